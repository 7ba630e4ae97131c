"""The workload generator's request model (Sec. III-B): the oracle pinned by a
hand-worked example and the properties the description fixes, then the
native model (C ABI) against the oracle, bit for bit."""
import json
import os

import numpy as np
import pytest

from oracle import workload as WG
from paper_2410_02425_amd import lp, synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "workload_example.json")


def golden():
    with open(GOLDEN) as f:
        return json.load(f)


# ------------------------------------------------------------------ oracle pins

def test_oracle_golden_example():
    g = golden()
    m = WG.fit(g["records"], g["max_bins"])
    e = g["expected"]
    assert [p[0] for p in m["params"]] == e["edges"]
    assert [p[1] for p in m["params"]] == e["centres"]
    assert m["marginal"] == e["counts"]
    assert [list(k) for k in m["keys"]] == e["joint_bins"] and m["counts"] == e["joint_counts"]
    got = WG.sample(m, e["samples"]["u"])
    assert [v for v, _ in got] == e["samples"]["values"] and [b for _, b in got] == e["samples"]["joint_bin"]
    assert WG.sample_independent(m, e["independent"]["u"]) == e["independent"]["values"]


@pytest.mark.parametrize("n,B", [(1000, 64), (1001, 64), (130, 64), (97, 7), (10, 3)])
def test_oracle_equal_frequency_bins_for_distinct_values(n, B):
    vals = np.random.default_rng(n).permutation(n) * 0.37 + 1.0
    edges, centres = WG.parameter_bins(vals, B)
    counts = [0] * len(centres)
    for x in vals:
        counts[WG.bin_index(edges, x)] += 1
    assert len(centres) == B and sum(counts) == n
    assert max(counts) - min(counts) <= 1 and min(counts) == n // B
    assert all(a < b for a, b in zip(edges[:-1], edges[1:-1]))  # strictly increasing lower ends
    assert all(edges[i] <= c <= edges[i + 1] for i, c in enumerate(centres))


def test_oracle_low_cardinality_gets_one_bin_per_value():
    vals = [3, 1, 2, 3, 3, 1]
    edges, centres = WG.parameter_bins(vals, 64)
    assert centres == [1.0, 2.0, 3.0]
    assert [WG.bin_index(edges, x) for x in vals] == [2, 0, 1, 2, 2, 0]


def test_oracle_heavy_ties_merge_bins():
    vals = [0.0] * 60 + list(np.linspace(0.1, 1.0, 40))
    edges, centres = WG.parameter_bins(vals, 10)
    assert edges[0] == 0.0 and edges[1] > 0.0  # the 60 zeros share one bin
    assert len(centres) < 10


def test_oracle_stratified_draws_reproduce_the_histogram():
    recs = synth.trace_records(3, 400)
    m = WG.fit(recs.tolist(), 16)
    N = m["n_records"]
    us = [(r + 0.5) / N for r in range(N)]  # one draw per record rank
    picks = [b for _, b in WG.sample(m, us)]
    assert np.bincount(picks, minlength=len(m["keys"])).tolist() == m["counts"]
    # every sample is a tuple that occurs in the records
    seen = {tuple(WG.bin_index(m["params"][p][0], r[p]) for p in range(recs.shape[1])) for r in recs}
    assert all(k in seen for k in m["keys"])


def test_oracle_independent_draws_reproduce_each_marginal():
    recs = synth.trace_records(4, 300)
    m = WG.fit(recs.tolist(), 8)
    N = m["n_records"]
    for p in range(recs.shape[1]):
        rows = [[0.5] * recs.shape[1] for _ in range(N)]
        for r in range(N):
            rows[r][p] = (r + 0.5) / N
        vals = [v[p] for v in WG.sample_independent(m, rows)]
        centres = m["params"][p][1]
        assert [vals.count(c) for c in centres] == m["marginal"][p]


# ------------------------------------------------------------------ native vs oracle

def test_native_golden_example():
    g = golden()
    m = lp.RequestModel(np.array(g["records"], dtype=np.float64), g["max_bins"])
    e = g["expected"]
    for p in range(2):
        edges, centres, counts = m.bins(p)
        assert edges.tolist() == e["edges"][p] and centres.tolist() == e["centres"][p]
        assert counts.tolist() == e["counts"][p]
    assert m.n_joint_bins() == len(e["joint_bins"])
    vals, jb = m.sample(e["samples"]["u"])
    assert vals.tolist() == e["samples"]["values"] and jb.tolist() == e["samples"]["joint_bin"]
    assert m.sample_independent(e["independent"]["u"]).tolist() == e["independent"]["values"]


@pytest.mark.parametrize("n,B,seed", [(3000, 64, 1), (2500, 8, 2), (700, 1, 3), (64, 64, 4)])
def test_native_matches_oracle(n, B, seed):
    recs = synth.trace_records(seed, n)
    nat = lp.RequestModel(recs, B)
    ora = WG.fit(recs.tolist(), B)
    for p in range(recs.shape[1]):
        edges, centres, counts = nat.bins(p)
        assert edges.tolist() == ora["params"][p][0]
        assert centres.tolist() == ora["params"][p][1]
        assert counts.tolist() == ora["marginal"][p]
    assert nat.n_joint_bins() == len(ora["keys"])
    rng = np.random.default_rng(seed)
    u = np.concatenate([rng.random(500), [0.0, np.nextafter(1.0, 0.0)]])
    vals, jb = nat.sample(u)
    exp = WG.sample(ora, u.tolist())
    assert vals.tolist() == [v for v, _ in exp] and jb.tolist() == [b for _, b in exp]
    ui = rng.random((200, recs.shape[1]))
    assert nat.sample_independent(ui).tolist() == WG.sample_independent(ora, ui.tolist())


def test_native_rejects_bad_input():
    with pytest.raises(lp.LPError):
        lp.RequestModel(np.array([[1.0, np.nan]]))
    m = lp.RequestModel(np.array([[1.0], [2.0]]))
    with pytest.raises(lp.LPError):
        m.sample([1.0])
    with pytest.raises(lp.LPError):
        m.sample([-0.1])
