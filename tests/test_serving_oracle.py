"""Pins for the scheduling and latency-accounting oracle: hand-worked golden
cases from the paper's definitions plus invariants and a brute-force check."""
import json
import os

import numpy as np
import pytest

from oracle import serving as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_latency_golden_example():
    g = load("latency_example.json")
    arr = {r["id"]: r["arrival_ns"] for r in g["requests"]}
    toks = {r["id"]: r["token_ns"] for r in g["requests"]}
    ins = {r["id"]: r["in_len"] for r in g["requests"]}
    for r in g["requests"]:
        ttft, itl, e2e = S.request_latencies(r["arrival_ns"], r["token_ns"])
        exp = g["expected"]["per_request"][str(r["id"])]
        assert (ttft, itl, e2e) == (exp["ttft"], exp["itl"], exp["e2e"])
        assert ttft / r["in_len"] == exp["nttft"]
    s = S.summarize(arr, toks, ins)
    for k in ("ttft_p50_ns", "nttft_p50_ns", "itl_p50_ns", "output_tokens", "e2e_p50_ns", "ttft_p90_ns",
              "itl_p90_ns", "itl_p99_ns", "n_requests", "itl_count"):
        assert s[k] == g["expected"][k]
    assert s["throughput_tok_s"] == pytest.approx(g["expected"]["throughput_tok_s"], rel=1e-12)


def test_e2e_equals_ttft_plus_itl_sum():
    rng = np.random.default_rng(0)
    for _ in range(100):
        arrival = int(rng.integers(0, 10**9))
        times = np.cumsum(rng.integers(1, 10**8, size=int(rng.integers(1, 50)))) + arrival
        ttft, itl, e2e = S.request_latencies(arrival, times)
        assert e2e == ttft + sum(itl) and len(itl) == len(times) - 1


def test_median_convention():
    assert S.median([3, 1, 2]) == 2.0
    assert S.median([4, 1, 3, 2]) == 2.5
    assert S.median([7]) == 7.0


def fake_step(kind, n_rows, n_tokens, sum_ctx):
    return 10 + n_tokens if kind == "prefill" else 5 + n_rows


@pytest.mark.parametrize("case", [0, 1])
def test_schedule_golden(case):
    g = load("schedule_example.json")
    reqs = [S.SimRequest(i, a, b) for i, a, b in g["requests"]]
    c = g["cases"][case]
    tr = S.simulate(reqs, g["max_batch"], c["max_batch_weight"], g["max_prefill_tokens"],
                    True, g["concurrency"], fake_step)
    got = [[st.kind, st.ids, st.slots, st.end_ns] for st in tr.steps]
    assert got == c["steps"]
    assert {str(k): v for k, v in tr.arrival_ns.items()} == c["arrival_ns"]
    assert {str(k): v for k, v in tr.token_ns.items()} == c["token_ns"]


def random_requests(rng, n, open_loop=False):
    t = 0
    out = []
    for i in range(n):
        t += int(rng.integers(0, 40))
        out.append(S.SimRequest(i, int(rng.integers(1, 30)), int(rng.integers(1, 12)), t if open_loop else 0))
    return out


@pytest.mark.parametrize("open_loop", [False, True])
def test_schedule_invariants(open_loop):
    rng = np.random.default_rng(11)
    for trial in range(30):
        reqs = random_requests(rng, 25, open_loop)
        mb, W, P = int(rng.integers(1, 6)), int(rng.integers(45, 120)), int(rng.integers(30, 90))
        tr = S.simulate(reqs, mb, W, P, not open_loop, int(rng.integers(1, 8)), fake_step)
        by_id = {r.id: r for r in reqs}
        # every request gets exactly out_len tokens, first from a prefill step
        for r in reqs:
            assert len(tr.token_ns[r.id]) == r.out_len
            assert tr.token_ns[r.id][0] >= tr.arrival_ns[r.id]
        active = {}
        admitted_order = []
        for st in tr.steps:
            if st.kind == "prefill":
                assert sum(by_id[i].in_len for i in st.ids) <= P
                for i, s in zip(st.ids, st.slots):
                    assert s not in active.values()
                    active[i] = s
                    admitted_order.append(i)
            assert len(active) <= mb
            assert sum(by_id[i].in_len + by_id[i].out_len for i in active) <= W
            emitted = {i: sum(1 for s2 in tr.steps[: tr.steps.index(st) + 1] if i in s2.ids) for i in active}
            for i in list(active):
                if emitted[i] == by_id[i].out_len:
                    del active[i]
        # strict FCFS: admission order is sorted by (arrival, id)
        assert admitted_order == sorted(admitted_order, key=lambda i: (tr.arrival_ns[i], i))


def brute_force_schedule(reqs, mb, W, P, U):
    """Closed-loop schedule by direct per-tick state evolution (independent
    re-derivation of the policy with explicit per-request counters)."""
    arrival = {r.id: 0 for r in reqs[:U]}
    queue = [r.id for r in reqs[:U]]
    nxt = U
    state = {}   # id -> [slot, emitted]
    weight = 0
    t = 0
    out = []
    L = {r.id: r for r in reqs}
    while len(out) < 10_000 and (queue or state):
        adm = []
        tok = 0
        for i in list(queue):
            r = L[i]
            if len(state) + len(adm) >= mb or weight + r.in_len + r.out_len > W or tok + r.in_len > P:
                break
            adm.append(i); tok += r.in_len; weight += r.in_len + r.out_len; queue.remove(i)
        done_t = []
        if adm:
            used = {v[0] for v in state.values()}
            slots = []
            for i in adm:
                s = 0
                while s in used:
                    s += 1
                used.add(s); slots.append(s); state[i] = [s, 1]
            t += 10 + tok
            out.append(("prefill", adm, slots, t))
            for i in adm:
                if L[i].out_len == 1:
                    del state[i]; weight -= L[i].in_len + L[i].out_len; done_t.append(t)
        rows = sorted((v[0], i) for i, v in state.items() if v[1] < L[i].out_len)
        if rows:
            t += 5 + len(rows)
            out.append(("decode", [i for _, i in rows], [s for s, _ in rows], t))
            for _, i in rows:
                state[i][1] += 1
            for _, i in rows:
                if state[i][1] == L[i].out_len:
                    del state[i]; weight -= L[i].in_len + L[i].out_len; done_t.append(t)
        for tt in done_t:
            if nxt < len(reqs):
                arrival[reqs[nxt].id] = tt; queue.append(reqs[nxt].id); nxt += 1
    return out


def test_schedule_matches_brute_force_closed_loop():
    rng = np.random.default_rng(5)
    for trial in range(40):
        reqs = random_requests(rng, 20)
        mb, W, P, U = int(rng.integers(1, 5)), int(rng.integers(45, 100)), int(rng.integers(30, 80)), int(rng.integers(1, 7))
        tr = S.simulate(reqs, mb, W, P, True, U, fake_step)
        got = [(st.kind, st.ids, st.slots, st.end_ns) for st in tr.steps]
        assert got == brute_force_schedule(reqs, mb, W, P, U)


def test_replay_reproduces_schedule():
    rng = np.random.default_rng(9)
    reqs = random_requests(rng, 30, open_loop=True)
    tr = S.simulate(reqs, 3, 80, 60, False, 0, fake_step)
    tr2 = S.simulate(reqs, 3, 80, 60, False, 0, [st.end_ns for st in tr.steps])
    assert [(s.kind, s.ids, s.end_ns) for s in tr2.steps] == [(s.kind, s.ids, s.end_ns) for s in tr.steps]
