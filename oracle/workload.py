"""Oracle of the workload generator's request model (Sec. III-B).

Test infrastructure: plain, slow Python that follows the paper's
description step by step; only the tests, the smoke check and the benchmark's
CPU baseline use it.

* Binning a parameter: at most B bins of about equal record counts; a
  parameter with at most B distinct values gets one bin per value.  With
  sorted values v and more distinct values than bins, bin j (j >= 1) starts
  at sorted position ceil(j n / B), so that distinct values give bins whose
  sizes differ by at most one; equal starting values merge.  Bins are the
  intervals between consecutive starting values (the last one closed at the
  largest value); a bin's value is its interval's centre.
* The joint model is the histogram of the tuples of bin indices of the
  records.
* A sample picks a tuple with probability proportional to its count and
  reports the centre of each interval.  The random draw is an input: a
  uniform u in [0, 1) selects record rank r = floor(u N), and the sample is
  the tuple (in lexicographic order) whose cumulative count first exceeds r.
"""
from __future__ import annotations

import math


def parameter_bins(values, max_bins: int):
    """(edges, centres) of one parameter: edges[i] is bin i's lower end,
    edges[-1] the largest value."""
    v = sorted(float(x) for x in values)
    n = len(v)
    distinct = []
    for x in v:
        if not distinct or x != distinct[-1]:
            distinct.append(x)
    if len(distinct) <= max_bins:
        return distinct + [distinct[-1]], list(distinct)
    starts = [v[0]]
    for j in range(1, max_bins):
        pos = -(-(j * n) // max_bins)  # ceil(j n / B)
        if v[pos] != starts[-1]:
            starts.append(v[pos])
    edges = starts + [v[-1]]
    centres = [(edges[i] + edges[i + 1]) / 2.0 for i in range(len(starts))]
    return edges, centres


def bin_index(edges, x: float) -> int:
    """The bin whose lower end is the largest one not above x."""
    nb = len(edges) - 1
    best = 0
    for i in range(nb):
        if edges[i] <= x:
            best = i
    return best


def fit(records, max_bins: int = 64):
    """The request model of a list of records (each a sequence of parameter
    values): per-parameter (edges, centres), the sorted non-empty joint bins
    with their counts, and each parameter's per-bin record counts."""
    n_params = len(records[0])
    params = [parameter_bins([r[p] for r in records], max_bins) for p in range(n_params)]
    counts = {}
    marginal = [[0] * len(c) for _, c in params]
    for r in records:
        key = tuple(bin_index(params[p][0], float(r[p])) for p in range(n_params))
        counts[key] = counts.get(key, 0) + 1
        for p in range(n_params):
            marginal[p][key[p]] += 1
    keys = sorted(counts)
    return {"params": params, "keys": keys, "counts": [counts[k] for k in keys], "marginal": marginal,
            "n_records": len(records)}


def _pick(counts, total: int, u: float) -> int:
    r = min(max(math.floor(u * total), 0), total - 1)
    acc = 0
    for i, c in enumerate(counts):
        acc += c
        if acc > r:
            return i
    raise AssertionError("counts do not sum to the total")


def sample(model, us):
    """One request (list of parameter values) and its joint-bin index per uniform."""
    out = []
    for u in us:
        b = _pick(model["counts"], model["n_records"], u)
        key = model["keys"][b]
        out.append(([model["params"][p][1][key[p]] for p in range(len(key))], b))
    return out


def sample_independent(model, us_rows):
    """Requests whose parameters are drawn from their own marginals, one
    uniform per parameter."""
    out = []
    for row in us_rows:
        vals = []
        for p, u in enumerate(row):
            b = _pick(model["marginal"][p], model["n_records"], u)
            vals.append(model["params"][p][1][b])
        out.append(vals)
    return out
