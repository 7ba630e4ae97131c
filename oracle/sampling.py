"""Oracle of next-token sampling under per-request parameters (temperature,
top-k, top-p), the decoding parameters carried by requests (Sec. III-A).

Test infrastructure: plain, slow Python; only the tests use it.

Definitions (the readings the engine implements):
* temperature <= 0 or top_p <= 0: greedy, the lowest index among the maxima;
* candidates: every token, or for 0 < top_k < V the tokens whose logit is at
  least the top_k-th largest logit (counting repeats), ties included;
* weight of a candidate: q = floor(exp((logit - max) / temperature) * 2^40);
* top_p < 1: with Z the candidates' total weight and
  need = ceil(Z * floor(top_p * 2^24) / 2^24), the kept candidates are those
  with q >= t, where t is the largest weight whose heavier-or-equal
  candidates sum to at least need;
* the draw: r = floor(Z_kept * u24 / 2^24) for a 24-bit uniform integer u24;
  the token is the kept candidate, in vocabulary order, whose cumulative
  weight interval [sum of earlier kept weights, + q) holds r.
Weights here use float64 exp; the kernel computes them in float32.
"""
from __future__ import annotations

import math

import numpy as np

SCALE = 1 << 40
PHILOX_WORD3 = 0x53414D50


def weights(logits, temperature: float, top_k: int):
    """(candidate mask, integer weights q) of one row."""
    l = [float(x) for x in logits]
    V = len(l)
    m = max(l)
    if 0 < top_k < V:
        kth = sorted(l, reverse=True)[top_k - 1]
        cand = [x >= kth for x in l]
    else:
        cand = [True] * V
    q = [int(math.floor(math.exp((x - m) / temperature) * SCALE)) if c else 0 for x, c in zip(l, cand)]
    return cand, q


def nucleus(cand, q, top_p: float):
    """(kept mask, kept total, threshold t) for top_p given as a float32 value."""
    Z = sum(qq for qq, c in zip(q, cand) if c)
    p32 = float(np.float32(top_p))
    if p32 >= 1.0:
        return list(cand), Z, 0
    pfix = max(1, int(math.floor(p32 * (1 << 24))))
    need = -(-(Z * pfix) // (1 << 24))
    # walk the candidates' weights from the heaviest down, a value (with all
    # its repeats) at a time, until their sum reaches need
    vals = sorted((qq for qq, c in zip(q, cand) if c), reverse=True)
    acc, t, i = 0, None, 0
    while i < len(vals):
        v = vals[i]
        while i < len(vals) and vals[i] == v:
            acc += v
            i += 1
        if acc >= need:
            t = v
            break
    keep = [c and qq >= t for qq, c in zip(q, cand)]
    return keep, sum(qq for qq, k in zip(q, keep) if k), t


def choose(logits, temperature: float, top_k: int, top_p: float, u24: int):
    """The chosen token and, for sampled rows, the details of the draw:
    (token, kept mask, weights, kept total, r)."""
    l = [float(x) for x in logits]
    greedy = max(range(len(l)), key=lambda i: (l[i], -i))
    if temperature <= 0 or float(np.float32(top_p)) <= 0 or len(l) == 1:
        return greedy, None
    cand, q = weights(l, temperature, top_k)
    keep, zk, _ = nucleus(cand, q, top_p)
    r = (zk * u24) >> 24
    acc = 0
    for i, (k, qq) in enumerate(zip(keep, q)):
        if k:
            if r < acc + qq:
                return i, (keep, q, zk, r)
            acc += qq
    raise AssertionError("r beyond the kept weight")


def draw_u24(key, counter) -> int:
    """24-bit uniform of a draw: the first Philox4x32-10 output word for the
    row's key and counter (fourth counter word PHILOX_WORD3), shifted right
    by 8."""
    from paper_2410_02425_amd import synth  # the shared seeded generator
    w = synth.philox4x32_10(counter[0], counter[1], counter[2], PHILOX_WORD3, key[0], key[1])[0]
    return int(np.asarray(w).reshape(-1)[0]) >> 8
