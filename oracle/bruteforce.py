"""Pure-Python brute-force transformer for tiny dimensions: TEST INFRASTRUCTURE ONLY.

An independent formulation used to pin the vectorised oracle in
``oracle/transformer.py``: explicit loops, Python floats, and RoPE written as a
complex multiplication (the pair (x_i, x_{i+hd/2}) is the complex number
x_i + i*x_{i+hd/2}, rotated by exp(i * pos * base^(-2i/hd))).  Keys and values
are recomputed for the whole prefix on every call (no cache).  It follows the
same readings of the paper's prompt-processing/decode description (Sec. II-A)
as the vectorised oracle.
"""
from __future__ import annotations

import cmath
import math


def _matvec(w, x):
    return [sum(w[r][c] * x[c] for c in range(len(x))) for r in range(len(w))]


def _norm(x, g, eps):
    ms = sum(v * v for v in x) / len(x)
    s = 1.0 / math.sqrt(ms + eps)
    return [x[i] * s * g[i] for i in range(len(x))]


def _rope(vec, pos, base):
    hd = len(vec)
    half = hd // 2
    out = [0.0] * hd
    for i in range(half):
        z = complex(vec[i], vec[i + half]) * cmath.exp(1j * pos * base ** (-2.0 * i / hd))
        out[i], out[i + half] = z.real, z.imag
    return out


def logits_all_positions(cfg, w, tokens):
    """Logits after every position of ``tokens`` (list of ints), by loops."""
    L, d, Hq, Hkv, V = cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["vocab"]
    hd = d // Hq
    base, eps = cfg.get("rope_theta", 10000.0), cfg.get("norm_eps", 1e-5)
    tl = lambda a: [list(map(float, row)) for row in a]
    n = len(tokens)
    xs = [list(map(float, w["embed"][t])) for t in tokens]
    for layer in range(L):
        lw = lambda nm: w[f"layers.{layer}.{nm}"]
        g_att, g_mlp = list(map(float, lw("attn_norm"))), list(map(float, lw("mlp_norm")))
        wq, wk, wv, wo = tl(lw("wq")), tl(lw("wk")), tl(lw("wv")), tl(lw("wo"))
        wg, wu, wd = tl(lw("wg")), tl(lw("wu")), tl(lw("wd"))
        hs = [_norm(x, g_att, eps) for x in xs]
        qs = [_matvec(wq, h) for h in hs]
        ks = [_matvec(wk, h) for h in hs]
        vs = [_matvec(wv, h) for h in hs]
        new_xs = []
        for i in range(n):
            attn = []
            for j in range(Hq):
                g = (j * Hkv) // Hq
                qj = _rope(qs[i][j * hd:(j + 1) * hd], i, base)
                scores = []
                for t in range(i + 1):
                    kt = _rope(ks[t][g * hd:(g + 1) * hd], t, base)
                    scores.append(sum(qj[c] * kt[c] for c in range(hd)) / math.sqrt(hd))
                mx = max(scores)
                ex = [math.exp(s - mx) for s in scores]
                tot = sum(ex)
                o = [0.0] * hd
                for t in range(i + 1):
                    for c in range(hd):
                        o[c] += ex[t] / tot * vs[t][g * hd + c]
                attn.extend(o)
            x1 = [xs[i][c] + v for c, v in enumerate(_matvec(wo, attn))]
            h2 = _norm(x1, g_mlp, eps)
            gate, up = _matvec(wg, h2), _matvec(wu, h2)
            act = [gate[f] / (1.0 + math.exp(-gate[f])) * up[f] for f in range(len(gate))]
            new_xs.append([x1[c] + v for c, v in enumerate(_matvec(wd, act))])
        xs = new_xs
    gf = list(map(float, w["final_norm"]))
    lm = tl(w["lm_head"])
    return [_matvec(lm, _norm(x, gf, eps)) for x in xs]


def greedy(logits):
    best = 0
    for i in range(1, len(logits)):
        if logits[i] > logits[best]:
            best = i
    return best
