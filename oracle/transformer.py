"""CPU oracle for the serving step's model arithmetic: TEST INFRASTRUCTURE ONLY.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg may
import this module.  It shares no code with the GPU path.

The paper (Sec. II-A) describes LLM inference as two phases: prompt processing,
which runs the prompt tokens through the model, populates the key-value cache
and produces the first output token; and decode, which appends to the KV cache
and produces the remaining output tokens one at a time.  The paper does not
define the transformer itself; the readings used here (a Llama-style pre-norm
decoder) are:

* RMSNorm with gain, eps = 1e-5, before attention, before the MLP and after the
  last layer.
* Multi-head / grouped-query attention, head_dim = d_model / n_heads; query head
  j reads key/value head floor(j * n_kv_heads / n_heads).
* Rotary position embedding in the rotate-half pairing: dimension i is paired
  with i + head_dim/2 and rotated by angle pos * base^(-2i/head_dim); positions
  are 0-based per request.
* Scores scaled by 1/sqrt(head_dim), strict causal mask (key position <= query
  position), softmax with the maximum subtracted.
* SwiGLU MLP: down(silu(gate(h)) * up(h)), silu(z) = z / (1 + exp(-z)).
* No biases, untied LM head, greedy decoding with ties going to the lowest
  index, exactly out_len output tokens per request (no end-of-sequence token).

All arithmetic is float64 on the stored weight values.
"""
from __future__ import annotations

import numpy as np


class Model:
    """Weights as float64 arrays keyed by canonical tensor name."""

    def __init__(self, cfg: dict, weights: dict):
        self.L = int(cfg["n_layers"])
        self.d = int(cfg["d_model"])
        self.Hq = int(cfg["n_heads"])
        self.Hkv = int(cfg["n_kv_heads"])
        self.hd = self.d // self.Hq
        self.F = int(cfg["ffn_dim"])
        self.V = int(cfg["vocab"])
        self.base = float(cfg.get("rope_theta", 10000.0))
        self.eps = float(cfg.get("norm_eps", 1e-5))
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}

    def layer(self, i: int, name: str) -> np.ndarray:
        return self.w[f"layers.{i}.{name}"]


# ------------------------------------------------------------------ building blocks

def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_cos_sin(positions: np.ndarray, hd: int, base: float):
    """Angles pos * base^(-2i/hd) for i < hd/2, as (cos, sin) of shape [n, hd/2]."""
    i = np.arange(hd // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half RoPE on x of shape [n, heads, hd] at per-row positions."""
    hd = x.shape[-1]
    cos, sin = rope_cos_sin(positions, hd, base)
    cos, sin = cos[:, None, :], sin[:, None, :]
    a, b = x[..., : hd // 2], x[..., hd // 2:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    """exp(s - max) / sum over the last axis; -inf entries get weight 0."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q, k, v, q_pos, k_pos, n_kv_heads: int):
    """Causal attention.  q: [n, Hq, hd]; k, v: [t, Hkv, hd]; positions 1-D.

    Query row i may attend to key t iff k_pos[t] <= q_pos[i].
    """
    n, Hq, hd = q.shape
    group = Hq // n_kv_heads
    out = np.empty_like(q)
    allowed = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    scale = 1.0 / np.sqrt(hd)
    for j in range(Hq):
        g = j // group
        s = (q[:, j, :] @ k[:, g, :].T) * scale
        s = np.where(allowed, s, -np.inf)
        out[:, j, :] = softmax(s) @ v[:, g, :]
    return out


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


# ------------------------------------------------------------------ forward passes

class KVCache:
    """Post-RoPE keys and values of every processed position, per layer."""

    def __init__(self, m: Model):
        self.k = [np.zeros((0, m.Hkv, m.hd)) for _ in range(m.L)]
        self.v = [np.zeros((0, m.Hkv, m.hd)) for _ in range(m.L)]

    @property
    def length(self) -> int:
        return self.k[0].shape[0]


def forward(m: Model, tokens, cache: KVCache, logits_rows="last"):
    """Run tokens at positions cache.length, cache.length+1, ... through the model.

    Appends their keys and values to ``cache`` and returns the logits of the
    requested rows ("last" or "all") as a [rows, V] float64 array.
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    n = tokens.size
    start = cache.length
    pos = np.arange(start, start + n)
    x = m.w["embed"][tokens].copy()
    for i in range(m.L):
        h = rmsnorm(x, m.layer(i, "attn_norm"), m.eps)
        q = (h @ m.layer(i, "wq").T).reshape(n, m.Hq, m.hd)
        k = (h @ m.layer(i, "wk").T).reshape(n, m.Hkv, m.hd)
        v = (h @ m.layer(i, "wv").T).reshape(n, m.Hkv, m.hd)
        q = rope(q, pos, m.base)
        k = rope(k, pos, m.base)
        cache.k[i] = np.concatenate([cache.k[i], k], axis=0)
        cache.v[i] = np.concatenate([cache.v[i], v], axis=0)
        kpos = np.arange(cache.k[i].shape[0])
        o = attention(q, cache.k[i], cache.v[i], pos, kpos, m.Hkv)
        x = x + o.reshape(n, m.Hq * m.hd) @ m.layer(i, "wo").T
        h2 = rmsnorm(x, m.layer(i, "mlp_norm"), m.eps)
        a = silu(h2 @ m.layer(i, "wg").T) * (h2 @ m.layer(i, "wu").T)
        x = x + a @ m.layer(i, "wd").T
    rows = x[-1:] if logits_rows == "last" else x
    z = rmsnorm(rows, m.w["final_norm"], m.eps)
    return z @ m.w["lm_head"].T


def greedy(logits: np.ndarray) -> int:
    """Index of the largest logit; ties go to the lowest index."""
    return int(np.argmax(logits))


def generate(m: Model, prompt, out_len: int, forced=None):
    """Greedy generation with the KV cache.

    The prompt pass yields the first token; each following step feeds the
    previous output token (or ``forced[s-1]`` when teacher forcing) and yields
    the next.  The last output token is never fed back.  Returns (tokens
    int32 [out_len], logits float64 [out_len, V]).
    """
    cache = KVCache(m)
    toks = np.empty(out_len, dtype=np.int32)
    logits = np.empty((out_len, m.V))
    lg = forward(m, prompt, cache)[0]
    logits[0], toks[0] = lg, greedy(lg)
    for s in range(1, out_len):
        feed = toks[s - 1] if forced is None else forced[s - 1]
        lg = forward(m, [feed], cache)[0]
        logits[s], toks[s] = lg, greedy(lg)
    return toks, logits


def generate_recompute(m: Model, prompt, out_len: int):
    """Greedy generation that reprocesses the whole prefix at every step."""
    seq = list(np.asarray(prompt, dtype=np.int64))
    toks = np.empty(out_len, dtype=np.int32)
    logits = np.empty((out_len, m.V))
    for s in range(out_len):
        lg = forward(m, seq, KVCache(m))[0]
        logits[s], toks[s] = lg, greedy(lg)
        seq.append(int(toks[s]))
    return toks, logits


# ------------------------------------------------------------------ single-step views

def decode_step_batch(m: Model, caches, tokens):
    """One decode step over several independent requests (each with its own
    cache); returns logits [B, V].  Requests never see each other's state."""
    return np.stack([forward(m, [t], c)[0] for t, c in zip(tokens, caches)])
