"""Seeded synthetic inputs shared by the GPU path, the oracle and the tests.

This module holds input generation only, none of the serving step's arithmetic:
model shapes, random weights, prompt token ids, request lengths and arrival
times.  The paper's inputs (trained LLM weights, the production-trace-derived
request generator of Sec. III-B, its prompt corpus) are not available, so the
workloads here are seeded stand-ins with the shapes and length ranges the paper
describes (Table II: input 1-4093 tokens, output 1-1500 tokens).

Weights are drawn with a counter-based generator so that any single element can
be produced on its own (the oracle needs a few rows of a 16 GB model) and so
that the device can generate the same values in HBM:

* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy
  as 1, 2, 3", SC'11): counter = (element index low word, element index high
  word, tensor id, 0), key = two 32-bit words derived from the seed.
* The 128 output bits give twelve 10-bit uniforms (bits 0-29 of each word);
  their sum S (Irwin-Hall with n = 12) has mean 6138 and variance 1024^2 - 1,
  so (S - 6138) / 1024 is approximately N(0, 1).  The fp32 value is
  ``fl(fl(S - 6138) * fl(std)) * 2**-10``: one correctly rounded product and an
  exact power-of-two scaling, so every IEEE implementation gets the same bits.
* bf16 models round that fp32 value to nearest-even once.
"""
from __future__ import annotations

import dataclasses
import numpy as np

# ---------------------------------------------------------------- model shapes

DTYPE_F32 = 0
DTYPE_BF16 = 1


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    ffn_dim: int
    vocab: int
    dtype: int = DTYPE_BF16
    rope_theta: float = 10000.0
    norm_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def with_layers(self, n_layers: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n_layers, name=f"{self.name}-L{n_layers}")

    def n_params(self) -> int:
        d, hd, F, V = self.d_model, self.head_dim, self.ffn_dim, self.vocab
        per_layer = (2 * d + d * (self.n_heads + 2 * self.n_kv_heads) * hd
                     + self.n_heads * hd * d + 3 * d * F)
        return V * d + self.n_layers * per_layer + d + V * d


@dataclasses.dataclass(frozen=True)
class Workload:
    """A seeded request stream: lengths, prompts and arrivals."""
    name: str
    base_seed: int
    n_requests: int
    max_batch: int
    in_range: tuple          # (lo, hi) clip of input lengths
    out_range: tuple         # (lo, hi) clip of output lengths
    in_lognormal: tuple = (6.0, 0.8)     # (mu, sigma); None for fixed lengths
    out_lognormal: tuple = (5.0, 0.7)
    fixed_in: int = 0
    fixed_out: int = 0
    mode: str = "closed"     # "closed" (fixed batch of users) or "open" (Poisson)
    rate_per_s: float = 0.0  # open-loop arrival rate


SHAPES = {
    "tiny": ModelShape("tiny", 2, 256, 4, 4, 688, 1024, dtype=DTYPE_F32),
    "7b": ModelShape("7b", 32, 4096, 32, 32, 11008, 32000),
    "13b": ModelShape("13b", 40, 5120, 40, 40, 13824, 32000),
    "8b": ModelShape("8b", 32, 4096, 32, 8, 14336, 128256),
    "70b": ModelShape("70b", 80, 8192, 64, 8, 28672, 128256),
}

WORKLOADS = {
    "tiny": Workload("tiny", 0, 4, 4, (32, 32), (16, 16), None, None, 32, 16),
    "7b": Workload("7b", 7, 64, 16, (16, 2048), (8, 512)),
    "13b": Workload("13b", 13, 128, 32, (16, 2048), (8, 512)),
    "8b": Workload("8b", 8, 256, 64, (16, 4096), (8, 1024)),
    "8b-poisson": Workload("8b-poisson", 8, 1200, 64, (16, 4096), (8, 1024),
                           mode="open", rate_per_s=20.0),
    "70b": Workload("70b", 70, 128, 32, (16, 4096), (8, 512)),
}

# canonical tensor order inside one layer (tensor id = 1 + 9 * layer + index)
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")


def tensor_shapes(shape: ModelShape):
    """Canonical (name, tensor id, (rows, cols)) list; matrices are [out x in]."""
    d, hd, F, V = shape.d_model, shape.head_dim, shape.ffn_dim, shape.vocab
    Hq, Hkv = shape.n_heads, shape.n_kv_heads
    dims = {"attn_norm": (1, d), "wq": (Hq * hd, d), "wk": (Hkv * hd, d), "wv": (Hkv * hd, d),
            "wo": (d, Hq * hd), "mlp_norm": (1, d), "wg": (F, d), "wu": (F, d), "wd": (d, F)}
    out = [("embed", 0, (V, d))]
    for layer in range(shape.n_layers):
        for j, nm in enumerate(LAYER_TENSORS):
            out.append((f"layers.{layer}.{nm}", 1 + 9 * layer + j, dims[nm]))
    out.append(("final_norm", 1 + 9 * shape.n_layers, (1, d)))
    out.append(("lm_head", 2 + 9 * shape.n_layers, (V, d)))
    return out


def is_gain(name: str) -> bool:
    return name.endswith("norm")


# ---------------------------------------------------------------- Philox4x32-10

_MASK32 = np.uint64(0xFFFFFFFF)
_PHILOX_M0 = np.uint64(0xD2511F53)
_PHILOX_M1 = np.uint64(0xCD9E8D57)
_PHILOX_W0 = 0x9E3779B9
_PHILOX_W1 = 0xBB67AE85


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Ten Philox-4x32 rounds on uint32 counter words (broadcastable arrays).

    Each round multiplies words 0 and 2 by the two Philox constants, keeps the
    64-bit products' high and low halves, and permutes them with the key; the
    key is bumped by the Weyl constants before every round but the first.
    Returns four uint32 arrays.
    """
    c = [np.asarray(x, dtype=np.uint64) & _MASK32 for x in (c0, c1, c2, c3)]
    c = [np.ascontiguousarray(x) for x in np.broadcast_arrays(*c)]
    k0 &= 0xFFFFFFFF
    k1 &= 0xFFFFFFFF
    sh = np.uint64(32)
    for r in range(10):
        if r:
            k0 = (k0 + _PHILOX_W0) & 0xFFFFFFFF
            k1 = (k1 + _PHILOX_W1) & 0xFFFFFFFF
        p0 = c[0] * _PHILOX_M0
        p1 = c[2] * _PHILOX_M1
        n0 = p1 >> sh
        n0 ^= c[1]
        n0 ^= np.uint64(k0)
        n2 = p0 >> sh
        n2 ^= c[3]
        n2 ^= np.uint64(k1)
        p1 &= _MASK32
        p0 &= _MASK32
        c = [n0, p1, n2, p0]
    return [x.astype(np.uint32) for x in c]


def seed_key(seed: int):
    """Split a 64-bit seed into the two Philox key words."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & 0xFFFFFFFF, seed >> 32


_CHUNK = 1 << 16


def _normal_chunk(idx: np.ndarray, tensor_id: int, k0: int, k1: int, std: float) -> np.ndarray:
    c = philox4x32_10(idx & _MASK32, idx >> np.uint64(32), np.uint64(tensor_id), 0, k0, k1)
    s = np.zeros(idx.shape, dtype=np.int64)
    for word in c:
        word = word.astype(np.int64)
        s += (word & 1023) + ((word >> 10) & 1023) + ((word >> 20) & 1023)
    k = (s - 6138).astype(np.float32)
    return (k * np.float32(std)) * np.float32(2.0 ** -10)


def normal_f32(seed: int, tensor_id: int, index, std: float) -> np.ndarray:
    """Approximately N(0, std^2) fp32 values for element indices ``index``.

    Large requests are split into cache-sized chunks spread over threads (the
    values do not depend on the split)."""
    idx = np.asarray(index, dtype=np.uint64)
    k0, k1 = seed_key(seed)
    flat = idx.reshape(-1)
    if flat.size <= _CHUNK:
        return _normal_chunk(flat, tensor_id, k0, k1, std).reshape(idx.shape)
    out = np.empty(flat.size, dtype=np.float32)
    starts = range(0, flat.size, _CHUNK)

    def work(a):
        out[a:a + _CHUNK] = _normal_chunk(flat[a:a + _CHUNK], tensor_id, k0, k1, std)

    import concurrent.futures as cf
    import os
    with cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(work, starts))
    return out.reshape(idx.shape)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest-even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_model_dtype(x_f32: np.ndarray, dtype: int) -> np.ndarray:
    """Values the model stores, as fp32 (bf16 models round once)."""
    if dtype == DTYPE_BF16:
        return bf16_bits_to_f32(f32_to_bf16_bits(x_f32))
    return np.asarray(x_f32, dtype=np.float32)


def tensor_values(seed: int, tensor_id: int, rows, n_cols: int, std: float,
                  dtype: int, gain_std: float = 0.0, gain: bool = False) -> np.ndarray:
    """Stored values (as fp32) of the listed rows of one canonical tensor.

    Element (r, c) has index r * n_cols + c.  Gains are 1.0 unless ``gain_std``
    is set, in which case they are 1 + N(0, gain_std^2) (used by tests so that
    a dropped gain multiplication is visible).
    """
    rows = np.atleast_1d(np.asarray(rows, dtype=np.int64))
    if gain:
        if gain_std == 0.0:
            return np.ones((rows.size, n_cols), dtype=np.float32)
        idx = rows[:, None].astype(np.uint64) * np.uint64(n_cols) + np.arange(n_cols, dtype=np.uint64)
        v = np.float32(1.0) + normal_f32(seed, tensor_id, idx, gain_std)
        return round_to_model_dtype(v, dtype)
    idx = rows[:, None].astype(np.uint64) * np.uint64(n_cols) + np.arange(n_cols, dtype=np.uint64)
    return round_to_model_dtype(normal_f32(seed, tensor_id, idx, std), dtype)


def model_weights(shape: ModelShape, seed: int, std: float = 0.02, gain_std: float = 0.0):
    """All canonical tensors as fp32 arrays holding the stored values."""
    out = {}
    for name, tid, (r, c) in tensor_shapes(shape):
        out[name] = tensor_values(seed, tid, np.arange(r), c, std, shape.dtype,
                                  gain_std=gain_std, gain=is_gain(name))
        if r == 1:
            out[name] = out[name].reshape(c)
    return out


def weights_blob(shape: ModelShape, weights: dict) -> bytes:
    """Concatenate tensors in canonical order in the model dtype."""
    parts = []
    for name, _, _ in tensor_shapes(shape):
        a = np.ascontiguousarray(weights[name], dtype=np.float32).reshape(-1)
        if shape.dtype == DTYPE_BF16:
            parts.append(f32_to_bf16_bits(a).tobytes())
        else:
            parts.append(a.tobytes())
    return b"".join(parts)


# ---------------------------------------------------------------- requests

@dataclasses.dataclass
class Request:
    id: int
    prompt: np.ndarray       # int32 [in_len]
    out_len: int
    arrival_ns: int = 0

    @property
    def in_len(self) -> int:
        return int(self.prompt.size)


def workload_seeds(base_seed: int):
    """[weights key, lengths rng, prompts rng, arrivals rng] from one base seed."""
    ss = np.random.SeedSequence(base_seed).spawn(4)
    w = ss[0].generate_state(2, dtype=np.uint32)
    key = int(w[0]) | (int(w[1]) << 32)
    return key, np.random.default_rng(ss[1]), np.random.default_rng(ss[2]), np.random.default_rng(ss[3])


def _lengths(rng, n, lognormal, clip, fixed):
    if lognormal is None:
        return np.full(n, fixed, dtype=np.int32)
    mu, sigma = lognormal
    v = np.rint(np.exp(rng.normal(mu, sigma, size=n)))
    return np.clip(v, clip[0], clip[1]).astype(np.int32)


def make_requests(wl: Workload, vocab: int, n_requests: int | None = None):
    """Seeded request list; lengths are drawn independently (the configs do not
    correlate input and output lengths)."""
    n = wl.n_requests if n_requests is None else n_requests
    # the stream holds the workload's own count; asking for more extends it
    # (the first wl.n_requests requests then differ from the stock ones)
    m = max(n, wl.n_requests)
    _, rl, rp, ra = workload_seeds(wl.base_seed)
    ins = _lengths(rl, m, wl.in_lognormal, wl.in_range, wl.fixed_in)[:n]
    outs = _lengths(rl, m, wl.out_lognormal, wl.out_range, wl.fixed_out)[:n]
    arrivals = np.zeros(n, dtype=np.int64)
    if wl.mode == "open":
        gaps = ra.exponential(1.0 / wl.rate_per_s, size=m)[:n]
        arrivals = np.rint(np.cumsum(gaps) * 1e9).astype(np.int64)
    reqs = []
    for i in range(n):
        prompt = rp.integers(0, vocab, size=int(ins[i]), dtype=np.int32)
        reqs.append(Request(i, prompt, int(outs[i]), int(arrivals[i])))
    return reqs


def uniform_f32(rng: np.random.Generator, shape, lo=-1.0, hi=1.0) -> np.ndarray:
    return rng.uniform(lo, hi, size=shape).astype(np.float32)


# ---------------------------------------------------------------- trace stand-in

# Columns of a synthetic trace record: the request parameters the paper finds
# matter most for latency (Sec. III-A): token counts, the number of prompts in
# the request, and the sampling parameters.
TRACE_COLUMNS = ("in_tokens", "out_tokens", "batch_size", "sampling", "temperature", "top_k")

# Rank correlation of the latent normals (Gaussian copula) behind the columns.
# The production traces are unavailable; the paper reports that input tokens,
# output tokens and batch size are strongly correlated with one another
# (Sec. III-A).  These values are a stand-in with that structure.
TRACE_CORRELATION = np.array([
    # in    out   batch  samp  temp  topk
    [1.00, 0.45, -0.50, 0.10, 0.00, 0.00],
    [0.45, 1.00, -0.35, 0.30, 0.00, 0.00],
    [-0.50, -0.35, 1.00, 0.00, 0.00, 0.00],
    [0.10, 0.30, 0.00, 1.00, 0.00, 0.00],
    [0.00, 0.00, 0.00, 0.00, 1.00, 0.50],
    [0.00, 0.00, 0.00, 0.00, 0.50, 1.00],
])


def trace_records(seed: int, n: int) -> np.ndarray:
    """n synthetic trace requests [n x 6] (TRACE_COLUMNS), seeded: input
    tokens lognormal(6.0, 0.9) in [1, 4093], output tokens lognormal(4.8, 0.9)
    in [1, 1500] (the ranges of the paper's Table II), batch size 1..5 (79%
    single prompts), greedy or sampling decoding (38% sampling), and for
    sampling requests a temperature in [0.05, 1.5] (two decimals) and top-k
    in {5, 10, 20, 40, 50, 100} (0 and 0 for greedy)."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((n, 6)) @ np.linalg.cholesky(TRACE_CORRELATION).T
    inp = np.clip(np.rint(np.exp(6.0 + 0.9 * z[:, 0])), 1, 4093)
    out = np.clip(np.rint(np.exp(4.8 + 0.9 * z[:, 1])), 1, 1500)
    batch = 1.0 + (z[:, 2] > 0.8) + (z[:, 2] > 1.4) + (z[:, 2] > 1.9) + (z[:, 2] > 2.3)
    sampling = (z[:, 3] > 0.3).astype(np.float64)
    temp = np.where(sampling > 0, np.round(np.clip(0.7 + 0.25 * z[:, 4], 0.05, 1.5), 2), 0.0)
    topk = np.where(sampling > 0, np.array([5, 10, 20, 40, 50, 100.0])[np.digitize(z[:, 5], [-1, -0.3, 0.3, 1, 1.6])],
                    0.0)
    return np.stack([inp, out, batch, sampling, temp, topk], axis=1)
