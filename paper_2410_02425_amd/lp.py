"""ctypes binding of the C ABI in include/lp.h and include/lp_ops.h.

Argument marshalling only: every step of the serving path runs inside
liblp.so.  PyTorch provides the device arena and the stream.  Loading fails
loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblp.so")

LP_OK, LP_EINVAL, LP_ENOMEM, LP_EHIP, LP_ESTATE = 0, -1, -2, -3, -4
LP_F32, LP_BF16, LP_F16 = 0, 1, 2
LP_OPEN_LOOP, LP_CLOSED_LOOP = 0, 1
LP_FLAG_KEEP_LOGITS, LP_FLAG_TIME_KERNEL, LP_FLAG_BF16_ACTIVATIONS, LP_FLAG_SEPARATE_QKV_FINISH = 1, 2, 4, 8

EXPORTED = [
    "lp_arena_bytes_required", "lp_engine_create", "lp_load_weights", "lp_init_weights_random",
    "lp_query_max_batch_weight", "lp_submit", "lp_set_forced_tokens", "lp_set_sampling", "lp_run", "lp_get_result",
    "lp_get_token_times", "lp_get_run_stats", "lp_get_step_log", "lp_get_logits", "lp_last_error",
    "lp_engine_destroy", "lp_sched_simulate", "lp_summarize_latencies", "lp_get_latency_summary",
    "lp_wg_fit", "lp_wg_info", "lp_wg_bins", "lp_wg_sample", "lp_wg_sample_independent", "lp_wg_free",
    "lp_op_gemm", "lp_op_gemm_plan", "lp_op_packed_weight_bytes", "lp_op_pack_weight", "lp_op_rmsnorm", "lp_op_decode_attention_ws_bytes", "lp_op_decode_attention",
    "lp_op_decode_attention_noalloc",
    "lp_op_prefill_attention", "lp_op_argmax", "lp_op_init_weight", "lp_op_sample",
]


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("ffn_dim", C.c_int32), ("vocab", C.c_int32),
                ("rope_theta", C.c_float), ("norm_eps", C.c_float), ("dtype", C.c_int32)]


class EngineOptions(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("max_seq_len", C.c_int32), ("max_batch_weight", C.c_int64),
                ("max_prefill_tokens", C.c_int64), ("hbm_reserve_bytes", C.c_int64), ("flags", C.c_uint32)]


class Request(C.Structure):
    _fields_ = [("id", C.c_int64), ("prompt", C.POINTER(C.c_int32)), ("in_len", C.c_int32),
                ("out_len", C.c_int32), ("arrival_ns", C.c_int64)]


class StepRecord(C.Structure):
    _fields_ = [("kind", C.c_int32), ("n_rows", C.c_int32), ("n_tokens", C.c_int64), ("sum_ctx", C.c_int64),
                ("plan_ns", C.c_int64), ("end_ns", C.c_int64)]


class RunStats(C.Structure):
    _fields_ = [("n_steps", C.c_int64), ("n_prefill_steps", C.c_int64), ("n_decode_steps", C.c_int64),
                ("output_tokens", C.c_int64), ("prompt_tokens", C.c_int64), ("wall_ns", C.c_int64),
                ("decode_ns", C.c_int64), ("decode_tokens", C.c_int64), ("full_decode_steps", C.c_int64),
                ("full_decode_ns", C.c_int64), ("full_decode_sum_ctx", C.c_int64),
                ("timed_kernel_launches", C.c_int64), ("timed_kernel_rows", C.c_int64),
                ("timed_kernel_ms", C.c_double)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class SampleParams(C.Structure):
    _fields_ = [("temperature", C.c_float), ("top_k", C.c_int32), ("top_p", C.c_float),
                ("key", C.c_uint32 * 2), ("counter", C.c_uint32 * 3)]


class LatencySummary(C.Structure):
    _fields_ = [("n_requests", C.c_int64), ("output_tokens", C.c_int64), ("itl_count", C.c_int64),
                ("ttft_p50_ns", C.c_double), ("nttft_p50_ns", C.c_double), ("itl_p50_ns", C.c_double),
                ("e2e_p50_ns", C.c_double), ("ttft_p90_ns", C.c_double), ("itl_p90_ns", C.c_double),
                ("itl_p99_ns", C.c_double), ("throughput_tok_s", C.c_double)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def lib():
    """The loaded liblp.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with paper_2410_02425_amd/build.py")
        L = C.CDLL(_LIB_PATH)
        vp, i32, i64, f32, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_size_t
        P = C.POINTER
        sig = {
            "lp_arena_bytes_required": [P(ModelConfig), P(EngineOptions), P(sz)],
            "lp_engine_create": [P(ModelConfig), P(EngineOptions), vp, sz, vp, P(vp)],
            "lp_load_weights": [vp, vp, sz],
            "lp_init_weights_random": [vp, C.c_uint64, f32],
            "lp_query_max_batch_weight": [vp, P(i64)],
            "lp_submit": [vp, P(Request), i32],
            "lp_set_forced_tokens": [vp, i64, P(i32), i32],
            "lp_set_sampling": [vp, i64, f32, i32, f32, C.c_uint64],
            "lp_run": [vp, i32, i32],
            "lp_get_result": [vp, i64, P(i32), P(i64), P(i64), P(i64), P(i64)],
            "lp_get_token_times": [vp, i64, P(i64)],
            "lp_get_run_stats": [vp, P(RunStats)],
            "lp_get_step_log": [vp, P(StepRecord), i64, P(i64), P(i64), P(i32), i64],
            "lp_get_logits": [vp, i64, i32, P(f32)],
            "lp_engine_destroy": [vp],
            "lp_sched_simulate": [P(Request), i32, i32, i64, i64, i32, i32, i64, i64, i64, i64, P(StepRecord),
                                  i64, P(i64), P(i64), P(i32), i64, P(i64), i64, P(i64)],
            "lp_summarize_latencies": [i32, P(i64), P(i32), P(i32), P(i64), P(LatencySummary)],
            "lp_wg_fit": [P(C.c_double), i64, i32, i32, P(vp)],
            "lp_wg_info": [vp, i32, P(i32), P(i64)],
            "lp_wg_bins": [vp, i32, P(C.c_double), P(C.c_double), P(i64)],
            "lp_wg_sample": [vp, P(C.c_double), i64, P(C.c_double), P(i64)],
            "lp_wg_sample_independent": [vp, P(C.c_double), i64, P(C.c_double)],
            "lp_get_latency_summary": [vp, P(LatencySummary)],
            "lp_op_gemm": [i32, vp, i64, vp, vp, i32, i32, i32, i32, vp, sz, vp],
            "lp_op_gemm_plan": [i32, i32, i32, i32, P(i32), P(i32), P(i32), P(i32)],
            "lp_op_pack_weight": [i32, vp, vp, i32, i32, vp],
            "lp_op_rmsnorm": [i32, vp, vp, i32, vp, vp, i32, i32, f32, vp],
            "lp_op_decode_attention": [i32, vp, vp, vp, vp, vp, i32, i64, vp, vp, i32, i32, i32, i32, i32, vp, sz,
                                       vp],
            "lp_op_decode_attention_noalloc": [i32, vp, vp, vp, vp, vp, i32, i64, vp, vp, i32, i32, i32, i32, i32,
                                               vp],
            "lp_op_prefill_attention": [i32, vp, vp, vp, vp, vp, i32, i64, vp, vp, i32, i32, i32, i32, i32, vp],
            "lp_op_argmax": [vp, i64, i32, i32, vp, vp],
            "lp_op_init_weight": [i32, vp, C.c_uint64, i32, i64, i64, f32, vp],
            "lp_op_sample": [vp, i64, i32, i32, vp, vp, vp],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = C.c_int
        L.lp_last_error.argtypes = [vp]
        L.lp_last_error.restype = C.c_char_p
        L.lp_op_decode_attention_ws_bytes.argtypes = [i32, i32, i32, i32]
        L.lp_op_decode_attention_ws_bytes.restype = sz
        L.lp_op_packed_weight_bytes.argtypes = [i32, i32, i32]
        L.lp_op_packed_weight_bytes.restype = sz
        L.lp_engine_destroy.restype = None
        L.lp_wg_free.argtypes = [vp]
        L.lp_wg_free.restype = None
        _lib = L
    return _lib


class LPError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"liblp error {code}: {msg}")
        self.code = code


def _check(rc, handle=None):
    if rc != LP_OK:
        msg = lib().lp_last_error(handle)
        raise LPError(rc, msg.decode() if msg else "")


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else None


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def make_config(shape, n_layers=None, dtype=None) -> ModelConfig:
    return ModelConfig(n_layers or shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                       shape.ffn_dim, shape.vocab, shape.rope_theta, shape.norm_eps,
                       shape.dtype if dtype is None else dtype)


def _requests(reqs):
    arr = (Request * len(reqs))()
    keep = []
    for i, r in enumerate(reqs):
        p = np.ascontiguousarray(r.prompt, dtype=np.int32)
        keep.append(p)
        arr[i] = Request(int(r.id), p.ctypes.data_as(C.POINTER(C.c_int32)), int(p.size), int(r.out_len),
                         int(r.arrival_ns))
    return arr, keep


def arena_bytes(cfg: ModelConfig, opt: EngineOptions) -> int:
    out = C.c_size_t()
    _check(lib().lp_arena_bytes_required(C.byref(cfg), C.byref(opt), C.byref(out)))
    return out.value


ARENA_ALIGN = 2 << 20


class Engine:
    """One serving engine on the current torch device and stream."""

    def __init__(self, cfg: ModelConfig, opt: EngineOptions, arena_bytes_: int | None = None, device="cuda"):
        import torch
        self.cfg, self.opt = cfg, opt
        n = arena_bytes_ if arena_bytes_ is not None else arena_bytes(cfg, opt)
        # the engine lays its buffers out on 2 MiB boundaries of the arena:
        # hand it a 2 MiB-aligned start (the allocation has that much slack)
        self.arena = torch.empty(n + ARENA_ALIGN, dtype=torch.uint8, device=device)
        base = (self.arena.data_ptr() + ARENA_ALIGN - 1) // ARENA_ALIGN * ARENA_ALIGN
        h = C.c_void_p()
        _check(lib().lp_engine_create(C.byref(cfg), C.byref(opt), C.c_void_p(base), n, _stream(), C.byref(h)))
        self.h = h
        self._reqs = {}

    def close(self):
        if getattr(self, "h", None):
            lib().lp_engine_destroy(self.h)
            self.h = None
        self.arena = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load_weights(self, blob: bytes):
        buf = C.create_string_buffer(blob, len(blob))
        _check(lib().lp_load_weights(self.h, buf, len(blob)), self.h)

    def init_weights_random(self, seed: int, std: float = 0.02):
        _check(lib().lp_init_weights_random(self.h, seed, std), self.h)

    def max_batch_weight(self) -> int:
        v = C.c_int64()
        _check(lib().lp_query_max_batch_weight(self.h, C.byref(v)), self.h)
        return v.value

    def submit(self, reqs):
        arr, _keep = _requests(reqs)
        _check(lib().lp_submit(self.h, arr, len(reqs)), self.h)
        self._reqs = {int(r.id): r for r in reqs}

    def set_forced_tokens(self, rid: int, toks):
        t = np.ascontiguousarray(toks, dtype=np.int32)
        _check(lib().lp_set_forced_tokens(self.h, rid, t.ctypes.data_as(C.POINTER(C.c_int32)), t.size), self.h)

    def run(self, mode=LP_CLOSED_LOOP, concurrency=None):
        if concurrency is None:
            concurrency = self.opt.max_batch
        _check(lib().lp_run(self.h, mode, concurrency), self.h)

    def result(self, rid: int):
        r = self._reqs[rid]
        toks = np.zeros(r.out_len, dtype=np.int32)
        itl = np.zeros(max(r.out_len - 1, 1), dtype=np.int64)
        ttft, e2e, arr = C.c_int64(), C.c_int64(), C.c_int64()
        _check(lib().lp_get_result(self.h, rid, toks.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(ttft),
                                   itl.ctypes.data_as(C.POINTER(C.c_int64)), C.byref(e2e), C.byref(arr)), self.h)
        return {"tokens": toks, "ttft_ns": ttft.value, "itl_ns": itl[: r.out_len - 1], "e2e_ns": e2e.value,
                "arrival_ns": arr.value}

    def set_sampling(self, rid: int, temperature: float, top_k: int = 0, top_p: float = 1.0, seed: int = 0):
        """Sampling parameters of submitted request rid (greedy until set)."""
        _check(lib().lp_set_sampling(self.h, rid, temperature, top_k, top_p, seed & 0xFFFFFFFFFFFFFFFF), self.h)

    def latency_summary(self) -> dict:
        """Load-test metrics of the last run over all submitted requests."""
        out = LatencySummary()
        _check(lib().lp_get_latency_summary(self.h, C.byref(out)), self.h)
        return out.as_dict()

    def token_times(self, rid: int):
        r = self._reqs[rid]
        t = np.zeros(r.out_len, dtype=np.int64)
        _check(lib().lp_get_token_times(self.h, rid, t.ctypes.data_as(C.POINTER(C.c_int64))), self.h)
        return t

    def stats(self) -> dict:
        s = RunStats()
        _check(lib().lp_get_run_stats(self.h, C.byref(s)), self.h)
        return s.as_dict()

    def step_log(self):
        n = C.c_int64()
        _check(lib().lp_get_step_log(self.h, None, 0, C.byref(n), None, None, 0), self.h)
        recs = (StepRecord * max(n.value, 1))()
        _check(lib().lp_get_step_log(self.h, recs, n.value, C.byref(n), None, None, 0), self.h)
        total = sum(recs[k].n_rows for k in range(n.value))
        ids = np.zeros(max(total, 1), dtype=np.int64)
        slots = np.zeros(max(total, 1), dtype=np.int32)
        _check(lib().lp_get_step_log(self.h, recs, n.value, C.byref(n), ids.ctypes.data_as(C.POINTER(C.c_int64)),
                                     slots.ctypes.data_as(C.POINTER(C.c_int32)), total), self.h)
        out, r = [], 0
        for k in range(n.value):
            rec = recs[k]
            out.append({"kind": "prefill" if rec.kind == 0 else "decode", "n_rows": rec.n_rows,
                        "n_tokens": rec.n_tokens, "sum_ctx": rec.sum_ctx, "plan_ns": rec.plan_ns,
                        "end_ns": rec.end_ns, "ids": ids[r:r + rec.n_rows].tolist(),
                        "slots": slots[r:r + rec.n_rows].tolist()})
            r += rec.n_rows
        return out

    def logits(self, rid: int, k: int) -> np.ndarray:
        out = np.zeros(self.cfg.vocab, dtype=np.float32)
        _check(lib().lp_get_logits(self.h, rid, k, out.ctypes.data_as(C.POINTER(C.c_float))), self.h)
        return out


# ------------------------------------------------------------------ host simulation

def sched_simulate(reqs, max_batch, max_batch_weight, max_prefill_tokens, closed_loop, concurrency,
                   a_prefill, b_prefill, a_decode, b_decode):
    """Runs the engine's scheduler on the host with a linear step-time model."""
    arr, _keep = _requests(reqs)
    n = len(reqs)
    total_out = sum(int(r.out_len) for r in reqs)
    cap = 4 * total_out + 16
    steps = (StepRecord * cap)()
    ns = C.c_int64()
    ids = np.zeros(cap * max_batch, dtype=np.int64)
    slots = np.zeros(cap * max_batch, dtype=np.int32)
    toks = np.zeros(total_out, dtype=np.int64)
    arrivals = np.zeros(n, dtype=np.int64)
    _check(lib().lp_sched_simulate(arr, n, max_batch, max_batch_weight, max_prefill_tokens,
                                   LP_CLOSED_LOOP if closed_loop else LP_OPEN_LOOP, concurrency, a_prefill,
                                   b_prefill, a_decode, b_decode, steps, cap, C.byref(ns),
                                   ids.ctypes.data_as(C.POINTER(C.c_int64)),
                                   slots.ctypes.data_as(C.POINTER(C.c_int32)), ids.size,
                                   toks.ctypes.data_as(C.POINTER(C.c_int64)), toks.size,
                                   arrivals.ctypes.data_as(C.POINTER(C.c_int64))))
    out, r = [], 0
    for k in range(ns.value):
        rec = steps[k]
        out.append({"kind": "prefill" if rec.kind == 0 else "decode", "ids": ids[r:r + rec.n_rows].tolist(),
                    "slots": slots[r:r + rec.n_rows].tolist(), "end_ns": rec.end_ns, "plan_ns": rec.plan_ns,
                    "sum_ctx": rec.sum_ctx, "n_tokens": rec.n_tokens})
        r += rec.n_rows
    token_ns, t = {}, 0
    for q in reqs:
        token_ns[int(q.id)] = toks[t:t + q.out_len].tolist()
        t += q.out_len
    return out, token_ns, {int(q.id): int(a) for q, a in zip(reqs, arrivals)}


def summarize_latencies(arrival_ns, in_len, out_len, token_ns) -> dict:
    """Load-test metrics of one experiment: per-request arrival times, input
    and output lengths, and output-token times packed in request order."""
    arr = np.ascontiguousarray(arrival_ns, dtype=np.int64)
    inl = np.ascontiguousarray(in_len, dtype=np.int32)
    outl = np.ascontiguousarray(out_len, dtype=np.int32)
    toks = np.ascontiguousarray(token_ns, dtype=np.int64)
    if toks.size != int(outl.sum()) or not (arr.size == inl.size == outl.size):
        raise ValueError("token_ns must hold sum(out_len) values; one arrival and length per request")
    out = LatencySummary()
    _check(lib().lp_summarize_latencies(arr.size, arr.ctypes.data_as(C.POINTER(C.c_int64)),
                                        inl.ctypes.data_as(C.POINTER(C.c_int32)),
                                        outl.ctypes.data_as(C.POINTER(C.c_int32)),
                                        toks.ctypes.data_as(C.POINTER(C.c_int64)), C.byref(out)))
    return out.as_dict()


class RequestModel:
    """The workload generator's joint request model (Sec. III-B), fitted to
    trace records [n x n_params]; sampling takes the uniforms it consumes."""

    def __init__(self, records, max_bins: int = 64):
        rec = np.ascontiguousarray(records, dtype=np.float64)
        if rec.ndim != 2:
            raise ValueError("records must be [n, n_params]")
        self.n_params = rec.shape[1]
        h = C.c_void_p()
        _check(lib().lp_wg_fit(rec.ctypes.data_as(C.POINTER(C.c_double)), rec.shape[0], self.n_params, max_bins,
                               C.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            lib().lp_wg_free(self.h)
            self.h = None

    def __del__(self):
        self.close()

    def n_joint_bins(self) -> int:
        nj = C.c_int64()
        _check(lib().lp_wg_info(self.h, -1, None, C.byref(nj)))
        return nj.value

    def bins(self, param: int):
        """(edges [n_bins + 1], centres [n_bins], record counts [n_bins])."""
        nb = C.c_int32()
        _check(lib().lp_wg_info(self.h, param, C.byref(nb), None))
        e, c = np.zeros(nb.value + 1), np.zeros(nb.value)
        k = np.zeros(nb.value, dtype=np.int64)
        _check(lib().lp_wg_bins(self.h, param, e.ctypes.data_as(C.POINTER(C.c_double)),
                                c.ctypes.data_as(C.POINTER(C.c_double)), k.ctypes.data_as(C.POINTER(C.c_int64))))
        return e, c, k

    def sample(self, u):
        """Requests [n x n_params] and their joint-bin indices for uniforms u [n]."""
        uu = np.ascontiguousarray(u, dtype=np.float64).reshape(-1)
        out = np.zeros((uu.size, self.n_params))
        jb = np.zeros(uu.size, dtype=np.int64)
        _check(lib().lp_wg_sample(self.h, uu.ctypes.data_as(C.POINTER(C.c_double)), uu.size,
                                  out.ctypes.data_as(C.POINTER(C.c_double)), jb.ctypes.data_as(C.POINTER(C.c_int64))))
        return out, jb

    def sample_independent(self, u):
        """Requests [n x n_params] with every parameter drawn from its own
        marginal, for uniforms u [n x n_params]."""
        uu = np.ascontiguousarray(u, dtype=np.float64).reshape(-1, self.n_params)
        out = np.zeros(uu.shape)
        _check(lib().lp_wg_sample_independent(self.h, uu.ctypes.data_as(C.POINTER(C.c_double)), uu.shape[0],
                                              out.ctypes.data_as(C.POINTER(C.c_double))))
        return out


# ------------------------------------------------------------------ single-kernel ops (torch tensors)

def _dt(t):
    import torch
    if t.dtype == torch.float16:
        return LP_F16
    return LP_BF16 if t.dtype in (torch.bfloat16, torch.int16, torch.uint16) else LP_F32


def packed_weight_elems(N: int, K: int) -> int:
    """Elements of an [N x K] 16-bit weight in the tiled layout."""
    return -(-N // 16) * -(-K // 32) * 512


def op_pack_weight(W, W_packed):
    """Row-major [N x K] 16-bit W -> the tiled layout the 16-bit GEMMs read
    (W_packed: a flat tensor of packed_weight_elems(N, K) elements)."""
    N, K = W.shape
    assert W_packed.numel() * W_packed.element_size() >= lib().lp_op_packed_weight_bytes(_dt(W), N, K)
    _check(lib().lp_op_pack_weight(_dt(W), _ptr(W), _ptr(W_packed), N, K, _stream()))


def op_gemm(X, W, Y, k_splits=1, ws=None, N=None):
    """Y = X W^T.  16-bit: W is the packed flat tensor and N its row count;
    fp32: W is row-major [N x K]."""
    M, K = X.shape
    if N is None:
        N = W.shape[0]
    _check(lib().lp_op_gemm(_dt(X), _ptr(X), X.stride(0), _ptr(W), _ptr(Y), M, N, K, k_splits, _ptr(ws),
                            0 if ws is None else ws.numel() * ws.element_size(), _stream()))


GEMM_KINDS = {0: "decode", 1: "prefill", 2: "prefill_pair", 3: "tiled"}


def op_gemm_plan(M, N, K, k_splits=1, with_order=False):
    """(kernel kind, rows per tile, K splits) that op_gemm runs for this shape,
    plus the row tiles per XCD group of its tile order (0: plain) when
    with_order; k_splits=0: what an engine prefill step of M > 64 rows runs."""
    kind, rows, splits, xg = C.c_int32(), C.c_int32(), C.c_int32(), C.c_int32()
    _check(lib().lp_op_gemm_plan(M, N, K, k_splits, C.byref(kind), C.byref(rows), C.byref(splits), C.byref(xg)))
    out = (GEMM_KINDS[kind.value], rows.value, splits.value)
    return out + (xg.value,) if with_order else out


def op_rmsnorm(x, g, y, eps, part=None, n_part=0):
    rows, d = x.shape
    _check(lib().lp_op_rmsnorm(_dt(y), _ptr(x), _ptr(part), n_part, _ptr(g), _ptr(y), rows, d, eps, _stream()))


def decode_attention_ws_bytes(M, n_heads, head_dim, max_ctx):
    return lib().lp_op_decode_attention_ws_bytes(M, n_heads, head_dim, max_ctx)


def op_decode_attention(q, out, kc, vc, block_table, row_slot, row_pos, n_kv_heads, max_ctx, ws):
    M, Hq, hd = q.shape
    _check(lib().lp_op_decode_attention(_dt(q), _ptr(q), _ptr(out), _ptr(kc), _ptr(vc), _ptr(block_table),
                                        block_table.shape[1], kc.shape[0], _ptr(row_slot), _ptr(row_pos), M, Hq,
                                        n_kv_heads, hd, max_ctx, _ptr(ws), ws.numel() * ws.element_size(),
                                        _stream()))


def op_decode_attention_noalloc(q, out, kc, vc, block_table, row_slot, row_pos, n_kv_heads, max_ctx):
    """lp_op_decode_attention_noalloc: the same call without a workspace."""
    M, Hq, hd = q.shape
    _check(lib().lp_op_decode_attention_noalloc(_dt(q), _ptr(q), _ptr(out), _ptr(kc), _ptr(vc), _ptr(block_table),
                                                block_table.shape[1], kc.shape[0], _ptr(row_slot), _ptr(row_pos), M,
                                                Hq, n_kv_heads, hd, max_ctx, _stream()))


def op_prefill_attention(q, out, kc, vc, block_table, seq_start, seq_slot, max_len, n_kv_heads):
    _, Hq, hd = q.shape
    _check(lib().lp_op_prefill_attention(_dt(q), _ptr(q), _ptr(out), _ptr(kc), _ptr(vc), _ptr(block_table),
                                         block_table.shape[1], kc.shape[0], _ptr(seq_start), _ptr(seq_slot),
                                         seq_slot.numel(), max_len, Hq, n_kv_heads, hd, _stream()))


def op_argmax(logits, tokens):
    M, V = logits.shape
    _check(lib().lp_op_argmax(_ptr(logits), logits.stride(0), M, V, _ptr(tokens), _stream()))


def op_sample(logits, params, tokens):
    """params: a device tensor holding M SampleParams records (uint8 view)."""
    M, V = logits.shape
    _check(lib().lp_op_sample(_ptr(logits), logits.stride(0), M, V, _ptr(params), _ptr(tokens), _stream()))


def sample_params_array(rows) -> np.ndarray:
    """Packs (temperature, top_k, top_p, (k0, k1), (c0, c1, c2)) tuples into
    the byte layout of lp_sample_params."""
    arr = (SampleParams * len(rows))()
    for i, (t, k, p, key, ctr) in enumerate(rows):
        arr[i] = SampleParams(t, k, p, (C.c_uint32 * 2)(*key), (C.c_uint32 * 3)(*ctr))
    return np.frombuffer(bytes(arr), dtype=np.uint8).copy()


def op_init_weight(dst, seed, tensor_id, std):
    rows, cols = dst.shape
    _check(lib().lp_op_init_weight(_dt(dst), _ptr(dst), seed, tensor_id, rows, cols, std, _stream()))
