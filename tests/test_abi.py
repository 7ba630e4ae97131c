"""Host-side checks of the C ABI: the library loads without a GPU, exports every
function the headers declare, and its scheduler (driven by a synthetic
step-time model) reproduces the oracle's schedule and accounting exactly."""
import os
import re

import numpy as np
import pytest

from oracle import serving as S
from paper_2410_02425_amd import lp, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("lp.h", "lp_ops.h"):
        with open(os.path.join(ROOT, "include", h)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(lp_\w+)\s*\(", text))
    return names


def test_library_exports_every_declared_function():
    L = lp.lib()
    names = declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), n
    assert names == set(lp.EXPORTED)


def test_config_validation_without_gpu():
    shape = synth.SHAPES["8b"]
    cfg = lp.make_config(shape)
    opt = lp.EngineOptions(64, 5120, 0, 65536, 0, 0)
    n = lp.arena_bytes(cfg, opt)
    # bf16 weights alone are 16.06 GB; KV for 64 x 5120 tokens is 42.9 GB
    assert 16.0e9 + 42.9e9 < n < 16.0e9 + 42.9e9 + 8e9
    bad = lp.make_config(shape)
    bad.n_kv_heads = 7
    with pytest.raises(lp.LPError):
        lp.arena_bytes(bad, opt)
    opt_bad = lp.EngineOptions(65, 5120, 0, 65536, 0, 0)
    with pytest.raises(lp.LPError):
        lp.arena_bytes(cfg, opt_bad)


def _oracle_trace(reqs, mb, W, P, closed, U, ap, bp, ad, bd):
    sreqs = [S.SimRequest(r.id, r.in_len, r.out_len, r.arrival_ns) for r in reqs]
    step = lambda kind, n_rows, n_tokens, sum_ctx: ap + bp * n_tokens if kind == "prefill" else ad + bd * n_rows
    return S.simulate(sreqs, mb, W, P, closed, U, step)


@pytest.mark.parametrize("closed", [True, False])
def test_engine_scheduler_matches_oracle(closed):
    rng = np.random.default_rng(7 if closed else 8)
    for trial in range(25):
        n = int(rng.integers(1, 40))
        reqs, t = [], 0
        for i in range(n):
            t += int(rng.integers(0, 3000))
            reqs.append(synth.Request(1000 + i, rng.integers(0, 50, size=int(rng.integers(1, 60))).astype(np.int32),
                                      int(rng.integers(1, 20)), t if not closed else 0))
        mb = int(rng.integers(1, 9))
        W = int(rng.integers(80, 400))
        P = int(rng.integers(60, 300))
        U = int(rng.integers(1, 12))
        ap, bp, ad, bd = 500, int(rng.integers(1, 20)), 300, int(rng.integers(1, 30))
        steps, toks, arr = lp.sched_simulate(reqs, mb, W, P, closed, U, ap, bp, ad, bd)
        tr = _oracle_trace(reqs, mb, W, P, closed, U, ap, bp, ad, bd)
        assert [(s["kind"], s["ids"], s["slots"], s["end_ns"]) for s in steps] == \
               [(s.kind, s.ids, s.slots, s.end_ns) for s in tr.steps]
        assert [s["plan_ns"] for s in steps] == [s.plan_ns for s in tr.steps]
        assert toks == tr.token_ns
        assert arr == tr.arrival_ns
        for r in reqs:
            ttft, itl, e2e = S.request_latencies(arr[r.id], toks[r.id])
            assert e2e == ttft + sum(itl)


def test_scheduler_rejects_unadmittable_request():
    reqs = [synth.Request(0, np.zeros(50, np.int32), 60)]
    with pytest.raises(lp.LPError):
        lp.sched_simulate(reqs, 2, 100, 1000, True, 1, 1, 1, 1, 1)


def test_scheduler_golden_schedule():
    import json
    with open(os.path.join(ROOT, "tests", "golden", "schedule_example.json")) as f:
        g = json.load(f)
    reqs = [synth.Request(i, np.zeros(a, np.int32), b) for i, a, b in g["requests"]]
    for c in g["cases"]:
        steps, toks, arr = lp.sched_simulate(reqs, g["max_batch"], c["max_batch_weight"], g["max_prefill_tokens"],
                                             True, g["concurrency"], 10, 1, 5, 1)
        assert [[s["kind"], s["ids"], s["slots"], s["end_ns"]] for s in steps] == c["steps"]
        assert {str(k): v for k, v in toks.items()} == c["token_ns"]
        assert {str(k): v for k, v in arr.items()} == c["arrival_ns"]


SUMMARY_KEYS = ("n_requests", "output_tokens", "itl_count", "ttft_p50_ns", "nttft_p50_ns", "itl_p50_ns",
                "e2e_p50_ns", "ttft_p90_ns", "itl_p90_ns", "itl_p99_ns", "throughput_tok_s")


def _native_summary(reqs, arr, toks):
    return lp.summarize_latencies([arr[r.id] for r in reqs], [r.in_len for r in reqs],
                                  [r.out_len for r in reqs], np.concatenate([toks[r.id] for r in reqs]))


def test_latency_summary_golden():
    import json
    with open(os.path.join(ROOT, "tests", "golden", "latency_example.json")) as f:
        g = json.load(f)
    rq = g["requests"]
    got = lp.summarize_latencies([r["arrival_ns"] for r in rq], [r["in_len"] for r in rq],
                                 [len(r["token_ns"]) for r in rq], np.concatenate([r["token_ns"] for r in rq]))
    for k in SUMMARY_KEYS:
        if k != "throughput_tok_s":
            assert got[k] == g["expected"][k], k
    assert got["throughput_tok_s"] == pytest.approx(g["expected"]["throughput_tok_s"], rel=1e-12)


@pytest.mark.parametrize("closed", [True, False])
def test_latency_summary_matches_oracle(closed):
    """The native load-test metrics equal the oracle's, bit for bit, over
    simulated schedules (odd and even counts, single-token requests)."""
    rng = np.random.default_rng(21 if closed else 22)
    for trial in range(30):
        n = int(rng.integers(1, 30))
        reqs, t = [], 0
        for i in range(n):
            t += int(rng.integers(0, 5000))
            reqs.append(synth.Request(i, np.zeros(int(rng.integers(1, 60)), np.int32), int(rng.integers(1, 12)),
                                      t if not closed else 0))
        steps, toks, arr = lp.sched_simulate(reqs, int(rng.integers(1, 8)), 400, 300, closed,
                                             int(rng.integers(1, 10)), 700, int(rng.integers(1, 9)), 300,
                                             int(rng.integers(1, 40)))
        got = _native_summary(reqs, arr, toks)
        exp = S.summarize(arr, toks, {r.id: r.in_len for r in reqs})
        for k in SUMMARY_KEYS:
            assert (got[k] == exp[k]) or (np.isnan(got[k]) and np.isnan(exp[k])), (trial, k, got[k], exp[k])


def test_latency_summary_rejects_bad_input():
    with pytest.raises(lp.LPError):
        lp.summarize_latencies([0], [0], [1], [5])
    with pytest.raises(ValueError):
        lp.summarize_latencies([0, 1], [1, 1], [2, 1], [5, 6])


def test_zero_row_op_calls_are_noops():
    """Op calls with no rows check their sizes and return LP_OK without a
    launch or a memory access, so null pointers pass (no GPU is touched);
    bad sizes are still LP_EINVAL."""
    L = lp.lib()
    F16, OK, EINVAL = lp.LP_F16, lp.LP_OK, lp.LP_EINVAL
    assert L.lp_op_gemm(F16, None, 64, None, None, 0, 128, 64, 1, None, 0, None) == OK
    assert L.lp_op_gemm(F16, None, 64, None, None, 0, 128, 64, 4, None, 0, None) == OK
    assert L.lp_op_gemm(F16, None, 64, None, None, -1, 128, 64, 1, None, 0, None) == EINVAL
    assert L.lp_op_gemm(F16, None, 64, None, None, 0, 128, 60, 1, None, 0, None) == EINVAL  # K % 8
    assert L.lp_op_rmsnorm(F16, None, None, 8, None, None, 0, 4096, 1e-5, None) == OK
    assert L.lp_op_rmsnorm(F16, None, None, 0, None, None, 0, 9000, 1e-5, None) == EINVAL  # d > 8192
    assert L.lp_op_decode_attention(F16, None, None, None, None, None, 2, 4, None, None, 0, 32, 8, 128, 128,
                                    None, 0, None) == OK
    assert L.lp_op_decode_attention(F16, None, None, None, None, None, 1, 4, None, None, 0, 32, 8, 128, 128,
                                    None, 0, None) == EINVAL  # max_blocks * 64 < max_ctx
    assert L.lp_op_decode_attention(F16, None, None, None, None, None, 2, 4, None, None, 0, 32, 3, 128, 128,
                                    None, 0, None) == EINVAL  # Hq not a multiple of Hkv
    assert L.lp_op_prefill_attention(F16, None, None, None, None, None, 2, 4, None, None, 0, 100, 32, 8, 128,
                                     None) == OK
    assert L.lp_op_prefill_attention(F16, None, None, None, None, None, 2, 4, None, None, -1, 100, 32, 8, 128,
                                     None) == EINVAL
    assert L.lp_op_argmax(None, 1000, 0, 1000, None, None) == OK
    assert L.lp_op_argmax(None, 999, 0, 1000, None, None) == EINVAL  # ld < V
    assert L.lp_op_sample(None, 1000, 0, 1000, None, None, None) == OK
    assert L.lp_op_sample(None, 1 << 22, 0, (1 << 21) + 2, None, None, None) == EINVAL  # V > 2^21
    # rows present but pointers null: rejected before any launch
    assert L.lp_op_argmax(None, 1000, 3, 1000, None, None) == EINVAL
    assert L.lp_op_gemm(F16, None, 64, None, None, 5, 128, 64, 1, None, 0, None) == EINVAL


def test_gemm_plan_query():
    """The host-side GEMM plan: decode kernel for M <= 64, the LDS-tiled kernel
    when K is not a multiple of 128, two 128-row workgroups per CU only with
    at least 512 tiles and no K split, split requests kept (rounded to whole
    128-wide K chunks)."""
    assert lp.op_gemm_plan(1, 4096, 4096) == ("decode", 16, 1)
    assert lp.op_gemm_plan(64, 4096, 4096, 8) == ("decode", 64, 8)
    assert lp.op_gemm_plan(65, 1376, 688) == ("tiled", 128, 1)
    assert lp.op_gemm_plan(777, 6144, 4096)[0] == "prefill"
    for M, N, K in [(553, 28672, 4096), (4223, 4096, 14336), (100, 131072, 256), (1500, 12000, 256)]:
        tiles = -(-M // 128) * -(-N // 256)
        assert tiles >= 512
        assert lp.op_gemm_plan(M, N, K) == ("prefill_pair", 128, 1)
        kind, rows, splits = lp.op_gemm_plan(M, N, K, 2)
        assert kind == "prefill" and splits == 2
    # fewer than 512 tiles of 128 rows never pair
    for M in range(65, 2049, 64):
        for N in (1024, 4096, 6144):
            kind, rows, splits = lp.op_gemm_plan(M, N, 4096)
            if -(-M // 128) * -(-N // 256) < 512:
                assert kind == "prefill", (M, N)
    # tile order: XCD groups of 16 row tiles for 64+ column tiles with 256-row
    # tiles, or with 128-row tiles once the weight exceeds the 256 MB
    # last-level cache; plain otherwise
    assert lp.op_gemm_plan(553, 57344, 8192, 0, with_order=True)[3] == 16   # 70B gate/up, 940 MB
    assert lp.op_gemm_plan(553, 28672, 4096, 0, with_order=True)[3] == 0    # 8B gate/up, 235 MB
    assert lp.op_gemm_plan(600, 16300, 1024, 1, with_order=True)[3] == 16
    assert lp.op_gemm_plan(1593, 8192, 28672, 0, with_order=True)[3] == 0   # 32 column tiles
    assert lp.op_gemm_plan(64, 28672, 4096, 1, with_order=True)[3] == 0     # decode kernel
    with pytest.raises(lp.LPError):
        lp.op_gemm_plan(0, 4096, 4096)
