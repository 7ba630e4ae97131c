"""The no-allocation decode attention entry point
(lp_op_decode_attention_noalloc) against the allocating one
(lp_op_decode_attention) through the C ABI: two calls in a row on the same
GPU, the second with a smaller batch, each bit-identical to the allocating
call on the same inputs and within the attention error bound of the float64
oracle; a call whose partials would exceed the scratch array is refused before
any launch."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import transformer as T
from paper_2410_02425_amd import lp
from test_gpu_kernels import DEV, attention_tol, bf16_values, make_paged_cache, to_dev

pytestmark = pytest.mark.gpu


def _call_both(rng, dtype, Hq, Hkv, hd, ctx):
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    (kc, vt, bt), Ks, Vs = make_paged_cache(rng, ctx, Hkv, hd, tdt)
    M = len(ctx)
    q = bf16_values(rng, (M, Hq, hd))
    qd = to_dev(q, tdt)
    max_ctx = max(ctx)
    row_slot = torch.arange(M, dtype=torch.int32, device=DEV)
    row_pos = torch.tensor([c - 1 for c in ctx], dtype=torch.int32, device=DEV)
    ws = torch.empty(lp.decode_attention_ws_bytes(M, Hq, hd, max_ctx) // 4 + 1, dtype=torch.float32, device=DEV)
    want = torch.full((M, Hq, hd), float("nan"), dtype=tdt, device=DEV)
    lp.op_decode_attention(qd, want, kc, vt, bt, row_slot, row_pos, Hkv, max_ctx, ws)
    got = torch.full((M, Hq, hd), float("nan"), dtype=tdt, device=DEV)
    lp.op_decode_attention_noalloc(qd, got, kc, vt, bt, row_slot, row_pos, Hkv, max_ctx)
    torch.cuda.synchronize()
    g, w = got.float().cpu().numpy(), want.float().cpu().numpy()
    assert not np.isnan(g).any()
    assert np.array_equal(g, w)                       # the same kernels on the same inputs
    for m, c in enumerate(ctx):
        args = (q[m:m + 1].astype(np.float64), Ks[m].astype(np.float64))
        ref = T.attention(*args, Vs[m].astype(np.float64), [c - 1], np.arange(c), Hkv)[0]
        mag = T.attention(*args, np.abs(Vs[m].astype(np.float64)), [c - 1], np.arange(c), Hkv)[0]
        assert np.all(np.abs(g[m] - ref) <= attention_tol(dtype, ref, mag)), (m, c)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_noalloc_decode_attention_matches_allocating_call(dtype):
    rng = np.random.default_rng(77)
    # a full 64-row 8B-shape batch, then a smaller one: the second call
    # reuses the scratch array the first left full of partials
    first = np.clip(rng.lognormal(6.4, 0.7, 64), 16, 4096).astype(int).tolist()
    _call_both(rng, dtype, 32, 8, 128, first)
    _call_both(rng, dtype, 32, 8, 128, [1, 65, 300, 2000, 257])


def test_noalloc_decode_attention_fp32_and_refusal():
    rng = np.random.default_rng(78)
    _call_both(rng, "f32", 4, 4, 64, [1, 40, 129, 600])
    _call_both(rng, "f32", 8, 2, 64, [64, 65])
    # 64 rows x 32 heads x 32 chunks x (128 + 2) x 4 bytes > 32 MiB: refused
    # from the sizes alone (LP_EINVAL), nothing launched
    q = torch.zeros(64, 32, 128, dtype=torch.float16, device=DEV)
    out = torch.zeros_like(q)
    kc = torch.zeros(1, 8, 64, 128, dtype=torch.float16, device=DEV)
    bt = torch.zeros(64, 128, dtype=torch.int32, device=DEV)
    rs = torch.zeros(64, dtype=torch.int32, device=DEV)
    with pytest.raises(lp.LPError) as err:
        lp.op_decode_attention_noalloc(q, out, kc, kc, bt, rs, rs, 8, 8192)
    assert err.value.code == lp.LP_EINVAL and "scratch" in str(err.value)
    torch.cuda.synchronize()
    assert torch.count_nonzero(out).item() == 0
