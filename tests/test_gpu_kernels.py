"""Kernel-level parity on the GPU: every kernel of the serving step, called
through the C ABI (include/lp_ops.h), against the float64 oracle on the same
seeded inputs.  Sizes span several tiles plus ragged tails, and include the
full 8B-shape decode shapes (checked on sampled outputs)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import transformer as T
from paper_2410_02425_amd import lp, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def bf16_values(rng, shape, scale=1.0):
    """Random fp32 values that bf16 represents exactly."""
    v = (rng.standard_normal(size=shape) * scale).astype(np.float32)
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(v)).reshape(shape)


def to_dev(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(dtype).to(DEV)


def gemm_bound(X, W, rows, cols):
    """|error| bound for fp32 accumulation of sampled outputs: 1e-5 * sum|x||w|."""
    return 1e-5 * np.abs(X[rows].astype(np.float64)) @ np.abs(W[cols].astype(np.float64)).T


GEMM_CASES = [
    # M, N, K, splits -- decode kernel (M <= 64) with and without split-K, tails in M, N and K
    (1, 96, 256, 1), (16, 768, 256, 1), (37, 1376, 688, 3), (64, 1024, 256, 2),
    (64, 6144, 4096, 6), (64, 4096, 14336, 8), (5, 2000, 1000, 4),
    # the 8B-shape decode launches as the engine issues them at 64 rows:
    # QKV with 5 splits, O with 8
    (64, 6144, 4096, 5), (64, 4096, 4096, 8),
    # prefill kernels: K not a multiple of 128 (LDS-tiled fallback), then the
    # pipelined kernel with tails in M and N, split-K, long K
    (65, 1376, 688, 1), (200, 768, 256, 1), (300, 640, 4096, 1), (300, 640, 4096, 4),
    (513, 1000, 1024, 2), (777, 6144, 4096, 1), (600, 1536, 14336, 4), (1030, 512, 384, 3),
    # wide weights (64 column tiles) with 256-row tiles take the XCD-grouped
    # tile order: a ragged last group of row tiles and a tail in N, without
    # and with split K
    (600, 16300, 1024, 1), (300, 16300, 1024, 2),
    # at least 512 tiles of 128 rows: two workgroups per CU, tails in M and N,
    # one row tile shorter than 128 rows; a weight larger than the 256 MB
    # last-level cache takes the XCD-grouped order there too
    (4200, 16300, 128, 1), (1500, 12000, 256, 1), (100, 131072, 256, 1), (600, 34800, 4096, 1),
    # 64 or more column tiles, not a multiple of 8: the grid is laid out over
    # the next multiple of 8 and its padding workgroups exit (86 tiles,
    # plain; 108 tiles of a 283 MB weight, grouped; 65 tiles with 256-row
    # tiles, grouped, and split K, plain)
    (700, 22000, 4096, 1), (600, 27600, 5120, 1), (600, 16500, 1024, 1), (300, 16500, 2048, 2),
    # odd split counts the planner takes for prompts of a few hundred tokens
    # (8B O at 553 rows: 3 splits; a 5-way split of a long K with tails)
    (553, 4096, 4096, 3), (632, 1000, 6400, 5),
]

# the kernel each case above is planned to take (the plan is host logic):
# kind, tile rows, row tiles per XCD group of the tile order (0: plain)
GEMM_CASE_KINDS = {(600, 16300, 1024, 1): ("prefill", 256, 16), (300, 16300, 1024, 2): ("prefill", 256, 16),
                   (4200, 16300, 128, 1): ("prefill_pair", 128, 0), (1500, 12000, 256, 1): ("prefill_pair", 128, 0),
                   (100, 131072, 256, 1): ("prefill_pair", 128, 0), (600, 34800, 4096, 1): ("prefill_pair", 128, 16),
                   (700, 22000, 4096, 1): ("prefill_pair", 128, 0), (600, 27600, 5120, 1): ("prefill_pair", 128, 16),
                   (600, 16500, 1024, 1): ("prefill", 256, 16), (300, 16500, 2048, 2): ("prefill", 128, 0)}


HALF = {"bf16": torch.bfloat16, "f16": torch.float16}


def packed(Wd):
    """W (device, row-major [N x K], 16-bit) in the tiled weight layout."""
    N, K = Wd.shape
    P = torch.full((lp.packed_weight_elems(N, K),), float("nan"), dtype=Wd.dtype, device=DEV)
    lp.op_pack_weight(Wd, P)
    return P


def tile_layout_reference(W):
    """The tiled layout written out from its definition: tiles of 16 rows x 32
    columns, tile (i, j) at index j * ceil(N/16) + i, element (r, c) of a tile
    at 8 * (r + 16 * (c // 8)) + c % 8, zeros past N and K."""
    N, K = W.shape
    nt, kt = -(-N // 16), -(-K // 32)
    full = np.zeros((nt * 16, kt * 32), dtype=W.dtype)
    full[:N, :K] = W
    out = np.zeros(nt * kt * 512, dtype=W.dtype)
    for i in range(nt):
        for j in range(kt):
            tile = full[16 * i:16 * i + 16, 32 * j:32 * j + 32]
            base = (j * nt + i) * 512
            for r in range(16):
                for c in range(32):
                    out[base + 8 * (r + 16 * (c // 8)) + c % 8] = tile[r, c]
    return out


@pytest.mark.parametrize("half", ["bf16", "f16"])
@pytest.mark.parametrize("N,K", [(16, 32), (48, 96), (50, 40), (1000, 1000), (33, 688)])
def test_pack_weight_layout(N, K, half):
    rng = np.random.default_rng(N * 31 + K)
    Wd = to_dev(bf16_values(rng, (N, K)), HALF[half])
    P = packed(Wd)
    torch.cuda.synchronize()
    got = P.float().cpu().numpy()
    want = tile_layout_reference(Wd.float().cpu().numpy())  # the values as stored in the half type
    assert got.shape == want.shape
    assert np.array_equal(got, want)                 # bit-exact, padding zero (no NaN left)


@pytest.mark.parametrize("half", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,splits", GEMM_CASES)
def test_gemm_16bit(M, N, K, splits, half):
    if (M, N, K, splits) in GEMM_CASE_KINDS:
        kind, rows, _, order = lp.op_gemm_plan(M, N, K, splits, with_order=True)
        assert (kind, rows, order) == GEMM_CASE_KINDS[(M, N, K, splits)]
    rng = np.random.default_rng(M * 7 + N + K)
    X = bf16_values(rng, (M, K))          # bf16 values are exact in fp16 too
    W = bf16_values(rng, (N, K), 0.02)
    Xd, Wd = to_dev(X, HALF[half]), to_dev(W, HALF[half])
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(max(splits, 1) * M * N, dtype=torch.float32, device=DEV)
    lp.op_gemm(Xd, packed(Wd), Y, splits, ws, N=N)
    torch.cuda.synchronize()
    got = Y.cpu().numpy()
    ref = X.astype(np.float64) @ W.astype(np.float64).T
    bound = 1e-5 * (np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)).T) + 1e-12
    assert np.all(np.abs(got - ref) <= bound), np.max(np.abs(got - ref) / bound)


@pytest.mark.parametrize("half", ["bf16", "f16"])
def test_gemm_full_8b_gate_up_sampled(half):
    """The decode gate/up GEMM at its full 8B-shape size (M=64, N=2*14336,
    K=4096), checked on 512 sampled outputs computed one by one."""
    M, N, K = 64, 28672, 4096
    g = torch.Generator().manual_seed(1234)
    X = torch.randn(M, K, generator=g).to(HALF[half])
    W = (torch.randn(N, K, generator=g) * 0.02).to(HALF[half])
    Y = torch.empty(M, N, dtype=torch.float32, device=DEV)
    lp.op_gemm(X.to(DEV), packed(W.to(DEV)), Y, 1, None, N=N)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    rows, cols = rng.integers(0, M, 512), rng.integers(0, N, 512)
    rows[:2], cols[:2] = [0, M - 1], [0, N - 1]
    Xn, Wn = X.float().numpy().astype(np.float64), W.float().numpy().astype(np.float64)
    got = Y.cpu().numpy()[rows, cols]
    ref = np.einsum("ik,ik->i", Xn[rows], Wn[cols])
    bound = 1e-5 * np.einsum("ik,ik->i", np.abs(Xn[rows]), np.abs(Wn[cols]))
    assert np.all(np.abs(got - ref) <= bound)


@pytest.mark.parametrize("half", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,order", [(553, 28672, 4096, 0), (4223, 4096, 14336, 0), (553, 57344, 8192, 16)])
def test_gemm_prefill_sampled(M, N, K, order, half):
    """Prefill projections at sizes that take two workgroups per CU (8B
    gate/up of a 553-token prompt and down of a 4,223-token step, both in the
    plain tile order; 70B gate/up of a 553-token prompt, whose 940 MB weight
    takes the XCD-grouped order), checked on 1024 sampled outputs plus the
    first and last row and column, computed one by one in fp64."""
    kind, _, _, xg = lp.op_gemm_plan(M, N, K, 1, with_order=True)
    assert kind == "prefill_pair" and xg == order
    g = torch.Generator().manual_seed(M + N)
    X = torch.randn(M, K, generator=g).to(HALF[half])
    W = (torch.randn(N, K, generator=g) * 0.02).to(HALF[half])
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    lp.op_gemm(X.to(DEV), packed(W.to(DEV)), Y, 1, None, N=N)
    torch.cuda.synchronize()
    rng = np.random.default_rng(M)
    rows, cols = rng.integers(0, M, 1024), rng.integers(0, N, 1024)
    rows[:4], cols[:4] = [0, M - 1, 0, M - 1], [0, N - 1, N - 1, 0]
    Xs = X[torch.from_numpy(rows)].float().numpy().astype(np.float64)   # only the sampled rows in fp64
    Ws = W[torch.from_numpy(cols)].float().numpy().astype(np.float64)
    Yc = Y.cpu().numpy()
    assert not np.isnan(Yc).any()
    got = Yc[rows, cols]
    ref = np.einsum("ik,ik->i", Xs, Ws)
    bound = 1e-5 * np.einsum("ik,ik->i", np.abs(Xs), np.abs(Ws))
    assert np.all(np.abs(got - ref) <= bound)


_LM_CACHE = {}


def _lm_head_weight(N, K, half):
    """One random [N x K] weight per (N, half), kept for the cases that share
    it: host values, their fp32 copy (exact), and the tiled device matrix."""
    key = (N, K, half)
    if key not in _LM_CACHE:
        _LM_CACHE.clear()
        g = torch.Generator().manual_seed(N)
        W = (torch.randn(N, K, generator=g) * 0.02).to(HALF[half])
        _LM_CACHE[key] = (W, W.float().numpy(), packed(W.to(DEV)))
    return _LM_CACHE[key]


@pytest.mark.parametrize("half", ["bf16", "f16"])
@pytest.mark.parametrize("N", [128256, 32000])
@pytest.mark.parametrize("M", [17, 40, 64])
def test_gemm_lm_head_decode_sampled(M, N, half):
    """The LM-head launch of a decode step (the last projection of Sec. II-A's
    decode phase, producing every greedy token) at 17..64 rows: N = 128,256
    takes the sixteen-wave plan with 2..4 row tiles per wave, N = 32,000 the
    eight-wave plan.  1,024 sampled outputs, the first and last column and row
    included, against the float64 product under the fp32-accumulation bound."""
    K = 4096
    g = torch.Generator().manual_seed(M * 1000 + N % 997)
    X = torch.randn(M, K, generator=g).to(HALF[half])
    W, Wf, Wp = _lm_head_weight(N, K, half)
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    lp.op_gemm(X.to(DEV), Wp, Y, 1, None, N=N)
    torch.cuda.synchronize()
    Yh = Y.cpu().numpy()
    assert not np.isnan(Yh).any()                     # every output written
    rng = np.random.default_rng(M + N)
    rows, cols = rng.integers(0, M, 1024), rng.integers(0, N, 1024)
    rows[:4], cols[:4] = [0, M - 1, 0, M - 1], [0, N - 1, N - 1, 0]
    Xn = X.float().numpy().astype(np.float64)
    Wc = Wf[cols].astype(np.float64)
    ref = np.einsum("ik,ik->i", Xn[rows], Wc)
    bound = 1e-5 * np.einsum("ik,ik->i", np.abs(Xn[rows]), np.abs(Wc))
    assert np.all(np.abs(Yh[rows, cols] - ref) <= bound)
    # whole last column block and whole last row, where the tails are
    Wl = Wf[N - 40:].astype(np.float64)
    ref_c = Xn @ Wl.T
    bnd_c = 1e-5 * (np.abs(Xn) @ np.abs(Wl).T)
    assert np.all(np.abs(Yh[:, N - 40:] - ref_c) <= bnd_c)
    cs = rng.integers(0, N, 4096)
    Wr = Wf[cs].astype(np.float64)
    ref_r = Wr @ Xn[M - 1]
    bnd_r = 1e-5 * (np.abs(Wr) @ np.abs(Xn[M - 1]))
    assert np.all(np.abs(Yh[M - 1, cs] - ref_r) <= bnd_r)


@pytest.mark.parametrize("M,N,K", [(3, 100, 64), (37, 1376, 688), (130, 768, 256)])
def test_gemm_f32(M, N, K):
    rng = np.random.default_rng(K)
    X = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * 0.05).astype(np.float32)
    Y = torch.empty(M, N, dtype=torch.float32, device=DEV)
    lp.op_gemm(to_dev(X, torch.float32), to_dev(W, torch.float32), Y)
    torch.cuda.synchronize()
    ref = X.astype(np.float64) @ W.astype(np.float64).T
    bound = 1e-5 * (np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)).T) + 1e-12
    assert np.all(np.abs(Y.cpu().numpy() - ref) <= bound)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("rows,d,n_part", [(4, 256, 0), (64, 4096, 3), (7, 8192, 0), (33, 5120, 1)])
def test_rmsnorm(dtype, rows, d, n_part):
    rng = np.random.default_rng(rows + d)
    x = (rng.standard_normal((rows, d)) * 3).astype(np.float32)
    part = (rng.standard_normal((max(n_part, 1), rows, d))).astype(np.float32)
    g = rng.uniform(0.5, 1.5, d).astype(np.float32)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    xd = to_dev(x, torch.float32)
    y = torch.empty(rows, d, dtype=tdt, device=DEV)
    lp.op_rmsnorm(xd, to_dev(g, torch.float32), y, 1e-5, to_dev(part, torch.float32) if n_part else None, n_part)
    torch.cuda.synchronize()
    xs = x.astype(np.float64) + (part[:n_part].astype(np.float64).sum(0) if n_part else 0)
    ref = T.rmsnorm(xs, g.astype(np.float64), 1e-5)
    got = y.float().cpu().numpy()
    tol = {"f32": 1e-5, "bf16": 2 ** -8, "f16": 2 ** -10}[dtype]
    assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 1e-6)
    if n_part:
        np.testing.assert_allclose(xd.cpu().numpy(), xs, rtol=1e-6, atol=1e-5)


def test_argmax_ties_and_tail():
    rng = np.random.default_rng(3)
    V = 128256
    logits = rng.standard_normal((9, V)).astype(np.float32)
    logits[0, [5, 77, 128255]] = 50.0      # tie: lowest index wins
    logits[1, V - 1] = 60.0                # last element
    logits[2, :] = 1.0                     # all equal -> 0
    logits[3, 0] = 80.0
    out = torch.empty(9, dtype=torch.int32, device=DEV)
    lp.op_argmax(to_dev(logits, torch.float32), out)
    torch.cuda.synchronize()
    assert out.cpu().numpy().tolist() == [int(np.argmax(r)) for r in logits]
    assert out.cpu().numpy()[:4].tolist() == [5, V - 1, 0, 0]


@pytest.mark.parametrize("V,ld", [(1001, 1001), (4100, 4104), (33, 36), (8192 * 4 + 3, 8192 * 4 + 4)])
def test_argmax_strides_and_tails(V, ld):
    """Row strides that are not a multiple of 4 (scalar path), a partly
    filled last batch of loads, and a tail past the last 16-byte chunk."""
    rng = np.random.default_rng(V)
    full = rng.standard_normal((5, ld)).astype(np.float32)
    full[0, V - 1] = 9.0                   # the last element of the row
    full[1, [3, V - 2]] = 7.0              # tie: lowest index
    full[2, :] = -np.inf                   # all -inf -> 0
    full[:, V:] = 100.0                    # padding past V is never read
    out = torch.empty(5, dtype=torch.int32, device=DEV)
    lp.op_argmax(to_dev(full, torch.float32)[:, :V], out)
    torch.cuda.synchronize()
    assert out.cpu().numpy().tolist() == [int(np.argmax(r[:V])) for r in full]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_device_weight_generator_matches_host(dtype):
    rows, cols, tid, seed = 300, 688, 17, 0x1234ABCD5678
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    dst = torch.empty(rows, cols, dtype=tdt, device=DEV)
    lp.op_init_weight(dst, seed, tid, 0.02)
    torch.cuda.synchronize()
    host = synth.tensor_values(seed, tid, np.arange(rows), cols, 0.02,
                               synth.DTYPE_F32 if dtype == "f32" else synth.DTYPE_BF16)
    got = dst.float().cpu().numpy()  # fp16 storage holds the bf16 values exactly
    assert np.array_equal(got.view(np.uint32), host.view(np.uint32))


# ------------------------------------------------------------------ attention

def make_paged_cache(rng, ctx_lens, Hkv, hd, tdt, extra_blocks=3):
    """Random KV cache in 64-token blocks with shuffled block tables.
    Returns device (kc, vt, block_table) and the host per-slot K/V [ctx, Hkv, hd]."""
    BS = 64
    nb_slot = [(c + BS - 1) // BS for c in ctx_lens]
    n_blocks = sum(nb_slot) + extra_blocks
    perm = rng.permutation(n_blocks)
    max_blocks = max(nb_slot)
    bt = np.zeros((len(ctx_lens), max_blocks), dtype=np.int32)
    kc = bf16_values(rng, (n_blocks, Hkv, BS, hd))
    vt = bf16_values(rng, (n_blocks, Hkv, hd, BS))
    used = 0
    Ks, Vs = [], []
    for s, c in enumerate(ctx_lens):
        blocks = perm[used:used + nb_slot[s]]
        used += nb_slot[s]
        bt[s, :nb_slot[s]] = blocks
        K = np.concatenate([kc[b] for b in blocks], axis=1)[:, :c]            # [Hkv, c, hd]
        V = np.concatenate([vt[b] for b in blocks], axis=2)[:, :, :c]         # [Hkv, hd, c]
        Ks.append(K.transpose(1, 0, 2))
        Vs.append(V.transpose(2, 0, 1))
    return (to_dev(kc, tdt), to_dev(vt, tdt), torch.from_numpy(bt).to(DEV)), Ks, Vs


def attention_tol(dtype, ref, mag):
    """Error bound of the GPU attention: fp32 scores and softmax; the 16-bit
    kernels round the softmax weights P to the element type before P.V (error
    <= u * sum p|v| / sum p, i.e. u times attention over |v|) and round the
    output (u |o|), with u the unit roundoff (2^-8 bf16, 2^-11 fp16)."""
    if dtype == "f32":
        return 2e-5
    u = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -11
    return 2 * u * (mag + np.abs(ref)) + 1e-5


# a full 8B-shape decode batch: 64 rows, lognormal contexts (median about
# 600, clipped to 16..4096) as in the closed-loop workload
FULL_BATCH_CTX = np.clip(np.random.default_rng(8).lognormal(6.4, 0.7, 64), 16, 4096).astype(int).tolist()

DECODE_CASES = [
    # dtype, Hq, Hkv, hd, context lengths
    ("f16", 32, 8, 128, FULL_BATCH_CTX),
    ("bf16", 32, 8, 128, [1, 63, 64, 65, 256, 257, 700, 5120]),
    ("f16", 32, 8, 128, [1, 63, 64, 65, 256, 257, 700, 5120]),
    ("f16", 64, 8, 128, [129, 4096]),
    ("bf16", 8, 8, 128, [300, 2, 1024]),
    ("bf16", 64, 8, 128, [77, 4096]),
    ("bf16", 4, 4, 64, [40, 33]),
    ("f32", 4, 4, 64, [1, 40, 129, 600]),
    ("f32", 8, 2, 64, [64, 65]),
]


@pytest.mark.parametrize("dtype,Hq,Hkv,hd,ctx", DECODE_CASES)
def test_decode_attention(dtype, Hq, Hkv, hd, ctx):
    rng = np.random.default_rng(len(ctx) * 100 + Hq)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    (kc, vt, bt), Ks, Vs = make_paged_cache(rng, ctx, Hkv, hd, tdt)
    M = len(ctx)
    q = bf16_values(rng, (M, Hq, hd))
    out = torch.full((M, Hq, hd), float("nan"), dtype=tdt, device=DEV)
    max_ctx = max(ctx)
    ws = torch.empty(lp.decode_attention_ws_bytes(M, Hq, hd, max_ctx) // 4 + 1, dtype=torch.float32, device=DEV)
    row_slot = torch.arange(M, dtype=torch.int32, device=DEV)
    row_pos = torch.tensor([c - 1 for c in ctx], dtype=torch.int32, device=DEV)
    lp.op_decode_attention(to_dev(q, tdt), out, kc, vt, bt, row_slot, row_pos, Hkv, max_ctx, ws)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    for m, c in enumerate(ctx):
        args = (q[m:m + 1].astype(np.float64), Ks[m].astype(np.float64))
        ref = T.attention(*args, Vs[m].astype(np.float64), [c - 1], np.arange(c), Hkv)[0]
        mag = T.attention(*args, np.abs(Vs[m].astype(np.float64)), [c - 1], np.arange(c), Hkv)[0]
        tol = attention_tol(dtype, ref, mag)
        assert np.all(np.abs(got[m] - ref) <= tol), (m, c, np.max(np.abs(got[m] - ref)))


PREFILL_CASES = [
    ("bf16", 32, 8, 128, [1, 17, 64, 65, 200]),
    ("f16", 32, 8, 128, [1, 17, 64, 65, 200]),
    ("bf16", 8, 8, 128, [130, 3]),
    # one to four prompts take the longest-first tile order: one long prompt,
    # and three of mixed lengths (tiles past a short prompt's end exit)
    ("f16", 32, 8, 128, [700]),
    ("bf16", 32, 8, 128, [300, 5, 129]),
    ("bf16", 4, 4, 64, [32, 32, 32, 32]),
    ("f32", 4, 4, 64, [32, 32, 5, 100]),
    ("f32", 8, 2, 64, [70]),
]


@pytest.mark.parametrize("dtype,Hq,Hkv,hd,lens", PREFILL_CASES)
def test_prefill_attention(dtype, Hq, Hkv, hd, lens):
    rng = np.random.default_rng(sum(lens) + Hq)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    (kc, vt, bt), Ks, Vs = make_paged_cache(rng, lens, Hkv, hd, tdt)
    rows = sum(lens)
    q = bf16_values(rng, (rows, Hq, hd))
    out = torch.full((rows, Hq, hd), float("nan"), dtype=tdt, device=DEV)
    seq_start = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device=DEV)
    seq_slot = torch.arange(len(lens), dtype=torch.int32, device=DEV)
    lp.op_prefill_attention(to_dev(q, tdt), out, kc, vt, bt, seq_start, seq_slot, max(lens), Hkv)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    r0 = 0
    for j, n in enumerate(lens):
        args = (q[r0:r0 + n].astype(np.float64), Ks[j].astype(np.float64))
        ref = T.attention(*args, Vs[j].astype(np.float64), np.arange(n), np.arange(n), Hkv)
        mag = T.attention(*args, np.abs(Vs[j].astype(np.float64)), np.arange(n), np.arange(n), Hkv)
        tol = attention_tol(dtype, ref, mag)
        assert np.all(np.abs(got[r0:r0 + n] - ref) <= tol), (j, np.max(np.abs(got[r0:r0 + n] - ref)))
        r0 += n


def test_zero_row_calls_through_the_binding():
    """Empty device tensors (null data pointers) through the binding: nothing
    is launched and the outputs of other calls are untouched."""
    z16 = torch.empty(0, 256, dtype=torch.float16, device=DEV)
    Wd = torch.zeros(64, 256, dtype=torch.float16, device=DEV)
    Y = torch.empty(0, 64, dtype=torch.float32, device=DEV)
    lp.op_gemm(z16, packed(Wd), Y, 1, None, N=64)
    x = torch.empty(0, 256, dtype=torch.float32, device=DEV)
    g = torch.ones(256, dtype=torch.float32, device=DEV)
    lp.op_rmsnorm(x, g, torch.empty(0, 256, dtype=torch.float16, device=DEV), 1e-5)
    logits = torch.empty(0, 1000, dtype=torch.float32, device=DEV)
    tok = torch.full((4,), -7, dtype=torch.int32, device=DEV)
    lp.op_argmax(logits, tok[:0])
    prm = torch.empty(0, dtype=torch.uint8, device=DEV)
    lp.op_sample(logits, prm, tok[:0])
    torch.cuda.synchronize()
    assert tok.cpu().tolist() == [-7] * 4
