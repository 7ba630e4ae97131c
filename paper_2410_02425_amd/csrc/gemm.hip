// Weight GEMMs Y = X W^T (X: [M x K] activations, W: [N x K] weights, both
// K-contiguous) with fused epilogues.
//
// 16-bit weights are in the tiled layout of kernels.hpp (16 x 32 tiles of
// 1 KB in MFMA operand order); fp32 weights are row-major.
//
//  * gemm_skinny: 16-bit MFMA for decode-sized M <= 64.  The weight matrix is
//    the large operand and is streamed once from HBM, each wave reading its
//    16-row slice tile after tile (1 KB contiguous per load) straight into
//    MFMA operand registers over the workgroup's K range; optional split-K
//    across workgroups writes fp32 partials that a finishing pass (or the
//    next RMSNorm) reduces.
//  * gemm_prefill: 16-bit MFMA for prefill-sized M when K is a multiple of
//    128: 256- or 128-row tiles of 256 columns, eight waves, operands loaded
//    straight from global memory into LDS stage buffers, weight tiles used
//    verbatim as MFMA operands, optional split-K; one workgroup per CU, or
//    two 128-row workgroups per CU for launches of at least 512 tiles.
//  * gemm_big: 16-bit MFMA for the remaining prefill shapes, 128x128x64 tiles
//    staged in LDS.
//  * gemm_f32: fp32 FMA tiles for the fp32 model path (any M).
#include <algorithm>

#include <hip/hip_ext.h>

#include "device.hpp"

namespace lp {


// ------------------------------------------------------------------ skinny (decode)
//
// Decode-sized M (<= 64 rows, MT 16-row tiles).  The weight stream is the whole
// cost: each wave owns NS 16-row slices of W and streams them over the
// workgroup's K range, one sub-chunk (KSUB 32-wide k-steps, one weight tile
// each) ahead of the MFMAs.  With the tiled layout every weight load is 1 KB
// of contiguous memory, and since the tiles of one K step lie side by side
// across the slices, all workgroups, starting together at their K range's
// first sub-chunk, sweep one compact region of the matrix.
// The activations of a sub-chunk are staged once per workgroup into LDS in
// MFMA-fragment order (one 1 KB block per (k-step, m-tile), lane-major), so
// they never occupy the vector-memory counter the weight prefetch waits on;
// each wave loads whole 128-byte row segments of them.
// The loop body has no exit between a prefetch and its use, and prefetches
// past the end re-read the last sub-chunk, so the compiler's wait counts stay
// exact.  Columns of the workgroup's chunk beyond K are zeroed in LDS; the
// weight loads there read valid neighbouring memory and meet those zeros.

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// GATE marks the gate/up launch (SiLU-gate epilogue): the same code under its
// own symbol, so that per-kernel profiles separate it from the other GEMMs.
// KW = 2: the workgroup holds two such groups of NW waves on the same columns,
// each over one half of the workgroup's K range with its own staging, and the
// second hands its sums to the first through LDS before the epilogue.  That
// halves each wave's loop where the MFMAs and fragment reads of 48-64 rows,
// not the weight stream, bound it (8B gate/up at 64 rows: 46.0 -> 43.3 us;
// at 16 or 32 rows it loses 5%).
template <typename T, int MT, int NS, int KSUB, int NW, bool GATE, int KW = 1>
__global__ __launch_bounds__(NW * KW * 64) void gemm_skinny_kernel(const T *__restrict__ X, int64_t ldx,
                                                                  const T *__restrict__ W, int M, int N, int K,
                                                                  int kchunk, float *__restrict__ part, Epi ep) {
  typedef typename Mfma<T>::v8 v8;
  static_assert(KW == 1 || KW == 2, "one or two K-ways");
  constexpr int KC = KSUB * 32;
  constexpr int XT = KSUB * MT * 64;                     // fragment entries per sub-chunk
  constexpr int XF = (XT + NW * 64 - 1) / (NW * 64);     // ... staged per thread
  __shared__ u32x4_t xsa[KW][2][KSUB][MT][64];
  const int kw = KW == 1 ? 0 : (int)threadIdx.x / (NW * 64);
  u32x4_t(&xs0)[KSUB][MT][64] = xsa[kw][0];
  u32x4_t(&xs1)[KSUB][MT][64] = xsa[kw][1];
  const int tid = KW == 1 ? (int)threadIdx.x : (int)threadIdx.x % (NW * 64), wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15;
  const int n0 = (blockIdx.x * NW + wave) * NS * 16;
  // K-way kw covers kchunk / KW of the workgroup's range (kchunk a multiple
  // of 2 KC KW); both K-ways run the same number of sub-chunks
  const int kcw = kchunk / KW;
  const int kbeg = blockIdx.y * kchunk + kw * kcw, kend = min(K, kbeg + kcw);
  const int klen = KW == 1 ? kend - kbeg : kcw;
  const int nsub = ((klen + 2 * KC - 1) / (2 * KC)) * 2;
  // every workgroup has K to cover, so the loop below runs at least once;
  // told so, the compiler keeps the first weight and activation requests
  // ahead of the prologue's barrier instead of sinking them into the loop's
  // preheader behind the first activation round trip
  __builtin_assume(nsub >= 2);
#define SK_SC(c) (kbeg + (c) * KC)
  const int klast = SK_SC(nsub - 1);

  const int64_t wkt = wpack_kt(K);
  const int nsl = (N + WT_ROWS - 1) / WT_ROWS;  // 16-row slices of W
  const T *wrow[NS];
#pragma unroll
  for (int j = 0; j < NS; ++j) wrow[j] = W + (int64_t)min((n0 >> 4) + j, nsl - 1) * WT_ELEMS + lane * 8;
  const int64_t wstep = (int64_t)nsl * WT_ELEMS;  // one tile further along K
  // staging of activation element e (16 bytes): thread e loads row
  // e / (4 KSUB), so a wave reads whole row segments of the sub-chunk, and
  // stores the bytes at their fragment position (k-step ks, m-tile i, lane l)
  const T *xsrc[XF];
  int xk[XF], xd[XF];
#pragma unroll
  for (int f = 0; f < XF; ++f) {
    const int e = min(tid + f * NW * 64, XT - 1);
    const int row = e / (4 * KSUB), c8 = e % (4 * KSUB);
    const int ks = c8 >> 2, i = row >> 4, l = (row & 15) + 16 * (c8 & 3);
    xsrc[f] = X + (int64_t)min(row, M - 1) * ldx;
    xk[f] = c8 * 8;
    xd[f] = (ks * MT + i) * 64 + l;
  }
  floatx4_t acc[MT][NS];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  v8 wA[KSUB][NS], wB[KSUB][NS];
  u32x4_t xA[XF], xB[XF];
  const u32x4_t z4 = {0u, 0u, 0u, 0u};

#define SK_XLOAD(XR, kb)                                                                        \
  _Pragma("unroll") for (int f = 0; f < XF; ++f) XR[f] = *(const u32x4_t *)(xsrc[f] + min((kb) + xk[f], K - 8));
#define SK_XSTORE(XS, XR, kb)                                                                   \
  _Pragma("unroll") for (int f = 0; f < XF; ++f) {                                              \
    const int e = tid + f * NW * 64;                                                            \
    if (XT % (NW * 64) == 0 || e < XT)                                                          \
      (&XS[0][0][0])[xd[f]] = ((kb) + xk[f] < kend) ? XR[f] : z4;                              \
  }
#define SK_WLOAD(WB, kb)                                                                        \
  _Pragma("unroll") for (int ks = 0; ks < KSUB; ++ks) {                                         \
    const int64_t t = min((int64_t)((kb) >> 5) + ks, wkt - 1);                                  \
    _Pragma("unroll") for (int j = 0; j < NS; ++j) WB[ks][j] = load8<T>(wrow[j] + t * wstep);    \
  }
#define SK_MMA(WB, XS)                                                                          \
  _Pragma("unroll") for (int ks = 0; ks < KSUB; ++ks) {                                         \
    _Pragma("unroll") for (int i = 0; i < MT; ++i) {                                            \
      const v8 a = __builtin_bit_cast(v8, XS[ks][i][lane]);                                     \
      _Pragma("unroll") for (int j = 0; j < NS; ++j) acc[i][j] = Mfma<T>::m16(a, WB[ks][j], acc[i][j]); \
    }                                                                                           \
  }
#define SK_SB __builtin_amdgcn_sched_barrier(0);

  SK_XLOAD(xA, SK_SC(0))
  SK_WLOAD(wA, SK_SC(0))
  SK_XLOAD(xB, SK_SC(1))
  SK_XSTORE(xs0, xA, SK_SC(0))
  __syncthreads();
  for (int c = 0; c < nsub; c += 2) {
    SK_SB
    SK_WLOAD(wB, SK_SC(c + 1))
    SK_XLOAD(xA, c + 2 < nsub ? SK_SC(c + 2) : klast)
    SK_SB
    SK_MMA(wA, xs0)
    SK_SB
    SK_XSTORE(xs1, xB, SK_SC(c + 1))
    __syncthreads();
    SK_SB
    SK_WLOAD(wA, c + 2 < nsub ? SK_SC(c + 2) : klast)
    SK_XLOAD(xB, c + 3 < nsub ? SK_SC(c + 3) : klast)
    SK_SB
    SK_MMA(wB, xs1)
    SK_SB
    SK_XSTORE(xs0, xA, c + 2 < nsub ? SK_SC(c + 2) : kend)
    __syncthreads();
  }
#undef SK_SC
#undef SK_XLOAD
#undef SK_XSTORE
#undef SK_WLOAD
#undef SK_MMA
#undef SK_SB

  if constexpr (KW == 2) {
    // the second K-way's sums go to the first through the staging buffers
    static_assert(sizeof(xsa) >= (size_t)NW * 64 * MT * NS * 4 * sizeof(float), "reduction space");
    float *red = (float *)&xsa[0][0][0][0][0];
    __syncthreads();
    if (kw == 1) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) red[(((wave * MT + i) * NS + j) * 4 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (kw == 1) return;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NS; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][j][r] += red[(((wave * MT + i) * NS + j) * 4 + r) * 64 + lane];
  }
  const bool split = gridDim.y > 1;
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int n = n0 + j * 16 + r16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = i * 16 + (lane >> 4) * 4 + r;
        const float v = acc[i][j][r];
        const float other = lane_xor1(v);
        if (split) {
          if (m < M && n < N) part[((int64_t)blockIdx.y * M + m) * N + n] = v;
        } else if ((lane & 1) == 0 && m < M && n < N) {
          epi_pair<T>(ep, m, n, v, other);
        }
      }
    }
}

// ------------------------------------------------------------------ split-K finish

template <typename T>
__global__ void gemm_finish_kernel(const float *__restrict__ part, int splits, int M, int N, Epi ep) {
  const int64_t half = (int64_t)N / 2;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= (int64_t)M * half) return;
  const int m = (int)(p / half);
  const int n = (int)(p % half) * 2;
  // partials are requested eight splits at a time before any is added, and
  // added in split order
  constexpr int U = 8;
  float v0 = 0.f, v1 = 0.f;
  for (int s0 = 0; s0 < splits; s0 += U) {
    float2 q[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      q[u] = *(const float2 *)(part + ((int64_t)min(s0 + u, splits - 1) * M + m) * N + n);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (s0 + u < splits) {
        v0 += q[u].x;
        v1 += q[u].y;
      }
  }
  epi_pair<T>(ep, m, n, v0, v1);
}

template <typename T>
void launch_gemm_finish(const float *part, int splits, int M, int N, const Epi &ep, hipStream_t s) {
  const int64_t pairs = (int64_t)M * (N / 2);
  if (pairs <= 0) return;
  gemm_finish_kernel<T><<<(unsigned)((pairs + 255) / 256), 256, 0, s>>>(part, splits, M, N, ep);
}

// ------------------------------------------------------------------ big (prefill)

constexpr int BG_BM = 128, BG_BN = 128, BG_BK = 64, BG_LDS = BG_BK + 8;

template <typename T>
__global__ __launch_bounds__(256) void gemm_big_kernel(const T *__restrict__ X, int64_t ldx,
                                                       const T *__restrict__ W, int M, int N,
                                                       int K, Epi ep) {
  typedef typename Mfma<T>::v8 v8;
  __shared__ T As[BG_BM][BG_LDS];
  __shared__ T Bs[BG_BN][BG_LDS];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BG_BM, n0 = blockIdx.x * BG_BN;
  const int64_t wns = wpack_ns(N);

  // global -> register staging: each thread moves 4 chunks of 16 B for A and B
  uint4 ra[4], rb[4];
#define BG_GLOAD(k0)                                                                            \
  _Pragma("unroll") for (int c = 0; c < 4; ++c) {                                               \
    const int idx = tid + c * 256;                                                              \
    const int row = idx >> 3, kk = (k0) + (idx & 7) * 8;                                        \
    const int m = m0 + row, n = n0 + row;                                                       \
    ra[c] = (m < M && kk < K) ? *(const uint4 *)(X + (int64_t)m * ldx + kk) : make_uint4(0, 0, 0, 0); \
    rb[c] = (n < N && kk < K) ? *(const uint4 *)(W + wpack_off(n, kk, wns)) : make_uint4(0, 0, 0, 0); \
  }
  floatx16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  BG_GLOAD(0)
  for (int k0 = 0; k0 < K; k0 += BG_BK) {
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int idx = tid + c * 256;
      const int row = idx >> 3, kc = (idx & 7) * 8;
      *(uint4 *)&As[row][kc] = ra[c];
      *(uint4 *)&Bs[row][kc] = rb[c];
    }
    __syncthreads();
    if (k0 + BG_BK < K) {
      BG_GLOAD(k0 + BG_BK)
    }
#pragma unroll
    for (int ks = 0; ks < BG_BK / 16; ++ks) {
      v8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = load8<T>(&As[wm * 64 + i * 32 + (lane & 31)][ks * 16 + (lane >> 5) * 8]);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = load8<T>(&Bs[wn * 64 + j * 32 + (lane & 31)][ks * 16 + (lane >> 5) * 8]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = Mfma<T>::m32(a[i], b[j], acc[i][j]);
    }
  }

  // epilogue through LDS: each wave stages one 32x32 tile at a time, then its
  // lanes apply the epilogue to column pairs
  __syncthreads();
  float *stage = (float *)&As[0][0] + wave * 32 * 33;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[((r & 3) + 4 * (lane >> 5) + 8 * (r >> 2)) * 33 + (lane & 31)] = acc[i][j][r];
      __syncthreads();
      for (int p = lane; p < 32 * 16; p += 64) {
        const int row = p >> 4, c = (p & 15) * 2;
        const int m = m0 + wm * 64 + i * 32 + row;
        const int n = n0 + wn * 64 + j * 32 + c;
        if (m < M && n < N) epi_pair<T>(ep, m, n, stage[row * 33 + c], stage[row * 33 + c + 1]);
      }
      __syncthreads();
    }
}

// ------------------------------------------------------------------ prefill (M > 64)
//
// BM x 256 output tiles (BM = 256 or 128), eight waves (4 x 2, each BM/4 x 128
// = BM/64 x 8 MFMA 16x16x32 tiles), 32-wide K stages.  Operands travel from global memory
// straight into LDS (global_load_lds_dwordx4: each lane's 16 bytes land at
// the instruction's LDS base + 16 x lane), with no register staging and no LDS
// store instructions.  NB stage buffers, NB - 1 stages in flight: at each
// stage a wave waits for its own loads of that stage (the in-order vmcnt
// counter, with the younger stages still outstanding), then a barrier makes
// every wave's loads visible, and the buffer freed by the previous stage is
// refilled before the MFMAs run.
//   * One workgroup per CU (NB = 4, 128 or 96 KB of LDS): the 128-row tile
//     reads the next stage's fragments while the MFMAs of the current one
//     run (two fragment sets).
//   * Two workgroups per CU (BM = 128, NB = 3, 72 KB of LDS, at most 128
//     registers a wave): each workgroup's barriers and epilogue then overlap
//     the other's MFMAs, which measured 4-8% faster once a GEMM has at least
//     two tiles per CU.
//   * A weight stage is one tile per 16-row slice, copied verbatim: its lanes
//     are already the B operand of a 16x16x32 MFMA, and the 16 tiles of a
//     stage lie side by side in memory.
//   * An activation stage holds BM rows of 64 bytes.  The four 16-byte
//     chunks of row r are stored XOR-swizzled by (r / 4) % 4, by choosing the
//     global address each lane loads, so that the 16-row fragment reads are
//     free of bank conflicts.
// More workgroups than output tiles split K: fp32 partials [z][M][N] replace
// the epilogue.  Rows and columns past M / N read clamped (valid) memory and
// are never stored; loads past the last stage re-read it into a buffer nobody
// reads, so every wave's load count (and the wait count) is the same at every
// stage.  K must be a multiple of 128.

constexpr int PF_BN = 256, PF_BK = 32, PF_NT = 512;
constexpr int PF_KQ = 128;  // K granularity of a split

// Waits until at most N vector loads of this wave remain, then joins the
// workgroup barrier (LDS reads drained first).
template <int N>
__device__ __forceinline__ void prefill_wait_barrier() {
  static_assert(N == 3 || N == 6 || N == 8, "stage wait count");
  if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else if constexpr (N == 6) asm volatile("s_waitcnt vmcnt(6) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(3) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Rows of a prefill epilogue pass whose global loads are requested together
// (a register budget of 128 VGPRs, two workgroups per CU, allows 8).
constexpr int PF_EPI_ROWS = 8;

// One 16-row MFMA tile row of a prefill wave's accumulators (16 x 128 fp32)
// into the wave's staging area, row-major with a row stride of PF_STG floats:
// the 4-float pad puts the 16 rows of one column in distinct LDS banks, for
// the column-wise reads of the V epilogue.
constexpr int PF_STG = 132;
__device__ __forceinline__ void prefill_stage16(const floatx4_t (&acc)[8], float *stg, int lane) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) stg[((lane >> 4) * 4 + r) * PF_STG + j * 16 + (lane & 15)] = acc[j][r];
}

// QKV epilogue of a prefill tile for one wave: rows wrow .. wrow + 16 TM - 1,
// this lane's column pair (n, n + 1).  Lane l < 16 TM looks up the KV slot,
// position and cache block of row wrow + l once, and every row reads them
// back with readlane; the rotary factors of PF_EPI_ROWS rows are requested
// before the first of their stores.  Same arithmetic and results as epi_pair.
template <typename T, int TM>
__device__ __forceinline__ void prefill_epi_qkv(const Epi &ep, const floatx4_t (&acc)[TM][8], float *stg, int wrow,
                                                int n, int M, int N, int lane) {
  const int hd = ep.kv.head_dim, half = hd >> 1;
  const int qdim = ep.n_heads * hd, kvdim = ep.kv.n_kv_heads * hd;
  int pos_l = 0, blk_l = 0;
  if (lane < 16 * TM && wrow + lane < M) {
    const int m = wrow + lane;
    const int slot = ep.rows.row_slot[m];
    pos_l = ep.rows.row_pos[m];
    blk_l = ep.kv.block_table[(int64_t)slot * ep.kv.max_blocks + pos_l / KV_BLOCK];
  }
  const bool ok = n < N, is_q = n < qdim, is_v = n >= qdim + kvdim;
  const int c = is_q ? n : (is_v ? n - qdim - kvdim : n - qdim);
  const int h = c / hd, j = c % hd, i = j >> 1;
  const int64_t layer_blocks = (int64_t)ep.layer * ep.kv.n_blocks;
  // A wave whose 128 columns are one whole V head writes the transposed
  // cache column-wise: lane (d4, r) = (lane / 16, lane % 16) stores row r's
  // dimensions 4 k + d4, so one store covers 16 consecutive rows (positions)
  // of four dimensions instead of one row across 128 scattered ones.
  const int n0 = n - lane * 2;  // the wave's first column
  if (hd == 128 && n0 >= qdim + kvdim && n0 + 128 <= N) {
    const int r = lane & 15, d4 = lane >> 4;
    const int hv = (n0 - qdim - kvdim) / hd;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      prefill_stage16(acc[t], stg, lane);
      const int pos = __shfl(pos_l, t * 16 + r, 64);
      const int blk = __shfl(blk_l, t * 16 + r, 64);
      const bool live = wrow + t * 16 + r < M;
      T *vt = (T *)ep.kv.v + ((layer_blocks + blk) * ep.kv.n_kv_heads + hv) * (int64_t)KV_BLOCK * hd + pos % KV_BLOCK;
      __syncthreads();
#pragma unroll 16
      for (int k = 0; k < 32; ++k) {
        const float v = stg[r * PF_STG + 4 * k + d4];
        if (live) vt[(int64_t)(4 * k + d4) * KV_BLOCK] = Act<T>::st(v);
      }
      __syncthreads();
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    prefill_stage16(acc[t], stg, lane);
    __syncthreads();
#pragma unroll
    for (int g = 0; g < 16; g += PF_EPI_ROWS) {
      float cs[PF_EPI_ROWS], sn[PF_EPI_ROWS];
#pragma unroll
      for (int u = 0; u < PF_EPI_ROWS; ++u) {
        const int pos = __builtin_amdgcn_readlane(pos_l, t * 16 + g + u);
        const bool rot = ok && !is_v && wrow + t * 16 + g + u < M;
        cs[u] = rot ? ep.rope_cos[(int64_t)pos * half + i] : 0.f;
        sn[u] = rot ? ep.rope_sin[(int64_t)pos * half + i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < PF_EPI_ROWS; ++u) {
        const int row = g + u, m = wrow + t * 16 + row;
        const int pos = __builtin_amdgcn_readlane(pos_l, t * 16 + row);
        const int blk = __builtin_amdgcn_readlane(blk_l, t * 16 + row);
        const float2 v = *(const float2 *)(stg + row * PF_STG + lane * 2);
        if (m < M && ok) {
          const int64_t cb = ((layer_blocks + blk) * ep.kv.n_kv_heads + h) * (int64_t)KV_BLOCK * hd;
          if (is_v) {
            T *vt = (T *)ep.kv.v + cb + pos % KV_BLOCK;
            vt[(int64_t)j * KV_BLOCK] = Act<T>::st(v.x);
            vt[(int64_t)(j + 1) * KV_BLOCK] = Act<T>::st(v.y);
          } else {
            float r0, r1;
            rope_rotate(v.x, v.y, cs[u], sn[u], r0, r1);
            T *dst = is_q ? (T *)ep.act_out + (int64_t)m * ep.ld_act + h * hd
                          : (T *)ep.kv.k + cb + (int64_t)(pos % KV_BLOCK) * hd;
            dst[i] = Act<T>::st(r0);
            dst[i + half] = Act<T>::st(r1);
          }
        }
      }
    }
    __syncthreads();
  }
}

// NB stage buffers; WPE waves per SIMD the registers are budgeted for (2: one
// workgroup per CU, 4: two).
template <typename T, int BM, int NB, int WPE>
__global__ __launch_bounds__(PF_NT, WPE) void gemm_prefill_kernel(const T *__restrict__ X, int64_t ldx,
                                                             const T *__restrict__ W, int M, int N, int K,
                                                             int kchunk, float *__restrict__ part, Epi ep,
                                                             int xg, int gx) {
  typedef typename Mfma<T>::v8 v8;
  constexpr int TM = BM / 64;                            // 16-row MFMA tiles per wave
  constexpr int PA = BM / 128;                           // activation loads per wave and stage
  constexpr int ABYTES = BM * PF_BK * 2;                 // activation bytes per stage
  constexpr int SBYTES = (BM + PF_BN) * PF_BK * 2;       // bytes per stage buffer
  __shared__ __attribute__((aligned(1024))) char lds[NB * SBYTES];
  static_assert(NB * SBYTES >= 8 * 16 * PF_STG * 4, "the epilogue stages 16 rows per wave in the stage buffers");
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;
  // 1-D grid over gx column tiles (the weight's, or that count rounded up
  // to a multiple of 8; workgroups of the padding columns exit at once).
  // Workgroup i runs on XCD i % 8, so with gx a multiple of 8 every row tile
  // of a column runs on one XCD and shares its L2.  xg == 0: plain order,
  // column tile fastest.  xg > 0 (gx a multiple of 8): XCD-aware order; each
  // XCD takes every eighth column tile, and its i / 8-th workgroup walks
  // groups of xg row tiles, row tile fastest inside a group and then the
  // XCD's column tiles.  The rows of a group share the XCD's L2 and stay in
  // the last-level cache while the XCD's weight columns pass.
  int bx, by, bz;
  const int gxw = (N + PF_BN - 1) / PF_BN, gy = (M + BM - 1) / BM;
  const bool split = (int)gridDim.x > gx * gy;  // K split over gridDim.x / (gx gy) ranges
  {
    const int lin = blockIdx.x;
    if (xg > 0) {
      const int cx = gx / 8, t = lin / 8;
      bz = t / (cx * gy);
      int r = t % (cx * gy);
      const int g0 = r / (xg * cx) * xg, ge = min(xg, gy - g0);  // the group's first row tile, its size
      r -= g0 * cx;
      by = g0 + r % ge;
      bx = r / ge * 8 + lin % 8;
    } else {
      bx = lin % gx;
      by = (lin / gx) % gy;
      bz = lin / (gx * gy);
    }
  }
  if (bx >= gxw) return;  // a padding column: no tile, before any barrier
  const int m0 = by * BM, n0 = bx * PF_BN;
  const int kb = bz * kchunk, ke = min(K, kb + kchunk);
  const int nk = (ke - kb) / PF_BK;
  const int nsl = (N + WT_ROWS - 1) / WT_ROWS;
  const int64_t wstep = (int64_t)nsl * WT_ELEMS;  // one tile further along K
  const uint32_t lds0 = lds_addr(lds);

  // this wave's share of a stage: PA 1 KB blocks of activations (16 rows
  // each) and two weight tiles
  const T *ga[PA];
  const T *gw[2];
  uint32_t la[PA], lw[2];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int blk = wave * PA + i;
    const int row = blk * 16 + (lane >> 2), slot = lane & 3;
    const int q = slot ^ ((row >> 2) & 3);  // the K chunk that this LDS slot holds
    ga[i] = X + (int64_t)min(m0 + row, M - 1) * ldx + kb + q * 8;
    la[i] = (uint32_t)__builtin_amdgcn_readfirstlane((int)(lds0 + blk * 1024));
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int blk = wave * 2 + i;
    gw[i] = W + ((int64_t)(kb / WT_COLS) * nsl + min((n0 >> 4) + blk, nsl - 1)) * WT_ELEMS + lane * 8;
    lw[i] = (uint32_t)__builtin_amdgcn_readfirstlane((int)(lds0 + ABYTES + blk * 1024));
  }
#define PF_ISSUE(kt)                                                                                 \
  {                                                                                                  \
    const int s_ = min((kt), nk - 1);                                                                \
    const uint32_t b_ = (uint32_t)(((kt) % NB) * SBYTES);                                           \
    _Pragma("unroll") for (int i = 0; i < PA; ++i) dma16(ga[i] + s_ * PF_BK, la[i] + b_);            \
    _Pragma("unroll") for (int i = 0; i < 2; ++i) dma16(gw[i] + s_ * wstep, lw[i] + b_);             \
  }
  floatx4_t acc[TM][8];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  int fa[TM];  // byte offsets of this lane's activation fragments in a stage
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * (BM / 4) + i * 16 + (lane & 15), q = lane >> 4;
    fa[i] = r * 64 + ((q ^ ((r >> 2) & 3)) << 4);
  }
  const int fb = ABYTES + wn * 8 * 1024 + lane * 16;

  // PA + 2 loads per stage and wave: with the NB - 2 younger stages' loads
  // still allowed outstanding, the oldest stage has landed; the barrier then
  // makes every wave's loads of it visible
#define PF_WAIT_BAR() prefill_wait_barrier<(PA + 2) * (NB - 2)>();
#define PF_READ(A, B, kt)                                                                          \
  {                                                                                                \
    const char *st_ = lds + ((kt) % NB) * SBYTES;                                                  \
    _Pragma("unroll") for (int i = 0; i < TM; ++i) A[i] = *(const v8 *)(st_ + fa[i]);              \
    _Pragma("unroll") for (int j = 0; j < 8; ++j) B[j] = *(const v8 *)(st_ + fb + j * 1024);       \
  }
#define PF_MMA(A, B)                                                                               \
  _Pragma("unroll") for (int i = 0; i < TM; ++i)                                                   \
    _Pragma("unroll") for (int j = 0; j < 8; ++j) acc[i][j] = Mfma<T>::m16(A[i], B[j], acc[i][j]);
#pragma unroll
  for (int p = 0; p < NB - 1; ++p) PF_ISSUE(p)
  if constexpr (BM == 128 && WPE == 2) {
    // software pipeline: stage kt+1's fragments are read into the other
    // register set while the MFMAs of stage kt run (two fragment sets fit
    // beside 128-row accumulators in a one-workgroup-per-CU register budget;
    // with 256 rows, or two workgroups per CU, they would spill)
    v8 a0[TM], b0[8], a1[TM], b1[8];
    PF_WAIT_BAR()
    PF_READ(a0, b0, 0)
    for (int kt = 0; kt < nk; kt += 2) {
      PF_ISSUE(kt + NB - 1)
      PF_WAIT_BAR()
      PF_READ(a1, b1, kt + 1)
      PF_MMA(a0, b0)
      if (kt + 1 >= nk) break;
      PF_ISSUE(kt + NB)
      PF_WAIT_BAR()
      PF_READ(a0, b0, kt + 2)
      PF_MMA(a1, b1)
    }
  } else {
    for (int kt = 0; kt < nk; ++kt) {
      PF_WAIT_BAR()
      PF_ISSUE(kt + NB - 1)
      v8 a[TM], b[8];
      PF_READ(a, b, kt)
      PF_MMA(a, b)
    }
  }
#undef PF_WAIT_BAR
#undef PF_READ
#undef PF_MMA
#undef PF_ISSUE
  // the last (re-read) stages land before LDS is reused below
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

  // accumulator (i, j) of lane l: row 4 (l / 16) + r of 16-row tile i, column l % 16 of tile j
  const int wrow = m0 + wm * (BM / 4), wcol = n0 + wn * 128;
  if (split) {
    float *pz = part + (int64_t)bz * M * N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int n = wcol + j * 16 + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = wrow + i * 16 + (lane >> 4) * 4 + r;
          if (m < M && n < N) pz[(int64_t)m * N + n] = acc[i][j][r];
        }
      }
    return;
  }
  // epilogue through LDS: each wave stages 16 rows x 128 columns of fp32 at a
  // time in its own 8.25 KB, then its lanes apply the epilogue to column pairs,
  // one 128-column row per pass of the wave.  What a pass reads from global
  // memory (residual rows, rotary factors, row metadata) is requested before
  // its first store: a load issued behind a store also waits for the store.
  float *stg = (float *)lds + wave * 16 * PF_STG;
  const int n = wcol + lane * 2;
  if (ep.kind == EPI_QKV) {
    prefill_epi_qkv<T, TM>(ep, acc, stg, wrow, n, M, N, lane);
    return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    prefill_stage16(acc[i], stg, lane);
    __syncthreads();
    if (ep.kind == EPI_RESID) {
#pragma unroll
      for (int g = 0; g < 16; g += PF_EPI_ROWS) {
        float2 r[PF_EPI_ROWS];
#pragma unroll
        for (int u = 0; u < PF_EPI_ROWS; ++u) {
          const int m = wrow + i * 16 + g + u;
          r[u] = (m < M && n < N) ? *(const float2 *)(ep.out + (int64_t)m * ep.ldo + n) : make_float2(0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < PF_EPI_ROWS; ++u) {
          const int m = wrow + i * 16 + g + u;
          const float2 v = *(const float2 *)(stg + (g + u) * PF_STG + lane * 2);
          if (m < M && n < N) {
            r[u].x += v.x;
            r[u].y += v.y;
            *(float2 *)(ep.out + (int64_t)m * ep.ldo + n) = r[u];
          }
        }
      }
    } else {
      for (int row = 0; row < 16; ++row) {
        const int m = wrow + i * 16 + row;
        const float2 v = *(const float2 *)(stg + row * PF_STG + lane * 2);
        if (m < M && n < N) epi_pair<T>(ep, m, n, v.x, v.y);
      }
    }
    __syncthreads();
  }
}

// Tile rows, K splits and workgroups per CU of a prefill GEMM, chosen by an
// estimate of its time.
//   * One workgroup per CU: the rounds of workgroups over the 256 CUs times
//     one tile's time at the tile shape's per-CU rate (PF_RATE_256,
//     PF_RATE_128), plus the fp32 partials of a split written and read once
//     (PF_FOLD_RATE, the folding pass included).  Splits of 1 to 8, keeping
//     at least 1024 K each.
//   * Two 128-row workgroups per CU (only with at least 512 tiles and no
//     split: with fewer, the dispatcher pairs workgroups on some CUs while
//     others idle): full rounds of 512 tiles at PF_RATE_PAIR per CU, then a
//     remainder of at most 256 tiles one per CU at the 128-row rate, or a
//     larger one as one more paired round.
// The rates were fitted to a sweep of every plan (tile rows, 1-8 splits,
// paired or not), each timed with the pass that consumes its partials, for
// the projections of the 8B, 13B and 70B shapes at M = 150..38,156: the plan
// picked is on average 0.15% (8B up to 4,223 rows), 0.6% (13B, 70B) and 0.6%
// (8B, 3,000 to 38,156 rows) slower than the best measured one, 9% at worst
// (13B down at M = 1,067), against 1.7%, 2.7% and 2.0% for the earlier rates
// (4.5, 4.8, 4.86 TFLOP/s, partials at 5 TB/s).
static constexpr double PF_RATE_128 = 4.1e12, PF_RATE_256 = 5.2e12, PF_RATE_PAIR = 4.86e12;  // flop/s per CU
static constexpr double PF_FOLD_RATE = 4.0e12;  // bytes/s of split partials, written and read back
static int prefill_kchunk(int K, int s) { return (K / s + PF_KQ - 1) / PF_KQ * PF_KQ; }

static double prefill_cost(int M, int N, int K, int bm, int s) {
  const int kchunk = prefill_kchunk(K, s);
  const int se = (K + kchunk - 1) / kchunk;
  const int64_t wgs = (int64_t)((M + bm - 1) / bm) * ((N + PF_BN - 1) / PF_BN) * se;
  const double rounds = (double)((wgs + 255) / 256);
  const double rate = bm == 256 ? PF_RATE_256 : PF_RATE_128;
  const double partials = se > 1 ? 2.0 * se * M * N * 4 / PF_FOLD_RATE : 0.0;
  return rounds * (2.0 * bm * PF_BN * kchunk / rate) + partials;
}

static constexpr int64_t PF_PAIR_MIN_TILES = 512;
static constexpr int64_t PF_LLC_BYTES = 256ll << 20;  // MI355X last-level (Infinity) cache

// Column tiles the prefill grid is laid out over, and row tiles per XCD
// group of its tile order (0: plain order), for a 16-bit [N x K] weight with
// bm-row tiles; the reasons are at the launch.
static int prefill_grid_columns(int N) {
  const int gx = (N + PF_BN - 1) / PF_BN;
  return gx >= 64 ? (gx + 7) / 8 * 8 : gx;
}
static int prefill_xcd_group(int N, int K, int bm) {
  const bool wide = (N + PF_BN - 1) / PF_BN >= 64;
  return (wide && (bm == 256 || (int64_t)N * K * 2 > PF_LLC_BYTES)) ? 16 : 0;
}

static double prefill_pair_cost(int M, int N, int K) {
  const int64_t tiles = (int64_t)((M + 127) / 128) * ((N + PF_BN - 1) / PF_BN);
  if (tiles < PF_PAIR_MIN_TILES) return -1.0;
  const double flops = 2.0 * 128 * PF_BN * K;
  const int64_t rest = tiles % 512;
  const double tail = rest == 0 ? 0.0 : (rest <= 256 ? flops / PF_RATE_128 : 2.0 * flops / PF_RATE_PAIR);
  return (double)(tiles / 512) * 2.0 * flops / PF_RATE_PAIR + tail;
}

struct PrefillPlan {
  int bm, splits;
  bool pair;  // two 128-row workgroups per CU
};

// splits > 0: the caller's split request (rounded to whole K chunks as
// gemm_effective_splits does), only the tile shape is chosen; splits == 0:
// both are chosen, from 1, 2 or 4 splits.
static PrefillPlan prefill_plan(int M, int N, int K, int splits) {
  PrefillPlan best{256, 1, false};
  if (M <= 64 || K % PF_KQ != 0) return best;
  double tbest = -1.0;
  for (int s = 1; s <= 8; ++s) {
    if (splits > 0 ? s != 1 : (s > 1 && K / s < 1024)) continue;
    const int req = splits > 0 ? splits : s;
    for (int bm : {256, 128}) {
      const double t = prefill_cost(M, N, K, bm, req);
      if (tbest < 0.0 || t < tbest) {
        tbest = t;
        const int kchunk = prefill_kchunk(K, req);
        best = {bm, (K + kchunk - 1) / kchunk, false};
      }
    }
  }
  if (splits <= 1) {
    const double t = prefill_pair_cost(M, N, K);
    if (t >= 0.0 && t < tbest) best = {128, 1, true};
  }
  return best;
}

int prefill_gemm_splits(int M, int N, int K) { return prefill_plan(M, N, K, 0).splits; }

// ------------------------------------------------------------------ fp32 path

constexpr int F_BM = 64, F_BN = 64, F_BK = 16;

__global__ __launch_bounds__(256) void gemm_f32_kernel(const float *__restrict__ X, int64_t ldx,
                                                       const float *__restrict__ W, int M, int N, int K,
                                                       Epi ep) {
  __shared__ float Xs[F_BK][F_BM + 4];
  __shared__ float Ws[F_BK][F_BN + 4];
  const int tid = threadIdx.x;
  const int ty = tid >> 4, tx = tid & 15;
  const int m0 = blockIdx.y * F_BM, n0 = blockIdx.x * F_BN;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += F_BK) {
    {
      const int row = tid >> 2, kk = (tid & 3) * 4;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = k0 + kk + u;
        const int m = m0 + row, n = n0 + row;
        Xs[kk + u][row] = (m < M && k < K) ? X[(int64_t)m * ldx + k] : 0.f;
        Ws[kk + u][row] = (n < N && k < K) ? W[(int64_t)n * K + k] : 0.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < F_BK; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = Xs[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Ws[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; j += 2) {
      const int n = n0 + tx * 4 + j;
      if (n < N) epi_pair<float>(ep, m, n, acc[i][j], acc[i][j + 1]);
    }
  }
}

// ------------------------------------------------------------------ dispatch

// Launch shapes of the decode kernel, chosen from the weight matrix shape by
// measured sweeps: one 16-column slice per wave and two weight tiles per
// sub-chunk, eight waves per workgroup sharing the staged activations; for
// the largest N (the LM head) sixteen waves with one tile per sub-chunk.
struct SkinnyPlan {
  int ns, ksub, nw, splits, kchunk;
};

SkinnyPlan skinny_plan(int N, int K, int want_splits) {
  SkinnyPlan p;
  if (N >= 65536) {
    p = {1, 1, 16, 1, 0};
  } else {
    p = {1, 2, 8, 1, 0};
  }
  const int KC2 = 2 * p.ksub * 32;
  int s = std::max(1, want_splits);
  int kchunk = (K + s - 1) / s;
  kchunk = (kchunk + KC2 - 1) / KC2 * KC2;
  p.kchunk = kchunk;
  p.splits = (K + kchunk - 1) / kchunk;
  return p;
}

int skinny_effective_splits(int N, int K, int splits) { return skinny_plan(N, K, splits).splits; }

void gemm_plan_info(int M, int N, int K, int splits, int *kind, int *rows, int *eff_splits, int *xcd_group) {
  *xcd_group = 0;
  if (M <= 64) {
    *kind = GEMM_KIND_DECODE;
    *rows = 16 * ((M + 15) / 16);
    *eff_splits = gemm_effective_splits(M, N, K, splits);
  } else if (K % PF_KQ == 0) {
    // 0: the engine's own choice (prefill_gemm_splits), otherwise lp_op_gemm's
    const int s = splits == 0 ? prefill_gemm_splits(M, N, K) : (splits < 1 ? 1 : gemm_effective_splits(M, N, K, splits));
    const PrefillPlan p = prefill_plan(M, N, K, s);
    *kind = p.pair ? GEMM_KIND_PREFILL_PAIR : GEMM_KIND_PREFILL;
    *rows = p.bm;
    *eff_splits = p.splits;
    *xcd_group = prefill_xcd_group(N, K, p.bm);
  } else {
    *kind = GEMM_KIND_TILED;
    *rows = BG_BM;
    *eff_splits = 1;
  }
}

int gemm_effective_splits(int M, int N, int K, int splits) {
  if (splits <= 1) return 1;
  if (M <= 64) return skinny_effective_splits(N, K, splits);
  if (K % PF_KQ != 0) return 1;
  const int kchunk = (K / splits + PF_KQ - 1) / PF_KQ * PF_KQ;
  return (K + kchunk - 1) / kchunk;
}

// Launches a kernel plainly, or with two events bound to its own dispatch.
template <typename... KArgs, typename... Args>
static void launch_k(void (*k)(KArgs...), dim3 grid, dim3 block, hipStream_t s, const hipEvent_t *timing,
                     Args... args) {
  if (timing)
    hipExtLaunchKernelGGL(k, grid, block, 0, s, timing[0], timing[1], 0, static_cast<KArgs>(args)...);
  else
    k<<<grid, block, 0, s>>>(static_cast<KArgs>(args)...);
}

template <typename T, int MT>
static void launch_skinny_mt(const T *X, int64_t ldx, const T *W, int M, int N, int K, int splits, float *part,
                             const Epi &ep, hipStream_t s, const hipEvent_t *timing) {
  const SkinnyPlan p = skinny_plan(N, K, splits);
  const int cols = p.nw * p.ns * 16;
  dim3 grid((N + cols - 1) / cols, p.splits);
  if constexpr (MT >= 3) {
    // gate/up over 33-64 rows: two K-ways a workgroup (K range a multiple of 256)
    if (p.nw == 8 && ep.kind == EPI_SILU && p.splits == 1 && p.kchunk % (2 * 2 * p.ksub * 32) == 0) {
      launch_k(gemm_skinny_kernel<T, MT, 1, 2, 8, true, 2>, grid, 2 * 8 * 64, s, timing, X, ldx, W, M, N, K,
               p.kchunk, part, ep);
      return;
    }
  }
  if (p.nw == 16)
    launch_k(gemm_skinny_kernel<T, MT, 1, 1, 16, false>, grid, 16 * 64, s, timing, X, ldx, W, M, N, K, p.kchunk,
             part, ep);
  else if (ep.kind == EPI_SILU && p.splits == 1)
    launch_k(gemm_skinny_kernel<T, MT, 1, 2, 8, true>, grid, 8 * 64, s, timing, X, ldx, W, M, N, K, p.kchunk,
             part, ep);
  else
    launch_k(gemm_skinny_kernel<T, MT, 1, 2, 8, false>, grid, 8 * 64, s, timing, X, ldx, W, M, N, K, p.kchunk,
             part, ep);
}

template <typename T>
static void launch_gemm_mfma(const T *X, int64_t ldx, const T *W, int M, int N, int K, int splits, float *part,
                             const Epi &ep, hipStream_t s, const hipEvent_t *timing) {
  if (M <= 0 || N <= 0) return;
  if (M <= 64) {
    if (splits < 1 || part == nullptr) splits = 1;
    switch ((M + 15) / 16) {
      case 1: launch_skinny_mt<T, 1>(X, ldx, W, M, N, K, splits, part, ep, s, timing); break;
      case 2: launch_skinny_mt<T, 2>(X, ldx, W, M, N, K, splits, part, ep, s, timing); break;
      case 3: launch_skinny_mt<T, 3>(X, ldx, W, M, N, K, splits, part, ep, s, timing); break;
      default: launch_skinny_mt<T, 4>(X, ldx, W, M, N, K, splits, part, ep, s, timing); break;
    }
    return;
  }
  if (K % PF_KQ == 0) {
    if (splits < 1 || part == nullptr) splits = 1;
    const PrefillPlan p = prefill_plan(M, N, K, splits);
    const int kchunk = prefill_kchunk(K, splits);
    const int gx = prefill_grid_columns(N);
    dim3 grid((unsigned)(gx * ((M + p.bm - 1) / p.bm) * p.splits));
    // Wide weights (64 or more column tiles) lay the grid over a multiple of
    // 8 column tiles, so that each column's row tiles share one XCD's L2
    // (7B gate/up, 86 column tiles: 20-25% faster at M = 700..3,500); the
    // padding leaves at most one column per XCD idle.  Narrower weights
    // keep their own count (padding 20 to 24 columns left XCDs 20% uneven).
    // XCD-aware order in groups of 16 row tiles for wide weights: 256-row
    // tiles always take it (measured 5-9% faster for the 28,672 x 4,096
    // gate/up matrix at most M).  128-row tiles take it only when the weight
    // is larger than the 256 MB last-level cache: in the plain order each
    // round of row tiles then re-reads it from HBM (70B gate/up, 57,344 x
    // 8,192: 31-35% slower plain; 13B gate/up, 283 MB: 6-11%), while a
    // weight that fits runs 3-9% faster plain (8B gate/up at M =
    // 1,024..4,223).
    const int xg = prefill_xcd_group(N, K, p.bm);
    if (p.pair)
      launch_k(gemm_prefill_kernel<T, 128, 3, 4>, grid, PF_NT, s, timing, X, ldx, W, M, N, K, kchunk, part, ep, xg, gx);
    else if (p.bm == 256)
      launch_k(gemm_prefill_kernel<T, 256, 4, 2>, grid, PF_NT, s, timing, X, ldx, W, M, N, K, kchunk, part, ep, xg, gx);
    else
      launch_k(gemm_prefill_kernel<T, 128, 4, 2>, grid, PF_NT, s, timing, X, ldx, W, M, N, K, kchunk, part, ep, xg, gx);
    return;
  }
  dim3 grid((N + BG_BN - 1) / BG_BN, (M + BG_BM - 1) / BG_BM);
  launch_k(gemm_big_kernel<T>, grid, 256, s, timing, X, ldx, W, M, N, K, ep);
}

template <>
void launch_gemm<bf16_t>(const bf16_t *X, int64_t ldx, const bf16_t *W, int M, int N, int K, int splits,
                         float *part, const Epi &ep, hipStream_t s, const hipEvent_t *timing) {
  launch_gemm_mfma<bf16_t>(X, ldx, W, M, N, K, splits, part, ep, s, timing);
}
template <>
void launch_gemm<f16_t>(const f16_t *X, int64_t ldx, const f16_t *W, int M, int N, int K, int splits,
                        float *part, const Epi &ep, hipStream_t s, const hipEvent_t *timing) {
  launch_gemm_mfma<f16_t>(X, ldx, W, M, N, K, splits, part, ep, s, timing);
}

template <>
void launch_gemm<float>(const float *X, int64_t ldx, const float *W, int M, int N, int K, int /*splits*/,
                        float * /*part*/, const Epi &ep, hipStream_t s, const hipEvent_t *timing) {
  if (M <= 0 || N <= 0) return;
  dim3 grid((N + F_BN - 1) / F_BN, (M + F_BM - 1) / F_BM);
  launch_k(gemm_f32_kernel, grid, 256, s, timing, X, ldx, W, M, N, K, ep);
}

// ------------------------------------------------------------------ weight packing

// One thread per 16-byte piece of the tiled output: piece p is lane p % 64 of
// tile p / 64.  Pieces past N or K are written as zeros.  K % 8 == 0.
template <typename T>
__global__ void wpack_kernel(const T *__restrict__ src, T *__restrict__ dst, int N, int K, int64_t pieces) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= pieces) return;
  const int64_t ns = wpack_ns(N), t = p >> 6;
  const int l = (int)(p & 63);
  const int64_t n = (t % ns) * WT_ROWS + (l & 15), k = (t / ns) * WT_COLS + (l >> 4) * 8;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (n < N && k < K) v = *(const uint4 *)(src + n * K + k);
  *(uint4 *)(dst + p * 8) = v;
}

template <typename T>
void launch_wpack(const T *src, T *dst, int N, int K, hipStream_t s) {
  const int64_t pieces = wpack_elems(N, K) / 8;
  if (pieces > 0) wpack_kernel<T><<<(unsigned)((pieces + 255) / 256), 256, 0, s>>>(src, dst, N, K, pieces);
}

template void launch_wpack<bf16_t>(const bf16_t *, bf16_t *, int, int, hipStream_t);
template void launch_wpack<f16_t>(const f16_t *, f16_t *, int, int, hipStream_t);

template void launch_gemm_finish<float>(const float *, int, int, int, const Epi &, hipStream_t);
template void launch_gemm_finish<bf16_t>(const float *, int, int, int, const Epi &, hipStream_t);
template void launch_gemm_finish<f16_t>(const float *, int, int, int, const Epi &, hipStream_t);

}  // namespace lp
