// Attention over the paged KV cache.
//
// Decode: each request row attends to its whole cached context.  The context
// is cut into chunks of DEC_CHUNK positions; one workgroup handles one (row,
// kv head, chunk) and all query heads of that kv head's group, four waves each
// taking one 64-position KV block.  The grid holds only live chunks: work
// item i is the i-th (row, chunk) pair in row-major order, found by a prefix
// sum over the rows' chunk counts.  Partial (max, sum, unnormalised output)
// triples are merged by a combine pass (log-sum-exp rescaling).
//
// Prefill: causal attention of packed prompt rows, one workgroup per 64 query
// rows of one (sequence, head), online softmax over 64-key blocks.
#include "device.hpp"

namespace lp {

typedef unsigned int u32x4_tt __attribute__((ext_vector_type(4)));

constexpr int DEC_CHUNK = 256;  // positions per decode workgroup

size_t decode_attention_ws_bytes(int M, int n_heads, int head_dim, int max_ctx) {
  const int splits = (max_ctx + DEC_CHUNK - 1) / DEC_CHUNK;
  return (size_t)M * n_heads * splits * (head_dim + 2) * sizeof(float);
}

int decode_attention_chunks(int ctx) { return (ctx + DEC_CHUNK - 1) / DEC_CHUNK; }

// The fused QKV finish gives each of the 256 threads one q pair of the group
// and requests all its partials at once.
constexpr int DEC_QKV_SPLITS = 6;
bool decode_attention_fuses_qkv(int group, int head_dim, int splits) {
  return group * head_dim / 2 <= 256 && splits >= 1 && splits <= DEC_QKV_SPLITS;
}

// Work item -> (row m, chunk s, slot, context) of a decode workgroup.  Item i
// is the i-th pair in the row-major list of every row's chunks (a row of
// context c has ceil(c / DEC_CHUNK)); contexts are clamped to max_ctx.  Each
// wave computes it on its own: lane l reads row base + l, an inclusive scan
// over the 64 lanes gives the chunks up to that row, and the first lane whose
// running count exceeds the item is the row.  False past the last item.
struct DecodeItem {
  int m, s, slot, ctx, pos;
};
__device__ __forceinline__ bool decode_item(const RowMeta &rows, int M, int max_ctx, int item, DecodeItem &it) {
  const int lane = threadIdx.x & 63;
  int before = 0;
  for (int base = 0; base < M; base += 64) {
    const int r = base + lane;
    const int pos = r < M ? rows.row_pos[r] : 0;
    const int ctx = r < M ? min(pos + 1, max_ctx) : 0;
    const int slot = r < M ? rows.row_slot[r] : 0;
    const int n = ctx > 0 ? (ctx + DEC_CHUNK - 1) / DEC_CHUNK : 0;
    int incl = n;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    const int total = __shfl(incl, 63, 64);
    const int rel = item - before;
    if (rel < total) {
      const int k = __popcll(__ballot(incl <= rel));  // rows wholly before the item
      it.m = base + k;
      it.s = rel - __shfl(incl - n, k, 64);
      it.slot = __shfl(slot, k, 64);
      it.ctx = __shfl(ctx, k, 64);
      it.pos = __shfl(pos, k, 64);
      return true;
    }
    before += total;
  }
  return false;
}

template <typename T>
struct Vec8;  // 8 consecutive activation elements as fp32
template <>
struct Vec8<bf16_t> {
  static __device__ __forceinline__ void load(const bf16_t *p, float *o) {
    const uint4 u = *(const uint4 *)p;
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(w[i] << 16);
      o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
};
template <>
struct Vec8<f16_t> {
  static __device__ __forceinline__ void load(const f16_t *p, float *o) {
    const f16x8_t v = __builtin_bit_cast(f16x8_t, *(const uint4 *)p);
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (float)v[i];
  }
};
template <>
struct Vec8<float> {
  static __device__ __forceinline__ void load(const float *p, float *o) {
    const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
};

template <typename T, int HD, int G>
__global__ __launch_bounds__(256) void decode_attn_kernel(const T *__restrict__ q, RowMeta rows,
                                                          KVCache kv, int layer, int M, int n_heads,
                                                          int max_ctx, int max_splits, float *__restrict__ ws) {
  constexpr int DPL = HD / 64;  // dims per lane in P.V
  __shared__ float qs[G][HD];
  __shared__ float ps[4][G][64];
  __shared__ float wm[4][G], wl[4][G];
  __shared__ float wo[4][G][HD];
  // KV head fastest: consecutive block ids, which the dispatcher deals out
  // round-robin over the XCDs, are the heads of one work item
  const int g = blockIdx.x % kv.n_kv_heads;
  DecodeItem it;
  if (!decode_item(rows, M, max_ctx, blockIdx.x / kv.n_kv_heads, it)) return;
  const int m = it.m, s = it.s, slot = it.slot, ctx = it.ctx;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

  for (int e = threadIdx.x; e < G * HD; e += 256)
    qs[e / HD][e % HD] = Act<T>::ld(q[((int64_t)m * n_heads + g * G) * HD + e]);
  __syncthreads();

  const int blk_pos = s * DEC_CHUNK + wave * 64;  // first position of this wave's block
  const bool active = blk_pos < ctx;
  float mw[G], lw[G], o[G][DPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    mw[h] = -INFINITY;
    lw[h] = 0.f;
#pragma unroll
    for (int t = 0; t < DPL; ++t) o[h][t] = 0.f;
  }
  if (active) {
    const int64_t base = kv_block_base(kv, layer, slot, blk_pos, g);
    const T *kb = (const T *)kv.k + base;
    const T *vb = (const T *)kv.v + base;
    const int p = blk_pos + lane;
    const bool valid = p < ctx;
    float sc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) sc[h] = 0.f;
    if (valid) {
#pragma unroll 4
      for (int d = 0; d < HD; d += 8) {
        float kk[8];
        Vec8<T>::load(kb + (int64_t)lane * HD + d, kk);
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
          for (int t = 0; t < 8; ++t) sc[h] += qs[h][d + t] * kk[t];
      }
    }
    const float scale = rsqrtf((float)HD);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float sv = valid ? sc[h] * scale : -INFINITY;
      mw[h] = wave_max(sv);
      const float pv = valid ? __expf(sv - mw[h]) : 0.f;
      lw[h] = wave_sum(pv);
      ps[wave][h][lane] = pv;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    const int nvalid = min(64, ctx - blk_pos);
#pragma unroll
    for (int t = 0; t < DPL; ++t) {
      const int d = lane * DPL + t;
      const T *vr = vb + (int64_t)d * KV_BLOCK;
      for (int pp = 0; pp < nvalid; pp += 8) {
        float vv[8];
        Vec8<T>::load(vr + pp, vv);
        // cache entries past the context are stale or uninitialised: never read them as numbers
#pragma unroll
        for (int u = 0; u < 8; ++u) vv[u] = (pp + u < nvalid) ? vv[u] : 0.f;
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
          for (int u = 0; u < 8; ++u) o[h][t] += ps[wave][h][pp + u] * vv[u];
      }
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      wm[wave][h] = mw[h];
      wl[wave][h] = lw[h];
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int t = 0; t < DPL; ++t) wo[wave][h][lane * DPL + t] = o[h][t];
  __syncthreads();

  // merge the four waves and write this split's partial
  for (int e = threadIdx.x; e < G * (HD + 2); e += 256) {
    const int h = e / (HD + 2), c = e % (HD + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, wm[w][h]);
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (wm[w][h] == -INFINITY) continue;
      const float f = __expf(wm[w][h] - M);
      acc += f * (c < HD ? wo[w][h][c] : wl[w][h]);
    }
    float *dst = ws + (((int64_t)m * n_heads + g * G + h) * max_splits + s) * (HD + 2);
    dst[c] = (c == HD) ? M : acc;  // [0, HD): output, HD: max, HD + 1: sum
  }
}

// Merges a row's chunk partials for one query head: out = sum_s e^(m_s - M) o_s
// / sum_s e^(m_s - M) l_s with M the largest chunk maximum, taken in one pass
// with a running maximum; each thread owns one output dimension and issues
// the loads of eight chunks before it uses any.
template <typename T, int HD>
__global__ __launch_bounds__(HD) void decode_combine_kernel(RowMeta rows, int n_heads, int max_ctx,
                                                            int max_splits, const float *__restrict__ ws,
                                                            T *__restrict__ out) {
  constexpr int U = 8;
  const int h = blockIdx.x, m = blockIdx.y;
  const int c = threadIdx.x;
  const int ctx = min(rows.row_pos[m] + 1, max_ctx);
  const int ns = ctx > 0 ? (ctx + DEC_CHUNK - 1) / DEC_CHUNK : 0;
  const float *src = ws + ((int64_t)m * n_heads + h) * max_splits * (HD + 2);
  float M = -INFINITY, num = 0.f, den = 0.f;
  for (int s0 = 0; s0 < ns; s0 += U) {
    float mv[U], ov[U], lv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float *p = src + (int64_t)min(s0 + u, ns - 1) * (HD + 2);
      mv[u] = p[HD];
      ov[u] = p[c];
      lv[u] = p[HD + 1];
    }
    float nm = M;
#pragma unroll
    for (int u = 0; u < U; ++u) nm = fmaxf(nm, mv[u]);
    if (nm == -INFINITY) continue;
    const float r = __expf(M - nm);  // 0 while M is still -inf
    num *= r;
    den *= r;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float f = (s0 + u < ns) ? __expf(mv[u] - nm) : 0.f;
      num += f * ov[u];
      den += f * lv[u];
    }
    M = nm;
  }
  out[((int64_t)m * n_heads + h) * HD + c] = Act<T>::st(num / den);
}

// 16-bit decode attention on MFMA.  One wave owns one 64-position KV block:
// S = Q K^T is four 16x16 tiles (query heads of the group padded to 16 rows,
// positions as columns, head_dim as the contraction), the softmax is reduced
// across the 16 lanes that hold a row (DPP lane moves, no LDS), P goes through
// LDS into the A-operand
// layout, and O = P V contracts over positions with V read from its
// transposed [hd][64] block as 16-byte B fragments.  All K fragments of the
// block are requested before any is used, then all V fragments.
//
// FUSED: q is not read; the workgroup finishes the split-K QKV projection of
// its row first (QkvParts): the fp32 partials of its G query heads summed in
// split order and rotated into LDS, and in the workgroup of the row's last
// chunk the new K (rotated) and V entry of head g, written to the cache and
// put into the last block's fragments in place of what the cache held there.
// Its registers are bounded for four waves per SIMD (112 VGPRs, no spills):
// the 8B-shape decode step ran 75 us faster than with the separate finishing
// pass, against 41 us at the compiler's own three.
template <typename T, int HD, int G, bool FUSED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(FUSED ? 4 : 1))) void decode_attn_mfma_kernel(
    const T *__restrict__ q, RowMeta rows, KVCache kv, int layer, int M, int n_heads, int max_ctx, int max_splits,
    float *__restrict__ ws, QkvParts qp) {
  typedef typename Mfma<T>::v8 v8;
  constexpr int KS = HD / 32;  // contraction steps over head_dim
  constexpr int NT = HD / 16;  // 16-wide output tiles over head_dim
  __shared__ T pls[4][16][64 + 8];
  __shared__ float wm[4][16], wl[4][16];
  __shared__ float wo[4][G][HD];
  __shared__ T qls[FUSED ? G : 1][HD];   // FUSED: the group's rotated q
  __shared__ T kvn[FUSED ? 2 : 1][HD];   // FUSED: the row's new K (rotated) and V entry
  // KV head fastest: consecutive block ids, which the dispatcher deals out
  // round-robin over the XCDs, are the heads of one work item
  const int g = blockIdx.x % kv.n_kv_heads;
  DecodeItem it;
  if (!decode_item(rows, M, max_ctx, blockIdx.x / kv.n_kv_heads, it)) return;
  const int m = it.m, s = it.s, slot = it.slot, ctx = it.ctx;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, quad = lane >> 4, kq = quad * 8;
  const int blk_pos = s * DEC_CHUNK + wave * 64;
  const int nvalid = max(0, min(64, ctx - blk_pos));

  const int64_t base = nvalid > 0 ? kv_block_base(kv, layer, slot, blk_pos, g) : 0;
  v8 kf[4][KS];
  v8 qa[KS];
  // the row's new position, when it lies in this wave's block (FUSED)
  const int pnew = (FUSED && it.pos == ctx - 1) ? it.pos - blk_pos : -1;
  if constexpr (FUSED) {
    // Thread t takes q pair t of the group's heads and, in the workgroup of
    // the row's last chunk, pair t of head g's new K (t < HD/2) or V entry.
    // All their loads are issued before the K fragments' (the wait counter
    // is in order), so q is ready when K is.
    static_assert(G * HD / 2 <= 256, "one q pair per thread (decode_attention_fuses_qkv)");
    // Every load below is unconditional, at a clamped (valid) address, so
    // that the compiler issues them back to back and can wait for them
    // without waiting for the K fragments requested after them.
    const bool last = (s + 1) * DEC_CHUNK >= ctx && it.pos == ctx - 1;
    const int pos = it.pos, half = HD / 2, t = threadIdx.x;
    const int qdim = n_heads * HD, kvdim = kv.n_kv_heads * HD;
    const bool has_q = t < G * half, has_kv = last && t < HD, kv_k = t < half;
    const int tq = min(t, G * half - 1), iq = tq % half, hq = tq / half;
    const int nq = (g * G + hq) * HD + 2 * iq;
    const int tk = min(t, HD - 1), ik = tk % half;
    const int nkv = has_kv ? (kv_k ? qdim + g * HD + 2 * tk : qdim + kvdim + g * HD + 2 * (tk - half)) : nq;
    // all partials requested together (decode_attention_fuses_qkv: at most
    // DEC_QKV_SPLITS splits)
    constexpr int U = DEC_QKV_SPLITS;
    const float csq = qp.rope_cos[(int64_t)pos * half + iq], snq = qp.rope_sin[(int64_t)pos * half + iq];
    const float csk = qp.rope_cos[(int64_t)pos * half + ik], snk = qp.rope_sin[(int64_t)pos * half + ik];
    const int64_t kvo = kv_block_base(kv, layer, slot, pos, g);
    float2 pq[U], pk[U];
    float q0 = 0.f, q1 = 0.f, k0 = 0.f, k1 = 0.f;
#define DA_PARTS(s0)                                                                            \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                               \
    const int64_t r = (int64_t)min((s0) + u, qp.splits - 1) * M + m;                            \
    pq[u] = *(const float2 *)(qp.part + r * qp.N + nq);                                         \
    pk[u] = *(const float2 *)(qp.part + r * qp.N + nkv);                                        \
  }
// splits past the count add +0, which leaves every sum as it is (a sum that
// starts at +0 is never -0), and keeps each load's use unconditional
#define DA_SUM(s0)                                                                              \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                               \
    /* the partials are in registers here: no load is deferred into a branch */                 \
    asm volatile("" ::"v"(pq[u].x), "v"(pq[u].y), "v"(pk[u].x), "v"(pk[u].y));                  \
  }                                                                                             \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                               \
    const bool in_ = (s0) + u < qp.splits;                                                      \
    q0 += in_ ? pq[u].x : 0.f;                                                                  \
    q1 += in_ ? pq[u].y : 0.f;                                                                  \
    k0 += in_ ? pk[u].x : 0.f;                                                                  \
    k1 += in_ ? pk[u].y : 0.f;                                                                  \
  }
    DA_PARTS(0)
    {
      // this wave's K fragments, requested right behind the partials and
      // before the wait for them, so that the K round trip runs under the
      // partials' (the wait counter is in order: the partials can be waited
      // for with these still outstanding); unconditional (a wave without a
      // block reads the cache's first block, zeroed below)
      const T *kb = (const T *)kv.k + base;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[nt][ks] = load8<T>(kb + (nt * 16 + r16) * HD + ks * 32 + kq);
    }
    DA_SUM(0)
#undef DA_PARTS
#undef DA_SUM
    if (nvalid <= 0) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[nt][ks] = zero8<T>();
    }
    if (has_q) {
      float r0, r1;
      rope_rotate(q0, q1, csq, snq, r0, r1);
      qls[hq][iq] = Act<T>::st(r0);
      qls[hq][iq + half] = Act<T>::st(r1);
    }
    if (has_kv) {
      T *kc = (T *)kv.k + kvo + (int64_t)(pos % KV_BLOCK) * HD;
      T *vc = (T *)kv.v + kvo + pos % KV_BLOCK;
      if (kv_k) {
        float r0, r1;
        rope_rotate(k0, k1, csk, snk, r0, r1);
        const T t0 = Act<T>::st(r0), t1 = Act<T>::st(r1);
        kvn[0][ik] = t0;
        kvn[0][ik + half] = t1;
        kc[ik] = t0;
        kc[ik + half] = t1;
      } else {
        const int j = 2 * (tk - half);
        const T t0 = Act<T>::st(k0), t1 = Act<T>::st(k1);
        kvn[1][j] = t0;
        kvn[1][j + 1] = t1;
        vc[(int64_t)j * KV_BLOCK] = t0;
        vc[(int64_t)(j + 1) * KV_BLOCK] = t1;
      }
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qa[ks] = (r16 < G) ? load8<T>(&qls[r16][ks * 32 + kq]) : zero8<T>();
    if (pnew >= 0 && pnew < 64) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
        if (nt * 16 + r16 == pnew) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) kf[nt][ks] = load8<T>(&kvn[0][ks * 32 + kq]);
        }
    }
  } else {
    const T *qrow = q + ((int64_t)m * n_heads + g * G + (r16 < G ? r16 : 0)) * HD;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qa[ks] = (r16 < G) ? load8<T>(qrow + ks * 32 + kq) : zero8<T>();
    if (nvalid > 0) {
      const T *kb = (const T *)kv.k + base;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[nt][ks] = load8<T>(kb + (nt * 16 + r16) * HD + ks * 32 + kq);
    } else {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[nt][ks] = zero8<T>();
    }
  }
  floatx4_t sacc[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    sacc[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) sacc[nt] = Mfma<T>::m16(qa[ks], kf[nt][ks], sacc[nt]);
  }
  // V is requested once the K fragments are consumed: the registers K held
  // take V, which keeps the kernel at three workgroups per CU
  v8 vf[NT][2];
  if (nvalid > 0) {
    const T *vb = (const T *)kv.v + base;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) vf[nt][kk] = load8<T>(vb + (nt * 16 + r16) * KV_BLOCK + kk * 32 + kq);
  } else {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) vf[nt][0] = vf[nt][1] = zero8<T>();
  }
  // sacc[nt][i]: row (head) 4*quad + i, position nt*16 + r16
  const float scale = rsqrtf((float)HD);
  float mx[4], sm[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const bool ok = nt * 16 + r16 < nvalid;
      sacc[nt][i] = ok ? sacc[nt][i] * scale : -INFINITY;
      v = fmaxf(v, sacc[nt][i]);
    }
    v = row16_max(v);
    mx[i] = v;
    float t = 0.f;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const float p = (v == -INFINITY) ? 0.f : __expf(sacc[nt][i] - v);
      sacc[nt][i] = p;
      t += p;
    }
    t = row16_sum(t);
    sm[i] = t;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) pls[wave][4 * quad + i][nt * 16 + r16] = Act<T>::st(sacc[nt][i]);
  }
  __syncthreads();
  v8 pa[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) pa[kk] = load8<T>(&pls[wave][r16][kk * 32 + kq]);
  // The V fragments are patched only now, after the softmax: a patch waits
  // for the fragments it edits, and placed right after their loads it held
  // the softmax of the wave (and, at the barrier above, its workgroup)
  // behind the V round trip.
  // Positions past the context hold stale or uninitialised cache entries.
  if (nvalid < 64) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (kk * 32 + kq + e >= nvalid) vf[nt][kk][e] = (typename Mfma<T>::v8){}[0];
  }
  // the row's new V entry (FUSED), in place of what the cache held there
  if (FUSED && pnew >= 0 && pnew < 64) {
    typedef __typeof__((typename Mfma<T>::v8){}[0]) elem_t;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const elem_t vn = __builtin_bit_cast(elem_t, kvn[FUSED ? 1 : 0][nt * 16 + r16]);
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (kk * 32 + kq + e == pnew) vf[nt][kk][e] = vn;
    }
  }
  floatx4_t oacc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    oacc[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) oacc[nt] = Mfma<T>::m16(pa[kk], vf[nt][kk], oacc[nt]);
  }
  if (r16 == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      wm[wave][4 * quad + i] = mx[i];
      wl[wave][4 * quad + i] = sm[i];
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * quad + i;
    if (h < G) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) wo[wave][h][nt * 16 + r16] = oacc[nt][i];
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * (HD + 2); e += 256) {
    const int h = e / (HD + 2), c = e % (HD + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, wm[w][h]);
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (wm[w][h] == -INFINITY) continue;
      const float f = __expf(wm[w][h] - M);
      acc += f * (c < HD ? wo[w][h][c] : wl[w][h]);
    }
    float *dst = ws + (((int64_t)m * n_heads + g * G + h) * max_splits + s) * (HD + 2);
    dst[c] = (c == HD) ? M : acc;  // [0, HD): output, HD: max, HD + 1: sum
  }
}

template <typename T, int HD, int G>
static void launch_decode_group(dim3 grid, const T *q, const RowMeta &rows, const KVCache &kv, int layer, int M,
                                int n_heads, int max_ctx, int splits, float *ws, hipStream_t s, const QkvParts *qkv) {
  if constexpr (sizeof(T) == 2) {
    if constexpr (G * HD / 2 <= 256) {
      if (qkv) {
        decode_attn_mfma_kernel<T, HD, G, true><<<grid, 256, 0, s>>>(q, rows, kv, layer, M, n_heads, max_ctx, splits,
                                                                     ws, *qkv);
        return;
      }
    }
    decode_attn_mfma_kernel<T, HD, G, false><<<grid, 256, 0, s>>>(q, rows, kv, layer, M, n_heads, max_ctx, splits,
                                                                    ws, QkvParts{});
  } else {
    decode_attn_kernel<T, HD, G><<<grid, 256, 0, s>>>(q, rows, kv, layer, M, n_heads, max_ctx, splits, ws);
  }
}

template <typename T, int HD>
static void launch_decode_hd(const T *q, T *out, const RowMeta &rows, const KVCache &kv, int layer,
                             int M, int n_heads, int max_ctx, int items, float *ws, hipStream_t s,
                             const QkvParts *qkv) {
  const int G = n_heads / kv.n_kv_heads;
  if (qkv && !decode_attention_fuses_qkv(G, HD, qkv->splits)) return;
  const int splits = (max_ctx + DEC_CHUNK - 1) / DEC_CHUNK;
  if (items <= 0 || items > M * splits) items = M * splits;
  dim3 grid((unsigned)(items * kv.n_kv_heads));
  switch (G) {
    case 1: launch_decode_group<T, HD, 1>(grid, q, rows, kv, layer, M, n_heads, max_ctx, splits, ws, s, qkv); break;
    case 2: launch_decode_group<T, HD, 2>(grid, q, rows, kv, layer, M, n_heads, max_ctx, splits, ws, s, qkv); break;
    case 4: launch_decode_group<T, HD, 4>(grid, q, rows, kv, layer, M, n_heads, max_ctx, splits, ws, s, qkv); break;
    case 8: launch_decode_group<T, HD, 8>(grid, q, rows, kv, layer, M, n_heads, max_ctx, splits, ws, s, qkv); break;
    default: return;
  }
  decode_combine_kernel<T, HD><<<dim3(n_heads, M), HD, 0, s>>>(rows, n_heads, max_ctx, splits, ws, out);
}

template <typename T>
void launch_decode_attention(const T *q, T *out, const RowMeta &rows, const KVCache &kv, int layer,
                             int M, int n_heads, int max_ctx, int items, float *ws, hipStream_t s,
                             const QkvParts *qkv) {
  if (M <= 0) return;
  if (sizeof(T) != 2) qkv = nullptr;  // the fp32 path has no split QKV projection
  if (kv.head_dim == 128)
    launch_decode_hd<T, 128>(q, out, rows, kv, layer, M, n_heads, max_ctx, items, ws, s, qkv);
  else if (kv.head_dim == 64)
    launch_decode_hd<T, 64>(q, out, rows, kv, layer, M, n_heads, max_ctx, items, ws, s, qkv);
}

// ------------------------------------------------------------------ prefill

template <typename T, int HD>
__global__ __launch_bounds__(256) void prefill_attn_kernel(const T *__restrict__ q, T *__restrict__ out,
                                                           const int32_t *seq_start,
                                                           const int32_t *seq_slot, KVCache kv,
                                                           int layer, int n_heads) {
  constexpr int Q4 = HD / 4;  // dims per thread
  __shared__ T ks[64][HD + 2];
  __shared__ T vs[64][HD + 2];
  const int qt = blockIdx.x, h = blockIdx.y, j = blockIdx.z;
  const int row0 = seq_start[j];
  const int len = seq_start[j + 1] - row0;
  if (qt * 64 >= len) return;
  const int slot = seq_slot[j];
  const int g = h / (n_heads / kv.n_kv_heads);
  const int qi = threadIdx.x >> 2, qq = threadIdx.x & 3;
  const int qpos = qt * 64 + qi;
  const bool qvalid = qpos < len;
  float qv[Q4], o[Q4];
  const T *qr = q + ((int64_t)(row0 + (qvalid ? qpos : 0)) * n_heads + h) * HD + qq * Q4;
#pragma unroll
  for (int t = 0; t < Q4; ++t) {
    qv[t] = Act<T>::ld(qr[t]);
    o[t] = 0.f;
  }
  float mx = -INFINITY, l = 0.f;
  const float scale = rsqrtf((float)HD);
  const int last_key = min(len, qt * 64 + 64);  // keys [0, last_key)
  for (int kb = 0; kb * 64 < last_key; ++kb) {
    __syncthreads();
    const int64_t base = kv_block_base(kv, layer, slot, kb * 64, g);
    const T *kbp = (const T *)kv.k + base;
    const T *vbp = (const T *)kv.v + base;
    for (int e = threadIdx.x; e < 64 * HD; e += 256) {
      const int p = e / HD, d = e % HD;
      ks[p][d] = kbp[e];
      const int d2 = e / 64, p2 = e % 64;
      vs[p2][d2] = vbp[e];
    }
    __syncthreads();
    const int nk = min(64, last_key - kb * 64);
    for (int p = 0; p < nk; ++p) {
      float sc = 0.f;
#pragma unroll
      for (int t = 0; t < Q4; ++t) sc += qv[t] * Act<T>::ld(ks[p][qq * Q4 + t]);
      sc += __shfl_xor(sc, 1, 64);
      sc += __shfl_xor(sc, 2, 64);
      const int kpos = kb * 64 + p;
      if (kpos > qpos) continue;  // causal (uniform across the 4 threads of a row)
      sc *= scale;
      const float mn = fmaxf(mx, sc);
      const float corr = __expf(mx - mn);
      const float pe = __expf(sc - mn);
      l = l * corr + pe;
#pragma unroll
      for (int t = 0; t < Q4; ++t) o[t] = o[t] * corr + pe * Act<T>::ld(vs[p][qq * Q4 + t]);
      mx = mn;
    }
  }
  if (qvalid) {
    T *orow = out + ((int64_t)(row0 + qpos) * n_heads + h) * HD + qq * Q4;
    const float inv = 1.0f / l;
#pragma unroll
    for (int t = 0; t < Q4; ++t) orow[t] = Act<T>::st(o[t] * inv);
  }
}

// 16-bit causal prefill attention on MFMA (flash-attention style).  A
// workgroup owns 64 query rows of one (sequence, head); each wave owns 16 of
// them.  Key blocks of 64 positions are staged in LDS (K as [key][dim], V
// transposed as [dim][key], rows padded so the 16-byte fragment reads of a
// wave fall in distinct banks) with the next block prefetched into registers
// while the current one is used.  S = Q K^T and O += P V are 16x16x32 MFMAs,
// the softmax is online (running max and sum per row, reduced across the 16
// lanes of a row by DPP lane moves), and only the diagonal block needs the
// causal mask.  The launch bound (at least two workgroups' worth of waves
// per SIMD) makes the compiler keep the 128-dim kernel at 148 VGPRs, so three
// waves share each SIMD and one wave's softmax runs under another's MFMAs.
// Grid: (query tile, head, sequence), or with longest_first (head, sequence,
// query tile) with the tiles walked from the last, so that the tiles with the
// most key blocks are dispatched first and the short ones fill in behind them.
template <typename T, int HD>
__global__ __launch_bounds__(256, 2) void prefill_attn_mfma_kernel(const T *__restrict__ q, T *__restrict__ out,
                                                                const int32_t *seq_start, const int32_t *seq_slot,
                                                                KVCache kv, int layer, int n_heads,
                                                                int longest_first) {
  typedef typename Mfma<T>::v8 v8;
  constexpr int KS = HD / 32;                 // contraction steps over head_dim
  constexpr int NT = HD / 16;                 // output tiles over head_dim
  constexpr int KPAD = HD + 8;                // K row stride (elements)
  constexpr int VPAD = 64 + 8;                // Vt row stride
  constexpr int CH = 64 * HD * 2 / 16 / 256;  // 16-byte chunks per thread per block (K and V)
  __shared__ T ks[64][KPAD];
  __shared__ T vs[HD][VPAD];
  __shared__ T pls[4][16][64 + 8];
  const int qt = longest_first ? (int)gridDim.z - 1 - (int)blockIdx.z : (int)blockIdx.x;
  const int h = longest_first ? (int)blockIdx.x : (int)blockIdx.y;
  const int j = longest_first ? (int)blockIdx.y : (int)blockIdx.z;
  const int row0 = seq_start[j];
  const int len = seq_start[j + 1] - row0;
  if (qt * 64 >= len) return;
  const int slot = seq_slot[j];
  const int g = h / (n_heads / kv.n_kv_heads);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, quad = lane >> 4, kq = quad * 8;
  const int q0 = qt * 64 + wave * 16;  // first query position of this wave

  v8 qa[KS];
  {
    const int qp = min(q0 + r16, len - 1);
    const T *qr = q + ((int64_t)(row0 + qp) * n_heads + h) * HD;
#pragma unroll
    for (int k = 0; k < KS; ++k) qa[k] = load8<T>(qr + k * 32 + kq);
  }
  floatx4_t oacc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) oacc[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    mrow[i] = -INFINITY;
    lrow[i] = 0.f;
  }
  // scores in base-2 units: e^x = 2^(x log2 e), with the factor folded into
  // the scale, so each exponential is one v_exp_f32
  const float scale = rsqrtf((float)HD) * 1.44269504088896341f;
  const int nblk = min(qt + 1, (len + 63) / 64);  // causal: key blocks up to the diagonal

  // staging: chunk c of a block -> K: key c / (HD/8), dims (c % (HD/8)) * 8;
  //                               Vt: dim c / 8, keys (c % 8) * 8
  u32x4_tt kr[CH], vr[CH];
  auto fetch = [&](int kb) __attribute__((always_inline)) {
    const int64_t base = kv_block_base(kv, layer, slot, kb * 64, g);
    const u32x4_tt *kp = (const u32x4_tt *)((const T *)kv.k + base);
    const u32x4_tt *vp = (const u32x4_tt *)((const T *)kv.v + base);
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      kr[c] = kp[tid + c * 256];
      vr[c] = vp[tid + c * 256];
    }
  };
  fetch(0);
  for (int kb = 0; kb < nblk; ++kb) {
    __syncthreads();  // previous block fully consumed
    const int kvalid = len - kb * 64;  // keys of this block inside the sequence
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int e = tid + c * 256;
      *(u32x4_tt *)&ks[e / (HD / 8)][(e % (HD / 8)) * 8] = kr[c];
      // cache entries past the sequence end are stale or uninitialised; their
      // softmax weight is 0 but 0 * NaN is not, so they become zeros here
      u32x4_tt v = vr[c];
      const int key0 = (e % 8) * 8;
      if (key0 + 8 > kvalid) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t lo = key0 + 2 * w < kvalid ? 0xFFFFu : 0u;
          const uint32_t hi = key0 + 2 * w + 1 < kvalid ? 0xFFFF0000u : 0u;
          v[w] &= (lo | hi);
        }
      }
      *(u32x4_tt *)&vs[e / 8][key0] = v;
    }
    __syncthreads();
    if (kb + 1 < nblk) fetch(kb + 1);
    // S = Q K^T over the 64 keys of this block
    floatx4_t sacc[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      sacc[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < KS; ++k) sacc[nt] = Mfma<T>::m16(qa[k], load8<T>(&ks[nt * 16 + r16][k * 32 + kq]), sacc[nt]);
    }
    // online softmax: row 4*quad + i of this wave, keys nt*16 + r16
    const bool diag = kb == nblk - 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qpos = q0 + 4 * quad + i;
      float mx = mrow[i];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int kpos = kb * 64 + nt * 16 + r16;
        const bool ok = !diag || (kpos <= qpos && kpos < len);
        sacc[nt][i] = ok ? sacc[nt][i] * scale : -INFINITY;
        mx = fmaxf(mx, sacc[nt][i]);
      }
      mx = row16_max(mx);
      // rows past the sequence end see no valid key: keep them finite
      const float mref = (mx == -INFINITY) ? 0.f : mx;
      const float corr = __builtin_amdgcn_exp2f(mrow[i] - mref);
      float t = 0.f;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const float p = __builtin_amdgcn_exp2f(sacc[nt][i] - mref);
        sacc[nt][i] = p;
        t += p;
      }
      t = row16_sum(t);
      lrow[i] = lrow[i] * corr + t;
      mrow[i] = mx;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) oacc[nt][i] *= corr;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) pls[wave][4 * quad + i][nt * 16 + r16] = Act<T>::st(sacc[nt][i]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    v8 pa[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) pa[kk] = load8<T>(&pls[wave][r16][kk * 32 + kq]);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        oacc[nt] = Mfma<T>::m16(pa[kk], load8<T>(&vs[nt * 16 + r16][kk * 32 + kq]), oacc[nt]);
  }
  // rows 4*quad + i, dims nt*16 + r16
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int qpos = q0 + 4 * quad + i;
    if (qpos < len) {
      const float inv = 1.0f / lrow[i];
      T *orow = out + ((int64_t)(row0 + qpos) * n_heads + h) * HD;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) orow[nt * 16 + r16] = Act<T>::st(oacc[nt][i] * inv);
    }
  }
}

// Steps of at most this many prompts dispatch the longest query tiles first:
// with few prompts the tiles of the most key blocks bound the launch (1.1-1.7x
// faster for one to three prompts of 547-4,000 tokens).  With many, walking
// each (prompt, head)'s tiles together keeps its keys and values in the L2
// (64 prompts of 43k tokens: 0.70 against 0.81 ms the other way).
constexpr int PF_ATTN_LONGEST_FIRST_MAX_SEQ = 4;

template <typename T, int HD>
static void launch_prefill_hd(dim3 grid, const T *q, T *out, const int32_t *seq_start, const int32_t *seq_slot,
                              const KVCache &kv, int layer, int n_heads, hipStream_t s) {
  if constexpr (sizeof(T) == 2) {
    if ((int)grid.z <= PF_ATTN_LONGEST_FIRST_MAX_SEQ)
      prefill_attn_mfma_kernel<T, HD><<<dim3(grid.y, grid.z, grid.x), 256, 0, s>>>(q, out, seq_start, seq_slot, kv,
                                                                                   layer, n_heads, 1);
    else
      prefill_attn_mfma_kernel<T, HD><<<grid, 256, 0, s>>>(q, out, seq_start, seq_slot, kv, layer, n_heads, 0);
  } else {
    prefill_attn_kernel<T, HD><<<grid, 256, 0, s>>>(q, out, seq_start, seq_slot, kv, layer, n_heads);
  }
}

template <typename T>
void launch_prefill_attention(const T *q, T *out, const int32_t *seq_start, const int32_t *seq_slot,
                              int n_seq, int max_len, const KVCache &kv, int layer, int n_heads,
                              hipStream_t s) {
  if (n_seq <= 0) return;
  dim3 grid((max_len + 63) / 64, n_heads, n_seq);
  if (kv.head_dim == 128)
    launch_prefill_hd<T, 128>(grid, q, out, seq_start, seq_slot, kv, layer, n_heads, s);
  else if (kv.head_dim == 64)
    launch_prefill_hd<T, 64>(grid, q, out, seq_start, seq_slot, kv, layer, n_heads, s);
}

#define INST(T)                                                                                     \
  template void launch_decode_attention<T>(const T *, T *, const RowMeta &, const KVCache &, int,   \
                                           int, int, int, int, float *, hipStream_t,                \
                                           const QkvParts *);                                       \
  template void launch_prefill_attention<T>(const T *, T *, const int32_t *, const int32_t *, int, \
                                            int, const KVCache &, int, int, hipStream_t);
INST(float)
INST(bf16_t)
INST(f16_t)
#undef INST

}  // namespace lp
