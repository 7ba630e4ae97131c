// Embedding gather, RMSNorm (with split-K residual folding), greedy argmax and
// the device-side weight generator.
#include "device.hpp"

namespace lp {

// ------------------------------------------------------------------ embedding

// One workgroup per row.  The row is read in 16-byte pieces, four per thread
// requested before any is stored, so a row of up to 4,096 16-bit (2,048
// fp32) values costs one memory round trip; rows whose length is not a
// multiple of the piece take the element loop.
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const T *__restrict__ E, const int32_t *pool,
                                                    const int32_t *tok_idx, const int32_t *row_slot,
                                                    const int32_t *slot_tok, float *__restrict__ x,
                                                    int d) {
  const int m = blockIdx.x;
  const int ti = tok_idx[m];
  const int tok = ti >= 0 ? pool[ti] : slot_tok[row_slot[m]];
  const T *src = E + (int64_t)tok * d;
  float *dst = x + (int64_t)m * d;
  constexpr int EV = 16 / sizeof(T);  // elements per 16-byte piece
  constexpr int U = 4;
  if (d % EV == 0) {
    const int nv = d / EV;
    for (int c0 = threadIdx.x; c0 < nv; c0 += 256 * U) {
      uint4 r[U];
#pragma unroll
      for (int u = 0; u < U; ++u) r[u] = ((const uint4 *)src)[min(c0 + u * 256, nv - 1)];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * 256;
        if (c < nv) {
          const T *e = (const T *)&r[u];
#pragma unroll
          for (int k = 0; k < EV; k += 4)
            *(float4 *)(dst + (int64_t)c * EV + k) =
                make_float4(Act<T>::ld(e[k]), Act<T>::ld(e[k + 1]), Act<T>::ld(e[k + 2]), Act<T>::ld(e[k + 3]));
        }
      }
    }
  } else {
    for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = Act<T>::ld(src[c]);
  }
}

template <typename T>
void launch_embed(const T *E, const int32_t *pool, const int32_t *tok_idx, const int32_t *row_slot,
                  const int32_t *slot_tok, float *x, int M, int d, hipStream_t s) {
  if (M <= 0) return;
  embed_kernel<T><<<M, 256, 0, s>>>(E, pool, tok_idx, row_slot, slot_tok, x, d);
}

// ------------------------------------------------------------------ RMSNorm

// One workgroup per row.  The residual row, every split-K partial of it and
// the gains are requested before any is used (NP is the partial count), so a
// row costs one memory latency rather than one per partial.  V4 float4 per
// thread: one for rows of up to 4,096, two up to 8,192, with d / (4 V4)
// threads (rounded to waves).  A 64 x 4,096 fold of eight partials took
// 4.2 us on 1,024 threads against 10.9 us on 256 with four float4 each
// (harness, partials cold): more waves keep more of the row in flight.
template <typename T, int NP, int V4>
__global__ __launch_bounds__(1024) void rmsnorm_kernel(float *x, const float *part, int64_t part_stride,
                                                       const int32_t *rows, const float *__restrict__ g,
                                                       T *__restrict__ y, int d, float eps) {
  __shared__ float red[16];
  const int j = blockIdx.x;
  const int src = rows ? rows[j] : j;
  const int d4 = d >> 2;
  const int nt = blockDim.x;
  float4 *xr = (float4 *)(x + (int64_t)src * d);
  const float4 *g4 = (const float4 *)g;
  float4 v[V4], gv[V4];
  float4 p[NP > 0 ? NP : 1][V4];
#pragma unroll
  for (int e = 0; e < V4; ++e) {
    const int c = threadIdx.x + e * nt;
    if (c < d4) {
      v[e] = xr[c];
      gv[e] = g4[c];
#pragma unroll
      for (int s = 0; s < NP; ++s) p[s][e] = ((const float4 *)(part + s * part_stride + (int64_t)src * d))[c];
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < V4; ++e) {
    const int c = threadIdx.x + e * nt;
    if (c < d4) {
#pragma unroll
      for (int s = 0; s < NP; ++s) {
        v[e].x += p[s][e].x;
        v[e].y += p[s][e].y;
        v[e].z += p[s][e].z;
        v[e].w += p[s][e].w;
      }
      if (NP) xr[c] = v[e];
      ss += v[e].x * v[e].x + v[e].y * v[e].y + v[e].z * v[e].z + v[e].w * v[e].w;
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < (nt >> 6); ++w) tot += red[w];
  const float r = rsqrtf(tot / (float)d + eps);
  T *yr = y + (int64_t)j * d;
#pragma unroll
  for (int e = 0; e < V4; ++e) {
    const int c = threadIdx.x + e * nt;
    if (c < d4) {
      const float4 gg = gv[e];
      yr[4 * c + 0] = Act<T>::st(v[e].x * r * gg.x);
      yr[4 * c + 1] = Act<T>::st(v[e].y * r * gg.y);
      yr[4 * c + 2] = Act<T>::st(v[e].z * r * gg.z);
      yr[4 * c + 3] = Act<T>::st(v[e].w * r * gg.w);
    }
  }
}

template <typename T>
void launch_rmsnorm(float *x, const float *part, int n_part, int64_t part_stride, const int32_t *rows,
                    const float *g, T *y, int M, int d, float eps, hipStream_t s) {
  if (M <= 0) return;
  // whole waves, V4 float4 per thread (d <= 8192)
  const int v4 = d / 4 <= 1024 ? 1 : 2;
  const int threads = std::min(1024, std::max(64, ((d / (4 * v4)) + 63) / 64 * 64));
#define NORM_CASE(NPV)                                                                                  \
  case NPV:                                                                                             \
    if (v4 == 1)                                                                                        \
      rmsnorm_kernel<T, NPV, 1><<<M, threads, 0, s>>>(x, part, part_stride, rows, g, y, d, eps);        \
    else                                                                                                \
      rmsnorm_kernel<T, NPV, 2><<<M, threads, 0, s>>>(x, part, part_stride, rows, g, y, d, eps);        \
    break;
  switch (n_part) {
    NORM_CASE(0) NORM_CASE(1) NORM_CASE(2) NORM_CASE(3) NORM_CASE(4) NORM_CASE(5) NORM_CASE(6)
    NORM_CASE(7) NORM_CASE(8) NORM_CASE(9) NORM_CASE(10) NORM_CASE(11) NORM_CASE(12)
    NORM_CASE(13) NORM_CASE(14) NORM_CASE(15) NORM_CASE(16)
    default: break;  // callers never pass more than 16 partials
  }
#undef NORM_CASE
}

// ------------------------------------------------------------------ argmax

// One workgroup of 1024 threads per row, 16-byte loads, eight of them
// requested before any is used (a row then costs four memory round trips, not
// thirty-two).  Merges prefer the larger value, then the lower index: a total
// order, so the result does not depend on the order of the merges.
__device__ __forceinline__ void argmax_merge(float &bv, int &bi, float ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

__global__ __launch_bounds__(1024) void argmax_kernel(const float *__restrict__ logits, int64_t ld, int V,
                                                      const int32_t *out_slot, int32_t *slot_tok, int32_t *tok_log) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const int m = blockIdx.x;
  const float *row = logits + (int64_t)m * ld;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  const int v4 = ((ld & 3) == 0) ? V >> 2 : 0;
  constexpr int U = 8;
  for (int c0 = threadIdx.x; c0 < v4; c0 += 1024 * U) {
    float4 q[U];
#pragma unroll
    for (int u = 0; u < U; ++u) q[u] = ((const float4 *)row)[min(c0 + u * 1024, v4 - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 1024;
      if (c < v4) {
        argmax_merge(best, bi, q[u].x, 4 * c);
        argmax_merge(best, bi, q[u].y, 4 * c + 1);
        argmax_merge(best, bi, q[u].z, 4 * c + 2);
        argmax_merge(best, bi, q[u].w, 4 * c + 3);
      }
    }
  }
  for (int c = 4 * v4 + threadIdx.x; c < V; c += 1024) argmax_merge(best, bi, row[c], c);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    argmax_merge(best, bi, ov, oi);
  }
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = best;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 16; ++w) argmax_merge(best, bi, sv[w], si[w]);
    if (out_slot) slot_tok[out_slot[m]] = bi;
    tok_log[m] = bi;
  }
}

void launch_argmax(const float *logits, int64_t ld, int M, int V, const int32_t *out_slot, int32_t *slot_tok,
                   int32_t *tok_log, hipStream_t s) {
  if (M <= 0) return;
  argmax_kernel<<<M, 1024, 0, s>>>(logits, ld, V, out_slot, slot_tok, tok_log);
}

// ------------------------------------------------------------------ weight generator

// Philox4x32 with ten rounds (Salmon et al., SC'11).
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c[0], hi0 = __umulhi(0xD2511F53u, c[0]);
    const uint32_t lo1 = 0xCD9E8D57u * c[2], hi1 = __umulhi(0xCD9E8D57u, c[2]);
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

// ------------------------------------------------------------------ sampling

// Non-greedy next-token choice per row (the sampling parameters carried by
// requests, Sec. III-A).  Every decision after the per-token weights is exact
// integer arithmetic, so the result does not depend on reduction order:
//  * temperature <= 0 or top_p <= 0: greedy (lowest index among maxima);
//  * candidates: all tokens, or with 0 < top_k < V those whose logit is at
//    least the top_k-th largest logit (ties at it kept), found by a radix
//    select over order-preserving integer keys of the logits;
//  * weight of a candidate: q = floor(exp((logit - max) / T) * 2^40);
//  * top_p < 1: with Z the candidates' total weight and
//    need = ceil(Z * floor(top_p * 2^24) / 2^24), keep the candidates whose q
//    is at least t, the largest value whose heavier-or-equal candidates sum to
//    at least need (a radix descent over q with 64-bit mass histograms);
//  * draw: u24 = the first Philox4x32-10 output word (key, counter as given)
//    shifted right by 8; r = floor(Z_kept * u24 / 2^24); the token is the kept
//    candidate, in vocabulary order, whose cumulative weight interval holds r.
// One workgroup per row.  The row is read in full at most five times: the
// maximum (with the first top-k level), the top-k bin's elements, the weight
// total (with the first top-p level), the top-p bin's elements, and the draw.
// The remaining radix levels run over those elements held in LDS (a full-row
// pass per level only when a bin holds more than SP_CAP elements).  When top-k
// leaves at most SP_DRAW candidates, their weights and the draw stay in LDS.

__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint64_t q_weight(float l, float mx, float inv_t) {
  const float w = __expf((l - mx) * inv_t);
  return (uint64_t)(w * 1099511627776.0f);  // 2^40; w <= 1
}

// (a * b) >> 24 for a < 2^58, b < 2^25, rounded up when `up`
__device__ __forceinline__ uint64_t mul_shift24(uint64_t a, uint64_t b, bool up) {
  const uint64_t lo = a * b, hi = __umul64hi(a, b);
  uint64_t r = (hi << 40) | (lo >> 24);
  if (up && (lo & 0xFFFFFFull)) ++r;
  return r;
}

constexpr int SP_T = 1024;     // threads per row
constexpr int SP_NB = 2048;    // bins of a radix level (11 bits)
constexpr int SP_CAP = 8192;   // values held in LDS after a compaction
constexpr int SP_DRAW = 1024;  // kept candidates drawn in LDS (one per thread)
// the full-row draw keeps a mass per 256 elements in the SP_CAP list
static_assert((int64_t)SP_CAP * 256 >= SAMPLE_MAX_V, "sampling rows longer than the draw's piece list");

struct SampleLds {
  uint64_t hist[SP_NB];
  uint64_t lv[SP_CAP];     // order key or weight of a listed element
  int32_t li[SP_CAP];      // its vocabulary index
  uint64_t cq[SP_DRAW];    // candidates of an LDS draw: weight
  int32_t ci[SP_DRAW];     // ... and index
  uint64_t red[16];
  uint64_t sel[4];
  float fmax[16];
  int imax[16];
  int n_list, n_cand, found, pick;
};

__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// inclusive scan of v over the block's threads (thread order), and the total
__device__ uint64_t sp_scan(uint64_t v, uint64_t *red, uint64_t &total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint64_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t t = __shfl_up(x, o, 64);
    if (lane >= o) x += t;
  }
  __syncthreads();
  if (lane == 63) red[w] = x;
  __syncthreads();
  uint64_t base = 0;
  total = 0;
  for (int i = 0; i < 16; ++i) {
    const uint64_t r = red[i];
    if (i < w) base += r;
    total += r;
  }
  return base + x;
}

// Radix level selection over hist[0..nb): the largest bin b >= 1 whose mass
// from the top (plus `above`) reaches need, else 0 -- the bin where a walk
// down from the highest bin first reaches need.  Writes sel[0] = mass above
// b (plus above), sel[1] = b, sel[2] = sel[0] + hist[b].  Thread t owns bins
// nb-1-2t and nb-2-2t.
__device__ void sp_select(SampleLds &S, int nb, uint64_t need, uint64_t above) {
  const int t = threadIdx.x;
  const int hi = nb - 1 - 2 * t, lo = hi - 1;
  const uint64_t hh = (t < nb / 2) ? S.hist[hi] : 0, hl = (t < nb / 2) ? S.hist[lo] : 0;
  uint64_t total;
  const uint64_t incl = sp_scan(hh + hl, S.red, total);
  const uint64_t excl = incl - hh - hl;
  if (t == 0) S.pick = 0;
  __syncthreads();
  if (t < nb / 2) {
    int b = -1;
    if (above + excl + hh >= need && hi >= 1) b = hi;
    else if (above + incl >= need && lo >= 1) b = lo;
    if (b >= 0) atomicMax(&S.pick, b);
  }
  __syncthreads();
  const int b = S.pick;
  if (t < nb / 2 && (b == hi || b == lo)) {
    const uint64_t a = above + excl + (b == lo ? hh : 0);
    S.sel[0] = a;
    S.sel[1] = (uint64_t)b;
    S.sel[2] = a + (b == lo ? hl : hh);
  }
  __syncthreads();
}

// First top-p level: a monotone, log-scale bin of a weight.  q < 64 has a
// bin of its own; larger q falls in bin 32 + 32 (e - 5) + m, e its highest
// set bit and m the 5 bits below, a bin of width 2^(e - 5).
__device__ __forceinline__ int sp_qbin(uint64_t q) {
  if (q < 64) return (int)q;
  const int e = 63 - __clzll((long long)q);
  return 32 + 32 * (e - 5) + (int)((q >> (e - 5)) & 31);
}
// lowest weight of bin b and the number of its free low bits
__device__ __forceinline__ void sp_qbin_range(int b, uint64_t &lo, int &bits) {
  if (b < 64) {
    lo = (uint64_t)b;
    bits = 0;
  } else {
    const int e = 5 + (b - 32) / 32, m = (b - 32) % 32;
    bits = e - 5;
    lo = (uint64_t)(32 + m) << bits;
  }
}

// hist[0] = total - hist[1..nb) (bin 0 was not accumulated)
__device__ void sp_fill_bin0(SampleLds &S, int nb, uint64_t total) {
  uint64_t v = 0;
  for (int b = 1 + (int)threadIdx.x; b < nb; b += SP_T) v += S.hist[b];
  uint64_t sum;
  sp_scan(v, S.red, sum);
  if (threadIdx.x == 0) S.hist[0] = total - sum;
  __syncthreads();
}

__device__ __forceinline__ void sp_clear(SampleLds &S, int nb) {
  for (int b = threadIdx.x; b < nb; b += SP_T) S.hist[b] = 0;
}

// wave-aggregated append: the slot of this lane's element when pred holds
__device__ __forceinline__ int sp_append(bool pred, int *counter) {
  const uint64_t mask = __ballot(pred);
  if (!mask) return -1;
  const int lane = threadIdx.x & 63, leader = __ffsll((unsigned long long)mask) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(counter, __popcll(mask));
  base = __shfl(base, leader, 64);
  return pred ? base + __popcll(mask & ((1ull << lane) - 1ull)) : -1;
}

// Calls f(index, logit, valid) for every element of the row, four per thread
// and step, all lanes active in every step (valid false past V).  Eight steps'
// loads are issued before any element is used.
__device__ __forceinline__ float4 sp_load4(const float *row, int c, int V, bool vec) {
  float4 v;
  if (vec && c + 3 < V) {
    v = *(const float4 *)(row + c);
  } else {
    v.x = c < V ? row[c] : 0.f;
    v.y = c + 1 < V ? row[c + 1] : 0.f;
    v.z = c + 2 < V ? row[c + 2] : 0.f;
    v.w = c + 3 < V ? row[c + 3] : 0.f;
  }
  return v;
}

template <typename F>
__device__ __forceinline__ void sp_row(const float *row, int V, bool vec, F f) {
  constexpr int U = 8;
  const int steps = (V + 4 * SP_T - 1) / (4 * SP_T);
  for (int s0 = 0; s0 < steps; s0 += U) {
    float4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = sp_load4(row, ((s0 + u) * SP_T + threadIdx.x) * 4, V, vec);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = ((s0 + u) * SP_T + threadIdx.x) * 4;
      f(c, v[u].x, c < V);
      f(c + 1, v[u].y, c + 1 < V);
      f(c + 2, v[u].z, c + 2 < V);
      f(c + 3, v[u].w, c + 3 < V);
    }
  }
}

__global__ __launch_bounds__(SP_T) void sample_kernel(const float *__restrict__ logits, int64_t ld, int V,
                                                       const SampleParams *__restrict__ prm, const int32_t *out_slot,
                                                       int32_t *slot_tok, int32_t *tok_out) {
  __shared__ SampleLds S;
  const int m = blockIdx.x, tid = threadIdx.x;
  const float *row = logits + (int64_t)m * ld;
  const bool vec = (ld % 4 == 0) && (((uintptr_t)logits & 15) == 0);
  const SampleParams P = prm[m];
  const bool sampled = P.temperature > 0.f && P.top_p > 0.f && V > 1;
  const bool topk = sampled && P.top_k > 0 && P.top_k < V;
  // 1. maximum (and the greedy answer), with the top-k first-level counts
  if (topk) sp_clear(S, SP_NB);
  __syncthreads();
  float best = -INFINITY;
  int bi = 0x7fffffff;
  sp_row(row, V, vec, [&](int c, float l, bool ok) {
    if (ok) {
      argmax_merge(best, bi, l, c);
      if (topk) atomicAdd((unsigned long long *)&S.hist[order_key(l) >> 21], 1ull);
    }
  });
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) argmax_merge(best, bi, __shfl_xor(best, o, 64), __shfl_xor(bi, o, 64));
  if ((tid & 63) == 0) {
    S.fmax[tid >> 6] = best;
    S.imax[tid >> 6] = bi;
  }
  __syncthreads();
  for (int w = 0; w < 16; ++w) argmax_merge(best, bi, S.fmax[w], S.imax[w]);
  int token = bi;
  if (sampled) {
    const float mx = best, inv_t = 1.f / P.temperature;
    uint32_t kmin = 0;
    bool in_lds = false;  // candidates (key >= kmin) listed in cq / ci
    if (topk) {
      // 2. top-k threshold: the top_k-th largest order key, in 11 + 11 + 10 bits
      sp_select(S, SP_NB, (uint64_t)P.top_k, 0);
      const uint32_t b0 = (uint32_t)S.sel[1];
      uint64_t above = S.sel[0];
      const uint64_t n_hi = S.sel[2];  // elements in bins >= b0
      __syncthreads();
      if (tid == 0) S.n_list = 0;
      __syncthreads();
      const bool listed = n_hi <= SP_CAP;
      if (listed) {
        sp_row(row, V, vec, [&](int c, float l, bool ok) {
          const uint32_t k = order_key(l);
          const int slot = sp_append(ok && (k >> 21) >= b0, &S.n_list);
          if (slot >= 0 && slot < SP_CAP) {
            S.lv[slot] = k;
            S.li[slot] = c;
          }
        });
        __syncthreads();
      }
      const int n = S.n_list;
      uint32_t prefix = b0 << 21;
      for (int level = 1; level < 3; ++level) {
        const int sh = level == 1 ? 10 : 0, nb = level == 1 ? SP_NB : 1024;
        const uint32_t pmask = level == 1 ? 0xFFE00000u : 0xFFFFFC00u;
        sp_clear(S, nb);
        __syncthreads();
        if (listed) {
          for (int j = tid; j < n; j += SP_T) {
            const uint32_t k = (uint32_t)S.lv[j];
            if ((k & pmask) == prefix) atomicAdd((unsigned long long *)&S.hist[(k >> sh) & (nb - 1)], 1ull);
          }
        } else {
          sp_row(row, V, vec, [&](int, float l, bool ok) {
            const uint32_t k = order_key(l);
            if (ok && (k & pmask) == prefix) atomicAdd((unsigned long long *)&S.hist[(k >> sh) & (nb - 1)], 1ull);
          });
        }
        __syncthreads();
        sp_select(S, nb, (uint64_t)P.top_k, above);
        above = S.sel[0];
        prefix |= (uint32_t)S.sel[1] << sh;
        __syncthreads();
      }
      kmin = prefix;
      // the candidates, when few, into the draw list
      if (listed) {
        if (tid == 0) S.n_cand = 0;
        __syncthreads();
        for (int j0 = 0; j0 < n; j0 += SP_T) {
          const int j = j0 + tid;
          const bool cand = j < n && (uint32_t)S.lv[j] >= kmin;
          const int slot = sp_append(cand, &S.n_cand);
          if (slot >= 0 && slot < SP_DRAW) {
            S.cq[slot] = q_weight(key_float((uint32_t)S.lv[j]), mx, inv_t);
            S.ci[slot] = S.li[j];
          }
        }
        __syncthreads();
        in_lds = S.n_cand <= SP_DRAW;
      }
    }
    // 3. candidate weights: their total and the top-p first-level masses
    const uint32_t pfix = P.top_p >= 1.f ? (1u << 24) : max(1u, (uint32_t)(P.top_p * 16777216.0f));
    const bool topp = pfix < (1u << 24);
    const int nc = in_lds ? S.n_cand : 0;
    uint64_t z = 0;
    if (topp) sp_clear(S, SP_NB);
    __syncthreads();
    // bin 0 (the many light weights) is left out and later set to the
    // total minus the other bins
    if (in_lds) {
      if (tid < nc) {
        const uint64_t q = S.cq[tid];
        z = q;
        if (topp && q) atomicAdd((unsigned long long *)&S.hist[sp_qbin(q)], (unsigned long long)q);
      }
    } else {
      sp_row(row, V, vec, [&](int, float l, bool ok) {
        if (ok && order_key(l) >= kmin) {
          const uint64_t q = q_weight(l, mx, inv_t);
          z += q;
          if (topp && q) atomicAdd((unsigned long long *)&S.hist[sp_qbin(q)], (unsigned long long)q);
        }
      });
    }
    uint64_t ztot;
    sp_scan(z, S.red, ztot);
    z = ztot;
    if (topp) sp_fill_bin0(S, SP_NB, z);
    // 4. top-p threshold on weights: a log-scale first level, then the free
    // low bits of the chosen bin, ten at a time
    uint64_t tmin = 0, zk = z;
    if (topp) {
      const uint64_t need = mul_shift24(z, pfix, true);
      sp_select(S, SP_NB, need, 0);
      const int b0 = (int)S.sel[1];
      uint64_t above = S.sel[0];
      zk = S.sel[2];
      __syncthreads();
      uint64_t prefix;
      int rem;
      sp_qbin_range(b0, prefix, rem);
      bool listed = in_lds;
      int n = nc;
      if (!in_lds && rem > 0) {
        // the weights of bin b0, which the remaining levels refine, when few,
        // into the list
        if (tid == 0) S.n_list = 0;
        __syncthreads();
        sp_row(row, V, vec, [&](int c, float l, bool ok) {
          bool keep = ok && order_key(l) >= kmin;
          uint64_t q = 0;
          if (keep) {
            q = q_weight(l, mx, inv_t);
            keep = q && sp_qbin(q) == b0;
          }
          const int slot = sp_append(keep, &S.n_list);
          if (slot >= 0 && slot < SP_CAP) {
            S.lv[slot] = q;
            S.li[slot] = c;
          }
        });
        __syncthreads();
        n = S.n_list;
        listed = n <= SP_CAP;
      }
      while (rem > 0) {
        const int take = min(10, rem), sh = rem - take, nb = 1 << take;
        const uint64_t pmask = ~0ull << rem;
        const uint64_t bucket = zk - above;  // mass of the bin being refined
        sp_clear(S, nb);
        __syncthreads();
        if (in_lds) {
          if (tid < nc) {
            const uint64_t q = S.cq[tid];
            if ((q & pmask) == prefix && ((q >> sh) & (nb - 1)))
              atomicAdd((unsigned long long *)&S.hist[(q >> sh) & (nb - 1)], (unsigned long long)q);
          }
        } else if (listed) {
          for (int j = tid; j < n; j += SP_T) {
            const uint64_t q = S.lv[j];
            if ((q & pmask) == prefix && ((q >> sh) & (nb - 1)))
              atomicAdd((unsigned long long *)&S.hist[(q >> sh) & (nb - 1)], (unsigned long long)q);
          }
        } else {
          sp_row(row, V, vec, [&](int, float l, bool ok) {
            if (ok && order_key(l) >= kmin) {
              const uint64_t q = q_weight(l, mx, inv_t);
              if ((q & pmask) == prefix && ((q >> sh) & (nb - 1)))
                atomicAdd((unsigned long long *)&S.hist[(q >> sh) & (nb - 1)], (unsigned long long)q);
            }
          });
        }
        __syncthreads();
        sp_fill_bin0(S, nb, bucket);
        sp_select(S, nb, need, above);
        above = S.sel[0];
        prefix |= S.sel[1] << sh;
        zk = S.sel[2];
        rem = sh;
        __syncthreads();
      }
      tmin = prefix;
    }
    // 5. draw: r in [0, zk), the kept candidate (q >= tmin) whose cumulative
    // interval in vocabulary order holds r
    uint32_t c4[4] = {P.counter[0], P.counter[1], P.counter[2], 0x53414D50u};
    philox4x32_10(c4, P.key[0], P.key[1]);
    const uint64_t r = mul_shift24(zk, c4[0] >> 8, false);
    if (tid == 0) S.found = bi;
    __syncthreads();
    if (in_lds) {
      const int nk = S.n_cand;
      if (tid < nk) {
        const uint64_t q = S.cq[tid];
        const int i = S.ci[tid];
        if (q >= tmin) {
          uint64_t pre = 0;
          for (int j = 0; j < nk; ++j) {
            const uint64_t qj = S.cq[j];
            if (qj >= tmin && S.ci[j] < i) pre += qj;
          }
          if (r >= pre && r < pre + q) S.found = i;
        }
      }
    } else {
      // kept mass of every (step, wave) piece of the row: 256 consecutive
      // elements, in vocabulary order; then the piece that holds r, then the
      // lane, then the element
      const int lane = tid & 63, w = tid >> 6;
      const int steps = (V + 4 * SP_T - 1) / (4 * SP_T), np = steps * 16;
      for (int s0 = 0; s0 < steps; s0 += 8) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = sp_load4(row, ((s0 + u) * SP_T + tid) * 4, V, vec);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int c = ((s0 + u) * SP_T + tid) * 4;
          const float lv4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
          uint64_t loc = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (c + e < V && order_key(lv4[e]) >= kmin) {
              const uint64_t q = q_weight(lv4[e], mx, inv_t);
              if (q >= tmin) loc += q;
            }
          }
#pragma unroll
          for (int o = 32; o > 0; o >>= 1) loc += __shfl_xor(loc, o, 64);
          if (lane == 0 && s0 + u < steps) S.lv[(s0 + u) * 16 + w] = loc;
        }
      }
      __syncthreads();
      // pieces are scanned in runs of per = ceil(np / SP_T) per thread
      const int per = (np + SP_T - 1) / SP_T;
      uint64_t run = 0;
      for (int i = 0; i < per; ++i) {
        const int p = tid * per + i;
        if (p < np) run += S.lv[p];
      }
      uint64_t tot;
      const uint64_t incl = sp_scan(run, S.red, tot);
      uint64_t pre = incl - run;
      if (tid == 0) S.pick = -1;
      __syncthreads();
      if (run > 0 && r >= pre && r < pre + run) {
        for (int i = 0; i < per; ++i) {
          const int p = tid * per + i;
          if (p >= np) break;
          const uint64_t q = S.lv[p];
          if (r < pre + q) {
            S.pick = p;
            S.sel[3] = pre;
            break;
          }
          pre += q;
        }
      }
      __syncthreads();
      const int p = S.pick;
      if (p >= 0 && w == p % 16) {
        const int c = ((p / 16) * SP_T + tid) * 4;
        uint64_t q4[4], loc = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          q4[e] = 0;
          if (c + e < V) {
            const float l = row[c + e];
            if (order_key(l) >= kmin) {
              const uint64_t q = q_weight(l, mx, inv_t);
              if (q >= tmin) q4[e] = q;
            }
          }
          loc += q4[e];
        }
        uint64_t x = loc;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint64_t t = __shfl_up(x, o, 64);
          if (lane >= o) x += t;
        }
        uint64_t pl = S.sel[3] + x - loc;
        if (loc > 0 && r >= pl && r < pl + loc) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (q4[e] && r < pl + q4[e]) {
              S.found = c + e;
              break;
            }
            pl += q4[e];
          }
        }
      }
    }
    __syncthreads();
    token = S.found;
  }
  if (tid == 0) {
    if (out_slot) slot_tok[out_slot[m]] = token;
    tok_out[m] = token;
  }
}

void launch_sample(const float *logits, int64_t ld, int M, int V, const SampleParams *prm, const int32_t *out_slot,
                   int32_t *slot_tok, int32_t *tok_out, hipStream_t s) {
  if (M <= 0) return;
  sample_kernel<<<M, 1024, 0, s>>>(logits, ld, V, prm, out_slot, slot_tok, tok_out);
}

template <typename T>
__global__ void init_weight_kernel(T *dst, uint32_t k0, uint32_t k1, uint32_t tid, int64_t rows,
                                   int64_t cols, float stdv, int perm, int hd, bool bf16_values, bool packed,
                                   int64_t row0, int64_t fused_ns) {
  const int64_t n = rows * cols;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    uint32_t c[4] = {(uint32_t)e, (uint32_t)((uint64_t)e >> 32), tid, 0u};
    philox4x32_10(c, k0, k1);
    int s = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) s += (c[w] & 1023u) + ((c[w] >> 10) & 1023u) + ((c[w] >> 20) & 1023u);
    float v = ((float)(s - 6138) * stdv) * 0x1p-10f;
    if (bf16_values) v = bf16_to_f32(f32_to_bf16(v));
    const int64_t r = e / cols, col = e % cols;
    int64_t dr = r;
    if (perm == PERM_ROPE) {
      const int64_t h = r / hd, i = r % hd;
      dr = h * hd + (i < hd / 2 ? 2 * i : 2 * (i - hd / 2) + 1);
    } else if (perm == PERM_GATE) {
      dr = 2 * r;
    } else if (perm == PERM_UP) {
      dr = 2 * r + 1;
    }
    dst[packed ? wpack_off(row0 + dr, col, fused_ns) : dr * cols + col] = Act<T>::st(v);
  }
}

template <typename T>
void launch_init_weight(T *dst, uint32_t k0, uint32_t k1, uint32_t tensor_id, int64_t rows,
                        int64_t cols, float stdv, int perm, int head_dim, bool bf16_values, bool packed,
                        int64_t row0, int64_t fused_rows, hipStream_t s) {
  const int64_t n = rows * cols;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
  init_weight_kernel<T><<<(unsigned)blocks, 256, 0, s>>>(dst, k0, k1, tensor_id, rows, cols, stdv, perm,
                                                        head_dim, bf16_values, packed, row0,
                                                        wpack_ns(fused_rows));
}

__global__ void fill_f32_kernel(float *dst, int64_t n, float v) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    dst[e] = v;
}

void launch_fill_f32(float *dst, int64_t n, float v, hipStream_t s) {
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  if (n > 0) fill_f32_kernel<<<(unsigned)blocks, 256, 0, s>>>(dst, n, v);
}

#define INST(T)                                                                                   \
  template void launch_embed<T>(const T *, const int32_t *, const int32_t *, const int32_t *,     \
                                const int32_t *, float *, int, int, hipStream_t);                 \
  template void launch_rmsnorm<T>(float *, const float *, int, int64_t, const int32_t *,          \
                                  const float *, T *, int, int, float, hipStream_t);              \
  template void launch_init_weight<T>(T *, uint32_t, uint32_t, uint32_t, int64_t, int64_t, float, \
                                      int, int, bool, bool, int64_t, int64_t, hipStream_t);
INST(float)
INST(bf16_t)
INST(f16_t)
#undef INST

}  // namespace lp
