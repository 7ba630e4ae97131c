// Embedding gather, RMSNorm (with split-K residual folding), greedy argmax and
// the device-side weight generator.
#include "device.hpp"

namespace lp {

// ------------------------------------------------------------------ embedding

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
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = Act<T>::ld(src[c]);
}

template <typename T>
void launch_embed(const T *E, const int32_t *pool, const int32_t *tok_idx, const int32_t *row_slot,
                  const int32_t *slot_tok, float *x, int M, int d, hipStream_t s) {
  if (M <= 0) return;
  embed_kernel<T><<<M, 256, 0, s>>>(E, pool, tok_idx, row_slot, slot_tok, x, d);
}

// ------------------------------------------------------------------ RMSNorm

constexpr int NORM_V4 = 4;  // float4 per thread; the block has d / 16 threads (rounded to waves)

// One workgroup per row.  The residual row, every split-K partial of it and
// the gains are requested before any is used (NP is the partial count), so a
// row costs one memory latency rather than one per partial.
template <typename T, int NP>
__global__ __launch_bounds__(512) void rmsnorm_kernel(float *x, const float *part, int64_t part_stride,
                                                       const int32_t *rows, const float *__restrict__ g,
                                                       T *__restrict__ y, int d, float eps) {
  __shared__ float red[16];
  const int j = blockIdx.x;
  const int src = rows ? rows[j] : j;
  const int d4 = d >> 2;
  const int nt = blockDim.x;
  float4 *xr = (float4 *)(x + (int64_t)src * d);
  const float4 *g4 = (const float4 *)g;
  float4 v[NORM_V4], gv[NORM_V4];
  float4 p[NP > 0 ? NP : 1][NORM_V4];
#pragma unroll
  for (int e = 0; e < NORM_V4; ++e) {
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
  for (int e = 0; e < NORM_V4; ++e) {
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
  for (int e = 0; e < NORM_V4; ++e) {
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
  // whole waves, NORM_V4 float4 per thread (d <= 8192)
  const int threads = std::min(512, std::max(64, ((d / (4 * NORM_V4)) + 63) / 64 * 64));
#define NORM_CASE(NPV)                                                                                  \
  case NPV:                                                                                             \
    rmsnorm_kernel<T, NPV><<<M, threads, 0, s>>>(x, part, part_stride, rows, g, y, d, eps);             \
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

// One workgroup of 1024 threads per row, 16-byte loads; each thread keeps the
// first maximum it meets in increasing index order, and merges prefer the
// larger value, then the lower index.
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
  for (int c = threadIdx.x; c < v4; c += 1024) {
    const float4 q = ((const float4 *)row)[c];
    argmax_merge(best, bi, q.x, 4 * c);
    argmax_merge(best, bi, q.y, 4 * c + 1);
    argmax_merge(best, bi, q.z, 4 * c + 2);
    argmax_merge(best, bi, q.w, 4 * c + 3);
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

__device__ uint64_t block_sum_u64(uint64_t v, uint64_t *red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t t = 0;
  for (int w = 0; w < 16; ++w) t += red[w];
  return t;
}

__global__ __launch_bounds__(1024) void sample_kernel(const float *__restrict__ logits, int64_t ld, int V,
                                                      const SampleParams *__restrict__ prm, const int32_t *out_slot,
                                                      int32_t *slot_tok, int32_t *tok_out) {
  __shared__ float sv[16];
  __shared__ int si[16];
  __shared__ uint64_t red[16];
  __shared__ uint64_t hist[256];
  __shared__ uint32_t cnt[256];
  __shared__ uint64_t sel[4];
  const int m = blockIdx.x, tid = threadIdx.x;
  const float *row = logits + (int64_t)m * ld;
  const SampleParams P = prm[m];
  // 1. maximum (and the greedy answer)
  float best = -INFINITY;
  int bi = 0x7fffffff;
  for (int c = tid; c < V; c += 1024) argmax_merge(best, bi, row[c], c);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) argmax_merge(best, bi, __shfl_xor(best, o, 64), __shfl_xor(bi, o, 64));
  if ((tid & 63) == 0) {
    sv[tid >> 6] = best;
    si[tid >> 6] = bi;
  }
  __syncthreads();
  for (int w = 0; w < 16; ++w) argmax_merge(best, bi, sv[w], si[w]);
  int token = bi;
  if (P.temperature > 0.f && P.top_p > 0.f && V > 1) {
    const float mx = best, inv_t = 1.f / P.temperature;
    // 2. top-k threshold on order keys: the top_k-th largest key
    uint32_t kmin = 0;
    if (P.top_k > 0 && P.top_k < V) {
      uint32_t prefix = 0, above = 0;
      for (int level = 0; level < 4; ++level) {
        const int sh = 24 - 8 * level;
        const uint32_t pmask = level ? (0xFFFFFFFFu << (32 - 8 * level)) : 0u;
        for (int b = tid; b < 256; b += 1024) cnt[b] = 0;
        __syncthreads();
        for (int c = tid; c < V; c += 1024) {
          const uint32_t k = order_key(row[c]);
          if ((k & pmask) == prefix) atomicAdd(&cnt[(k >> sh) & 255u], 1u);
        }
        __syncthreads();
        if (tid == 0) {
          uint32_t acc = above;
          int b = 255;
          for (; b > 0; --b) {
            if (acc + cnt[b] >= (uint32_t)P.top_k) break;
            acc += cnt[b];
          }
          sel[0] = acc;
          sel[1] = (uint64_t)b;
        }
        __syncthreads();
        above = (uint32_t)sel[0];
        prefix |= (uint32_t)sel[1] << sh;
        __syncthreads();
      }
      kmin = prefix;
    }
    // 3. candidate weights and their total
    uint64_t z = 0;
    for (int c = tid; c < V; c += 1024) {
      const float l = row[c];
      if (order_key(l) >= kmin) z += q_weight(l, mx, inv_t);
    }
    z = block_sum_u64(z, red);
    // 4. top-p threshold on weights
    uint64_t tmin = 0, zk = z;
    const uint32_t pfix = P.top_p >= 1.f ? (1u << 24) : max(1u, (uint32_t)(P.top_p * 16777216.0f));
    if (pfix < (1u << 24)) {
      const uint64_t need = mul_shift24(z, pfix, true);
      uint64_t prefix = 0, above = 0;
      for (int level = 0; level < 6; ++level) {
        const int sh = 40 - 8 * level;
        const uint64_t pmask = level ? (~0ull << (48 - 8 * level)) & 0xFFFFFFFFFFFFull : 0ull;
        for (int b = tid; b < 256; b += 1024) hist[b] = 0;
        __syncthreads();
        for (int c = tid; c < V; c += 1024) {
          const float l = row[c];
          if (order_key(l) < kmin) continue;
          const uint64_t q = q_weight(l, mx, inv_t);
          if ((q & pmask) == prefix) atomicAdd((unsigned long long *)&hist[(q >> sh) & 255u], (unsigned long long)q);
        }
        __syncthreads();
        if (tid == 0) {
          uint64_t acc = above;
          int b = 255;
          for (; b > 0; --b) {
            if (acc + hist[b] >= need) break;
            acc += hist[b];
          }
          sel[0] = acc;
          sel[1] = (uint64_t)b;
          sel[2] = acc + hist[b];
        }
        __syncthreads();
        above = sel[0];
        prefix |= sel[1] << sh;
        zk = sel[2];
        __syncthreads();
      }
      tmin = prefix;
    }
    // 5. draw: r in [0, zk), located by a scan over contiguous index chunks
    uint32_t c4[4] = {P.counter[0], P.counter[1], P.counter[2], 0x53414D50u};
    philox4x32_10(c4, P.key[0], P.key[1]);
    const uint64_t r = mul_shift24(zk, c4[0] >> 8, false);
    const int chunk = (V + 1023) / 1024;
    const int c0 = tid * chunk, c1 = min(V, c0 + chunk);
    uint64_t local = 0;
    for (int c = c0; c < c1; ++c) {
      const float l = row[c];
      if (order_key(l) < kmin) continue;
      const uint64_t q = q_weight(l, mx, inv_t);
      if (q >= tmin) local += q;
    }
    // exclusive scan of the per-thread sums (thread order = index order)
    uint64_t incl = local;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t t = __shfl_up(incl, o, 64);
      if ((tid & 63) >= o) incl += t;
    }
    __syncthreads();
    if ((tid & 63) == 63) red[tid >> 6] = incl;
    __syncthreads();
    uint64_t base = 0;
    for (int w = 0; w < (tid >> 6); ++w) base += red[w];
    uint64_t pre = base + incl - local;
    __shared__ int found;
    if (tid == 0) found = bi;
    __syncthreads();
    if (local > 0 && r >= pre && r < pre + local) {
      for (int c = c0; c < c1; ++c) {
        const float l = row[c];
        if (order_key(l) < kmin) continue;
        const uint64_t q = q_weight(l, mx, inv_t);
        if (q < tmin) continue;
        if (r < pre + q) {
          found = c;
          break;
        }
        pre += q;
      }
    }
    __syncthreads();
    token = found;
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
