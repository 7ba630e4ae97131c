// Device-side helpers shared by the kernel sources.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace lp {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest even (finite inputs).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T>
struct Act;
template <>
struct Act<float> {
  static __device__ __forceinline__ float ld(float v) { return v; }
  static __device__ __forceinline__ float st(float v) { return v; }
};
template <>
struct Act<bf16_t> {
  static __device__ __forceinline__ float ld(bf16_t v) { return bf16_to_f32(v); }
  static __device__ __forceinline__ bf16_t st(float v) { return f32_to_bf16(v); }
};

template <>
struct Act<f16_t> {
  static __device__ __forceinline__ float ld(f16_t v) { return (float)v; }
  static __device__ __forceinline__ f16_t st(float v) { return (f16_t)v; }
};

// MFMA instructions per 16-bit element type: 16x16x32 and 32x32x16 tiles,
// fp32 accumulation.
template <typename T>
struct Mfma;
template <>
struct Mfma<bf16_t> {
  typedef bf16x8_t v8;
  static __device__ __forceinline__ floatx4_t m16(v8 a, v8 b, floatx4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ floatx16_t m32(v8 a, v8 b, floatx16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<f16_t> {
  typedef f16x8_t v8;
  static __device__ __forceinline__ floatx4_t m16(v8 a, v8 b, floatx4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ floatx16_t m32(v8 a, v8 b, floatx16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

template <typename T>
__device__ __forceinline__ typename Mfma<T>::v8 load8(const T *p) {
  return __builtin_bit_cast(typename Mfma<T>::v8, *(const uint4 *)p);
}
template <typename T>
__device__ __forceinline__ typename Mfma<T>::v8 zero8() {
  return __builtin_bit_cast(typename Mfma<T>::v8, make_uint4(0, 0, 0, 0));
}


__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// Element offset of (layer, slot-position, kv head) in the K cache (row of hd)
// and the V cache (column inside a transposed [hd][BS] block).
__device__ __forceinline__ int64_t kv_block_base(const KVCache &kv, int layer, int slot, int pos,
                                                 int h) {
  const int blk = kv.block_table[(int64_t)slot * kv.max_blocks + pos / KV_BLOCK];
  return (((int64_t)layer * kv.n_blocks + blk) * kv.n_kv_heads + h) * (int64_t)KV_BLOCK * kv.head_dim;
}

// Max / sum over the 16 lanes of a DPP row (lanes 16r .. 16r+15), the result
// in every lane of the row, in registers: swap within quads (xor 1, xor 2),
// then combine mirrored half-rows and mirrored rows.  Each step combines two
// equal partial results in either order, so all lanes end with the same value.
template <typename F>
__device__ __forceinline__ float row16_reduce(float v, F op) {
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false)));  // quad_perm 1,0,3,2
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false)));  // quad_perm 2,3,0,1
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false))); // row_half_mirror
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false))); // row_mirror
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  return row16_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float row16_sum(float v) {
  return row16_reduce(v, [](float a, float b) { return a + b; });
}

// Sum / max over the 64 lanes of a wave, the same value in every lane: the
// four row results combined in a fixed order.
__device__ __forceinline__ float wave_sum(float v) {
  v = row16_sum(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}
__device__ __forceinline__ float wave_max(float v) {
  v = row16_max(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

// The value of lane l ^ 1 (the neighbour within a lane pair).
__device__ __forceinline__ float lane_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

// 16 bytes per lane from global memory straight into LDS (gfx950's
// global_load_lds_dwordx4): lane l's bytes land at LDS byte address
// `lds` + 16 l, `lds` wave-uniform.  The load counts on vmcnt like any vector
// load but is invisible to the compiler's wait-count tracking: callers wait
// for it explicitly (s_waitcnt vmcnt) before a barrier and reading the data.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(g) : "memory", "m0");
}

// LDS byte address of a __shared__ object (for dma16).
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char *)p;
}

// Rotary embedding of one pair (x0, x1) = (dimension i, dimension i + hd/2)
// at angle theta, cs = cos theta, sn = sin theta.  Every kernel that rotates
// a pair rounds it the same way: the fused multiply-adds are explicit, and
// the results are held as fp32 (the empty asm), so that a 16-bit store of
// them is not fused into a mixed-precision FMA that rounds once to 16 bits.
__device__ __forceinline__ void rope_rotate(float x0, float x1, float cs, float sn, float &r0, float &r1) {
  r0 = fmaf(x0, cs, -(x1 * sn));
  r1 = fmaf(x1, cs, x0 * sn);
  asm("" : "+v"(r0), "+v"(r1));
}

// Applies the epilogue to output columns (n, n+1) of row m, n even.
template <typename T>
__device__ __forceinline__ void epi_pair(const Epi &ep, int m, int n, float v0, float v1) {
  switch (ep.kind) {
    case EPI_STORE:
    case EPI_LOGITS: {
      float2 *p = (float2 *)(ep.out + (int64_t)m * ep.ldo + n);
      *p = make_float2(v0, v1);
      break;
    }
    case EPI_RESID: {
      float2 *p = (float2 *)(ep.out + (int64_t)m * ep.ldo + n);
      float2 r = *p;
      r.x += v0;
      r.y += v1;
      *p = r;
      break;
    }
    case EPI_SILU: {
      T *h = (T *)ep.act_out;
      h[(int64_t)m * ep.ld_act + (n >> 1)] = Act<T>::st(silu(v0) * v1);
      break;
    }
    case EPI_QKV: {
      const int hd = ep.kv.head_dim;
      const int qdim = ep.n_heads * hd;
      const int kvdim = ep.kv.n_kv_heads * hd;
      const int slot = ep.rows.row_slot[m];
      const int pos = ep.rows.row_pos[m];
      if (n < qdim + kvdim) {
        const bool is_q = n < qdim;
        const int c = is_q ? n : n - qdim;
        const int h = c / hd;
        const int i = (c % hd) >> 1;  // rotary pair index
        const float cs = ep.rope_cos[(int64_t)pos * (hd >> 1) + i];
        const float sn = ep.rope_sin[(int64_t)pos * (hd >> 1) + i];
        float r0, r1;
        rope_rotate(v0, v1, cs, sn, r0, r1);
        if (is_q) {
          T *q = (T *)ep.act_out + (int64_t)m * ep.ld_act + h * hd;
          q[i] = Act<T>::st(r0);
          q[i + (hd >> 1)] = Act<T>::st(r1);
        } else {
          T *k = (T *)ep.kv.k + kv_block_base(ep.kv, ep.layer, slot, pos, h) +
                 (int64_t)(pos % KV_BLOCK) * hd;
          k[i] = Act<T>::st(r0);
          k[i + (hd >> 1)] = Act<T>::st(r1);
        }
      } else {
        const int c = n - qdim - kvdim;
        const int h = c / hd;
        const int j = c % hd;
        T *vt = (T *)ep.kv.v + kv_block_base(ep.kv, ep.layer, slot, pos, h) + (pos % KV_BLOCK);
        vt[(int64_t)j * KV_BLOCK] = Act<T>::st(v0);
        vt[(int64_t)(j + 1) * KV_BLOCK] = Act<T>::st(v1);
      }
      break;
    }
  }
}

}  // namespace lp
