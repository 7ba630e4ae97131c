// Single-kernel entry points (include/lp_ops.h).
#include <hip/hip_runtime.h>

#include <string>

#include "../../include/lp_ops.h"
#include "kernels.hpp"

using namespace lp;

std::string &lp_global_error();
#define lp_ops_err lp_global_error()

#define OPCHK(cond, msg)          \
  do {                            \
    if (!(cond)) {                \
      lp_ops_err = (msg);         \
      return LP_EINVAL;           \
    }                             \
  } while (0)

static int op_status() {
  hipError_t s = hipGetLastError();
  if (s != hipSuccess) {
    lp_ops_err = hipGetErrorString(s);
    return LP_EHIP;
  }
  return LP_OK;
}

extern "C" int lp_op_gemm(int32_t dtype, const void *X, int64_t ldx, const void *W, float *Y, int32_t M, int32_t N,
                          int32_t K, int32_t k_splits, void *ws, size_t ws_bytes, void *stream) {
  OPCHK(M >= 0 && N > 0 && K > 0, "gemm: bad sizes");
  OPCHK(K % 8 == 0 && N % 2 == 0 && ldx >= K && ldx % 8 == 0, "gemm: K % 8, N % 2, ldx");
  OPCHK(dtype == LP_F32 || dtype == LP_BF16 || dtype == LP_F16, "gemm: dtype");
  if (M == 0) return LP_OK;  // no rows: nothing is read or written
  OPCHK(X && W && Y, "gemm: bad pointers");
  hipStream_t s = (hipStream_t)stream;
  Epi ep{};
  ep.kind = EPI_STORE;
  ep.out = Y;
  ep.ldo = N;
  if (dtype != LP_F32) {
    int splits = 1;
    if (k_splits > 1) {
      splits = gemm_effective_splits(M, N, K, k_splits);
      OPCHK(splits == 1 || (ws && ws_bytes >= (size_t)splits * M * N * 4), "gemm: workspace too small for split-K");
    }
    if (dtype == LP_BF16) {
      launch_gemm<bf16_t>((const bf16_t *)X, ldx, (const bf16_t *)W, M, N, K, splits, (float *)ws, ep, s);
      if (splits > 1) launch_gemm_finish<bf16_t>((const float *)ws, splits, M, N, ep, s);
    } else {
      launch_gemm<f16_t>((const f16_t *)X, ldx, (const f16_t *)W, M, N, K, splits, (float *)ws, ep, s);
      if (splits > 1) launch_gemm_finish<f16_t>((const float *)ws, splits, M, N, ep, s);
    }
  } else {
    launch_gemm<float>((const float *)X, ldx, (const float *)W, M, N, K, 1, nullptr, ep, s);
  }
  return op_status();
}

extern "C" int lp_op_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t k_splits, int32_t *kind,
                               int32_t *tile_rows, int32_t *splits, int32_t *xcd_group) {
  OPCHK(M > 0 && N > 0 && K > 0 && kind && tile_rows && splits && xcd_group, "gemm plan: bad sizes or pointers");
  int k = 0, r = 0, sp = 0, xg = 0;
  gemm_plan_info(M, N, K, k_splits, &k, &r, &sp, &xg);
  *kind = k;
  *tile_rows = r;
  *splits = sp;
  *xcd_group = xg;
  return LP_OK;
}

extern "C" size_t lp_op_packed_weight_bytes(int32_t dtype, int32_t N, int32_t K) {
  if ((dtype != LP_BF16 && dtype != LP_F16) || N <= 0 || K <= 0) return 0;
  return (size_t)wpack_elems(N, K) * 2;
}

extern "C" int lp_op_pack_weight(int32_t dtype, const void *W, void *W_packed, int32_t N, int32_t K, void *stream) {
  OPCHK(W && W_packed && N > 0 && K > 0 && K % 8 == 0, "pack weight: bad pointers or sizes (K % 8 == 0)");
  OPCHK(dtype == LP_BF16 || dtype == LP_F16, "pack weight: 16-bit dtypes only");
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LP_BF16)
    launch_wpack<bf16_t>((const bf16_t *)W, (bf16_t *)W_packed, N, K, s);
  else
    launch_wpack<f16_t>((const f16_t *)W, (f16_t *)W_packed, N, K, s);
  return op_status();
}

extern "C" int lp_op_rmsnorm(int32_t dtype, float *x, const float *part, int32_t n_part, const float *g, void *y,
                             int32_t rows, int32_t d, float eps, void *stream) {
  OPCHK(rows >= 0 && d > 0 && d <= 8192 && n_part >= 0, "rmsnorm: sizes");
  if (rows == 0) return LP_OK;  // no rows: nothing is read or written
  OPCHK(x && g && y && (n_part == 0 || part), "rmsnorm: pointers");
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LP_BF16)
    launch_rmsnorm<bf16_t>(x, part, n_part, (int64_t)rows * d, nullptr, g, (bf16_t *)y, rows, d, eps, s);
  else if (dtype == LP_F16)
    launch_rmsnorm<f16_t>(x, part, n_part, (int64_t)rows * d, nullptr, g, (f16_t *)y, rows, d, eps, s);
  else if (dtype == LP_F32)
    launch_rmsnorm<float>(x, part, n_part, (int64_t)rows * d, nullptr, g, (float *)y, rows, d, eps, s);
  else
    OPCHK(false, "rmsnorm: dtype");
  return op_status();
}

extern "C" size_t lp_op_decode_attention_ws_bytes(int32_t M, int32_t n_heads, int32_t head_dim, int32_t max_ctx) {
  return decode_attention_ws_bytes(M, n_heads, head_dim, max_ctx);
}

static int check_heads(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int32_t dtype) {
  OPCHK(n_heads > 0 && n_kv_heads > 0 && n_heads % n_kv_heads == 0, "attention: heads");
  const int G = n_heads / n_kv_heads;
  OPCHK(G == 1 || G == 2 || G == 4 || G == 8, "attention: group size must be 1, 2, 4 or 8");
  OPCHK(head_dim == 64 || head_dim == 128, "attention: head_dim must be 64 or 128");
  OPCHK(dtype == LP_BF16 || dtype == LP_F16 || (dtype == LP_F32 && head_dim == 64), "attention: dtype / head_dim");
  return LP_OK;
}

extern "C" int lp_op_decode_attention(int32_t dtype, const void *q, void *out, const void *k_cache,
                                      const void *v_cache, const int32_t *block_table, int32_t max_blocks,
                                      int64_t n_blocks, const int32_t *row_slot, const int32_t *row_pos, int32_t M,
                                      int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx,
                                      void *ws, size_t ws_bytes, void *stream) {
  int rc = check_heads(n_heads, n_kv_heads, head_dim, dtype);
  if (rc) return rc;
  OPCHK(M >= 0 && max_ctx > 0, "decode attention: sizes");
  OPCHK(max_blocks * 64 >= max_ctx, "decode attention: max_blocks too small for max_ctx");
  if (M == 0) return LP_OK;  // no rows: nothing is read or written
  OPCHK(q && out && k_cache && v_cache && block_table && row_slot && row_pos, "decode attention: pointers");
  OPCHK(ws && ws_bytes >= decode_attention_ws_bytes(M, n_heads, head_dim, max_ctx), "decode attention: ws");
  KVCache kv{(void *)k_cache, (void *)v_cache, block_table, max_blocks, n_blocks, n_kv_heads, head_dim};
  RowMeta rows{row_slot, row_pos};
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LP_BF16)
    launch_decode_attention<bf16_t>((const bf16_t *)q, (bf16_t *)out, rows, kv, 0, M, n_heads, max_ctx, 0,
                                    (float *)ws, s);
  else if (dtype == LP_F16)
    launch_decode_attention<f16_t>((const f16_t *)q, (f16_t *)out, rows, kv, 0, M, n_heads, max_ctx, 0,
                                   (float *)ws, s);
  else
    launch_decode_attention<float>((const float *)q, (float *)out, rows, kv, 0, M, n_heads, max_ctx, 0,
                                   (float *)ws, s);
  return op_status();
}

extern "C" int lp_op_prefill_attention(int32_t dtype, const void *q, void *out, const void *k_cache,
                                       const void *v_cache, const int32_t *block_table, int32_t max_blocks,
                                       int64_t n_blocks, const int32_t *seq_start, const int32_t *seq_slot,
                                       int32_t n_seq, int32_t max_len, int32_t n_heads, int32_t n_kv_heads,
                                       int32_t head_dim, void *stream) {
  int rc = check_heads(n_heads, n_kv_heads, head_dim, dtype);
  if (rc) return rc;
  OPCHK(n_seq >= 0 && max_len > 0, "prefill attention: sizes");
  OPCHK(max_blocks * 64 >= max_len, "prefill attention: max_blocks too small for max_len");
  if (n_seq == 0) return LP_OK;  // no sequences: nothing is read or written
  OPCHK(q && out && k_cache && v_cache && block_table && seq_start && seq_slot, "prefill attention: pointers");
  KVCache kv{(void *)k_cache, (void *)v_cache, block_table, max_blocks, n_blocks, n_kv_heads, head_dim};
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LP_BF16)
    launch_prefill_attention<bf16_t>((const bf16_t *)q, (bf16_t *)out, seq_start, seq_slot, n_seq, max_len, kv, 0,
                                     n_heads, s);
  else if (dtype == LP_F16)
    launch_prefill_attention<f16_t>((const f16_t *)q, (f16_t *)out, seq_start, seq_slot, n_seq, max_len, kv, 0,
                                    n_heads, s);
  else
    launch_prefill_attention<float>((const float *)q, (float *)out, seq_start, seq_slot, n_seq, max_len, kv, 0,
                                    n_heads, s);
  return op_status();
}

extern "C" int lp_op_argmax(const float *logits, int64_t ld, int32_t M, int32_t V, int32_t *tokens, void *stream) {
  OPCHK(M >= 0 && V > 0 && ld >= V, "argmax: sizes");
  if (M == 0) return LP_OK;  // no rows: nothing is read or written
  OPCHK(logits && tokens, "argmax: pointers");
  launch_argmax(logits, ld, M, V, nullptr, nullptr, tokens, (hipStream_t)stream);
  return op_status();
}

extern "C" int lp_op_sample(const float *logits, int64_t ld, int32_t M, int32_t V, const lp_sample_params *params,
                            int32_t *tokens, void *stream) {
  OPCHK(M >= 0 && V > 0 && ld >= V, "sample: sizes");
  OPCHK(V <= SAMPLE_MAX_V, "sample: rows of at most 2^21 logits");
  if (M == 0) return LP_OK;  // no rows: nothing is read or written
  OPCHK(logits && params && tokens, "sample: pointers");
  static_assert(sizeof(lp_sample_params) == sizeof(SampleParams), "sampling parameter layout");
  launch_sample(logits, ld, M, V, (const SampleParams *)params, nullptr, nullptr, tokens, (hipStream_t)stream);
  return op_status();
}

extern "C" int lp_op_init_weight(int32_t dtype, void *dst, uint64_t seed, int32_t tensor_id, int64_t rows,
                                 int64_t cols, float stdv, void *stream) {
  OPCHK(dst && rows > 0 && cols > 0 && tensor_id >= 0, "init_weight: args");
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LP_BF16)
    launch_init_weight<bf16_t>((bf16_t *)dst, (uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)tensor_id, rows,
                               cols, stdv, PERM_NONE, 0, false, false, 0, 0, s);
  else if (dtype == LP_F16)
    launch_init_weight<f16_t>((f16_t *)dst, (uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)tensor_id, rows,
                              cols, stdv, PERM_NONE, 0, true, false, 0, 0, s);
  else if (dtype == LP_F32)
    launch_init_weight<float>((float *)dst, (uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)tensor_id, rows, cols,
                              stdv, PERM_NONE, 0, false, false, 0, 0, s);
  else
    OPCHK(false, "init_weight: dtype");
  return op_status();
}
