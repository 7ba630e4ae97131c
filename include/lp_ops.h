/* lp_ops.h -- single-kernel entry points of the serving step, for parity
 * checks and kernel timing.  They launch exactly the kernels the engine runs,
 * on caller-provided device buffers, asynchronously on `hip_stream` (a
 * hipStream_t, NULL for the null stream).  All pointers are device pointers
 * unless stated otherwise; the caller owns every buffer.  Each returns LP_OK or
 * LP_EINVAL (bad sizes; checked before any launch) or LP_EHIP (launch error);
 * lp_last_error(NULL) then holds a message.  A call with no rows (M, rows or
 * n_seq equal to 0) checks its sizes, then returns LP_OK without a launch or
 * any memory access; its pointers may be null.
 *
 * `dtype` is LP_F32, LP_BF16 or LP_F16: the element type of weights and
 * activations (bf16 as raw 16-bit patterns).  Accumulation is fp32 in all.
 */
#ifndef LP_OPS_H
#define LP_OPS_H

#include <stddef.h>
#include <stdint.h>

#include "lp.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Y[M x N] (fp32, row stride N) = X[M x K] (row stride ldx) times W[N x K]^T:
 * the weight-GEMM contraction of every projection of the decoder (Q/K/V,
 * output, gate/up, down, LM head) that both phases of Sec. II-A run every
 * token through (the paper fixes no layer math; the Llama-style decoder is
 * a reading).  For LP_BF16 / LP_F16, W is in the tiled
 * weight layout that lp_op_pack_weight writes; for LP_F32 it is row-major
 * [N x K].  16-bit types with M <= 64 take the decode kernel, larger M the
 * prefill kernel; `k_splits` > 1 splits K across workgroups (prefill: only
 * when K is a multiple of 128; the count is rounded to whole K chunks) and
 * needs `ws` of at least k_splits * M * N * 4 bytes (fp32 partials).  K must
 * be a multiple of 8, N even; 16-byte aligned rows. */
int lp_op_gemm(int32_t dtype, const void *X, int64_t ldx, const void *W, float *Y, int32_t M, int32_t N,
               int32_t K, int32_t k_splits, void *ws, size_t ws_bytes, void *hip_stream);

/* Which kernel lp_op_gemm (16-bit types) runs for this shape and split
 * request, for the same contraction as above: `kind` 0 = decode kernel
 * (M <= 64), 1 = prefill kernel with one workgroup per CU, 2 = prefill
 * kernel with two 128-row workgroups per CU, 3 = LDS-tiled kernel (K not a
 * multiple of 128); `tile_rows` = rows per output tile; `splits` = the K
 * splits it uses; `xcd_group` = row tiles per group of the prefill kernel's
 * XCD-aware tile order, 0 for the plain order.  `k_splits` as for lp_op_gemm, except that 0 asks for the
 * split count a prefill step of the engine chooses by itself for M > 64.
 * Host-only, no device call.  Returns LP_EINVAL for non-positive sizes or
 * null outputs. */
int lp_op_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t k_splits, int32_t *kind, int32_t *tile_rows,
                    int32_t *splits, int32_t *xcd_group);

/* The tiled weight layout of the 16-bit GEMMs (weights of Sec. II-A's
 * decoder, stored for the decode phase's weight stream).  A row-major [N x K]
 * matrix W (row n = output feature n, stride K, K % 8 == 0) becomes
 * ceil(N/16) * ceil(K/32) tiles of 16 rows x 32 columns, 512 elements (1 KB) each;
 * tile (i, j) has index j * ceil(N/16) + i (the tiles of one 32-column step
 * side by side) and holds rows 16i..16i+15, columns 32j..32j+31, its element
 * (r, c) at position
 * 8 * (r + 16 * (c / 8)) + c % 8.  Rows >= N and columns >= K are zero.
 * lp_op_packed_weight_bytes gives the size (0 for other dtypes or
 * non-positive sizes); lp_op_pack_weight writes W_packed (device, that many
 * bytes, caller-owned, 16-byte aligned like W) on `hip_stream`.  LP_EINVAL for
 * null pointers, bad sizes or a dtype other than LP_BF16 / LP_F16. */
size_t lp_op_packed_weight_bytes(int32_t dtype, int32_t N, int32_t K);
int lp_op_pack_weight(int32_t dtype, const void *W, void *W_packed, int32_t N, int32_t K, void *hip_stream);

/* RMSNorm of the decoder layer (run by both phases of Sec. II-A; the norm is
 * a reading of the architecture, which the paper leaves open):
 * y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g for r < rows; x fp32
 * [rows x d] (first incremented in place by the n_part fp32 partial arrays
 * part[s][rows][d] when n_part > 0), g fp32 [d], y [rows x d] in dtype.
 * d <= 8192. */
int lp_op_rmsnorm(int32_t dtype, float *x, const float *part, int32_t n_part, const float *g, void *y,
                  int32_t rows, int32_t d, float eps, void *hip_stream);

/* Decode attention of one layer (Sec. II-A's decode phase reads the KV cache
 * of every earlier position).  q, out: [M x Hq x hd] in dtype.  KV cache of
 * one layer in blocks of 64 tokens: k_cache [n_blocks][Hkv][64][hd],
 * v_cache [n_blocks][Hkv][hd][64] (transposed per block); block_table
 * [*][max_blocks] int32 lists each slot's blocks.  Row m reads slot
 * row_slot[m] over positions 0..row_pos[m] (ctx = row_pos[m] + 1 <= max_ctx;
 * a larger ctx is clamped to max_ctx, so the kernels stay inside ws and the
 * first max_ctx positions of the block table).
 * ws: at least lp_op_decode_attention_ws_bytes(M, Hq, hd, max_ctx) bytes. */
size_t lp_op_decode_attention_ws_bytes(int32_t M, int32_t n_heads, int32_t head_dim, int32_t max_ctx);
int lp_op_decode_attention(int32_t dtype, const void *q, void *out, const void *k_cache, const void *v_cache,
                           const int32_t *block_table, int32_t max_blocks, int64_t n_blocks,
                           const int32_t *row_slot, const int32_t *row_pos, int32_t M, int32_t n_heads,
                           int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx, void *ws, size_t ws_bytes,
                           void *hip_stream);

/* lp_op_decode_attention without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Arguments, layouts and results
 * are those of lp_op_decode_attention; the chunk partials go to a static
 * device array of LP_NOALLOC_SCRATCH_BYTES (32 MiB) that the library holds on
 * every GPU it runs on until the process ends.  The call allocates and frees
 * nothing.  LP_EINVAL when lp_op_decode_attention_ws_bytes(M, n_heads,
 * head_dim, max_ctx) exceeds the array (64 rows of 32 heads of head_dim 128
 * fit contexts up to 7,936 positions), checked before any device call.  Every
 * call on one GPU shares that GPU's array: calls that overlap in time on one
 * GPU (other streams, other threads) race and must be serialised by the
 * caller. */
#define LP_NOALLOC_SCRATCH_BYTES (32u << 20)
int lp_op_decode_attention_noalloc(int32_t dtype, const void *q, void *out, const void *k_cache,
                                   const void *v_cache, const int32_t *block_table, int32_t max_blocks,
                                   int64_t n_blocks, const int32_t *row_slot, const int32_t *row_pos, int32_t M,
                                   int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx,
                                   void *hip_stream);

/* Causal prefill attention of one layer over packed prompts (Sec. II-A's
 * prompt processing): sequence j owns rows [seq_start[j], seq_start[j+1]) of
 * q/out ([rows x Hq x hd]) at positions 0.., and its keys/values are already
 * in the cache of slot seq_slot[j] (layout as above).  max_len bounds every
 * sequence length. */
int lp_op_prefill_attention(int32_t dtype, const void *q, void *out, const void *k_cache, const void *v_cache,
                            const int32_t *block_table, int32_t max_blocks, int64_t n_blocks,
                            const int32_t *seq_start, const int32_t *seq_slot, int32_t n_seq, int32_t max_len,
                            int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, void *hip_stream);

/* Greedy decoding, the token choice of each prefill and decode step of Sec.
 * II-A under greedy requests: tokens[m] = argmax of logits row m (fp32, row
 * stride ld), lowest index on ties.  tokens [M] int32 (device). */
int lp_op_argmax(const float *logits, int64_t ld, int32_t M, int32_t V, int32_t *tokens, void *hip_stream);

/* The device weight generator (see lp_init_weights_random): dst[rows x cols]
 * in dtype gets element (r, c) of canonical tensor `tensor_id`, unpermuted;
 * LP_F16 stores the bf16-rounded value (as a bf16 model held in fp16). */
int lp_op_init_weight(int32_t dtype, void *dst, uint64_t seed, int32_t tensor_id, int64_t rows, int64_t cols,
                      float std, void *hip_stream);

/* Sampling parameters of one row (requests carry them, Sec. III-A):
 * temperature <= 0 or top_p <= 0 mean greedy; top_k 0 means no top-k limit;
 * top_p >= 1 means no nucleus limit; key / counter: the Philox4x32-10 key
 * and the first three counter words of the row's random draw (the fourth is
 * the constant 0x53414D50). */
typedef struct {
  float temperature;
  int32_t top_k;
  float top_p;
  uint32_t key[2];
  uint32_t counter[3];
} lp_sample_params;

/* Next token of each of M rows of fp32 logits (row stride ld >= V) under its
 * sampling parameters; tokens [M] int32 (device).  Greedy rows take the
 * lowest index among the maxima.  Otherwise, with m the row maximum:
 * candidates are all tokens, or for 0 < top_k < V the tokens whose logit is
 * at least the top_k-th largest (ties kept); a candidate's weight is
 * q = floor(exp((logit - m) / temperature) * 2^40); for top_p < 1 the kept
 * candidates are those with q >= t, t the largest value whose heavier-or-
 * equal candidates weigh at least ceil(Z * floor(top_p * 2^24) / 2^24) (Z the
 * candidates' total); the draw r = floor(Z_kept * u24 / 2^24), u24 the first
 * Philox output word >> 8, picks the kept candidate, in vocabulary order,
 * whose cumulative weight interval holds r.  V <= 2^21 (LP_EINVAL beyond). */
int lp_op_sample(const float *logits, int64_t ld, int32_t M, int32_t V, const lp_sample_params *params,
                 int32_t *tokens, void *hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* LP_OPS_H */
