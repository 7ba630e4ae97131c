// Kernel launch interface shared by the engine and the op-level entry points.
// All pointers are device pointers; every launch goes on the given stream.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lp {

constexpr int KV_BLOCK = 64;  // tokens per KV-cache block

// bf16 stored as raw 16-bit patterns; fp16 as the native half type.
typedef uint16_t bf16_t;
typedef _Float16 f16_t;

// Tiled layout of 16-bit weight matrices, read by every 16-bit GEMM kernel.
// An [N x K] matrix (row n is output feature n, K its inputs) is cut into
// tiles of 16 rows x 32 columns, 1 KB each.  Tile (i, j) holds rows
// 16i..16i+15 and columns 32j..32j+31 and has index j * ceil(N/16) + i: the
// tiles of one K step follow each other across the slices, so waves that
// stream their slices side by side in K read one compact, moving region of
// the matrix.  Inside a tile the 8 elements of lane l = r + 16q (r < 16,
// q < 4) are row 16i + r, columns 32j + 8q .. 32j + 8q + 7: the B operand of
// a 16x16x32 MFMA, so a wave reads a tile with one contiguous 1 KB load.
// Rows past N and columns past K are zero.
constexpr int WT_ROWS = 16, WT_COLS = 32, WT_ELEMS = WT_ROWS * WT_COLS;
__host__ __device__ inline int64_t wpack_kt(int64_t K) { return (K + WT_COLS - 1) / WT_COLS; }
__host__ __device__ inline int64_t wpack_ns(int64_t N) { return (N + WT_ROWS - 1) / WT_ROWS; }
__host__ __device__ inline int64_t wpack_elems(int64_t N, int64_t K) { return wpack_ns(N) * wpack_kt(K) * WT_ELEMS; }
// Element offset of (n, k) for a matrix with ns = wpack_ns(N) 16-row slices.
__host__ __device__ inline int64_t wpack_off(int64_t n, int64_t k, int64_t ns) {
  return ((k >> 5) * ns + (n >> 4)) * WT_ELEMS + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7);
}

// Where the rows of a step read their token and write their results.
struct RowMeta {
  const int32_t *row_slot;  // [M] KV slot of each row
  const int32_t *row_pos;   // [M] position of the row's token in its sequence
};

// KV cache of all layers: K [L][NB][Hkv][BS][hd], V transposed per block:
// Vt [L][NB][Hkv][hd][BS]; element type = activation type.
struct KVCache {
  void *k;
  void *v;
  const int32_t *block_table;  // [max_batch][max_blocks]
  int32_t max_blocks;          // blocks per slot
  int64_t n_blocks;            // blocks per layer
  int32_t n_kv_heads, head_dim;
};

enum EpiKind : int {
  EPI_STORE = 0,   // out_f32[m, n] = acc
  EPI_QKV = 1,     // RoPE on q/k pairs, q -> q_out, k/v -> KV cache
  EPI_RESID = 2,   // resid[m, n] += acc
  EPI_SILU = 3,    // h[m, n/2] = silu(acc[2f]) * acc[2f+1]
  EPI_LOGITS = 4,  // logits[m, n] = acc (fp32)
};

// Arguments of the GEMM epilogues.  Columns are processed in pairs (n, n+1),
// n even; the weight rows are stored so that each pair belongs together
// (rotary pairs of q/k, gate/up rows of the MLP).
struct Epi {
  int kind;
  float *out;        // EPI_STORE / EPI_LOGITS: [M x ldo] fp32; EPI_RESID: [M x ldo]
  int64_t ldo;
  void *act_out;     // EPI_QKV: q [M x Hq*hd]; EPI_SILU: h [M x F] (activation type)
  int64_t ld_act;
  // EPI_QKV
  RowMeta rows;
  KVCache kv;
  int32_t layer, n_heads;
  const float *rope_cos;  // [max_pos][hd/2]
  const float *rope_sin;
};

// ---------------------------------------------------------------- launches

// x[M, d] (fp32) = embedding rows; token of row m: pool[tok_idx[m]] if
// tok_idx[m] >= 0, else slot_tok[row_slot[m]].
template <typename T>
void launch_embed(const T *E, const int32_t *pool, const int32_t *tok_idx, const int32_t *row_slot,
                  const int32_t *slot_tok, float *x, int M, int d, hipStream_t s);

// Optionally folds split-K partials into the residual (x[r] += sum_s part[s][r]),
// then y[j] = rmsnorm(x[src(j)]) * g where src(j) = rows ? rows[j] : j.
template <typename T>
void launch_rmsnorm(float *x, const float *part, int n_part, int64_t part_stride,
                    const int32_t *rows, const float *g, T *y, int M, int d, float eps,
                    hipStream_t s);

// Generic GEMM Y = X W^T with epilogue.  T = float, bf16_t or f16_t.  W is
// in the tiled weight layout for 16-bit T, row-major [N x K] for float.
// splits > 1 (16-bit only): writes partials [splits][M][N] into `part` and a
// following launch_gemm_finish (or an RMSNorm fold) applies the epilogue;
// gemm_effective_splits gives the count a launch uses for a requested one.
// timing (optional, two events): recorded with the kernel's own dispatch, so
// their interval is the kernel's execution alone.
template <typename T>
void launch_gemm(const T *X, int64_t ldx, const T *W, int M, int N, int K, int splits,
                 float *part, const Epi &ep, hipStream_t s, const hipEvent_t *timing = nullptr);

int gemm_effective_splits(int M, int N, int K, int splits);
// The kernel a launch_gemm of this shape and split request runs: its kind,
// rows per output tile, effective K splits and the row tiles per XCD group of
// its tile order (0: plain order).
enum GemmKind : int { GEMM_KIND_DECODE = 0, GEMM_KIND_PREFILL = 1, GEMM_KIND_PREFILL_PAIR = 2, GEMM_KIND_TILED = 3 };
void gemm_plan_info(int M, int N, int K, int splits, int *kind, int *rows, int *eff_splits, int *xcd_group);
// K splits the prefill GEMM (M > 64) takes for its shape (1 when the tile grid
// fills the chip); an effective count.
int prefill_gemm_splits(int M, int N, int K);

// Packs a row-major [N x K] 16-bit matrix (row stride K) into the tiled
// weight layout at dst (wpack_elems(N, K) elements, padding zeroed).
template <typename T>
void launch_wpack(const T *src, T *dst, int N, int K, hipStream_t s);

template <typename T>
void launch_gemm_finish(const float *part, int splits, int M, int N, const Epi &ep, hipStream_t s);

// Decode attention: row m attends to ctx = min(row_pos[m] + 1, max_ctx)
// cached positions of its slot.  q [M][Hq][hd], out [M][Hq][hd] (activation
// type).  Uses workspace `ws` (see decode_attention_ws_bytes).  `items` is the
// rows' total chunk count, the sum of decode_attention_chunks(ctx) over the
// rows, which sizes the grid to the live work; 0 launches the upper bound
// M * decode_attention_chunks(max_ctx), whose surplus workgroups exit.
//
// With `qkv` (16-bit types only): q is not read.  The attention kernel
// finishes the split-K QKV projection itself: it sums the fp32 partials
// [splits][M][N] of its row and heads in split order, applies the rotary
// embedding to q and k, writes the row's new K and V entry into the cache
// (the workgroup of the row's last chunk) and uses that entry in registers,
// all with the arithmetic of launch_gemm_finish's EPI_QKV epilogue.
struct QkvParts {
  const float *part;  // [splits][M][N] fp32, N = (Hq + 2 Hkv) hd, rotary pairs adjacent
  int splits, N;
  const float *rope_cos, *rope_sin;  // [positions][hd / 2]
};
// Whether launch_decode_attention can take `qkv` for a query-head group of
// that size and that many QKV splits (it launches nothing where it cannot).
bool decode_attention_fuses_qkv(int group, int head_dim, int splits);
size_t decode_attention_ws_bytes(int M, int n_heads, int head_dim, int max_ctx);
int decode_attention_chunks(int ctx);
template <typename T>
void launch_decode_attention(const T *q, T *out, const RowMeta &rows, const KVCache &kv, int layer,
                             int M, int n_heads, int max_ctx, int items, float *ws, hipStream_t s,
                             const QkvParts *qkv = nullptr);

// Prefill (causal) attention over packed sequences: sequence j covers rows
// [seq_start[j], seq_start[j+1]) at positions 0.., KV slot seq_slot[j].
template <typename T>
void launch_prefill_attention(const T *q, T *out, const int32_t *seq_start, const int32_t *seq_slot,
                              int n_seq, int max_len, const KVCache &kv, int layer, int n_heads,
                              hipStream_t s);

// Greedy token per row (lowest index on ties): tok -> slot_tok[out_slot[m]]
// and tok_log[m].
void launch_argmax(const float *logits, int64_t ld, int M, int V, const int32_t *out_slot,
                   int32_t *slot_tok, int32_t *tok_log, hipStream_t s);

// Sampling parameters of one row: temperature (<= 0: greedy), top_k (0: off),
// top_p (>= 1: off), and the Philox key / counter words of its random draw.
struct SampleParams {
  float temperature;
  int32_t top_k;
  float top_p;
  uint32_t key[2];
  uint32_t counter[3];
};

// Next token per row under its sampling parameters (see the kernel):
// tok -> slot_tok[out_slot[m]] (when out_slot) and tok_out[m].  Rows hold at
// most SAMPLE_MAX_V logits.
constexpr int SAMPLE_MAX_V = 1 << 21;
void launch_sample(const float *logits, int64_t ld, int M, int V, const SampleParams *prm, const int32_t *out_slot,
                   int32_t *slot_tok, int32_t *tok_out, hipStream_t s);

// Weight generator: writes rows x cols values of canonical tensor `tensor_id`
// to dst with row r stored at perm(r), in T, row-major or (`packed`) in the
// tiled weight layout of a cols-wide matrix.  `bf16_values`: round each value
// to bf16 first (a bf16 model held in fp16 storage keeps its exact values).
enum RowPerm : int { PERM_NONE = 0, PERM_ROPE = 1, PERM_GATE = 2, PERM_UP = 3 };
// packed: dst is the tiled matrix of fused_rows rows that holds this tensor's
// (permuted) rows from row0 on; otherwise dst is the tensor's row 0 of a
// row-major matrix.
template <typename T>
void launch_init_weight(T *dst, uint32_t k0, uint32_t k1, uint32_t tensor_id, int64_t rows,
                        int64_t cols, float stdv, int perm, int head_dim, bool bf16_values, bool packed,
                        int64_t row0, int64_t fused_rows, hipStream_t s);
void launch_fill_f32(float *dst, int64_t n, float v, hipStream_t s);

}  // namespace lp
