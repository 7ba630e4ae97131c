// The serving engine behind the C ABI: arena layout, weight loading, the KV
// block pool, prefill and decode steps, the real-time run loop and the
// per-request latency accounting.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

#include "../../include/lp.h"
#include "kernels.hpp"
#include "scheduler.hpp"


using namespace lp;

namespace {

constexpr int LOOKAHEAD = 2;           // steps the host may run ahead of the GPU
constexpr int RING = LOOKAHEAD + 2;    // event / staging ring depth
constexpr int64_t TOKLOG_CAP = 1 << 22;     // output tokens per run
constexpr int64_t POOL_CAP = 1 << 24;       // prompt + forced token ids
constexpr int64_t LOGITS_LOG_BYTES = 256ll << 20;

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
// A large pool sized from the arena holds a multiple of KV_NB_ROUND blocks, so
// that every layer's part of the K and V pools starts at the same (2 MiB)
// alignment.
constexpr int64_t KV_NB_ROUND = 16;
constexpr size_t KV_ALIGN = 2u << 20;  // offset alignment of the K pool and the workspace buffers in the arena

struct Layout {
  // weights
  size_t embed, lm_head, final_norm;
  std::vector<size_t> attn_norm, wqkv, wo, mlp_norm, wgu, wd;
  size_t weights_end;
  // KV
  size_t kcache, vcache;
  int64_t n_blocks;
  size_t kv_end;
  // workspace
  size_t x, xn, q, attn, h, logits, part, attn_ws, rope_cos, rope_sin, meta, slot_tok, tok_log,
      pool, logits_log;
  size_t part_bytes, meta_bytes, logits_log_bytes;
  size_t total;
};

// Activation / weight storage type of the GPU path.
enum ActType { ACT_F32 = 0, ACT_BF16 = 1, ACT_F16 = 2 };

struct Dims {
  int L, d, Hq, Hkv, hd, F, V, qkv_n;
  size_t esz;  // bytes per activation / weight element
  int act;     // ActType
};

Dims dims_of(const lp_model_config &c, uint32_t flags = 0) {
  Dims D;
  D.L = c.n_layers;
  D.d = c.d_model;
  D.Hq = c.n_heads;
  D.Hkv = c.n_kv_heads;
  D.hd = c.d_model / c.n_heads;
  D.F = c.ffn_dim;
  D.V = c.vocab;
  D.qkv_n = (D.Hq + 2 * D.Hkv) * D.hd;
  D.esz = c.dtype == LP_BF16 ? 2 : 4;
  // a bf16 model computes with fp16 MFMA inputs by default: the bf16 weight
  // values are held exactly and activations / KV entries round 8x finer
  D.act = c.dtype == LP_F32 ? ACT_F32 : ((flags & LP_FLAG_BF16_ACTIVATIONS) ? ACT_BF16 : ACT_F16);
  return D;
}

int64_t rows_cap(const lp_engine_options &o) { return std::max<int64_t>(o.max_batch, o.max_prefill_tokens); }

int decode_splits(int N, int K) {
  // K splits of the decode GEMMs whose epilogue can be deferred: at most
  // eight waves per CU (one 16-column slice per wave), with chunks of >= 512
  // k.  Measured at M = 64: QKV (384 slices) 5 splits 14.8 us against 6
  // splits 16.4 us, O and down (256 slices) best at 8.
  const int waves_per_split = std::max(1, N / 16);
  int s = std::max(1, 2048 / waves_per_split);
  s = std::min(s, std::max(1, K / 512));
  return lp::gemm_effective_splits(64, N, K, s);
}

// K splits of a GEMM over M rows whose epilogue can be deferred to a folding
// pass: decode-sized M by the weight shape, prefill-sized M by the tile grid.
int step_splits(int M, int N, int K) { return M <= 64 ? decode_splits(N, K) : lp::prefill_gemm_splits(M, N, K); }

size_t part_bytes_for(const Dims &D, const lp_model_config &c, const lp_engine_options &o) {
  if (c.dtype != LP_BF16) return 256;
  size_t m = 0;
  const int64_t Ns[3] = {D.qkv_n, D.d, D.d};
  const int64_t Ks[3] = {D.d, D.Hq * D.hd, D.F};
  const int64_t R = rows_cap(o);
  // every row count a step can have (the split plan is not monotone in M)
  for (int i = 0; i < 3; ++i)
    for (int64_t M = 1; M <= R; ++M)
      m = std::max(m, (size_t)step_splits((int)M, (int)Ns[i], (int)Ks[i]) * M * Ns[i] * sizeof(float));
  return m;
}

// Bytes of an [N x K] GEMM weight: the tiled layout for 16-bit models,
// row-major fp32 otherwise.
size_t wbytes(const Dims &D, int64_t N, int64_t K) {
  return D.esz == 2 ? (size_t)wpack_elems(N, K) * 2 : (size_t)N * K * D.esz;
}

// Lays out everything but the KV pool size, which is decided by the caller.
Layout plan_layout(const lp_model_config &c, const lp_engine_options &o, int64_t n_blocks) {
  const Dims D = dims_of(c);
  Layout Ly;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  // the norm gains first, then the matrices, each on a 2 MiB boundary (no
  // padding where the matrices' sizes are multiples of 2 MiB, as at every
  // 16-bit shape here)
  auto take_w = [&](size_t bytes) {
    off = (off + KV_ALIGN - 1) / KV_ALIGN * KV_ALIGN;
    return take(bytes);
  };
  for (int l = 0; l < D.L; ++l) {
    Ly.attn_norm.push_back(take((size_t)D.d * 4));
    Ly.mlp_norm.push_back(take((size_t)D.d * 4));
  }
  Ly.final_norm = take((size_t)D.d * 4);
  Ly.embed = take_w((size_t)D.V * D.d * D.esz);
  for (int l = 0; l < D.L; ++l) {
    Ly.wqkv.push_back(take_w(wbytes(D, D.qkv_n, D.d)));
    Ly.wo.push_back(take_w(wbytes(D, D.d, (int64_t)D.Hq * D.hd)));
    Ly.wgu.push_back(take_w(wbytes(D, 2 * (int64_t)D.F, D.d)));
    Ly.wd.push_back(take_w(wbytes(D, D.d, D.F)));
  }
  Ly.lm_head = take_w(wbytes(D, D.V, D.d));
  Ly.weights_end = off;
  // every workspace buffer starts on a 2 MiB boundary as well: its alignment
  // then does not depend on the sizes of the buffers before it
  auto take_al = [&](size_t bytes) {
    off = (off + KV_ALIGN - 1) / KV_ALIGN * KV_ALIGN;
    return take(bytes);
  };
  const int64_t R = rows_cap(o);
  const int max_pos = o.max_seq_len;
  Ly.x = take_al((size_t)R * D.d * 4);
  Ly.xn = take_al((size_t)R * D.d * D.esz);
  Ly.q = take_al((size_t)R * D.Hq * D.hd * D.esz);
  Ly.attn = take_al((size_t)R * D.Hq * D.hd * D.esz);
  Ly.h = take_al((size_t)R * D.F * D.esz);
  Ly.logits = take_al((size_t)o.max_batch * D.V * 4);
  Ly.part_bytes = part_bytes_for(D, c, o);
  Ly.part = take_al(Ly.part_bytes);
  Ly.attn_ws = take_al(decode_attention_ws_bytes(o.max_batch, D.Hq, D.hd, max_pos));
  Ly.rope_cos = take_al((size_t)max_pos * (D.hd / 2) * 4);
  Ly.rope_sin = take_al((size_t)max_pos * (D.hd / 2) * 4);
  const int max_blocks = (o.max_seq_len + KV_BLOCK - 1) / KV_BLOCK;
  // eight regions, each padded to 64 ints: row slot / position / token,
  // sequence starts / slots / LM rows, block table, sampling parameters
  Ly.meta_bytes =
      (size_t)(3 * R + 4 * (o.max_batch + 1) + (int64_t)o.max_batch * max_blocks + 8 * o.max_batch + 8 * 64) * 4;
  Ly.meta = take_al(Ly.meta_bytes);
  Ly.slot_tok = take((size_t)o.max_batch * 4);
  Ly.tok_log = take((size_t)TOKLOG_CAP * 4);
  Ly.pool = take((size_t)POOL_CAP * 4);
  Ly.logits_log_bytes = (o.flags & LP_FLAG_KEEP_LOGITS) ? LOGITS_LOG_BYTES : 0;
  Ly.logits_log = take_al(Ly.logits_log_bytes);
  Ly.n_blocks = n_blocks;
  const size_t kv_bytes = (size_t)D.L * n_blocks * D.Hkv * KV_BLOCK * D.hd * D.esz;
  // the K pool starts on a 2 MiB boundary of the arena, whatever the sizes
  // before it; the V pool follows it directly, so the arena grows by exactly
  // one block's bytes per block (and V is 2 MiB-aligned too whenever a
  // block's K bytes over all layers and heads are, as for every 16-bit shape)
  off = (off + KV_ALIGN - 1) / KV_ALIGN * KV_ALIGN;
  Ly.kcache = take(kv_bytes);
  Ly.vcache = take(kv_bytes);
  Ly.kv_end = off;
  Ly.total = off;
  return Ly;
}

size_t block_bytes(const lp_model_config &c) {
  const Dims D = dims_of(c);
  return (size_t)2 * D.L * D.Hkv * KV_BLOCK * D.hd * D.esz;
}

int check_config(const lp_model_config *c, const lp_engine_options *o, std::string &err) {
  if (!c || !o) return err = "null config", LP_EINVAL;
  if (c->n_layers < 1 || c->d_model < 64 || c->n_heads < 1 || c->n_kv_heads < 1 || c->ffn_dim < 8 ||
      c->vocab < 2)
    return err = "non-positive dimension", LP_EINVAL;
  if (c->d_model % c->n_heads || c->n_heads % c->n_kv_heads)
    return err = "d_model % n_heads or n_heads % n_kv_heads != 0", LP_EINVAL;
  const int hd = c->d_model / c->n_heads;
  if (hd != 64 && hd != 128) return err = "head_dim must be 64 or 128", LP_EINVAL;
  const int G = c->n_heads / c->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return err = "query heads per kv head must be 1, 2, 4 or 8", LP_EINVAL;
  if (c->d_model > 8192 || c->d_model % 8 || c->ffn_dim % 8 || c->vocab % 2 || c->vocab > SAMPLE_MAX_V)
    return err = "d_model <= 8192, d_model and ffn_dim multiples of 8, even vocab <= 2^21 required", LP_EINVAL;
  if (c->dtype != LP_F32 && c->dtype != LP_BF16) return err = "dtype", LP_EINVAL;
  if (c->dtype == LP_F32 && hd != 64) return err = "the fp32 path supports head_dim 64", LP_EINVAL;
  if (o->max_batch < 1 || o->max_batch > 64) return err = "max_batch must be 1..64", LP_EINVAL;
  if (o->max_seq_len < 2) return err = "max_seq_len", LP_EINVAL;
  if (o->max_prefill_tokens < 1) return err = "max_prefill_tokens", LP_EINVAL;
  if (o->max_batch_weight < 0 || o->hbm_reserve_bytes < 0) return err = "negative budget", LP_EINVAL;
  return LP_OK;
}

int64_t now_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(
             std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

}  // namespace

struct lp_engine {
  lp_model_config cfg;
  lp_engine_options opt;
  Dims D;
  Layout Ly;
  char *arena = nullptr;
  hipStream_t stream = nullptr;
  int64_t max_weight = 0;
  int max_blocks = 0;
  bool weights_ready = false;
  std::string err;

  // requests
  std::vector<SReq> reqs;
  std::unordered_map<int64_t, int32_t> by_id;
  std::vector<int64_t> prompt_off;   // into the device pool
  std::vector<int64_t> forced_off;   // -1: none
  std::vector<int32_t> forced_n;
  std::vector<SampleParams> sampling;  // per request (temperature 0: greedy)
  int64_t pool_used = 0;
  std::vector<int32_t> host_pool;

  // results of the last run
  std::vector<std::vector<int32_t>> out_tokens;
  std::vector<std::vector<int64_t>> out_times;
  std::vector<int64_t> out_arrival;
  std::vector<lp_step_record> steps;
  std::vector<int64_t> step_row_ids;
  std::vector<int32_t> step_row_slots;
  std::vector<int64_t> log_off_of_step;  // tok_log offset per step
  std::vector<std::vector<int64_t>> tok_log_index;  // per request: tok_log index per token
  lp_run_stats stats{};
  bool have_results = false;

  // run-time objects
  hipEvent_t ev_start = nullptr;
  hipEvent_t ev_step[RING] = {};
  std::vector<hipEvent_t> ev_kern;  // RING * L * 2 when timing
  int32_t *staging[RING] = {};
  size_t staging_bytes = 0;

  template <typename T>
  T *ptr(size_t off) const {
    return (T *)(arena + off);
  }
};

#define HIPCHK(e, call)                                                    \
  do {                                                                     \
    hipError_t _s = (call);                                                \
    if (_s != hipSuccess) {                                                \
      (e)->err = std::string(#call) + ": " + hipGetErrorString(_s);        \
      return LP_EHIP;                                                      \
    }                                                                      \
  } while (0)

static thread_local std::string g_err;
std::string &lp_global_error() { return g_err; }

extern "C" int lp_arena_bytes_required(const lp_model_config *cfg, const lp_engine_options *opt,
                                       size_t *out_bytes) {
  std::string err;
  int rc = check_config(cfg, opt, err);
  if (rc) return g_err = err, rc;
  const int64_t W = opt->max_batch_weight > 0 ? opt->max_batch_weight
                                              : (int64_t)opt->max_batch * opt->max_seq_len;
  const int64_t nb = (W + KV_BLOCK - 1) / KV_BLOCK + opt->max_batch;
  Layout Ly = plan_layout(*cfg, *opt, nb);
  *out_bytes = Ly.total + (size_t)opt->hbm_reserve_bytes + 4096;
  return LP_OK;
}

static int setup_rope(lp_engine *e) {
  const int half = e->D.hd / 2;
  const int P = e->opt.max_seq_len;
  std::vector<float> c((size_t)P * half), s((size_t)P * half);
  for (int p = 0; p < P; ++p)
    for (int i = 0; i < half; ++i) {
      const double theta = std::pow((double)e->cfg.rope_theta, -2.0 * i / e->D.hd);
      const double a = (double)p * theta;
      c[(size_t)p * half + i] = (float)std::cos(a);
      s[(size_t)p * half + i] = (float)std::sin(a);
    }
  HIPCHK(e, hipMemcpy(e->ptr<float>(e->Ly.rope_cos), c.data(), c.size() * 4, hipMemcpyHostToDevice));
  HIPCHK(e, hipMemcpy(e->ptr<float>(e->Ly.rope_sin), s.data(), s.size() * 4, hipMemcpyHostToDevice));
  return LP_OK;
}

extern "C" int lp_engine_create(const lp_model_config *cfg, const lp_engine_options *opt, void *arena,
                                size_t arena_bytes, void *hip_stream, lp_engine **out) {
  if (!out) return LP_EINVAL;
  *out = nullptr;
  std::string err;
  int rc = check_config(cfg, opt, err);
  if (rc) return g_err = err, rc;
  if (!arena || ((uintptr_t)arena & 255)) return g_err = "arena must be non-null and 256-byte aligned", LP_EINVAL;
  lp_engine *e = new lp_engine();
  e->cfg = *cfg;
  e->opt = *opt;
  e->D = dims_of(*cfg, opt->flags);
  e->arena = (char *)arena;
  e->stream = (hipStream_t)hip_stream;
  e->max_blocks = (opt->max_seq_len + KV_BLOCK - 1) / KV_BLOCK;
  const size_t usable = arena_bytes > (size_t)opt->hbm_reserve_bytes ? arena_bytes - opt->hbm_reserve_bytes : 0;
  const Layout base = plan_layout(*cfg, *opt, 0);
  int64_t nb;
  if (opt->max_batch_weight > 0) {
    nb = (opt->max_batch_weight + KV_BLOCK - 1) / KV_BLOCK + opt->max_batch;
    e->max_weight = opt->max_batch_weight;
  } else {
    nb = base.total < usable ? (int64_t)((usable - base.total - 1024) / (block_bytes(*cfg) + 1)) : 0;
    if (nb >= 64 * KV_NB_ROUND) nb = nb / KV_NB_ROUND * KV_NB_ROUND;  // large pools only: a small one keeps every block
    e->max_weight = (nb - opt->max_batch) * KV_BLOCK;
  }
  e->Ly = plan_layout(*cfg, *opt, nb);
  if (e->Ly.total > usable || e->max_weight < 2) {
    g_err = "arena of " + std::to_string(arena_bytes) + " bytes cannot hold weights + workspace + KV cache (" +
            std::to_string(e->Ly.total) + " bytes needed)";
    delete e;
    return LP_ENOMEM;
  }
  if (setup_rope(e)) {
    g_err = e->err;
    delete e;
    return LP_EHIP;
  }
  hipError_t s = hipEventCreate(&e->ev_start);
  for (int i = 0; i < RING && s == hipSuccess; ++i) s = hipEventCreate(&e->ev_step[i]);
  if (s == hipSuccess && (opt->flags & LP_FLAG_TIME_KERNEL)) {
    e->ev_kern.resize((size_t)RING * 2);
    for (auto &ev : e->ev_kern)
      if (s == hipSuccess) s = hipEventCreate(&ev);
  }
  e->staging_bytes = e->Ly.meta_bytes;
  for (int i = 0; i < RING && s == hipSuccess; ++i) s = hipHostMalloc((void **)&e->staging[i], e->staging_bytes, 0);
  if (s != hipSuccess) {
    g_err = std::string("engine setup: ") + hipGetErrorString(s);
    lp_engine_destroy(e);
    return LP_EHIP;
  }
  // slot tokens start at 0
  hipMemsetAsync(e->ptr<int32_t>(e->Ly.slot_tok), 0, opt->max_batch * 4, e->stream);
  hipStreamSynchronize(e->stream);
  *out = e;
  return LP_OK;
}

extern "C" void lp_engine_destroy(lp_engine *e) {
  if (!e) return;
  if (e->stream) hipStreamSynchronize(e->stream);
  if (e->ev_start) hipEventDestroy(e->ev_start);
  for (auto ev : e->ev_step)
    if (ev) hipEventDestroy(ev);
  for (auto ev : e->ev_kern)
    if (ev) hipEventDestroy(ev);
  for (auto p : e->staging)
    if (p) hipHostFree(p);
  delete e;
}

extern "C" const char *lp_last_error(const lp_engine *e) { return e ? e->err.c_str() : g_err.c_str(); }

extern "C" int lp_query_max_batch_weight(lp_engine *e, int64_t *out) {
  if (!e || !out) return LP_EINVAL;
  *out = e->max_weight;
  return LP_OK;
}

// ------------------------------------------------------------------ weights

namespace {

struct TensorDesc {
  int64_t rows, cols;
  bool gain;
};

// canonical order: embed, per layer 9 tensors, final_norm, lm_head
std::vector<TensorDesc> canonical(const Dims &D) {
  std::vector<TensorDesc> t;
  t.push_back({D.V, D.d, false});
  for (int l = 0; l < D.L; ++l) {
    t.push_back({1, D.d, true});
    t.push_back({(int64_t)D.Hq * D.hd, D.d, false});
    t.push_back({(int64_t)D.Hkv * D.hd, D.d, false});
    t.push_back({(int64_t)D.Hkv * D.hd, D.d, false});
    t.push_back({D.d, (int64_t)D.Hq * D.hd, false});
    t.push_back({1, D.d, true});
    t.push_back({D.F, D.d, false});
    t.push_back({D.F, D.d, false});
    t.push_back({D.d, D.F, false});
  }
  t.push_back({1, D.d, true});
  t.push_back({D.V, D.d, false});
  return t;
}

// Destination of canonical tensor i: row permutation, whether it is a norm
// gain (fp32), and whether it is stored in the tiled weight layout (every GEMM
// weight of a 16-bit model; the embedding table stays row-major for the row
// gather).  Row-major: `off` is the byte offset of the tensor's row 0.  Tiled:
// `off` is the byte offset of the whole fused matrix (fused_rows rows), whose
// rows from row0 on are this tensor's (q, k and v share one matrix).
struct Dest {
  size_t off;
  int perm;
  bool gain;
  bool packed;
  int64_t row0 = 0, fused_rows = 0;
};

Dest dest_of(const lp_engine *e, int i) {
  const Dims &D = e->D;
  const bool pk = D.esz == 2;
  if (i == 0) return {e->Ly.embed, PERM_NONE, false, false};
  const int last = 1 + 9 * D.L;
  if (i == last) return {e->Ly.final_norm, PERM_NONE, true, false};
  if (i == last + 1) return {e->Ly.lm_head, PERM_NONE, false, pk, 0, D.V};
  const int l = (i - 1) / 9, j = (i - 1) % 9;
  // q, k and v are rows [0, Hq hd), [Hq hd, (Hq + Hkv) hd) and the rest of
  // one fused matrix
  const int64_t qr = (int64_t)D.Hq * D.hd, kr = (int64_t)D.Hkv * D.hd;
  const size_t rowb = (size_t)D.d * D.esz;
  switch (j) {
    case 0: return {e->Ly.attn_norm[l], PERM_NONE, true, false};
    case 1: return {e->Ly.wqkv[l], PERM_ROPE, false, pk, 0, D.qkv_n};
    case 2: return {e->Ly.wqkv[l] + (pk ? 0 : qr * rowb), PERM_ROPE, false, pk, qr, D.qkv_n};
    case 3: return {e->Ly.wqkv[l] + (pk ? 0 : (qr + kr) * rowb), PERM_NONE, false, pk, qr + kr, D.qkv_n};
    case 4: return {e->Ly.wo[l], PERM_NONE, false, pk, 0, D.d};
    case 5: return {e->Ly.mlp_norm[l], PERM_NONE, true, false};
    case 6: return {e->Ly.wgu[l], PERM_GATE, false, pk, 0, 2 * (int64_t)D.F};
    case 7: return {e->Ly.wgu[l], PERM_UP, false, pk, 0, 2 * (int64_t)D.F};
    default: return {e->Ly.wd[l], PERM_NONE, false, pk, 0, D.d};
  }
}

// Host-side packing of a row-major rows x K matrix of 16-bit values into the
// tiled weight layout (K % 8 == 0; padding zeroed).
std::vector<uint16_t> pack_tiles(const uint16_t *src, int64_t rows, int64_t K) {
  const int64_t ns = wpack_ns(rows);
  std::vector<uint16_t> out((size_t)wpack_elems(rows, K), 0);
  for (int64_t n = 0; n < rows; ++n)
    for (int64_t k = 0; k < K; k += 8) memcpy(&out[(size_t)wpack_off(n, k, ns)], src + n * K + k, 16);
  return out;
}

int64_t perm_row(int perm, int64_t r, int hd) {
  switch (perm) {
    case PERM_ROPE: {
      const int64_t h = r / hd, i = r % hd;
      return h * hd + (i < hd / 2 ? 2 * i : 2 * (i - hd / 2) + 1);
    }
    case PERM_GATE: return 2 * r;
    case PERM_UP: return 2 * r + 1;
    default: return r;
  }
}

}  // namespace

extern "C" int lp_load_weights(lp_engine *e, const void *blob, size_t bytes) {
  if (!e || !blob) return LP_EINVAL;
  const Dims &D = e->D;
  auto ts = canonical(D);
  size_t need = 0;
  for (auto &t : ts) need += (size_t)t.rows * t.cols * D.esz;
  if (bytes != need) {
    e->err = "weight blob is " + std::to_string(bytes) + " bytes, expected " + std::to_string(need);
    return LP_EINVAL;
  }
  const char *src = (const char *)blob;
  std::vector<char> tmp;
  std::vector<char> conv;
  if (D.act == ACT_F16) {
    // bf16 bit patterns -> fp16 bit patterns, exactly or not at all
    const size_t n = bytes / 2;
    conv.resize(bytes);
    const uint16_t *b = (const uint16_t *)blob;
    uint16_t *h = (uint16_t *)conv.data();
    for (size_t i = 0; i < n; ++i) {
      uint32_t u = (uint32_t)b[i] << 16;
      float f;
      memcpy(&f, &u, 4);
      const _Float16 hv = (_Float16)f;
      if ((float)hv != f) {
        e->err = "a bf16 weight is not exactly representable in fp16; create the engine with "
                 "LP_FLAG_BF16_ACTIVATIONS";
        return LP_EINVAL;
      }
      memcpy(&h[i], &hv, 2);
    }
    src = conv.data();
  }
  for (int i = 0; i < (int)ts.size(); ++i) {
    const auto &t = ts[i];
    const Dest ds = dest_of(e, i);
    const size_t rowb = (size_t)t.cols * D.esz;
    if (ds.gain) {
      std::vector<float> g(t.cols);
      for (int64_t c = 0; c < t.cols; ++c) {
        if (D.act == ACT_F16) {
          _Float16 hv;
          memcpy(&hv, src + c * 2, 2);
          g[c] = (float)hv;
        } else if (D.esz == 2) {
          uint16_t b;
          memcpy(&b, src + c * 2, 2);
          uint32_t u = (uint32_t)b << 16;
          memcpy(&g[c], &u, 4);
        } else {
          memcpy(&g[c], src + c * 4, 4);
        }
      }
      HIPCHK(e, hipMemcpy(e->arena + ds.off, g.data(), t.cols * 4, hipMemcpyHostToDevice));
    } else if (ds.packed) {
      // assemble the destination rows (q/k rotary pairs adjacent; gate and
      // up, which follow each other in the blob, interleaved into rows 2f and
      // 2f + 1), then tile them
      if (ds.perm == PERM_UP) {  // written together with the gate rows
        src += rowb * t.rows;
        continue;
      }
      const int64_t out_rows = ds.perm == PERM_GATE ? 2 * t.rows : t.rows;
      tmp.assign(rowb * out_rows, 0);
      for (int64_t r = 0; r < t.rows; ++r) {
        memcpy(tmp.data() + perm_row(ds.perm, r, D.hd) * rowb, src + r * rowb, rowb);
        if (ds.perm == PERM_GATE)
          memcpy(tmp.data() + perm_row(PERM_UP, r, D.hd) * rowb, src + (t.rows + r) * rowb, rowb);
      }
      // the tensor's tiles of one K step are one run of its slices inside
      // the fused matrix's K step: one strided copy places them all
      const std::vector<uint16_t> pk = pack_tiles((const uint16_t *)tmp.data(), out_rows, t.cols);
      const int64_t ns = wpack_ns(out_rows), fused_ns = wpack_ns(ds.fused_rows);
      if (ds.row0 % WT_ROWS || (ds.row0 + out_rows < ds.fused_rows && out_rows % WT_ROWS) ||
          ds.row0 / WT_ROWS + ns > fused_ns) {
        e->err = "a fused weight piece does not start and end at whole 16-row slices";
        return LP_EINVAL;
      }
      const size_t tile_b = (size_t)WT_ELEMS * 2;
      HIPCHK(e, hipMemcpy2D(e->arena + ds.off + (size_t)(ds.row0 / WT_ROWS) * tile_b, fused_ns * tile_b,
                            pk.data(), ns * tile_b, ns * tile_b, wpack_kt(t.cols), hipMemcpyHostToDevice));
    } else if (ds.perm == PERM_NONE) {
      HIPCHK(e, hipMemcpy(e->arena + ds.off, src, rowb * t.rows, hipMemcpyHostToDevice));
    } else {
      // gate/up interleave into rows 2f / 2f+1 of the fused matrix; q/k rotary pairs adjacent
      const int64_t out_rows = (ds.perm == PERM_ROPE) ? t.rows : 2 * t.rows;
      tmp.assign(rowb * out_rows, 0);
      if (ds.perm != PERM_ROPE) {  // keep the rows the other half already wrote
        HIPCHK(e, hipMemcpy(tmp.data(), e->arena + ds.off, rowb * out_rows, hipMemcpyDeviceToHost));
      }
      for (int64_t r = 0; r < t.rows; ++r)
        memcpy(tmp.data() + perm_row(ds.perm, r, D.hd) * rowb, src + r * rowb, rowb);
      HIPCHK(e, hipMemcpy(e->arena + ds.off, tmp.data(), rowb * out_rows, hipMemcpyHostToDevice));
    }
    src += rowb * t.rows;
  }
  e->weights_ready = true;
  return LP_OK;
}

extern "C" int lp_init_weights_random(lp_engine *e, uint64_t seed, float stdv) {
  if (!e) return LP_EINVAL;
  const Dims &D = e->D;
  auto ts = canonical(D);
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  // tiles past a matrix's last column (K not a multiple of 32) must read as
  // zeros: the generator writes only the matrix's own elements
  if (D.esz == 2 && (D.d % WT_COLS || D.F % WT_COLS || (D.Hq * D.hd) % WT_COLS))
    HIPCHK(e, hipMemsetAsync(e->arena, 0, e->Ly.weights_end, e->stream));
  for (int i = 0; i < (int)ts.size(); ++i) {
    const auto &t = ts[i];
    const Dest ds = dest_of(e, i);
    if (ds.gain) {
      launch_fill_f32((float *)(e->arena + ds.off), t.cols, 1.0f, e->stream);
    } else if (D.act == ACT_F16) {
      launch_init_weight<f16_t>((f16_t *)(e->arena + ds.off), k0, k1, (uint32_t)i, t.rows, t.cols, stdv,
                                ds.perm, D.hd, true, ds.packed, ds.row0, ds.fused_rows, e->stream);
    } else if (D.act == ACT_BF16) {
      launch_init_weight<bf16_t>((bf16_t *)(e->arena + ds.off), k0, k1, (uint32_t)i, t.rows, t.cols, stdv,
                                 ds.perm, D.hd, false, ds.packed, ds.row0, ds.fused_rows, e->stream);
    } else {
      launch_init_weight<float>((float *)(e->arena + ds.off), k0, k1, (uint32_t)i, t.rows, t.cols, stdv,
                                ds.perm, D.hd, false, false, 0, 0, e->stream);
    }
  }
  HIPCHK(e, hipGetLastError());
  HIPCHK(e, hipStreamSynchronize(e->stream));
  e->weights_ready = true;
  return LP_OK;
}

// ------------------------------------------------------------------ requests

extern "C" int lp_submit(lp_engine *e, const lp_request *reqs, int32_t n) {
  if (!e || (n > 0 && !reqs) || n < 0) return LP_EINVAL;
  std::vector<SReq> rs;
  std::unordered_map<int64_t, int32_t> ids;
  std::vector<int32_t> pool;
  std::vector<int64_t> offs;
  int64_t total_out = 0;
  for (int i = 0; i < n; ++i) {
    const lp_request &q = reqs[i];
    if (q.in_len < 1 || q.out_len < 1 || !q.prompt) return e->err = "request lengths must be >= 1", LP_EINVAL;
    if ((int64_t)q.in_len + q.out_len > e->opt.max_seq_len)
      return e->err = "in_len + out_len exceeds max_seq_len", LP_EINVAL;
    if ((int64_t)q.in_len + q.out_len > e->max_weight)
      return e->err = "request exceeds the maximum batch weight", LP_EINVAL;
    if (q.in_len > e->opt.max_prefill_tokens) return e->err = "in_len exceeds max_prefill_tokens", LP_EINVAL;
    if (q.arrival_ns < 0) return e->err = "negative arrival", LP_EINVAL;
    if (!ids.emplace(q.id, i).second) return e->err = "duplicate request id", LP_EINVAL;
    for (int t = 0; t < q.in_len; ++t)
      if (q.prompt[t] < 0 || q.prompt[t] >= e->D.V) return e->err = "token id out of range", LP_EINVAL;
    SReq s;
    s.id = q.id;
    s.in_len = q.in_len;
    s.out_len = q.out_len;
    s.arrival_ns = q.arrival_ns;
    s.order = i;
    rs.push_back(s);
    offs.push_back((int64_t)pool.size());
    pool.insert(pool.end(), q.prompt, q.prompt + q.in_len);
    total_out += q.out_len;
  }
  if ((int64_t)pool.size() > POOL_CAP) return e->err = "too many prompt tokens in one submission", LP_EINVAL;
  if (total_out > TOKLOG_CAP) return e->err = "too many output tokens in one submission", LP_EINVAL;
  if (!pool.empty())
    HIPCHK(e, hipMemcpy(e->ptr<int32_t>(e->Ly.pool), pool.data(), pool.size() * 4, hipMemcpyHostToDevice));
  e->reqs.swap(rs);
  e->by_id.swap(ids);
  e->prompt_off.swap(offs);
  e->host_pool.swap(pool);
  e->pool_used = (int64_t)e->host_pool.size();
  e->forced_off.assign(n, -1);
  e->forced_n.assign(n, 0);
  e->sampling.assign(n, SampleParams{});
  e->have_results = false;
  return LP_OK;
}

extern "C" int lp_set_sampling(lp_engine *e, int64_t id, float temperature, int32_t top_k, float top_p,
                               uint64_t seed) {
  if (!e) return LP_EINVAL;
  auto it = e->by_id.find(id);
  if (it == e->by_id.end()) return e->err = "unknown request id", LP_EINVAL;
  if (!(temperature >= 0.f) || top_k < 0 || !(top_p >= 0.f)) return e->err = "sampling parameters", LP_EINVAL;
  SampleParams &sp = e->sampling[it->second];
  sp.temperature = temperature;
  sp.top_k = top_k;
  sp.top_p = top_p;
  sp.key[0] = (uint32_t)seed;
  sp.key[1] = (uint32_t)(seed >> 32);
  return LP_OK;
}

extern "C" int lp_set_forced_tokens(lp_engine *e, int64_t id, const int32_t *toks, int32_t n) {
  if (!e || (!toks && n > 0)) return LP_EINVAL;
  auto it = e->by_id.find(id);
  if (it == e->by_id.end()) return e->err = "unknown request id", LP_EINVAL;
  const SReq &q = e->reqs[it->second];
  if (n < 0 || n > q.out_len - 1) return e->err = "forced tokens must number 0..out_len-1", LP_EINVAL;
  for (int i = 0; i < n; ++i)
    if (toks[i] < 0 || toks[i] >= e->D.V) return e->err = "token id out of range", LP_EINVAL;
  if (e->pool_used + n > POOL_CAP) return e->err = "token pool full", LP_EINVAL;
  if (n > 0)
    HIPCHK(e, hipMemcpy(e->ptr<int32_t>(e->Ly.pool) + e->pool_used, toks, (size_t)n * 4, hipMemcpyHostToDevice));
  e->forced_off[it->second] = e->pool_used;
  e->forced_n[it->second] = n;
  e->pool_used += n;
  return LP_OK;
}

// ------------------------------------------------------------------ steps

namespace {

struct StepMeta {
  int32_t *row_slot, *row_pos, *row_tok, *seq_start, *seq_slot, *lm_rows, *block_table;
  const SampleParams *sample;  // per output row; null when every row is greedy
};

template <typename T>
KVCache kv_of(lp_engine *e, const int32_t *block_table) {
  KVCache kv;
  kv.k = e->arena + e->Ly.kcache;
  kv.v = e->arena + e->Ly.vcache;
  kv.block_table = block_table;
  kv.max_blocks = e->max_blocks;
  kv.n_blocks = e->Ly.n_blocks;
  kv.n_kv_heads = e->D.Hkv;
  kv.head_dim = e->D.hd;
  return kv;
}

// Runs every layer and the LM head over M rows already embedded into x.
// prefill: n_seq sequences described by seq_start/seq_slot, LM head over
// lm_rows; decode: rows attend to their slots' caches.
template <typename T>
int run_layers(lp_engine *e, bool prefill, int M, int n_out, int n_seq, int max_len, int attn_items,
               const StepMeta &dm, int64_t log_off, int64_t step) {
  const int step_ring = (int)(step % RING);
  // LP_FLAG_TIME_KERNEL: one layer's gate/up launch per decode step, rotating
  // over the layers, carries two events bound to its dispatch
  const int timed_layer = (int)(step % e->D.L);
  const Dims &D = e->D;
  hipStream_t st = e->stream;
  float *x = e->ptr<float>(e->Ly.x);
  T *xn = e->ptr<T>(e->Ly.xn);
  T *qb = e->ptr<T>(e->Ly.q);
  T *ab = e->ptr<T>(e->Ly.attn);
  T *hb = e->ptr<T>(e->Ly.h);
  float *part = e->ptr<float>(e->Ly.part);
  const bool bf = D.act != ACT_F32;
  const float eps = e->cfg.norm_eps;
  RowMeta rows{dm.row_slot, dm.row_pos};
  KVCache kv = kv_of<T>(e, dm.block_table);
  const int qd = D.Hq * D.hd;
  // split-K plan (16-bit paths only)
  const int s_qkv = bf ? step_splits(M, D.qkv_n, D.d) : 1;
  const int s_o = bf ? step_splits(M, D.d, qd) : 1;
  const int s_dn = bf ? step_splits(M, D.d, D.F) : 1;
  int pending_parts = 0;  // partials of the last residual GEMM not yet folded into x
  int64_t pending_stride = 0;
  for (int l = 0; l < D.L; ++l) {
    launch_rmsnorm<T>(x, part, pending_parts, pending_stride, nullptr, e->ptr<float>(e->Ly.attn_norm[l]), xn, M,
                      D.d, eps, st);
    pending_parts = 0;
    Epi eq{};
    eq.kind = EPI_QKV;
    eq.act_out = qb;
    eq.ld_act = qd;
    eq.rows = rows;
    eq.kv = kv;
    eq.layer = l;
    eq.n_heads = D.Hq;
    eq.rope_cos = e->ptr<float>(e->Ly.rope_cos);
    eq.rope_sin = e->ptr<float>(e->Ly.rope_sin);
    launch_gemm<T>(xn, D.d, e->ptr<T>(e->Ly.wqkv[l]), M, D.qkv_n, D.d, s_qkv, part, eq, st);
    // a decode step's split QKV projection is finished inside the attention
    // kernel (sum of partials, rotary embedding, KV append); prefill finishes
    // it in its own pass
    const bool fuse_qkv = !prefill && bf && s_qkv > 1 && !(e->opt.flags & LP_FLAG_SEPARATE_QKV_FINISH) &&
                          decode_attention_fuses_qkv(D.Hq / D.Hkv, D.hd, s_qkv);
    if (s_qkv > 1 && !fuse_qkv) launch_gemm_finish<T>(part, s_qkv, M, D.qkv_n, eq, st);
    if (prefill) {
      launch_prefill_attention<T>(qb, ab, dm.seq_start, dm.seq_slot, n_seq, max_len, kv, l, D.Hq, st);
    } else {
      const QkvParts qp{part, s_qkv, D.qkv_n, eq.rope_cos, eq.rope_sin};
      launch_decode_attention<T>(qb, ab, rows, kv, l, M, D.Hq, max_len, attn_items, e->ptr<float>(e->Ly.attn_ws),
                                 st, fuse_qkv ? &qp : nullptr);
    }
    Epi eo{};
    eo.kind = EPI_RESID;
    eo.out = x;
    eo.ldo = D.d;
    launch_gemm<T>(ab, qd, e->ptr<T>(e->Ly.wo[l]), M, D.d, qd, s_o, part, eo, st);
    if (s_o > 1) {
      pending_parts = s_o;
      pending_stride = (int64_t)M * D.d;
    }
    launch_rmsnorm<T>(x, part, pending_parts, pending_stride, nullptr, e->ptr<float>(e->Ly.mlp_norm[l]), xn, M,
                      D.d, eps, st);
    pending_parts = 0;
    Epi eg{};
    eg.kind = EPI_SILU;
    eg.act_out = hb;
    eg.ld_act = D.F;
    const hipEvent_t *tk = nullptr;
    if (!prefill && !e->ev_kern.empty() && l == timed_layer) tk = &e->ev_kern[(size_t)step_ring * 2];
    launch_gemm<T>(xn, D.d, e->ptr<T>(e->Ly.wgu[l]), M, 2 * D.F, D.d, 1, part, eg, st, tk);
    Epi ed{};
    ed.kind = EPI_RESID;
    ed.out = x;
    ed.ldo = D.d;
    launch_gemm<T>(hb, D.F, e->ptr<T>(e->Ly.wd[l]), M, D.d, D.F, s_dn, part, ed, st);
    if (s_dn > 1) {
      pending_parts = s_dn;
      pending_stride = (int64_t)M * D.d;
    }
  }
  // final norm over the rows that produce tokens, then LM head and argmax
  launch_rmsnorm<T>(x, part, pending_parts, pending_stride, prefill ? dm.lm_rows : nullptr,
                    e->ptr<float>(e->Ly.final_norm), xn, n_out, D.d, eps, st);
  float *logits = e->ptr<float>(e->Ly.logits);
  Epi el{};
  el.kind = EPI_LOGITS;
  el.out = logits;
  el.ldo = D.V;
  launch_gemm<T>(xn, D.d, e->ptr<T>(e->Ly.lm_head), n_out, D.V, D.d, 1, part, el, st);
  const int32_t *out_slot = prefill ? dm.seq_slot : dm.row_slot;
  if (dm.sample)
    launch_sample(logits, D.V, n_out, D.V, dm.sample, out_slot, e->ptr<int32_t>(e->Ly.slot_tok),
                  e->ptr<int32_t>(e->Ly.tok_log) + log_off, st);
  else
    launch_argmax(logits, D.V, n_out, D.V, out_slot, e->ptr<int32_t>(e->Ly.slot_tok),
                  e->ptr<int32_t>(e->Ly.tok_log) + log_off, st);
  if (e->Ly.logits_log_bytes) {
    const size_t row_bytes = (size_t)D.V * 4;
    const size_t cap_rows = e->Ly.logits_log_bytes / row_bytes;
    if ((size_t)log_off + n_out <= cap_rows)
      hipMemcpyAsync(e->arena + e->Ly.logits_log + (size_t)log_off * row_bytes, logits, (size_t)n_out * row_bytes,
                     hipMemcpyDeviceToDevice, st);
  }
  HIPCHK(e, hipGetLastError());
  return LP_OK;
}

}  // namespace

// Issues one planned step; returns its tok_log offset via log_off.
static int launch_step(lp_engine *e, const PlanStep &ps, int64_t step, int64_t log_off,
                       const std::vector<int32_t> &block_table_host) {
  const int ring = (int)(step % RING);
  const int M = ps.kind == 0 ? (int)ps.n_tokens : (int)ps.reqs.size();
  const int n_rows = (int)ps.reqs.size();
  int32_t *h = e->staging[ring];
  int32_t *d = e->ptr<int32_t>(e->Ly.meta);
  size_t o = 0;
  auto region = [&](size_t n) {
    const size_t at = o;
    o += (n + 63) & ~size_t(63);
    return at;
  };
  const size_t o_slot = region(M), o_pos = region(M), o_tok = region(M);
  const size_t o_ss = region(n_rows + 1), o_sq = region(n_rows), o_lm = region(n_rows);
  const size_t o_bt = region(block_table_host.size());
  const size_t o_smp = region((size_t)n_rows * (sizeof(SampleParams) / 4));
  if (o * 4 > e->staging_bytes) return e->err = "step metadata overflow", LP_EINVAL;
  // sampling parameters of the rows that emit a token; the draw's counter is
  // (request id, index of the output token being produced)
  bool any_sampling = false;
  SampleParams *hs = (SampleParams *)(h + o_smp);
  for (int j = 0; j < n_rows; ++j) {
    const int ri = ps.reqs[j];
    const SampleParams &sp = e->sampling[ri];
    const int64_t id = e->reqs[ri].id;
    const int k = ps.kind == 0 ? 0 : ps.pos[j] - e->reqs[ri].in_len + 1;
    hs[j] = sp;
    hs[j].counter[0] = (uint32_t)id;
    hs[j].counter[1] = (uint32_t)((uint64_t)id >> 32);
    hs[j].counter[2] = (uint32_t)k;
    any_sampling |= sp.temperature > 0.f && sp.top_p > 0.f;
  }
  int max_len = 0, attn_items = 0;
  if (ps.kind == 0) {
    int64_t row = 0;
    for (int j = 0; j < n_rows; ++j) {
      const int ri = ps.reqs[j];
      const SReq &q = e->reqs[ri];
      h[o_ss + j] = (int32_t)row;
      h[o_sq + j] = ps.slots[j];
      for (int p = 0; p < q.in_len; ++p, ++row) {
        h[o_slot + row] = ps.slots[j];
        h[o_pos + row] = p;
        h[o_tok + row] = (int32_t)(e->prompt_off[ri] + p);
      }
      h[o_lm + j] = (int32_t)(row - 1);
      max_len = std::max(max_len, q.in_len);
    }
    h[o_ss + n_rows] = (int32_t)row;
  } else {
    for (int j = 0; j < n_rows; ++j) {
      const int ri = ps.reqs[j];
      const SReq &q = e->reqs[ri];
      h[o_slot + j] = ps.slots[j];
      h[o_pos + j] = ps.pos[j];
      max_len = std::max(max_len, ps.pos[j] + 1);  // decode: the longest context
      attn_items += decode_attention_chunks(ps.pos[j] + 1);
      // the token fed at position pos is output token number pos - in_len
      const int k = ps.pos[j] - q.in_len;
      const bool forced = e->forced_off[ri] >= 0 && k < e->forced_n[ri];
      h[o_tok + j] = forced ? (int32_t)(e->forced_off[ri] + k) : -1;
    }
  }
  memcpy(h + o_bt, block_table_host.data(), block_table_host.size() * 4);
  HIPCHK(e, hipMemcpyAsync(d, h, o * 4, hipMemcpyHostToDevice, e->stream));
  StepMeta dm{d + o_slot, d + o_pos, d + o_tok, d + o_ss, d + o_sq, d + o_lm, d + o_bt,
              any_sampling ? (const SampleParams *)(d + o_smp) : nullptr};
  int rc;
  const bool pf = ps.kind == 0;
  int32_t *pool = e->ptr<int32_t>(e->Ly.pool), *stok = e->ptr<int32_t>(e->Ly.slot_tok);
  float *x = e->ptr<float>(e->Ly.x);
  switch (e->D.act) {
    case ACT_F16:
      launch_embed<f16_t>(e->ptr<f16_t>(e->Ly.embed), pool, dm.row_tok, dm.row_slot, stok, x, M, e->D.d, e->stream);
      rc = run_layers<f16_t>(e, pf, M, n_rows, n_rows, max_len, attn_items, dm, log_off, step);
      break;
    case ACT_BF16:
      launch_embed<bf16_t>(e->ptr<bf16_t>(e->Ly.embed), pool, dm.row_tok, dm.row_slot, stok, x, M, e->D.d,
                           e->stream);
      rc = run_layers<bf16_t>(e, pf, M, n_rows, n_rows, max_len, attn_items, dm, log_off, step);
      break;
    default:
      launch_embed<float>(e->ptr<float>(e->Ly.embed), pool, dm.row_tok, dm.row_slot, stok, x, M, e->D.d, e->stream);
      rc = run_layers<float>(e, pf, M, n_rows, n_rows, max_len, attn_items, dm, log_off, step);
  }
  if (rc) return rc;
  HIPCHK(e, hipEventRecord(e->ev_step[ring], e->stream));
  return LP_OK;
}

// ------------------------------------------------------------------ run loop

namespace {

struct RunState {
  std::vector<int64_t> end_ns;   // per step
  int64_t read = 0;              // steps whose end time is known
};

int read_step(lp_engine *e, RunState &rs, int64_t k) {
  const int ring = (int)(k % RING);
  HIPCHK(e, hipEventSynchronize(e->ev_step[ring]));
  float ms = 0.f;
  const hipEvent_t prev = k == 0 ? e->ev_start : e->ev_step[(k - 1) % RING];
  HIPCHK(e, hipEventElapsedTime(&ms, prev, e->ev_step[ring]));
  const int64_t base = k == 0 ? 0 : rs.end_ns[k - 1];
  rs.end_ns[k] = base + (int64_t)std::llround((double)ms * 1e6);
  if (!e->ev_kern.empty() && e->steps[k].kind == 1) {
    float km = 0.f;
    hipEvent_t *tk = &e->ev_kern[(size_t)ring * 2];
    if (hipEventElapsedTime(&km, tk[0], tk[1]) == hipSuccess) {
      e->stats.timed_kernel_ms += km;
      e->stats.timed_kernel_launches += 1;
      e->stats.timed_kernel_rows += e->steps[k].n_rows;
    }
  }
  rs.read = k + 1;
  return LP_OK;
}

}  // namespace

extern "C" int lp_run(lp_engine *e, int32_t mode, int32_t concurrency) {
  if (!e) return LP_EINVAL;
  if (!e->weights_ready) return e->err = "weights not loaded", LP_ESTATE;
  if (e->reqs.empty()) return e->err = "no requests submitted", LP_ESTATE;
  if (mode != LP_OPEN_LOOP && mode != LP_CLOSED_LOOP) return e->err = "mode", LP_EINVAL;
  if (mode == LP_CLOSED_LOOP && concurrency < 1) return e->err = "concurrency must be >= 1", LP_EINVAL;
  const bool closed = mode == LP_CLOSED_LOOP;
  Scheduler sched(e->reqs, e->opt.max_batch, e->max_weight, e->opt.max_prefill_tokens, closed, concurrency);
  e->steps.clear();
  e->step_row_ids.clear();
  e->step_row_slots.clear();
  e->log_off_of_step.clear();
  e->stats = lp_run_stats{};
  // KV block pool
  std::vector<int32_t> free_blocks;
  for (int64_t b = e->Ly.n_blocks - 1; b >= 0; --b) free_blocks.push_back((int32_t)b);
  std::vector<std::vector<int32_t>> slot_blocks(e->opt.max_batch);
  std::vector<int32_t> bt((size_t)e->opt.max_batch * e->max_blocks, 0);
  RunState rs;
  int64_t log_off = 0;
  HIPCHK(e, hipStreamSynchronize(e->stream));
  const int64_t t0 = now_ns();
  HIPCHK(e, hipEventRecord(e->ev_start, e->stream));
  std::vector<PlanStep> plan;
  while (!sched.finished()) {
    int64_t now = now_ns() - t0;
    if (!closed) {
      const int64_t wake = sched.idle_until(now);
      if (wake > 0) {
        std::this_thread::sleep_for(std::chrono::nanoseconds(wake - now));
        while ((now = now_ns() - t0) < wake) {
        }
      }
    }
    plan.clear();
    const size_t first_new = e->steps.size();
    sched.plan(now, (int64_t)first_new, plan);
    for (auto &ps : plan) {
      const int64_t k = (int64_t)e->steps.size();
      if (ps.kind == 0) {
        for (size_t j = 0; j < ps.reqs.size(); ++j) {
          const SReq &q = e->reqs[ps.reqs[j]];
          const int nb = (q.in_len + q.out_len + KV_BLOCK - 1) / KV_BLOCK;
          if ((int)free_blocks.size() < nb) return e->err = "KV block pool exhausted", LP_ENOMEM;
          auto &sb = slot_blocks[ps.slots[j]];
          sb.clear();
          for (int b = 0; b < nb; ++b) {
            sb.push_back(free_blocks.back());
            free_blocks.pop_back();
          }
          for (int b = 0; b < nb; ++b) bt[(size_t)ps.slots[j] * e->max_blocks + b] = sb[b];
        }
      }
      lp_step_record rec{};
      rec.kind = ps.kind;
      rec.n_rows = (int32_t)ps.reqs.size();
      rec.n_tokens = ps.n_tokens;
      rec.sum_ctx = ps.sum_ctx;
      rec.plan_ns = now;
      e->steps.push_back(rec);
      for (size_t j = 0; j < ps.reqs.size(); ++j) {
        e->step_row_ids.push_back(e->reqs[ps.reqs[j]].id);
        e->step_row_slots.push_back(ps.slots[j]);
      }
      e->log_off_of_step.push_back(log_off);
      rs.end_ns.push_back(0);
      if (k >= LOOKAHEAD) {
        int rc = read_step(e, rs, k - LOOKAHEAD);
        if (rc) return rc;
      }
      int rc = launch_step(e, ps, k, log_off, bt);
      if (rc) return rc;
      log_off += (int64_t)ps.reqs.size();
    }
    // return the KV blocks of requests that finished in this iteration (their
    // slots are not reused before the next plan, and stream order protects
    // the in-flight steps that still read them)
    for (int32_t s : sched.take_retired_slots()) {
      for (int32_t b : slot_blocks[s]) free_blocks.push_back(b);
      slot_blocks[s].clear();
    }
  }
  const int64_t n_steps = (int64_t)e->steps.size();
  for (int64_t k = rs.read; k < n_steps; ++k) {
    int rc = read_step(e, rs, k);
    if (rc) return rc;
  }
  // tokens and times per request
  std::vector<int32_t> toklog((size_t)log_off);
  if (log_off)
    HIPCHK(e, hipMemcpy(toklog.data(), e->ptr<int32_t>(e->Ly.tok_log), (size_t)log_off * 4, hipMemcpyDeviceToHost));
  const size_t n = e->reqs.size();
  e->out_tokens.assign(n, {});
  e->out_times.assign(n, {});
  e->out_arrival.assign(n, 0);
  e->tok_log_index.assign(n, {});
  std::vector<int64_t> row_of_step_start(n_steps + 1, 0);
  for (int64_t k = 0; k < n_steps; ++k) {
    e->steps[k].end_ns = rs.end_ns[k];
    row_of_step_start[k + 1] = row_of_step_start[k] + e->steps[k].n_rows;
  }
  std::vector<int32_t> seen(n, 0);
  for (int64_t k = 0; k < n_steps; ++k) {
    for (int64_t r = row_of_step_start[k]; r < row_of_step_start[k + 1]; ++r) {
      const int32_t ri = e->by_id[e->step_row_ids[r]];
      const int64_t li = e->log_off_of_step[k] + (r - row_of_step_start[k]);
      e->out_tokens[ri].push_back(toklog[li]);
      e->out_times[ri].push_back(rs.end_ns[k]);
      e->tok_log_index[ri].push_back(li);
    }
  }
  int64_t first_arrival = INT64_MAX, last_tok = 0;
  for (size_t i = 0; i < n; ++i) {
    const SReq &q = e->reqs[i];
    e->out_arrival[i] = closed ? (q.arrival_step < 0 ? 0 : rs.end_ns[q.arrival_step]) : q.arrival_ns;
    first_arrival = std::min(first_arrival, e->out_arrival[i]);
    if (!e->out_times[i].empty()) last_tok = std::max(last_tok, e->out_times[i].back());
    e->stats.output_tokens += (int64_t)e->out_tokens[i].size();
    e->stats.prompt_tokens += q.in_len;
  }
  e->stats.n_steps = n_steps;
  for (int64_t k = 0; k < n_steps; ++k) {
    const int64_t dur = rs.end_ns[k] - (k ? rs.end_ns[k - 1] : 0);
    if (e->steps[k].kind == 0) {
      e->stats.n_prefill_steps++;
    } else {
      e->stats.n_decode_steps++;
      e->stats.decode_ns += dur;
      e->stats.decode_tokens += e->steps[k].n_rows;
      if (e->steps[k].n_rows == e->opt.max_batch) {
        e->stats.full_decode_steps++;
        e->stats.full_decode_ns += dur;
        e->stats.full_decode_sum_ctx += e->steps[k].sum_ctx;
      }
    }
  }
  e->stats.wall_ns = last_tok - first_arrival;
  e->have_results = true;
  return LP_OK;
}

extern "C" int lp_get_result(lp_engine *e, int64_t id, int32_t *tokens, int64_t *ttft_ns, int64_t *itl_ns,
                             int64_t *e2e_ns, int64_t *arrival_ns) {
  if (!e) return LP_EINVAL;
  if (!e->have_results) return e->err = "no results", LP_ESTATE;
  auto it = e->by_id.find(id);
  if (it == e->by_id.end()) return e->err = "unknown request id", LP_EINVAL;
  const int i = it->second;
  const auto &tk = e->out_tokens[i];
  const auto &tt = e->out_times[i];
  if (tokens) memcpy(tokens, tk.data(), tk.size() * 4);
  const int64_t a = e->out_arrival[i];
  if (ttft_ns) *ttft_ns = tt.front() - a;
  if (itl_ns)
    for (size_t k = 0; k + 1 < tt.size(); ++k) itl_ns[k] = tt[k + 1] - tt[k];
  if (e2e_ns) *e2e_ns = tt.back() - a;
  if (arrival_ns) *arrival_ns = a;
  return LP_OK;
}

extern "C" int lp_get_token_times(lp_engine *e, int64_t id, int64_t *token_ns) {
  if (!e || !token_ns) return LP_EINVAL;
  if (!e->have_results) return e->err = "no results", LP_ESTATE;
  auto it = e->by_id.find(id);
  if (it == e->by_id.end()) return e->err = "unknown request id", LP_EINVAL;
  const auto &tt = e->out_times[it->second];
  memcpy(token_ns, tt.data(), tt.size() * 8);
  return LP_OK;
}

extern "C" int lp_get_latency_summary(lp_engine *e, lp_latency_summary *out) {
  if (!e || !out) return LP_EINVAL;
  if (!e->have_results) return e->err = "no results", LP_ESTATE;
  const int32_t n = (int32_t)e->reqs.size();
  std::vector<int64_t> arr(n), toks;
  std::vector<int32_t> in(n), outl(n);
  for (int32_t i = 0; i < n; ++i) {
    arr[i] = e->out_arrival[i];
    in[i] = e->reqs[i].in_len;
    outl[i] = e->reqs[i].out_len;
    toks.insert(toks.end(), e->out_times[i].begin(), e->out_times[i].end());
  }
  return lp_summarize_latencies(n, arr.data(), in.data(), outl.data(), toks.data(), out);
}

extern "C" int lp_get_run_stats(lp_engine *e, lp_run_stats *out) {
  if (!e || !out) return LP_EINVAL;
  *out = e->stats;
  return LP_OK;
}

extern "C" int lp_get_step_log(lp_engine *e, lp_step_record *out, int64_t cap, int64_t *n_out, int64_t *ids,
                               int32_t *slots, int64_t ids_cap) {
  if (!e || !n_out) return LP_EINVAL;
  *n_out = (int64_t)e->steps.size();
  if (out)
    for (int64_t k = 0; k < std::min<int64_t>(cap, *n_out); ++k) out[k] = e->steps[k];
  const int64_t nr = std::min<int64_t>(ids_cap, (int64_t)e->step_row_ids.size());
  if (ids)
    for (int64_t r = 0; r < nr; ++r) ids[r] = e->step_row_ids[r];
  if (slots)
    for (int64_t r = 0; r < nr; ++r) slots[r] = e->step_row_slots[r];
  return LP_OK;
}

extern "C" int lp_get_logits(lp_engine *e, int64_t id, int32_t k, float *logits) {
  if (!e || !logits) return LP_EINVAL;
  if (!(e->opt.flags & LP_FLAG_KEEP_LOGITS)) return e->err = "engine created without LP_FLAG_KEEP_LOGITS", LP_ESTATE;
  if (!e->have_results) return e->err = "no results", LP_ESTATE;
  auto it = e->by_id.find(id);
  if (it == e->by_id.end()) return e->err = "unknown request id", LP_EINVAL;
  const auto &idx = e->tok_log_index[it->second];
  if (k < 0 || k >= (int)idx.size()) return e->err = "token index out of range", LP_EINVAL;
  const size_t row_bytes = (size_t)e->D.V * 4;
  if ((size_t)(idx[k] + 1) * row_bytes > e->Ly.logits_log_bytes) return e->err = "logits not kept (log full)", LP_ENOMEM;
  HIPCHK(e, hipMemcpy(logits, e->arena + e->Ly.logits_log + (size_t)idx[k] * row_bytes, row_bytes,
                      hipMemcpyDeviceToHost));
  return LP_OK;
}

// ------------------------------------------------------------------ host simulation

extern "C" int lp_sched_simulate(const lp_request *reqs, int32_t n, int32_t max_batch, int64_t max_batch_weight,
                                 int64_t max_prefill_tokens, int32_t mode, int32_t concurrency, int64_t a_prefill,
                                 int64_t b_prefill, int64_t a_decode, int64_t b_decode, lp_step_record *steps,
                                 int64_t step_cap, int64_t *n_steps, int64_t *row_ids, int32_t *row_slots,
                                 int64_t row_cap, int64_t *token_ns, int64_t tok_cap, int64_t *arrival_ns) {
  if (!reqs || n < 1 || max_batch < 1 || !n_steps) return LP_EINVAL;
  const bool closed = mode == LP_CLOSED_LOOP;
  std::vector<SReq> rs(n);
  for (int i = 0; i < n; ++i) {
    rs[i].id = reqs[i].id;
    rs[i].in_len = reqs[i].in_len;
    rs[i].out_len = reqs[i].out_len;
    rs[i].arrival_ns = reqs[i].arrival_ns;
    rs[i].order = i;
    if (reqs[i].in_len < 1 || reqs[i].out_len < 1 || reqs[i].in_len + (int64_t)reqs[i].out_len > max_batch_weight ||
        reqs[i].in_len > max_prefill_tokens)
      return g_err = "a request can never be admitted", LP_EINVAL;
  }
  Scheduler sched(rs, max_batch, max_batch_weight, max_prefill_tokens, closed, concurrency);
  std::vector<PlanStep> plan;
  std::vector<int64_t> ends;
  int64_t now = 0, nrow = 0, k = 0;
  while (!sched.finished()) {
    if (!closed) {
      const int64_t wake = sched.idle_until(now);
      if (wake > 0) now = wake;
    }
    plan.clear();
    sched.plan(now, k, plan);
    const int64_t plan_t = now;
    for (auto &ps : plan) {
      const int64_t dur = ps.kind == 0 ? a_prefill + b_prefill * ps.n_tokens
                                       : a_decode + b_decode * (int64_t)ps.reqs.size();
      now += dur;
      ends.push_back(now);
      if (k < step_cap && steps) {
        lp_step_record r{};
        r.kind = ps.kind;
        r.n_rows = (int32_t)ps.reqs.size();
        r.n_tokens = ps.n_tokens;
        r.sum_ctx = ps.sum_ctx;
        r.plan_ns = plan_t;
        r.end_ns = now;
        steps[k] = r;
      }
      for (size_t j = 0; j < ps.reqs.size(); ++j, ++nrow) {
        if (nrow < row_cap) {
          if (row_ids) row_ids[nrow] = rs[ps.reqs[j]].id;
          if (row_slots) row_slots[nrow] = ps.slots[j];
        }
      }
      ++k;
    }
  }
  *n_steps = k;
  int64_t t = 0;
  for (int i = 0; i < n; ++i) {
    if (arrival_ns) arrival_ns[i] = closed ? (rs[i].arrival_step < 0 ? 0 : ends[rs[i].arrival_step]) : rs[i].arrival_ns;
    for (int64_t s : rs[i].tok_step) {
      if (token_ns && t < tok_cap) token_ns[t] = ends[s];
      ++t;
    }
  }
  return LP_OK;
}
