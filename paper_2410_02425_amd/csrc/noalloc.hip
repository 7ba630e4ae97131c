// Decode attention for callers that cannot allocate device memory.
//
// The chunk partials that lp_op_decode_attention keeps in the caller's `ws`
// live here in a file-scope device array instead.  Host code never passes the
// array's name to a kernel (in host code it names a host-side stand-in, not
// device memory): on the first call on a device, with that device current,
// hipGetSymbolAddress gives the device's own copy of the array, and that
// address is what the kernels receive.  No call allocates or frees memory.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/lp_ops.h"
#include "kernels.hpp"

using namespace lp;

std::string &lp_global_error();

namespace {

constexpr size_t SCRATCH_BYTES = size_t(32) << 20;  // LP_NOALLOC_SCRATCH_BYTES
constexpr int MAX_DEVICES = 64;

__device__ __align__(256) char scratch[SCRATCH_BYTES];

std::mutex g_mu;
void *g_ptr[MAX_DEVICES] = {};

// The current device's copy of `scratch`, looked up once per device.
int scratch_ptr(void **out) {
  int dev = -1;
  hipError_t s = hipGetDevice(&dev);
  if (s != hipSuccess || dev < 0 || dev >= MAX_DEVICES) {
    lp_global_error() = std::string("no-alloc decode attention: device: ") +
                        (s != hipSuccess ? hipGetErrorString(s) : "index beyond 64");
    return LP_EHIP;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    s = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (s != hipSuccess || !p) {
      lp_global_error() = std::string("no-alloc decode attention: hipGetSymbolAddress: ") + hipGetErrorString(s);
      return LP_EHIP;
    }
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return LP_OK;
}

}  // namespace

static_assert(SCRATCH_BYTES == LP_NOALLOC_SCRATCH_BYTES, "scratch size in the header");

extern "C" int lp_op_decode_attention_noalloc(int32_t dtype, const void *q, void *out, const void *k_cache,
                                              const void *v_cache, const int32_t *block_table, int32_t max_blocks,
                                              int64_t n_blocks, const int32_t *row_slot, const int32_t *row_pos,
                                              int32_t M, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                              int32_t max_ctx, void *stream) {
  // sizes first: a call too large for the scratch array fails before any
  // device call
  if (M > 0 && max_ctx > 0 && n_heads > 0 && head_dim > 0 &&
      decode_attention_ws_bytes(M, n_heads, head_dim, max_ctx) > SCRATCH_BYTES) {
    lp_global_error() = "no-alloc decode attention: M * n_heads * ceil(max_ctx / 256) * (head_dim + 2) * 4 = " +
                        std::to_string(decode_attention_ws_bytes(M, n_heads, head_dim, max_ctx)) +
                        " bytes of partials exceed the " + std::to_string(SCRATCH_BYTES) + "-byte scratch array";
    return LP_EINVAL;
  }
  void *ws = nullptr;
  if (M > 0) {
    const int rc = scratch_ptr(&ws);
    if (rc) return rc;
  }
  // the allocating entry point's checks and launches, with the scratch array
  // as its workspace (every partial the combine pass reads is written first
  // by the same call, so nothing needs clearing)
  return lp_op_decode_attention(dtype, q, out, k_cache, v_cache, block_table, max_blocks, n_blocks, row_slot,
                                row_pos, M, n_heads, n_kv_heads, head_dim, max_ctx, ws, SCRATCH_BYTES, stream);
}
