// Load-test metrics over recorded token times (LLM-Pilot Sec. III-C-3): per
// request time to first token (from its arrival), normalised by its input
// length, the inter-token latencies pooled over all requests, end-to-end
// latency, and output-token throughput over the experiment.  Pure host code.
#include <algorithm>
#include <cmath>
#include <limits>
#include <vector>

#include "../../include/lp.h"

namespace {

// Median of v (sorted in place): the mean of the two middle values for an
// even count, NaN when empty.
template <typename V>
double median_of(std::vector<V> &v) {
  const size_t n = v.size();
  if (n == 0) return std::numeric_limits<double>::quiet_NaN();
  std::sort(v.begin(), v.end());
  if (n % 2) return (double)v[n / 2];
  if constexpr (std::is_integral<V>::value)
    return (double)(v[n / 2 - 1] + v[n / 2]) / 2.0;
  else
    return (v[n / 2 - 1] + v[n / 2]) / 2.0;
}

// p-th percentile by the nearest-rank rule on sorted v.
template <typename V>
double nearest_rank(const std::vector<V> &v, double p) {
  if (v.empty()) return std::numeric_limits<double>::quiet_NaN();
  const int64_t k = std::max<int64_t>(1, (int64_t)std::ceil(p / 100.0 * (double)v.size()));
  return (double)v[(size_t)std::min<int64_t>(k, (int64_t)v.size()) - 1];
}

}  // namespace

extern "C" int lp_summarize_latencies(int32_t n, const int64_t *arrival_ns, const int32_t *in_len,
                                      const int32_t *out_len, const int64_t *token_ns, lp_latency_summary *out) {
  if (n < 1 || !arrival_ns || !in_len || !out_len || !token_ns || !out) return LP_EINVAL;
  std::vector<int64_t> ttft, itl, e2e;
  std::vector<double> nttft;
  ttft.reserve(n);
  nttft.reserve(n);
  e2e.reserve(n);
  int64_t off = 0, tokens = 0;
  int64_t start = arrival_ns[0], end = std::numeric_limits<int64_t>::min();
  for (int32_t i = 0; i < n; ++i) {
    if (in_len[i] < 1 || out_len[i] < 1) return LP_EINVAL;
    const int64_t *t = token_ns + off;
    const int64_t first = t[0] - arrival_ns[i];
    ttft.push_back(first);
    nttft.push_back((double)first / (double)in_len[i]);
    for (int32_t k = 0; k + 1 < out_len[i]; ++k) itl.push_back(t[k + 1] - t[k]);
    e2e.push_back(t[out_len[i] - 1] - arrival_ns[i]);
    start = std::min(start, arrival_ns[i]);
    for (int32_t k = 0; k < out_len[i]; ++k) end = std::max(end, t[k]);
    off += out_len[i];
    tokens += out_len[i];
  }
  lp_latency_summary s{};
  s.n_requests = n;
  s.output_tokens = tokens;
  s.itl_count = (int64_t)itl.size();
  s.ttft_p50_ns = median_of(ttft);
  s.nttft_p50_ns = median_of(nttft);
  s.itl_p50_ns = median_of(itl);
  s.e2e_p50_ns = median_of(e2e);
  s.ttft_p90_ns = nearest_rank(ttft, 90.0);  // sorted by median_of
  s.itl_p90_ns = nearest_rank(itl, 90.0);
  s.itl_p99_ns = nearest_rank(itl, 99.0);
  s.throughput_tok_s = end > start ? (double)tokens / ((double)(end - start) * 1e-9)
                                   : std::numeric_limits<double>::infinity();
  *out = s;
  return LP_OK;
}
