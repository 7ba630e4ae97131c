// Request model of the workload generator (LLM-Pilot Sec. III-B): every
// request parameter is binned into at most `max_bins` intervals holding about
// equal numbers of trace records (or one bin per value when it has fewer
// distinct values); the joint model is the sparse histogram of the
// multi-dimensional bins that records fall in; a sample picks a bin with
// probability proportional to its count and reports the centre of each
// parameter's interval.  Pure host code.
//
// Binning of one parameter with n records, sorted values v[0..n-1], k
// distinct values and B = max_bins:
//   k <= B: one bin per distinct value, its centre the value itself;
//   k >  B: bin j would start at sorted position c_j = ceil(j n / B)
//           (0-based) for j = 1..B-1, so that with distinct values bin sizes
//           differ by at most one; its lower edge is v[c_j]; equal
//           consecutive edges merge, as does an edge equal to v[0]; bin i
//           spans [e_i, e_{i+1}) with e_0 = v[0] and the last bin closed at
//           v[n-1]; its centre is (lower + upper) / 2.
//   A value falls in the bin whose lower edge is the largest edge <= value.
// Sampling with a uniform u in [0, 1): r = floor(u * N) (N records, r clamped
// to N - 1); the chosen bin is the first in lexicographic order of bin-index
// tuples whose cumulative count exceeds r.
#include <algorithm>
#include <cmath>
#include <map>
#include <vector>

#include "../../include/lp.h"

struct lp_wg_model {
  int32_t n_params = 0;
  int64_t n_records = 0;
  std::vector<std::vector<double>> edges;    // per parameter: lower edges, then the top value
  std::vector<std::vector<double>> centres;  // per parameter: bin centres
  std::vector<std::vector<int64_t>> marginal_cum;  // per parameter: cumulative record counts per bin
  std::vector<std::vector<int32_t>> keys;    // non-empty joint bins, lexicographic order
  std::vector<int64_t> cum;                  // cumulative counts over `keys`
};

namespace {

void bin_parameter(std::vector<double> v, int32_t max_bins, std::vector<double> &edges, std::vector<double> &centres) {
  std::sort(v.begin(), v.end());
  const int64_t n = (int64_t)v.size();
  std::vector<double> distinct;
  for (int64_t i = 0; i < n; ++i)
    if (i == 0 || v[i] != v[i - 1]) distinct.push_back(v[i]);
  edges.clear();
  centres.clear();
  if ((int64_t)distinct.size() <= max_bins) {
    for (double d : distinct) {
      edges.push_back(d);
      centres.push_back(d);
    }
    edges.push_back(distinct.back());
    return;
  }
  edges.push_back(v[0]);
  for (int32_t j = 1; j < max_bins; ++j) {
    const int64_t c = ((int64_t)j * n + max_bins - 1) / max_bins;  // ceil(j n / B)
    if (v[c] != edges.back()) edges.push_back(v[c]);
  }
  const size_t nb = edges.size();
  edges.push_back(v[n - 1]);
  for (size_t i = 0; i < nb; ++i) centres.push_back((edges[i] + edges[i + 1]) / 2.0);
}

// Index of the bin holding value x: the last lower edge <= x (values below the
// first edge go to bin 0, values above the top to the last bin).
int32_t bin_of(const std::vector<double> &edges, double x) {
  const int32_t nb = (int32_t)edges.size() - 1;
  const auto it = std::upper_bound(edges.begin(), edges.begin() + nb, x);
  const int32_t i = (int32_t)(it - edges.begin()) - 1;
  return std::min(std::max(i, 0), nb - 1);
}

int64_t draw(const std::vector<int64_t> &cum, int64_t total, double u) {
  int64_t r = (int64_t)std::floor(u * (double)total);
  r = std::min(std::max<int64_t>(r, 0), total - 1);
  return (int64_t)(std::upper_bound(cum.begin(), cum.end(), r) - cum.begin());
}

}  // namespace

extern "C" int lp_wg_fit(const double *records, int64_t n, int32_t n_params, int32_t max_bins, lp_wg_model **out) {
  if (!records || !out || n < 1 || n_params < 1 || max_bins < 1) return LP_EINVAL;
  for (int64_t i = 0; i < n * n_params; ++i)
    if (!std::isfinite(records[i])) return LP_EINVAL;
  lp_wg_model *m = new lp_wg_model();
  m->n_params = n_params;
  m->n_records = n;
  m->edges.resize(n_params);
  m->centres.resize(n_params);
  m->marginal_cum.resize(n_params);
  std::vector<std::vector<int32_t>> idx(n_params, std::vector<int32_t>(n));
  for (int32_t p = 0; p < n_params; ++p) {
    std::vector<double> v(n);
    for (int64_t i = 0; i < n; ++i) v[i] = records[i * n_params + p];
    bin_parameter(v, max_bins, m->edges[p], m->centres[p]);
    std::vector<int64_t> cnt(m->centres[p].size(), 0);
    for (int64_t i = 0; i < n; ++i) {
      idx[p][i] = bin_of(m->edges[p], v[i]);
      ++cnt[idx[p][i]];
    }
    int64_t c = 0;
    for (int64_t x : cnt) m->marginal_cum[p].push_back(c += x);
  }
  std::map<std::vector<int32_t>, int64_t> hist;  // ordered: lexicographic tuples
  std::vector<int32_t> key(n_params);
  for (int64_t i = 0; i < n; ++i) {
    for (int32_t p = 0; p < n_params; ++p) key[p] = idx[p][i];
    ++hist[key];
  }
  int64_t c = 0;
  for (const auto &kv : hist) {
    m->keys.push_back(kv.first);
    m->cum.push_back(c += kv.second);
  }
  *out = m;
  return LP_OK;
}

extern "C" int lp_wg_info(const lp_wg_model *m, int32_t param, int32_t *n_bins, int64_t *n_joint_bins) {
  if (!m || param < -1 || param >= m->n_params) return LP_EINVAL;
  if (n_bins) *n_bins = param < 0 ? 0 : (int32_t)m->centres[param].size();
  if (n_joint_bins) *n_joint_bins = (int64_t)m->keys.size();
  return LP_OK;
}

extern "C" int lp_wg_bins(const lp_wg_model *m, int32_t param, double *edges, double *centres, int64_t *counts) {
  if (!m || param < 0 || param >= m->n_params) return LP_EINVAL;
  const size_t nb = m->centres[param].size();
  if (edges) std::copy(m->edges[param].begin(), m->edges[param].end(), edges);
  if (centres) std::copy(m->centres[param].begin(), m->centres[param].end(), centres);
  if (counts)
    for (size_t i = 0; i < nb; ++i) counts[i] = m->marginal_cum[param][i] - (i ? m->marginal_cum[param][i - 1] : 0);
  return LP_OK;
}

extern "C" int lp_wg_sample(const lp_wg_model *m, const double *u, int64_t n, double *out, int64_t *joint_bin) {
  if (!m || (!u && n > 0) || (!out && n > 0) || n < 0) return LP_EINVAL;
  const int64_t total = m->cum.back();
  for (int64_t s = 0; s < n; ++s) {
    if (!(u[s] >= 0.0 && u[s] < 1.0)) return LP_EINVAL;
    const int64_t b = draw(m->cum, total, u[s]);
    for (int32_t p = 0; p < m->n_params; ++p) out[s * m->n_params + p] = m->centres[p][m->keys[b][p]];
    if (joint_bin) joint_bin[s] = b;
  }
  return LP_OK;
}

extern "C" int lp_wg_sample_independent(const lp_wg_model *m, const double *u, int64_t n, double *out) {
  if (!m || (!u && n > 0) || (!out && n > 0) || n < 0) return LP_EINVAL;
  for (int64_t s = 0; s < n; ++s)
    for (int32_t p = 0; p < m->n_params; ++p) {
      const double x = u[s * m->n_params + p];
      if (!(x >= 0.0 && x < 1.0)) return LP_EINVAL;
      const int64_t b = draw(m->marginal_cum[p], m->n_records, x);
      out[s * m->n_params + p] = m->centres[p][b];
    }
  return LP_OK;
}

extern "C" void lp_wg_free(lp_wg_model *m) { delete m; }
