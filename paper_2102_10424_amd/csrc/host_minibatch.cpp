// Cluster mini-batch CSR (Section 2.2; eq. (1); Appendix C.2), host side.
//
// The mini-batch is the subgraph induced by a union of clusters.  Rows are
// the selected nodes in ascending global id; a global edge is kept when both
// ends are selected; degrees are induced degrees.  Values are computed in
// double precision (exact integer products, correctly rounded sqrt and
// division) and rounded once to float, so the GCN and theory matrices come
// out bitwise symmetric.

#include <algorithm>
#include <cmath>
#include <vector>

#include "gist_internal.h"

namespace {

// Global -> local id map reused across calls on one thread: an entry is
// valid only if its stamp equals the current call's stamp, so the O(n)
// clear happens once per graph size rather than once per call.
struct LocalMap {
  std::vector<int32_t> local;
  std::vector<uint32_t> stamp;
  uint32_t cur = 0;
  void reset(int64_t n) {
    if (static_cast<int64_t>(local.size()) != n) {
      local.assign(static_cast<size_t>(n), 0);
      stamp.assign(static_cast<size_t>(n), 0);
      cur = 0;
    }
    if (++cur == 0) {  // wrapped: clear
      std::fill(stamp.begin(), stamp.end(), 0u);
      cur = 1;
    }
  }
  void set(int64_t g, int32_t l) { local[g] = l; stamp[g] = cur; }
  int32_t get(int64_t g) const { return stamp[g] == cur ? local[g] : -1; }
};

thread_local LocalMap t_map;

// Diagonal entry: the general formula with j = i (GCN), 1 for the theory form.
float self_value(gist_norm norm, double di) {
  if (norm == GIST_NORM_THEORY) return 1.0f;
  return static_cast<float>(1.0 / std::sqrt((di + 1.0) * (di + 1.0)));
}

}  // namespace

extern "C" gist_status gist_build_minibatch_csr(const gist_graph* g,
                                                const int32_t* clusters,
                                                int32_t n_clusters, gist_norm norm,
                                                gist_csr* out) {
  using gist::set_error;
  gist::clear_error();
  if (!g || !out) return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: NULL argument");
  if (norm != GIST_NORM_GCN_SYM && norm != GIST_NORM_SAGE_MEAN && norm != GIST_NORM_THEORY)
    return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: unknown norm");
  if (g->n < 0 || (g->n > 0 && (!g->rowptr || !g->col)))
    return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: bad graph arrays");
  const int64_t n = g->n;

  // 1. selected nodes, ascending
  std::vector<int32_t> nodes;
  if (n_clusters == -1) {
    if (n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "graph exceeds int32 ids");
    nodes.resize(static_cast<size_t>(n));
    for (int64_t i = 0; i < n; ++i) nodes[i] = static_cast<int32_t>(i);
  } else {
    if (n_clusters < 1 || !clusters)
      return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: empty cluster selection");
    if (!g->cluster_ptr || !g->cluster_nodes || g->n_clusters < 1)
      return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: graph has no clusters");
    std::vector<int32_t> sel(clusters, clusters + n_clusters);
    for (int32_t c : sel)
      if (c < 0 || c >= g->n_clusters)
        return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: cluster id out of range");
    std::sort(sel.begin(), sel.end());
    sel.erase(std::unique(sel.begin(), sel.end()), sel.end());
    for (int32_t c : sel)
      for (int64_t k = g->cluster_ptr[c]; k < g->cluster_ptr[c + 1]; ++k) {
        const int32_t v = g->cluster_nodes[k];
        if (v < 0 || v >= n)
          return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: cluster node out of range");
        nodes.push_back(v);
      }
    std::sort(nodes.begin(), nodes.end());
    nodes.erase(std::unique(nodes.begin(), nodes.end()), nodes.end());
  }
  const int64_t nb = static_cast<int64_t>(nodes.size());

  // 2. induced degrees
  LocalMap& map = t_map;
  map.reset(n);
  for (int64_t i = 0; i < nb; ++i) map.set(nodes[i], static_cast<int32_t>(i));
  std::vector<int32_t> deg(static_cast<size_t>(nb), 0);
  int64_t edges = 0;
  for (int64_t i = 0; i < nb; ++i) {
    const int64_t u = nodes[i];
    int32_t k = 0;
    for (int64_t e = g->rowptr[u]; e < g->rowptr[u + 1]; ++e) k += map.get(g->col[e]) >= 0;
    deg[i] = k;
    edges += k;
  }
  const bool loops = norm != GIST_NORM_SAGE_MEAN;
  const int64_t nnz = edges + (loops ? nb : 0);
  out->n = nb;
  out->nnz = nnz;
  if (nb > INT32_MAX - 1 || nnz > INT32_MAX)
    return set_error(GIST_E_UNSUPPORTED, "gist_build_minibatch_csr: mini-batch exceeds int32 CSR");
  if (!out->rowptr) return GIST_OK;  // size query
  const bool sage = norm == GIST_NORM_SAGE_MEAN;
  if (!out->col || !out->val || !out->node_map ||
      (sage && (!out->t_rowptr || !out->t_col || !out->t_val)))
    return set_error(GIST_E_INVAL, "gist_build_minibatch_csr: NULL output array");
  if (out->cap_n < nb || out->cap_nnz < nnz)
    return set_error(GIST_E_NOMEM, "gist_build_minibatch_csr: output capacity too small");

  // 3. rows, columns ascending (global columns ascend and local order is
  //    ascending global id, so induced columns come out ascending; the
  //    self-loop is inserted at its place)
  int32_t* rp = out->rowptr;
  int32_t* ci = out->col;
  float* vv = out->val;
  int64_t w = 0;
  rp[0] = 0;
  for (int64_t i = 0; i < nb; ++i) {
    const int64_t u = nodes[i];
    out->node_map[i] = nodes[i];
    bool placed = !loops;
    const double di = static_cast<double>(deg[i]);
    for (int64_t e = g->rowptr[u]; e < g->rowptr[u + 1]; ++e) {
      const int32_t j = map.get(g->col[e]);
      if (j < 0) continue;
      if (!placed && j > i) {
        ci[w] = static_cast<int32_t>(i);
        vv[w] = self_value(norm, di);
        ++w;
        placed = true;
      }
      const double dj = static_cast<double>(deg[j]);
      double v;
      if (norm == GIST_NORM_GCN_SYM) v = 1.0 / std::sqrt((di + 1.0) * (dj + 1.0));
      else if (norm == GIST_NORM_THEORY) v = 1.0 / std::sqrt(di * dj);
      else v = 1.0 / di;
      ci[w] = j;
      vv[w] = static_cast<float>(v);
      ++w;
    }
    if (!placed) {
      ci[w] = static_cast<int32_t>(i);
      vv[w] = self_value(norm, di);
      ++w;
    }
    rp[i + 1] = static_cast<int32_t>(w);
  }

  // 4. explicit transpose for the mean aggregator (counting sort by column;
  //    rows are visited in ascending order, so transposed columns ascend)
  if (sage) {
    int32_t* trp = out->t_rowptr;
    std::fill(trp, trp + nb + 1, 0);
    for (int64_t e = 0; e < nnz; ++e) ++trp[ci[e] + 1];
    for (int64_t i = 0; i < nb; ++i) trp[i + 1] += trp[i];
    std::vector<int32_t> fill(trp, trp + nb);
    for (int64_t i = 0; i < nb; ++i)
      for (int32_t e = rp[i]; e < rp[i + 1]; ++e) {
        const int32_t p = fill[ci[e]]++;
        out->t_col[p] = static_cast<int32_t>(i);
        out->t_val[p] = vv[e];
      }
  }
  return GIST_OK;
}
