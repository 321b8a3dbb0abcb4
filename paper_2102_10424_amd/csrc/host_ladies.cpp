// LADIES layer-sampled mini-batch (Section 5.4; Appendix A.6), host side.
//
// LADIES (Zou et al., NeurIPS 2019) samples the nodes of each GCN layer from
// the output layer down.  The importance of a node j for layer l is the
// squared norm of column j of the full matrix restricted to the rows V_{l+1}
// already kept; s nodes are drawn from that distribution, the kept set V_l
// adds them to V_{l+1}, and the layer's matrix keeps A_ij / (s p_j) on the
// kept columns, normalised to unit row sums.
//
// Every floating-point step is a single IEEE double operation in a fixed
// order (squares and sums in ascending row / column order, one division per
// probability and weight, one rounding to float), so the result does not
// depend on threads or vector width.  Only the columns the rows V_{l+1}
// touch are visited: the distribution is kept compact (touched columns in
// ascending order, read off a bitmap of the graph's nodes), which gives the
// same prefix sums as the full vector, since the untouched columns add
// exact zeros.  Membership in V_l is a second bitmap (a few tens of KB, so
// it stays in cache): the pass that builds the rows reads a node's
// importance and position only for the few entries that are kept.

#include <algorithm>
#include <cmath>
#include <cstring>
#include <iterator>
#include <vector>

#include "gist_internal.h"

namespace {

inline void set_bit(std::vector<uint64_t>& b, int32_t j) {
  b[static_cast<size_t>(j) >> 6] |= 1ull << (j & 63);
}
inline bool get_bit(const std::vector<uint64_t>& b, int32_t j) {
  return (b[static_cast<size_t>(j) >> 6] >> (j & 63)) & 1ull;
}

// Per-thread scratch, sized to the graph once.  Between calls q is zero and
// both bitmaps are clear.
struct Scratch {
  std::vector<double> q;         // importance per node (non-zero: touched this layer)
  std::vector<int32_t> pos;      // position in V_l, valid where `member` is set
  std::vector<uint64_t> seen;    // columns touched by the current layer's rows
  std::vector<uint64_t> member;  // V_l
  std::vector<int32_t> touched;  // columns with q > 0, ascending
  std::vector<double> prefix;    // running sums of q over `touched`
  void resize(int64_t n) {
    if (static_cast<int64_t>(q.size()) != n) {
      q.assign(static_cast<size_t>(n), 0.0);
      pos.assign(static_cast<size_t>(n), 0);
      seen.assign(static_cast<size_t>((n + 63) / 64), 0ull);
      member.assign(static_cast<size_t>((n + 63) / 64), 0ull);
    }
  }
};

thread_local Scratch t_scr;

// One sampled layer, built into vectors before the caller's buffers are checked.
struct Layer {
  std::vector<int32_t> nodes, rowptr, col, t_rowptr, t_col;
  std::vector<float> val, t_val;
};

}  // namespace

extern "C" gist_status gist_ladies_sample(const gist_csr* A, const int32_t* batch, int64_t b,
                                          int32_t L, int32_t s, uint64_t seed,
                                          gist_ladies_layer* layers) {
  using gist::set_error;
  gist::clear_error();
  if (!A || !layers || (b > 0 && !batch))
    return set_error(GIST_E_INVAL, "gist_ladies_sample: NULL argument");
  if (L < 1 || s < 0 || b < 0)
    return set_error(GIST_E_INVAL, "gist_ladies_sample: need L >= 1, s >= 0, b >= 0");
  const int64_t n = A->n;
  if (n < 0 || (n > 0 && (!A->rowptr || (A->nnz > 0 && (!A->col || !A->val)))))
    return set_error(GIST_E_INVAL, "gist_ladies_sample: bad matrix arrays");
  if (n > INT32_MAX) return set_error(GIST_E_UNSUPPORTED, "gist_ladies_sample: n exceeds int32");
  for (int64_t k = 0; k < b; ++k) {
    if (batch[k] < 0 || batch[k] >= n)
      return set_error(GIST_E_INVAL, "gist_ladies_sample: batch node out of range");
    if (k > 0 && batch[k] <= batch[k - 1])
      return set_error(GIST_E_INVAL, "gist_ladies_sample: batch not strictly ascending");
  }
  const int32_t* rp = A->rowptr;
  const int32_t* ac = A->col;
  const float* av = A->val;

  Scratch& S = t_scr;
  S.resize(n);
  gist::SplitMix64 rng(seed);
  const double s_eff = static_cast<double>(s > 0 ? s : 1);
  std::vector<Layer> out(static_cast<size_t>(L));
  std::vector<int32_t> V(batch, batch + b);   // V_{l+1} of the layer being sampled
  std::vector<int32_t> draws;
  for (int32_t l = L - 1; l >= 0; --l) {
    Layer& Y = out[static_cast<size_t>(l)];
    const int64_t n_out = static_cast<int64_t>(V.size());
    Y.rowptr.assign(static_cast<size_t>(n_out) + 1, 0);
    if (n_out == 0) {
      Y.t_rowptr.assign(1, 0);
      continue;
    }
    // importance of every column the rows V_{l+1} touch, rows in ascending
    // order; the next rows' entries and the importance slots a row is about
    // to update are prefetched (the rows lie anywhere in the graph)
    for (size_t r = 0; r < V.size(); ++r) {
      if (r + 2 < V.size()) {
        __builtin_prefetch(ac + rp[V[r + 2]]);
        __builtin_prefetch(av + rp[V[r + 2]]);
      }
      const int32_t i = V[r];
      const int32_t e0 = rp[i], e1 = rp[i + 1];
      for (int32_t e = e0; e < e1 && e < e0 + 8; ++e) __builtin_prefetch(&S.q[ac[e]], 1);
      for (int32_t e = e0; e < e1; ++e) {
        if (e + 8 < e1) __builtin_prefetch(&S.q[ac[e + 8]], 1);
        const int32_t j = ac[e];
        const double a = static_cast<double>(av[e]);
        S.q[j] += a * a;
        set_bit(S.seen, j);
      }
    }
    // touched columns in ascending order with their running sums (clearing the
    // bitmap); a column whose entries were all zero keeps q = 0, never drawn
    S.touched.clear();
    S.prefix.clear();
    double run = 0.0;
    for (size_t w = 0; w < S.seen.size(); ++w) {
      uint64_t x = S.seen[w];
      if (!x) continue;
      S.seen[w] = 0;
      while (x) {
        const int32_t j = static_cast<int32_t>(w * 64 + static_cast<size_t>(__builtin_ctzll(x)));
        x &= x - 1;
        const double qj = S.q[j];
        if (qj > 0.0) {
          S.touched.push_back(j);
          run += qj;
          S.prefix.push_back(run);
        }
      }
    }
    const double Q = run;
    draws.clear();
    if (s > 0 && S.touched.empty())   // every q is zero (and the bitmaps clear)
      return set_error(GIST_E_INVAL, "gist_ladies_sample: no node has positive importance");
    if (s > 0) {
      for (int32_t k = 0; k < s; ++k) {
        const double u = static_cast<double>(rng.next() >> 11) * 0x1.0p-53;
        const double t = u * Q;
        size_t idx = static_cast<size_t>(
            std::upper_bound(S.prefix.begin(), S.prefix.end(), t) - S.prefix.begin());
        if (idx == S.prefix.size()) idx = S.prefix.size() - 1;
        draws.push_back(S.touched[idx]);
      }
    }
    // V_l = distinct draws together with V_{l+1}
    std::sort(draws.begin(), draws.end());
    draws.erase(std::unique(draws.begin(), draws.end()), draws.end());
    Y.nodes.clear();
    std::set_union(draws.begin(), draws.end(), V.begin(), V.end(), std::back_inserter(Y.nodes));
    for (size_t k = 0; k < Y.nodes.size(); ++k) {
      S.pos[Y.nodes[k]] = static_cast<int32_t>(k);
      set_bit(S.member, Y.nodes[k]);
    }
    // rows: A_ij / (s p_j) over the kept columns, normalised by the row sum
    Y.col.clear();
    Y.val.clear();
    std::vector<double> w;
    for (int64_t r = 0; r < n_out; ++r) {
      if (r + 2 < n_out) {
        __builtin_prefetch(ac + rp[V[static_cast<size_t>(r) + 2]]);
        __builtin_prefetch(av + rp[V[static_cast<size_t>(r) + 2]]);
      }
      const int32_t i = V[static_cast<size_t>(r)];
      w.clear();
      for (int32_t e = rp[i]; e < rp[i + 1]; ++e) {
        const int32_t j = ac[e];
        if (!get_bit(S.member, j)) continue;
        const double p = S.q[j] / Q;
        w.push_back(static_cast<double>(av[e]) / (s_eff * p));
        Y.col.push_back(S.pos[j]);
      }
      double sum = 0.0;
      for (double x : w) sum += x;
      for (size_t k = 0; k < w.size(); ++k) Y.val.push_back(static_cast<float>(w[k] / sum));
      Y.rowptr[static_cast<size_t>(r) + 1] = static_cast<int32_t>(Y.col.size());
    }
    // transpose by counting sort (entries of a transposed row in ascending row)
    const int64_t n_in = static_cast<int64_t>(Y.nodes.size());
    const size_t nnz = Y.col.size();
    Y.t_rowptr.assign(static_cast<size_t>(n_in) + 1, 0);
    for (int32_t c : Y.col) ++Y.t_rowptr[static_cast<size_t>(c) + 1];
    for (int64_t k = 0; k < n_in; ++k) Y.t_rowptr[k + 1] += Y.t_rowptr[k];
    Y.t_col.resize(nnz);
    Y.t_val.resize(nnz);
    std::vector<int32_t> fill(Y.t_rowptr.begin(), Y.t_rowptr.end() - 1);
    for (int64_t r = 0; r < n_out; ++r) {
      for (int32_t e = Y.rowptr[r]; e < Y.rowptr[r + 1]; ++e) {
        const int32_t d = fill[Y.col[e]]++;
        Y.t_col[d] = static_cast<int32_t>(r);
        Y.t_val[d] = Y.val[e];
      }
    }
    for (int32_t j : S.touched) S.q[j] = 0.0;   // leave the scratch zeroed
    for (int32_t j : Y.nodes) S.member[static_cast<size_t>(j) >> 6] = 0;
    V = Y.nodes;
  }

  // report sizes, then copy into the caller's buffers if they fit
  bool query = true, fits = true;
  for (int32_t l = 0; l < L; ++l) {
    gist_ladies_layer& D = layers[l];
    const Layer& Y = out[static_cast<size_t>(l)];
    D.n_out = static_cast<int64_t>(Y.rowptr.size()) - 1;
    D.n_in = static_cast<int64_t>(Y.nodes.size());
    D.nnz = static_cast<int64_t>(Y.col.size());
    if (D.rowptr) query = false;
    if (D.n_in > D.cap_n || D.nnz > D.cap_nnz) fits = false;
  }
  if (query) return GIST_OK;
  if (!fits) return set_error(GIST_E_NOMEM, "gist_ladies_sample: layer capacity too small");
  for (int32_t l = 0; l < L; ++l) {
    const gist_ladies_layer& D = layers[l];
    if (!D.rowptr || !D.t_rowptr || (D.n_in > 0 && !D.nodes) ||
        (D.nnz > 0 && (!D.col || !D.val || !D.t_col || !D.t_val)))
      return set_error(GIST_E_INVAL, "gist_ladies_sample: NULL layer array");
  }
  for (int32_t l = 0; l < L; ++l) {
    gist_ladies_layer& D = layers[l];
    const Layer& Y = out[static_cast<size_t>(l)];
    auto put = [](auto* dst, const auto& v) {
      if (!v.empty()) std::memcpy(dst, v.data(), v.size() * sizeof(v[0]));
    };
    put(D.nodes, Y.nodes);
    put(D.rowptr, Y.rowptr);
    put(D.col, Y.col);
    put(D.val, Y.val);
    put(D.t_rowptr, Y.t_rowptr);
    put(D.t_col, Y.t_col);
    put(D.t_val, Y.t_val);
  }
  return GIST_OK;
}
