// subGCNs feature partition (Section 2.1, Algorithm 1), host side.
//
// A random disjoint partition of [0, d) into m equal blocks.  The random
// stream is SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) seeded with the
// caller's seed; a Fisher-Yates shuffle with rejection-sampled bounded draws
// orders the indices; block k takes shuffled positions [k d/m, (k+1) d/m)
// and sorts them.  The categorical flag instead assigns each index r
// (ascending) to a uniformly drawn block, as in the masks of Appendix C.1.

#include <algorithm>
#include <cstring>
#include <vector>

#include "gist_internal.h"

using gist::SplitMix64;

extern "C" gist_status gist_partition(int64_t d, int32_t m, uint64_t seed,
                                      uint32_t flags, int32_t* idx_out,
                                      int64_t* offs_out) {
  using gist::set_error;
  gist::clear_error();
  if (!idx_out || !offs_out) return set_error(GIST_E_INVAL, "gist_partition: NULL output");
  if (flags & ~GIST_PART_CATEGORICAL)
    return set_error(GIST_E_INVAL, "gist_partition: unknown flags");
  if (d < 1 || m < 1 || m > d)
    return set_error(GIST_E_INVAL, "gist_partition: need 1 <= m <= d");
  if (d > INT32_MAX) return set_error(GIST_E_INVAL, "gist_partition: d exceeds int32 indices");
  SplitMix64 rng(seed);
  if (flags & GIST_PART_CATEGORICAL) {
    std::vector<int32_t> owner(static_cast<size_t>(d));
    std::vector<int64_t> count(static_cast<size_t>(m) + 1, 0);
    for (int64_t r = 0; r < d; ++r) {
      owner[r] = static_cast<int32_t>(rng.below(static_cast<uint64_t>(m)));
      ++count[owner[r] + 1];
    }
    for (int32_t j = 0; j < m; ++j) count[j + 1] += count[j];
    std::memcpy(offs_out, count.data(), sizeof(int64_t) * (m + 1));
    for (int64_t r = 0; r < d; ++r) idx_out[count[owner[r]]++] = static_cast<int32_t>(r);
    return GIST_OK;
  }
  if (d % m) return set_error(GIST_E_INVAL, "gist_partition: m must divide d");
  std::vector<int32_t> p(static_cast<size_t>(d));
  for (int64_t i = 0; i < d; ++i) p[i] = static_cast<int32_t>(i);
  for (int64_t i = d - 1; i >= 1; --i) {
    const uint64_t j = rng.below(static_cast<uint64_t>(i) + 1);
    std::swap(p[i], p[j]);
  }
  const int64_t s = d / m;
  for (int32_t k = 0; k <= m; ++k) offs_out[k] = k * s;
  for (int32_t k = 0; k < m; ++k) std::sort(p.begin() + k * s, p.begin() + (k + 1) * s);
  std::memcpy(idx_out, p.data(), sizeof(int32_t) * d);
  return GIST_OK;
}

extern "C" gist_status gist_partition_inverse(int64_t d, int32_t m, const int32_t* idx,
                                              const int64_t* offs, int32_t* rank_out) {
  using gist::set_error;
  gist::clear_error();
  if (!idx || !offs || !rank_out)
    return set_error(GIST_E_INVAL, "gist_partition_inverse: NULL pointer");
  if (d < 1 || m < 1 || d > INT32_MAX)
    return set_error(GIST_E_INVAL, "gist_partition_inverse: bad sizes");
  if (offs[0] != 0 || offs[m] != d)
    return set_error(GIST_E_INVAL, "gist_partition_inverse: offsets do not cover [0, d)");
  for (int32_t b = 0; b < m; ++b)
    if (offs[b + 1] < offs[b])
      return set_error(GIST_E_INVAL, "gist_partition_inverse: offsets not ascending");
  std::vector<char> seen(static_cast<size_t>(d), 0);
  for (int64_t k = 0; k < d; ++k) {
    const int32_t r = idx[k];
    if (r < 0 || r >= d || seen[r])
      return set_error(GIST_E_INVAL, "gist_partition_inverse: index out of range or repeated");
    seen[r] = 1;
    rank_out[r] = static_cast<int32_t>(k);
  }
  return GIST_OK;
}
