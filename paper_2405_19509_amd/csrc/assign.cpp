// Host-side assignment tables (gc_assign), version and status strings.
//
// The assignment matrix A of Sec. 1 is described by its support plus the order
// in which each worker processes its chunks, i.e. the ordering matrix O of
// Sec. 3.  Everything downstream works from three dense tables derived from O:
// order (worker -> chunk by position), holder and hpos (chunk -> worker and
// the position of the chunk inside that worker).
#include <cstdint>
#include <vector>

#include "gcx.h"

extern "C" int gc_version(void) { return 100; }  // 0.1.0

extern "C" const char *gc_strerror(int status) {
  switch (status) {
    case GC_OK: return "ok";
    case GC_EINVAL: return "invalid argument";
    case GC_ELAUNCH: return "HIP launch or runtime error";
    case GC_ENOTSUP: return "device is not gfx950";
    default: return "unknown status";
  }
}

namespace {

int tables_from_order(int32_t N, int32_t m, const int32_t *O, int32_t delta, int32_t gamma,
                      int32_t *order, int32_t *holder, int32_t *hpos) {
  for (int64_t a = 0; a < int64_t(m) * delta; ++a) order[a] = -1;
  for (int64_t a = 0; a < int64_t(N) * gamma; ++a) holder[a] = hpos[a] = -1;
  // worker side: every column of O holds positions 1..delta_j exactly once
  for (int32_t j = 0; j < m; ++j) {
    int32_t load = 0;
    for (int32_t i = 0; i < N; ++i) {
      const int32_t o = O[int64_t(i) * m + j];
      if (o < 0) return GC_EINVAL;
      if (o == 0) continue;
      if (o > delta) return GC_EINVAL;
      int32_t &slot = order[int64_t(j) * delta + (o - 1)];
      if (slot != -1) return GC_EINVAL;  // two chunks at the same position
      slot = i;
      ++load;
    }
    for (int32_t t = 0; t < load; ++t)  // positions must be 1..load, no gaps
      if (order[int64_t(j) * delta + t] < 0) return GC_EINVAL;
  }
  // chunk side, holders in ascending worker order
  for (int32_t i = 0; i < N; ++i) {
    int32_t u = 0;
    for (int32_t j = 0; j < m; ++j) {
      const int32_t o = O[int64_t(i) * m + j];
      if (o == 0) continue;
      if (u >= gamma) return GC_EINVAL;
      holder[int64_t(i) * gamma + u] = j;
      hpos[int64_t(i) * gamma + u] = o - 1;
      ++u;
    }
  }
  return GC_OK;
}

}  // namespace

extern "C" int gc_assign(int32_t kind, int32_t N, int32_t m, int32_t s, int32_t *O, int32_t delta,
                         int32_t gamma, int32_t *order, int32_t *holder, int32_t *hpos) {
  if (!order || !holder || !hpos) return GC_EINVAL;
  if (N < 1 || m < 1 || delta < 1 || gamma < 1) return GC_EINVAL;
  if (kind == GC_ASSIGN_CYCLIC) {
    if (N != m || s < 0 || s >= m || delta != s + 1 || gamma != s + 1) return GC_EINVAL;
    std::vector<int32_t> cyc(size_t(N) * m, 0);
    for (int32_t j = 0; j < m; ++j)
      for (int32_t t = 0; t <= s; ++t) cyc[size_t((j + t) % N) * m + j] = t + 1;
    const int st = tables_from_order(N, m, cyc.data(), delta, gamma, order, holder, hpos);
    if (st == GC_OK && O)
      for (size_t a = 0; a < cyc.size(); ++a) O[a] = cyc[a];
    return st;
  }
  if (kind == GC_ASSIGN_ORDER) {
    if (!O) return GC_EINVAL;
    return tables_from_order(N, m, O, delta, gamma, order, holder, hpos);
  }
  return GC_EINVAL;
}
