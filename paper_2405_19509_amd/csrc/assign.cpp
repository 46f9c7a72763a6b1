// Host-side assignment tables (gc_assign), version and status strings.
//
// The assignment matrix A of Sec. 1 is described by its support plus the order
// in which each worker processes its chunks, i.e. the ordering matrix O of
// Sec. 3.  Everything downstream works from three dense tables derived from O:
// order (worker -> chunk by position), holder and hpos (chunk -> worker and
// the position of the chunk inside that worker).
#include <cstdint>
#include <queue>
#include <vector>

#include "gcx.h"

extern "C" int gc_version(void) { return 100; }  // 0.1.0

extern "C" const char *gc_strerror(int status) {
  switch (status) {
    case GC_OK: return "ok";
    case GC_EINVAL: return "invalid argument";
    case GC_ELAUNCH: return "HIP launch or runtime error";
    case GC_ENOTSUP: return "device is not gfx950";
    case GC_ESCRATCH: return "request exceeds the fixed scratch array of the no-allocation call";
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

// Maximum bipartite matching by Hopcroft-Karp: chunks on the left, workers on the
// right, adj[i] the workers still available to chunk i.  Returns the matching size
// and fills match_l (chunk -> worker) and match_r (worker -> chunk).
int hopcroft_karp(const std::vector<std::vector<int32_t>> &adj, int32_t m,
                  std::vector<int32_t> &match_l, std::vector<int32_t> &match_r) {
  const int32_t N = int32_t(adj.size());
  const int32_t INF = 1 << 30;
  match_l.assign(N, -1);
  match_r.assign(m, -1);
  std::vector<int32_t> dist(N), it(N), stack;
  int size = 0;
  for (;;) {
    // BFS layers from the free chunks
    std::queue<int32_t> q;
    for (int32_t i = 0; i < N; ++i) {
      dist[i] = match_l[i] < 0 ? 0 : INF;
      if (match_l[i] < 0) q.push(i);
    }
    bool found = false;
    while (!q.empty()) {
      const int32_t i = q.front();
      q.pop();
      for (int32_t j : adj[i]) {
        const int32_t k = match_r[j];
        if (k < 0) {
          found = true;
        } else if (dist[k] == INF) {
          dist[k] = dist[i] + 1;
          q.push(k);
        }
      }
    }
    if (!found) break;
    // vertex-disjoint shortest augmenting paths, iterative DFS
    for (int32_t i = 0; i < N; ++i) it[i] = 0;
    for (int32_t root = 0; root < N; ++root) {
      if (match_l[root] >= 0) continue;
      stack.assign(1, root);
      while (!stack.empty()) {
        const int32_t i = stack.back();
        if (it[i] >= int32_t(adj[i].size())) {
          dist[i] = INF;  // dead end
          stack.pop_back();
          continue;
        }
        const int32_t j = adj[i][it[i]++];
        const int32_t k = match_r[j];
        if (k < 0) {
          // augment along the stack: each chunk on it takes the worker it last tried
          for (int32_t a = int32_t(stack.size()) - 1; a >= 0; --a) {
            const int32_t u = stack[a];
            const int32_t w = adj[u][it[u] - 1];
            match_l[u] = w;
            match_r[w] = u;
          }
          ++size;
          stack.clear();
        } else if (dist[k] == dist[i] + 1) {
          stack.push_back(k);
        }
      }
    }
  }
  return size;
}

// Algorithm 2 (Chunk-Ordering, Sec. 3): peel delta perfect matchings P_1..P_delta
// off a delta-regular support and set O = sum_i i P_i.  Claim 1 guarantees each
// perfect matching exists.  O is overwritten with the ordering.
int regular_ordering(int32_t N, int32_t m, int32_t delta, int32_t *O) {
  if (N != m) return GC_EINVAL;
  std::vector<std::vector<int32_t>> adj(N);
  std::vector<int32_t> coldeg(m, 0);
  for (int32_t i = 0; i < N; ++i) {
    for (int32_t j = 0; j < m; ++j)
      if (O[int64_t(i) * m + j] != 0) {
        adj[i].push_back(j);
        ++coldeg[j];
      }
    if (int32_t(adj[i].size()) != delta) return GC_EINVAL;
  }
  for (int32_t j = 0; j < m; ++j)
    if (coldeg[j] != delta) return GC_EINVAL;
  std::vector<int32_t> out(size_t(N) * m, 0), ml, mr;
  for (int32_t step = 1; step <= delta; ++step) {
    if (hopcroft_karp(adj, m, ml, mr) != N) return GC_EINVAL;  // cannot happen for a regular support
    for (int32_t i = 0; i < N; ++i) {
      out[size_t(i) * m + ml[i]] = step;
      auto &a = adj[i];
      for (size_t u = 0; u < a.size(); ++u)
        if (a[u] == ml[i]) {
          a.erase(a.begin() + long(u));
          break;
        }
    }
  }
  for (size_t a = 0; a < out.size(); ++a) O[a] = out[a];
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
  if (kind == GC_ASSIGN_REGULAR) {
    if (!O || delta != gamma) return GC_EINVAL;
    std::vector<int32_t> work(O, O + size_t(N) * m);
    const int st = regular_ordering(N, m, delta, work.data());
    if (st != GC_OK) return st;
    const int st2 = tables_from_order(N, m, work.data(), delta, gamma, order, holder, hpos);
    if (st2 == GC_OK)
      for (size_t a = 0; a < work.size(); ++a) O[a] = work[a];
    return st2;
  }
  return GC_EINVAL;
}

// Q_i(O) (Sec. 3): the most chunks the cluster can process while no copy of D_i has been
// processed -- every holder j of D_i stops just before it (O_ij - 1 chunks), every other
// worker processes all of its delta_j chunks.  With N = m and every load and replication
// equal to delta this is the paper's sum_j O_ij + (m - delta - 1) delta over the holders.
extern "C" int gc_qmax(const int32_t *O, int32_t N, int32_t m, int64_t *Q, int64_t *qmax) {
  if (N < 1 || m < 1 || m > GC_MAX_M || !O || !qmax) return GC_EINVAL;
  std::vector<int64_t> load(m, 0);
  std::vector<std::vector<char>> seen(m);
  for (int32_t j = 0; j < m; ++j) {
    for (int32_t i = 0; i < N; ++i) {
      const int32_t o = O[int64_t(i) * m + j];
      if (o < 0 || o > N) return GC_EINVAL;
      if (o > 0) ++load[j];
    }
    // the positions of a worker are 1..delta_j, once each
    seen[j].assign(size_t(load[j]) + 1, 0);
    for (int32_t i = 0; i < N; ++i) {
      const int32_t o = O[int64_t(i) * m + j];
      if (o == 0) continue;
      if (o > load[j] || seen[j][o]) return GC_EINVAL;
      seen[j][o] = 1;
    }
  }
  int64_t total = 0;
  for (int32_t j = 0; j < m; ++j) total += load[j];
  int64_t best = -1;
  for (int32_t i = 0; i < N; ++i) {
    int64_t q = total;  // everyone finishes ...
    for (int32_t j = 0; j < m; ++j) {
      const int32_t o = O[int64_t(i) * m + j];
      if (o > 0) q -= load[j] - (o - 1);  // ... except the holders of D_i, who stop before it
    }
    if (Q) Q[i] = q;
    if (q > best) best = q;
  }
  *qmax = best;
  return GC_OK;
}
