// The paper's straggler simulation (Sec. 4) on the GPU: worker progress at a
// grid of deadlines, and exact-GC completion times for the proposed protocol and
// for original GC.  Worker j processes the chunks of its order one after the
// other; the chunk at position t is finished at sum_{u <= t} tau[r][j][u]; a
// failed worker finishes nothing.  All times are fp64 and summed in position
// order, so every comparison with a deadline is reproducible bit for bit.
#include "common.h"

namespace gcx {
namespace {

constexpr int kSimThreads = 256;
constexpr int kSimWaves = kSimThreads / kWave;

// psi[r][g][j] = #{t : sum_{u <= t} tau[r][j][u] <= T[g]}, 0 for failed workers.
__global__ __launch_bounds__(kSimThreads) void progress_kernel(const double *__restrict__ tau,
                                                               const uint8_t *__restrict__ failed,
                                                               int64_t R, int m, int delta,
                                                               const double *__restrict__ T, int G,
                                                               int32_t *__restrict__ psi) {
  const int64_t e = int64_t(blockIdx.x) * kSimThreads + threadIdx.x;  // (r, j)
  if (e >= R * m) return;
  const int64_t r = e / m;
  const int j = int(e % m);
  const double *tj = tau + e * delta;
  const bool dead = failed != nullptr && failed[e] != 0;
  for (int g = 0; g < G; ++g) {
    int cnt = 0;
    if (!dead) {
      double c = 0.0;
      for (int t = 0; t < delta; ++t) {
        c += tj[t];
        cnt += c <= T[g] ? 1 : 0;
      }
    }
    psi[(r * G + g) * m + j] = cnt;
  }
}

// The ell-th smallest of a stream of values, kept as a sorted prefix of ELLMAX.
template <int ELLMAX>
struct Smallest {
  double v[ELLMAX];
  __device__ void init() {
#pragma unroll
    for (int a = 0; a < ELLMAX; ++a) v[a] = INFINITY;
  }
  __device__ void push(double x) {
#pragma unroll
    for (int a = 0; a < ELLMAX; ++a) {
      const double lo = fmin(v[a], x), hi = fmax(v[a], x);
      v[a] = lo;
      x = hi;
    }
  }
};

// One wavefront per trial, one lane per chunk.  Chunk i reaches ell processed
// copies at the ell-th smallest finish time over its holders; the protocol can
// decode once every chunk has (the proposed protocol), and original GC once
// every chunk has ell holders that finished *all* their chunks.
__global__ __launch_bounds__(kSimThreads) void completion_kernel(
    const double *__restrict__ tau, const uint8_t *__restrict__ failed, int64_t R, int N, int m,
    int delta, const int32_t *__restrict__ holder, const int32_t *__restrict__ hpos, int gamma,
    int ell, double *__restrict__ partial, double *__restrict__ original) {
  const int lane = threadIdx.x % kWave;
  const int64_t r = int64_t(blockIdx.x) * kSimWaves + threadIdx.x / kWave;
  if (r >= R) return;
  const double *tr = tau + r * int64_t(m) * delta;
  double worst_p = 0.0, worst_o = 0.0;
  for (int i = lane; i < N; i += kWave) {
    Smallest<GC_MAX_ELL> sp, so;
    sp.init();
    so.init();
    for (int u = 0; u < gamma; ++u) {
      const int j = holder[int64_t(i) * gamma + u], t = hpos[int64_t(i) * gamma + u];
      if (j < 0 || j >= m || t < 0 || t >= delta) continue;
      if (failed != nullptr && failed[r * m + j] != 0) continue;
      const double *tj = tr + int64_t(j) * delta;
      double c = 0.0, at = 0.0;
      for (int v = 0; v < delta; ++v) {
        c += tj[v];
        if (v == t) at = c;
      }
      sp.push(at);
      so.push(c);
    }
    double fp = INFINITY, fo = INFINITY;
#pragma unroll
    for (int a = 0; a < GC_MAX_ELL; ++a)
      if (a == ell - 1) {
        fp = sp.v[a];
        fo = so.v[a];
      }
    worst_p = fmax(worst_p, fp);
    worst_o = fmax(worst_o, fo);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    worst_p = fmax(worst_p, __shfl_xor(worst_p, off, kWave));
    worst_o = fmax(worst_o, __shfl_xor(worst_o, off, kWave));
  }
  if (lane == 0) {
    partial[r] = worst_p;
    original[r] = worst_o;
  }
}


constexpr int kLsThreads = 256;

__device__ __forceinline__ double block_sum(double v, double *scratch) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();  // scratch free from any previous use
  if (threadIdx.x % kWave == 0) scratch[w] = v;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int a = 0; a < kLsThreads / kWave; ++a) t += scratch[a];
  return t;
}

// Original GC's approximate decoding for one pattern per block: CGLS on
// min ||A_F r - 1|| (A the 0/1 support, F the workers that processed all their
// chunks), from r = 0 so it converges to the minimum-norm solution; fp64.
// err = ||A_F r - 1||^2 at exit.
__global__ __launch_bounds__(kLsThreads) void original_ls_kernel(
    const int32_t *__restrict__ psi, int N, int m, const int32_t *__restrict__ order, int delta,
    const int32_t *__restrict__ holder, int gamma, int max_iter, double tol,
    double *__restrict__ err, int32_t *__restrict__ iters) {
  extern __shared__ double sh[];
  double *res = sh;           // [N]  1 - A_F r
  double *q = res + N;        // [N]  A_F p
  double *sv = q + N;         // [m]  A_F^T res
  double *pv = sv + m;        // [m]  search direction
  double *rv = pv + m;        // [m]  the decoding vector r
  __shared__ double scratch[kLsThreads / kWave];
  __shared__ uint8_t fin[GC_MAX_M];
  const int64_t p = blockIdx.x;
  const int32_t *ps = psi + p * m;
  for (int j = threadIdx.x; j < m; j += kLsThreads) {
    int load = 0;
    for (int t = 0; t < delta; ++t) {
      const int c = order[int64_t(j) * delta + t];
      load += (c >= 0 && c < N) ? 1 : 0;
    }
    fin[j] = (load > 0 && ps[j] >= load) ? 1 : 0;
    rv[j] = 0.0;
  }
  for (int i = threadIdx.x; i < N; i += kLsThreads) res[i] = 1.0;
  __syncthreads();
  auto AT = [&](const double *v, double *out) {  // out = A_F^T v
    for (int j = threadIdx.x; j < m; j += kLsThreads) {
      double a = 0.0;
      if (fin[j])
        for (int t = 0; t < delta; ++t) {
          const int c = order[int64_t(j) * delta + t];
          if (c >= 0 && c < N) a += v[c];
        }
      out[j] = a;
    }
  };
  auto Ax = [&](const double *v, double *out) {  // out = A_F v
    for (int i = threadIdx.x; i < N; i += kLsThreads) {
      double a = 0.0;
      for (int u = 0; u < gamma; ++u) {
        const int j = holder[int64_t(i) * gamma + u];
        if (j >= 0 && j < m && fin[j]) a += v[j];
      }
      out[i] = a;
    }
  };
  AT(res, sv);
  __syncthreads();
  double part = 0.0;
  for (int j = threadIdx.x; j < m; j += kLsThreads) {
    pv[j] = sv[j];
    part += sv[j] * sv[j];
  }
  double gam = block_sum(part, scratch);
  const double stop = tol * tol * gam;
  int it = 0;
  while (it < max_iter && gam > stop && gam > 0.0) {
    __syncthreads();
    Ax(pv, q);
    __syncthreads();
    part = 0.0;
    for (int i = threadIdx.x; i < N; i += kLsThreads) part += q[i] * q[i];
    const double qq = block_sum(part, scratch);
    if (!(qq > 0.0)) break;
    const double alpha = gam / qq;
    for (int j = threadIdx.x; j < m; j += kLsThreads) rv[j] += alpha * pv[j];
    for (int i = threadIdx.x; i < N; i += kLsThreads) res[i] -= alpha * q[i];
    __syncthreads();
    AT(res, sv);
    __syncthreads();
    part = 0.0;
    for (int j = threadIdx.x; j < m; j += kLsThreads) part += sv[j] * sv[j];
    const double gnew = block_sum(part, scratch);
    const double beta = gnew / gam;
    for (int j = threadIdx.x; j < m; j += kLsThreads) pv[j] = sv[j] + beta * pv[j];
    gam = gnew;
    ++it;
  }
  // recompute the residual from r for the reported error
  __syncthreads();
  Ax(rv, q);
  __syncthreads();
  part = 0.0;
  for (int i = threadIdx.x; i < N; i += kLsThreads) {
    const double e = q[i] - 1.0;
    part += e * e;
  }
  const double e2 = block_sum(part, scratch);
  if (threadIdx.x == 0) {
    err[p] = e2;
    if (iters) iters[p] = it;
  }
}

}  // namespace
}  // namespace gcx

extern "C" int gc_progress(const double *tau, const uint8_t *failed, int64_t R, int32_t m,
                           int32_t delta, const double *T, int32_t G, int32_t *psi,
                           hipStream_t stream) {
  using namespace gcx;
  if (R < 0 || m < 1 || m > GC_MAX_M || delta < 1 || delta > GC_MAX_DELTA || G < 1) return GC_EINVAL;
  // tau [R][m][delta], psi [R][G][m]
  if (!sizes_ok({R, m, delta}) || !sizes_ok({R, G, m})) return GC_EINVAL;
  if (R == 0) return GC_OK;
  if (!tau || !T || !psi) return GC_EINVAL;
  const int64_t blocks = ceil_div(R * m, kSimThreads);
  if (!grid_ok(blocks, kSimThreads)) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  (void)hipGetLastError();
  hipLaunchKernelGGL(progress_kernel, dim3(unsigned(blocks)), dim3(kSimThreads), 0, stream, tau,
                     failed, R, m, delta, T, G, psi);
  return launch_status();
}

extern "C" int gc_completion_times(const double *tau, const uint8_t *failed, int64_t R, int32_t N,
                                   int32_t m, int32_t delta, const int32_t *holder,
                                   const int32_t *hpos, int32_t gamma, int32_t ell,
                                   double *partial, double *original, hipStream_t stream) {
  using namespace gcx;
  if (R < 0 || N < 1 || m < 1 || m > GC_MAX_M || delta < 1 || delta > GC_MAX_DELTA || gamma < 1 ||
      gamma > GC_MAX_DELTA || ell < 1 || ell > GC_MAX_ELL)
    return GC_EINVAL;
  if (!sizes_ok({R, m, delta}) || !sizes_ok({N, gamma})) return GC_EINVAL;  // tau, tables
  if (R == 0) return GC_OK;
  if (!tau || !holder || !hpos || !partial || !original) return GC_EINVAL;
  const int64_t blocks = ceil_div(R, kSimWaves);
  if (!grid_ok(blocks, kSimThreads)) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  (void)hipGetLastError();
  hipLaunchKernelGGL(completion_kernel, dim3(unsigned(blocks)), dim3(kSimThreads), 0, stream, tau,
                     failed, R, N, m, delta, holder, hpos, gamma, ell, partial, original);
  return launch_status();
}

extern "C" int gc_original_ls(const int32_t *psi, int64_t P, int32_t N, int32_t m,
                              const int32_t *order, int32_t delta, const int32_t *holder,
                              int32_t gamma, int32_t max_iter, double tol, double *err,
                              int32_t *iters, hipStream_t stream) {
  using namespace gcx;
  if (P < 0 || N < 1 || N > GC_MAX_M || m < 1 || m > GC_MAX_M || delta < 1 ||
      delta > GC_MAX_DELTA || gamma < 1 || gamma > GC_MAX_DELTA || max_iter < 0 || !(tol >= 0.0))
    return GC_EINVAL;
  if (!sizes_ok({P, m})) return GC_EINVAL;  // psi [P][m]
  if (P == 0) return GC_OK;
  if (!psi || !order || !holder || !err) return GC_EINVAL;
  if (!grid_ok(P, kLsThreads)) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  (void)hipGetLastError();
  const size_t lds = sizeof(double) * (2 * size_t(N) + 3 * size_t(m));
  hipLaunchKernelGGL(original_ls_kernel, dim3(unsigned(P)), dim3(kLsThreads), lds, stream, psi, N,
                     m, order, delta, holder, gamma, max_iter, tol, err, iters);
  return launch_status();
}
