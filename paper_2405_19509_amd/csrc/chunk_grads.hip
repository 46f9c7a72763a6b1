// gc_chunk_grads: per-chunk gradients g_{D_i} = X_i^T r_i (Sec. 1), with
// r_i = X_i w - y_i (linear) or sigmoid(X_i w) - y_i (logistic), at b
// evaluation points.
//
// For one evaluation point this is two matrix-vector products per chunk at
// about 1 flop per byte of X: HBM-bound.  Two streaming kernels:
//   residual_kernel  one wavefront per sample row: dot(x, w) reduced across
//                    the wave, then the loss residual  -> workspace r [b][N][n]
//   xtr_kernel       one block per (point, chunk, 256*VEC columns): the
//                    chunk's residuals staged in LDS, every thread streams its
//                    VEC columns down all n rows (coalesced, several loads in
//                    flight), fixed summation order -> deterministic.
#include "common.h"

namespace gcx {
namespace {

constexpr int kGradThreads = 256;
constexpr int kGradWaves = kGradThreads / kWave;
constexpr int kResidStage = 2048;  // residuals staged in LDS per step

template <int VEC>
__global__ __launch_bounds__(kGradThreads) void residual_kernel(
    const float *__restrict__ X, const float *__restrict__ y, const float *__restrict__ W, int64_t rows,
    int64_t Nn, int64_t d, int loss, float *__restrict__ resid) {
  const int lane = threadIdx.x % kWave;
  const int64_t row = int64_t(blockIdx.x) * kGradWaves + threadIdx.x / kWave;  // q*N*n + i*n + r
  if (row >= rows) return;
  const int64_t q = row / Nn, ir = row % Nn;
  const float *x = X + ir * d;
  const float *w = W + q * d;
  float s = 0.f;
  if constexpr (VEC == 4) {
    const int64_t d4 = d / 4;
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    const float4 *w4 = reinterpret_cast<const float4 *>(w);
    for (int64_t c = lane; c < d4; c += kWave) {
      const float4 a = x4[c], b = w4[c];
      s = fmaf(a.x, b.x, s);
      s = fmaf(a.y, b.y, s);
      s = fmaf(a.z, b.z, s);
      s = fmaf(a.w, b.w, s);
    }
  } else {
    for (int64_t c = lane; c < d; c += kWave) s = fmaf(x[c], w[c], s);
  }
  s = wave_sum(s);
  if (lane == 0) {
    const float yv = y[ir];
    resid[row] = loss == GC_LOSS_LOGISTIC ? 1.0f / (1.0f + expf(-s)) - yv : s - yv;
  }
}

template <int VEC>
__global__ __launch_bounds__(kGradThreads) void xtr_kernel(const float *__restrict__ X,
                                                           const float *__restrict__ resid, int N,
                                                           int n, int64_t d, int64_t tiles,
                                                           float *__restrict__ G) {
  __shared__ float rs[kResidStage];
  const int64_t tile = blockIdx.x % tiles;
  const int64_t qi = blockIdx.x / tiles;  // q*N + i
  const int64_t i = qi % N;
  const int64_t x = (tile * kGradThreads + threadIdx.x) * VEC;
  const float *Xi = X + i * int64_t(n) * d;
  const float *ri = resid + qi * n;
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
  for (int r0 = 0; r0 < n; r0 += kResidStage) {
    const int rn = n - r0 < kResidStage ? n - r0 : kResidStage;
    __syncthreads();
    for (int a = threadIdx.x; a < rn; a += kGradThreads) rs[a] = ri[r0 + a];
    __syncthreads();
    if (x < d) {
      const float *xp = Xi + int64_t(r0) * d + x;
      int r = 0;
      for (; r + 8 <= rn; r += 8) {
        float v[8][VEC];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if constexpr (VEC == 4) {
            const float4 t = *reinterpret_cast<const float4 *>(xp + int64_t(r + u) * d);
            v[u][0] = t.x; v[u][1] = t.y; v[u][2] = t.z; v[u][3] = t.w;
          } else {
            v[u][0] = xp[int64_t(r + u) * d];
          }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float c = rs[r + u];
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] = fmaf(c, v[u][e], acc[e]);
        }
      }
      for (; r < rn; ++r) {
        const float c = rs[r];
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = fmaf(c, xp[int64_t(r) * d + e], acc[e]);
      }
    }
  }
  if (x < d) {
    float *dst = G + qi * d + x;
    if constexpr (VEC == 4) {
      *reinterpret_cast<float4 *>(dst) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    } else {
      dst[0] = acc[0];
    }
  }
}

}  // namespace
}  // namespace gcx

extern "C" size_t gc_chunk_grads_workspace_size(int32_t N, int32_t n, int64_t d, int32_t b) {
  if (N < 1 || n < 1 || d < 1 || b < 1) return 0;
  return sizeof(float) * size_t(b) * size_t(N) * size_t(n);
}

extern "C" int gc_chunk_grads(const float *X, const float *y, const float *W, int32_t N, int32_t n,
                              int64_t d, int32_t b, int32_t loss, float *G, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  using namespace gcx;
  if (N < 1 || n < 1 || d < 1 || b < 1) return GC_EINVAL;
  if (loss != GC_LOSS_LINEAR && loss != GC_LOSS_LOGISTIC) return GC_EINVAL;
  if (!X || !y || !W || !G || !workspace) return GC_EINVAL;
  if (workspace_bytes < gc_chunk_grads_workspace_size(N, n, d, b)) return GC_EINVAL;
  const int64_t rows = int64_t(b) * N * n;
  const bool vec4 = d % 4 == 0 && aligned16(X) && aligned16(W) && aligned16(G);
  const int vec = vec4 ? 4 : 1;
  const int64_t tiles = ceil_div(d, int64_t(kGradThreads) * vec);
  if (!grid_ok(ceil_div(rows, kGradWaves), kGradThreads) || !grid_ok(int64_t(b) * N * tiles, kGradThreads))
    return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  float *resid = static_cast<float *>(workspace);
  (void)hipGetLastError();
  const dim3 g1(unsigned(ceil_div(rows, kGradWaves))), g2(unsigned(int64_t(b) * N * tiles));
  if (vec4) {
    hipLaunchKernelGGL(residual_kernel<4>, g1, dim3(kGradThreads), 0, stream, X, y, W, rows,
                       int64_t(N) * n, d, loss, resid);
    hipLaunchKernelGGL(xtr_kernel<4>, g2, dim3(kGradThreads), 0, stream, X, resid, N, n, d, tiles, G);
  } else {
    hipLaunchKernelGGL(residual_kernel<1>, g1, dim3(kGradThreads), 0, stream, X, y, W, rows,
                       int64_t(N) * n, d, loss, resid);
    hipLaunchKernelGGL(xtr_kernel<1>, g2, dim3(kGradThreads), 0, stream, X, resid, N, n, d, tiles, G);
  }
  return launch_status();
}
