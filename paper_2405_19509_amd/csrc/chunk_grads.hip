// gc_chunk_grads: per-chunk gradients g_{D_i} = X_i^T r_i (Sec. 1), with
// r_i = X_i w - y_i (linear) or sigmoid(X_i w) - y_i (logistic), at b
// evaluation points.
//
// For one evaluation point this is two matrix-vector products per chunk at
// about 1 flop per byte of X: HBM-bound, and X is the only large operand, so
// the goal is to read it exactly once.
//
// Fused path (d <= 16384, d % 4 == 0): fused_grad_kernel gives each block a
// contiguous range of sample rows (at most n, so it touches at most two
// chunks).  A 512-thread block holds a whole row in registers (8 float4 per
// thread at d = 16384) together with w and its running partial gradient:
// load the row once, reduce x.w across the block, form the residual, and add
// r * x into the partial.  Partials go to the workspace (two slots per
// block) and reduce_partials_kernel sums, for every chunk, the partials of
// the blocks that touched it, in block order: one read of X, deterministic.
//
// Many points (b >= 16, b % 4 == 0, d % 4 == 0): two fp32 MFMA GEMMs per chunk
// (chunk_grads_mfma.hip).
//
// General path (any d): two streaming kernels
//   residual_kernel  one wavefront per sample row: dot(x, w) reduced across
//                    the wave, then the loss residual  -> workspace r [b][N][n]
//   xtr_kernel       one block per (point, chunk, 256*VEC columns): the
//                    chunk's residuals staged in LDS, every thread streams its
//                    VEC columns down all n rows (coalesced, several loads in
//                    flight), fixed summation order -> deterministic.
#include "common.h"

namespace gcx {

// multi-point path on the matrix cores (chunk_grads_mfma.hip)
bool mfma_eligible(int64_t d, int b);
size_t mfma_workspace_bytes(int N, int n, int64_t d, int b);
int launch_mfma_grads(const float *X, const float *y, const float *W, int N, int n, int64_t d, int b,
                      int loss, float *G, void *workspace, hipStream_t st);

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


constexpr int kFusedThreads = 512;
constexpr int kFusedWaves = kFusedThreads / kWave;
constexpr int kFusedMaxNV = 8;  // float4 per thread: d <= 512 * 4 * 8 = 16384

struct FusedPlan {
  int64_t blocks;          // blocks per evaluation point
  int64_t rows_per_block;  // <= n
};

inline FusedPlan fused_plan(int N, int n) {
  const int64_t R = int64_t(N) * n;
  int64_t blocks = 512;  // two 512-thread blocks per CU on 256 CUs
  if (blocks < N) blocks = N;
  int64_t rpb = ceil_div(R, blocks);
  if (rpb > n) rpb = n;
  return FusedPlan{ceil_div(R, rpb), rpb};
}

__device__ __forceinline__ float loss_residual(float z, float yv, int loss) {
  return loss == GC_LOSS_LOGISTIC ? 1.0f / (1.0f + expf(-z)) - yv : z - yv;
}

template <int NV>
__global__ __launch_bounds__(kFusedThreads) void fused_grad_kernel(
    const float *__restrict__ X, const float *__restrict__ y, const float *__restrict__ W, int N,
    int n, int64_t d, int loss, int64_t rows_per_block, int64_t blocks, float *__restrict__ part) {
  __shared__ float red[2][kFusedWaves];
  const int q = blockIdx.y;
  const int64_t b = blockIdx.x;
  const int64_t R = int64_t(N) * n;
  const int64_t r0 = b * rows_per_block;
  const int64_t r1 = r0 + rows_per_block < R ? r0 + rows_per_block : R;
  const int64_t d4 = d / 4;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;

  float4 w[NV], acc[NV];
  const float4 *w4 = reinterpret_cast<const float4 *>(W + int64_t(q) * d);
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int64_t c = threadIdx.x + int64_t(kFusedThreads) * v;
    w[v] = c < d4 ? w4[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    acc[v] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const int64_t c0 = r0 / n;  // first chunk of this block
  int64_t cur = c0;
  float *slot = part + ((int64_t(q) * blocks + b) * 2) * d;

  auto flush = [&](int64_t chunk) {
    float4 *dst = reinterpret_cast<float4 *>(slot + (chunk - c0) * d);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int64_t c = threadIdx.x + int64_t(kFusedThreads) * v;
      if (c < d4) dst[c] = acc[v];
      acc[v] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };

  for (int64_t r = r0; r < r1; ++r) {
    const int64_t c = r / n;
    if (c != cur) {
      flush(cur);
      cur = c;
    }
    const float4 *x4 = reinterpret_cast<const float4 *>(X + r * d);
    float4 x[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int64_t cc = threadIdx.x + int64_t(kFusedThreads) * v;
      x[v] = cc < d4 ? x4[cc] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      s = fmaf(x[v].x, w[v].x, s);
      s = fmaf(x[v].y, w[v].y, s);
      s = fmaf(x[v].z, w[v].z, s);
      s = fmaf(x[v].w, w[v].w, s);
    }
    s = wave_sum(s);
    const int par = int(r & 1);  // two buffers: one barrier per row suffices
    if (lane == 0) red[par][wave] = s;
    __syncthreads();
    float z = 0.f;
#pragma unroll
    for (int k = 0; k < kFusedWaves; ++k) z += red[par][k];
    const float u = loss_residual(z, y[r], loss);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      acc[v].x = fmaf(u, x[v].x, acc[v].x);
      acc[v].y = fmaf(u, x[v].y, acc[v].y);
      acc[v].z = fmaf(u, x[v].z, acc[v].z);
      acc[v].w = fmaf(u, x[v].w, acc[v].w);
    }
  }
  if (r1 > r0) flush(cur);
}

// G[q][i][x] = sum over the blocks b that touched chunk i (ascending) of their partial.
__global__ void reduce_partials_kernel(const float *__restrict__ part, int N, int n, int64_t d,
                                       int64_t rows_per_block, int64_t blocks, float *__restrict__ G) {
  const int64_t x4 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t i = blockIdx.y;
  const int q = blockIdx.z;
  if (x4 * 4 >= d) return;
  const int64_t bfirst = (i * n) / rows_per_block;
  const int64_t blast = ((i + 1) * n - 1) / rows_per_block;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t b = bfirst; b <= blast; ++b) {
    const int64_t c0 = (b * rows_per_block) / n;
    const float4 v = reinterpret_cast<const float4 *>(part + ((int64_t(q) * blocks + b) * 2 + (i - c0)) * d)[x4];
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  reinterpret_cast<float4 *>(G + (int64_t(q) * N + i) * d)[x4] = s;
}

}  // namespace
}  // namespace gcx

namespace {
bool fused_ok(int64_t d) { return d % 4 == 0 && d <= int64_t(gcx::kFusedThreads) * 4 * gcx::kFusedMaxNV; }
}  // namespace

namespace {
// X [N][n][d], W [b][d], G [b][N][d], residuals [b][N][n]
bool grad_sizes_ok(int32_t N, int32_t n, int64_t d, int32_t b) {
  return N >= 1 && n >= 1 && d >= 1 && b >= 1 && gcx::sizes_ok({N, n, d}) && gcx::sizes_ok({b, N, d}) &&
         gcx::sizes_ok({b, N, n});
}
}  // namespace

extern "C" size_t gc_chunk_grads_workspace_size(int32_t N, int32_t n, int64_t d, int32_t b) {
  if (!grad_sizes_ok(N, n, d, b)) return 0;
  if (gcx::mfma_eligible(d, b)) return gcx::mfma_workspace_bytes(N, n, d, b);
  if (fused_ok(d)) {
    const gcx::FusedPlan fp = gcx::fused_plan(N, n);
    return sizeof(float) * size_t(b) * size_t(fp.blocks) * 2 * size_t(d);
  }
  return sizeof(float) * size_t(b) * size_t(N) * size_t(n);
}

extern "C" int gc_chunk_grads(const float *X, const float *y, const float *W, int32_t N, int32_t n,
                              int64_t d, int32_t b, int32_t loss, float *G, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  using namespace gcx;
  if (!grad_sizes_ok(N, n, d, b)) return GC_EINVAL;
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
  (void)hipGetLastError();
  if (mfma_eligible(d, b)) {
    if (!vec4 || !aligned16(y) || !aligned16(workspace)) return GC_EINVAL;
    const int st = launch_mfma_grads(X, y, W, N, n, d, b, loss, G, workspace, stream);
    if (st != GC_OK) return st;
    return launch_status();
  }
  if (vec4 && fused_ok(d) && aligned16(workspace)) {
    const FusedPlan fp = fused_plan(N, n);
    if (!grid_ok(fp.blocks * b, kFusedThreads)) return GC_EINVAL;
    float *part = static_cast<float *>(workspace);
    const int nv = int(ceil_div(d, int64_t(kFusedThreads) * 4));
    const dim3 g1(unsigned(fp.blocks), unsigned(b));
#define GC_FUSED(NV)                                                                              \
  hipLaunchKernelGGL(fused_grad_kernel<NV>, g1, dim3(kFusedThreads), 0, stream, X, y, W, N, n, d, \
                     loss, fp.rows_per_block, fp.blocks, part)
    if (nv <= 1) GC_FUSED(1);
    else if (nv <= 2) GC_FUSED(2);
    else if (nv <= 4) GC_FUSED(4);
    else GC_FUSED(8);
#undef GC_FUSED
    const dim3 g2(unsigned(ceil_div(d / 4, 256)), unsigned(N), unsigned(b));
    hipLaunchKernelGGL(reduce_partials_kernel, g2, dim3(256), 0, stream, part, N, n, d,
                       fp.rows_per_block, fp.blocks, G);
    return launch_status();
  }
  float *resid = static_cast<float *>(workspace);
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
