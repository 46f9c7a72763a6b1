// gc_reconstruct: the PS combine of Sec. 2.2 -- block k of the estimate is
// sum_j R[k][j] g_j -- with an optional fused squared error against the exact
// target; and gc_sum_chunks, the exact target sum_i g_{D_i} itself.
//
// Bandwidth design (HBM-bound on the T read, ~0.5 flop per byte): a block
// owns one pattern and one slice of 4096 consecutive x positions; each thread
// keeps Q = 4096 / (256 * VEC) vectors of ell accumulators and, for every
// worker j, issues its Q independent vector loads of T[p][j][slice] before
// using any of them (Q loads in flight per thread, every T byte read once).
// R[k][j] is a wave-uniform value read from LDS.  The squared error is
// accumulated in fp64 per block and reduced across slices in a fixed order by
// a second small kernel, so it is deterministic.
#include "common.h"

namespace gcx {
namespace {

constexpr int kRecThreads = 256;
constexpr int64_t kRecSlice = 4096;

size_t rec_slices(int64_t L) { return size_t(ceil_div(L, kRecSlice)); }

template <int ELL, int VEC>
__global__ __launch_bounds__(kRecThreads) void reconstruct_kernel(
    const float *__restrict__ T, const float *__restrict__ R, int m, int64_t d, int64_t L,
    int nslices, float *__restrict__ ghat, const float *__restrict__ gsum,
    double *__restrict__ partial) {
  constexpr int Q = int(kRecSlice / (kRecThreads * VEC));
  extern __shared__ float Rs[];  // [ELL][m]
  __shared__ double red[kRecThreads / kWave];
  for (int a = threadIdx.x; a < ELL * m; a += kRecThreads) Rs[a] = R[a];
  __syncthreads();

  const int64_t p = blockIdx.x / nslices;
  const int64_t s = blockIdx.x % nslices;
  const int64_t xs = s * kRecSlice;

  float acc[ELL][Q][VEC];
#pragma unroll
  for (int k = 0; k < ELL; ++k)
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[k][q][e] = 0.f;

  const float *Tp = T + p * int64_t(m) * L;
  for (int j = 0; j < m; ++j) {
    float v[Q][VEC];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int64_t x = xs + (int64_t(q) * kRecThreads + threadIdx.x) * VEC;
      if (x < L) {
        const float *src = Tp + int64_t(j) * L + x;
        if constexpr (VEC == 4) {
          const float4 t4 = *reinterpret_cast<const float4 *>(src);
          v[q][0] = t4.x; v[q][1] = t4.y; v[q][2] = t4.z; v[q][3] = t4.w;
        } else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[q][e] = src[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[q][e] = 0.f;
      }
    }
#pragma unroll
    for (int k = 0; k < ELL; ++k) {
      const float r = Rs[k * m + j];
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[k][q][e] = fmaf(r, v[q][e], acc[k][q][e]);
    }
  }

  double se = 0.0;
#pragma unroll
  for (int k = 0; k < ELL; ++k)
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int64_t x = xs + (int64_t(q) * kRecThreads + threadIdx.x) * VEC;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int64_t col = int64_t(k) * L + x + e;
        if (x + e < L && col < d) {
          const float gv = acc[k][q][e];
          if (ghat) ghat[p * d + col] = gv;
          if (partial) {
            const double diff = double(gv) - double(gsum[col]);
            se += diff * diff;
          }
        }
      }
    }
  if (partial) {
    se = wave_sum(se);
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = se;
    __syncthreads();
    if (threadIdx.x == 0) {
      double tot = 0.0;
      for (int w = 0; w < kRecThreads / kWave; ++w) tot += red[w];
      partial[p * nslices + s] = tot;
    }
  }
}

__global__ void sqerr_finalize_kernel(const double *__restrict__ partial, int64_t P, int nslices,
                                      double *__restrict__ sqerr) {
  const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (p >= P) return;
  double tot = 0.0;
  for (int s = 0; s < nslices; ++s) tot += partial[p * nslices + s];
  sqerr[p] = tot;
}

template <int ELL>
void launch_rec(bool vec4, const float *T, const float *R, int64_t P, int m, int64_t d, int64_t L,
                int nslices, float *ghat, const float *gsum, double *partial, hipStream_t st) {
  const int64_t blocks = P * nslices;
  const size_t lds = sizeof(float) * ELL * m;
  if (vec4)
    hipLaunchKernelGGL((reconstruct_kernel<ELL, 4>), dim3(unsigned(blocks)), dim3(kRecThreads), lds,
                       st, T, R, m, d, L, nslices, ghat, gsum, partial);
  else
    hipLaunchKernelGGL((reconstruct_kernel<ELL, 1>), dim3(unsigned(blocks)), dim3(kRecThreads), lds,
                       st, T, R, m, d, L, nslices, ghat, gsum, partial);
}

__global__ void sum_chunks_kernel(const void *__restrict__ G, int bf16, int N, int64_t d,
                                  float *__restrict__ gsum) {
  const int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (x >= d) return;
  double acc = 0.0;
  if (bf16) {
    const uint16_t *g = static_cast<const uint16_t *>(G);
    for (int i = 0; i < N; ++i) acc += double(bf16_to_f32(g[int64_t(i) * d + x]));
  } else {
    const float *g = static_cast<const float *>(G);
    for (int i = 0; i < N; ++i) acc += double(g[int64_t(i) * d + x]);
  }
  gsum[x] = float(acc);
}

}  // namespace
}  // namespace gcx

extern "C" size_t gc_reconstruct_workspace_size(int64_t P, int32_t m, int64_t d, int32_t ell) {
  (void)m;
  if (P < 1 || d < 1 || ell < 1 || ell > GC_MAX_ELL) return 0;
  const size_t ns = gcx::rec_slices(gcx::ceil_div(d, ell));
  return ns > 1 ? sizeof(double) * size_t(P) * ns : 0;
}

extern "C" int gc_reconstruct(const float *T, const float *R, int64_t P, int32_t m, int64_t d,
                              int32_t ell, float *ghat, const float *gsum, double *sqerr,
                              void *workspace, size_t workspace_bytes, hipStream_t stream) {
  using namespace gcx;
  if (P < 0 || m < 1 || m > GC_MAX_M || d < 1 || ell < 1 || ell > GC_MAX_ELL) return GC_EINVAL;
  if (P == 0) return GC_OK;
  if (!T || !R) return GC_EINVAL;
  const bool want_err = sqerr != nullptr;
  if (want_err && !gsum) return GC_EINVAL;
  if (!ghat && !want_err) return GC_OK;  // nothing requested
  const int64_t L = ceil_div(d, ell);
  const int nslices = int(rec_slices(L));
  if (P * nslices > 0x7fffffffLL) return GC_EINVAL;
  double *partial = nullptr;
  if (want_err) {
    if (nslices == 1) {
      partial = sqerr;
    } else {
      const size_t need = gc_reconstruct_workspace_size(P, m, d, ell);
      if (!workspace || workspace_bytes < need) return GC_EINVAL;
      partial = static_cast<double *>(workspace);
    }
  }
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  const bool vec4 = (L % 4 == 0) && aligned16(T);
  (void)hipGetLastError();
  switch (ell) {
#define GC_CASE(E)                                                                           \
  case E:                                                                                    \
    launch_rec<E>(vec4, T, R, P, m, d, L, nslices, ghat, gsum, partial, stream);             \
    break;
    GC_CASE(1) GC_CASE(2) GC_CASE(3) GC_CASE(4) GC_CASE(5) GC_CASE(6) GC_CASE(7) GC_CASE(8)
#undef GC_CASE
    default: return GC_EINVAL;
  }
  if (want_err && nslices > 1)
    hipLaunchKernelGGL(sqerr_finalize_kernel, dim3(unsigned(ceil_div(P, 256))), dim3(256), 0,
                       stream, partial, P, nslices, sqerr);
  return launch_status();
}

extern "C" int gc_sum_chunks(const void *G, int32_t g_dtype, int32_t N, int64_t d, float *gsum,
                             hipStream_t stream) {
  using namespace gcx;
  if (N < 1 || d < 1 || !G || !gsum || (g_dtype != GC_F32 && g_dtype != GC_BF16)) return GC_EINVAL;
  if (ceil_div(d, 256) > 0x7fffffffLL) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  (void)hipGetLastError();
  hipLaunchKernelGGL(sum_chunks_kernel, dim3(unsigned(ceil_div(d, 256))), dim3(256), 0, stream, G,
                     g_dtype == GC_BF16 ? 1 : 0, N, d, gsum);
  return launch_status();
}
