// gc_reconstruct: the PS combine of Sec. 2.2 -- block k of the estimate is
// sum_j R[k][j] g_j -- with an optional fused squared error against the exact
// target; and gc_sum_chunks, the exact target sum_i g_{D_i} itself.
//
// Bandwidth design (HBM-bound on the T read, ~0.5 flop per byte): a block of
// 1024 threads takes items, each one pattern and one piece of 4096 consecutive x
// positions (16 KB of every transmitting worker's row, read as one coalesced sweep
// per row); consecutive items are consecutive pieces of a pattern, and a block
// takes several consecutive items when the estimate is written (see below).
// Measured on MI355X, 16 KB per row and item beats 4 KB and 8 KB (2-3%), and one
// float4 per thread and row beats two or four.  Each thread holds one float4 of ell
// accumulators and keeps kRecUnroll rows of loads in flight; the transmitting
// rows and their weights R[k][j] are compacted into LDS first.  T is read with
// non-temporal loads (it is consumed once).  The squared error is accumulated
// in fp64 per block and reduced across pieces in a fixed order by a second
// small kernel, so it is deterministic.  Given psi, rows of workers with
// psi = 0 (which transmitted nothing) are neither read nor needed.
// The block's writes come last: every item's squared error (with its barrier) first,
// then the estimates with non-temporal stores and the partial sums.  A barrier waits
// for every outstanding memory access of the block's waves, stores included, so an
// estimate stored before one held the block until it had reached memory (the combine
// ran 5% slower at ell = 1 and 10% at ell = 2).  The estimate's 4 bytes per position,
// interleaved into the read stream, still cost far more than their share of the
// traffic (~0.6 ms at the 16384 x 10,000-pattern size with one 16 KB write per item);
// written in 128 KB bursts, 8 / ell items' worth held in LDS per block, they cost
// about a third less.
#include <mutex>

#include "common.h"

namespace gcx {
namespace {

constexpr int kRecThreads = 1024;
constexpr int kRecNV = 1;            // float4 (or 4 scalars) per thread and row
constexpr int kRecV = 4 * kRecNV;    // x positions per thread
constexpr int64_t kRecPiece = int64_t(kRecThreads) * kRecV;  // x positions per block
constexpr int kRecUnroll = 8;        // rows of T loads in flight per thread

typedef float v4f __attribute__((ext_vector_type(4)));

int64_t rec_pieces(int64_t L) { return ceil_div(L, kRecPiece); }

// VEC = 4: thread t owns x = piece*kRecPiece + 4(t + kRecThreads v) + e, v < kRecNV, e < 4
// (needs L % 4 == 0 and aligned T); VEC = 1: x = piece*kRecPiece + t + kRecThreads i,
// i < kRecV (any L).  Either way each load instruction of a block reads consecutive bytes.
template <int VEC>
__device__ __forceinline__ int64_t rec_x(int64_t q, int i) {
  return VEC == 4 ? q * kRecPiece + (int64_t(threadIdx.x) + int64_t(kRecThreads) * (i / 4)) * 4 + i % 4
                  : q * kRecPiece + threadIdx.x + int64_t(kRecThreads) * i;
}

template <int VEC>
__device__ __forceinline__ void rec_load(const float *__restrict__ row, int64_t q, int64_t L,
                                         float (&v)[kRecV]) {
  if constexpr (VEC == 4) {
#pragma unroll
    for (int u = 0; u < kRecNV; ++u) {
      const int64_t x = rec_x<4>(q, 4 * u);
      if (x < L) {
        const v4f t = __builtin_nontemporal_load(reinterpret_cast<const v4f *>(row + x));
        v[4 * u] = t.x; v[4 * u + 1] = t.y; v[4 * u + 2] = t.z; v[4 * u + 3] = t.w;
      } else {
        v[4 * u] = v[4 * u + 1] = v[4 * u + 2] = v[4 * u + 3] = 0.f;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < kRecV; ++i) {
      const int64_t x = rec_x<1>(q, i);
      v[i] = x < L ? __builtin_nontemporal_load(row + x) : 0.f;
    }
  }
}

// Items per block when the estimate is written: K consecutive (pattern, piece) items,
// each item's estimate held in LDS (ell * 16 KB) and all K written at the block's end.
// Interleaved into the read stream, the estimate's writes cost far more than their bytes;
// 128 KB bursts per block cost a third less than one 16 KB write per item.
template <int ELL>
constexpr int rec_items() { return ELL == 1 ? 8 : (ELL == 2 ? 4 : (ELL <= 4 ? 2 : 1)); }

// the estimate's stores of one item (positions as rec_x; the whole float4 where it lies
// inside the gradient, else element by element)
template <int ELL, int VEC>
__device__ __forceinline__ void rec_store(float *__restrict__ ghat, int64_t p, int64_t q, int64_t d,
                                          int64_t L, const float (&acc)[ELL][kRecV]) {
#pragma unroll
  for (int k = 0; k < ELL; ++k) {
#pragma unroll
    for (int u = 0; u < kRecNV; ++u) {
      const int64_t x0 = rec_x<VEC>(q, 4 * u);
      const int64_t c0 = int64_t(k) * L + x0;
      if (VEC == 4 && x0 < L && c0 + 3 < d) {
        const float *a4 = &acc[k][4 * u];
        __builtin_nontemporal_store(v4f{a4[0], a4[1], a4[2], a4[3]},
                                    reinterpret_cast<v4f *>(ghat + p * d + c0));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t x = rec_x<VEC>(q, 4 * u + e);
          const int64_t col = int64_t(k) * L + x;
          if (x < L && col < d) __builtin_nontemporal_store(acc[k][4 * u + e], ghat + p * d + col);
        }
      }
    }
  }
}

// K items per block: item it = blockIdx.x * K + i (pattern it / pieces, piece it % pieces).
// With K > 1 the estimates wait in LDS (`held`, K * ELL * 16 KB of dynamic LDS) and the
// partial sums in `part_s` until every item is done: a barrier waits for every
// outstanding memory access of the block's waves, stores included, so the block's stores
// all come after its last barrier.
template <int ELL, int VEC, int K>
__global__ __launch_bounds__(kRecThreads) void reconstruct_kernel(
    const float *__restrict__ T, const float *__restrict__ R, const int32_t *__restrict__ psi,
    int m, int64_t d, int64_t L, int64_t pieces, int64_t items, float *__restrict__ ghat,
    const float *__restrict__ gsum, double *__restrict__ partial) {
  __shared__ double red[kRecThreads / kWave];
  __shared__ double part_s[K];
  __shared__ int rows[GC_MAX_M];      // the workers that transmitted, ascending
  __shared__ float rw[ELL][GC_MAX_M];  // their R[k][j]
  __shared__ int nrows;
  extern __shared__ __align__(16) unsigned char rec_dyn[];
  v4f *held = reinterpret_cast<v4f *>(rec_dyn);  // [K][ELL][kRecThreads] (K > 1)
  const int64_t it0 = int64_t(blockIdx.x) * K;
  const int nit = int(items - it0 < K ? items - it0 : K);
  int64_t cur_p = -1;
  for (int item = 0; item < nit; ++item) {
  const int64_t p = (it0 + item) / pieces;
  const int64_t q = (it0 + item) % pieces;
  const float *Tp = T + p * int64_t(m) * L;
  __syncthreads();  // the previous item's rows, weights and reduction slots are free

  // compact the transmitting workers (psi > 0) with ballots in wave 0, with their
  // weights R[k][j]
  if (p != cur_p) {
    if (threadIdx.x < kWave) {
      int cnt = 0;
      for (int base = 0; base < m; base += kWave) {
        const int j = base + int(threadIdx.x);
        const bool on = j < m && psi[p * m + j] > 0;
        const unsigned long long mask = __ballot(on);
        if (on) {
          const int a = cnt + __popcll(mask & ((1ull << threadIdx.x) - 1));
          rows[a] = j;
#pragma unroll
          for (int k = 0; k < ELL; ++k) rw[k][a] = R[int64_t(k) * m + j];
        }
        cnt += __popcll(mask);
      }
      if (threadIdx.x == 0) nrows = cnt;
    }
    __syncthreads();
    cur_p = p;
  }
  const int nr = nrows;

  float acc[ELL][kRecV];
#pragma unroll
  for (int k = 0; k < ELL; ++k)
#pragma unroll
    for (int i = 0; i < kRecV; ++i) acc[k][i] = 0.f;
  // software pipeline: the loads of the next kRecUnroll rows are in flight while the
  // current ones are consumed
  float va[kRecUnroll][kRecV], vb[kRecUnroll][kRecV];
  auto issue = [&](int a0, float (&v)[kRecUnroll][kRecV]) {
#pragma unroll
    for (int u = 0; u < kRecUnroll; ++u)
      if (a0 + u < nr) rec_load<VEC>(Tp + int64_t(rows[a0 + u]) * L, q, L, v[u]);
  };
  auto consume = [&](int a0, const float (&v)[kRecUnroll][kRecV]) {
#pragma unroll
    for (int u = 0; u < kRecUnroll; ++u)
      if (a0 + u < nr)
#pragma unroll
      for (int k = 0; k < ELL; ++k) {
        const float r = rw[k][a0 + u];
#pragma unroll
        for (int i = 0; i < kRecV; ++i) acc[k][i] = fmaf(r, v[u][i], acc[k][i]);
      }
  };
  if (nr > 0) issue(0, va);
  for (int a = 0; a < nr; a += 2 * kRecUnroll) {
    if (a + kRecUnroll < nr) issue(a + kRecUnroll, vb);
    consume(a, va);
    if (a + kRecUnroll >= nr) break;
    if (a + 2 * kRecUnroll < nr) issue(a + 2 * kRecUnroll, va);
    consume(a + kRecUnroll, vb);
  }

  // the squared error (gsum reads, the block reduction and its barrier) of this item
  if (partial) {
    double se = 0.0;
#pragma unroll
    for (int k = 0; k < ELL; ++k) {
#pragma unroll
      for (int u = 0; u < kRecNV; ++u) {
        const int64_t x0 = rec_x<VEC>(q, 4 * u);
        const int64_t c0 = int64_t(k) * L + x0;
        if (VEC == 4 && x0 < L && c0 + 3 < d) {  // whole float4 inside the gradient
          const float *a4 = &acc[k][4 * u];
          const float4 g = *reinterpret_cast<const float4 *>(gsum + c0);
          const double e0 = double(a4[0]) - g.x, e1 = double(a4[1]) - g.y;
          const double e2 = double(a4[2]) - g.z, e3 = double(a4[3]) - g.w;
          se += e0 * e0 + e1 * e1 + e2 * e2 + e3 * e3;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int64_t x = rec_x<VEC>(q, 4 * u + e);
            const int64_t col = int64_t(k) * L + x;
            if (x < L && col < d) {
              const double diff = double(acc[k][4 * u + e]) - double(gsum[col]);
              se += diff * diff;
            }
          }
        }
      }
    }
    se = wave_sum(se);
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = se;
    __syncthreads();
    if (threadIdx.x == 0) {
      double tot = 0.0;
      for (int w = 0; w < kRecThreads / kWave; ++w) tot += red[w];
      part_s[item] = tot;
    }
  }
  if constexpr (K == 1) {
    // one item: nothing follows, so its stores can go out directly
    if (ghat) rec_store<ELL, VEC>(ghat, p, q, d, L, acc);
  } else {
#pragma unroll
    for (int k = 0; k < ELL; ++k)
      held[(item * ELL + k) * kRecThreads + threadIdx.x] = v4f{acc[k][0], acc[k][1], acc[k][2], acc[k][3]};
  }
  }  // items

  // the block's stores, after its last barrier
  if constexpr (K > 1) {
    for (int item = 0; item < nit; ++item) {
      const int64_t p = (it0 + item) / pieces, q = (it0 + item) % pieces;
      float acc[ELL][kRecV];
#pragma unroll
      for (int k = 0; k < ELL; ++k) {
        const v4f h = held[(item * ELL + k) * kRecThreads + threadIdx.x];
        acc[k][0] = h.x; acc[k][1] = h.y; acc[k][2] = h.z; acc[k][3] = h.w;
      }
      rec_store<ELL, VEC>(ghat, p, q, d, L, acc);
    }
  }
  if (partial && threadIdx.x == 0)
    for (int item = 0; item < nit; ++item) partial[it0 + item] = part_s[item];
}

__global__ void sqerr_finalize_kernel(const double *__restrict__ partial, int64_t P, int nslices,
                                      double *__restrict__ sqerr) {
  const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (p >= P) return;
  double tot = 0.0;
  for (int s = 0; s < nslices; ++s) tot += partial[p * nslices + s];
  sqerr[p] = tot;
}

template <int ELL, int VEC, int K>
int launch_rec_k(const float *T, const float *R, const int32_t *psi, int64_t P, int m, int64_t d,
                 int64_t L, int64_t pieces, float *ghat, const float *gsum, double *partial,
                 hipStream_t st) {
  const int64_t items = P * pieces;
  const int64_t blocks = ceil_div(items, int64_t(K));
  if (!grid_ok(blocks, kRecThreads)) return GC_EINVAL;
  const size_t dyn = K > 1 ? sizeof(v4f) * size_t(K) * ELL * kRecThreads : 0;
  if (dyn > 0 && hipFuncSetAttribute(reinterpret_cast<const void *>(&reconstruct_kernel<ELL, VEC, K>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(dyn)) != hipSuccess)
    return GC_ELAUNCH;
  hipLaunchKernelGGL((reconstruct_kernel<ELL, VEC, K>), dim3(unsigned(blocks)), dim3(kRecThreads), dyn, st,
                     T, R, psi, m, d, L, pieces, items, ghat, gsum, partial);
  return GC_OK;
}

// items per block: rec_items<ELL>() when the estimate is written, else one
template <int ELL>
int launch_rec(bool vec4, const float *T, const float *R, const int32_t *psi, int64_t P, int m,
               int64_t d, int64_t L, int64_t pieces, float *ghat, const float *gsum, double *partial,
               hipStream_t st) {
  constexpr int KB = rec_items<ELL>();
  if (ghat && KB > 1)
    return vec4 ? launch_rec_k<ELL, 4, KB>(T, R, psi, P, m, d, L, pieces, ghat, gsum, partial, st)
                : launch_rec_k<ELL, 1, KB>(T, R, psi, P, m, d, L, pieces, ghat, gsum, partial, st);
  return vec4 ? launch_rec_k<ELL, 4, 1>(T, R, psi, P, m, d, L, pieces, ghat, gsum, partial, st)
              : launch_rec_k<ELL, 1, 1>(T, R, psi, P, m, d, L, pieces, ghat, gsum, partial, st);
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
  if (P < 1 || m < 1 || d < 1 || ell < 1 || ell > GC_MAX_ELL || !gcx::sizes_ok({P, d}) ||
      !gcx::sizes_ok({P, m, gcx::ceil_div(d, ell)}))
    return 0;
  const int64_t pieces = gcx::rec_pieces(gcx::ceil_div(d, ell));
  return pieces > 1 ? sizeof(double) * size_t(P) * size_t(pieces) : 0;
}

namespace gcx {
namespace {

// The combine behind both entry points: `partial` holds the squared error's per-piece sums
// (P * pieces doubles) when there is more than one piece per pattern.
int reconstruct_impl(const float *T, const float *R, const int32_t *psi, int64_t P, int32_t m, int64_t d,
                     int32_t ell, float *ghat, const float *gsum, double *sqerr, double *partial,
                     hipStream_t stream) {
  const int64_t L = ceil_div(d, ell);
  const int64_t pieces = rec_pieces(L);
  if (sqerr && pieces == 1) partial = sqerr;
  // float4 path: rows of T, the estimate's rows and gsum all 16-byte aligned
  const bool vec4 = L % 4 == 0 && d % 4 == 0 && aligned16(T) && (!ghat || aligned16(ghat)) &&
                    (!gsum || aligned16(gsum));
  (void)hipGetLastError();
  int st = GC_OK;
  switch (ell) {
#define GC_CASE(E)                                                                                 \
  case E:                                                                                          \
    st = launch_rec<E>(vec4, T, R, psi, P, m, d, L, pieces, ghat, sqerr ? gsum : nullptr,          \
                       sqerr ? partial : nullptr, stream);                                         \
    break;
    GC_CASE(1) GC_CASE(2) GC_CASE(3) GC_CASE(4) GC_CASE(5) GC_CASE(6) GC_CASE(7) GC_CASE(8)
#undef GC_CASE
    default: return GC_EINVAL;
  }
  if (st != GC_OK) return st;
  if (sqerr && pieces > 1)
    hipLaunchKernelGGL(sqerr_finalize_kernel, dim3(unsigned(ceil_div(P, 256))), dim3(256), 0, stream,
                       partial, P, int(pieces), sqerr);
  return launch_status();
}

// Argument checks shared by both entry points (sizes, pointers, grid limits).  Returns
// GC_OK to go on, or the status to return; *done = true when there is nothing to do.
int reconstruct_check(const float *T, const float *R, const int32_t *psi, int64_t P, int32_t m, int64_t d,
                      int32_t ell, const float *ghat, const float *gsum, const double *sqerr, bool *done) {
  *done = false;
  if (P < 0 || m < 1 || m > GC_MAX_M || d < 1 || ell < 1 || ell > GC_MAX_ELL) return GC_EINVAL;
  // T [P][m][L], the estimate [P][d]
  if (!sizes_ok({P, d}) || !sizes_ok({P, m, ceil_div(d, ell)})) return GC_EINVAL;
  if (P == 0) {
    *done = true;
    return GC_OK;
  }
  if (!T || !R || !psi) return GC_EINVAL;
  if (sqerr && !gsum) return GC_EINVAL;
  if (!ghat && !sqerr) {  // nothing requested
    *done = true;
    return GC_OK;
  }
  if (!grid_ok(P * rec_pieces(ceil_div(d, ell)), kRecThreads)) return GC_EINVAL;
  return GC_OK;
}

}  // namespace
}  // namespace gcx

extern "C" int gc_reconstruct(const float *T, const float *R, const int32_t *psi, int64_t P,
                              int32_t m, int64_t d, int32_t ell, float *ghat, const float *gsum, double *sqerr,
                              void *workspace, size_t workspace_bytes, hipStream_t stream) {
  using namespace gcx;
  bool done = false;
  const int chk = reconstruct_check(T, R, psi, P, m, d, ell, ghat, gsum, sqerr, &done);
  if (chk != GC_OK || done) return chk;
  const size_t need = sqerr ? gc_reconstruct_workspace_size(P, m, d, ell) : 0;
  if (need && (!workspace || workspace_bytes < need)) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  return reconstruct_impl(T, R, psi, P, m, d, ell, ghat, gsum, sqerr, static_cast<double *>(workspace),
                          stream);
}

// ---------------------------------------------------------------------------------------
// gc_reconstruct_noalloc: the same combine with its scratch (the squared error's per-piece
// sums) in a fixed device array, for callers that cannot allocate.  Each device holds its
// own copy of `scratch`; its address is looked up once per device with the device current
// (the array's name in host code is only a stand-in for the symbol, not a device address).
// Every call on a device shares that device's array: calls that overlap on one device race.
// Nothing needs clearing: every partial sum a call reads, the same call has written.

static __device__ __align__(256) double scratch[GC_NOALLOC_SCRATCH_BYTES / sizeof(double)];

namespace gcx {
namespace {

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices];

int scratch_address(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return GC_ELAUNCH;
  if (dev < 0 || dev >= kMaxDevices) return GC_ENOTSUP;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return GC_ELAUNCH;
    }
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return GC_OK;
}

}  // namespace
}  // namespace gcx

extern "C" int gc_reconstruct_noalloc(const float *T, const float *R, const int32_t *psi, int64_t P,
                                      int32_t m, int64_t d, int32_t ell, float *ghat, const float *gsum,
                                      double *sqerr, hipStream_t stream) {
  using namespace gcx;
  bool done = false;
  const int chk = reconstruct_check(T, R, psi, P, m, d, ell, ghat, gsum, sqerr, &done);
  if (chk != GC_OK || done) return chk;
  const size_t need = sqerr ? gc_reconstruct_workspace_size(P, m, d, ell) : 0;
  if (need > GC_NOALLOC_SCRATCH_BYTES) return GC_ESCRATCH;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  void *ws = nullptr;
  if (need) {
    const int st = scratch_address(&ws);
    if (st != GC_OK) return st;
  }
  return reconstruct_impl(T, R, psi, P, m, d, ell, ghat, gsum, sqerr, static_cast<double *>(ws), stream);
}

extern "C" int gc_sum_chunks(const void *G, int32_t g_dtype, int32_t N, int64_t d, float *gsum,
                             hipStream_t stream) {
  using namespace gcx;
  if (N < 1 || d < 1 || !G || !gsum || (g_dtype != GC_F32 && g_dtype != GC_BF16)) return GC_EINVAL;
  if (!sizes_ok({N, d})) return GC_EINVAL;
  if (!grid_ok(ceil_div(d, 256), 256)) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  (void)hipGetLastError();
  hipLaunchKernelGGL(sum_chunks_kernel, dim3(unsigned(ceil_div(d, 256))), dim3(256), 0, stream, G,
                     g_dtype == GC_BF16 ? 1 : 0, N, d, gsum);
  return launch_status();
}
