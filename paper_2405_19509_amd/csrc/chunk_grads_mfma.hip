// Chunk gradients at many evaluation points on the fp32 matrix cores.
//
// With b evaluation points W [b][d] the per-chunk gradient (Sec. 1) is two
// dense contractions per chunk i:
//   Z_i = X_i W^T          [n][b]   (K = d)
//   U_i = loss'(Z_i) - y_i [n][b]   (residuals, broadcast over the points)
//   G_i = U_i^T X_i        [b][d]   (K = n),   stored as G[q][i][:]
// Both run as 128 x 128-tiled GEMMs on v_mfma_f32_32x32x2f32: a 256-thread
// block holds a 128 x 128 output tile as four 64 x 64 wave tiles (2 x 2 MFMA
// tiles of 32 x 32 each); operands are staged through double-buffered LDS,
// 32 values of K per stage, with the global loads of the stage after next in
// flight (two register sets) while the current one feeds the MFMAs.  fp32 in,
// fp32 accumulation.
//
//   zw_kernel     Z partials over a split of K = d (split-K keeps >= ~3 waves
//                 of blocks on 256 CUs); both operands are K-contiguous, held
//                 in LDS as [row][k] and read four k at a time: within a
//                 stage lane half h takes the k in [16h, 16h + 16), so each
//                 lane's operands for four consecutive MFMAs are one 16-byte
//                 LDS read (the K order inside a stage is a permutation shared
//                 by both operands, so the sum is unchanged).
//   resid_kernel  U = loss'(sum of the partials, in split order) - y.
//   utx_kernel    G tiles; both operands are row-contiguous along M and N,
//                 held in LDS as [k][row].
// Along the points both kernels use 128-wide tiles when b is a multiple of 128 and
// 64-wide tiles otherwise, so b = 64 does not spend half the MFMAs on padding.
#include <type_traits>

#include "common.h"

namespace gcx {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kTM = 128;  // tile rows
constexpr int kTN = 128;  // tile cols
constexpr int kTK = 32;   // K per stage
constexpr int kMThreads = 256;
constexpr int kPadK = 4;  // [row][k] LDS rows: 36 floats apart, conflict-free 16-byte reads

__device__ __forceinline__ v16f mfma32(float a, float b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }

__device__ __forceinline__ float comp(const float4 &v, int e) {
  return e == 0 ? v.x : (e == 1 ? v.y : (e == 2 ? v.z : v.w));
}

// Z partial: Zp[s][i][r][q] = sum_{x in split s} X[i][r][x] * W[q][x].  TB = tile width
// along the points (128, or 64 when b is not a multiple of 128: no padded half tile).
template <int TB>
__global__ __launch_bounds__(kMThreads, 2) void zw_kernel(const float *__restrict__ X,
                                                          const float *__restrict__ W, int N, int n,
                                                          int64_t d, int b, int splits, int64_t kper,
                                                          int mtiles, int ntiles,
                                                          float *__restrict__ Zp) {
  constexpr int NB = TB / 64;  // 32-wide MFMA blocks per wave along the points
  __shared__ __align__(16) float As[2][kTM][kTK + kPadK];
  __shared__ __align__(16) float Bs[2][TB][kTK + kPadK];
  int64_t bid = blockIdx.x;
  const int nt = int(bid % ntiles);
  bid /= ntiles;
  const int mt = int(bid % mtiles);
  bid /= mtiles;
  const int s = int(bid % splits);
  const int64_t i = bid / splits;
  const int t = threadIdx.x, lane = t % kWave, wave = t / kWave;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, li = lane & 31;
  const float *Xi = X + i * int64_t(n) * d;
  const int64_t k0 = int64_t(s) * kper;
  const int64_t k1 = k0 + kper < d ? k0 + kper : d;
  const int lrow = t >> 3, lk = (t & 7) * 4;

  // two register sets: the stage after next loads while this stage feeds the MFMAs
  float4 ra[2][4], rb[2][4];
  auto gload = [&](int set, int64_t kb) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int row = lrow + 32 * p;
      const int64_t k = kb + lk;
      const int r = mt * kTM + row, q = nt * TB + row;
      ra[set][p] = (r < n && k < k1) ? ld4(Xi + int64_t(r) * d + k) : make_float4(0.f, 0.f, 0.f, 0.f);
      rb[set][p] = (row < TB && q < b && k < k1) ? ld4(W + int64_t(q) * d + k)
                                                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto lstore = [&](int set, int buf) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      *reinterpret_cast<float4 *>(&As[buf][lrow + 32 * p][lk]) = ra[set][p];
      if (lrow + 32 * p < TB) *reinterpret_cast<float4 *>(&Bs[buf][lrow + 32 * p][lk]) = rb[set][p];
    }
  };

  v16f acc[2][NB];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.f;

  const int64_t nst = ceil_div(k1 - k0, kTK);
  gload(0, k0);
  if (nst > 1) gload(1, k0 + kTK);
  lstore(0, 0);
  __syncthreads();
  // stage st is in LDS buffer st & 1, stage st + 1 in register set (st + 1) & 1
  auto stage = [&](int64_t st, auto setc) {
    constexpr int SET = decltype(setc)::value;  // st & 1
    if (st + 2 < nst) gload(SET, k0 + (st + 2) * kTK);
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      float4 a[2], bb[NB];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) a[mb] = ld4(&As[SET][wm * 64 + mb * 32 + li][h * 16 + s4 * 4]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        bb[nb] = ld4(&Bs[SET][wn * (TB / 2) + nb * 32 + li][h * 16 + s4 * 4]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = mfma32(comp(a[mb], e), comp(bb[nb], e), acc[mb][nb]);
    }
    if (st + 1 < nst) lstore(SET ^ 1, SET ^ 1);
    __syncthreads();
  };
  for (int64_t st = 0; st < nst; st += 2) {
    stage(st, std::integral_constant<int, 0>{});
    if (st + 1 < nst) stage(st + 1, std::integral_constant<int, 1>{});
  }

  float *Zs = Zp + (int64_t(s) * N + i) * int64_t(n) * b;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = mt * kTM + wm * 64 + mb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        const int q = nt * TB + wn * (TB / 2) + nb * 32 + li;
        if (r < n && q < b) Zs[int64_t(r) * b + q] = acc[mb][nb][v];
      }
}

// U[i][r][q] = loss'(sum_s Zp[s][i][r][q]) - y[i][r], the splits summed in order.
__global__ void resid_kernel(const float *__restrict__ Zp, const float *__restrict__ y, int64_t total,
                             int b, int splits, int loss, float *__restrict__ Uo) {
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  float z = 0.f;
  for (int s = 0; s < splits; ++s) z += Zp[int64_t(s) * total + e];
  const float yv = y[e / b];
  Uo[e] = loss == GC_LOSS_LOGISTIC ? 1.0f / (1.0f + expf(-z)) - yv : z - yv;
}

// G[q][i][x] = sum_r U[i][r][q] * X[i][r][x]; TB = tile height along the points.
template <int TB>
__global__ __launch_bounds__(kMThreads, 2) void utx_kernel(const float *__restrict__ Ui,
                                                           const float *__restrict__ X, int N, int n,
                                                           int64_t d, int b, int mtiles,
                                                           int64_t ntiles, float *__restrict__ G) {
  constexpr int MB = TB / 64;  // 32-high MFMA blocks per wave along the points
  __shared__ __align__(16) float As[2][kTK][TB + 4];
  __shared__ __align__(16) float Bs[2][kTK][kTN + 4];
  int64_t bid = blockIdx.x;
  const int mt = int(bid % mtiles);  // the point tiles of one X tile run back to back
  bid /= mtiles;
  const int64_t nt = bid % ntiles;
  const int64_t i = bid / ntiles;
  const int t = threadIdx.x, lane = t % kWave, wave = t / kWave;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, li = lane & 31;
  const float *Xi = X + i * int64_t(n) * d;
  const float *Uc = Ui + i * int64_t(n) * b;
  const int lrow = t >> 5, lc = (t & 31) * 4;

  // two register sets: the stage after next loads while this stage feeds the MFMAs
  float4 ra[2][4], rb[2][4];
  auto gload = [&](int set, int kb) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int r = kb + lrow + 8 * p;
      const int q = mt * TB + lc;
      const int64_t x = nt * kTN + lc;
      ra[set][p] = (lc < TB && r < n && q < b) ? ld4(Uc + int64_t(r) * b + q)
                                               : make_float4(0.f, 0.f, 0.f, 0.f);
      rb[set][p] = (r < n && x < d) ? ld4(Xi + int64_t(r) * d + x) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto lstore = [&](int set, int buf) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (lc < TB) *reinterpret_cast<float4 *>(&As[buf][lrow + 8 * p][lc]) = ra[set][p];
      *reinterpret_cast<float4 *>(&Bs[buf][lrow + 8 * p][lc]) = rb[set][p];
    }
  };

  v16f acc[MB][2];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.f;

  const int nst = int(ceil_div(n, kTK));
  gload(0, 0);
  if (nst > 1) gload(1, kTK);
  lstore(0, 0);
  __syncthreads();
  // stage st is in LDS buffer st & 1, stage st + 1 in register set (st + 1) & 1
  auto stage = [&](int st, auto setc) {
    constexpr int SET = decltype(setc)::value;  // st & 1
    if (st + 2 < nst) gload(SET, (st + 2) * kTK);
#pragma unroll
    for (int s = 0; s < kTK / 2; ++s) {
      float a[MB], bb[2];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) a[mb] = As[SET][2 * s + h][wm * (TB / 2) + mb * 32 + li];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) bb[nb] = Bs[SET][2 * s + h][wn * 64 + nb * 32 + li];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = mfma32(a[mb], bb[nb], acc[mb][nb]);
    }
    if (st + 1 < nst) lstore(SET ^ 1, SET ^ 1);
    __syncthreads();
  };
  for (int st = 0; st < nst; st += 2) {
    stage(st, std::integral_constant<int, 0>{});
    if (st + 1 < nst) stage(st + 1, std::integral_constant<int, 1>{});
  }

#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int q = mt * TB + wm * (TB / 2) + mb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        const int64_t x = nt * kTN + wn * 64 + nb * 32 + li;
        if (q < b && x < d) G[(int64_t(q) * N + i) * d + x] = acc[mb][nb][v];
      }
}

}  // namespace

// Launch plan shared by the workspace-size query and the launch.
struct MfmaPlan {
  int tb;  // tile width along the points: 128, or 64 when b is not a multiple of 128
  int splits;
  int64_t kper;
  int mtiles1, ntiles1;  // zw tiles over (rows r, points q)
  size_t zp_floats, u_floats;
};

MfmaPlan mfma_plan(int N, int n, int64_t d, int b) {
  MfmaPlan pl{};
  pl.tb = b % 128 == 0 ? 128 : 64;
  pl.mtiles1 = int(ceil_div(n, kTM));
  pl.ntiles1 = int(ceil_div(b, pl.tb));
  const int64_t tiles = int64_t(N) * pl.mtiles1 * pl.ntiles1;
  // K = d split (at most 16 ways) so that the blocks fill whole rounds of the 512 resident
  // ones (two per CU on 256 CUs): a grid that overshoots a round by a little runs its last
  // round mostly empty.  Each split is charged half a percent (its Z partials, written and
  // summed again, and a block prologue per tile); ties go to fewer splits.
  constexpr int64_t kResident = 512;
  int64_t splits = 1;
  double best = -1.0;
  for (int64_t sp = 1; sp <= 16; ++sp) {
    const int64_t kp = ceil_div(ceil_div(d, sp), kTK) * kTK;
    if (ceil_div(d, kp) != sp) continue;  // stage rounding merges splits: a smaller sp covers it
    const int64_t blocks = tiles * sp;
    const double fill = double(blocks) / double(ceil_div(blocks, kResident) * kResident);
    const double score = fill - 0.005 * double(sp);
    if (score > best + 1e-9) {
      best = score;
      splits = sp;
    }
  }
  const int64_t kper = ceil_div(ceil_div(d, splits), kTK) * kTK;
  splits = ceil_div(d, kper);
  pl.splits = int(splits);
  pl.kper = kper;
  pl.zp_floats = size_t(splits) * N * size_t(n) * b;
  pl.u_floats = size_t(N) * n * size_t(b);
  return pl;
}

bool mfma_eligible(int64_t d, int b) { return b >= 16 && b % 4 == 0 && d % 4 == 0; }

size_t mfma_workspace_bytes(int N, int n, int64_t d, int b) {
  const MfmaPlan pl = mfma_plan(N, n, d, b);
  return sizeof(float) * (pl.zp_floats + pl.u_floats);
}

int launch_mfma_grads(const float *X, const float *y, const float *W, int N, int n, int64_t d, int b,
                      int loss, float *G, void *workspace, hipStream_t st) {
  const MfmaPlan pl = mfma_plan(N, n, d, b);
  float *Zp = static_cast<float *>(workspace);
  float *Uo = Zp + pl.zp_floats;
  const int64_t blocks1 = int64_t(N) * pl.splits * pl.mtiles1 * pl.ntiles1;
  const int mtiles2 = int(ceil_div(b, pl.tb));
  const int64_t ntiles2 = ceil_div(d, kTN);
  const int64_t blocks2 = int64_t(N) * ntiles2 * mtiles2;
  const int64_t total = int64_t(N) * n * b;
  if (!grid_ok(blocks1, kMThreads) || !grid_ok(blocks2, kMThreads) || !grid_ok(ceil_div(total, 256), 256))
    return GC_EINVAL;
  if (pl.tb == 128)
    hipLaunchKernelGGL(zw_kernel<128>, dim3(unsigned(blocks1)), dim3(kMThreads), 0, st, X, W, N, n,
                       d, b, pl.splits, pl.kper, pl.mtiles1, pl.ntiles1, Zp);
  else
    hipLaunchKernelGGL(zw_kernel<64>, dim3(unsigned(blocks1)), dim3(kMThreads), 0, st, X, W, N, n,
                       d, b, pl.splits, pl.kper, pl.mtiles1, pl.ntiles1, Zp);
  hipLaunchKernelGGL(resid_kernel, dim3(unsigned(ceil_div(total, 256))), dim3(256), 0, st, Zp, y,
                     total, b, pl.splits, loss, Uo);
  if (pl.tb == 128)
    hipLaunchKernelGGL(utx_kernel<128>, dim3(unsigned(blocks2)), dim3(kMThreads), 0, st, Uo, X, N, n,
                       d, b, mtiles2, ntiles2, G);
  else
    hipLaunchKernelGGL(utx_kernel<64>, dim3(unsigned(blocks2)), dim3(kMThreads), 0, st, Uo, X, N, n,
                       d, b, mtiles2, ntiles2, G);
  return GC_OK;
}

}  // namespace gcx
