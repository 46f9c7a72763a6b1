// gc_decode_direct: the PS's estimate without materialising what the workers
// transmit.  Substituting the worker encode (Sec. 2) into the PS combine
// (Sec. 2.2):
//   block k of the estimate = sum_j R[k][j] g_j
//                           = sum_i sum_k' (R[:, S_i] B^(i)[S_i, :])[k][k'] g_{D_i}[k']
// and R[:, S_i] B^(i)[S_i, :] = X X^+ with X = R[:, S_i]: the identity when
// Delta_i >= ell (every decodable chunk passes through unchanged), the
// orthogonal projection onto range(X) when 0 < Delta_i < ell, zero when
// Delta_i = 0.  So the estimate of all patterns is one dense contraction
//   ghat[(p, k)][x] = sum_{(i, k')} C[(p, k)][(i, k')] * g_i[k' L + x]
// with C [P*ell][N*ell] the per-pattern mixing matrices, run on the fp32
// matrix cores.  Reads G and C (small, L2-resident), writes the estimate.
//
//   mix_kernel      one wavefront per pattern, one lane per chunk: coverage and
//                   the ell x ell mixing block in fp64 (Cholesky of X^T X),
//                   rounded once to fp32 into C (row stride padded to Kp).
//   direct_kernel   128 x 128-tiled v_mfma_f32_32x32x2f32 GEMM of C and the
//                   block-split gradients; A tiles [row][k] in LDS, B tiles
//                   [k][col]; the estimate written with column guards.
//                   With a target it also sums each row's squared error over the
//                   tile's columns into per-(row, tile) fp64 partials.
//   direct_sqerr_kernel  adds the partials of each pattern in a fixed order.
#include "common.h"

namespace gcx {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kDM = 128, kDN = 128, kDK = 32, kDThreads = 256, kDPad = 4;

template <int ELL>
__device__ __forceinline__ void chol(double (&A)[ELL][ELL]) {
#pragma unroll
  for (int c = 0; c < ELL; ++c) {
    double s = A[c][c];
#pragma unroll
    for (int q = 0; q < c; ++q) s -= A[c][q] * A[c][q];
    const double dcc = sqrt(s);
    A[c][c] = dcc;
#pragma unroll
    for (int r = c + 1; r < ELL; ++r) {
      double v = A[r][c];
#pragma unroll
      for (int q = 0; q < c; ++q) v -= A[r][q] * A[c][q];
      A[r][c] = v / dcc;
    }
  }
}

template <int ELL>
__device__ __forceinline__ void chol_solve(const double (&Lf)[ELL][ELL], double (&b)[ELL]) {
#pragma unroll
  for (int r = 0; r < ELL; ++r) {
    double v = b[r];
#pragma unroll
    for (int q = 0; q < r; ++q) v -= Lf[r][q] * b[q];
    b[r] = v / Lf[r][r];
  }
#pragma unroll
  for (int r = ELL - 1; r >= 0; --r) {
    double v = b[r];
#pragma unroll
    for (int q = r + 1; q < ELL; ++q) v -= Lf[q][r] * b[q];
    b[r] = v / Lf[r][r];
  }
}

// C[(p*ell + k)*Kp + i*ell + k'] = (X X^+)[k][k'] for chunk i of pattern p.
template <int ELL>
__global__ __launch_bounds__(256) void mix_kernel(const int32_t *__restrict__ psi, int64_t P, int N,
                                                  int m, int delta, const int32_t *__restrict__ holder,
                                                  const int32_t *__restrict__ hpos, int gamma,
                                                  const float *__restrict__ R, int64_t Kp,
                                                  float *__restrict__ C) {
  const int lane = threadIdx.x % kWave;
  const int64_t p = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave;
  if (p >= P) return;
  const int32_t *ps = psi + p * m;
  float *Cp = C + p * ELL * Kp;
  for (int i = lane; i < N; i += kWave) {
    const int32_t *hi = holder + int64_t(i) * gamma;
    const int32_t *hp = hpos + int64_t(i) * gamma;
    int Delta = 0;
    int selj[ELL];
#pragma unroll
    for (int a = 0; a < ELL; ++a) selj[a] = 0;
    for (int u = 0; u < gamma; ++u) {
      const int j = hi[u], t = hp[u];
      if (j >= 0 && j < m && t >= 0 && t < delta && ps[j] > t) {
#pragma unroll
        for (int a = 0; a < ELL; ++a)
          if (a == Delta) selj[a] = j;
        ++Delta;
      }
    }
    double Mx[ELL][ELL];  // mixing block X X^+
#pragma unroll
    for (int k = 0; k < ELL; ++k)
#pragma unroll
      for (int kk = 0; kk < ELL; ++kk) Mx[k][kk] = (Delta >= ELL && k == kk) ? 1.0 : 0.0;
    if (Delta > 0 && Delta < ELL) {
      // X = R[:, S_i] (ell x Delta), H = X^T X padded with the identity, X X^+ = X H^-1 X^T
      double X[ELL][ELL];
#pragma unroll
      for (int a = 0; a < ELL; ++a)
#pragma unroll
        for (int k = 0; k < ELL; ++k) X[k][a] = a < Delta ? double(R[k * m + selj[a]]) : 0.0;
      double H[ELL][ELL];
#pragma unroll
      for (int a = 0; a < ELL; ++a)
#pragma unroll
        for (int b = 0; b < ELL; ++b) {
          double v = 0.0;
#pragma unroll
          for (int k = 0; k < ELL; ++k) v += X[k][a] * X[k][b];
          H[a][b] = (a < Delta && b < Delta) ? v : (a == b ? 1.0 : 0.0);
        }
      chol<ELL>(H);
#pragma unroll
      for (int kk = 0; kk < ELL; ++kk) {
        double z[ELL];  // H^-1 X^T e_kk
#pragma unroll
        for (int a = 0; a < ELL; ++a) z[a] = X[kk][a];
        chol_solve<ELL>(H, z);
#pragma unroll
        for (int k = 0; k < ELL; ++k) {
          double v = 0.0;
#pragma unroll
          for (int a = 0; a < ELL; ++a) v += X[k][a] * z[a];
          Mx[k][kk] = v;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < ELL; ++k)
#pragma unroll
      for (int kk = 0; kk < ELL; ++kk) Cp[k * Kp + int64_t(i) * ELL + kk] = float(Mx[k][kk]);
  }
  // zero the padding columns of this pattern's rows
  for (int64_t c = int64_t(N) * ELL + lane; c < Kp; c += kWave)
#pragma unroll
    for (int k = 0; k < ELL; ++k) Cp[k * Kp + c] = 0.f;
}

template <typename GT>
__device__ __forceinline__ float gval(const GT *p);
template <>
__device__ __forceinline__ float gval<float>(const float *p) { return *p; }
template <>
__device__ __forceinline__ float gval<uint16_t>(const uint16_t *p) { return bf16_to_f32(*p); }

// ghat[p*d + k*L + x] = sum_c C[(p*ell + k)*Kp + c] * G_blk[c][x],
// G_blk[i*ell + k'][x] = g_i[k'*L + x] (zero past d).  With part != NULL the block also
// writes part[r*ntiles + nt] = sum over its columns of (ghat[r][x] - gsum[k*L + x])^2 (fp64).
constexpr int kDLdsA = 2 * kDM * (kDK + kDPad), kDLdsB = 2 * kDK * (kDN + 4);
constexpr int kDRedStride = 2 * 32 + 1;  // doubles per row of the error reduction
static_assert((kDLdsA + kDLdsB) * 4 >= kDM * kDRedStride * 8, "reduction fits the tile buffers");

template <typename GT, bool VEC4, int ELL>
__global__ __launch_bounds__(kDThreads, 2) void direct_kernel(const float *__restrict__ C,
                                                               const GT *__restrict__ G, int N,
                                                               int64_t d, int64_t L,
                                                               int64_t Kp, int64_t rows,
                                                               int64_t ntiles,
                                                               float *__restrict__ ghat,
                                                               const float *__restrict__ gsum,
                                                               double *__restrict__ part) {
  __shared__ __align__(16) float smem[kDLdsA + kDLdsB];
  auto As = reinterpret_cast<float(*)[kDM][kDK + kDPad]>(smem);
  auto Bs = reinterpret_cast<float(*)[kDK][kDN + 4]>(smem + kDLdsA);
  // consecutive blocks take the column tiles of one row tile of C
  const int64_t nt = blockIdx.x % ntiles;
  const int64_t mt = blockIdx.x / ntiles;
  const int t = threadIdx.x, lane = t % kWave, wave = t / kWave;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, li = lane & 31;
  const int K = N * ELL;
  const int arow = t >> 3, ak = (t & 7) * 4;   // A loader: 8 threads per row, 32 rows per pass
  const int brow = t >> 5, bc = (t & 31) * 4;  // B loader: 32 threads per row, 8 rows per pass

  float4 ra[4], rb[4];
  auto gload = [&](int64_t kb) {
#pragma unroll
    for (int p4 = 0; p4 < 4; ++p4) {
      const int64_t r = mt * kDM + arow + 32 * p4;
      ra[p4] = r < rows ? *reinterpret_cast<const float4 *>(C + r * Kp + kb + ak)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
      const int c = int(kb) + brow + 8 * p4;  // (chunk, block) index
      const int64_t x = nt * kDN + bc;
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (c < K) {
        const int i = c / ELL, kk = c % ELL;
        const int64_t col = kk * L + x;
        const GT *src = G + int64_t(i) * d + col;
        if (VEC4 && x + 3 < L && col + 3 < d) {
          if constexpr (sizeof(GT) == 4) {
            const float4 f = *reinterpret_cast<const float4 *>(src);
            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
          } else {
            const uint2 u = *reinterpret_cast<const uint2 *>(src);
            v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
            v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (x + e < L && col + e < d) v[e] = gval<GT>(src + e);
        }
      }
      rb[p4] = make_float4(v[0], v[1], v[2], v[3]);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int p4 = 0; p4 < 4; ++p4) {
      *reinterpret_cast<float4 *>(&As[buf][arow + 32 * p4][ak]) = ra[p4];
      *reinterpret_cast<float4 *>(&Bs[buf][brow + 8 * p4][bc]) = rb[p4];
    }
  };

  v16f acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.f;

  const int64_t nst = Kp / kDK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int64_t st = 0; st < nst; ++st) {
    const int buf = int(st & 1);
    if (st + 1 < nst) gload((st + 1) * kDK);
    // lane half h takes k in [16h, 16h + 16) of the stage; both operands of one MFMA
    // come from the same k in each half
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      float4 a[2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
        a[mb] = *reinterpret_cast<const float4 *>(&As[buf][wm * 64 + mb * 32 + li][h * 16 + s4 * 4]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int kk = h * 16 + s4 * 4 + e;
        float bv[2];
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) bv[nb] = Bs[buf][kk][wn * 64 + nb * 32 + li];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          const float av = e == 0 ? a[mb].x : (e == 1 ? a[mb].y : (e == 2 ? a[mb].z : a[mb].w));
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv[nb], acc[mb][nb], 0, 0, 0);
        }
      }
    }
    if (st + 1 < nst) lstore(buf ^ 1);
    __syncthreads();
  }

  // lane (h, li) of wave (wm, wn) holds rows wm*64 + mb*32 + 8*(v/4) + 4h + v%4, columns
  // wn*64 + nb*32 + li of the tile
  double *red = reinterpret_cast<double *>(smem);  // [kDM][kDRedStride], free after the loop
  const int64_t p0 = mt * kDM / ELL;                // pattern and block of the tile's first row
  const int k0 = int(mt * kDM % ELL);
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int rl = wm * 64 + mb * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
      const int64_t r = mt * kDM + rl;
      const int64_t p = p0 + (k0 + rl) / ELL;
      const int k = (k0 + rl) % ELL;
      double e2 = 0.0;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int64_t x = nt * kDN + wn * 64 + nb * 32 + li;
        const int64_t col = k * L + x;
        if (r < rows && x < L && col < d) {
          const float g = acc[mb][nb][v];
          if (ghat) __builtin_nontemporal_store(g, ghat + p * d + col);
          if (part) {
            const double e = double(g) - double(gsum[col]);
            e2 += e * e;
          }
        }
      }
      if (part) red[rl * kDRedStride + wn * 32 + li] = e2;
    }
  if (part) {
    __syncthreads();
    // two threads per row, 32 entries each, then the pair is added: a fixed order
    const int rl = t >> 1;
    const double *src = red + rl * kDRedStride + (t & 1) * 32;
    double s = 0.0;
#pragma unroll 8
    for (int c = 0; c < 32; ++c) s += src[c];
    s += __shfl_xor(s, 1, kWave);
    const int64_t r = mt * kDM + rl;
    if ((t & 1) == 0 && r < rows) part[r * ntiles + nt] = s;
  }
}

// sqerr[p] = sum over k < ell and column tiles of part, in a fixed order.
__global__ __launch_bounds__(256) void direct_sqerr_kernel(const double *__restrict__ part,
                                                            int64_t P, int ell, int64_t ntiles,
                                                            double *__restrict__ sqerr) {
  __shared__ double red[4];
  const int64_t p = blockIdx.x;
  const int64_t n = ell * ntiles;
  const double *src = part + p * n;
  double s = 0.0;
  for (int64_t c = threadIdx.x; c < n; c += 256) s += src[c];
  s = wave_sum(s);
  if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = s;
  __syncthreads();
  if (threadIdx.x == 0 && p < P) sqerr[p] = (red[0] + red[1]) + (red[2] + red[3]);
}

int64_t direct_kp(int N, int ell) { return ceil_div(int64_t(N) * ell, kDK) * kDK; }

// workspace: C [P*ell][Kp] fp32, then the error partials [P*ell][ntiles] fp64
size_t direct_c_bytes(int64_t P, int N, int ell) {
  return ceil_div(sizeof(float) * size_t(P) * ell * size_t(direct_kp(N, ell)), 256) * 256;
}

}  // namespace
}  // namespace gcx

extern "C" size_t gc_decode_direct_workspace_size(int64_t P, int32_t N, int64_t d, int32_t ell) {
  using namespace gcx;
  if (P < 1 || N < 1 || d < 1 || ell < 1 || ell > GC_MAX_ELL) return 0;
  const int64_t ntiles = ceil_div(ceil_div(d, ell), kDN);
  return direct_c_bytes(P, N, ell) + sizeof(double) * size_t(P) * ell * size_t(ntiles);
}

extern "C" int gc_decode_direct(const void *G, int32_t g_dtype, int32_t N, int64_t d,
                                const int32_t *psi, int64_t P, int32_t m, int32_t delta,
                                const int32_t *holder, const int32_t *hpos, int32_t gamma,
                                const float *R, int32_t ell, float *ghat, const float *gsum,
                                double *sqerr, void *workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  using namespace gcx;
  if (N < 1 || N > GC_MAX_M || d < 1 || P < 0 || m < 1 || m > GC_MAX_M || delta < 1 ||
      delta > GC_MAX_DELTA ||
      gamma < 1 || gamma > GC_MAX_DELTA || ell < 1 || ell > GC_MAX_ELL ||
      (g_dtype != GC_F32 && g_dtype != GC_BF16))
    return GC_EINVAL;
  if (P == 0) return GC_OK;
  if (!G || !psi || !holder || !hpos || !R || !workspace) return GC_EINVAL;
  if (!ghat && !sqerr) return GC_EINVAL;
  if (sqerr && !gsum) return GC_EINVAL;
  if (workspace_bytes < gc_decode_direct_workspace_size(P, N, d, ell) || !aligned16(workspace))
    return GC_EINVAL;
  const int64_t L = ceil_div(d, ell);
  const int64_t Kp = direct_kp(N, ell);
  const int64_t rows = P * ell;
  const int64_t ntiles = ceil_div(L, kDN);
  const int64_t blocks = ceil_div(rows, kDM) * ntiles;
  if (!grid_ok(blocks, kDThreads) || !grid_ok(ceil_div(P, 4), 256) || !grid_ok(P, 256))
    return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  float *Cm = static_cast<float *>(workspace);
  double *part = sqerr ? reinterpret_cast<double *>(static_cast<char *>(workspace) +
                                                    direct_c_bytes(P, N, ell))
                       : nullptr;
  (void)hipGetLastError();
  switch (ell) {
#define GC_CASE(E)                                                                                 \
  case E:                                                                                          \
    hipLaunchKernelGGL(mix_kernel<E>, dim3(unsigned(ceil_div(P, 4))), dim3(256), 0, stream, psi, P, \
                       N, m, delta, holder, hpos, gamma, R, Kp, Cm);                               \
    break;
    GC_CASE(1) GC_CASE(2) GC_CASE(3) GC_CASE(4) GC_CASE(5) GC_CASE(6) GC_CASE(7) GC_CASE(8)
#undef GC_CASE
    default: return GC_EINVAL;
  }
  const size_t es = g_dtype == GC_F32 ? 4 : 2;
  const bool vec4 = d % 4 == 0 && L % 4 == 0 && (reinterpret_cast<uintptr_t>(G) % (4 * es)) == 0;
  const dim3 grid{static_cast<uint32_t>(blocks)};
  const bool f32 = g_dtype == GC_F32;
#define GC_DIRECT(GT, V, E)                                                                        \
  hipLaunchKernelGGL((direct_kernel<GT, V, E>), grid, dim3(kDThreads), 0, stream, Cm,              \
                     static_cast<const GT *>(G), N, d, L, Kp, rows, ntiles, ghat, gsum, part)
#define GC_DIRECT_ELL(E)                                                                           \
  case E:                                                                                          \
    if (f32) {                                                                                     \
      if (vec4) GC_DIRECT(float, true, E); else GC_DIRECT(float, false, E);                        \
    } else {                                                                                       \
      if (vec4) GC_DIRECT(uint16_t, true, E); else GC_DIRECT(uint16_t, false, E);                  \
    }                                                                                              \
    break;
  switch (ell) {
    GC_DIRECT_ELL(1) GC_DIRECT_ELL(2) GC_DIRECT_ELL(3) GC_DIRECT_ELL(4)
    GC_DIRECT_ELL(5) GC_DIRECT_ELL(6) GC_DIRECT_ELL(7) GC_DIRECT_ELL(8)
    default: return GC_EINVAL;
  }
#undef GC_DIRECT_ELL
#undef GC_DIRECT
  if (sqerr)
    hipLaunchKernelGGL(direct_sqerr_kernel, dim3(unsigned(P)), dim3(256), 0, stream, part, P, ell,
                       ntiles, sqerr);
  return launch_status();
}
