// gc_decode_coeffs: coverage, decodability, coefficient error and the
// encoding coefficients of Algorithm 1 (Find-Encoding-Coeff), batched over
// straggler patterns.  One wavefront per pattern, one lane per chunk.
//
// For chunk i with processed holders S_i (Delta = |S_i|) and X = R[:, S_i]
// (ell x Delta), Algorithm 1's minimum-norm least-squares coefficients are
// the rows of pinv(X) (the Frobenius objective separates per column, Sec. 2.1
// and the W_5 example of Sec. 2.2).  Each lane forms them in fp64 from the
// smaller Gram matrix:
//   Delta >= ell:  M = X X^T (ell x ell),  row j of pinv(X) = (M^-1 x_j)^T
//   Delta <  ell:  H = X^T X (Delta x Delta, padded with the identity to
//                  ell x ell),  pinv(X) = H^-1 X^T
// with a Cholesky factorisation of M or H.  ell = 1 reduces to Remark 1:
// coefficient R_j / sum_{S_i} R^2.  Coverage and decodability are integer
// decisions and never depend on the floating-point solve.
#include <algorithm>

#include "common.h"
#include "small_solve.h"

namespace gcx {
namespace {

constexpr int kDecodeThreads = 256;
constexpr int kDecodeWaves = kDecodeThreads / kWave;

// Coefficients are written once and read only by later calls: non-temporal stores (measured
// 15% faster for the 1.6 GB of coefficients of 100,000 patterns at m = 200, delta = 20 than
// plain ones).  Coverage rows (4N bytes per pattern, not whole cache lines) stay plain:
// non-temporal stores of them measured slower.
__device__ __forceinline__ void st_nt(float *p, float v) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ void st_nt4(float *p, float a, float b, float c, float d) {
  typedef float v4f_ __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(v4f_{a, b, c, d}, reinterpret_cast<v4f_ *>(p));
}

// One pattern by one wavefront, one lane per chunk: coverage, decodability, coefficient
// error and the chunk's coefficients written straight to their (worker, position) slots.
template <int ELL>
__device__ __forceinline__ void decode_one(const int32_t *__restrict__ psi, int64_t p, int N, int m,
                                           const int32_t *__restrict__ order, int delta,
                                           const int32_t *__restrict__ holder, const int32_t *__restrict__ hpos,
                                           int gamma, const float *__restrict__ Rs, int32_t *__restrict__ cov,
                                           uint8_t *__restrict__ dec, int32_t *__restrict__ coef_err,
                                           float *__restrict__ Bc, int lane) {
  const int32_t *ps = psi + p * m;
  const int64_t wstride = int64_t(delta) * ELL;       // floats per worker in Bc
  const bool want_bc = Bc != nullptr;                  // else coverage only
  float *Bp = want_bc ? Bc + p * int64_t(m) * wstride : nullptr;

  // psi_j must lie in [0, delta_j]; padded order slots get zero coefficients.
  bool bad = false;
  for (int j = lane; j < m; j += kWave) {
    int load = 0;
    for (int t = 0; t < delta; ++t) {
      const int c = order[int64_t(j) * delta + t];
      if (c >= 0 && c < N) {
        ++load;
      } else if (want_bc) {
#pragma unroll
        for (int k = 0; k < ELL; ++k) st_nt(Bp + j * wstride + t * ELL + k, 0.f);
      }
    }
    const int v = ps[j];
    bad = bad || v < 0 || v > load;
  }
  const bool invalid = __any(bad);

  int err = 0;
  bool all_ok = true;
  for (int i = lane; i < N; i += kWave) {
    const int32_t *hi = holder + int64_t(i) * gamma;
    const int32_t *hp = hpos + int64_t(i) * gamma;
    // W_j processed chunk i iff chunk i sits at a position t < psi_j of W_j
    int Delta = 0;
    for (int u = 0; u < gamma; ++u) {
      const int j = hi[u], t = hp[u];
      if (j >= 0 && j < m && t >= 0 && t < delta && ps[j] > t) ++Delta;
    }
    if (cov != nullptr) cov[p * N + i] = Delta;
    err += Delta < ELL ? ELL - Delta : 0;
    all_ok = all_ok && Delta >= ELL;
    if (!want_bc) continue;

    if (Delta == 0 || invalid) {
      for (int u = 0; u < gamma; ++u) {
        const int j = hi[u], t = hp[u];
        if (j >= 0 && j < m && t >= 0 && t < delta) {
#pragma unroll
          for (int k = 0; k < ELL; ++k) st_nt(Bp + j * wstride + t * ELL + k, 0.f);
        }
      }
      continue;
    }

    if constexpr (ELL == 1) {
      double ss = 0.0;
      for (int u = 0; u < gamma; ++u) {
        const int j = hi[u], t = hp[u];
        if (j >= 0 && j < m && t >= 0 && t < delta && ps[j] > t) {
          const double x = Rs[j];
          ss += x * x;
        }
      }
      for (int u = 0; u < gamma; ++u) {
        const int j = hi[u], t = hp[u];
        if (j >= 0 && j < m && t >= 0 && t < delta)
          st_nt(Bp + j * wstride + t, ps[j] > t ? float(double(Rs[j]) / ss) : 0.f);
      }
    } else if (Delta >= ELL) {
      // M = X X^T, lower triangle
      double M[ELL][ELL];
#pragma unroll
      for (int a = 0; a < ELL; ++a)
#pragma unroll
        for (int b = 0; b < ELL; ++b) M[a][b] = 0.0;
      for (int u = 0; u < gamma; ++u) {
        const int j = hi[u], t = hp[u];
        if (j >= 0 && j < m && t >= 0 && t < delta && ps[j] > t) {
          double x[ELL];
#pragma unroll
          for (int k = 0; k < ELL; ++k) x[k] = Rs[k * m + j];
#pragma unroll
          for (int a = 0; a < ELL; ++a)
#pragma unroll
            for (int b = 0; b <= a; ++b) M[a][b] += x[a] * x[b];
        }
      }
      cholesky<ELL>(M);
      for (int u = 0; u < gamma; ++u) {
        const int j = hi[u], t = hp[u];
        if (!(j >= 0 && j < m && t >= 0 && t < delta)) continue;
        float *dst = Bp + j * wstride + t * ELL;
        if (ps[j] > t) {
          double c[ELL];
#pragma unroll
          for (int k = 0; k < ELL; ++k) c[k] = Rs[k * m + j];
          chol_solve<ELL>(M, c);
#pragma unroll
          for (int k = 0; k < ELL; ++k) st_nt(dst + k, float(c[k]));
        } else {
#pragma unroll
          for (int k = 0; k < ELL; ++k) st_nt(dst + k, 0.f);
        }
      }
    } else {
      // 0 < Delta < ell: collect the members (at most ell - 1 of them)
      int selj[ELL], selt[ELL];
#pragma unroll
      for (int a = 0; a < ELL; ++a) selj[a] = selt[a] = -1;
      int cnt = 0;
      for (int u = 0; u < gamma; ++u) {
        const int j = hi[u], t = hp[u];
        if (!(j >= 0 && j < m && t >= 0 && t < delta)) continue;
        if (ps[j] > t) {
#pragma unroll
          for (int a = 0; a < ELL; ++a)
            if (a == cnt) {
              selj[a] = j;
              selt[a] = t;
            }
          ++cnt;
        } else {
#pragma unroll
          for (int k = 0; k < ELL; ++k) st_nt(Bp + j * wstride + t * ELL + k, 0.f);
        }
      }
      double X[ELL][ELL];  // X[k][a] = R[k][selj[a]], zero for a >= Delta
#pragma unroll
      for (int a = 0; a < ELL; ++a) {
        const int ja = a < Delta ? selj[a] : 0;  // index stays in range even if speculated
#pragma unroll
        for (int k = 0; k < ELL; ++k) X[k][a] = a < Delta ? double(Rs[k * m + ja]) : 0.0;
      }
      double H[ELL][ELL];
#pragma unroll
      for (int a = 0; a < ELL; ++a)
#pragma unroll
        for (int b = 0; b <= a; ++b) {
          double v = 0.0;
#pragma unroll
          for (int k = 0; k < ELL; ++k) v += X[k][a] * X[k][b];
          H[a][b] = (a < Delta) ? v : (a == b ? 1.0 : 0.0);
        }
      cholesky<ELL>(H);
#pragma unroll
      for (int a = 0; a < ELL; ++a) {
        if (a >= Delta) break;
        double z[ELL];  // column a of H^-1 (= row a, H symmetric)
#pragma unroll
        for (int b = 0; b < ELL; ++b) z[b] = (a == b) ? 1.0 : 0.0;
        chol_solve<ELL>(H, z);
        float *dst = Bp + selj[a] * wstride + selt[a] * ELL;
#pragma unroll
        for (int k = 0; k < ELL; ++k) {
          double c = 0.0;
#pragma unroll
          for (int b = 0; b < ELL; ++b) c += z[b] * X[k][b];
          st_nt(dst + k, float(c));
        }
      }
    }
  }

  err = wave_sum(err);
  const bool ok = __all(all_ok);
  if (lane == 0) {
    dec[p] = invalid ? GC_DEC_INVALID : (ok ? GC_DEC_YES : GC_DEC_NO);
    coef_err[p] = err;
  }
}

template <int ELL>
__global__ __launch_bounds__(kDecodeThreads) void decode_kernel(
    const int32_t *__restrict__ psi, int64_t P, int N, int m, const int32_t *__restrict__ order,
    int delta, const int32_t *__restrict__ holder, const int32_t *__restrict__ hpos, int gamma,
    const float *__restrict__ R, int32_t *__restrict__ cov, uint8_t *__restrict__ dec,
    int32_t *__restrict__ coef_err, float *__restrict__ Bc) {
  extern __shared__ float Rs[];  // [ELL][m]
  if (R != nullptr)
    for (int a = threadIdx.x; a < ELL * m; a += blockDim.x) Rs[a] = R[a];
  __syncthreads();  // the only barrier; every thread reaches it

  const int lane = threadIdx.x % kWave;
  const int64_t p = int64_t(blockIdx.x) * kDecodeWaves + threadIdx.x / kWave;
  if (p >= P) return;
  decode_one<ELL>(psi, p, N, m, order, delta, holder, hpos, gamma, Rs, cov, dec, coef_err, Bc, lane);
}

// Two-phase variant, used whenever the assignment tables fit in LDS.  A persistent block
// stages the tables transposed ([gamma][N], so lane i's holder reads are consecutive
// words) and each worker's load once; each wave then takes patterns in turn:
//   phase 1, one lane per chunk: coverage, and the fp64 factor of the chunk's small
//     system (ell = 1: sum_{S_i} R^2; Delta >= ell: Cholesky of X X^T; 0 < Delta < ell:
//     Cholesky of the padded X^T X and the members), kept in the wave's LDS region;
//   phase 2, one lane per coefficient row (j, t) in Bc order: the chunk order[j][t], and
//     the coefficients recomputed from the stored factor with the same operations as the
//     one-phase kernel, written contiguously.
// Both phases read psi from the wave's LDS copy.  Results equal decode_kernel's, except
// that at ell = 1 the coefficient R_j / sum R^2 is formed as R_j * (1 / sum R^2) in fp64
// before the fp32 rounding.
template <int ELL>
struct DecodeLayout {
  static constexpr int NF = ELL * (ELL + 1) / 2;  // packed lower triangle
  // words (4 bytes) of the block-shared part and of one wave's region
  // at ell = 1 with Bc the squares R_j^2 in fp64 [m + 1] (exact: fp32 squared fits fp64);
  // holder table [gamma][N] (worker | position << 16), loads [m], Rs [ELL][m] + a zero
  // for the sentinel worker m, and with Bc the order table [m][delta] as int16 (entries
  // past the chunks: the sentinel chunk N)
  __host__ __device__ static int64_t r2_words(int m, bool bc) {
    return (ELL == 1 && bc) ? 2 * int64_t(m + 1) : 0;
  }
  __host__ __device__ static int64_t shared_words(int N, int m, int gamma, int delta, bool bc) {
    const int64_t ord = bc ? (int64_t(m) * delta + 1) / 2 : 0;
    return (r2_words(m, bc) + int64_t(gamma) * N + m + int64_t(ELL) * m + 1 + ord + 3) & ~int64_t(3);
  }
  // F [N + 1][NF] doubles (row N: the sentinel chunk, zero), covS [N + 1], sel [N][ELL]
  // (ell > 1), psi [m + 1] (entry m: the sentinel worker)
  __host__ __device__ static int64_t wave_words(int N, int m, bool bc) {
    const int64_t f = bc ? 2 * int64_t(N + 1) * NF : 0;
    const int64_t sel = (bc && ELL > 1) ? int64_t(N) * ELL : 0;
    return (f + N + 1 + sel + m + 1 + 3) & ~int64_t(3);
  }
};

// Blocks of up to 16 waves while the per-lane solve is small, 4 beyond (more registers).
template <int ELL>
constexpr int decode_tiled_max_waves() { return ELL <= 4 ? 16 : 4; }

template <int ELL>
__global__ __launch_bounds__(decode_tiled_max_waves<ELL>() * 64)
__attribute__((amdgpu_waves_per_eu(ELL <= 2 ? 8 : 1))) void decode_tiled_kernel(
    const int32_t *__restrict__ psi, int64_t P, int N, int m, const int32_t *__restrict__ order,
    int delta, const int32_t *__restrict__ holder, const int32_t *__restrict__ hpos, int gamma,
    const float *__restrict__ R, int32_t *__restrict__ cov, uint8_t *__restrict__ dec,
    int32_t *__restrict__ coef_err, float *__restrict__ Bc) {
  using Lay = DecodeLayout<ELL>;
  constexpr int NF = Lay::NF;
  extern __shared__ __align__(16) int32_t sh[];
  const bool want_bc = Bc != nullptr;
  double *R2s = reinterpret_cast<double *>(sh);  // [m + 1] (ell = 1 with Bc)
  int32_t *hjt = sh + Lay::r2_words(m, want_bc);  // [gamma][N]: j | t << 16
  int32_t *loads = hjt + int64_t(gamma) * N;     // [m]
  float *Rs = reinterpret_cast<float *>(loads + m);  // [ELL][m] + 1
  int16_t *ordS = reinterpret_cast<int16_t *>(Rs + ELL * m + 1);  // [m][delta] (with Bc)
  // table entries outside [0, m) x [0, delta) point at the sentinel worker m, whose psi
  // entry is -1 (never past any position) and whose weight is 0
  for (int e = threadIdx.x; e < N * gamma; e += blockDim.x) {
    const int i = e / gamma, u = e % gamma;
    const int j = holder[e], t = hpos[e];
    const bool ok = j >= 0 && j < m && t >= 0 && t < delta;
    hjt[int64_t(u) * N + i] = ok ? (j | (t << 16)) : m;
  }
  for (int j = threadIdx.x; j < m; j += blockDim.x) {
    int load = 0;
    for (int t = 0; t < delta; ++t) {
      const int c = order[int64_t(j) * delta + t];
      load += (c >= 0 && c < N) ? 1 : 0;
    }
    loads[j] = load;
  }
  if (want_bc) {
    for (int a = threadIdx.x; a < ELL * m; a += blockDim.x) Rs[a] = R[a];
    if (threadIdx.x == 0) Rs[ELL * m] = 0.f;
    if (ELL == 1)
      for (int j = threadIdx.x; j <= m; j += blockDim.x) {
        const double x = j < m ? double(R[j]) : 0.0;
        R2s[j] = x * x;
      }
    for (int e = threadIdx.x; e < m * delta; e += blockDim.x) {
      const int c = order[e];
      ordS[e] = int16_t((c >= 0 && c < N) ? c : N);
    }
  }
  __syncthreads();  // the only block barrier; every thread reaches it

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  int32_t *region = sh + Lay::shared_words(N, m, gamma, delta, want_bc) +
                    int64_t(wave) * Lay::wave_words(N, m, want_bc);
  double *F = reinterpret_cast<double *>(region);                      // [N + 1][NF]
  int32_t *covS = region + (want_bc ? 2 * int64_t(N + 1) * NF : 0);    // [N + 1]
  int32_t *sel = covS + N + 1;                                          // [N][ELL] (ELL > 1)
  int32_t *pss = sel + ((want_bc && ELL > 1) ? int64_t(N) * ELL : 0);  // [m]
  const int64_t wstride = int64_t(delta) * ELL;
  // phase 2 walks e = lane, lane + 64, ... as (worker, position) = (e / delta, e % delta)
  const int j_first = lane / delta, t_first = lane % delta;
  const int j_step = kWave / delta, t_step = kWave % delta;
  if (want_bc && lane == 0) {  // the sentinel chunk: no coverage, zero coefficients
    covS[N] = 0;
#pragma unroll
    for (int a = 0; a < NF; ++a) F[int64_t(N) * NF + a] = 0.0;
  }

  for (int64_t p = int64_t(blockIdx.x) * nw + wave; p < P; p += int64_t(gridDim.x) * nw) {
    bool bad = false;
    for (int j = lane; j < m; j += kWave) {
      const int v = psi[p * m + j];
      pss[j] = v;
      bad = bad || v < 0 || v > loads[j];
    }
    if (lane == 0) pss[m] = -1;
    const bool invalid = __any(bad);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- phase 1: one lane per chunk
    int err = 0;
    bool all_ok = true;
    for (int i = lane; i < N; i += kWave) {
      int Delta = 0;
      double ss = 0.0;  // ell = 1: sum of R_j^2 over the members, in holder order
      if (ELL == 1 && want_bc) {
        // branch-free, every load unconditional (the sentinel worker m has psi -1 and
        // weight 0), so the unrolled holders' LDS reads overlap
#pragma unroll 4
        for (int u = 0; u < gamma; ++u) {
          const int jt = hjt[u * N + i], j = jt & 0xffff, t = jt >> 16;
          const int pv = pss[j];
          const double x2 = R2s[j];
          const bool member = pv > t;
          Delta += member ? 1 : 0;
          ss += member ? x2 : 0.0;
        }
      } else {
#pragma unroll 4
        for (int u = 0; u < gamma; ++u) {
          const int jt = hjt[u * N + i], j = jt & 0xffff, t = jt >> 16;
          Delta += pss[j] > t ? 1 : 0;
        }
      }
      if (cov != nullptr) cov[p * N + i] = Delta;
      err += Delta < ELL ? ELL - Delta : 0;
      all_ok = all_ok && Delta >= ELL;
      covS[i] = Delta;
      if (!want_bc) continue;
      double *Fi = F + int64_t(i) * NF;
      if constexpr (ELL == 1) {
        // phase 2 multiplies by the reciprocal (one rounding more than a division); zero
        // when nothing is covered or the pattern is invalid, so phase 2 writes zeros
        Fi[0] = (invalid || Delta == 0) ? 0.0 : 1.0 / ss;
        continue;
      }
      if (invalid || Delta == 0) continue;
      if constexpr (ELL == 1) {
      } else if (Delta >= ELL) {
        double M[ELL][ELL];
#pragma unroll
        for (int a = 0; a < ELL; ++a)
#pragma unroll
          for (int b = 0; b < ELL; ++b) M[a][b] = 0.0;
        for (int u = 0; u < gamma; ++u) {
          const int jt = hjt[u * N + i], j = jt & 0xffff, t = jt >> 16;
          if (pss[j] > t) {
            double x[ELL];
#pragma unroll
            for (int k = 0; k < ELL; ++k) x[k] = Rs[k * m + j];
#pragma unroll
            for (int a = 0; a < ELL; ++a)
#pragma unroll
              for (int b = 0; b <= a; ++b) M[a][b] += x[a] * x[b];
          }
        }
        cholesky<ELL>(M);
#pragma unroll
        for (int a = 0; a < ELL; ++a)
#pragma unroll
          for (int b = 0; b <= a; ++b) Fi[a * (a + 1) / 2 + b] = M[a][b];
      } else {
        int selj[ELL];
#pragma unroll
        for (int a = 0; a < ELL; ++a) selj[a] = -1;
        int cnt = 0;
        for (int u = 0; u < gamma; ++u) {
          const int jt = hjt[u * N + i], j = jt & 0xffff, t = jt >> 16;
          if (pss[j] > t) {
#pragma unroll
            for (int a = 0; a < ELL; ++a)
              if (a == cnt) selj[a] = j;
            ++cnt;
          }
        }
        double X[ELL][ELL];
#pragma unroll
        for (int a = 0; a < ELL; ++a) {
          const int ja = a < Delta ? selj[a] : 0;
#pragma unroll
          for (int k = 0; k < ELL; ++k) X[k][a] = a < Delta ? double(Rs[k * m + ja]) : 0.0;
        }
        double H[ELL][ELL];
#pragma unroll
        for (int a = 0; a < ELL; ++a)
#pragma unroll
          for (int b = 0; b <= a; ++b) {
            double v = 0.0;
#pragma unroll
            for (int k = 0; k < ELL; ++k) v += X[k][a] * X[k][b];
            H[a][b] = (a < Delta) ? v : (a == b ? 1.0 : 0.0);
          }
        cholesky<ELL>(H);
#pragma unroll
        for (int a = 0; a < ELL; ++a) {
          sel[int64_t(i) * ELL + a] = selj[a];
#pragma unroll
          for (int b = 0; b <= a; ++b) Fi[a * (a + 1) / 2 + b] = H[a][b];
        }
      }
    }
    err = wave_sum(err);
    const bool ok = __all(all_ok);
    if (lane == 0) {
      dec[p] = invalid ? GC_DEC_INVALID : (ok ? GC_DEC_YES : GC_DEC_NO);
      coef_err[p] = err;
    }
    if (!want_bc) continue;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- phase 2: one lane per coefficient row (j, t), Bc order
    float *Bp = Bc + p * int64_t(m) * wstride;
    const int nrow = m * delta;
    if (ELL == 1 && delta >= 4 && (nrow & 3) == 0 && (reinterpret_cast<uintptr_t>(Bp) & 15) == 0) {
      // four consecutive rows per lane, one 16-byte store
      int j4 = (4 * lane) / delta, t4 = (4 * lane) % delta;
      const int j4_step = (4 * kWave) / delta, t4_step = (4 * kWave) % delta;
      for (int e0 = 4 * lane; (delta & 3) == 0 && e0 < nrow; e0 += 4 * kWave) {
        // delta a multiple of 4: the four rows are positions t4 .. t4 + 3 of one worker
        double f[4];  // zero for the sentinel chunk, Delta = 0, invalid
#pragma unroll
        for (int q = 0; q < 4; ++q) f[q] = F[ordS[e0 + q]];
        const int pv = pss[j4];
        const double r = Rs[j4];
        float o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float v = float(r * f[q]);
          o[q] = (pv > t4 + q && f[q] != 0.0) ? v : 0.f;
        }
        st_nt4(Bp + e0, o[0], o[1], o[2], o[3]);
        j4 += j4_step;
        t4 += t4_step;
        if (t4 >= delta) {
          t4 -= delta;
          ++j4;
        }
      }
      for (int e0 = 4 * lane; (delta & 3) != 0 && e0 < nrow; e0 += 4 * kWave) {
        // the four rows' (worker, position), then every LDS read, then the selects: no
        // branches, so the reads of the four rows overlap
        int jq[4], tq[4], cq[4];
        int jj = j4, tt = t4;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          jq[q] = jj;
          tq[q] = tt;
          cq[q] = ordS[e0 + q];
          if (++tt == delta) {
            tt = 0;
            ++jj;
          }
        }
        double f[4];  // zero for the sentinel chunk, Delta = 0, invalid
        int pv[4];
        float r[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          f[q] = F[cq[q]];
          pv[q] = pss[jq[q]];
          r[q] = Rs[jq[q]];
        }
        float o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float v = float(double(r[q]) * f[q]);
          o[q] = (pv[q] > tq[q] && f[q] != 0.0) ? v : 0.f;
        }
        st_nt4(Bp + e0, o[0], o[1], o[2], o[3]);
        j4 += j4_step;
        t4 += t4_step;
        if (t4 >= delta) {
          t4 -= delta;
          ++j4;
        }
      }
    } else {
      int j = j_first, t = t_first;
  #pragma unroll 4
      for (int e = lane; e < nrow; e += kWave) {
        const int c = ordS[e];
        float out[ELL];
  #pragma unroll
        for (int k = 0; k < ELL; ++k) out[k] = 0.f;
        const bool valid = c < N && pss[j] > t;
        if constexpr (ELL == 1) {
          if (valid && F[c] != 0.0) out[0] = float(double(Rs[j]) * F[c]);  // +0 otherwise
        }
        const int Delta = (ELL > 1 && valid) ? covS[c] : 0;
        if (ELL > 1 && !invalid && Delta > 0) {
          const double *Fc = F + int64_t(c) * NF;
          if constexpr (ELL == 1) {
          } else if (Delta >= ELL) {
            double Lf[ELL][ELL];
  #pragma unroll
            for (int a = 0; a < ELL; ++a)
  #pragma unroll
              for (int b = 0; b < ELL; ++b) Lf[a][b] = b <= a ? Fc[a * (a + 1) / 2 + b] : 0.0;
            double cc[ELL];
  #pragma unroll
            for (int k = 0; k < ELL; ++k) cc[k] = Rs[k * m + j];
            chol_solve<ELL>(Lf, cc);
  #pragma unroll
            for (int k = 0; k < ELL; ++k) out[k] = float(cc[k]);
          } else {
            double Lf[ELL][ELL];
  #pragma unroll
            for (int a = 0; a < ELL; ++a)
  #pragma unroll
              for (int b = 0; b < ELL; ++b) Lf[a][b] = b <= a ? Fc[a * (a + 1) / 2 + b] : 0.0;
            int selj[ELL];
            int me = 0;  // j's place among the members
  #pragma unroll
            for (int a = 0; a < ELL; ++a) {
              selj[a] = sel[int64_t(c) * ELL + a];
              if (a < Delta && selj[a] == j) me = a;
            }
            double X[ELL][ELL];
  #pragma unroll
            for (int a = 0; a < ELL; ++a) {
              const int ja = a < Delta ? selj[a] : 0;
  #pragma unroll
              for (int k = 0; k < ELL; ++k) X[k][a] = a < Delta ? double(Rs[k * m + ja]) : 0.0;
            }
            double z[ELL];
  #pragma unroll
            for (int b = 0; b < ELL; ++b) z[b] = (me == b) ? 1.0 : 0.0;
            chol_solve<ELL>(Lf, z);
  #pragma unroll
            for (int k = 0; k < ELL; ++k) {
              double v = 0.0;
  #pragma unroll
              for (int b = 0; b < ELL; ++b) v += z[b] * X[k][b];
              out[k] = float(v);
            }
          }
        }
  #pragma unroll
        for (int k = 0; k < ELL; ++k) st_nt(Bp + int64_t(e) * ELL + k, out[k]);
        j += j_step;
        t += t_step;
        if (t >= delta) {
          t -= delta;
          ++j;
        }
      }
    }
    // the next pattern overwrites this wave's region only after every lane is done with it
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// ell = 1 with coefficients, N = m and gamma = delta: the cyclic assignment is checked
// entry by entry on the device (chunk i held by worker (i - u) mod N at position u, worker j
// holding chunk (j + t) mod N at position t) and, when it holds, each wave runs the
// pattern with the tables replaced by index arithmetic.  psi and the squares R_j^2 are laid
// out extended around the cycle (entry k holds worker (k - delta) mod N), so holder u of
// chunk i sits at entry i - u + delta, and the reciprocals 1 / sum R^2 too (entry k holds
// chunk k mod N), so position t of worker j reads entry j + t: no table reads, no modulo.
// The arithmetic is the tiled kernel's (sum of R^2 over the holders in fp64, the
// reciprocal, R_j times it in fp64, one rounding to fp32), with the holders summed in
// ascending cyclic order (the tables' ascending worker order except for the chunks whose
// holders wrap past worker N - 1).  Other tables: the one-phase path, per wave.
//   LDS: R2x [m + delta] fp64, Rs [m] (+ pad); per wave F [N + delta] fp64, psi [m + delta].
constexpr int kCycMaxWaves = 16;

__host__ __device__ inline int64_t cyc_shared_bytes(int m, int delta) {
  return ((8 * int64_t(m + delta) + 4 * int64_t(m)) + 15) & ~int64_t(15);
}
// per wave: the reciprocals F [N + delta] fp64 and psi extended [m + delta]
__host__ __device__ inline int64_t cyc_wave_bytes(int N, int m, int delta) {
  return ((8 * int64_t(N + delta) + 4 * int64_t(m + delta)) + 15) & ~int64_t(15);
}

__device__ __forceinline__ void decode_cyclic_l1(const int32_t *__restrict__ psi, int64_t p, int N, int delta,
                                                 const double *__restrict__ R2x,
                                                 const float *__restrict__ Rs, int32_t *pss, double *F,
                                                 int32_t *__restrict__ cov, uint8_t *__restrict__ dec,
                                                 int32_t *__restrict__ coef_err, float *__restrict__ Bc,
                                                 int lane) {
  const int m = N;
  bool bad = false;
  for (int j = lane; j < m; j += kWave) {
    const int v = psi[p * m + j];
    pss[j + delta] = v;
    if (j >= m - delta) pss[j - (m - delta)] = v;
    bad = bad || v < 0 || v > delta;
  }
  const bool invalid = __any(bad);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // phase 1, one lane per chunk: coverage and the reciprocal of sum_{S_i} R^2
  int err = 0;
  bool all_ok = true;
  for (int i = lane; i < N; i += kWave) {
    int Delta = 0;
    double ss = 0.0;
    // holders in ascending cyclic order: worker i - delta + 1 + v (entry i + 1 + v) at
    // position delta - 1 - v
    const int32_t *pc = pss + i + 1;
    const double *rc = R2x + i + 1;
#pragma unroll 4
    for (int v = 0; v < delta; ++v) {
      const int pv = pc[v];
      const double x2 = rc[v];
      const bool member = pv > delta - 1 - v;
      Delta += member ? 1 : 0;
      ss += member ? x2 : 0.0;
    }
    if (cov != nullptr) cov[p * N + i] = Delta;
    err += Delta < 1 ? 1 : 0;
    all_ok = all_ok && Delta >= 1;
    const double f = (invalid || Delta == 0) ? 0.0 : 1.0 / ss;
    F[i] = f;
    if (i < delta) F[i + N] = f;
  }
  err = wave_sum(err);
  const bool ok = __all(all_ok);
  if (lane == 0) {
    dec[p] = invalid ? GC_DEC_INVALID : (ok ? GC_DEC_YES : GC_DEC_NO);
    coef_err[p] = err;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // phase 2, four consecutive coefficient rows per lane (worker j, positions t .. t + 3,
  // reciprocals at F[j + t ..]); zero past the processed prefix.  A position inside the
  // prefix always has a covered chunk (its own worker processed it), so its reciprocal is
  // set; an invalid pattern writes zeros throughout (wave-uniform).
  float *Bp = Bc + p * int64_t(m) * delta;
  const int nrow = m * delta;
  if (invalid) {
    for (int e = lane; e < nrow; e += kWave) st_nt(Bp + e, 0.f);
  } else if ((delta & 3) == 0 && (reinterpret_cast<uintptr_t>(Bp) & 15) == 0) {
    int j4 = (4 * lane) / delta, t4 = (4 * lane) % delta;
    const int j4_step = (4 * kWave) / delta, t4_step = (4 * kWave) % delta;
    for (int e0 = 4 * lane; e0 < nrow; e0 += 4 * kWave) {
      const double *fr = F + j4 + t4;
      const int lim = pss[j4 + delta] - t4;  // positions t4 + q with q < lim are processed
      const double r = Rs[j4];
      // every F entry read here is set, so the four reads are unconditional (paired LDS
      // reads) and the prefix is applied as a bit mask
      uint32_t o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = __float_as_uint(float(r * fr[q])) & (q < lim ? ~0u : 0u);
      st_nt4(Bp + e0, __uint_as_float(o[0]), __uint_as_float(o[1]), __uint_as_float(o[2]), __uint_as_float(o[3]));
      j4 += j4_step;
      t4 += t4_step;
      if (t4 >= delta) {
        t4 -= delta;
        ++j4;
      }
    }
  } else {
    int j = lane / delta, t = lane % delta;
    const int j_step = kWave / delta, t_step = kWave % delta;
    for (int e = lane; e < nrow; e += kWave) {
      const uint32_t v = __float_as_uint(float(double(Rs[j]) * F[j + t]));
      st_nt(Bp + e, __uint_as_float(v & (pss[j + delta] > t ? ~0u : 0u)));
      j += j_step;
      t += t_step;
      if (t >= delta) {
        t -= delta;
        ++j;
      }
    }
  }
  // the next pattern overwrites this wave's arrays only after every lane is done with them
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__global__ __launch_bounds__(kCycMaxWaves * 64) __attribute__((amdgpu_waves_per_eu(8))) void
decode_cyclic_l1_kernel(const int32_t *__restrict__ psi, int64_t P, int N, int m,
                        const int32_t *__restrict__ order, int delta, const int32_t *__restrict__ holder,
                        const int32_t *__restrict__ hpos, int gamma, const float *__restrict__ R,
                        int32_t *__restrict__ cov, uint8_t *__restrict__ dec, int32_t *__restrict__ coef_err,
                        float *__restrict__ Bc) {
  extern __shared__ __align__(16) unsigned char lds_c[];
  double *R2x = reinterpret_cast<double *>(lds_c);       // [m + delta]
  float *Rs = reinterpret_cast<float *>(R2x + m + delta);  // [m]
  // chunk i: its gamma = delta holders are the workers (i - t) mod N at positions t, in any
  // order (gc_assign lists them by ascending worker)
  bool cyc = N == m && gamma == delta && delta <= 64;
  for (int i = threadIdx.x; i < N && cyc; i += blockDim.x) {
    unsigned long long seen = 0;
    for (int u = 0; u < gamma; ++u) {
      const int j = holder[int64_t(i) * gamma + u], t = hpos[int64_t(i) * gamma + u];
      const bool ok = t >= 0 && t < delta && j == (i - t + N) % N;
      cyc = cyc && ok;
      if (ok) seen |= 1ull << t;
    }
    cyc = cyc && seen == (delta == 64 ? ~0ull : (1ull << delta) - 1);
  }
  for (int e = threadIdx.x; e < m * delta; e += blockDim.x)
    cyc = cyc && order[e] == (e / delta + e % delta) % N;
  for (int k = threadIdx.x; k < m + delta; k += blockDim.x) {
    const double x = double(R[((k - delta) % m + m) % m]);
    R2x[k] = x * x;
  }
  for (int j = threadIdx.x; j < m; j += blockDim.x) Rs[j] = R[j];
  const bool all_cyc = __syncthreads_and(cyc ? 1 : 0) != 0;  // the only block barrier

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  unsigned char *region = lds_c + cyc_shared_bytes(m, delta) + size_t(wave) * cyc_wave_bytes(N, m, delta);
  double *F = reinterpret_cast<double *>(region);                    // [N + delta]
  int32_t *pss = reinterpret_cast<int32_t *>(F + N + delta);         // [m + delta]
  for (int64_t p = int64_t(blockIdx.x) * nw + wave; p < P; p += int64_t(gridDim.x) * nw) {
    if (all_cyc)
      decode_cyclic_l1(psi, p, N, delta, R2x, Rs, pss, F, cov, dec, coef_err, Bc, lane);
    else
      decode_one<1>(psi, p, N, m, order, delta, holder, hpos, gamma, Rs, cov, dec, coef_err, Bc, lane);
  }
}

constexpr size_t kDecodeLdsCU = 160 * 1024;  // LDS of one CU

// the cyclic ell = 1 kernel when its LDS leaves at least 8 waves per CU; false otherwise
bool launch_decode_cyclic_l1(const int32_t *psi, int64_t P, int N, int m, const int32_t *order, int delta,
                             const int32_t *holder, const int32_t *hpos, int gamma, const float *R,
                             int32_t *cov, uint8_t *dec, int32_t *coef_err, float *Bc, hipStream_t st,
                             bool *launched) {
  *launched = false;
  const size_t shared = size_t(cyc_shared_bytes(m, delta)), per_wave = size_t(cyc_wave_bytes(N, m, delta));
  int best_w = 0, best_total = 0;
  for (int w = kCycMaxWaves; w >= 1; w >>= 1) {
    const size_t lds = shared + w * per_wave;
    if (lds > kDecodeLdsCU) continue;
    const int per_cu = int(std::min<size_t>(kDecodeLdsCU / lds, 32 / w));
    if (per_cu * w > best_total) {
      best_total = per_cu * w;
      best_w = w;
    }
  }
  if (best_total < 8) return true;
  const size_t lds = shared + best_w * per_wave;
  const int64_t blocks = std::min(ceil_div(P, best_w), int64_t(best_total / best_w) * cu_count());
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(reinterpret_cast<const void *>(&decode_cyclic_l1_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
    return false;
  hipLaunchKernelGGL(decode_cyclic_l1_kernel, dim3(unsigned(blocks)), dim3(best_w * kWave), lds, st, psi, P,
                     N, m, order, delta, holder, hpos, gamma, R, cov, dec, coef_err, Bc);
  *launched = true;
  return true;
}

template <int ELL>
bool launch_decode(const int32_t *psi, int64_t P, int N, int m, const int32_t *order, int delta,
                   const int32_t *holder, const int32_t *hpos, int gamma, const float *R,
                   int32_t *cov, uint8_t *dec, int32_t *coef_err, float *Bc, hipStream_t st) {
  using Lay = DecodeLayout<ELL>;
  const bool bc = Bc != nullptr;
  if (ELL == 1 && bc && N == m && gamma == delta) {
    bool launched = false;
    if (!launch_decode_cyclic_l1(psi, P, N, m, order, delta, holder, hpos, gamma, R, cov, dec, coef_err, Bc,
                                 st, &launched))
      return false;
    if (launched) return true;
  }
  const size_t shared = 4 * size_t(Lay::shared_words(N, m, gamma, delta, bc));
  const size_t per_wave = 4 * size_t(Lay::wave_words(N, m, bc));
  // the most waves per CU the LDS allows (at most 32), in blocks of up to 16 waves
  int best_w = 0, best_total = 0;
  for (int w = decode_tiled_max_waves<ELL>(); w >= 1; w >>= 1) {
    const size_t lds = shared + w * per_wave;
    if (lds > kDecodeLdsCU) continue;
    const int per_cu = int(std::min<size_t>(kDecodeLdsCU / lds, 32 / w));
    if (per_cu * w > best_total) {
      best_total = per_cu * w;
      best_w = w;
    }
  }
  // else the one-phase kernel, which needs no LDS per wave (the two-phase kernel's order
  // table holds chunk indices as int16)
  if (best_total >= 8 && N < 32768) {
    const size_t lds = shared + best_w * per_wave;
    const int64_t want = ceil_div(P, best_w);
    const int64_t resident = int64_t(best_total / best_w) * cu_count();
    const int64_t blocks = std::min(want, resident);
    if (lds > 64 * 1024 &&
        hipFuncSetAttribute(reinterpret_cast<const void *>(&decode_tiled_kernel<ELL>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
      return false;
    hipLaunchKernelGGL(decode_tiled_kernel<ELL>, dim3(unsigned(blocks)), dim3(best_w * kWave), lds,
                       st, psi, P, N, m, order, delta, holder, hpos, gamma, R, cov, dec, coef_err, Bc);
    return true;
  }
  const int64_t blocks = ceil_div(P, kDecodeWaves);
  const size_t lds = sizeof(float) * ELL * m;
  hipLaunchKernelGGL(decode_kernel<ELL>, dim3(unsigned(blocks)), dim3(kDecodeThreads), lds, st,
                     psi, P, N, m, order, delta, holder, hpos, gamma, R, cov, dec, coef_err, Bc);
  return true;
}

}  // namespace
}  // namespace gcx

extern "C" int gc_decode_coeffs(const int32_t *psi, int64_t P, int32_t N, int32_t m,
                                const int32_t *order, int32_t delta, const int32_t *holder,
                                const int32_t *hpos, int32_t gamma, const float *R, int32_t ell,
                                int32_t *cov, uint8_t *dec, int32_t *coef_err, float *Bc,
                                hipStream_t stream) {
  using namespace gcx;
  if (P < 0 || N < 1 || m < 1 || m > GC_MAX_M || delta < 1 || delta > GC_MAX_DELTA ||
      gamma < 1 || gamma > GC_MAX_DELTA || ell < 1 || ell > GC_MAX_ELL)
    return GC_EINVAL;
  // psi [P][m], cov [P][N], Bc [P][m][delta][ell]
  if (!sizes_ok({P, m, delta, ell}) || !sizes_ok({P, N}) || !sizes_ok({N, gamma})) return GC_EINVAL;
  if (P == 0) return GC_OK;
  if (!grid_ok(ceil_div(P, kDecodeWaves), kDecodeThreads)) return GC_EINVAL;
  if (!psi || !order || !holder || !hpos || !dec || !coef_err) return GC_EINVAL;
  if (Bc && !R) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  (void)hipGetLastError();
  switch (ell) {
#define GC_CASE(E)                                                                              \
  case E:                                                                                       \
    if (!launch_decode<E>(psi, P, N, m, order, delta, holder, hpos, gamma, R, cov, dec, coef_err, \
                          Bc, stream))                                                          \
      return GC_ELAUNCH;                                                                        \
    break;
    GC_CASE(1) GC_CASE(2) GC_CASE(3) GC_CASE(4) GC_CASE(5) GC_CASE(6) GC_CASE(7) GC_CASE(8)
#undef GC_CASE
    default: return GC_EINVAL;
  }
  return launch_status();
}
