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
//   direct_short_kernel  K = N*ell <= 64: persistent blocks walk 128 x 128 output
//                   tiles with the mixing rows resident in LDS and the next gradient
//                   tile prefetched into registers.
//   direct_kernel   any K: one 128 x 128 tile per block, k staged through
//                   double-buffered LDS.
//   Both run v_mfma_f32_32x32x2f32 with the gradients as first operand, so each
//   lane ends with runs of four positions of one estimate row: 16-byte stores,
//   and with a target the row's squared error over the tile (per-(row, tile)
//   fp64 partials) needs one cross-lane exchange.
//   direct_sqerr_kernel  adds the partials of each pattern in a fixed order.
#include <algorithm>

#include "common.h"
#include "small_solve.h"

namespace gcx {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kDM = 128, kDN = 128, kDK = 32, kDThreads = 256, kDPad = 4;

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
      cholesky<ELL>(H);
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

typedef float v4f __attribute__((ext_vector_type(4)));

// Four gradient entries G_blk[c][x .. x+3], G_blk[i*ell + k'][x] = g_i[k'*L + x], zero past
// the block (x >= L) or the gradient (k'*L + x >= d) and for c >= K.
template <typename GT, bool VEC4, int ELL>
__device__ __forceinline__ float4 gload4(const GT *__restrict__ G, int K, int64_t d, int64_t L,
                                         int c, int64_t x) {
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (c < K) {
    const int i = c / ELL, kk = c % ELL;
    const int64_t col = kk * L + x;
    const GT *src = G + int64_t(i) * d + col;
    if (VEC4) {  // d and L multiples of 4, G aligned: all four in or all four out
      if (x < L && col < d) {
        if constexpr (sizeof(GT) == 4) {
          const float4 f = *reinterpret_cast<const float4 *>(src);
          v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
        } else {
          const uint2 u = *reinterpret_cast<const uint2 *>(src);
          v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
          v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (x + e < L && col + e < d) v[e] = gval<GT>(src + e);
    }
  }
  return make_float4(v[0], v[1], v[2], v[3]);
}

// The MFMAs take the gradient tile as their first operand and the mixing rows as their
// second, so they produce the transposed tile: lane (h, li) of acc[xb][rb] holds estimate
// row rb*32 + li (of the wave's 64 rows) at positions xb*32 + 8*(v/4) + 4h + v%4 (of the
// wave's 64 columns).  Each lane thus owns runs of four consecutive positions of one row:
// the estimate leaves as 16-byte stores, and a row's squared error over the wave's columns
// is a sum inside the lane plus one exchange between the lane halves.
//
// Writes the tile's estimate (if ghat) and, if red2, red2[wn][row] = squared error of the
// row over the wave's 64 columns: each difference, square and sum of four neighbours in
// fp32, the rest in fp64, in a fixed order.  gs = target tile [ELL][kDN] in LDS.
template <int ELL, bool VST>
__device__ __forceinline__ void direct_epilogue(const v16f (&acc)[2][2], int64_t mt, int64_t nt,
                                                int64_t rows, int64_t d, int64_t L,
                                                float *__restrict__ ghat, const float *gs,
                                                double (*red2)[kDM], int wm, int wn, int h,
                                                int li) {
  const int64_t p0 = mt * kDM / ELL;  // pattern and block of the tile's first row
  const int k0 = int(mt * kDM % ELL);
  const int64_t x0 = nt * kDN;
  const bool tail = (ELL - 1) * L + x0 + kDN > d;  // the tile reaches past d somewhere
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int rl = wm * 64 + rb * 32 + li;
    const int64_t p = p0 + (k0 + rl) / ELL;
    const int k = (k0 + rl) % ELL;
    // tile columns xl < lim lie inside the block (x < L) and the gradient (k*L + x < d);
    // -1 for a row past the last pattern
    const int lim = mt * kDM + rl < rows ? int(std::min<int64_t>(std::min(L, d - k * L) - x0, kDN)) : -1;
    float *row = ghat ? ghat + p * d + k * L + x0 : nullptr;
    const float *grow = gs + k * kDN;
    double rs = 0.0;
#pragma unroll
    for (int xb = 0; xb < 2; ++xb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int xl = wn * 64 + xb * 32 + 8 * g + 4 * h;
        const float e0 = acc[xb][rb][4 * g], e1 = acc[xb][rb][4 * g + 1];
        const float e2 = acc[xb][rb][4 * g + 2], e3 = acc[xb][rb][4 * g + 3];
        if (ghat) {
          // plain stores: a wave completes each 128-byte line of a row in eight 16-byte
          // pieces, which the L2 merges before writing back
          if constexpr (VST) {  // d, L multiples of 4, ghat aligned: all four in or all out
            if (xl < lim) *reinterpret_cast<v4f *>(row + xl) = v4f{e0, e1, e2, e3};
          } else {
            const float ev[4] = {e0, e1, e2, e3};
#pragma unroll
            for (int u = 0; u < 4; ++u)
              if (xl + u < lim) row[xl + u] = ev[u];
          }
        }
        if (red2) {
          // past the block (x >= L) both sides hold zero; the zero-padded tail of the last
          // block (k*L + x >= d) is not part of the estimate and is masked out
          const float4 t4 = *reinterpret_cast<const float4 *>(grow + xl);
          float d0 = e0 - t4.x, d1 = e1 - t4.y, d2 = e2 - t4.z, d3 = e3 - t4.w;
          if (tail) {
            d0 = xl < lim ? d0 : 0.f;
            d1 = xl + 1 < lim ? d1 : 0.f;
            d2 = xl + 2 < lim ? d2 : 0.f;
            d3 = xl + 3 < lim ? d3 : 0.f;
          }
          rs += double((d0 * d0 + d1 * d1) + (d2 * d2 + d3 * d3));
        }
      }
    if (red2) {
      const double o = __shfl_xor(rs, 32, kWave);
      if (h == 0) red2[wn][rl] = rs + o;
    }
  }
}

// Fills the target tile gs[k][x] = gsum[k*L + nt*kDN + x] (zero past the block or d).
template <int ELL>
__device__ __forceinline__ void load_target(const float *__restrict__ gsum, int64_t nt, int64_t d,
                                            int64_t L, float *gs, int t) {
  for (int e = t; e < ELL * kDN; e += kDThreads) {
    const int k = e / kDN;
    const int64_t x = nt * kDN + e % kDN, col = k * L + x;
    gs[e] = (x < L && col < d) ? gsum[col] : 0.f;
  }
}

// ghat[p*d + k*L + x] = sum_c C[(p*ell + k)*Kp + c] * G_blk[c][x] for any K, in k stages of
// kDK through double-buffered LDS; one 128 x 128 tile per block.  With part != NULL it also
// writes part[r*ntiles + nt] = the row's squared error over the tile's columns.
constexpr int kDLdsA = 2 * kDM * (kDK + kDPad), kDLdsB = 2 * kDK * (kDN + 4);

template <typename GT, bool VEC4, int ELL>
__global__ __launch_bounds__(kDThreads, 2) void direct_kernel(
    const float *__restrict__ C, const GT *__restrict__ G, int N, int64_t d, int64_t L, int64_t Kp,
    int64_t rows, int64_t ntiles, float *__restrict__ ghat,
    const float *__restrict__ gsum, double *__restrict__ part) {
  __shared__ __align__(16) float As[2][kDM][kDK + kDPad];
  __shared__ __align__(16) float Bs[2][kDK][kDN + 4];
  __shared__ __align__(16) float gs[ELL * kDN];
  __shared__ double red2[2][kDM];
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
      rb[p4] = gload4<GT, VEC4, ELL>(G, K, d, L, int(kb) + brow + 8 * p4, nt * kDN + bc);
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

  if (part) load_target<ELL>(gsum, nt, d, L, gs, t);
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
      for (int rbk = 0; rbk < 2; ++rbk)
        a[rbk] = *reinterpret_cast<const float4 *>(&As[buf][wm * 64 + rbk * 32 + li][h * 16 + s4 * 4]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int kk = h * 16 + s4 * 4 + e;
        float bv[2];
#pragma unroll
        for (int xb = 0; xb < 2; ++xb) bv[xb] = Bs[buf][kk][wn * 64 + xb * 32 + li];
#pragma unroll
        for (int rbk = 0; rbk < 2; ++rbk) {
          const float av = e == 0 ? a[rbk].x : (e == 1 ? a[rbk].y : (e == 2 ? a[rbk].z : a[rbk].w));
#pragma unroll
          for (int xb = 0; xb < 2; ++xb)
            acc[xb][rbk] = __builtin_amdgcn_mfma_f32_32x32x2f32(bv[xb], av, acc[xb][rbk], 0, 0, 0);
        }
      }
    }
    if (st + 1 < nst) lstore(buf ^ 1);
    __syncthreads();
  }

  direct_epilogue<ELL, VEC4>(acc, mt, nt, rows, d, L, ghat, gs, part ? red2 : nullptr, wm, wn, h, li);
  if (part) {
    __syncthreads();
    const int64_t r = mt * kDM + t;
    if (t < kDM && r < rows) part[r * ntiles + nt] = red2[0][t] + red2[1][t];
  }
}

// Short contractions (K = N*ell <= 64, padded to Kq, a multiple of 4): a persistent grid walks
// the (row tile, column tile) pairs in row-tile-major order, each block a contiguous range.
// The block's A rows (128 x Kq) stay in LDS while its row tile does not change; the next
// column tile of the gradients is loaded into registers while the current one is
// multiplied.  Lane half h takes k in [h*Kh, (h+1)*Kh), Kh = Kq/2, from LDS layouts whose
// two halves sit 32 banks apart, so the 64 lanes of a read hit 64 distinct banks.
constexpr int kSKMax = 64;                           // largest Kq of the short path
constexpr int kSAStride = 33;                        // words per A row of one half (odd)
constexpr int kSAHalf = kDM * kSAStride + 32;        // A half 1 starts 32 banks after half 0
constexpr int kSBHalf = (kSKMax / 2) * kDN + 32;     // likewise for B
constexpr int kSLds = 2 * kSAHalf + 2 * kSBHalf + GC_MAX_ELL * kDN;  // floats; + red2 below

template <typename GT, bool VEC4, int ELL>
__global__ __launch_bounds__(kDThreads, 2) void direct_short_kernel(
    const float *__restrict__ C, const GT *__restrict__ G, int N, int64_t d, int64_t L, int64_t Kp,
    int Kq, int64_t rows, int64_t ntiles, int64_t ntotal, float *__restrict__ ghat,
    const float *__restrict__ gsum, double *__restrict__ part) {
  __shared__ __align__(16) float smem[kSLds];
  __shared__ double red2[2][kDM];
  float *As = smem;                  // [2][kDM][kSAStride] (+ gap)
  float *Bs = smem + 2 * kSAHalf;    // [2][Kh][kDN] (+ gap)
  float *gs = Bs + 2 * kSBHalf;      // [ELL][kDN]
  const int t = threadIdx.x, lane = t % kWave, wave = t / kWave;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, li = lane & 31;
  const int K = N * ELL, Kh = Kq >> 1;
  const int64_t q0 = int64_t(blockIdx.x) * ntotal / gridDim.x;
  const int64_t q1 = int64_t(blockIdx.x + 1) * ntotal / gridDim.x;

  // B rows c = (t >> 5) + 8j, columns 4*(t & 31) .. +3; target entries t + 256j
  constexpr int kTgt = (ELL * kDN + kDThreads - 1) / kDThreads;
  float4 rb[kSKMax / 8];
  float rg[kTgt];
  auto prefetch = [&](int64_t q) {
    const int64_t nt = q % ntiles;
    const int64_t x = nt * kDN + (t & 31) * 4;
#pragma unroll
    for (int j = 0; j < kSKMax / 8; ++j) rb[j] = gload4<GT, VEC4, ELL>(G, K, d, L, (t >> 5) + 8 * j, x);
    if (part) {
#pragma unroll
      for (int j = 0; j < kTgt; ++j) {
        const int e = t + j * kDThreads, k = e / kDN;
        const int64_t xx = nt * kDN + e % kDN, col = k * L + xx;
        rg[j] = (e < ELL * kDN && xx < L && col < d) ? gsum[col] : 0.f;
      }
    }
  };
  auto commit = [&]() {
#pragma unroll
    for (int j = 0; j < kSKMax / 8; ++j) {
      const int c = (t >> 5) + 8 * j;
      if (c < Kq) {
        const int hh = c >= Kh ? 1 : 0;
        *reinterpret_cast<float4 *>(Bs + hh * kSBHalf + (c - hh * Kh) * kDN + (t & 31) * 4) = rb[j];
      }
    }
    if (part) {
#pragma unroll
      for (int j = 0; j < kTgt; ++j)
        if (t + j * kDThreads < ELL * kDN) gs[t + j * kDThreads] = rg[j];
    }
  };

  int64_t cur_mt = -1;
  if (q0 < q1) prefetch(q0);
  for (int64_t q = q0; q < q1; ++q) {
    const int64_t mt = q / ntiles, nt = q % ntiles;
    if (mt != cur_mt) {
      // A rows of the new row tile: C[(mt*128 + r)][0 .. Kq), zero past the last row
      for (int e = t; e < kDM * (Kq >> 2); e += kDThreads) {
        const int r = e / (Kq >> 2), c = (e % (Kq >> 2)) * 4;
        const int64_t gr = mt * kDM + r;
        const float4 a = gr < rows ? *reinterpret_cast<const float4 *>(C + gr * Kp + c)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
        const float av[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int cc = c + u, hh = cc >= Kh ? 1 : 0;
          As[hh * kSAHalf + r * kSAStride + (cc - hh * Kh)] = av[u];
        }
      }
      cur_mt = mt;
    }
    commit();
    __syncthreads();
    if (q + 1 < q1) prefetch(q + 1);

    v16f acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.f;
    const float *Ah = As + h * kSAHalf + (wm * 64 + li) * kSAStride;
    const float *Bh = Bs + h * kSBHalf + wn * 64 + li;
#pragma unroll 2
    for (int ks = 0; ks < Kh; ++ks) {
      const float a0 = Ah[ks], a1 = Ah[32 * kSAStride + ks];
      const float b0 = Bh[ks * kDN], b1 = Bh[ks * kDN + 32];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(b0, a0, acc[0][0], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(b1, a0, acc[1][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(b0, a1, acc[0][1], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(b1, a1, acc[1][1], 0, 0, 0);
    }

    direct_epilogue<ELL, VEC4>(acc, mt, nt, rows, d, L, ghat, gs, part ? red2 : nullptr, wm, wn, h,
                               li);
    __syncthreads();
    if (part && t < kDM) {
      const int64_t r = mt * kDM + t;
      if (r < rows) part[r * ntiles + nt] = red2[0][t] + red2[1][t];
    }
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
  if (P < 1 || N < 1 || d < 1 || ell < 1 || ell > GC_MAX_ELL || !sizes_ok({P, ell, direct_kp(N, ell)}) ||
      !sizes_ok({P, d}))
    return 0;
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
  // G [N][d], psi [P][m], the estimate [P][d], mixing rows [P ell][Kp]
  if (!sizes_ok({N, d}) || !sizes_ok({P, m}) || !sizes_ok({P, d}) || !sizes_ok({P, ell, direct_kp(N, ell)}))
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
  // the VEC4 kernels load the gradients and store the estimate 16 bytes at a time
  const bool vec4 = d % 4 == 0 && L % 4 == 0 && (reinterpret_cast<uintptr_t>(G) % (4 * es)) == 0 &&
                    (reinterpret_cast<uintptr_t>(ghat) % 16) == 0;
  const dim3 grid{static_cast<uint32_t>(blocks)};
  const bool f32 = g_dtype == GC_F32;
  const int Kq = int(ceil_div(int64_t(N) * ell, 4) * 4);
  const int64_t ntotal = ceil_div(rows, kDM) * ntiles;
  const bool short_k = Kq <= kSKMax;
  const dim3 sgrid{static_cast<uint32_t>(std::min<int64_t>(ntotal, 2 * int64_t(cu_count())))};
#define GC_DIRECT(GT, V, E)                                                                        \
  if (short_k)                                                                                     \
    hipLaunchKernelGGL((direct_short_kernel<GT, V, E>), sgrid, dim3(kDThreads), 0, stream, Cm,     \
                       static_cast<const GT *>(G), N, d, L, Kp, Kq, rows, ntiles, ntotal, ghat,    \
                       gsum, part);                                                                \
  else                                                                                             \
    hipLaunchKernelGGL((direct_kernel<GT, V, E>), grid, dim3(kDThreads), 0, stream, Cm,            \
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
