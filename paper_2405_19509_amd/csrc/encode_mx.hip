// gc_encode on the bf16 matrix cores (Sec. 2, worker encode):
//   T[p][j][x] = sum_{t < psi[p][j]} sum_{k < ell} Bc[p][j][t][k] * g_{order[j][t]}[k*L + x]
//
// Why matrix cores: every output value of the encode takes psi*ell multiply-adds, 4-5 per
// byte of T at delta = 20, ell = 1 and 4x that at ell = 4, which the vector units cannot
// sustain at the HBM write rate.  Per worker group the encode is a dense contraction
//   T[(pattern, worker)][x] = sum_kk A[(pattern, worker)][kk] * Gs[kk][x]
// over kk = (chunk slot s of the group's union, block k), with A the coefficients of the
// row's worker (zero where the worker does not hold the chunk or has not processed it).
//
// Arithmetic: each fp32 coefficient a is split into three bf16 parts a = a1 + a2 + a3 + r
// with |r| <= 2^-24 |a| (each part the bf16 rounding of what the previous ones leave).
// bf16 chunk gradients enter as they are: three products per term.  An fp32 chunk gradient
// g is split exactly into three bf16 parts by truncation (g1 its top 16 bits, g2 the top 16
// bits of g - g1, g3 the rest), and the six products a_i g_j with i + j <= 4 are kept: the
// dropped ones stay below 2^-21 |a g|.  Every product of two bf16 values is exact in fp32;
// v_mfma_f32_32x32x16_bf16 accumulates them in fp32.
//
// Layout: a block owns a group of J consecutive workers, a window of PB patterns
// (J * PB = 64 or 128 candidate rows (pattern, worker), candidate r = pb * J + jb) and a
// range of at most 32 slices of x walked in turn.  The window's transmitting rows (psi > 0) are
// compacted into full 32-row tiles (stragglers cost nothing), whose coefficients, split
// into three bf16 planes, are built once per block.  Per slice the block stages the slices
// of the group's union of chunks (J + delta - 1 chunks under the cyclic order), one row per
// (slot, block), and every row tile is computed against them:
//   bf16: 512-wide slices staged straight from memory to LDS (1 KB rows); each of the 8
//         waves takes two 32 x 32 output tiles per row tile, per 16-deep K step three bf16x8
//         coefficient loads, eight 16-bit gathers of the staged column per tile, six MFMAs.
//         Where the group's rows need 3+ K steps, 128-candidate windows with 256-wide
//         slices: the union of twice the workers is not much larger, so the rows staged per
//         row written nearly halve; each wave takes one 32-wide column, gathered once per K
//         step for all (up to four) row tiles.  From 4 K steps on a block fills a CU's LDS
//         and the K loop is unrolled into the registers that frees;
//   fp32: 512-wide slices (256-wide from 4 K steps on) staged through registers with the
//         staged rows fastest, so that a lane's eight K values of one position are two
//         16-byte reads, split once per slice for both row tiles; each wave takes one
//         32-position tile, six MFMAs per row tile and K step.
// Stores are 4 bytes per lane, two 128-byte row segments per instruction, non-temporal;
// rows of workers that transmit nothing (psi = 0) are not written.  Blocks of a slice range
// run back to back on one XCD (round-robin dispatch), so its L2 serves the groups'
// overlapping chunk slices.  If a block's union exceeds its slots (orders other than the
// cyclic one), it walks its workers one at a time (a pass per worker, each staging only
// that worker's chunks).
#include <type_traits>

#include "common.h"
#include "encode_mx.h"

namespace gcx {
namespace {

constexpr int kMxThreads = 512;              // bf16, and fp32 with more than 3 K steps
constexpr int kMxW = 512;                    // positions per slice (1 KB of bf16 per staged row)
constexpr int kMxfMaxWideKS = 3;             // fp32: 512-wide slices (1024 threads) up to 3 K steps
static_assert(kMxW == (kMxThreads / 64) * 64 && kMxW * 2 == 64 * 16, "bf16: two 32-wide tiles per wave, 16 bytes per lane and staged row");
constexpr int kMxMaxKS = 6;                  // K steps of 16 (at most 96 staged rows)
// slices a block walks at most: runs of 32 wrote T up to 8% faster than the 128-373-slice
// runs that about 16 blocks per CU gave at d = 2^20 and 2^24 (a store-only kernel with
// this grid showed the same: its write rate rose with the number of shorter blocks)
constexpr int64_t kMxSliceRun = 32;
// bf16: 128-candidate windows (256-wide slices, one tile per wave) where a 64-candidate
// window would need this many K steps
constexpr int kMxWinKS = 3;
constexpr size_t kMxLds = 152 * 1024;

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

// round-to-nearest-even bf16 bits of a finite fp32 value
__device__ __forceinline__ uint32_t bf16_rne(float v) {
  const uint32_t b = __float_as_uint(v);
  return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// Exact split of eight finite fp32 values into three bf16 parts each, g = g1 + g2 + g3:
// g1 keeps the top 16 bits of g (sign, exponent, 7 fraction bits), g - g1 is exact with at
// most 16 significant bits, g2 its top 16 bits, and what remains has at most 8 significant
// bits, a bf16 value (|g2| < 2^-7 |g|, |g3| < 2^-15 |g|; exact for |g| >= 2^-100).
__device__ __forceinline__ void split3(float4 u0, float4 u1, v8bf &g1, v8bf &g2, v8bf &g3) {
  const float v[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
  uint32_t h1[8], h2[8], h3[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    h1[i] = __float_as_uint(v[i]) & 0xffff0000u;
    const float r1 = v[i] - __uint_as_float(h1[i]);
    h2[i] = __float_as_uint(r1) & 0xffff0000u;
    h3[i] = __float_as_uint(r1 - __uint_as_float(h2[i]));
  }
  v4u p1, p2, p3;
#pragma unroll
  for (int j = 0; j < 4; ++j) {  // high halves: element 2j low, element 2j + 1 high
    p1[j] = __builtin_amdgcn_perm(h1[2 * j + 1], h1[2 * j], 0x07060302u);
    p2[j] = __builtin_amdgcn_perm(h2[2 * j + 1], h2[2 * j], 0x07060302u);
    p3[j] = __builtin_amdgcn_perm(h3[2 * j + 1], h3[2 * j], 0x07060302u);
  }
  g1 = __builtin_bit_cast(v8bf, p1);
  g2 = __builtin_bit_cast(v8bf, p2);
  g3 = __builtin_bit_cast(v8bf, p3);
}

struct MxArgs {
  const void *G;
  int N;
  int64_t d, L;
  const int32_t *psi;
  const int32_t *order;
  const float *Bc;
  int64_t P;
  int m, delta, ell;
  float *T;
  bool stage16;   // bf16: G 16-byte aligned and d, L multiples of 8; fp32: 8-byte, multiples of 2
  int J;          // workers per window
  int PB;         // patterns per window (J * PB = 64 or 128 candidate rows, at most)
  int ngroups;
  int64_t ntp;    // pattern windows
  int slots;      // union slots staged per block
  int nslices;
  int64_t spb;    // slices per range
  int64_t nsr;    // slice ranges (a multiple of 8)
};

// Slice region of the LDS, by chunk-gradient type:
//   bf16: Kp staged rows x RB bytes, position fastest (filled straight from memory)
//   fp32: W positions x (Kp + 4) floats, staged row fastest (a lane's eight K values of
//         one position are two 16-byte reads)
template <typename GT, int KS, int CW>
struct MxLayout {
  static constexpr bool F32 = sizeof(GT) == 4;
  static constexpr int Kp = 16 * KS;
  static_assert(CW == 64 || (CW == 128 && !F32), "64 candidates, or 128 with bf16 chunk gradients");
  static constexpr bool WIN = CW == 128;  // 256-wide slices, one 32-wide tile per wave
  static constexpr int NT = CW / 32;      // row tiles at most
  // fp32: one 32-wide tile per wave, 2 KB row segments of T per slice (16 waves) while the
  // staged rows fit, else 256 positions (8 waves); bf16: two tiles per wave, 512 positions
  // (128-candidate windows: one tile per wave, 256 positions)
  static constexpr int THREADS = F32 && KS <= kMxfMaxWideKS ? 1024 : kMxThreads;
  static constexpr int WAVES = THREADS / 64;
  static constexpr int W = F32 || WIN ? 32 * WAVES : kMxW;  // positions per slice
  static constexpr int RB = W * 2 + 16;  // bf16: staged row stride in bytes, padded so rows 8 apart differ in bank
  static constexpr int BS = Kp + 4;                  // fp32: floats per staged position
  static constexpr size_t slice_bytes = F32 ? size_t(W) * BS * 4 : size_t(Kp) * RB;
  // bf16 from 4 K steps on the staged rows allow one block per CU: registers for the K loop
  // unrolled, so the LDS reads of one step overlap the products of the previous one
  static constexpr int WPE = !F32 && KS >= 4 ? 2 : 4;
  static constexpr int UNR = !F32 && KS >= 4 ? KS : 1;
  static_assert(!F32 || (W / 2) % 128 == 0, "fp32 staging: two positions per thread, whole waves per row group");
};

// LDS: [ slice region ][ Ap: CW/32 tiles x 3 planes x 32 rows x AP bf16 ]
//      [ rdesc: 2 int64 per row ][ map: N int32 ][ slotc: slots int32 ][ code: J*delta int32 ]
// The coefficient rows are first assembled in fp32 over the slice region, then split into Ap.
template <typename GT, int KS, int CW>
__global__ __launch_bounds__((MxLayout<GT, KS, CW>::THREADS)) __attribute__((amdgpu_waves_per_eu(MxLayout<GT, KS, CW>::WPE))) void encode_mx_kernel(
    MxArgs a) {
  using Lay = MxLayout<GT, KS, CW>;
  constexpr int NTH = Lay::THREADS;
  constexpr bool F32 = Lay::F32;
  constexpr int Kp = Lay::Kp;
  constexpr int AP = Kp + 8;  // plane row stride (bf16): 16-byte aligned rows, staggered banks
  extern __shared__ __align__(16) unsigned char lds[];
  unsigned char *Gs = lds;
  uint16_t *Ap = reinterpret_cast<uint16_t *>(lds + Lay::slice_bytes);
  int64_t *rdesc = reinterpret_cast<int64_t *>(Ap + Lay::NT * 3 * 32 * AP);
  int32_t *map = reinterpret_cast<int32_t *>(rdesc + 2 * Kp);
  int32_t *slotc = map + a.N;
  int32_t *code = slotc + a.slots;
  float *Af = reinterpret_cast<float *>(Gs);  // [CW][Kp] fp32, before the slices are staged
  static_assert(size_t(CW) * Kp * 4 <= Lay::slice_bytes, "coefficient rows fit the slice region");
  __shared__ int nslot_s, nuni_s, nsend_s;
  __shared__ int8_t ccomp_s[CW];    // compacted row of each candidate, or -1
  // each compacted row's element offset in T from the window's first row (pattern p0,
  // worker j0): (pb * m + jb) * L; read two at a time by the stores
  __shared__ __align__(16) int64_t rowoff_s[CW];

  // block -> (slice range, unit = (group, pattern tile)); XCD x takes ranges x, x + 8, ...
  const int64_t b = blockIdx.x;
  const int64_t units = int64_t(a.ngroups) * a.ntp;
  const int64_t sr = (b & 7) + 8 * ((b >> 3) / units);
  const int64_t unit = (b >> 3) % units;
  const int64_t s_begin = sr * a.spb;
  const int64_t s_end = s_begin + a.spb < a.nslices ? s_begin + a.spb : a.nslices;
  if (s_begin >= s_end) return;  // the whole block: an empty range at the end
  const int gi = int(unit % a.ngroups);
  const int64_t p0 = (unit / a.ngroups) * a.PB;
  const int j0 = gi * a.J;
  const int nj = a.m - j0 < a.J ? a.m - j0 : a.J;
  const int ell = a.ell;
  float *const Tw = a.T + (p0 * a.m + j0) * a.L;  // row (pattern p0, worker j0) of T
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave, h = lane >> 5, li = lane & 31;

  // which chunks the whole group uses; if they exceed the slots, one worker per pass
  for (int c = tid; c < a.N; c += NTH) map[c] = 0;
  __syncthreads();
  for (int e = tid; e < nj * a.delta; e += NTH) {
    const int c = a.order[int64_t(j0) * a.delta + e];
    if (c >= 0 && c < a.N) map[c] = 1;
  }
  __syncthreads();
  if (tid < kWave) {
    int cnt = 0;
    for (int base = 0; base < a.N; base += kWave) {
      const int c = base + tid;
      const unsigned long long mk = __ballot(c < a.N && map[c] != 0);
      cnt += __popcll(mk);
    }
    if (tid == 0) nuni_s = cnt;
  }
  __syncthreads();
  const bool split = nuni_s > a.slots;
  const int npass = split ? nj : 1;

  for (int pass = 0; pass < npass; ++pass) {
    // active workers of this pass: all nj, or worker jb = pass
    const int ja = split ? pass : 0, jn = split ? pass + 1 : nj;
    __syncthreads();  // the previous pass is done with every table
    for (int c = tid; c < a.N; c += NTH) map[c] = 0;
    __syncthreads();
    for (int e = tid; e < (jn - ja) * a.delta; e += NTH) {
      const int c = a.order[int64_t(j0 + ja) * a.delta + e];
      if (c >= 0 && c < a.N) map[c] = 1;
    }
    __syncthreads();
    // slots in ascending chunk order
    if (tid < kWave) {
      int cnt = 0;
      for (int base = 0; base < a.N; base += kWave) {
        const int c = base + tid;
        const bool on = c < a.N && map[c] != 0;
        const unsigned long long mk = __ballot(on);
        if (on) {
          const int s = cnt + __popcll(mk & ((1ull << tid) - 1));
          map[c] = s;  // < slots: the active set fits by construction
          slotc[s] = c;
        } else if (c < a.N) {
          map[c] = -1;
        }
        cnt += __popcll(mk);
      }
      if (tid == 0) nslot_s = cnt;
    }
    __syncthreads();
    const int nslot = nslot_s;
    const int K = nslot * ell;
    // per (worker, position): the slot of the chunk there, or -1
    for (int e = tid; e < nj * a.delta; e += NTH) {
      const int jb = e / a.delta;
      const int c = a.order[int64_t(j0 + jb) * a.delta + e % a.delta];
      code[e] = (jb >= ja && jb < jn && c >= 0 && c < a.N) ? map[c] : -1;
    }
    // the transmitting candidates of the pass, compacted in candidate order
    if (tid < kWave) {
      int cnt = 0;
      for (int r0 = 0; r0 < CW; r0 += kWave) {
        const int r = r0 + tid, pb = r / a.J, jb = r % a.J;
        const int64_t p = p0 + pb;
        const bool on = pb < a.PB && p < a.P && jb >= ja && jb < jn && a.psi[p * a.m + j0 + jb] > 0;
        const unsigned long long mk = __ballot(on);
        const int c = cnt + __popcll(mk & ((1ull << tid) - 1));
        ccomp_s[r] = on ? int8_t(c) : int8_t(-1);
        if (on) rowoff_s[c] = (int64_t(pb) * a.m + jb) * a.L;
        cnt += __popcll(mk);
      }
      if (tid == 0) nsend_s = cnt;
    }
    for (int e = tid; e < CW * Kp; e += NTH) Af[e] = 0.f;
    __syncthreads();
    const int nsend = nsend_s;
    const int ntile = (nsend + 31) / 32;
    // compacted row c (candidate (pattern p0 + r / J, worker j0 + r % J)), column s*ell + k:
    // zero past the row's processed prefix
    for (int e = tid; e < CW * a.delta; e += NTH) {
      const int r = e / a.delta, t = e % a.delta;
      const int c = ccomp_s[r];
      if (c < 0) continue;
      const int jb = r % a.J;
      const int64_t p = p0 + r / a.J;
      const int s = code[jb * a.delta + t];
      if (s < 0) continue;
      int v = a.psi[p * a.m + j0 + jb];
      v = v < 0 ? 0 : (v > a.delta ? a.delta : v);
      if (t >= v) continue;
      const float *src = a.Bc + ((p * a.m + j0 + jb) * a.delta + t) * ell;
      for (int k = 0; k < ell; ++k) Af[c * Kp + s * ell + k] = src[k];
    }
    __syncthreads();
    // three bf16 planes per row tile: a1 = bf16(a), a2 = bf16(a - a1), a3 = bf16(a - a1 - a2),
    // all exact steps
    for (int e = tid; e < 32 * ntile * Kp; e += NTH) {
      const int c = e / Kp, kk = e % Kp;
      const int rt = c / 32, r = c % 32;
      const float v = Af[e];
      const uint32_t b1 = bf16_rne(v);
      const float r1 = v - __uint_as_float(b1 << 16);
      const uint32_t b2 = bf16_rne(r1);
      const float r2 = r1 - __uint_as_float(b2 << 16);
      const uint32_t b3 = bf16_rne(r2);
      uint16_t *tp = Ap + rt * 3 * 32 * AP;
      tp[(0 * 32 + r) * AP + kk] = uint16_t(b1);
      tp[(1 * 32 + r) * AP + kk] = uint16_t(b2);
      tp[(2 * 32 + r) * AP + kk] = uint16_t(b3);
    }
    // staged rows: element offset of block k of slot s's chunk, and the end of its valid
    // positions min(L, d - k L)
    for (int row = tid; row < K; row += NTH) {
      const int s = row / ell, k = row % ell;
      rdesc[2 * row] = int64_t(slotc[s]) * a.d + int64_t(k) * a.L;
      const int64_t rem = a.d - int64_t(k) * a.L;
      rdesc[2 * row + 1] = rem < a.L ? rem : a.L;
    }
    __syncthreads();  // Af consumed: the slice region is free
    // bf16: rows K .. Kp of the slice region stay zero for the whole pass (fp32: the
    // staging writes them)
    if constexpr (!F32)
      for (int e = tid; e < (Kp - K) * (Lay::RB / 16); e += NTH)
        reinterpret_cast<uint4 *>(Gs + size_t(K) * Lay::RB)[e] = make_uint4(0u, 0u, 0u, 0u);
    if (ntile == 0) continue;  // nothing transmitted in this window: no slice to stage

    for (int64_t slice = s_begin; slice < s_end; ++slice) {
      const int64_t x0 = slice * Lay::W;
      __syncthreads();  // the previous slice is consumed
      if constexpr (F32) {
        // stage: a thread takes positions xp, xp + 1 and groups of 8 staged rows, and writes
        // each position's 8 values as two 16-byte words (zero past L, d or K)
        float *Bf = reinterpret_cast<float *>(Gs);
        const float *Gf = static_cast<const float *>(a.G);
        const int xp = 2 * (tid % (Lay::W / 2));
        const int64_t x = x0 + xp;
#pragma unroll 1
        for (int g = tid / (Lay::W / 2); g < Kp / 8; g += (NTH / (Lay::W / 2))) {
          float v0[8], v1[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int kk = 8 * g + i;
            v0[i] = 0.f;
            v1[i] = 0.f;
            if (kk < K) {
              const int64_t base = rdesc[2 * kk], lim = rdesc[2 * kk + 1];
              if (a.stage16 && x + 2 <= lim) {
                const float2 u = *reinterpret_cast<const float2 *>(Gf + base + x);
                v0[i] = u.x;
                v1[i] = u.y;
              } else {
                if (x < lim) v0[i] = Gf[base + x];
                if (x + 1 < lim) v1[i] = Gf[base + x + 1];
              }
            }
          }
          float *d0 = Bf + xp * Lay::BS + 8 * g, *d1 = d0 + Lay::BS;
          *reinterpret_cast<float4 *>(d0) = make_float4(v0[0], v0[1], v0[2], v0[3]);
          *reinterpret_cast<float4 *>(d0 + 4) = make_float4(v0[4], v0[5], v0[6], v0[7]);
          *reinterpret_cast<float4 *>(d1) = make_float4(v1[0], v1[1], v1[2], v1[3]);
          *reinterpret_cast<float4 *>(d1 + 4) = make_float4(v1[4], v1[5], v1[6], v1[7]);
        }
      } else {
        // stage: staged row `row` <- W positions of its block from x0 (zero past L or d),
        // straight from memory to LDS: one wave instruction per row, lane i filling bytes
        // 16i .. 16i + 15 (256-wide slices: lanes 0 .. 31)
        const uint16_t *Gh = static_cast<const uint16_t *>(a.G);
        for (int row = wave; row < K && (!Lay::WIN || lane < 32); row += Lay::WAVES) {
          const int64_t base = rdesc[2 * row], lim = rdesc[2 * row + 1];
          const int64_t x = x0 + 8 * lane;
          unsigned char *dst = Gs + size_t(row) * Lay::RB;
          if (a.stage16 && x0 + Lay::W <= lim) {
            __builtin_amdgcn_global_load_lds(Gh + base + x, dst, 16, 0, 0);
          } else {
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const uint32_t lo = x + 2 * q < lim ? Gh[base + x + 2 * q] : 0u;
              const uint32_t hi = x + 2 * q + 1 < lim ? Gh[base + x + 2 * q + 1] : 0u;
              w[q] = lo | (hi << 16);
            }
            *reinterpret_cast<uint4 *>(dst + 16 * lane) = make_uint4(w[0], w[1], w[2], w[3]);
          }
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's direct-to-LDS loads have landed
      }
      __syncthreads();  // the slice is staged

      if constexpr (F32) {
        // one 32-position tile per wave (x0 + 32 wave + li), every row tile in one K loop so
        // that each staged value is split once
        const float *Bw = reinterpret_cast<const float *>(Gs) + (32 * wave + li) * Lay::BS + 8 * h;
        auto tiles = [&](auto ntc) {
          constexpr int NT = decltype(ntc)::value;
          v16f acc[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[t] = v16f{};
#pragma unroll 1
          for (int q = 0; q < KS; ++q) {
            const float4 u0 = *reinterpret_cast<const float4 *>(Bw + 16 * q);
            const float4 u1 = *reinterpret_cast<const float4 *>(Bw + 16 * q + 4);
            v8bf g1, g2, g3;
            split3(u0, u1, g1, g2, g3);
            const int kb = 16 * q + 8 * h;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              const uint16_t *At = Ap + t * 3 * 32 * AP;
              const v8bf a1 = *reinterpret_cast<const v8bf *>(At + (0 * 32 + li) * AP + kb);
              const v8bf a2 = *reinterpret_cast<const v8bf *>(At + (1 * 32 + li) * AP + kb);
              const v8bf a3 = *reinterpret_cast<const v8bf *>(At + (2 * 32 + li) * AP + kb);
              // the six products of parts above 2^-24 relative, smallest first
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, g1, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, g2, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, g3, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, g1, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, g2, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, g1, acc[t], 0, 0, 0);
            }
          }
          const int64_t xa = x0 + 32 * wave + li;
          if (xa >= a.L) return;
          // lane (h, li) holds D[8(v/4) + 4h + v%4][li]: rows 32t + 8g + 4h + i, their
          // offsets read four at a time (two 16-byte reads)
          float *Tx = Tw + xa;
#pragma unroll
          for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int cb = 32 * t + 8 * g + 4 * h;
              const longlong2 o0 = *reinterpret_cast<const longlong2 *>(rowoff_s + cb);
              const longlong2 o1 = *reinterpret_cast<const longlong2 *>(rowoff_s + cb + 2);
              const int64_t off[4] = {o0.x, o0.y, o1.x, o1.y};
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (cb + i < nsend) __builtin_nontemporal_store(acc[t][4 * g + i], Tx + off[i]);
            }
        };
        if (ntile == 2)
          tiles(std::integral_constant<int, 2>{});
        else
          tiles(std::integral_constant<int, 1>{});
      } else if constexpr (Lay::WIN) {
        // one 32-position tile per wave (x0 + 32 wave + li), every row tile in one K loop so
        // that each gathered column feeds all of them
        const uint16_t *Gc = reinterpret_cast<const uint16_t *>(Gs) + 32 * wave + li;
        constexpr int GR = Lay::RB / 2;  // staged row stride in bf16
        auto tiles = [&](auto ntc) {
          constexpr int NT = decltype(ntc)::value;
          v16f acc[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[t] = v16f{};
#pragma unroll Lay::UNR
          for (int q = 0; q < KS; ++q) {
            const int kb = 16 * q + 8 * h;
            v8bf bq;
#pragma unroll
            for (int i = 0; i < 8; ++i) bq[i] = __builtin_bit_cast(__bf16, Gc[(kb + i) * GR]);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              const uint16_t *At = Ap + t * 3 * 32 * AP;
              const v8bf a1 = *reinterpret_cast<const v8bf *>(At + (0 * 32 + li) * AP + kb);
              const v8bf a2 = *reinterpret_cast<const v8bf *>(At + (1 * 32 + li) * AP + kb);
              const v8bf a3 = *reinterpret_cast<const v8bf *>(At + (2 * 32 + li) * AP + kb);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, bq, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, bq, acc[t], 0, 0, 0);
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, bq, acc[t], 0, 0, 0);
            }
          }
          const int64_t xa = x0 + 32 * wave + li;
          if (xa >= a.L) return;
          // lane (h, li) holds D[8(v/4) + 4h + v%4][li]: rows 32t + 8g + 4h + i, their
          // offsets read four at a time (two 16-byte reads)
          float *Tx = Tw + xa;
#pragma unroll
          for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int cb = 32 * t + 8 * g + 4 * h;
              const longlong2 o0 = *reinterpret_cast<const longlong2 *>(rowoff_s + cb);
              const longlong2 o1 = *reinterpret_cast<const longlong2 *>(rowoff_s + cb + 2);
              const int64_t off[4] = {o0.x, o0.y, o1.x, o1.y};
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (cb + i < nsend) __builtin_nontemporal_store(acc[t][4 * g + i], Tx + off[i]);
            }
        };
        if (ntile == 1)
          tiles(std::integral_constant<int, 1>{});
        else if (ntile == 2)
          tiles(std::integral_constant<int, 2>{});
        else if (ntile == 3)
          tiles(std::integral_constant<int, 3>{});
        else
          tiles(std::integral_constant<int, Lay::NT>{});
      } else {
        // per row tile, two 32 x 32 tiles per wave: positions x0 + 64 wave + 32 c + li
        const uint16_t *Gc = reinterpret_cast<const uint16_t *>(Gs) + 64 * wave + li;
        constexpr int GR = Lay::RB / 2;  // staged row stride in bf16
        for (int rt = 0; rt < ntile; ++rt) {
          const uint16_t *At = Ap + rt * 3 * 32 * AP;
          v16f acc0 = {}, acc1 = {};
#pragma unroll Lay::UNR
          for (int q = 0; q < KS; ++q) {
            const int kb = 16 * q + 8 * h;
            const v8bf a1 = *reinterpret_cast<const v8bf *>(At + (0 * 32 + li) * AP + kb);
            const v8bf a2 = *reinterpret_cast<const v8bf *>(At + (1 * 32 + li) * AP + kb);
            const v8bf a3 = *reinterpret_cast<const v8bf *>(At + (2 * 32 + li) * AP + kb);
            v8bf b0, b1;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              b0[i] = __builtin_bit_cast(__bf16, Gc[(kb + i) * GR]);
              b1[i] = __builtin_bit_cast(__bf16, Gc[(kb + i) * GR + 32]);
            }
            acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b1, acc1, 0, 0, 0);
            acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b1, acc1, 0, 0, 0);
            acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc1, 0, 0, 0);
          }
          // lane (h, li) holds D[8(v/4) + 4h + v%4][li] of each tile: rows 32 rt + 8g + 4h +
          // i, their offsets read four at a time (two 16-byte reads)
          const int64_t xa = x0 + 64 * wave + li, xb = xa + 32;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int cb = 32 * rt + 8 * g + 4 * h;
            const longlong2 o0 = *reinterpret_cast<const longlong2 *>(rowoff_s + cb);
            const longlong2 o1 = *reinterpret_cast<const longlong2 *>(rowoff_s + cb + 2);
            const int64_t off[4] = {o0.x, o0.y, o1.x, o1.y};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if (cb + i >= nsend) continue;
              float *row = Tw + off[i];
              if (xa < a.L) __builtin_nontemporal_store(acc0[4 * g + i], row + xa);
              if (xb < a.L) __builtin_nontemporal_store(acc1[4 * g + i], row + xb);
            }
          }
        }
      }
    }
  }
}

template <typename GT, int KS, int CW>
int launch_mx_ks(const MxArgs &m, size_t lds, hipStream_t st) {
  if constexpr (CW == 128 && KS < kMxWinKS) {
    return kEncodeMxNotApplicable;  // never planned: a 128-candidate window has as many K steps
  } else {                          // as a 64-candidate one, or more
    const int64_t blocks = m.nsr * m.ngroups * m.ntp;
    constexpr int NTH = MxLayout<GT, KS, CW>::THREADS;
    if (!grid_ok(blocks, NTH)) return GC_EINVAL;
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&encode_mx_kernel<GT, KS, CW>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
      return GC_ELAUNCH;
    hipLaunchKernelGGL((encode_mx_kernel<GT, KS, CW>), dim3(unsigned(blocks)), dim3(NTH), lds, st, m);
    return GC_OK;
  }
}

template <typename GT, int CW>
int launch_mx(const MxArgs &a, int KS, size_t lds, hipStream_t st) {
  switch (KS) {
    case 1: return launch_mx_ks<GT, 1, CW>(a, lds, st);
    case 2: return launch_mx_ks<GT, 2, CW>(a, lds, st);
    case 3: return launch_mx_ks<GT, 3, CW>(a, lds, st);
    case 4: return launch_mx_ks<GT, 4, CW>(a, lds, st);
    case 5: return launch_mx_ks<GT, 5, CW>(a, lds, st);
    case 6: return launch_mx_ks<GT, 6, CW>(a, lds, st);
    default: return kEncodeMxNotApplicable;
  }
}

}  // namespace

int encode_mx(const void *G, bool f32, int32_t N, int64_t d, const int32_t *psi, const int32_t *order,
              const float *Bc, int64_t P, int32_t m, int32_t delta, int32_t ell, float *T, hipStream_t stream) {
  MxArgs a{};
  a.G = G;
  a.N = N;
  a.d = d;
  a.L = ceil_div(d, ell);
  a.psi = psi;
  a.order = order;
  a.Bc = Bc;
  a.P = P;
  a.m = m;
  a.delta = delta;
  a.ell = ell;
  a.T = T;
  const uintptr_t ga = reinterpret_cast<uintptr_t>(G);
  a.stage16 = f32 ? (d % 2 == 0 && a.L % 2 == 0 && (ga & 7) == 0) : (d % 8 == 0 && a.L % 8 == 0 && (ga & 15) == 0);
  // slots for the cyclic union of a group; a block whose union is larger walks its workers
  // one at a time, each needing delta slots
  auto union_slots = [&](int64_t J) {
    int64_t sl = J + delta - 1;
    if (sl > N) sl = N;
    return sl < delta ? int64_t(delta) : sl;
  };
  // a window of cw candidate rows: PB patterns (a power of two covering the call, at most
  // cw) x J workers, J halved while the group's cyclic union would need more than kMxMaxKS
  // K steps
  struct Plan {
    int pb, J, KS, W;
    int64_t slots;
    size_t lds;
  };
  auto plan = [&](int cw, Plan &q) {
    q.pb = 1;
    while (q.pb < cw && q.pb < P) q.pb *= 2;
    int64_t J = cw / q.pb;
    if (J > m) J = m;
    while (J > 1 && ceil_div(union_slots(J) * ell, 16) > kMxMaxKS) J /= 2;
    q.J = int(J);
    q.slots = union_slots(J);
    const int64_t KS = ceil_div(q.slots * ell, 16);
    if (KS > kMxMaxKS) return false;
    q.KS = int(KS);
    const int Kp = 16 * q.KS;
    q.W = f32 ? (q.KS <= kMxfMaxWideKS ? 512 : 256) : (cw == 128 ? 256 : kMxW);
    const size_t slice = f32 ? size_t(q.W) * (Kp + 4) * sizeof(float) : size_t(Kp) * (q.W * 2 + 16);
    q.lds = slice + sizeof(uint16_t) * (cw / 32) * 3 * 32 * (Kp + 8) + 2 * sizeof(int64_t) * size_t(Kp) +
            sizeof(int32_t) * (size_t(N) + q.slots + size_t(q.J) * delta);
    return q.lds <= kMxLds;
  };
  Plan q{}, q2{};
  const bool ok64 = plan(64, q);
  // bf16: 128-candidate windows, which stage the group's chunks once for up to twice the
  // rows, where a 64-candidate window would need kMxWinKS or more K steps and the larger
  // window holds more candidates
  const bool win = !f32 && (!ok64 || q.KS >= kMxWinKS) && plan(128, q2) &&
                   (!ok64 || int64_t(q2.pb) * q2.J > int64_t(q.pb) * q.J);
  if (win) q = q2;
  else if (!ok64) return kEncodeMxNotApplicable;
  a.PB = q.pb;
  a.J = q.J;
  a.ngroups = int(ceil_div(m, a.J));
  a.ntp = ceil_div(P, q.pb);
  a.slots = int(q.slots);
  const int KS = q.KS, W = q.W;
  const size_t lds = q.lds;
  a.nslices = int(ceil_div(a.L, W));
  // slice ranges: a multiple of 8 (one share per XCD), at least about 16 blocks per CU in
  // all, and at most kMxSliceRun slices each
  const int64_t units = int64_t(a.ngroups) * a.ntp;
  const int64_t want = 16 * int64_t(cu_count());
  int64_t nsr = ceil_div(ceil_div(want, units), 8) * 8;
  if (nsr > ceil_div(a.nslices, 8) * 8) nsr = ceil_div(a.nslices, 8) * 8;
  a.spb = ceil_div(a.nslices, nsr);
  // shorter runs while the grid stays within the launch limits (1024 threads per block at most)
  if (a.spb > kMxSliceRun && ceil_div(ceil_div(a.nslices, kMxSliceRun), 8) * 8 * units <= 0xffffffffLL / 1024)
    a.spb = kMxSliceRun;
  a.nsr = ceil_div(ceil_div(a.nslices, a.spb), 8) * 8;
  if (f32) return launch_mx<float, 64>(a, KS, lds, stream);
  return win ? launch_mx<uint16_t, 128>(a, KS, lds, stream) : launch_mx<uint16_t, 64>(a, KS, lds, stream);
}

}  // namespace gcx
