// gc_encode: every simulated worker's transmitted vector (Sec. 2, worker encode)
//   T[p][j][x] = sum_{t < psi[p][j]} sum_{k < ell} Bc[p][j][t][k] * g_{order[j][t]}[k*L + x]
// Workers with psi = 0 transmit nothing (they are the stragglers of Sec. 1);
// their rows of T are not written.
//
// Bandwidth design (HBM-bound on the T write, ~1 flop per byte):
//   - a block owns one slice of W consecutive x positions and a contiguous
//     range of rows r = p*m + j;  it stages the W-wide slice of every block k
//     of every chunk gradient in LDS once (N*ell*W values, stored type), so
//     the ~psi*ell reads per output element hit LDS, not HBM or L2;
//   - per-row metadata (psi, the chunk indices and the coefficients of the
//     row's processed prefix) is staged group by group in LDS with coalesced
//     loads, then read back as wave-uniform broadcasts;
//   - a wave writes one row segment of W floats (64 lanes x VEC floats)
//     per row: fully coalesced, and every T byte is written exactly once;
//   - block -> (slice, row range) is XCD-aware: blocks are dispatched
//     round-robin over the 8 XCDs, and every block of a slice runs on the
//     same XCD, so its L2 serves the repeated slice staging.
#include "common.h"

namespace gcx {
namespace {

constexpr int kEncThreads = 1024;
constexpr int kEncWaves = kEncThreads / kWave;
constexpr size_t kEncSliceLds = 96 * 1024;   // G slice budget
constexpr size_t kEncMetaLds = 24 * 1024;    // row metadata budget
constexpr int64_t kEncRowsPerBlock = 4096;
constexpr int kEncMaxGroup = 1024;           // rows of metadata staged per step, at most

template <typename GT>
__device__ __forceinline__ float to_f32(GT v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf16_to_f32(v); }

template <typename GT, int VEC>
struct Vec;
template <>
struct Vec<float, 4> { using T = float4; };
template <>
struct Vec<float, 2> { using T = float2; };
template <>
struct Vec<float, 1> { using T = float; };
template <>
struct Vec<uint16_t, 4> { using T = uint2; };
template <>
struct Vec<uint16_t, 2> { using T = uint32_t; };
template <>
struct Vec<uint16_t, 1> { using T = uint16_t; };

template <typename GT, int VEC>
__device__ __forceinline__ void load_vec(const GT *p, float (&v)[VEC]) {
  using VT = typename Vec<GT, VEC>::T;
  const VT raw = *reinterpret_cast<const VT *>(p);
  const GT *e = reinterpret_cast<const GT *>(&raw);
#pragma unroll
  for (int q = 0; q < VEC; ++q) v[q] = to_f32<GT>(e[q]);
}

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));

// T is written once and read back only by the combine: non-temporal stores
// keep it from displacing the chunk-gradient slices in L2.
template <int VEC>
__device__ __forceinline__ void store_vec(float *p, const float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const v4f t = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(t, reinterpret_cast<v4f *>(p));
  } else if constexpr (VEC == 2) {
    const v2f t = {v[0], v[1]};
    __builtin_nontemporal_store(t, reinterpret_cast<v2f *>(p));
  } else {
    __builtin_nontemporal_store(v[0], p);
  }
}

struct EncodeArgs {
  const void *G;
  int N;
  int64_t d;
  int64_t L;
  const int32_t *psi;
  const int32_t *order;
  const float *Bc;
  int64_t rows;  // P * m
  int m;
  int delta;
  int ell;
  float *T;
  int nslices;
  int64_t rows_per_block;
  int group_rows;  // rows of metadata staged per step
  bool stage16;    // d and L multiples of 16 bytes of G, G 16-byte aligned
};

// LDS layout: [ G slice : N*ell*W GT ][ psi : group ][ chunk : group*delta ][ coef : group*delta*ell ]
// STAGE = false (the slice of every chunk does not fit in LDS): no slice in
// LDS; the gradient values are read from global memory, where L2 holds the
// slice for the block's many rows.
template <typename GT, int VEC, bool STAGE>
__global__ __launch_bounds__(kEncThreads) void encode_kernel(EncodeArgs a) {
  constexpr int W = kWave * VEC;
  extern __shared__ __align__(16) unsigned char lds[];
  GT *Gs = reinterpret_cast<GT *>(lds);
  const size_t gbytes =
      STAGE ? (size_t(a.N) * a.ell * W * sizeof(GT) + 15) & ~size_t(15) : size_t(0);
  int32_t *mpsi = reinterpret_cast<int32_t *>(lds + gbytes);
  int32_t *mchunk = mpsi + a.group_rows;
  float *mcoef = reinterpret_cast<float *>(mchunk + size_t(a.group_rows) * a.delta);

  // block -> (slice, row block); every block of a slice lands on one XCD
  const int64_t b = blockIdx.x;
  int64_t slice, rblock;
  if ((a.nslices & 7) == 0) {
    const int64_t per = a.nslices >> 3;
    slice = (b & 7) + 8 * ((b >> 3) % per);
    rblock = b / a.nslices;
  } else {
    slice = b % a.nslices;
    rblock = b / a.nslices;
  }
  const int64_t x0 = slice * W;
  const int64_t r0 = rblock * a.rows_per_block;
  const int64_t r1 = r0 + a.rows_per_block < a.rows ? r0 + a.rows_per_block : a.rows;

  // stage the slice: Gs[(c*ell + k)*W + w] = g_c[k*L + x0 + w] (zero past L or past d),
  // 16 bytes per load where the run lies inside the gradient (d, L and G aligned to it)
  const GT *G = reinterpret_cast<const GT *>(a.G);
  const int nrow = STAGE ? a.N * a.ell : 0;
  constexpr int SV = 16 / sizeof(GT);
  using SVT = uint4;
  for (int e = threadIdx.x * SV; e < nrow * W; e += kEncThreads * SV) {
    const int ck = e / W, w = e % W;  // W is a multiple of SV
    const int c = ck / a.ell, k = ck % a.ell;
    const int64_t x = x0 + w;
    const int64_t col = int64_t(k) * a.L + x;
    if (a.stage16 && x + SV <= a.L && col + SV <= a.d) {
      *reinterpret_cast<SVT *>(Gs + e) = *reinterpret_cast<const SVT *>(G + int64_t(c) * a.d + col);
    } else {
#pragma unroll
      for (int u = 0; u < SV; ++u)
        Gs[e + u] = (x + u < a.L && col + u < a.d) ? G[int64_t(c) * a.d + col + u] : GT(0);
    }
  }

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int stride_row = a.delta * a.ell;
  const int64_t xl = x0 + int64_t(lane) * VEC;  // this lane's first x
  __shared__ int nact;                          // rows of the group that transmit
  __shared__ int16_t act[kEncMaxGroup];
  for (int64_t g0 = r0; g0 < r1; g0 += a.group_rows) {
    const int gn = int(r1 - g0 < a.group_rows ? r1 - g0 : a.group_rows);
    __syncthreads();  // previous group fully consumed (and the slice staged)
    if (threadIdx.x == 0) nact = 0;
    __syncthreads();
    for (int e = threadIdx.x; e < gn; e += kEncThreads) {
      const int64_t r = g0 + e;
      const int j = int(r % a.m);
      int v = a.psi[r];
      v = v < 0 ? 0 : (v > a.delta ? a.delta : v);
      mpsi[e] = v;
      // a worker that has processed nothing transmits nothing: only the other
      // rows are queued, so the waves share the transmitted rows evenly
      if (v > 0) act[atomicAdd(&nact, 1)] = int16_t(e);
      for (int t = 0; t < a.delta; ++t) {
        int c = a.order[int64_t(j) * a.delta + t];
        mchunk[e * a.delta + t] = (c >= 0 && c < a.N) ? c : -1;
      }
    }
    const float *src = a.Bc + g0 * stride_row;
    for (int e = threadIdx.x; e < gn * stride_row; e += kEncThreads) mcoef[e] = src[e];
    __syncthreads();

    const int na = nact;
    for (int ai = wave; ai < na; ai += kEncWaves) {
      const int e = act[ai];
      const int64_t r = g0 + e;
      const int np = mpsi[e];
      float acc[VEC];
#pragma unroll
      for (int q = 0; q < VEC; ++q) acc[q] = 0.f;
      for (int t = 0; t < np; ++t) {
        const int c = mchunk[e * a.delta + t];
        if (c < 0) continue;
        for (int k = 0; k < a.ell; ++k) {
          const float w = mcoef[e * stride_row + t * a.ell + k];
          float g[VEC];
          if constexpr (STAGE) {
            load_vec<GT, VEC>(Gs + (size_t(c) * a.ell + k) * W + lane * VEC, g);
          } else {
            const int64_t col = int64_t(k) * a.L + xl;
            if (xl < a.L && col < a.d) {
              load_vec<GT, VEC>(G + int64_t(c) * a.d + col, g);
            } else {
#pragma unroll
              for (int q = 0; q < VEC; ++q) g[q] = 0.f;
            }
          }
#pragma unroll
          for (int q = 0; q < VEC; ++q) acc[q] = fmaf(w, g[q], acc[q]);
        }
      }
      if (xl < a.L) store_vec<VEC>(a.T + r * a.L + xl, acc);
    }
  }
}

// Per-worker layout, for ell >= 2 or many chunks, where the W-wide slice of every chunk
// no longer fits in LDS at W = 256 floats: a block owns one worker j, one WW-wide slice of x
// (WW = 1024, 512 or 256 floats: the widest whose delta*ell slices fit in kEwLds) and a
// range of patterns, and stages only the slices of j's own delta chunks.  Consecutive
// blocks take the slices of one row, then the next worker (the next row in memory), then
// the next pattern range, so the blocks in flight write whole consecutive rows of T.
// A wave writes one WW-wide row piece per transmitting pattern.
constexpr int kEwThreads = 256;
constexpr size_t kEwLds = 64 * 1024;   // slice budget
constexpr int64_t kEwPatterns = 100;   // patterns per block

template <typename GT, int WW>
__global__ __launch_bounds__(kEwThreads) void encode_worker_kernel(EncodeArgs a, int64_t P,
                                                                   int nsl) {
  constexpr int NV = WW / (4 * kWave);  // 16-byte pieces per lane
  extern __shared__ __align__(16) unsigned char lds[];
  GT *Gs = reinterpret_cast<GT *>(lds);  // [delta*ell][WW]
  const int64_t b = blockIdx.x;
  const int s = int(b % nsl);
  const int j = int((b / nsl) % a.m);
  const int64_t g = b / (int64_t(nsl) * a.m);
  const int64_t x0 = int64_t(s) * WW;
  const int nk = a.delta * a.ell;
  const GT *G = reinterpret_cast<const GT *>(a.G);
  for (int e = threadIdx.x; e < nk * WW; e += kEwThreads) {
    const int tk = e / WW, w = e % WW;
    const int t = tk / a.ell, k = tk % a.ell;
    const int c = a.order[int64_t(j) * a.delta + t];
    const int64_t x = x0 + w, col = int64_t(k) * a.L + x;
    Gs[e] = (c >= 0 && c < a.N && x < a.L && col < a.d) ? G[int64_t(c) * a.d + col] : GT(0);
  }
  __syncthreads();

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t p0 = g * kEwPatterns;
  const int64_t p1 = p0 + kEwPatterns < P ? p0 + kEwPatterns : P;
  for (int64_t p = p0 + wave; p < p1; p += kEwThreads / kWave) {
    const int64_t r = p * a.m + j;
    int np = a.psi[r];
    np = np < 0 ? 0 : (np > a.delta ? a.delta : np);
    if (np == 0) continue;  // a worker that has processed nothing transmits nothing
    const float *co = a.Bc + r * nk;
    float acc[NV][4];
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[i][q] = 0.f;
    for (int tk = 0; tk < np * a.ell; ++tk) {  // positions in order, blocks within a position
      const float w = co[tk];
      const GT *src = Gs + size_t(tk) * WW + lane * 4;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        float gv[4];
        load_vec<GT, 4>(src + i * 4 * kWave, gv);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][q] = fmaf(w, gv[q], acc[i][q]);
      }
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int64_t x = x0 + i * 4 * kWave + lane * 4;
      if (x < a.L) store_vec<4>(a.T + r * a.L + x, acc[i]);
    }
  }
}

template <typename GT, int WW>
int launch_encode_worker(const EncodeArgs &a, int64_t P, hipStream_t st) {
  const int nsl = int(ceil_div(a.L, WW));
  const int64_t blocks = int64_t(nsl) * a.m * ceil_div(P, kEwPatterns);
  if (!grid_ok(blocks, kEwThreads)) return GC_EINVAL;
  const size_t lds = size_t(a.delta) * a.ell * WW * sizeof(GT);
  hipLaunchKernelGGL((encode_worker_kernel<GT, WW>), dim3(unsigned(blocks)), dim3(kEwThreads), lds,
                     st, a, P, nsl);
  return GC_OK;
}

template <typename GT, int VEC, bool STAGE>
int launch_encode(EncodeArgs a, hipStream_t st) {
  constexpr int W = kWave * VEC;
  a.nslices = int(ceil_div(a.L, W));
  const size_t gbytes =
      STAGE ? (size_t(a.N) * a.ell * W * sizeof(GT) + 15) & ~size_t(15) : size_t(0);
  const size_t per_row = sizeof(int32_t) * (1 + a.delta) + sizeof(float) * a.delta * a.ell;
  int group = int(kEncMetaLds / per_row);
  if (group > kEncMaxGroup) group = kEncMaxGroup;
  if (group < 1) group = 1;
  a.group_rows = group;
  // at most kEncRowsPerBlock rows per block, and a grid that is a whole number of rounds of
  // the blocks the chip holds at once (two per CU), so no round runs partly empty
  const int64_t conc = 2 * int64_t(cu_count());
  int64_t g = a.nslices, h = conc;
  while (h) { const int64_t t = g % h; g = h; h = t; }
  const int64_t step = conc / g;  // row blocks per round of the grid
  const int64_t rblocks = ceil_div(ceil_div(a.rows, kEncRowsPerBlock), step) * step;
  a.rows_per_block = ceil_div(a.rows, rblocks);
  const int64_t blocks = rblocks * a.nslices;
  if (!grid_ok(blocks, kEncThreads)) return GC_EINVAL;
  const size_t lds = gbytes + per_row * group;
  if (hipFuncSetAttribute(reinterpret_cast<const void *>(&encode_kernel<GT, VEC, STAGE>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
    return GC_ELAUNCH;
  hipLaunchKernelGGL((encode_kernel<GT, VEC, STAGE>), dim3(unsigned(blocks)), dim3(kEncThreads), lds,
                     st, a);
  return GC_OK;
}

template <typename GT>
int dispatch_encode(const EncodeArgs &a, int vec, bool stage, hipStream_t st) {
  if (stage) {
    return vec == 4 ? launch_encode<GT, 4, true>(a, st)
                    : (vec == 2 ? launch_encode<GT, 2, true>(a, st) : launch_encode<GT, 1, true>(a, st));
  }
  return vec == 4 ? launch_encode<GT, 4, false>(a, st)
                  : (vec == 2 ? launch_encode<GT, 2, false>(a, st) : launch_encode<GT, 1, false>(a, st));
}

}  // namespace
}  // namespace gcx

extern "C" int gc_encode(const void *G, int32_t g_dtype, int32_t N, int64_t d, const int32_t *psi,
                         const int32_t *order, const float *Bc, int64_t P, int32_t m,
                         int32_t delta, int32_t ell, float *T, hipStream_t stream) {
  using namespace gcx;
  if (N < 1 || d < 1 || P < 0 || m < 1 || m > GC_MAX_M || delta < 1 || delta > GC_MAX_DELTA ||
      ell < 1 || ell > GC_MAX_ELL || (g_dtype != GC_F32 && g_dtype != GC_BF16))
    return GC_EINVAL;
  if (P == 0) return GC_OK;
  if (!G || !psi || !order || !Bc || !T) return GC_EINVAL;
  const int dev = check_device();
  if (dev != GC_OK) return dev;
  EncodeArgs a{};
  a.G = G;
  a.N = N;
  a.d = d;
  a.L = ceil_div(d, ell);
  a.psi = psi;
  a.order = order;
  a.Bc = Bc;
  a.rows = P * m;
  a.m = m;
  a.delta = delta;
  a.ell = ell;
  a.T = T;
  // widest vector the row length and the alignment of T allow; stage the
  // slice of every chunk in LDS when it fits, else read G through L2
  const size_t esize = g_dtype == GC_F32 ? 4 : 2;
  const uintptr_t ta = reinterpret_cast<uintptr_t>(T), ga = reinterpret_cast<uintptr_t>(G);
  const int64_t sv = int64_t(16 / esize);
  a.stage16 = d % sv == 0 && a.L % sv == 0 && (ga & 15) == 0;
  int vec = (a.L % 4 == 0 && (ta & 15) == 0) ? 4 : ((a.L % 2 == 0 && (ta & 7) == 0) ? 2 : 1);
  int svec = vec;
  while (svec > 1 && size_t(N) * ell * kWave * svec * esize > kEncSliceLds) svec >>= 1;
  const bool stage = size_t(N) * ell * kWave * svec * esize <= kEncSliceLds;
  if (stage) {
    vec = svec;
  } else {
    // direct vector loads of G need d and the base to be multiples of the vector
    while (vec > 1 && (d % vec != 0 || (ga & (size_t(vec) * esize - 1)) != 0)) vec >>= 1;
  }
  (void)hipGetLastError();
  // when the all-chunk slice cannot stay 256 wide, the per-worker layout at the widest slice
  // (1024, 512 or 256) that fits, given 16-byte rows of T and enough patterns per block to
  // repay the staging of each worker's slices: its staged bytes, ceil(P/100)*delta*ell*esize
  // per row position, at most half of the 4*P bytes of T there (with very few patterns the
  // all-chunk layout stages every chunk's slice once for all the rows)
  const bool ew_pays = 2 * ceil_div(P, kEwPatterns) * delta * ell * int64_t(esize) <= 4 * P;
  if (a.L % 4 == 0 && (ta & 15) == 0 && (!stage || svec < 4) && ew_pays) {
    const size_t per = size_t(delta) * ell * esize;  // LDS bytes per slice position
    int ww = 0;
    for (int w = 1024; w >= 256 && !ww; w >>= 1)
      if (per * w <= kEwLds) ww = w;
    if (ww) {
      int st;
      if (g_dtype == GC_F32)
        st = ww == 1024 ? launch_encode_worker<float, 1024>(a, P, stream)
             : ww == 512 ? launch_encode_worker<float, 512>(a, P, stream)
                         : launch_encode_worker<float, 256>(a, P, stream);
      else
        st = ww == 1024 ? launch_encode_worker<uint16_t, 1024>(a, P, stream)
             : ww == 512 ? launch_encode_worker<uint16_t, 512>(a, P, stream)
                         : launch_encode_worker<uint16_t, 256>(a, P, stream);
      if (st != GC_OK) return st;
      return launch_status();
    }
  }
  const int st = g_dtype == GC_F32 ? dispatch_encode<float>(a, vec, stage, stream)
                                   : dispatch_encode<uint16_t>(a, vec, stage, stream);
  if (st != GC_OK) return st;
  return launch_status();
}
