// gc_encode: every simulated worker's transmitted vector (Sec. 2, worker encode)
//   T[p][j][x] = sum_{t < psi[p][j]} sum_{k < ell} Bc[p][j][t][k] * g_{order[j][t]}[k*L + x]
// Workers with psi = 0 transmit nothing (they are the stragglers of Sec. 1);
// their rows of T are not written.
//
// Bandwidth design (HBM-bound on the T write, ~1 flop per byte):
//   - a block owns one slice of W consecutive x positions and a run of about 512
//     consecutive rows r = p*m + j; it stages the W-wide slice of every block k
//     of every chunk gradient in LDS (N*ell*W values, stored type), straight
//     from memory to LDS with every piece in flight at once, so the ~psi*ell
//     reads per output element hit LDS, not HBM or L2;
//   - the rows' metadata is staged group by group as a table of (LDS offset,
//     coefficient) per term, four terms per pair of 16-byte LDS reads; its loads
//     are independent of each other (one round trip per group);
//   - a wave writes one row segment of W floats (64 lanes x VEC floats) per
//     row: fully coalesced, and every T byte is written exactly once;
//   - the run length trades the slice staging (N*ell*W values per block, from
//     L2) against the spread of the write front: the blocks in flight cover
//     every slice of a few thousand rows, and runs of ~512 rows wrote T ~4%
//     faster than runs of 4096 (runs of 64-128 lose more to the per-block
//     staging and latency than they gain);
//   - block -> (slice, row run) is XCD-aware: blocks are dispatched round-robin
//     over the 8 XCDs, and every block of a slice runs on the same XCD, so its
//     L2 serves the repeated slice staging.
// When the slice of every chunk does not fit in LDS (many chunks, ell >= 2, bf16 at
// large N) the worker-group layout below takes over.
#include "common.h"
#include "encode_mx.h"

namespace gcx {
namespace {

constexpr int kEncThreads = 1024;
constexpr int kEncWaves = kEncThreads / kWave;
constexpr size_t kEncSliceLds = 96 * 1024;   // G slice budget
constexpr size_t kEncMetaLds = 24 * 1024;    // row metadata budget
constexpr int kEncGroup = 256;               // rows of metadata staged per step, at most
constexpr int kEncGroupsPerBlock = 2;        // rows per block = 2 groups

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
typedef float v16f __attribute__((ext_vector_type(16)));

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

// 16 bytes per lane from global memory straight into LDS: lane i of the wave writes
// bytes 16i..16i+15 of the 1 KB run at `lds_run` (which must be the same for every lane).
// Completion is counted by vmcnt like any vector load.
__device__ __forceinline__ void load_lds16(const void *src, void *lds_run) {
  __builtin_amdgcn_global_load_lds(src, lds_run, 16, 0, 0);
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
  int term_stride; // delta*ell rounded up to 4
  bool stage16;    // d and L multiples of 16 bytes of G, G 16-byte aligned
};

// LDS layout: [ G slice : N*ell*W GT ][ zero row : W GT ][ nterm : group ][ off : group*SR ]
//             [ coef : group*SR ],  SR = delta*ell rounded up to 4.
// Row e's terms u < SR: off = LDS element offset of the slice term u reads (chunk
// order[j][u / ell], block u % ell), coef its coefficient; terms past the row's processed
// prefix, and chunk indices outside [0, N), read the zero row with coefficient 0.
// nterm = the row's psi*ell rounded up to 4 (0: the row transmits nothing).
template <typename GT, int VEC>
__global__ __launch_bounds__(kEncThreads) void encode_kernel(EncodeArgs a) {
  constexpr int W = kWave * VEC;
  constexpr int SV = 16 / sizeof(GT);  // elements per 16-byte piece
  constexpr int PPR = W / SV;          // pieces per staged row
  extern __shared__ __align__(16) unsigned char lds[];
  GT *Gs = reinterpret_cast<GT *>(lds);
  const int nrow = a.N * a.ell;
  const size_t gbytes = size_t(nrow + 1) * W * sizeof(GT);  // W*sizeof(GT) is a multiple of 16
  const int SR = a.term_stride;
  int32_t *mnt = reinterpret_cast<int32_t *>(lds + gbytes);
  int32_t *moff = mnt + ((a.group_rows + 3) & ~3);
  float *mcoef = reinterpret_cast<float *>(moff + size_t(a.group_rows) * SR);
  const int zoff = nrow * W;

  // block -> (slice, row run); every block of a slice lands on one XCD
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
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;

  // the slice: Gs[(c*ell + k)*W + w] = g_c[k*L + x0 + w] (zero past L or past d).  A
  // 16-byte piece inside the gradient (d, L and G aligned to it) goes straight from
  // memory to LDS (global_load_lds_dwordx4: lane i of a wave fills bytes 16i..16i+15
  // of the wave's 1 KB run), every piece in flight at once; the rest element by element.
  const GT *G = reinterpret_cast<const GT *>(a.G);
  const int npieces = nrow * PPR;
  for (int p0 = 0; p0 < npieces; p0 += kEncThreads) {
    const int p = p0 + int(threadIdx.x);
    const int ck = p / PPR, w = (p % PPR) * SV;
    const int c = ck / a.ell, k = ck - c * a.ell;
    const int64_t x = x0 + w;
    const int64_t col = int64_t(k) * a.L + x;
    const bool fast = p < npieces && a.stage16 && x + SV <= a.L && col + SV <= a.d;
    if (fast) load_lds16(G + int64_t(c) * a.d + col, Gs + size_t(p0 + wave * kWave) * SV);
    else if (p < npieces)
      for (int u = 0; u < SV; ++u)
        Gs[size_t(p) * SV + u] = (x + u < a.L && col + u < a.d) ? G[int64_t(c) * a.d + col + u] : GT(0);
  }
  for (int e = threadIdx.x; e < W; e += kEncThreads) Gs[zoff + e] = GT(0);

  const int64_t xl = x0 + int64_t(lane) * VEC;  // this lane's first x
  for (int64_t g0 = r0; g0 < r1; g0 += a.group_rows) {
    const int gn = int(r1 - g0 < a.group_rows ? r1 - g0 : a.group_rows);
    if (g0 != r0) __syncthreads();  // previous group fully consumed
    for (int e = threadIdx.x; e < gn * SR; e += kEncThreads) {
      const int row = e / SR, u = e - row * SR;
      const int64_t r = g0 + row;
      // three independent loads (one round trip), then the selection
      int np = a.psi[r];
      const int t = u / a.ell, k = u - t * a.ell;
      int c = -1;
      float w = 0.f;
      if (u < a.delta * a.ell) {
        c = a.order[int64_t(r % a.m) * a.delta + t];
        w = a.Bc[r * a.delta * a.ell + u];
      }
      np = np < 0 ? 0 : (np > a.delta ? a.delta : np);
      const bool live = u < np * a.ell && c >= 0 && c < a.N;
      moff[e] = live ? (c * a.ell + k) * W : zoff;
      mcoef[e] = live ? w : 0.f;
      if (u == 0) mnt[row] = (np * a.ell + 3) & ~3;
    }
    __builtin_amdgcn_s_waitcnt(0);  // the slice's direct-to-LDS loads have landed
    __syncthreads();

    // a worker that has processed nothing transmits nothing: its row is skipped
    for (int e = wave; e < gn; e += kEncWaves) {
      const int nt = mnt[e];
      if (nt == 0) continue;
      const int64_t r = g0 + e;
      float acc[VEC];
#pragma unroll
      for (int q = 0; q < VEC; ++q) acc[q] = 0.f;
      const int32_t *ro = moff + size_t(e) * SR;
      const float *rc = mcoef + size_t(e) * SR;
      for (int u = 0; u < nt; u += 4) {
        const int4 o = *reinterpret_cast<const int4 *>(ro + u);
        const float4 cw = *reinterpret_cast<const float4 *>(rc + u);
        float g0v[VEC], g1v[VEC], g2v[VEC], g3v[VEC];
        load_vec<GT, VEC>(Gs + o.x + lane * VEC, g0v);
        load_vec<GT, VEC>(Gs + o.y + lane * VEC, g1v);
        load_vec<GT, VEC>(Gs + o.z + lane * VEC, g2v);
        load_vec<GT, VEC>(Gs + o.w + lane * VEC, g3v);
#pragma unroll
        for (int q = 0; q < VEC; ++q) {
          acc[q] = fmaf(cw.x, g0v[q], acc[q]);
          acc[q] = fmaf(cw.y, g1v[q], acc[q]);
          acc[q] = fmaf(cw.z, g2v[q], acc[q]);
          acc[q] = fmaf(cw.w, g3v[q], acc[q]);
        }
      }
      if (xl < a.L) store_vec<VEC>(a.T + r * a.L + xl, acc);
    }
  }
}

// Worker-group layout, for when the slice of every chunk does not fit in LDS at the
// chosen width (many chunks, ell >= 2, bf16 at N = 200, ...).  A block owns one
// W-wide slice of x, a group of J consecutive workers and a range of patterns.
// It stages the slices of the union of the group's chunks (J + delta - 1 chunks
// under the cyclic assignment, so J is sized for that), up to the LDS capacity;
// chunks past the capacity, possible under other orders, are read through L2.
// A wave computes one worker for PB patterns at once: each gradient value read
// from LDS feeds PB accumulators.  The coefficients of the PB rows arrive as one
// coalesced load per 16 terms (lane 16*pb + i holds term tk0 + i of pattern pb)
// and are broadcast with readlane; the LDS offset of each term's slice comes from
// a per-group table the same way.  The blocks of a slice run back to back on one
// XCD, so its L2 serves the groups' overlapping chunk slices.
// Shapes with many terms per output normally take the bf16 matrix-core encode
// (encode_mx.hip); where its staged rows do not fit, with a full 32-pattern tile per call
// and delta*ell >= 32 terms per output (a dense contraction [32 patterns][terms] x
// [terms][128 positions] per worker), a block whose group's chunks are all staged runs its
// items on the fp32 matrix cores instead (v_mfma_f32_32x32x2f32; coefficients past a
// pattern's prefix enter as zeros, so the gradient values must be finite).  With fewer
// patterns, the tile rows are 16 (pattern, worker) pairs and its K the group's staged
// chunk blocks (v_mfma_f32_16x16x4f32).
// fp32 chunk gradients take the bf16 matrix-core encode from this many terms per output
// (measured at m = 100, d = 2^20: at delta*ell = 10 the vector path writes 7% faster; at 20
// the two are within a few percent either way, at 80 the matrix cores win by far)
constexpr int kMxF32Terms = 32;
constexpr int kGrpThreads = 512;
constexpr int kGrpWaves = kGrpThreads / kWave;
constexpr size_t kGrpLds = 72 * 1024;     // per block: two blocks per CU
constexpr size_t kGrpLdsMF = 144 * 1024;  // matrix cores, 32-pattern tiles: one block per CU
static_assert(kGrpLds <= size_t(9) * 512 * 16, "one staging pass covers the slice budget");
constexpr int kGrpTerms = 16;          // terms per coefficient load
constexpr int kGrpStage = 9;           // 16-byte staging loads per thread: the whole slice
constexpr int kGrpSkip = INT32_MIN;    // a padded order slot: no term

// 16 bytes of G from src (positions x.. of a block row valid below lim), zero from lim on
__device__ __forceinline__ uint4 load16_lim(const float *src, int64_t x, int64_t lim) {
  uint32_t r[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = x + v < lim ? __float_as_uint(src[v]) : 0u;
  return make_uint4(r[0], r[1], r[2], r[3]);
}
__device__ __forceinline__ uint4 load16_lim(const uint16_t *src, int64_t x, int64_t lim) {
  uint32_t r[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const uint32_t lo = x + 2 * v < lim ? src[2 * v] : 0u;
    const uint32_t hi = x + 2 * v + 1 < lim ? src[2 * v + 1] : 0u;
    r[v] = lo | (hi << 16);
  }
  return make_uint4(r[0], r[1], r[2], r[3]);
}

struct GroupArgs {
  int J;          // workers per group
  int ngroups;
  int64_t PR;     // patterns per block
  int64_t npr;    // pattern ranges
  int slots;      // chunk slices the block can stage
  int64_t P;
  int64_t nsr;    // slice ranges (a multiple of 8)
  int64_t spb;    // slices per range
  int dense;      // 1: chunk -> slot map over all N chunks; 0 (J = 1): slot t = position t
};

__device__ __forceinline__ int readlane_i(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}
__device__ __forceinline__ float readlane_f(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// The items of one staged slice on the vector units: (pattern batch of PB, worker), worker
// fastest, so the waves write neighbouring rows.
template <typename GT, int VEC, int NV, int PB>
__device__ __forceinline__ void group_vector(const EncodeArgs &a, const GT *__restrict__ Gs,
                                             const int32_t *__restrict__ code, int64_t x0, int j0, int nj,
                                             int64_t p0, int64_t p1, int wave, int lane) {
  const int dl = a.delta * a.ell;
  const GT *G = reinterpret_cast<const GT *>(a.G);
  constexpr int W = kWave * VEC * NV;
  const int64_t nb = ceil_div(p1 - p0, PB);
  const int64_t items = nb * nj;
  const int tl = lane % kGrpTerms, pl = lane / kGrpTerms;  // this lane's term and pattern
  for (int64_t it = wave; it < items; it += kGrpWaves) {
    const int jb = int(it % nj);
    const int j = j0 + jb;
    const int64_t pb0 = p0 + (it / nj) * PB;
    // term tk0 + (lane % 16) of pattern pb0 + lane / 16: its coefficient, and the LDS offset
    // of its slice (staged) or -1 - (c*ell + k) (chunk c, block k, read through L2)
    const float *brow = a.Bc + ((pb0 + pl) * a.m + j) * int64_t(dl);
    auto term_info = [&](int tk0, float &cv, int &cd) {
      const int tk = tk0 + tl;
      cv = (pl < PB && pb0 + pl < p1 && tk < dl) ? brow[tk] : 0.f;
      cd = tk < dl ? code[jb * dl + tk] : kGrpSkip;
    };
    float cvn;
    int cdn;
    term_info(0, cvn, cdn);  // issued before psi is known
    // term limits psi*ell per pattern of the batch (0 past the range)
    int lim_l = 0;
    if (lane < PB && pb0 + lane < p1) {
      int v = a.psi[(pb0 + lane) * a.m + j];
      lim_l = (v < 0 ? 0 : (v > a.delta ? a.delta : v)) * a.ell;
    }
    int lim[PB];
    int tmax = 0;
#pragma unroll
    for (int q = 0; q < PB; ++q) {
      lim[q] = readlane_i(lim_l, q);
      tmax = lim[q] > tmax ? lim[q] : tmax;
    }
    if (tmax == 0) continue;  // every pattern of the batch: a straggler, nothing sent
    float acc[PB][NV][VEC];
#pragma unroll
    for (int q = 0; q < PB; ++q)
#pragma unroll
      for (int u = 0; u < NV; ++u)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[q][u][v] = 0.f;
    for (int tk0 = 0; tk0 < tmax; tk0 += kGrpTerms) {
      const float cv = cvn;
      const int cd = cdn;
      // the next 16 terms' coefficients and slice offsets load while these are applied
      if (tk0 + kGrpTerms < tmax) term_info(tk0 + kGrpTerms, cvn, cdn);
#pragma unroll
      for (int i = 0; i < kGrpTerms; ++i) {
        if (tk0 + i >= tmax) break;
        const int ci = readlane_i(cd, i);
        if (ci == kGrpSkip) continue;
        float gv[NV][VEC];
        if (ci >= 0) {
#pragma unroll
          for (int u = 0; u < NV; ++u) load_vec<GT, VEC>(Gs + ci + (u * kWave + lane) * VEC, gv[u]);
        } else {
          const int ck = -1 - ci, c = ck / a.ell, k = ck - c * a.ell;
#pragma unroll
          for (int u = 0; u < NV; ++u) {
            const int64_t x = x0 + int64_t(u * kWave + lane) * VEC;
            const int64_t col = int64_t(k) * a.L + x;
#pragma unroll
            for (int v = 0; v < VEC; ++v)
              gv[u][v] = (x + v < a.L && col + v < a.d) ? to_f32<GT>(G[int64_t(c) * a.d + col + v]) : 0.f;
          }
        }
#pragma unroll
        for (int q = 0; q < PB; ++q) {
          if (tk0 + i < lim[q]) {
            const float w = readlane_f(cv, q * kGrpTerms + i);
#pragma unroll
            for (int u = 0; u < NV; ++u)
#pragma unroll
              for (int v = 0; v < VEC; ++v) acc[q][u][v] = fmaf(w, gv[u][v], acc[q][u][v]);
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < PB; ++q) {
      if (lim[q] == 0) continue;
      float *row = a.T + ((pb0 + q) * a.m + j) * a.L;
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const int64_t x = x0 + int64_t(u * kWave + lane) * VEC;
        if (x < a.L) store_vec<VEC>(row + x, acc[q][u]);
      }
    }
  }
}

// The items of one staged slice on the matrix cores, every term of the group staged.
template <typename GT>
__device__ __forceinline__ void group_mfma(const EncodeArgs &a, const GT *__restrict__ Gs,
                                             const int32_t *__restrict__ code, int64_t x0, int j0, int nj,
                                             int64_t p0, int64_t p1, int wave, int lane) {
  const int dl = a.delta * a.ell;
  const GT *G = reinterpret_cast<const GT *>(a.G);
  constexpr int W = 128;
  // a wave computes one worker for 32 patterns and 4 x 32 positions on the matrix cores:
  // D[pattern][x] += A[pattern][term] B[term][x] two terms at a time, A the coefficients
  // (zero past each pattern's prefix), B the staged slices.  The two terms of step i are
  // tk0 + i (lanes 0-31) and tk0 + 8 + i (lanes 32-63).
  const int h = lane >> 5, li = lane & 31;
  const int64_t items = ceil_div(p1 - p0, 32) * nj;
  const bool a16 = (dl & 7) == 0 && (reinterpret_cast<uintptr_t>(a.Bc) & 15) == 0;
  for (int64_t it = wave; it < items; it += kGrpWaves) {
    const int jb = int(it % nj);
    const int j = j0 + jb;
    const int64_t pb0 = p0 + (it / nj) * 32;
    const int64_t p = pb0 + li;
    const float *crow = a.Bc + ((p < p1 ? p : pb0) * a.m + j) * int64_t(dl);
    // this lane's coefficients of terms tk0 + 8h .. + 7 (raw; masked once psi is known),
    // issued a chunk ahead of their use
    auto load_a = [&](int tk0, float (&r)[8]) {
      int tb = tk0 + 8 * h;
      if (a16) {  // dl a multiple of 8: a lane's eight terms lie all inside the row or all past it
        if (tb >= dl) tb = 0;  // past the row: values that the prefix mask zeroes
        const float4 u0 = *reinterpret_cast<const float4 *>(crow + tb);
        const float4 u1 = *reinterpret_cast<const float4 *>(crow + tb + 4);
        r[0] = u0.x; r[1] = u0.y; r[2] = u0.z; r[3] = u0.w;
        r[4] = u1.x; r[5] = u1.y; r[6] = u1.z; r[7] = u1.w;
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) r[i] = tb + i < dl ? crow[tb + i] : 0.f;
      }
    };
    float an[8];
    load_a(0, an);
    int lim = 0;  // psi*ell of pattern p (0 past the range)
    if (p < p1) {
      const int v = a.psi[p * a.m + j];
      lim = (v < 0 ? 0 : (v > a.delta ? a.delta : v)) * a.ell;
    }
    const unsigned long long sendm = __ballot(h == 0 && lim > 0);  // bit i: pattern pb0 + i sends
    int tmax = lim;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const int v = __shfl_xor(tmax, o, kWave);
      tmax = v > tmax ? v : tmax;
    }
    tmax = __builtin_amdgcn_readfirstlane(tmax);  // equal in every lane
    if (tmax == 0) continue;  // every pattern of the tile: a straggler, nothing sent
    v16f acc[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[nt][v] = 0.f;
    for (int tk0 = 0; tk0 < tmax; tk0 += kGrpTerms) {
      float av[8];
      int off[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) av[i] = an[i];
      load_a(tk0 + kGrpTerms, an);  // unconditional: in-row addresses, masked at use
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int tk = tk0 + 8 * h + i;
        const int o = tk < dl ? code[jb * dl + tk] : kGrpSkip;
        off[i] = o >= 0 ? o : 0;  // a padded slot (or past the row): any staged value, times 0
        av[i] = (tk < lim && o >= 0) ? av[i] : 0.f;  // lim <= dl
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const GT *src = Gs + off[i] + li;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          acc[nt] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], to_f32<GT>(src[32 * nt]), acc[nt], 0, 0,
                                                         0);
      }
    }
    // lane (h, li) holds D[8(v/4) + 4h + v%4][li] of each tile
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const int64_t x = x0 + 32 * nt + li;
      if (x >= a.L) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int pi = 8 * (v >> 2) + 4 * h + (v & 3);
        if ((sendm >> pi) & 1ull)
          __builtin_nontemporal_store(acc[nt][v], a.T + ((pb0 + pi) * a.m + j) * a.L + x);
      }
    }
  }
}

// The items of one staged slice on the matrix cores with (pattern, worker) rows: the 16 rows
// of the block (P_block patterns x J workers) against the K staged chunk-block slices,
// D[row][x] += A[row][k] B[k][x] four terms at a time (v_mfma_f32_16x16x4f32), A the
// coefficient tile built once per block (zero where a worker does not hold or has not
// processed a chunk), B the staged slices; each wave owns 32 positions (two 16-wide tiles).
template <typename GT>
__device__ __forceinline__ void group_mrows(const EncodeArgs &a, const GT *__restrict__ Gs,
                                            const float *__restrict__ Asm, int as, int Kp, uint32_t rsend,
                                            int64_t x0, int j0, int J, int64_t p0, int wave, int lane) {
  constexpr int W = kGrpWaves * 32;
  const int r16 = lane & 15, kq = lane >> 4;
  const int xw = wave * 32;
  v4f acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  const float *arow = Asm + r16 * as + kq;
  const GT *brow = Gs + kq * W + xw + r16;
  for (int ks = 0; ks < Kp; ks += 4) {
    const float av = arow[ks];
    const GT *bp = brow + ks * W;
    acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av, to_f32<GT>(bp[0]), acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av, to_f32<GT>(bp[16]), acc1, 0, 0, 0);
  }
  // lane (kq, r16) holds D[4 kq + v][r16] of each tile; rows that do not transmit are skipped
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int64_t x = x0 + xw + 16 * nt + r16;
    if (x >= a.L) continue;
    const v4f &acc = nt == 0 ? acc0 : acc1;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = 4 * kq + v;
      if ((rsend >> i) & 1u) {
        const int64_t row = (p0 + i / J) * a.m + j0 + i % J;
        __builtin_nontemporal_store(acc[v], a.T + row * a.L + x);
      }
    }
  }
}

// rows of staged slices in the matrix-rows layout: a multiple of 4 (zero rows pad K)
__host__ __device__ inline int mr_rows(int slots, int ell) { return (slots * ell + 3) & ~3; }

// LDS: [ G slices : slots*ell*W GT ][ code : J*delta*ell int32 ][ slot chunk : slots int32 ][ map : N int32 ]
// W = 64*VEC*NV: lane l owns x = x0 + (64u + l)*VEC + v for u < NV, v < VEC, so every
// load and store instruction of a wave covers 64*VEC consecutive positions.
template <typename GT, int VEC, int NV, int PB, bool MF = false, bool MR = false>
__global__ __launch_bounds__(kGrpThreads) __attribute__((amdgpu_waves_per_eu(MF ? 2 : 4))) void encode_group_kernel(
    EncodeArgs a, GroupArgs g) {
  constexpr int W = kWave * VEC * NV;
  static_assert(MF || (PB >= 1 && PB * kGrpTerms <= kWave), "PB rows of 16 terms fill at most one wave");
  static_assert(!MF || (W == 4 * 32 && PB == 32), "matrix cores: 32 patterns x 4 tiles of 32 positions");
  static_assert(!MR || W == kGrpWaves * 32, "matrix rows: each wave two tiles of 16 positions");
  extern __shared__ __align__(16) unsigned char lds[];
  GT *Gs = reinterpret_cast<GT *>(lds);
  const int grows = MR ? mr_rows(g.slots, a.ell) : g.slots * a.ell;  // staged slice rows
  const size_t gbytes = (size_t(grows) * W * sizeof(GT) + 15) & ~size_t(15);
  float *Asm = reinterpret_cast<float *>(lds + gbytes);  // MR: [16][grows + 1]
  const int as = grows + 1;
  const size_t abytes = MR ? sizeof(float) * 16 * size_t(as) : 0;
  // per staged row s*ell + k: element offset of block k of chunk slotc[s] in G, and the end
  // of that block's valid positions (min(L, d - k*L))
  int64_t *rdesc = reinterpret_cast<int64_t *>(lds + gbytes + abytes);
  int32_t *code = reinterpret_cast<int32_t *>(lds + gbytes + abytes + 2 * sizeof(int64_t) * size_t(grows));
  int32_t *slotc = code + g.J * a.delta * a.ell;
  int32_t *map = slotc + g.slots;  // [N] (dense)
  __shared__ int nslot, nuni;  // chunks staged; distinct chunks the group uses
  __shared__ uint32_t rsend;   // MR: bit r set when row r (pattern, worker) transmits

  // block -> (slice range, unit = (group, pattern range)).  Blocks are dispatched
  // round-robin over the 8 XCDs; XCD x takes ranges x, x + 8, ..., and the blocks of all
  // units of one range run back to back there, so its L2 serves the groups' overlapping
  // chunk slices.  A block walks its range slice by slice with its group's tables built once.
  const int64_t b = blockIdx.x;
  const int64_t units = int64_t(g.ngroups) * g.npr;
  const int64_t sr = (b & 7) + 8 * ((b >> 3) / units);
  const int64_t unit = (b >> 3) % units;
  const int64_t s_begin = sr * g.spb;
  const int64_t s_end = s_begin + g.spb < a.nslices ? s_begin + g.spb : a.nslices;
  if (s_begin >= s_end) return;  // the whole block: an empty range at the end
  const int gi = int(unit % g.ngroups);
  const int64_t pi = unit / g.ngroups;
  const int j0 = gi * g.J;
  const int nj = a.m - j0 < g.J ? a.m - j0 : g.J;
  const int64_t p0 = pi * g.PR;
  const int64_t p1 = p0 + g.PR < g.P ? p0 + g.PR : g.P;
  const int dl = a.delta * a.ell;

  if constexpr (MR)
    for (int e = threadIdx.x; e < 16 * as; e += kGrpThreads) Asm[e] = 0.f;
  // 1. which chunks the group uses, then slots in ascending chunk order
  if (g.dense) {
    for (int c = threadIdx.x; c < a.N; c += kGrpThreads) map[c] = 0;
    __syncthreads();
    for (int e = threadIdx.x; e < nj * a.delta; e += kGrpThreads) {
      const int c = a.order[int64_t(j0) * a.delta + e];  // rows j0.. of order are contiguous
      if (c >= 0 && c < a.N) map[c] = 1;
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
      int cnt = 0;
      for (int base = 0; base < a.N; base += kWave) {
        const int c = base + int(threadIdx.x);
        const bool on = c < a.N && map[c] != 0;
        const unsigned long long mask = __ballot(on);
        if (on) {
          const int s_ = cnt + __popcll(mask & ((1ull << threadIdx.x) - 1));
          map[c] = s_ < g.slots ? s_ : -1;
          if (s_ < g.slots) slotc[s_] = c;
        } else if (c < a.N) {
          map[c] = -1;
        }
        cnt += __popcll(mask);
      }
      if (threadIdx.x == 0) {
        nslot = cnt < g.slots ? cnt : g.slots;
        nuni = cnt;
      }
    }
    __syncthreads();
    // per (worker, term tk = t*ell + k): the LDS offset of block k of the chunk at
    // position t (>= 0), or -1 - (c*ell + k) for a chunk read through L2, or kGrpSkip for
    // a padded slot
    const int dlt = a.delta * a.ell;
    for (int e = threadIdx.x; e < nj * dlt; e += kGrpThreads) {
      const int jb = e / dlt, tk = e % dlt, t = tk / a.ell, k = tk % a.ell;
      const int c = a.order[int64_t(j0 + jb) * a.delta + t];
      int v = kGrpSkip;
      if (c >= 0 && c < a.N) v = map[c] >= 0 ? (map[c] * a.ell + k) * W : -1 - (c * a.ell + k);
      code[e] = v;
    }
  } else {
    // one worker (a worker's chunks are distinct): slot t holds position t
    for (int t = threadIdx.x; t < a.delta; t += kGrpThreads) {
      const int c = a.order[int64_t(j0) * a.delta + t];
      const bool ok = c >= 0 && c < a.N;
      if (t < g.slots) slotc[t] = ok ? c : 0;  // a padded slot stages chunk 0, never read
      for (int k = 0; k < a.ell; ++k)
        code[t * a.ell + k] = !ok ? kGrpSkip : (t < g.slots ? (t * a.ell + k) * W : -1 - (c * a.ell + k));
    }
    if (threadIdx.x == 0) {
      nslot = a.delta < g.slots ? a.delta : g.slots;
      nuni = a.delta;  // every position has a slot when delta <= slots (a padded one: chunk 0)
    }
    __syncthreads();
  }
  if constexpr (MR) {
    // the coefficient tile: row r = (pattern p0 + r / J, worker j0 + r % J), column
    // s*ell + k = block k of the chunk in slot s; zero where the worker does not hold the
    // chunk or has not processed it; and zero rows of slices past the staged ones
    __syncthreads();
    const int J = g.J;
    for (int e = threadIdx.x; e < 16 * a.delta; e += kGrpThreads) {
      const int r = e / a.delta, t = e % a.delta;
      const int pb = r / J, jb = r % J;
      if (p0 + pb >= p1 || jb >= nj) continue;
      const int64_t p = p0 + pb;
      const int j = j0 + jb;
      int v = a.psi[p * a.m + j];
      v = v < 0 ? 0 : (v > a.delta ? a.delta : v);
      const int c = a.order[int64_t(j) * a.delta + t];
      if (t >= v || c < 0 || c >= a.N) continue;
      const int u = g.dense ? map[c] : (t < g.slots ? t : -1);
      if (u < 0) continue;
      const float *src = a.Bc + ((p * a.m + j) * a.delta + t) * a.ell;
      for (int k = 0; k < a.ell; ++k) Asm[r * as + u * a.ell + k] = src[k];
    }
    const int K = nslot * a.ell, Kp = (K + 3) & ~3;
    for (int e = threadIdx.x; e < (Kp - K) * W; e += kGrpThreads) Gs[K * W + e] = GT(0);
    if (threadIdx.x < kWave) {
      bool on = false;
      const int r = int(threadIdx.x), pb = r / J, jb = r % J;
      if (r < 16 && p0 + pb < p1 && jb < nj) on = a.psi[(p0 + pb) * a.m + j0 + jb] > 0;
      const unsigned long long mask = __ballot(on);
      if (threadIdx.x == 0) rsend = uint32_t(mask);
    }
  }
  for (int row = threadIdx.x; row < nslot * a.ell; row += kGrpThreads) {
    const int sl = row / a.ell, k = row % a.ell;
    rdesc[2 * row] = int64_t(slotc[sl]) * a.d + int64_t(k) * a.L;
    const int64_t rem = a.d - int64_t(k) * a.L;
    rdesc[2 * row + 1] = rem < a.L ? rem : a.L;
  }
  __syncthreads();
  // 2. staging of a slice: Gs[(s*ell + k)*W + w] = g_{slotc[s]}[k*L + x0 + w] (zero past L
  // or d), 16 bytes per thread and step, all of it in registers first; where the compute
  // leaves room (PREF) the next slice's loads are issued before the current slice is
  // computed, else each slice is loaded and stored in turn
  const GT *G = reinterpret_cast<const GT *>(a.G);
  constexpr int SV = 16 / sizeof(GT);
  const int total = nslot * a.ell * W;
  uint4 buf[kGrpStage];
  // one pass covers kGrpStage * kGrpThreads * 16 bytes from element e0 on
  auto stage_load = [&](int64_t x0, int e0 = 0) {
#pragma unroll
    for (int u = 0; u < kGrpStage; ++u) {
      int e = e0 + (int(threadIdx.x) + u * kGrpThreads) * SV;
      // recomputed per slice rather than kept live through the compute
      asm volatile("" : "+v"(e));
      buf[u] = make_uint4(0u, 0u, 0u, 0u);
      if (e < total) {
        const int row = e / W, w = e % W;
        const int64_t x = x0 + w, lim = rdesc[2 * row + 1];
        const GT *src = G + rdesc[2 * row] + x;
        if (a.stage16 && x + SV <= lim)
          buf[u] = *reinterpret_cast<const uint4 *>(src);
        else
          buf[u] = load16_lim(src, x, lim);
      }
    }
  };
  auto stage_store = [&](int e0 = 0) {
#pragma unroll
    for (int u = 0; u < kGrpStage; ++u) {
      const int e = e0 + (int(threadIdx.x) + u * kGrpThreads) * SV;
      if (e < total) *reinterpret_cast<uint4 *>(Gs + e) = buf[u];
    }
  };
  constexpr bool PREF = !MF && PB * NV * VEC <= 16;
  if constexpr (PREF) stage_load(s_begin * W);

  // 3. items (pattern batch, worker), worker fastest: the waves write neighbouring rows
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
  const int lane = threadIdx.x % kWave;
  for (int64_t slice = s_begin; slice < s_end; ++slice) {
  const int64_t x0 = slice * W;
  __syncthreads();  // tables built; the previous slice's terms all applied
  if constexpr (!PREF) {
    for (int e0 = 0; e0 < total; e0 += kGrpStage * kGrpThreads * SV) {
      stage_load(x0, e0);
      stage_store(e0);
    }
  } else {
    stage_store();
  }
  __syncthreads();
  if constexpr (PREF) {
    if (slice + 1 < s_end) stage_load(x0 + W);
  }
  if constexpr (MF) {
    if (nslot > 0 && nuni <= nslot)
      group_mfma<GT>(a, Gs, code, x0, j0, nj, p0, p1, wave, lane);
    else  // a union past the slots (orders other than the cyclic one): the vector layout
      group_vector<GT, 2, 1, 4>(a, Gs, code, x0, j0, nj, p0, p1, wave, lane);
  } else if constexpr (MR) {
    if (nslot > 0 && nuni <= nslot)
      group_mrows<GT>(a, Gs, Asm, as, (nslot * a.ell + 3) & ~3, rsend, x0, j0, g.J, p0, wave, lane);
    else
      group_vector<GT, VEC, NV, PB>(a, Gs, code, x0, j0, nj, p0, p1, wave, lane);
  } else {
    group_vector<GT, VEC, NV, PB>(a, Gs, code, x0, j0, nj, p0, p1, wave, lane);
  }
  }  // slice
}

// Sizes of the worker-group layout for a slice width W: the group J (for the cyclic
// union of J + delta - 1 chunks), the slice capacity, the patterns per block (staged bytes
// at most an eighth of those written, where the patterns allow).  Returns the ratio of
// staged to written bytes, or a negative value when the layout does not fit.
double plan_group(const EncodeArgs &a, int64_t P, int64_t W, size_t esize, int pb, GroupArgs &g,
                  size_t &lds, size_t budget = kGrpLds) {
  const int64_t sb = int64_t(a.ell) * W * int64_t(esize);  // one chunk's slices
  const int64_t B = int64_t(budget) - 16;
  const int64_t dm1 = a.delta - 1;
  // the dense chunk map needs 4N bytes; past a quarter of the budget, single-worker
  // groups, whose slots need no map
  g.dense = 4 * int64_t(a.N) <= (int64_t(kGrpLds) - 16) / 4 ? 1 : 0;
  const int64_t mapw = g.dense ? a.N : 0;
  const int64_t dl = int64_t(a.delta) * a.ell;  // table words per worker
  int64_t J = g.dense ? (B - 4 * mapw - (sb + 4 + 16 * a.ell) * dm1) / (sb + 4 + 16 * a.ell + 4 * dl) : 1;
  if (J > a.m) J = a.m;
  if (J < 1) J = 1;
  g.ngroups = int(ceil_div(a.m, J));
  J = ceil_div(a.m, g.ngroups);  // balanced groups
  int64_t slots = (B - 4 * (J * dl + mapw)) / (sb + 4 + 16 * a.ell);
  const int64_t most = J * a.delta < a.N ? J * a.delta : a.N;
  if (slots > most) slots = most;
  if (slots < 1) return -1.0;
  const int64_t uni = J + dm1 < slots ? J + dm1 : slots;
  int64_t pr = ceil_div(8 * uni * sb, J * W * 4);
  pr = ceil_div(pr < 1 ? 1 : pr, pb) * pb;
  if (pr > P) pr = P;
  g.J = int(J);
  g.PR = pr;
  g.npr = ceil_div(P, pr);
  g.slots = int(slots);
  g.P = P;
  lds = ((size_t(sb) * slots + 15) & ~size_t(15)) + 2 * sizeof(int64_t) * size_t(slots) * a.ell +
        sizeof(int32_t) * size_t(J * dl + slots + mapw);
  if (lds > budget) return -1.0;
  return double(uni * sb) / double(J * pr * W * 4);
}

// Sizes of the matrix-rows layout (fewer than 32 patterns per call, many terms): 16 rows of
// (pattern, worker) per block, P_block = min(P, 16) patterns by J = 16 / P_block workers; the
// cyclic union of the group's chunks must fit, with the coefficient tile, in the LDS budget.
bool plan_rows(const EncodeArgs &a, int64_t P, size_t esize, GroupArgs &g, size_t &lds) {
  const int64_t W = kGrpWaves * 32;
  const int64_t sb = int64_t(a.ell) * W * int64_t(esize);
  const int64_t B = int64_t(kGrpLds) - 16;
  const int pblk = P < 16 ? int(P) : 16;
  int64_t J = 16 / pblk;
  if (J > a.m) J = a.m;
  g.dense = 4 * int64_t(a.N) <= B / 4 ? 1 : 0;
  if (!g.dense) J = 1;
  g.ngroups = int(ceil_div(a.m, J));
  J = ceil_div(a.m, g.ngroups);  // balanced groups
  const int64_t dl = int64_t(a.delta) * a.ell, mapw = g.dense ? a.N : 0;
  // per slot: its slices, its coefficient columns, its slot word; fixed: the per-term table,
  // the map, the tile's padding column and up to three zero rows of slices
  const int64_t fixed = 4 * (J * dl + mapw) + 16 * 4 * 4 + 3 * (W * int64_t(esize) + 16);
  int64_t slots = (B - fixed) / (sb + 64 * a.ell + 16 * a.ell + 4);
  const int64_t most = J * a.delta < a.N ? J * a.delta : a.N;
  if (slots > most) slots = most;
  const int64_t need = J + a.delta - 1 < a.N ? J + a.delta - 1 : a.N;
  if (slots < need || slots < 1) return false;
  g.J = int(J);
  g.PR = pblk;
  g.npr = ceil_div(P, pblk);
  g.slots = int(slots);
  g.P = P;
  const int gr = mr_rows(int(slots), a.ell);
  lds = ((size_t(gr) * W * esize + 15) & ~size_t(15)) + sizeof(float) * 16 * size_t(gr + 1) +
        2 * sizeof(int64_t) * size_t(gr) + sizeof(int32_t) * size_t(J * dl + slots + mapw);
  return lds <= kGrpLds;
}

template <typename GT, int VEC, int NV, int PB, bool MF = false, bool MR = false>
int launch_group(const EncodeArgs &a, const GroupArgs &g, size_t lds, hipStream_t st) {
  const int64_t blocks = g.nsr * g.ngroups * g.npr;
  if (!grid_ok(blocks, kGrpThreads)) return GC_EINVAL;
  if (hipFuncSetAttribute(reinterpret_cast<const void *>(&encode_group_kernel<GT, VEC, NV, PB, MF, MR>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
    return GC_ELAUNCH;
  hipLaunchKernelGGL((encode_group_kernel<GT, VEC, NV, PB, MF, MR>), dim3(unsigned(blocks)),
                     dim3(kGrpThreads), lds, st, a, g);
  return GC_OK;
}

// Candidate slice widths, widest first: (VEC, NV) = (4,4), (4,2), (4,1), (2,1), (1,1), i.e.
// rows of 4 KB down to 256 B per wave, as far as the row length and T's alignment allow.
// The widest candidate that stages the cyclic union of its group's chunks is taken (measured
// on MI355X, wider rows always won once the union fits; a union that spills to L2 reads
// costs 2-10x), else the narrowest.
constexpr int kGrpCand = 5;
constexpr int kGrpVec[kGrpCand] = {4, 4, 4, 2, 1};
constexpr int kGrpNv[kGrpCand] = {4, 2, 1, 1, 1};

int pick_group(const EncodeArgs &a, int64_t P, int vec, size_t esize, GroupArgs &g, size_t &lds) {
  int pick = -1;
  for (int i = 0; i < kGrpCand; ++i) {
    if (kGrpVec[i] > vec) continue;
    GroupArgs gi{};
    size_t li = 0;
    if (plan_group(a, P, int64_t(kWave) * kGrpVec[i] * kGrpNv[i], esize, P >= 4 ? 4 : 2, gi, li) < 0)
      continue;
    g = gi;
    lds = li;
    pick = i;
    const int64_t uni = int64_t(gi.J) + a.delta - 1 < a.N ? int64_t(gi.J) + a.delta - 1 : a.N;
    if (gi.slots >= uni) break;
  }
  return pick;
}

template <typename GT, int VEC>
int launch_encode_group(EncodeArgs a, int64_t P, hipStream_t st) {
  GroupArgs g{};
  size_t lds = 0;
  // the matrix cores when a call has a full 32-pattern tile and at least 32 terms per
  // output, and the cyclic union of a group's chunks fits 128 positions wide
  bool mf = false;
  if (P >= 32 && a.delta * a.ell >= 32) {
    GroupArgs gm{};
    size_t lm = 0;
    if (plan_group(a, P, 128, sizeof(GT), 32, gm, lm, kGrpLdsMF) >= 0) {
      const int64_t uni = int64_t(gm.J) + a.delta - 1 < a.N ? int64_t(gm.J) + a.delta - 1 : a.N;
      if (gm.slots >= uni) {
        g = gm;
        lds = lm;
        mf = true;
      }
    }
  }
  // fewer patterns per call: the matrix cores with (pattern, worker) rows, 256 positions wide
  bool mr = false;
  if (!mf && P < 32 && a.delta * a.ell >= 32) {
    GroupArgs gr{};
    size_t lr = 0;
    if (plan_rows(a, P, sizeof(GT), gr, lr)) {
      g = gr;
      lds = lr;
      mr = true;
    }
  }
  const int c = (mf || mr) ? -1 : pick_group(a, P, VEC, sizeof(GT), g, lds);
  if (!mf && !mr && c < 0) return GC_EINVAL;
  const int64_t W = mf ? 128 : (mr ? int64_t(kGrpWaves) * 32 : int64_t(kWave) * kGrpVec[c] * kGrpNv[c]);
  a.nslices = int(ceil_div(a.L, W));
  // enough work units to fill the chip: fewer patterns per block while they are short
  const int pb = mf ? 32 : (mr ? int(g.PR) : (P >= 4 ? 4 : 2));
  const int64_t want = 128 * int64_t(cu_count());  // blocks: about 64 rounds of resident ones
  while (a.nslices * g.ngroups * g.npr < want / 2 && g.PR > pb) {
    g.PR = ceil_div(g.PR / 2, pb) * pb;
    g.npr = ceil_div(P, g.PR);
  }
  // slice ranges: a multiple of 8 (one share per XCD), about `want` blocks in all
  const int64_t units = int64_t(g.ngroups) * g.npr;
  int64_t nsr = ceil_div(ceil_div(want, units), 8) * 8;
  if (nsr > ceil_div(a.nslices, 8) * 8) nsr = ceil_div(a.nslices, 8) * 8;
  g.spb = ceil_div(a.nslices, nsr);
  g.nsr = ceil_div(ceil_div(a.nslices, g.spb), 8) * 8;
  if (mf) return launch_group<GT, 2, 1, 32, true>(a, g, lds, st);
  if (mr)
    return P >= 4 ? launch_group<GT, 1, 4, 4, false, true>(a, g, lds, st)
                  : launch_group<GT, 1, 4, 2, false, true>(a, g, lds, st);
  const bool pb4 = P >= 4;
  if constexpr (VEC == 4) {
    if (c == 0)
      return pb4 ? launch_group<GT, 4, 4, 4>(a, g, lds, st) : launch_group<GT, 4, 4, 2>(a, g, lds, st);
    if (c == 1)
      return pb4 ? launch_group<GT, 4, 2, 4>(a, g, lds, st) : launch_group<GT, 4, 2, 2>(a, g, lds, st);
    if (c == 2)
      return pb4 ? launch_group<GT, 4, 1, 4>(a, g, lds, st) : launch_group<GT, 4, 1, 2>(a, g, lds, st);
  }
  if constexpr (VEC >= 2) {
    if (c == 3)
      return pb4 ? launch_group<GT, 2, 1, 4>(a, g, lds, st) : launch_group<GT, 2, 1, 2>(a, g, lds, st);
  }
  return pb4 ? launch_group<GT, 1, 1, 4>(a, g, lds, st) : launch_group<GT, 1, 1, 2>(a, g, lds, st);
}

template <typename GT, int VEC>
int launch_encode(EncodeArgs a, hipStream_t st) {
  constexpr int W = kWave * VEC;
  a.nslices = int(ceil_div(a.L, W));
  a.term_stride = (a.delta * a.ell + 3) & ~3;
  const size_t gbytes = size_t(a.N * a.ell + 1) * W * sizeof(GT);
  const size_t per_row = sizeof(int32_t) + (sizeof(int32_t) + sizeof(float)) * a.term_stride;
  int group = int(kEncMetaLds / per_row);
  if (group > kEncGroup) group = kEncGroup;
  if (group < 1) group = 1;
  // runs of a few hundred rows: long enough to amortise the slice staging, short enough
  // that the blocks in flight keep a compact write front (longer only where the grid
  // would otherwise exceed the launch limits)
  const int64_t max_blocks = 0xffffffffLL / kEncThreads;
  int64_t rblocks = ceil_div(a.rows, int64_t(group) * kEncGroupsPerBlock);
  if (rblocks * a.nslices > max_blocks) rblocks = max_blocks / a.nslices;
  if (rblocks < 1) return GC_EINVAL;
  a.rows_per_block = ceil_div(a.rows, rblocks);
  if (a.rows_per_block < group) group = int(a.rows_per_block);
  a.group_rows = group;
  rblocks = ceil_div(a.rows, a.rows_per_block);
  const int64_t blocks = rblocks * a.nslices;
  if (!grid_ok(blocks, kEncThreads)) return GC_EINVAL;
  const size_t lds = gbytes + sizeof(int32_t) * ((group + 3) & ~3) +
                     (sizeof(int32_t) + sizeof(float)) * a.term_stride * size_t(group);
  if (hipFuncSetAttribute(reinterpret_cast<const void *>(&encode_kernel<GT, VEC>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
    return GC_ELAUNCH;
  hipLaunchKernelGGL((encode_kernel<GT, VEC>), dim3(unsigned(blocks)), dim3(kEncThreads), lds, st, a);
  return GC_OK;
}

template <typename GT>
int dispatch_encode(const EncodeArgs &a, int64_t P, int vec, bool all_chunks, hipStream_t st) {
  if (all_chunks)
    return vec == 4 ? launch_encode<GT, 4>(a, st)
                    : (vec == 2 ? launch_encode<GT, 2>(a, st) : launch_encode<GT, 1>(a, st));
  return vec == 4 ? launch_encode_group<GT, 4>(a, P, st)
                  : (vec == 2 ? launch_encode_group<GT, 2>(a, P, st) : launch_encode_group<GT, 1>(a, P, st));
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
  // G [N][d], Bc [P][m][delta][ell], T [P][m][L]
  if (!sizes_ok({N, d}) || !sizes_ok({P, m, delta, ell}) || !sizes_ok({P, m, ceil_div(d, ell)}))
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
  // widest vector the row length and the alignment of T allow; the all-chunk layout
  // when the slice of every chunk fits in LDS at that width, else the worker groups
  const size_t esize = g_dtype == GC_F32 ? 4 : 2;
  const uintptr_t ta = reinterpret_cast<uintptr_t>(T), ga = reinterpret_cast<uintptr_t>(G);
  const int64_t sv = int64_t(16 / esize);
  a.stage16 = d % sv == 0 && a.L % sv == 0 && (ga & 15) == 0;
  const int vec = (a.L % 4 == 0 && (ta & 15) == 0) ? 4 : ((a.L % 2 == 0 && (ta & 7) == 0) ? 2 : 1);
  const bool all_chunks = size_t(N) * ell * kWave * vec * esize <= kEncSliceLds;
  (void)hipGetLastError();
  // beyond the all-chunk layout, the bf16 matrix cores where they fit: always for bf16 chunk
  // gradients; for fp32 ones from kMxF32Terms terms per output on
  if (!all_chunks && (g_dtype == GC_BF16 || delta * ell >= kMxF32Terms)) {
    const int st = encode_mx(G, g_dtype == GC_F32, N, d, psi, order, Bc, P, m, delta, ell, T, stream);
    if (st != kEncodeMxNotApplicable) return st != GC_OK ? st : launch_status();
  }
  const int st = g_dtype == GC_F32 ? dispatch_encode<float>(a, P, vec, all_chunks, stream)
                                   : dispatch_encode<uint16_t>(a, P, vec, all_chunks, stream);
  if (st != GC_OK) return st;
  return launch_status();
}
