// Host driver for the sanitizer build of libgcx (address and undefined-behaviour checks on
// the host side of the C ABI).  Runs without a GPU: the host-only entry points with valid
// and invalid input, every device entry point's argument validation, and the device entry
// points with valid arguments up to their device check (no device: a non-OK status, nothing
// launched).  Prints "ok" and returns 0 when every check holds.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <vector>

#include "gcx.h"

static int failures = 0;

#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

// a small deterministic generator (no library state)
static uint64_t lcg_state = 88172645463325252ull;
static uint32_t next_u32() {
  lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
  return uint32_t(lcg_state >> 33);
}

struct Tables {
  std::vector<int32_t> O, order, holder, hpos;
  Tables(int N, int m, int delta, int gamma)
      : O(size_t(N) * m, 0), order(size_t(m) * delta), holder(size_t(N) * gamma), hpos(size_t(N) * gamma) {}
};

static int assign(int kind, int N, int m, int s, int delta, int gamma, Tables &t, bool pass_O = true) {
  return gc_assign(kind, N, m, s, pass_O ? t.O.data() : nullptr, delta, gamma, t.order.data(),
                   t.holder.data(), t.hpos.data());
}

// order/holder/hpos agree with O: order[j][O_ij - 1] = i, and (holder, hpos) list O's column
static bool consistent(const Tables &t, int N, int m, int delta, int gamma) {
  for (int j = 0; j < m; ++j)
    for (int i = 0; i < N; ++i) {
      const int o = t.O[size_t(i) * m + j];
      if (o > 0 && t.order[size_t(j) * delta + o - 1] != i) return false;
    }
  for (int i = 0; i < N; ++i) {
    int u = 0;
    for (int j = 0; j < m; ++j) {
      const int o = t.O[size_t(i) * m + j];
      if (o == 0) continue;
      if (u >= gamma || t.holder[size_t(i) * gamma + u] != j || t.hpos[size_t(i) * gamma + u] != o - 1)
        return false;
      ++u;
    }
    for (; u < gamma; ++u)
      if (t.holder[size_t(i) * gamma + u] != -1) return false;
  }
  return true;
}

static void host_entry_points() {
  CHECK(gc_version() >= 100);
  for (int st = -6; st <= 2; ++st) CHECK(gc_strerror(st) != nullptr && std::strlen(gc_strerror(st)) > 0);

  // cyclic tables at the workloads' sizes
  const int cyc[][2] = {{1, 0}, {3, 1}, {6, 2}, {20, 3}, {50, 4}, {100, 9}, {200, 19}, {9, 8}};
  for (const auto &c : cyc) {
    const int m = c[0], s = c[1], dl = s + 1;
    Tables t(m, m, dl, dl);
    CHECK(assign(GC_ASSIGN_CYCLIC, m, m, s, dl, dl, t) == GC_OK);
    CHECK(consistent(t, m, m, dl, dl));
    for (int j = 0; j < m; ++j)
      for (int u = 0; u < dl; ++u) CHECK(t.order[size_t(j) * dl + u] == (j + u) % m);
    Tables t2(m, m, dl, dl);
    CHECK(assign(GC_ASSIGN_CYCLIC, m, m, s, dl, dl, t2, false) == GC_OK);  // O not requested
  }

  // random orderings through GC_ASSIGN_ORDER, then their Q metric
  for (int rep = 0; rep < 200; ++rep) {
    const int N = 1 + int(next_u32() % 12), m = 1 + int(next_u32() % 12);
    std::vector<int32_t> O(size_t(N) * m, 0);
    int delta = 1, gamma = 1;
    for (int j = 0; j < m; ++j) {
      int pos = 0;
      for (int i = 0; i < N; ++i)
        if (next_u32() % 10 < 4) O[size_t(i) * m + j] = ++pos;
      // shuffle the positions among the column's chunks
      for (int i = N - 1; i > 0; --i) {
        const int k = int(next_u32() % uint32_t(i + 1));
        if (O[size_t(i) * m + j] && O[size_t(k) * m + j]) std::swap(O[size_t(i) * m + j], O[size_t(k) * m + j]);
      }
      delta = pos > delta ? pos : delta;
    }
    for (int i = 0; i < N; ++i) {
      int g = 0;
      for (int j = 0; j < m; ++j) g += O[size_t(i) * m + j] ? 1 : 0;
      gamma = g > gamma ? g : gamma;
    }
    Tables t(N, m, delta, gamma);
    t.O = O;
    CHECK(assign(GC_ASSIGN_ORDER, N, m, -1, delta, gamma, t) == GC_OK);
    CHECK(consistent(t, N, m, delta, gamma));
    std::vector<int64_t> Q(N);
    int64_t qmax = -1;
    CHECK(gc_qmax(O.data(), N, m, Q.data(), &qmax) == GC_OK);
    CHECK(qmax >= 0);
    CHECK(gc_qmax(O.data(), N, m, nullptr, &qmax) == GC_OK);
  }

  // Algorithm 2 on circulant delta-regular supports: every row of O sums to delta(delta+1)/2
  const int reg[][2] = {{4, 2}, {10, 3}, {50, 5}, {200, 8}, {300, 8}};
  for (const auto &r : reg) {
    const int m = r[0], dl = r[1];
    Tables t(m, m, dl, dl);
    for (int j = 0; j < m; ++j)
      for (int u = 0; u < dl; ++u) t.O[size_t((j + 3 * u) % m) * m + j] = 1;  // a support, not an order
    bool regular = true;  // (j + 3u) mod m distinct for u < dl when m is not divisible by 3 below dl*3
    for (int i = 0; i < m; ++i) {
      int g = 0;
      for (int j = 0; j < m; ++j) g += t.O[size_t(i) * m + j] ? 1 : 0;
      regular = regular && g == dl;
    }
    if (!regular) continue;
    CHECK(assign(GC_ASSIGN_REGULAR, m, m, -1, dl, dl, t) == GC_OK);
    CHECK(consistent(t, m, m, dl, dl));
    for (int i = 0; i < m; ++i) {
      int sum = 0;
      for (int j = 0; j < m; ++j) sum += t.O[size_t(i) * m + j];
      CHECK(sum == dl * (dl + 1) / 2);
    }
  }

  // invalid assignments
  {
    Tables t(6, 6, 3, 3);
    CHECK(assign(GC_ASSIGN_CYCLIC, 5, 6, 1, 2, 2, t) == GC_EINVAL);   // N != m
    CHECK(assign(GC_ASSIGN_CYCLIC, 5, 5, 5, 6, 6, t) == GC_EINVAL);   // s >= m
    CHECK(assign(GC_ASSIGN_CYCLIC, 5, 5, 1, 3, 2, t) == GC_EINVAL);   // delta != s + 1
    CHECK(assign(GC_ASSIGN_CYCLIC, 5, 5, -1, 0, 0, t) == GC_EINVAL);  // s < 0
    CHECK(assign(7, 5, 5, 1, 2, 2, t) == GC_EINVAL);                  // unknown kind
    CHECK(assign(GC_ASSIGN_ORDER, 3, 3, -1, 2, 2, t, false) == GC_EINVAL);  // O missing
    CHECK(gc_assign(GC_ASSIGN_CYCLIC, 3, 3, 1, nullptr, 2, 2, nullptr, t.holder.data(), t.hpos.data()) ==
          GC_EINVAL);
    Tables b(3, 3, 3, 3);
    const int32_t dup[9] = {1, 0, 0, 1, 0, 0, 0, 0, 0};  // two chunks at position 1
    std::memcpy(b.O.data(), dup, sizeof dup);
    CHECK(assign(GC_ASSIGN_ORDER, 3, 3, -1, 3, 3, b) == GC_EINVAL);
    const int32_t gap[9] = {1, 0, 0, 3, 0, 0, 0, 0, 0};  // positions 1 and 3
    std::memcpy(b.O.data(), gap, sizeof gap);
    CHECK(assign(GC_ASSIGN_ORDER, 3, 3, -1, 3, 3, b) == GC_EINVAL);
    const int32_t neg[9] = {-1, 0, 0, 0, 0, 0, 0, 0, 0};
    std::memcpy(b.O.data(), neg, sizeof neg);
    CHECK(assign(GC_ASSIGN_ORDER, 3, 3, -1, 3, 3, b) == GC_EINVAL);
    const int32_t big[9] = {9, 0, 0, 0, 0, 0, 0, 0, 0};
    std::memcpy(b.O.data(), big, sizeof big);
    CHECK(assign(GC_ASSIGN_ORDER, 3, 3, -1, 3, 3, b) == GC_EINVAL);
    Tables n(3, 3, 1, 2);
    const int32_t wide[9] = {1, 1, 1, 0, 0, 0, 0, 0, 0};  // gamma 3 > table width 2
    std::memcpy(n.O.data(), wide, sizeof wide);
    CHECK(assign(GC_ASSIGN_ORDER, 3, 3, -1, 1, 2, n) == GC_EINVAL);
    Tables irr(5, 5, 1, 1);
    for (int i = 0; i < 5; ++i) irr.O[size_t(i) * 5 + i] = 1;
    irr.O[1] = 1;  // row 0 of degree 2
    CHECK(assign(GC_ASSIGN_REGULAR, 5, 5, -1, 1, 1, irr) == GC_EINVAL);
    int64_t q = 0;
    CHECK(gc_qmax(b.O.data(), 3, 3, nullptr, &q) == GC_EINVAL);       // position 9 > load
    CHECK(gc_qmax(nullptr, 3, 3, nullptr, &q) == GC_EINVAL);
    CHECK(gc_qmax(b.O.data(), 3, 3, nullptr, nullptr) == GC_EINVAL);
    CHECK(gc_qmax(b.O.data(), 0, 3, nullptr, &q) == GC_EINVAL);
  }
}

static void workspace_sizes() {
  const int64_t big64 = std::numeric_limits<int64_t>::max();
  const int32_t big32 = std::numeric_limits<int32_t>::max();
  const int32_t ns[] = {-1, 0, 1, 50, big32};
  const int64_t ds[] = {-1, 0, 1, 16384, 1 << 24, big64};
  for (int32_t N : ns)
    for (int64_t d : ds) {
      (void)gc_chunk_grads_workspace_size(N, N, d, 1);
      (void)gc_chunk_grads_workspace_size(N, 512, d, 256);
      (void)gc_reconstruct_workspace_size(int64_t(N), 50, d, 1);
      (void)gc_reconstruct_workspace_size(big64, N, d, 8);
      (void)gc_decode_direct_workspace_size(int64_t(N), N, d, 1);
      (void)gc_decode_direct_workspace_size(big64, N, d, 8);
    }
  CHECK(gc_reconstruct_workspace_size(10000, 50, 16384, 1) == 8u * 10000 * 4);
}

static void device_validation() {
  void *p = reinterpret_cast<void *>(uintptr_t(256));  // never dereferenced
  const float *fp = static_cast<const float *>(p);
  float *fo = static_cast<float *>(p);
  const int32_t *ip = static_cast<const int32_t *>(p);
  int32_t *io = static_cast<int32_t *>(p);
  uint8_t *u8 = static_cast<uint8_t *>(p);
  double *dp = static_cast<double *>(p);
  const int E = GC_EINVAL;

  // chunk gradients
  CHECK(gc_chunk_grads(fp, fp, fp, 2, 3, 8, 1, 5, fo, p, 1 << 20, nullptr) == E);  // loss
  CHECK(gc_chunk_grads(fp, fp, fp, 2, 3, 8, 1, 0, fo, p, 4, nullptr) == E);        // small ws
  CHECK(gc_chunk_grads(nullptr, fp, fp, 2, 3, 8, 1, 0, fo, p, 1 << 20, nullptr) == E);
  CHECK(gc_chunk_grads(fp, fp, fp, 0, 3, 8, 1, 0, fo, p, 1 << 20, nullptr) == E);   // N = 0
  CHECK(gc_chunk_grads(fp, fp, fp, 2, 3, -8, 1, 0, fo, p, 1 << 20, nullptr) == E);  // d < 0
  CHECK(gc_chunk_grads(fp, fp, fp, 2, 3, 8, 0, 0, fo, p, 1 << 20, nullptr) == E);   // b = 0
  CHECK(gc_sum_chunks(p, 3, 2, 8, fo, nullptr) == E);
  CHECK(gc_sum_chunks(nullptr, GC_F32, 2, 8, fo, nullptr) == E);
  CHECK(gc_sum_chunks(p, GC_F32, 2, 0, fo, nullptr) == E);

  // coefficients
  CHECK(gc_decode_coeffs(ip, 4, 6, 0, ip, 3, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) == E);     // m = 0
  CHECK(gc_decode_coeffs(ip, 4, 6, 6, ip, 3, ip, ip, 3, fp, 9, io, u8, io, fo, nullptr) == E);     // ell > 8
  CHECK(gc_decode_coeffs(ip, 4, 6, 6, ip, 3, ip, ip, 3, fp, 0, io, u8, io, fo, nullptr) == E);     // ell = 0
  CHECK(gc_decode_coeffs(nullptr, 4, 6, 6, ip, 3, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) == E);  // psi
  CHECK(gc_decode_coeffs(ip, 4, 6, 2000, ip, 3, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) == E);  // m big
  CHECK(gc_decode_coeffs(ip, -1, 6, 6, ip, 3, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) == E);    // P < 0
  CHECK(gc_decode_coeffs(ip, 4, 6, 6, ip, 99, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) == E);    // delta
  CHECK(gc_decode_coeffs(ip, 4, 6, 6, ip, 3, ip, ip, 99, fp, 1, io, u8, io, fo, nullptr) == E);    // gamma
  CHECK(gc_decode_coeffs(ip, 0, 6, 6, ip, 3, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) == GC_OK);  // P = 0

  // encode
  CHECK(gc_encode(p, 5, 6, 64, ip, ip, fp, 4, 6, 3, 1, fo, nullptr) == E);        // dtype
  CHECK(gc_encode(p, GC_F32, 6, 0, ip, ip, fp, 4, 6, 3, 1, fo, nullptr) == E);    // d = 0
  CHECK(gc_encode(nullptr, GC_F32, 6, 64, ip, ip, fp, 4, 6, 3, 1, fo, nullptr) == E);
  CHECK(gc_encode(p, GC_F32, 6, 64, ip, ip, fp, 4, 6, 3, 9, fo, nullptr) == E);   // ell
  CHECK(gc_encode(p, GC_F32, 6, 64, ip, ip, fp, 4, 6, 0, 1, fo, nullptr) == E);   // delta
  CHECK(gc_encode(p, GC_F32, 6, 64, ip, ip, fp, 4, 6, 3, 1, nullptr, nullptr) == E);  // T
  CHECK(gc_encode(p, GC_F32, 6, 64, ip, ip, fp, 0, 6, 3, 1, fo, nullptr) == GC_OK);   // P = 0

  // combine, with and without a workspace
  CHECK(gc_reconstruct(fp, fp, ip, 4, 6, 64, 0, fo, nullptr, nullptr, nullptr, 0, nullptr) == E);  // ell
  CHECK(gc_reconstruct(fp, fp, ip, 4, 6, 64, 1, fo, nullptr, dp, nullptr, 0, nullptr) == E);       // gsum
  CHECK(gc_reconstruct(fp, fp, ip, 4, 6, 1 << 20, 1, nullptr, fp, dp, nullptr, 0, nullptr) == E);  // ws
  CHECK(gc_reconstruct(fp, fp, nullptr, 4, 6, 64, 1, fo, nullptr, nullptr, nullptr, 0, nullptr) == E);  // psi
  CHECK(gc_reconstruct(fp, fp, ip, 4, 6, 64, 1, nullptr, nullptr, nullptr, nullptr, 0, nullptr) == GC_OK);
  CHECK(gc_reconstruct_noalloc(fp, fp, ip, 1000, 4, 1 << 24, 1, nullptr, fp, dp, nullptr) == GC_ESCRATCH);
  CHECK(gc_reconstruct_noalloc(fp, fp, nullptr, 4, 6, 64, 1, fo, nullptr, nullptr, nullptr) == E);
  CHECK(gc_reconstruct_noalloc(fp, fp, ip, 4, 6, 64, 9, fo, nullptr, nullptr, nullptr) == E);

  // PS-side estimate
  const size_t ws = gc_decode_direct_workspace_size(4, 6, 64, 1);
  CHECK(gc_decode_direct(p, GC_F32, 6, 64, ip, 4, 6, 3, ip, ip, 3, fp, 0, fo, nullptr, nullptr, p, ws,
                         nullptr) == E);  // ell
  CHECK(gc_decode_direct(p, 3, 6, 64, ip, 4, 6, 3, ip, ip, 3, fp, 1, fo, nullptr, nullptr, p, ws, nullptr) ==
        E);  // dtype
  CHECK(gc_decode_direct(p, GC_F32, 6, 64, ip, 4, 6, 3, ip, ip, 3, fp, 1, nullptr, nullptr, nullptr, p, ws,
                         nullptr) == E);  // no output
  CHECK(gc_decode_direct(p, GC_F32, 6, 64, ip, 4, 6, 3, ip, ip, 3, fp, 1, fo, nullptr, dp, p, ws, nullptr) ==
        E);  // sqerr without gsum
  CHECK(gc_decode_direct(p, GC_F32, 6, 64, ip, 4, 6, 3, ip, ip, 3, fp, 1, fo, nullptr, nullptr, p, ws - 1,
                         nullptr) == E);  // workspace
  CHECK(gc_decode_direct(p, GC_F32, 6, 64, ip, 4, 6, 3, ip, ip, 3, fp, 1, fo, nullptr, nullptr,
                         static_cast<char *>(p) + 4, ws, nullptr) == E);  // unaligned workspace
  CHECK(gc_decode_direct(p, GC_F32, 6, 64, ip, 0, 6, 3, ip, ip, 3, fp, 1, fo, nullptr, nullptr, p, ws,
                         nullptr) == GC_OK);  // P = 0

  // simulations
  CHECK(gc_progress(static_cast<const double *>(p), nullptr, 4, 0, 3, dp, 5, io, nullptr) == E);  // m = 0
  CHECK(gc_progress(nullptr, nullptr, 4, 6, 3, dp, 5, io, nullptr) == E);
  CHECK(gc_completion_times(static_cast<const double *>(p), nullptr, 4, 6, 6, 3, ip, ip, 3, 0, dp, dp,
                            nullptr) == E);  // ell = 0
  CHECK(gc_completion_times(nullptr, nullptr, 4, 6, 6, 3, ip, ip, 3, 1, dp, dp, nullptr) == E);
  CHECK(gc_original_ls(nullptr, 4, 6, 6, ip, 3, ip, 3, 100, 1e-12, dp, io, nullptr) == E);
  CHECK(gc_original_ls(ip, 4, 6, 6, ip, 3, ip, 3, 100, 1e-12, nullptr, io, nullptr) == E);
}

// sizes whose buffers could not exist: rejected on the host, with no overflow on the way
static void extreme_sizes() {
  void *p = reinterpret_cast<void *>(uintptr_t(256));
  const float *fp = static_cast<const float *>(p);
  float *fo = static_cast<float *>(p);
  const int32_t *ip = static_cast<const int32_t *>(p);
  int32_t *io = static_cast<int32_t *>(p);
  uint8_t *u8 = static_cast<uint8_t *>(p);
  double *dp = static_cast<double *>(p);
  const int64_t H = std::numeric_limits<int64_t>::max();
  const int32_t H32 = std::numeric_limits<int32_t>::max();
  const size_t Z = std::numeric_limits<size_t>::max();
  CHECK(gc_chunk_grads(fp, fp, fp, H32, H32, H, H32, 0, fo, p, Z, nullptr) != GC_OK);
  CHECK(gc_chunk_grads(fp, fp, fp, 50, 512, H, 256, 0, fo, p, Z, nullptr) != GC_OK);
  CHECK(gc_chunk_grads(fp, fp, fp, H32, H32, 16384, 1, 1, fo, p, Z, nullptr) != GC_OK);
  CHECK(gc_sum_chunks(p, GC_BF16, H32, H, fo, nullptr) != GC_OK);
  CHECK(gc_decode_coeffs(ip, H, 1024, 1024, ip, 64, ip, ip, 64, fp, 8, io, u8, io, fo, nullptr) != GC_OK);
  CHECK(gc_decode_coeffs(ip, H, H32, 1024, ip, 64, ip, ip, 64, fp, 8, io, u8, io, fo, nullptr) != GC_OK);
  CHECK(gc_encode(p, GC_F32, H32, H, ip, ip, fp, H, 1024, 64, 8, fo, nullptr) != GC_OK);
  CHECK(gc_encode(p, GC_BF16, 200, H, ip, ip, fp, 8, 200, 20, 1, fo, nullptr) != GC_OK);
  CHECK(gc_encode(p, GC_F32, 100, 1 << 20, ip, ip, fp, H, 100, 10, 2, fo, nullptr) != GC_OK);
  CHECK(gc_reconstruct(fp, fp, ip, H, 1024, H, 1, fo, fp, dp, p, Z, nullptr) != GC_OK);
  CHECK(gc_reconstruct(fp, fp, ip, 8, 1024, H, 8, fo, nullptr, nullptr, nullptr, 0, nullptr) != GC_OK);
  CHECK(gc_reconstruct_noalloc(fp, fp, ip, H, 1024, H, 1, fo, fp, dp, nullptr) != GC_OK);
  CHECK(gc_decode_direct(p, GC_F32, H32, H, ip, H, 1024, 64, ip, ip, 64, fp, 8, fo, fp, dp, p, Z, nullptr) !=
        GC_OK);
  CHECK(gc_decode_direct(p, GC_F32, 1024, H, ip, 10, 1024, 64, ip, ip, 64, fp, 1, fo, nullptr, nullptr, p, Z,
                         nullptr) != GC_OK);
  CHECK(gc_progress(static_cast<const double *>(p), nullptr, H, 1024, 64, dp, H32, io, nullptr) != GC_OK);
  CHECK(gc_completion_times(static_cast<const double *>(p), nullptr, H, H32, 1024, 64, ip, ip, 64, 8, dp, dp,
                            nullptr) != GC_OK);
  CHECK(gc_original_ls(ip, H, 1024, 1024, ip, 64, ip, 64, H32, 1e-12, dp, io, nullptr) != GC_OK);
}

// valid arguments: with no GPU the device check fails (a non-OK status, nothing launched)
static void device_check_without_gpu() {
  void *p = reinterpret_cast<void *>(uintptr_t(256));
  const float *fp = static_cast<const float *>(p);
  float *fo = static_cast<float *>(p);
  const int32_t *ip = static_cast<const int32_t *>(p);
  int32_t *io = static_cast<int32_t *>(p);
  uint8_t *u8 = static_cast<uint8_t *>(p);
  double *dp = static_cast<double *>(p);
  CHECK(gc_decode_coeffs(ip, 4, 6, 6, ip, 3, ip, ip, 3, fp, 1, io, u8, io, fo, nullptr) != GC_OK);
  CHECK(gc_encode(p, GC_F32, 6, 64, ip, ip, fp, 4, 6, 3, 1, fo, nullptr) != GC_OK);
  CHECK(gc_reconstruct(fp, fp, ip, 4, 6, 64, 1, fo, nullptr, nullptr, nullptr, 0, nullptr) != GC_OK);
  CHECK(gc_reconstruct_noalloc(fp, fp, ip, 4, 6, 1 << 16, 1, fo, fp, dp, nullptr) != GC_OK);
  CHECK(gc_sum_chunks(p, GC_F32, 2, 8, fo, nullptr) != GC_OK);
}

int main(int argc, char **argv) {
  const bool with_device_check = !(argc > 1 && std::strcmp(argv[1], "--gpu-present") == 0);
  host_entry_points();
  workspace_sizes();
  device_validation();
  extreme_sizes();
  if (with_device_check) device_check_without_gpu();
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("ok\n");
  return 0;
}
