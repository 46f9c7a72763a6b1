// Internal helpers shared by the gcx HIP sources (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <initializer_list>

#include "gcx.h"

namespace gcx {

constexpr int kWave = 64;

// The library is built for gfx950 only; refuse other devices up front rather
// than failing at the first launch with an opaque "invalid device function".
inline int check_device() {
  static int cached[64];  // 0 unknown, 1 ok, 2 not supported
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return GC_ELAUNCH;
  if (dev >= 0 && dev < 64 && cached[dev]) return cached[dev] == 1 ? GC_OK : GC_ENOTSUP;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return GC_ELAUNCH;
  const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev >= 0 && dev < 64) cached[dev] = ok ? 1 : 2;
  return ok ? GC_OK : GC_ENOTSUP;
}

// Compute units of the current device (cached per device); 256 on MI355X.
inline int cu_count() {
  static int cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < 64 && cached[dev]) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
    n = 256;
  if (dev >= 0 && dev < 64) cached[dev] = n;
  return n;
}

inline int launch_status() {
  return hipGetLastError() == hipSuccess ? GC_OK : GC_ELAUNCH;
}

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ceil(a / b) for a >= 0, b > 0, without forming a + b - 1 (no overflow near INT64_MAX)
__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return a / b + (a % b != 0 ? 1 : 0); }

// Host-side size limits: no array extent above 2^40 and no array above 2^48 elements
// (neither fits on any device), so that every size the entry points derive from their
// arguments is formed without int64 overflow.
constexpr int64_t kMaxExtent = int64_t(1) << 40;
constexpr int64_t kMaxElems = int64_t(1) << 48;

// every extent in [0, kMaxExtent] and their product at most kMaxElems
inline bool sizes_ok(std::initializer_list<int64_t> dims) {
  bool zero = false;
  for (int64_t v : dims) {
    if (v < 0 || v > kMaxExtent) return false;
    zero = zero || v == 0;
  }
  if (zero) return true;
  int64_t prod = 1;
  for (int64_t v : dims) {
    if (prod > kMaxElems / v) return false;
    prod *= v;
  }
  return true;
}

// A 1-D launch must keep gridDim.x < 2^31 and the total thread count < 2^32.
inline bool grid_ok(int64_t blocks, int threads) {
  return blocks >= 1 && blocks <= 0x7fffffffLL && blocks * threads <= 0xffffffffLL;
}

// bf16 bits -> fp32 (exact)
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

}  // namespace gcx
