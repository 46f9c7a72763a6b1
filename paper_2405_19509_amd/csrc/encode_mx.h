// The bf16 matrix-core encode (encode_mx.hip), called by gc_encode.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gcx {

// returned (nothing enqueued) when the group's staged rows or LDS would not fit
constexpr int kEncodeMxNotApplicable = 1;

// G [N][d], fp32 (f32) or bf16 bits; other arguments as gc_encode.  GC_OK, a GC_ status,
// or kEncodeMxNotApplicable.
int encode_mx(const void *G, bool f32, int32_t N, int64_t d, const int32_t *psi, const int32_t *order, const float *Bc,
              int64_t P, int32_t m, int32_t delta, int32_t ell, float *T, hipStream_t stream);

}  // namespace gcx
