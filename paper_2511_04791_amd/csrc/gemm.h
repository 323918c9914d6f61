// Plain bf16 GEMMs of the token-level operators (internal), on hipBLASLt.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>

namespace duet {

struct GemmCache;  // the hipBLASLt handle and one planned algorithm per problem shape

// Bytes of hipBLASLt workspace each concurrently running GEMM is given.
constexpr size_t kGemmWorkspaceBytes = (size_t)32 << 20;

// Returns nullptr when hipBLASLt cannot be initialised.
GemmCache* gemm_cache_create();
void gemm_cache_destroy(GemmCache* c);

// Row-major y[n, d_out] = x[n, d_in] @ w[d_in, d_out] (+ y when accumulate), bf16 operands and
// result, fp32 accumulation; rows of x and y are packed (strides d_in and d_out).  ws holds
// kGemmWorkspaceBytes bytes of device memory no other concurrent GEMM uses.  Returns 0, or -1
// with a message in *msg (a static string).
int gemm_bf16(GemmCache* c, const void* x, const void* w, void* y, int n, int d_in, int d_out, bool accumulate,
              void* ws, hipStream_t s, const char** msg);

}  // namespace duet
