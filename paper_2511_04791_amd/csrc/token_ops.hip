// Token-level operators of a transformer block (paper, Section 4.1, "Token-Level Operators"):
// RMSNorm, the SwiGLU activation, and the step between the QKV projection and attention that
// takes the query rows out of the projection and writes the new tokens' keys and values into the
// paged cache (Section 2: a token's key and value are appended before attention reads them).
// The projections themselves are plain GEMMs (hipBLASLt, issued by the runtime).
//
// All three are HBM-bound elementwise passes over [rows, width] bf16 activations: 16-byte
// accesses, one workgroup per token row, fp32 arithmetic, round-to-nearest-even on store.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace duet {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  return t;
}

// y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * w, for rows r of [rows, d] (d a multiple of 8).
__global__ __launch_bounds__(256) void rmsnorm_bf16(const __bf16* x, const __bf16* w, __bf16* y, int d, float eps) {
  __shared__ float red[4];
  const size_t row = blockIdx.x;
  const bf16x8* xr = reinterpret_cast<const bf16x8*>(x + row * d);
  float ss = 0.f;
  for (int c = threadIdx.x; c < d / 8; c += blockDim.x) {
    const bf16x8 v = xr[c];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float f = static_cast<float>(v[e]);
      ss += f * f;
    }
  }
  const float inv = 1.0f / sqrtf(block_sum(ss, red) / (float)d + eps);
  const bf16x8* wr = reinterpret_cast<const bf16x8*>(w);
  bf16x8* yr = reinterpret_cast<bf16x8*>(y + row * d);
  for (int c = threadIdx.x; c < d / 8; c += blockDim.x) {
    const bf16x8 v = xr[c], g = wr[c];
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = static_cast<__bf16>(static_cast<float>(v[e]) * inv * static_cast<float>(g[e]));
    yr[c] = o;
  }
}

// a[r, i] = silu(gu[r, i]) * gu[r, m + i]: gate columns first, then up (m a multiple of 8).
__global__ __launch_bounds__(256) void swiglu_bf16(const __bf16* gu, __bf16* a, int m) {
  const size_t row = blockIdx.x;
  const bf16x8* g = reinterpret_cast<const bf16x8*>(gu + row * 2 * m);
  const bf16x8* u = reinterpret_cast<const bf16x8*>(gu + row * 2 * m + m);
  bf16x8* o = reinterpret_cast<bf16x8*>(a + row * m);
  for (int c = threadIdx.x; c < m / 8; c += blockDim.x) {
    const bf16x8 gv = g[c], uv = u[c];
    bf16x8 r;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float gf = static_cast<float>(gv[e]);
      r[e] = static_cast<__bf16>(gf / (1.0f + expf(-gf)) * static_cast<float>(uv[e]));
    }
    o[c] = r;
  }
}

// Row r0 + blockIdx.x of the QKV projection [rows, (h_q + 2 h_kv) d]: its h_q d query columns go
// to q (row stride h_q d); its key and value columns go to slot pos % 16 of the physical page
// holding absolute position pos = cached_len + (row - q_start) of its request (found by binary
// search over the request table, whose q_start rise with the request index), or, in a look-ahead
// step, of decode request `row` of the step (its token at the step's cached_len).  A page id outside
// [0, num_phys_pages) is not written through: it sets bit 0 of the error word.
__global__ __launch_bounds__(256) void qkv_split_bf16(QkvSplitArgs s) {
  const int row = s.row0 + blockIdx.x;
  const int nq = s.h_q * s.head_dim, nk = s.h_kv * s.head_dim;
  const __bf16* src = s.qkv + (size_t)row * (nq + 2 * nk);
  {
    const bf16x8* qs = reinterpret_cast<const bf16x8*>(src);
    bf16x8* qd = reinterpret_cast<bf16x8*>(s.q + (size_t)row * nq);
    for (int c = threadIdx.x; c < nq / 8; c += blockDim.x) qd[c] = qs[c];
  }
  int lo = 0, hi = s.num_reqs - 1;  // last request with q_start <= row
  if (s.dreq) {
    lo = s.dreq[row].x;
  } else {
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s.meta[mid].y <= row) lo = mid;
      else hi = mid - 1;
    }
  }
  const int4 m = s.meta[lo];
  const int pos = s.dreq ? m.w : m.w + (row - m.y);
  const int id = s.page_table[(size_t)lo * s.max_pages + (pos >> 4)];
  if (id < 0 || (long long)id >= s.num_phys_pages) {
    if (threadIdx.x == 0) atomicOr(s.err, 1);
    return;
  }
  const int slot = pos & 15, d = s.head_dim;
  for (int i = threadIdx.x; i < nk; i += blockDim.x) {
    const int j = i / d, e = i - j * d;
    const size_t slab = (size_t)id * s.h_kv + j;
    s.k_cache[(slab * 16 + slot) * d + e] = src[nq + i];
    s.v_cache[(slab * d + e) * 16 + slot] = src[nq + nk + i];
  }
}

}  // namespace

hipError_t launch_rmsnorm(const __bf16* x, const __bf16* w, __bf16* y, int rows, int d, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_bf16, dim3(rows), dim3(256), 0, s, x, w, y, d, eps);
  return hipGetLastError();
}

hipError_t launch_swiglu(const __bf16* gu, __bf16* a, int rows, int m, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_bf16, dim3(rows), dim3(256), 0, s, gu, a, m);
  return hipGetLastError();
}

hipError_t launch_qkv_split(const QkvSplitArgs& a, int rows, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(qkv_split_bf16, dim3(rows), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace duet
