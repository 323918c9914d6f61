// Paged cache write of one decode step's new token (look-ahead decode).
//
// A decode step appends its token's keys and values to the request's cache before attention
// reads them (paper, Section 2).  Look-ahead decode (Section 4.3) runs k decode steps back to
// back on preallocated KV slots, so every step after the first starts by writing its token:
// for decode request i of the step's work list, the token at absolute position p (the step's
// cached_len) goes to slot p % 16 of physical page page_table[r][p / 16].  K pages are
// token-major ([page][kv head][slot][d]): the key row is one contiguous d-element run.  V pages
// are dim-major ([page][kv head][d][slot]): the value row is a column with a 16-element stride.
//
// One wave per (decode request, kv head); lane e copies dims e, e + 64, ...  The copies are
// exact, so the written cache is bit-identical to an index assignment on the host.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace duet {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void kv_append(AppendArgs a, WorkArgs w) {
  const int pair = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (pair >= w.n_dreq * a.h_kv) return;
  const int i = pair / a.h_kv;
  const int j = pair - i * a.h_kv;
  const int4 dr = w.dreq[i];    // (req, item_base, n_split, n_pages)
  const int4 m = w.meta[dr.x];  // (kind, row of the step's q / new K / new V, 1, position of the new token)
  const int pos = m.w;
  const int id = a.page_table[(size_t)dr.x * a.max_pages + (pos >> 4)];
  if (id < 0 || (long long)id >= a.num_phys_pages) {
    if (lane == 0) atomicOr(w.err, 1);
    return;
  }
  const int d = a.head_dim;
  const int slot = pos & 15;
  const T* kr = static_cast<const T*>(a.k_new) + ((size_t)m.y * a.h_kv + j) * d;
  const T* vr = static_cast<const T*>(a.v_new) + ((size_t)m.y * a.h_kv + j) * d;
  T* kd = static_cast<T*>(a.k_cache) + (((size_t)id * a.h_kv + j) * 16 + slot) * d;
  T* vd = static_cast<T*>(a.v_cache) + ((size_t)id * a.h_kv + j) * d * 16 + slot;
  for (int e = lane; e < d; e += 64) {
    kd[e] = kr[e];
    vd[(size_t)e * 16] = vr[e];
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendArgs& a, const WorkArgs& w, hipStream_t s) {
  if (w.n_dreq == 0) return hipSuccess;
  const dim3 grid((w.n_dreq * a.h_kv + 3) / 4);
  if (a.dtype == 0) hipLaunchKernelGGL(kv_append<__bf16>, grid, dim3(256), 0, s, a, w);
  else hipLaunchKernelGGL(kv_append<float>, grid, dim3(256), 0, s, a, w);
  return hipGetLastError();
}

}  // namespace duet
