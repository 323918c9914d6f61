// Decode attention over the paged KV cache: split-K partial kernel and reduce kernel.
//
// Each decode request has one query token at absolute position kv_len - 1 that attends all
// kv_len keys (paper, Section 2: the new token's key and value are appended before attention;
// Section 4.1: decode is q = 1, c > 0).  The work is HBM-bound: every key and value is read
// once.  A work item is (request, kv head, split) where a split is a fixed run of logical pages
// (pages_per_split).  One wave owns one item and reads each page of its kv head once for all
// query heads of the GQA group, so the bytes moved are the algorithmic K/V bytes.
//
// bf16 path, per pair of pages (32 tokens), on the 16x16x32 bf16 MFMA (fp32 accumulate):
//   S^T [16 tokens x 16 heads] = K_page [16 x d] . Q^T [d x 16]     (one MFMA per 32 dims)
//   O^T [16 dims x 16 heads]  += V^T   [16 x 32] . P^T [32 x 16]    (one MFMA per 16 dims)
// Heads beyond the group size are zero columns.  K is read token-major (16 B per lane, the
// MFMA A layout); V pages are stored dim-major, so a lane's 4 consecutive tokens of one dim
// are 8 contiguous bytes and P^T never leaves registers.  Online softmax keeps a running max
// and denominator per head; partials (unnormalised output, max, denominator) go to the
// workspace and the reduce kernel merges the splits.  All arithmetic order depends on logical
// token positions only.
#include <hip/hip_runtime.h>

#include <cmath>

#include "kernels.h"

namespace duet {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ uint64_t low_elems_mask(int n) {  // keep the first n of 4 bf16
  return n >= 4 ? ~0ull : (n <= 0 ? 0ull : ((1ull << (16 * n)) - 1ull));
}

template <int D>
struct PagePair {
  uint4 k0[D / 32], k1[D / 32];  // K rows (token = lane % 16), 8 dims per lane per 32-dim step
  uint2 v0[D / 16], v1[D / 16];  // V^T rows (dim = 16 n + lane % 16), tokens 4 (lane / 16) .. +4
};

template <int D>
__device__ __forceinline__ void load_pair(PagePair<D>& pp, const char* kbase, const char* vbase, int id0, int id1,
                                          bool ok0, bool ok1, int lane) {
  const int row = lane & 15, quad = lane >> 4;
  constexpr size_t kPageBytes = 16 * D * 2;  // one (page, kv head) slab
  if (ok0) {
    const char* kp = kbase + (size_t)id0 * kPageBytes + row * D * 2 + quad * 16;
    const char* vp = vbase + (size_t)id0 * kPageBytes + row * 32 + quad * 8;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) pp.k0[ks] = *reinterpret_cast<const uint4*>(kp + ks * 64);
#pragma unroll
    for (int n = 0; n < D / 16; ++n) pp.v0[n] = *reinterpret_cast<const uint2*>(vp + n * 16 * 32);
  } else {
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) pp.k0[ks] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int n = 0; n < D / 16; ++n) pp.v0[n] = make_uint2(0, 0);
  }
  if (ok1) {
    const char* kp = kbase + (size_t)id1 * kPageBytes + row * D * 2 + quad * 16;
    const char* vp = vbase + (size_t)id1 * kPageBytes + row * 32 + quad * 8;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) pp.k1[ks] = *reinterpret_cast<const uint4*>(kp + ks * 64);
#pragma unroll
    for (int n = 0; n < D / 16; ++n) pp.v1[n] = *reinterpret_cast<const uint2*>(vp + n * 16 * 32);
  } else {
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) pp.k1[ks] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int n = 0; n < D / 16; ++n) pp.v1[n] = make_uint2(0, 0);
  }
}

__device__ __forceinline__ bool page_ok(int id, long long num_phys) { return id >= 0 && (long long)id < num_phys; }

template <int D>
__global__ __launch_bounds__(256) void decode_partial_bf16(AttnArgs a, WorkArgs w) {
  const int wave = uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int4 dr = w.dreq[blockIdx.y];  // (req, item_base, n_split, n_pages)
  const int witem = blockIdx.x * 4 + wave;
  const int j = witem / dr.z;
  const int s = witem - j * dr.z;
  if (j >= a.h_kv) return;  // no barriers in this kernel: idle waves leave early
  const int4 m = w.meta[dr.x];  // (kind, q_start, q_len, cached_len)
  const int L = m.w + m.z;
  const int g = a.group;
  const int col = lane & 15, quad = lane >> 4;
  const int pb = s * w.pages_per_split;
  const int pe = min(pb + w.pages_per_split, dr.w);

  // Q^T as the B operand: column = head of the group, k = dims 32 ks + 8 quad .. +8.
  bf16x8 qf[D / 32];
  {
    const __bf16* qrow = reinterpret_cast<const __bf16*>(a.q) + ((size_t)m.y * a.h_q + j * g + col) * D + quad * 8;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      uint4 u = col < g ? *reinterpret_cast<const uint4*>(qrow + ks * 32) : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, u);
    }
  }

  const char* kbase = reinterpret_cast<const char*>(a.k_cache) + (size_t)j * 16 * D * 2;
  const char* vbase = reinterpret_cast<const char*>(a.v_cache) + (size_t)j * 16 * D * 2;
  // Both caches are [P, h_kv, 16 * d] in bytes per (page, head) slab; fold h_kv into the page stride.
  const long long slab_stride_pages = a.h_kv;
  const int* prow = a.page_table + (size_t)dr.x * a.max_pages;

  f32x4 acc[D / 16];
#pragma unroll
  for (int n = 0; n < D / 16; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  int bad = 0;

  auto page_ids = [&](int p, int& id0, int& id1, bool& ok0, bool& ok1) {
    id0 = uniform(prow[p]);
    ok0 = page_ok(id0, a.num_phys_pages);
    const bool has1 = p + 1 < pe;
    id1 = has1 ? uniform(prow[p + 1]) : 0;
    ok1 = has1 && page_ok(id1, a.num_phys_pages);
    bad |= (!ok0) | (has1 && !ok1);
  };

  PagePair<D> cur, nxt;
  int id0, id1;
  bool ok0, ok1;
  page_ids(pb, id0, id1, ok0, ok1);
  load_pair<D>(cur, kbase, vbase, (int)(id0 * slab_stride_pages), (int)(id1 * slab_stride_pages), ok0, ok1, lane);

  for (int p = pb; p < pe; p += 2) {
    const bool c_ok0 = ok0, c_ok1 = ok1;
    if (p + 2 < pe) {
      page_ids(p + 2, id0, id1, ok0, ok1);
      load_pair<D>(nxt, kbase, vbase, (int)(id0 * slab_stride_pages), (int)(id1 * slab_stride_pages), ok0, ok1,
                   lane);
    }
    // Scores S^T: lane holds head `col`, tokens 4 quad + i of each page.
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, cur.k0[ks]), qf[ks], s0, 0, 0, 0);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, cur.k1[ks]), qf[ks], s1, 0, 0, 0);

    const int t0 = 16 * p + 4 * quad;
    float x[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[i] = (c_ok0 && t0 + i < L) ? s0[i] * a.scale_log2 : -INFINITY;
      x[4 + i] = (c_ok1 && t0 + 16 + i < L) ? s1[i] * a.scale_log2 : -INFINITY;
    }
    float mx = x[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = fmaxf(mx, x[i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float pr[8], psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      pr[i] = fast_exp2(x[i] - m_new);
      psum += pr[i];
    }
    l_run = l_run * alpha + psum;
    bf16x8 pb8;
#pragma unroll
    for (int i = 0; i < 8; ++i) pb8[i] = static_cast<__bf16>(pr[i]);

    // Values of tokens past the end (NaN-poisoned slots) must not reach the MFMA.
    if (16 * (p + 2) > L) {
      const uint64_t mk0 = low_elems_mask(L - t0), mk1 = low_elems_mask(L - t0 - 16);
#pragma unroll
      for (int n = 0; n < D / 16; ++n) {
        uint64_t v0 = ((uint64_t)cur.v0[n].y << 32 | cur.v0[n].x) & mk0;
        uint64_t v1 = ((uint64_t)cur.v1[n].y << 32 | cur.v1[n].x) & mk1;
        cur.v0[n] = make_uint2((uint32_t)v0, (uint32_t)(v0 >> 32));
        cur.v1[n] = make_uint2((uint32_t)v1, (uint32_t)(v1 >> 32));
      }
    }
#pragma unroll
    for (int n = 0; n < D / 16; ++n) {
      acc[n] *= alpha;
      const uint4 vv = make_uint4(cur.v0[n].x, cur.v0[n].y, cur.v1[n].x, cur.v1[n].y);
      acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vv), pb8, acc[n], 0, 0, 0);
    }
    if (p + 2 < pe) cur = nxt;
  }

  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  if (bad && lane == 0) atomicOr(w.err, 1);
  const int item = dr.y + j * dr.z + s;
  if (col < g) {
    float* pa = w.pacc + ((size_t)item * g + col) * D + 4 * quad;
#pragma unroll
    for (int n = 0; n < D / 16; ++n) *reinterpret_cast<f32x4*>(pa + 16 * n) = acc[n];
    if (quad == 0) {
      w.pml[((size_t)item * g + col) * 2 + 0] = m_run;
      w.pml[((size_t)item * g + col) * 2 + 1] = l_tot;
    }
  }
}

// fp32 path (small shapes): one wave per item, lane = dim, scores reduced across the wave.
template <int D>
__global__ __launch_bounds__(256) void decode_partial_f32(AttnArgs a, WorkArgs w) {
  constexpr int E = D / 64;
  const int wave = uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int4 dr = w.dreq[blockIdx.y];
  const int witem = blockIdx.x * 4 + wave;
  const int j = witem / dr.z;
  const int s = witem - j * dr.z;
  if (j >= a.h_kv) return;
  const int4 m = w.meta[dr.x];
  const int L = m.w + m.z;
  const int g = a.group;
  const int pb = s * w.pages_per_split;
  const int pe = min(pb + w.pages_per_split, dr.w);
  const float* K = reinterpret_cast<const float*>(a.k_cache);
  const float* V = reinterpret_cast<const float*>(a.v_cache);
  const int* prow = a.page_table + (size_t)dr.x * a.max_pages;
  const int item = dr.y + j * dr.z + s;
  int bad = 0;
  for (int col = 0; col < g; ++col) {
    const float* qrow = reinterpret_cast<const float*>(a.q) + ((size_t)m.y * a.h_q + j * g + col) * D;
    float qv[E], acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      qv[e] = qrow[lane + 64 * e];
      acc[e] = 0.f;
    }
    float m_run = -INFINITY, l_run = 0.f;
    for (int p = pb; p < pe; ++p) {
      const int id = uniform(prow[p]);
      if (!page_ok(id, a.num_phys_pages)) {
        bad = 1;
        continue;
      }
      const size_t slab = ((size_t)id * a.h_kv + j) * 16 * D;
      for (int t = 0; t < 16 && 16 * p + t < L; ++t) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) dot += qv[e] * K[slab + (size_t)t * D + lane + 64 * e];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) dot += __shfl_xor(dot, off);
        const float x = dot * a.scale_log2;
        const float m_new = fmaxf(m_run, x);
        const float alpha = fast_exp2(m_run - m_new);
        const float pr = fast_exp2(x - m_new);
        l_run = l_run * alpha + pr;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = acc[e] * alpha + pr * V[slab + (size_t)(lane + 64 * e) * 16 + t];
        m_run = m_new;
      }
    }
    float* pa = w.pacc + ((size_t)item * g + col) * D;
#pragma unroll
    for (int e = 0; e < E; ++e) pa[lane + 64 * e] = acc[e];
    if (lane == 0) {
      w.pml[((size_t)item * g + col) * 2 + 0] = m_run;
      w.pml[((size_t)item * g + col) * 2 + 1] = l_run;
    }
  }
  if (bad && lane == 0) atomicOr(w.err, 1);
}

// Merge the splits of one (decode request, query head): one wave, lane = dim.
template <int D, typename OutT>
__global__ __launch_bounds__(256) void decode_reduce(AttnArgs a, WorkArgs w) {
  constexpr int E = D / 64;
  const int lane = threadIdx.x & 63;
  const int pair = blockIdx.x * 4 + uniform(threadIdx.x >> 6);
  const int i = pair / a.h_q;
  const int h = pair - i * a.h_q;
  if (i >= w.n_dreq) return;
  const int4 dr = w.dreq[i];
  const int4 m = w.meta[dr.x];
  const int g = a.group;
  const int j = h / g, col = h - j * g;
  const int base = dr.y + j * dr.z;
  float M = -INFINITY;
  for (int s = 0; s < dr.z; ++s) M = fmaxf(M, w.pml[((size_t)(base + s) * g + col) * 2]);
  float den = 0.f, num[E];
#pragma unroll
  for (int e = 0; e < E; ++e) num[e] = 0.f;
  for (int s = 0; s < dr.z; ++s) {
    const size_t it = (size_t)(base + s) * g + col;
    const float wgt = fast_exp2(w.pml[it * 2] - M);
    den += wgt * w.pml[it * 2 + 1];
#pragma unroll
    for (int e = 0; e < E; ++e) num[e] += wgt * w.pacc[it * D + lane + 64 * e];
  }
  const float inv = 1.0f / den;
  OutT* o = reinterpret_cast<OutT*>(a.out) + ((size_t)m.y * a.h_q + h) * D;
#pragma unroll
  for (int e = 0; e < E; ++e) o[lane + 64 * e] = static_cast<OutT>(num[e] * inv);
}

}  // namespace

hipError_t launch_decode_partial(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  if (w.n_dreq == 0) return hipSuccess;
  const dim3 grid((a.h_kv * w.max_split + 3) / 4, w.n_dreq);
  if (a.dtype == 0) {
    if (a.head_dim == 128) hipLaunchKernelGGL(decode_partial_bf16<128>, grid, dim3(256), 0, s, a, w);
    else hipLaunchKernelGGL(decode_partial_bf16<64>, grid, dim3(256), 0, s, a, w);
  } else {
    if (a.head_dim == 128) hipLaunchKernelGGL(decode_partial_f32<128>, grid, dim3(256), 0, s, a, w);
    else hipLaunchKernelGGL(decode_partial_f32<64>, grid, dim3(256), 0, s, a, w);
  }
  return hipGetLastError();
}

hipError_t launch_decode_reduce(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  if (w.n_dreq == 0) return hipSuccess;
  const dim3 grid((w.n_dreq * a.h_q + 3) / 4);
  if (a.dtype == 0) {
    if (a.head_dim == 128) hipLaunchKernelGGL((decode_reduce<128, __bf16>), grid, dim3(256), 0, s, a, w);
    else hipLaunchKernelGGL((decode_reduce<64, __bf16>), grid, dim3(256), 0, s, a, w);
  } else {
    if (a.head_dim == 128) hipLaunchKernelGGL((decode_reduce<128, float>), grid, dim3(256), 0, s, a, w);
    else hipLaunchKernelGGL((decode_reduce<64, float>), grid, dim3(256), 0, s, a, w);
  }
  return hipGetLastError();
}

}  // namespace duet
