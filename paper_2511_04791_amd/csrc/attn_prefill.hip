// Prefill-chunk attention over the paged KV cache (causal, with a cached prefix).
//
// A prefill request schedules q tokens after c cached ones; its keys and values, including
// those of the q new tokens, are already in the cache (paper, Section 2).  Query i sits at
// absolute position c + i and attends keys 0 .. c + i (Section 4.1: chunked prefill is q > 1,
// c > 0).  The work is a dense contraction, so it runs on MFMA: bf16 operands, fp32 accumulate.
//
// Work unit: one workgroup of 8 waves owns NH query heads of one GQA group (NH = group size, at
// most 8) and 256 / NH consecutive queries; each wave owns 32 (head, query) rows.  All waves of
// the unit read the same keys, so each K/V tile is fetched once for NH heads.  Keys stream
// through LDS 64 at a time (4 pages) in a 3-deep ring: K as [64 keys][d] and V as
// V^T [d][64 keys] (V pages are stored dim-major, so staging V^T is a straight copy).  Per
// 64-key step each wave computes, on the 32x32x16 bf16 MFMA,
//   S^T [64 keys x 32 queries] = K . Q^T       (Q^T held in registers for the whole loop)
//   O^T [d x 32 queries]      += V^T . P^T     (P^T never leaves registers)
// With S^T and O^T transposed, every per-query quantity (running max, denominator, rescale
// factor) lives in one lane pair (lane, lane ^ 32), so the online softmax needs one cross-lane
// exchange per step.  Rows of the K tile are fed to the MFMA in an order that makes each
// lane's score registers hold 8 consecutive keys, exactly the B layout P^T needs.
// The running max is only moved when a score exceeds it by more than 2^8 (in base-2 units);
// otherwise probabilities are taken against the stale max.  The result is the same softmax
// (numerator and denominator share the reference), and the O rescale is skipped on most steps.
// Key tiles past a wave's last query are skipped; only tiles crossing the diagonal are masked.
#include <hip/hip_runtime.h>

#include <cmath>

#include "kernels.h"

namespace duet {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kStages = 3;
constexpr float kRescaleSlack = 8.0f;  // base-2 units: probabilities stay below 2^8

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ bool page_ok(int id, long long num_phys) { return id >= 0 && (long long)id < num_phys; }

// A-operand row rho of a 32-row MFMA tile carries key swap_bits23(rho): within each group of 16,
// bits 2 and 3 are exchanged, so output register v of lane l holds key 16 (v / 8) + 8 (l / 32) + v % 8.
__device__ __forceinline__ int swap_bits23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// LDS chunk swizzles.  A wave's K-operand reads touch rows swap_bits23(0..31) in groups of 8 or
// 16 lanes; its V-operand reads touch rows 0..31 in order.  Both maps give every such lane group
// distinct 16-byte bank groups, for both 8-lane and 16-lane LDS service.
#ifndef DUET_PREFILL_PLAIN_SWIZZLE
__device__ __forceinline__ int kswz(int row) { return swap_bits23(row & 15); }
__device__ __forceinline__ int vswz(int row) { return (row & 7) ^ ((row >> 3) & 1); }
#else
__device__ __forceinline__ int kswz(int row) { return row & 15; }
__device__ __forceinline__ int vswz(int row) { return row & 7; }
#endif

__device__ __forceinline__ uint32_t keep_pairs(uint32_t word, int n_valid_in_pair) {
  return n_valid_in_pair >= 2 ? word : (n_valid_in_pair == 1 ? (word & 0xffffu) : 0u);
}

constexpr int kIdCap = kMaxPrefillKeys / 16;  // page ids staged in LDS for a whole unit

template <int D>
struct PrefillSmem {
  static constexpr int kStageElems = 2 * kPrefillKeys * D;  // K tile + V^T tile, bf16
  static constexpr size_t kTileBytes = (size_t)kStages * kStageElems * 2;
  static constexpr size_t kBytes = kTileBytes + kIdCap * sizeof(int);
};

template <int D, int NH>
__global__ __launch_bounds__(kThreads, 1) void prefill_bf16(AttnArgs a, WorkArgs w) {
  constexpr int BN = kPrefillKeys;       // keys per stage
  constexpr int KCH = D / 8;             // 16-byte chunks per K row
  constexpr int VCH = BN / 8;            // 16-byte chunks per V^T row
  constexpr int CH = (BN * D / 8) / kThreads;  // chunks per thread per tensor per stage
  constexpr int NK = D / 16;             // MFMA k-steps over the head dim
  constexpr int NO = D / 32;             // 32-dim output tiles
  constexpr int WPH = kWaves / NH;       // waves per head
  constexpr int QB = 32 * WPH;           // queries per unit
  extern __shared__ __attribute__((aligned(16))) __bf16 lds[];

  const int tid = threadIdx.x;
  const int wave = uniform(tid >> 6);
  const int lane = tid & 63;
  const int hh = lane >> 5;
  const int4 it = w.pitems[blockIdx.x];  // (req, first query head, q_row0, 0)
  const int r = it.x, h = it.y + wave / WPH, q_row0 = it.z;
  const int4 m = w.meta[r];
  const int q_start = m.y, q_len = m.z, c = m.w;
  const int L = c + q_len;
  const int n_pages = (L + 15) >> 4;
  const int j = it.y / a.group;

  const int wrow0 = q_row0 + 32 * (wave % WPH);
  const int qi = wrow0 + (lane & 31);
  const bool row_ok = qi < q_len;
  const int qpos = c + qi;

  bf16x8 qf[NK];
  {
    const __bf16* qp = reinterpret_cast<const __bf16*>(a.q) + ((size_t)(q_start + (row_ok ? qi : 0)) * a.h_q + h) * D +
                       8 * hh;
#pragma unroll
    for (int ks = 0; ks < NK; ++ks) {
      const uint4 u = row_ok ? *reinterpret_cast<const uint4*>(qp + 16 * ks) : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, u);
    }
  }

  const int n_tiles = (c + min(q_row0 + QB - 1, q_len - 1)) / BN + 1;
  const int w_tiles = wrow0 < q_len ? (c + min(wrow0 + 31, q_len - 1)) / BN + 1 : 0;
  const int w_first_pos = c + wrow0;

  const char* kbase = reinterpret_cast<const char*>(a.k_cache);
  const char* vbase = reinterpret_cast<const char*>(a.v_cache);
  const int* prow = a.page_table + (size_t)r * a.max_pages;
  constexpr size_t kSlab = 16 * D * 2;  // bytes of one (page, kv head) slab, K or V
  int bad = 0;

  // The unit's page ids go to LDS once, so a tile load never waits on a page-table read.
  int* ids = reinterpret_cast<int*>(reinterpret_cast<char*>(lds) + PrefillSmem<D>::kTileBytes);
  const int n_used_pages = min(n_pages, (n_tiles * BN + 15) >> 4);
  for (int i = tid; i < n_used_pages; i += kThreads) ids[i] = prow[i];
  __syncthreads();

  uint4 kst[CH], vst[CH];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int x = 0; x < CH; ++x) {
      const int chunk = tid + kThreads * x;
      const int pi = chunk / (2 * D);
      const int y = chunk - pi * (2 * D);
      const int lp = 4 * kt + pi;
      const bool in_range = lp < n_pages;
      const int id = in_range ? ids[lp] : 0;
      const bool ok = in_range && page_ok(id, a.num_phys_pages);
      bad |= in_range & !ok;
      // Loads are unconditional (page 0 stands in for a missing page); keys of a missing page
      // lie past the end and are masked, so only their values need zeroing.
      const size_t off = ((size_t)(ok ? id : 0) * a.h_kv + j) * kSlab + (size_t)y * 16;
      kst[x] = *reinterpret_cast<const uint4*>(kbase + off);
      uint4 v = *reinterpret_cast<const uint4*>(vbase + off);
      // Values of keys >= L are NaN-poisoned slots: they must not reach the MFMA.
      const int nv = ok ? L - (BN * kt + 16 * pi + 8 * (y & 1)) : 0;
      if (nv < 8) {
        v.x = keep_pairs(v.x, nv);
        v.y = keep_pairs(v.y, nv - 2);
        v.z = keep_pairs(v.z, nv - 4);
        v.w = keep_pairs(v.w, nv - 6);
      }
      vst[x] = v;
    }
  };
  auto store_tile = [&](int buf) {
    __bf16* ks = lds + buf * PrefillSmem<D>::kStageElems;
    __bf16* vs = ks + BN * D;
#pragma unroll
    for (int x = 0; x < CH; ++x) {
      const int chunk = tid + kThreads * x;
      const int pi = chunk / (2 * D);
      const int y = chunk - pi * (2 * D);
      const int krow = 16 * pi + y / KCH;
      const int kch = (y % KCH) ^ (kswz(krow) & (KCH - 1));
      *reinterpret_cast<uint4*>(ks + krow * D + kch * 8) = kst[x];
      const int vrow = y >> 1;
      const int vch = (2 * pi + (y & 1)) ^ (vswz(vrow) & (VCH - 1));
      *reinterpret_cast<uint4*>(vs + vrow * BN + vch * 8) = vst[x];
    }
  };

  f32x16 oacc[NO];
#pragma unroll
  for (int n = 0; n < NO; ++n)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[n][v] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;

  load_tile(0);
  store_tile(0);
  if (n_tiles > 1) {
    load_tile(1);
    store_tile(1);
  }
  __syncthreads();
  if (n_tiles > 2) load_tile(2);

  for (int kt = 0; kt < n_tiles; ++kt) {
    if (kt < w_tiles) {
      const __bf16* ks = lds + (kt % kStages) * PrefillSmem<D>::kStageElems;
      const __bf16* vs = ks + BN * D;
      // All K fragments of the step are read before the first MFMA, so LDS latency is paid once.
      bf16x8 kf[2][NK];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int row = 32 * nb + swap_bits23(lane & 31);
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
          const int ch = (2 * kk + hh) ^ (kswz(row) & (KCH - 1));
          kf[nb][kk] = *reinterpret_cast<const bf16x8*>(ks + row * D + ch * 8);
        }
      }
      f32x16 sacc[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[nb][v] = 0.f;
#ifdef DUET_PREFILL_SETPRIO
      __builtin_amdgcn_s_setprio(1);
#endif
#pragma unroll
      for (int kk = 0; kk < NK; ++kk)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          sacc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[nb][kk], qf[kk], sacc[nb], 0, 0, 0);
#ifdef DUET_PREFILL_SETPRIO
      __builtin_amdgcn_s_setprio(0);
#endif
      // V fragments are read now; their LDS latency hides behind the softmax below.  With
      // DUET_PREFILL_VHALF only the first half is read ahead (fewer live registers).
#ifdef DUET_PREFILL_VHALF
      constexpr int NV = NO / 2;
#else
      constexpr int NV = NO;
#endif
      bf16x8 vf[NO][4];
#pragma unroll
      for (int n = 0; n < NV; ++n) {
        const int vrow = 32 * n + (lane & 31);
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) {
          const int ch = (2 * k2 + hh) ^ (vswz(vrow) & (VCH - 1));
          vf[n][k2] = *reinterpret_cast<const bf16x8*>(vs + vrow * BN + ch * 8);
        }
      }
      // Only tiles that cross this wave's diagonal need the causal mask.
      if (BN * kt + BN - 1 > w_first_pos) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = BN * kt + 32 * nb + 16 * (v >> 3) + 8 * hh + (v & 7);
            if (key > qpos) sacc[nb][v] = -INFINITY;
          }
      }
      // Max over raw scores; the scale (log2(e) / sqrt(d) > 0) is applied once to the max and
      // folded into each exponent as an FMA.
      float mx = -INFINITY;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[nb][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * a.scale_log2;
      // Move the reference max only when some score exceeds it by more than the slack.
      if (__any(mx > m_ref + kRescaleSlack)) {
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = fast_exp2(m_ref - m_new);
        m_ref = m_new;
        l_run *= alpha;
#pragma unroll
        for (int n = 0; n < NO; ++n) oacc[n] *= alpha;
      }
      bf16x8 pb[4];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          pb[2 * nb + (v >> 3)][v & 7] = static_cast<__bf16>(fast_exp2(__builtin_fmaf(sacc[nb][v], a.scale_log2, -m_ref)));
      // The denominator sums the bf16 probabilities the PV product consumes.
      const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
      for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 two = {pb[k2][2 * e], pb[k2][2 * e + 1]};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(two, ones, l_run, false);
        }
#pragma unroll
      for (int n = NV; n < NO; ++n) {
        const int vrow = 32 * n + (lane & 31);
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) {
          const int ch = (2 * k2 + hh) ^ (vswz(vrow) & (VCH - 1));
          vf[n][k2] = *reinterpret_cast<const bf16x8*>(vs + vrow * BN + ch * 8);
        }
      }
#ifdef DUET_PREFILL_SETPRIO
      __builtin_amdgcn_s_setprio(1);
#endif
#pragma unroll
      for (int n = 0; n < NO; ++n)
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2)
          oacc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[n][k2], pb[k2], oacc[n], 0, 0, 0);
#ifdef DUET_PREFILL_SETPRIO
      __builtin_amdgcn_s_setprio(0);
#endif
    }
    if (kt + 2 < n_tiles) store_tile((kt + 2) % kStages);
    if (kt + 3 < n_tiles) load_tile(kt + 3);
    __syncthreads();
  }

  if (bad) atomicOr(w.err, 1);
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (row_ok) {
    const float inv = 1.0f / l_tot;
    __bf16* op = reinterpret_cast<__bf16*>(a.out) + ((size_t)(q_start + qi) * a.h_q + h) * D + 4 * hh;
#pragma unroll
    for (int n = 0; n < NO; ++n)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        __bf16 o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = static_cast<__bf16>(oacc[n][4 * g4 + e] * inv);
        *reinterpret_cast<uint2*>(op + 32 * n + 8 * g4) = __builtin_bit_cast(uint2, o4);
      }
  }
}

// fp32 path (small shapes): each wave walks its 32 rows one by one, lane = dim.
template <int D>
__global__ __launch_bounds__(256) void prefill_f32(AttnArgs a, WorkArgs w) {
  constexpr int E = D / 64;
  const int wave = uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int4 it = w.pitems[blockIdx.x];  // (req, query head, q_row0, 0)
  const int r = it.x, h = it.y, q_row0 = it.z;
  const int4 m = w.meta[r];
  const int q_start = m.y, q_len = m.z, c = m.w;
  const int j = h / a.group;
  const float* K = reinterpret_cast<const float*>(a.k_cache);
  const float* V = reinterpret_cast<const float*>(a.v_cache);
  const int* prow = a.page_table + (size_t)r * a.max_pages;
  int bad = 0;
  for (int i = 0; i < 32; ++i) {
    const int qi = q_row0 + 32 * wave + i;
    if (qi >= q_len) break;
    const float* qrow = reinterpret_cast<const float*>(a.q) + ((size_t)(q_start + qi) * a.h_q + h) * D;
    float qv[E], acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      qv[e] = qrow[lane + 64 * e];
      acc[e] = 0.f;
    }
    float m_run = -INFINITY, l_run = 0.f;
    const int pos = c + qi;
    for (int t = 0; t <= pos; ++t) {
      const int id = uniform(prow[t >> 4]);
      if (!page_ok(id, a.num_phys_pages)) {
        bad = 1;
        continue;
      }
      const size_t slab = ((size_t)id * a.h_kv + j) * 16 * D;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dot += qv[e] * K[slab + (size_t)(t & 15) * D + lane + 64 * e];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) dot += __shfl_xor(dot, off);
      const float x = dot * a.scale_log2;
      const float m_new = fmaxf(m_run, x);
      const float alpha = fast_exp2(m_run - m_new);
      const float pr = fast_exp2(x - m_new);
      l_run = l_run * alpha + pr;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = acc[e] * alpha + pr * V[slab + (size_t)(lane + 64 * e) * 16 + (t & 15)];
      m_run = m_new;
    }
    float* orow = reinterpret_cast<float*>(a.out) + ((size_t)(q_start + qi) * a.h_q + h) * D;
#pragma unroll
    for (int e = 0; e < E; ++e) orow[lane + 64 * e] = acc[e] / l_run;
  }
  if (bad && lane == 0) atomicOr(w.err, 1);
}

template <int D, int NH>
hipError_t launch_bf16(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  static bool attr_set = false;  // the attribute is per function and process
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&prefill_bf16<D, NH>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)PrefillSmem<D>::kBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((prefill_bf16<D, NH>), dim3(w.n_pitems), dim3(kThreads), PrefillSmem<D>::kBytes, s, a, w);
  return hipGetLastError();
}

template <int D>
hipError_t launch_bf16_nh(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  switch (prefill_heads_per_unit(a.group)) {
    case 1: return launch_bf16<D, 1>(a, w, s);
    case 2: return launch_bf16<D, 2>(a, w, s);
    case 4: return launch_bf16<D, 4>(a, w, s);
    default: return launch_bf16<D, 8>(a, w, s);
  }
}

}  // namespace

int prefill_heads_per_unit(int group) {
  // largest power of two <= min(group, 8) that divides the group
  int nh = 1;
  while (nh * 2 <= 8 && group % (nh * 2) == 0) nh *= 2;
  return nh;
}

int prefill_rows_per_unit(int group, int dtype) {
  return dtype == 0 ? 256 / prefill_heads_per_unit(group) : kPrefillRows;
}

hipError_t launch_prefill(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  if (w.n_pitems == 0) return hipSuccess;
  if (a.dtype == 0) return a.head_dim == 128 ? launch_bf16_nh<128>(a, w, s) : launch_bf16_nh<64>(a, w, s);
  const dim3 grid(w.n_pitems);
  if (a.head_dim == 128) hipLaunchKernelGGL(prefill_f32<128>, grid, dim3(256), 0, s, a, w);
  else hipLaunchKernelGGL(prefill_f32<64>, grid, dim3(256), 0, s, a, w);
  return hipGetLastError();
}

}  // namespace duet
