// Decode attention over the paged KV cache: split-K partial kernel and reduce kernel.
//
// Each decode request has one query token at absolute position kv_len - 1 that attends all
// kv_len keys (paper, Section 2: the new token's key and value are appended before attention;
// Section 4.1: decode is q = 1, c > 0).  The work is HBM-bound: every key and value is read
// once.  A work item is (request, kv head, split) where a split is a fixed run of logical pages
// (pages_per_split).  One wave owns one item and reads each page of its kv head once for all
// query heads of the GQA group, so the bytes moved are the algorithmic K/V bytes.
//
// bf16 path, per page (16 tokens), on MFMA with fp32 accumulate:
//   S^T [16 tokens x 16 heads] = K_page [16 x d] . Q^T [d x 16]   (16x16x32, one per 32 dims)
//   O^T [16 dims x 16 heads]  += V^T   [16 x 16] . P^T [16 x 16]  (16x16x16, one per 16 dims)
// Heads beyond the group size are zero columns.  K is read token-major (16 B per lane, the
// MFMA A layout); V pages are stored dim-major, so a lane's 4 consecutive tokens of one dim
// are 8 contiguous bytes and P^T never leaves registers.  Pages cycle through four register
// buffers, so three pages are in flight while one is computed, across item boundaries too.
// Online softmax keeps a reference max per head that only moves when a score exceeds it by
// more than 2^8 (base-2 units), so the output rescale is rare.  Partials (unnormalised output,
// reference max, denominator) go to the workspace, and one wave per (request, query head) merges
// the splits: the reduce kernel, or, for the layers of a call but the last, the next layer's bf16
// partial kernel, in the waves whose item queue has run dry.
// All arithmetic order depends on logical token positions only.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>
#include <cmath>

#include "kernels.h"

namespace duet {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr float kRescaleSlack = 8.0f;  // base-2 units: probabilities stay below 2^8
constexpr int kRing = 4;  // page buffers per wave: kRing - 1 pages in flight
typedef float f32x4 __attribute__((ext_vector_type(4)));


__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Combine a value across the four 16-lane rows of a wave (lanes l, l ^ 16, l ^ 32, l ^ 48) with
// the row-swap permutes, which stay in the vector ALU: an LDS permute would be counted with the
// scalar loads, so waiting for it would also wait for them.
__device__ __forceinline__ float max_rows(float x) {
  const unsigned u = __float_as_uint(x);
  auto s32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const float m = fmaxf(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
  const unsigned v = __float_as_uint(m);
  auto s16 = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return fmaxf(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
}
__device__ __forceinline__ float sum_rows(float x) {
  const unsigned u = __float_as_uint(x);
  auto s16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float m = __uint_as_float(s16[0]) + __uint_as_float(s16[1]);  // rows (0+1, 0+1, 2+3, 2+3)
  const unsigned v = __float_as_uint(m);
  auto s32 = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(s32[0]) + __uint_as_float(s32[1]);
}

// K/V pages are read exactly once per iteration (plain loads: non-temporal loads were measured
// slower under the split).
template <typename T>
__device__ __forceinline__ T stream_load(const char* p) {
  return *reinterpret_cast<const T*>(p);
}

__device__ __forceinline__ uint64_t low_elems_mask(int n) {  // keep the first n of 4 bf16
  return n >= 4 ? ~0ull : (n <= 0 ? 0ull : ((1ull << (16 * n)) - 1ull));
}

template <int D>
struct Page {
  uint4 k[D / 32];  // K rows (token = lane % 16), 8 dims per lane per 32-dim step
  uint2 v[D / 16];  // V^T rows (dim = 16 n + lane % 16), tokens 4 (lane / 16) .. +4
};

template <int D>
__device__ __forceinline__ void load_page(Page<D>& pg, const char* kbase, const char* vbase, size_t slab, int lane) {
  const int row = lane & 15, quad = lane >> 4;
  constexpr size_t kPageBytes = 16 * D * 2;  // one (page, kv head) slab
  const char* kp = kbase + slab * kPageBytes + row * D * 2 + quad * 16;
  const char* vp = vbase + slab * kPageBytes + row * 32 + quad * 8;
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) pg.k[ks] = stream_load<uint4>(kp + ks * 64);
#pragma unroll
  for (int n = 0; n < D / 16; ++n) pg.v[n] = stream_load<uint2>(vp + n * 16 * 32);
}

__device__ __forceinline__ bool page_ok(int id, long long num_phys) { return id >= 0 && (long long)id < num_phys; }

// Uniform loads of the read-only work list through the scalar cache (used before the page stream
// starts; inside it a scalar load would be waited for together with every LDS operation).
__device__ __forceinline__ i32x4 sload4(const void* p) { return *(const __attribute__((address_space(4))) i32x4*)(p); }

// A decode work item as the host lists it: (q_start, req | kv head << 24, first page |
// (tokens - 1) << 22, row of its split-K partial).  The item covers `tokens` keys (at most 16 PPS)
// from its first logical page on.
struct DItem {
  int q_start, req, j, first_page, n_tok, slot;
  bool valid;
};
__device__ __forceinline__ DItem unpack_item(i32x4 v, bool valid) {
  DItem d;
  d.q_start = v.x;
  d.req = v.y & 0xffffff;
  d.j = (int)((unsigned)v.y >> 24);
  d.first_page = v.z & 0x3fffff;
  d.n_tok = (int)((unsigned)v.z >> 22) + 1;
  d.slot = v.w;
  d.valid = valid;
  return d;
}

// Merges the splits of one (decode request, query head) pair, pair = request * h_q + head, with
// one wave.  Lanes first take one split each to find the common max and the denominator, then take
// one dim each to sum the weighted outputs.
template <int D, typename OutT>
__device__ __forceinline__ void merge_pair(const AttnArgs& a, const WorkArgs& w, const float* pacc, const float* pml,
                                           void* out, int pair, int lane) {
  constexpr int E = D / 64;
  const int i = pair / a.h_q;
  const int h = pair - i * a.h_q;
  const int4 dr = w.dreq[i];
  const int g = a.group;
  const int j = h / g, col = h - j * g;
  const size_t base = (size_t)(dr.y + j * dr.z) * g + col;  // partial row of split 0
  const int n = dr.z;
  // Eight partial rows (splits s0 + t0 .. + 7 of the cnt from s0) are loaded before any is used,
  // so their loads overlap.
  float part[8][E];
  auto load_rows = [&](int s0, int t0, int cnt) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = min(t0 + u, cnt - 1);
      const float* pa = pacc + (base + (size_t)(s0 + t) * g) * D + lane;
#pragma unroll
      for (int e = 0; e < E; ++e) part[u][e] = pa[64 * e];
    }
  };
  auto load_ml = [&](int s) {
    return s < n ? *reinterpret_cast<const float2*>(pml + (base + (size_t)s * g) * 2) : make_float2(-INFINITY, 0.f);
  };
  // The first 64 splits' (max, denominator) pairs, the first eight partial rows and the output
  // row's request metadata are all in flight together: a request of up to eight splits costs one
  // memory round trip before its arithmetic.
  float2 ml = load_ml(lane);
  if (n > 0) load_rows(0, 0, min(64, n));  // every decode request has at least one split
  const int4 m = w.meta[dr.x];
  float M = ml.x;
  for (int s = lane + 64; s < n; s += 64) M = fmaxf(M, pml[(base + (size_t)s * g) * 2]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  float den = 0.f, num[E];
#pragma unroll
  for (int e = 0; e < E; ++e) num[e] = 0.f;
  for (int s0 = 0; s0 < n; s0 += 64) {
    const int s = s0 + lane;
    if (s0 > 0) ml = load_ml(s);
    const float wgt = s < n ? fast_exp2(ml.x - M) : 0.f;
    den += s < n ? wgt * ml.y : 0.f;
    const int cnt = min(64, n - s0);
    for (int t0 = 0; t0 < cnt; t0 += 8) {
      if (s0 > 0 || t0 > 0) load_rows(s0, t0, cnt);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float wt = t0 + u < cnt ? __shfl(wgt, t0 + u) : 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) num[e] += wt * part[u][e];
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) den += __shfl_xor(den, off);
  const float inv = 1.0f / den;
  OutT* o = reinterpret_cast<OutT*>(out) + ((size_t)m.y * a.h_q + h) * D;
#pragma unroll
  for (int e = 0; e < E; ++e) o[lane + 64 * e] = static_cast<OutT>(num[e] * inv);
}

// Persistent: the grid holds as many waves as fit on the CUs the stream may use; each wave takes
// one item by its index, then the next ones from a counter until the list is exhausted (every
// wave reaches the exit).  Items are listed longest first.  Which wave computes an item never changes its arithmetic.
//
// A wave streams pages through a ring of kRing register buffers without a break at item
// boundaries: while it works on one item it takes the next one from the counter, reads the
// item's descriptor, then its page ids and query; the next item's first pages are loaded while
// the current item's last pages are computed.  Each item is processed in groups of kRing pages
// (the last group padded with masked pages that re-read the item's last page), so a page's
// buffer is known at compile time and a load is never separated from its use by an early exit.
// Per-wave LDS staging of finished items' partials (floats): up to kStageFloats / (g d + 2 g)
// items (7 for g = 4, d = 128) are written out together, when the buffer is full or the wave's
// work is done.  A store's completion comes back late while the memory system streams reads, and
// vector memory operations complete in order, so every store burst stalls the page loads issued
// after it until it completes: one burst per buffer instead of one per item.
constexpr int kStageFloats = 4096;
template <int D, int PPS>
__global__ __launch_bounds__(256, 1) void decode_partial_bf16(AttnArgs a, WorkArgs w) {
  constexpr int R = kRing;
  static_assert(PPS % R == 0, "a split must hold whole groups of ring pages");
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, quad = lane >> 4;
  const int g = a.group;
  const int n_items = w.n_ditems;
  const char* kcache = reinterpret_cast<const char*>(a.k_cache);
  const char* vcache = reinterpret_cast<const char*>(a.v_cache);
  // Both caches are [P, h_kv, 16 * d] in bytes per (page, head) slab; fold h_kv into the page stride.
  const long long slab_stride_pages = a.h_kv;

  __shared__ __align__(16) float stage_lds[4 * kStageFloats];
  float* const stage = stage_lds + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * kStageFloats;
  const int ml_floats = (2 * g + 3) & ~3;
  const int item_floats = g * D + ml_floats;  // [g][d] output, then (m, l) per head
  const int n_slots = kStageFloats / item_floats;
  int n_staged = 0;     // items in the buffer
  int staged_rows = 0;  // lane k: partial row of buffered item k
  // Writes the buffered items to their partial rows, coalesced (LDS operations of one wave complete
  // in order, so the reads see the staging writes).
  auto flush = [&]() {
    for (int k = 0; k < n_staged; ++k) {
      const int row = __builtin_amdgcn_readlane(staged_rows, k);
      const float* src = stage + k * item_floats;
      float* dst = w.pacc + (size_t)row * g * D;
      for (int i = 4 * lane; i < g * D; i += 256)
        *reinterpret_cast<f32x4*>(dst + i) = *reinterpret_cast<const f32x4*>(src + i);
      if (lane < 2 * g) w.pml[(size_t)row * 2 * g + lane] = src[g * D + lane];
    }
    n_staged = 0;
  };

  // Wave v of the grid starts with item v; every item past the first n_waves is dealt round-robin
  // to n_queues counters (one atomic per item on a single counter would saturate it), and wave v
  // takes them from counter v % n_queues: ticket t is item n_waves + t n_queues + c.  Only one
  // item per wave is static, so from its second item on a wave that streams more slowly takes
  // fewer.  Every queue has a wave (n_waves >= n_queues), and a wave's tickets rise, as do their
  // items, all of them above the static ones: when a wave stops at an item past the end, every
  // ticket it still holds is past the end too.
  const int n_waves = gridDim.x * (blockDim.x >> 6);
  const int n_queues = n_waves >= kDecodeQueues ? kDecodeQueues : 1;
  const int first = blockIdx.x * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int queue = first % n_queues;
  int* const counter = w.work_counter + queue * kDecodeQueueStride;
  // The counter's old value, in lane 0; nothing touches it in the branch, so the load is waited
  // for only where it is read.
  auto grab = [&]() {
    int ticket = 0;
    if (lane == 0) ticket = atomicAdd(counter, 1);
    return ticket;
  };
  // An item's descriptor through the vector memory path, one word per lane: it completes in order
  // with the page loads issued before it, so waiting for it never drains the page stream.
  auto load_desc = [&](int idx) {
    return reinterpret_cast<const int*>(w.ditems)[(size_t)min(idx, n_items - 1) * 4 + (lane & 3)];
  };
  auto desc_item = [&](int words, int idx) {
    i32x4 v;
    v.x = __builtin_amdgcn_readlane(words, 0);
    v.y = __builtin_amdgcn_readlane(words, 1);
    v.z = __builtin_amdgcn_readlane(words, 2);
    v.w = __builtin_amdgcn_readlane(words, 3);
    return unpack_item(v, idx < n_items);
  };
  auto pages_of = [&](const DItem& it) { return min(PPS, (it.n_tok + 15) >> 4); };
  // The item's page ids, one per lane (at most PPS <= 64), and Q^T as the MFMA B operand:
  // column = head of the group, k = dims 32 ks + 8 quad .. +8.
  auto fetch_lane_data = [&](const DItem& it, int& ids, bf16x8 (&qf)[D / 32]) {
    const int* prow = a.page_table + (size_t)it.req * a.max_pages + it.first_page;
    ids = lane < pages_of(it) ? prow[lane] : 0;
    const __bf16* qrow = reinterpret_cast<const __bf16*>(a.q) + ((size_t)it.q_start * a.h_q + it.j * g + col) * D + quad * 8;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const uint4 u = col < g ? *reinterpret_cast<const uint4*>(qrow + ks * 32) : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, u);
    }
  };
  struct Ids {
    size_t slab;
    bool ok;
  };
  int bad = 0;
  // Page p (clamped to the item's last page) of an item whose ids a lane-distributed register holds.
  auto page_id = [&](int id_reg, int p, int n_pages, int j) {
    Ids r;
    const int id = __builtin_amdgcn_readlane(id_reg, min(p, n_pages - 1));
    r.ok = page_ok(id, a.num_phys_pages);
    bad |= !r.ok;
    r.slab = (size_t)(r.ok ? id : 0) * slab_stride_pages + j;
    return r;
  };

  // The deferred merge of the layer before: once a wave's item queue is empty (the launch's
  // tail, where waves would otherwise idle until the last items finish), it takes (request,
  // query head) pairs from merge queue `queue`: ticket t is pair t n_queues + queue.  Every queue
  // has a wave and every wave ends here, so every pair is merged.
  auto merge_tail = [&]() {
    if (w.n_merge == 0) return;
    int* const mcounter = w.work_counter + (kDecodeQueues + queue) * kDecodeQueueStride;
    for (;;) {
      int t = 0;
      if (lane == 0) t = atomicAdd(mcounter, 1);
      const int pair = __builtin_amdgcn_readfirstlane(t) * n_queues + queue;
      if (pair >= w.n_merge) break;
      merge_pair<D, __bf16>(a, w, w.merge_pacc, w.merge_pml, w.merge_out, pair, lane);
    }
  };
  // The counter set of the partial kernel before this one on the stream (it has finished).
  if (w.clear_counter && blockIdx.x == 0 && threadIdx.x < kDecodeSetLines)
    w.clear_counter[threadIdx.x * kDecodeQueueStride] = 0;

  if (first >= n_items) {
    merge_tail();
    return;
  }
  DItem cur = unpack_item(sload4(w.ditems + first), true);
  // The second item's ticket: its atomic returns while the first item's data loads.
  DItem nxt;
  {
    const int idx = n_waves + __builtin_amdgcn_readfirstlane(grab()) * n_queues + queue;
    nxt = desc_item(load_desc(idx), idx);
  }
  int cur_ids;
  bf16x8 qf[D / 32];
  fetch_lane_data(cur, cur_ids, qf);

  Page<D> buf[R];
  Ids ids[R];
  {
    const int np = pages_of(cur);
#pragma unroll
    for (int k = 0; k < R - 1; ++k) {
      ids[k] = page_id(cur_ids, k, np, cur.j);
      load_page<D>(buf[k], kcache, vcache, ids[k].slab, lane);
    }
  }

  for (;;) {
    const int n_pages = pages_of(cur);
    // At least two groups, so the next item's descriptor and ids (fetched in the first group)
    // are in before the last group loads its first pages.
    const int n_groups = max(2, (n_pages + R - 1) / R);
    const int n_tok = cur.n_tok;  // the item's tokens, from its first page on

    int ticket = 0, nn_words = 0, nn_idx = n_items, nxt_ids = 0;
    bf16x8 qn[D / 32];

    f32x4 acc[D / 16];
#pragma unroll
    for (int n = 0; n < D / 16; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    float l_run = 0.f;
    float m_ref = -INFINITY;  // reference max (base-2 units) the probabilities are taken against

    auto compute = [&](const Page<D>& pg, int p, const Ids& pid) {
      // Scores S^T: lane holds head `col`, tokens 4 quad + i of the page.
      f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pg.k[ks]), qf[ks], sc, 0, 0, 0);
      const int t0 = 16 * p + 4 * quad;
      // Tokens past the end (NaN-poisoned slots, and the padding pages of the last group) and
      // tokens of a bad page are masked; only the last pages of an item or a bad page need it.
      const bool tail = 16 * (p + 1) > n_tok || !pid.ok;
      if (tail) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!pid.ok || t0 + i >= n_tok) sc[i] = -INFINITY;
      }
      float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
      mx = max_rows(mx);
      mx *= a.scale_log2;  // the scale is positive: max of scaled = scaled max
      // The reference max moves only when a score exceeds it by more than the slack, so the
      // output rescale is rare; numerator and denominator share the reference.
      if (__any(mx > m_ref + kRescaleSlack)) {
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = fast_exp2(m_ref - m_new);
        m_ref = m_new;
        l_run *= alpha;
#pragma unroll
        for (int n = 0; n < D / 16; ++n) acc[n] *= alpha;
      }
      bf16x4 pb4;
#pragma unroll
      for (int i = 0; i < 4; ++i) pb4[i] = static_cast<__bf16>(fast_exp2(__builtin_fmaf(sc[i], a.scale_log2, -m_ref)));
      // The denominator sums the bf16 probabilities the PV product consumes.
      const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
      l_run = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb4[0], pb4[1]}, ones, l_run, false);
      l_run = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb4[2], pb4[3]}, ones, l_run, false);
      const s16x4 pbs = __builtin_bit_cast(s16x4, pb4);
      // Their values must not reach the MFMA either (0 x NaN is NaN).
      const uint64_t mk = !pid.ok ? 0ull : (tail ? low_elems_mask(n_tok - t0) : ~0ull);
#pragma unroll
      for (int n = 0; n < D / 16; ++n) {
        const uint64_t v = ((uint64_t)pg.v[n].y << 32 | pg.v[n].x) & mk;
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, v), pbs, acc[n], 0, 0, 0);
      }
    };

    // One group of R pages.  Every group issues the same loads in the same order (sources are
    // selected, never branched on), so the wait counts stay exact across the loop.  Items move
    // through a pipeline two deep: the first group takes a ticket for the item after next and
    // fetches the next item's ids and query; the last group reads the ticket (its atomic has
    // returned while the pages loaded after it did), loads that item's descriptor, then the next
    // item's first R - 1 pages (or, with no next item, re-reads).  No result is used right after
    // its load.
    auto group = [&](int grp, auto first_tag, auto last_tag) {
      constexpr bool kFirst = decltype(first_tag)::value;
      constexpr bool kLast = decltype(last_tag)::value;
#pragma unroll
      for (int u = 0; u < R; ++u) {
        if constexpr (kFirst) {
          if (u == 0) ticket = grab();
          if (u == 2) fetch_lane_data(nxt, nxt_ids, qn);  // a valid address even without a next item
        }
        if constexpr (kLast) {
          if (u == 0) {
            nn_idx = n_waves + __builtin_amdgcn_readfirstlane(ticket) * n_queues + queue;
            nn_words = load_desc(nn_idx);
          }
        }
        const int p = grp * R + u;
        const bool from_nxt = kLast && u > 0 && nxt.valid;
        const int src_ids = from_nxt ? nxt_ids : cur_ids;
        const int src_page = from_nxt ? u - 1 : p + R - 1;
        const int src_pages = from_nxt ? pages_of(nxt) : n_pages;
        const int src_j = from_nxt ? nxt.j : cur.j;
        ids[(u + R - 1) % R] = page_id(src_ids, src_page, src_pages, src_j);
        load_page<D>(buf[(u + R - 1) % R], kcache, vcache, ids[(u + R - 1) % R].slab, lane);
        compute(buf[u], p, ids[u]);
      }
    };
    using T = std::true_type;
    using F = std::false_type;
    group(0, T{}, F{});
    for (int grp = 1; grp < n_groups - 1; ++grp) group(grp, F{}, F{});
    group(n_groups - 1, F{}, T{});

    const float l_tot = sum_rows(l_run);
    {
      float* st = stage + n_staged * item_floats;
      if (col < g) {
#pragma unroll
        for (int n = 0; n < D / 16; ++n) *reinterpret_cast<f32x4*>(st + col * D + 16 * n + 4 * quad) = acc[n];
        if (quad == 0) {
          st[g * D + 2 * col + 0] = m_ref;
          st[g * D + 2 * col + 1] = l_tot;
        }
      }
      staged_rows = lane == n_staged ? cur.slot : staged_rows;
      ++n_staged;
    }
    if (n_staged == n_slots || !nxt.valid) flush();
    if (!nxt.valid) break;
    cur = nxt;
    nxt = desc_item(nn_words, nn_idx);
    cur_ids = nxt_ids;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) qf[ks] = qn[ks];
  }
  if (bad && lane == 0) atomicOr(w.err, 1);
  merge_tail();
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

// Merges every (decode request, query head) pair of one layer: one wave per pair.
template <int D, typename OutT>
__global__ __launch_bounds__(256) void decode_reduce(AttnArgs a, WorkArgs w) {
  // The partial kernel before this one on the stream has finished with its counter set: clear it
  // for the next call.
  if (blockIdx.x == 0 && threadIdx.x < kDecodeSetLines) w.work_counter[threadIdx.x * kDecodeQueueStride] = 0;
  const int pair = blockIdx.x * 4 + uniform(threadIdx.x >> 6);
  if (pair >= w.n_dreq * a.h_q) return;
  merge_pair<D, OutT>(a, w, w.pacc, w.pml, a.out, pair, threadIdx.x & 63);
}

}  // namespace

constexpr int kMinRounds = 4;      // items per wave the persistent grid is sized for, at least
constexpr int kMinWavesPerCu = 4;  // waves per CU of the share, at least

// Persistent grid size.  The memory system needs far fewer waves in flight than fit, so the grid
// is sized for at least kMinRounds items per wave (a short tail when the last items
// finish), but never below kMinWavesPerCu waves per CU (bandwidth on small CU
// shares) nor above what is resident at once.
template <int D>
hipError_t launch_persistent(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  static int per_cu = 0;  // resident 256-thread blocks per CU, from the occupancy calculator
  if (per_cu == 0) {
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, reinterpret_cast<const void*>(&decode_partial_bf16<D, kDecodePagesPerSplit>), 256, 0);
    if (e != hipSuccess) return e;
    if (per_cu < 1) per_cu = 1;
  }
  const int capacity = w.decode_cus * per_cu * 4;
  const int floor_waves = w.decode_cus * kMinWavesPerCu;
  const int want = (w.n_ditems + kMinRounds - 1) / kMinRounds;
  const int waves = std::max(1, std::min(capacity, std::max(want, floor_waves)));
  hipLaunchKernelGGL((decode_partial_bf16<D, kDecodePagesPerSplit>), dim3((waves + 3) / 4), dim3(256), 0, s, a, w);
  return hipGetLastError();
}

hipError_t launch_decode_partial(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  if (w.n_dreq == 0) return hipSuccess;
  const dim3 grid((a.h_kv * w.max_split + 3) / 4, w.n_dreq);
  if (a.dtype == 0) {
    if (w.pages_per_split != kDecodePagesPerSplit) return hipErrorInvalidValue;
    return a.head_dim == 128 ? launch_persistent<128>(a, w, s) : launch_persistent<64>(a, w, s);
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
