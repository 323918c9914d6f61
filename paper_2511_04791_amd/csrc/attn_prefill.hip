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
// through LDS 64 at a time (4 pages) in a 4-slot ring: K as [64 keys][d] and V as
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
//
// A unit with a long key range may run as several pieces, each over a run of its key tiles
// (kernels.h).  A piece keeps the same per-row state as a whole unit (reference max, denominator,
// unnormalised O^T) and stores it; the last piece of the unit to finish combines the stored
// states in piece order, m = max(m_a, m_b), O = 2^(m_a - m) O_a + 2^(m_b - m) O_b (likewise the
// denominator), and writes the normalised rows.  Inside a piece a row may see no key at all
// (its position lies before the piece's first key): its state stays (-inf, 0, 0).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "kernels.h"

namespace duet {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;  // two waves per SIMD
constexpr int kThreads = 64 * kWaves;
// LDS ring of kStages tiles: the tile in use plus kStages - 1 in flight.
constexpr int kStages = 4;
static_assert(kStages >= 2, "the ring needs a tile in use and one in flight");
constexpr float kRescaleSlack = 8.0f;  // base-2 units: probabilities stay below 2^8

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// Direct global-to-LDS load of 16 bytes per lane: lane i of the wave writes lds_block + 16 i.
// lds_block must be the same for the whole wave.
__device__ __forceinline__ void load_lds16(const char* src, __bf16* lds_block) {
  __builtin_amdgcn_global_load_lds(src, lds_block, 16, 0, 0);
}
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ bool page_ok(int id, long long num_phys) { return id >= 0 && (long long)id < num_phys; }

// Max and sum of a value over lanes l and l ^ 32, by the half-wave swap permute (a vector-ALU op;
// an LDS permute would wait behind the fragment reads in flight).  The swap returns the lane's own
// value and its partner's, in an order that depends on the half; both combinations are symmetric.
__device__ __forceinline__ float pair_max(float x) {
  const unsigned u = __float_as_uint(x);
  auto s = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const unsigned u = __float_as_uint(x);
  auto s = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// A-operand row rho of a 32-row MFMA tile carries key swap_bits23(rho): within each group of 16,
// bits 2 and 3 are exchanged, so output register v of lane l holds key 16 (v / 8) + 8 (l / 32) + v % 8.
__device__ __forceinline__ int swap_bits23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// LDS chunk swizzles.  A wave's K-operand reads touch rows swap_bits23(0..31) in groups of 8 or
// 16 lanes; its V-operand reads touch rows 0..31 in order.  Both maps give every such lane group
// distinct 16-byte bank groups, for both 8-lane and 16-lane LDS service.
__device__ __forceinline__ int kswz(int row) { return swap_bits23(row & 15); }
__device__ __forceinline__ int vswz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

__device__ __forceinline__ uint32_t keep_pairs(uint32_t word, int n_valid_in_pair) {
  return n_valid_in_pair >= 2 ? word : (n_valid_in_pair == 1 ? (word & 0xffffu) : 0u);
}

constexpr int kIdCap = kMaxPrefillKeys / 16;  // most page ids a unit can stage in LDS

// Dynamic LDS: the K/V ring, then the page ids of the unit (sized per launch for the longest
// prefill request, so short requests leave room for a second workgroup per CU).
template <int D>
struct PrefillSmem {
  static constexpr int kStageElems = 2 * kPrefillKeys * D;  // K tile + V^T tile, bf16
  static constexpr size_t kTileBytes = (size_t)kStages * kStageElems * 2;
  static constexpr size_t kMaxBytes = kTileBytes + kIdCap * sizeof(int);
  static size_t bytes(int id_cap) { return kTileBytes + (((size_t)id_cap + 3) & ~(size_t)3) * sizeof(int); }
};

template <int D, int NH>
__global__ __launch_bounds__(kThreads, 1) void prefill_bf16(AttnArgs a, WorkArgs w) {
  constexpr int BN = kPrefillKeys;       // keys per stage
  constexpr int KCH = D / 8;             // 16-byte chunks per K row
  constexpr int VCH = BN / 8;            // 16-byte chunks per V^T row
  constexpr int NK = D / 16;             // MFMA k-steps over the head dim
  constexpr int NO = D / 32;             // 32-dim output tiles
  constexpr int WPH = kWaves / NH;       // waves per head
  constexpr int QB = 32 * WPH;           // queries per unit
  extern __shared__ __attribute__((aligned(16))) __bf16 lds[];

  const int tid = threadIdx.x;
  const int wave = uniform(tid >> 6);
  const int lane = tid & 63;
  const int hh = lane >> 5;
  const int4 it = w.pitems[blockIdx.x];  // (req, first query head, q_row0, piece)
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

  // Key tiles [kt0, kt1) of the unit: all of them, or one piece's run.
  const int unit_tiles = (c + min(q_row0 + QB - 1, q_len - 1)) / BN + 1;
  const int piece = it.w & ((1 << kPrefillPieceBits) - 1);
  const int split_unit = (it.w >> kPrefillPieceBits) - 1;  // -1: whole unit
  // (first slot, pieces | tiles per piece << 16)
  const int2 su = split_unit >= 0 ? w.psplit[split_unit] : make_int2(0, 1 | (unit_tiles << 16));
  const int n_pieces = su.y & 0xffff, piece_tiles = su.y >> 16;
  const int kt0 = piece * piece_tiles;
  const int kt1 = min(unit_tiles, kt0 + piece_tiles);
  const int w_tiles = wrow0 < q_len ? (c + min(wrow0 + 31, q_len - 1)) / BN + 1 : 0;
  const int w_first_pos = c + wrow0;

  const char* kbase = reinterpret_cast<const char*>(a.k_cache);
  const char* vbase = reinterpret_cast<const char*>(a.v_cache);
  const int* prow = a.page_table + (size_t)r * a.max_pages;
  constexpr size_t kSlab = 16 * D * 2;  // bytes of one (page, kv head) slab, K or V
  int bad = 0;

  // The page ids of tiles kt0 .. kt1 - 1 go to LDS once (ids[i] = page 4 kt0 + i), so a tile
  // load never waits on a page-table read.
  int* ids = reinterpret_cast<int*>(reinterpret_cast<char*>(lds) + PrefillSmem<D>::kTileBytes);
  const int id0 = (BN / 16) * kt0;
  const int n_used_pages = min(n_pages, (kt1 * BN + 15) >> 4) - id0;
  // Ids are checked here, once: a missing page is recorded and replaced by page 0 (its keys lie
  // past the end, or the request is flagged).
  for (int i = tid; i < n_used_pages; i += kThreads) {
    const int id = prow[id0 + i];
    const bool ok = page_ok(id, a.num_phys_pages);
    bad |= !ok;
    ids[i] = ok ? id : 0;
  }
  __syncthreads();

  // Tiles arrive by direct global-to-LDS loads (16 bytes per lane; lane i of a wave writes bytes
  // 16 i .. 16 i + 15 of a 1 KiB LDS block).  Each tile is KB blocks of K and KB blocks of V^T;
  // wave w loads blocks w, w + kWaves, ...  A lane's source is fixed by the block and the lane
  // (the inverse of the LDS chunk swizzle) except for the page id, so only the id changes per
  // tile.  Loads run kStages - 1 tiles ahead of the tile in use.
  constexpr int KB = BN * D * 2 / 1024;   // 1 KiB blocks per tile per tensor
  constexpr int BPW = KB / kWaves;        // blocks per wave per tensor
  static_assert(BPW >= 1 && KB % kWaves == 0, "tile blocks must divide evenly among waves");
  int k_pi[BPW], k_off[BPW], v_pi[BPW], v_off[BPW];
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int blk = wave + kWaves * i;
    const int krow = (64 / KCH) * blk + lane / KCH;           // key row of the K tile
    const int kc = (lane % KCH) ^ (kswz(krow) & (KCH - 1));   // logical 16-byte chunk of the row
    k_pi[i] = krow >> 4;
    k_off[i] = (krow & 15) * (D * 2) + kc * 16;
    const int vrow = 8 * blk + lane / 8;                      // dim row of the V^T tile
    const int vc = (lane % 8) ^ (vswz(vrow) & (VCH - 1));     // logical chunk: 8 keys
    v_pi[i] = vc >> 1;
    v_off[i] = vrow * 32 + (vc & 1) * 16;
  }
  // Per-lane parts of the tile addresses.  A K block lies inside one page (uniform over the wave),
  // so its address is a scalar page base plus the lane's 32-bit offset; a V^T block spans the
  // tile's pages, so each lane adds its page's slab to a 64-bit base.  Pages past the request's
  // end (only in its last tile) re-read its last page: their keys are masked and their values
  // zeroed before use.
  const size_t page_stride = (size_t)a.h_kv * kSlab;
  const char* kbase_j = kbase + (size_t)j * kSlab;
  const char* vlane[BPW];
#pragma unroll
  for (int i = 0; i < BPW; ++i) vlane[i] = vbase + (size_t)j * kSlab + v_off[i];
  const int last_page = n_pages - 1 - id0;
  auto issue_tile = [&](int kt) {
    __bf16* kdst = lds + (kt % kStages) * PrefillSmem<D>::kStageElems;
    __bf16* vdst = kdst + BN * D;
    int kid[BPW], vid[BPW];  // all ids first: one LDS wait for the tile
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      kid[i] = ids[min(4 * kt + k_pi[i] - id0, last_page)];
      vid[i] = ids[min(4 * kt + v_pi[i] - id0, last_page)];
    }
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int blk = wave + kWaves * i;
      load_lds16(kbase_j + (size_t)uniform(kid[i]) * page_stride + k_off[i], kdst + blk * 512);
      load_lds16(vlane[i] + (size_t)(unsigned)vid[i] * page_stride, vdst + blk * 512);
    }
  };
  // Waits until this wave's loads of all but the `later` most recent tiles have landed
  // (later <= kStages - 2).
  auto wait_tiles = [&](int later) {
    constexpr int L1 = 2 * BPW, L2 = 4 * BPW;  // loads of one and of two tiles
    static_assert(kStages <= 4 && L2 < 64, "wait counts are spelled out for up to two later tiles");
    // s_waitcnt: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt left at their maxima
    if (kStages >= 4 && later >= 2) __builtin_amdgcn_s_waitcnt((L2 & 15) | ((L2 >> 4) << 14) | 0x0F70);
    else if (kStages >= 3 && later >= 1) __builtin_amdgcn_s_waitcnt((L1 & 15) | ((L1 >> 4) << 14) | 0x0F70);
    else __builtin_amdgcn_s_waitcnt(0x0F70);
  };
  // Values of keys >= L (NaN-poisoned tail slots, stand-in pages) must not reach the MFMA: the
  // tile holding key L - 1 has them zeroed in LDS before first use.
  const int kt_tail = (L - 1) / BN;
  const int tail_keys = L - BN * kt_tail;  // valid keys of that tile, 1 .. BN
  auto zero_tail = [&](int kt) {
    if (kt != kt_tail || tail_keys == BN) return false;
    __bf16* vs = lds + (kt % kStages) * PrefillSmem<D>::kStageElems + BN * D;
    for (int x = tid; x < D * VCH; x += kThreads) {
      const int vrow = x / VCH;
      const int sc = x % VCH;
      const int c = sc ^ (vswz(vrow) & (VCH - 1));
      const int first = 8 * c;
      if (first + 8 <= tail_keys) continue;
      uint4* p = reinterpret_cast<uint4*>(vs + vrow * BN + sc * 8);
      if (first >= tail_keys) {
        *p = make_uint4(0, 0, 0, 0);
      } else {
        uint4 v = *p;
        const int nv = tail_keys - first;
        v.x = keep_pairs(v.x, nv);
        v.y = keep_pairs(v.y, nv - 2);
        v.z = keep_pairs(v.z, nv - 4);
        v.w = keep_pairs(v.w, nv - 6);
        *p = v;
      }
    }
    return true;
  };
  // Makes tile kt visible to every wave: this wave's loads of it have landed (the `later`
  // newer tiles may still be in flight), then a barrier; the tail tile gets its fix-up.
  auto publish = [&](int kt, int later) {
    wait_tiles(later);
    __builtin_amdgcn_s_barrier();
    if (zero_tail(kt)) {
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the fix-up's LDS writes are done
      __builtin_amdgcn_s_barrier();
    }
  };

  f32x16 oacc[NO];
#pragma unroll
  for (int n = 0; n < NO; ++n)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[n][v] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;
  float m_sub = 0.f;  // m_ref where it is finite, else 0: a row with no key yet gets 2^-inf = 0

  for (int t = kt0; t < kt0 + kStages - 1 && t < kt1; ++t) issue_tile(t);
  publish(kt0, min(kt1 - 1, kt0 + kStages - 2) - kt0);
  // The query fragments have landed before the loop (tile 0's wait above covers them in
  // hardware, but the compiler would otherwise keep them pending at the loop head and make every
  // step's first MFMA wait for all tile loads in flight, collapsing the ring to one tile).
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)

  // S^T of key tile kt for this wave's 32 rows: K fragments from LDS, Q^T from registers.
  auto scores = [&](int kt, f32x16 (&sacc)[2]) {
    const __bf16* ks = lds + (kt % kStages) * PrefillSmem<D>::kStageElems;
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
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[nb][v] = 0.f;
    // The score MFMAs and the V fragment reads after them issue at a raised wave priority: a wave
    // that reaches them first keeps the matrix core while its SIMD partner is still in its
    // softmax, so the two waves of a SIMD drift out of phase (measured 1-3% faster; priority
    // around the PV products was slower).
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        sacc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[nb][kk], qf[kk], sacc[nb], 0, 0, 0);
  };

  for (int kt = kt0; kt < kt1; ++kt) {
    // Stage (kt + kStages - 1) % kStages held tile kt - 1, which every wave has left (the barrier
    // that ended step kt - 1).  Issuing at the top of the step, right after that barrier, gives
    // the loads a whole step more than issuing at its end (measured: 2-3% on long chunks).
    if (kt + kStages - 1 < kt1) issue_tile(kt + kStages - 1);
    if (kt < w_tiles) {
      f32x16 sacc[2];
      scores(kt, sacc);
      const __bf16* vs = lds + (kt % kStages) * PrefillSmem<D>::kStageElems + BN * D;
      // V fragments are read now; their LDS latency hides behind the softmax below.
      bf16x8 vf[NO][4];
#pragma unroll
      for (int n = 0; n < NO; ++n) {
        const int vrow = 32 * n + (lane & 31);
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) {
          const int ch = (2 * k2 + hh) ^ (vswz(vrow) & (VCH - 1));
          vf[n][k2] = *reinterpret_cast<const bf16x8*>(vs + vrow * BN + ch * 8);
        }
      }
      __builtin_amdgcn_s_setprio(0);
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
      mx = pair_max(mx) * a.scale_log2;
      // Move the reference max only when some score exceeds it by more than the slack.
      if (__any(mx > m_ref + kRescaleSlack)) {
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_ref - m_new);
        m_ref = m_new;
        m_sub = m_new == -INFINITY ? 0.f : m_new;
        l_run *= alpha;
#pragma unroll
        for (int n = 0; n < NO; ++n) oacc[n] *= alpha;
      }
      bf16x8 pb[4];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          pb[2 * nb + (v >> 3)][v & 7] = static_cast<__bf16>(fast_exp2(__builtin_fmaf(sacc[nb][v], a.scale_log2, -m_sub)));
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
      for (int n = 0; n < NO; ++n)
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2)
          oacc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[n][k2], pb[k2], oacc[n], 0, 0, 0);
    }
    // Tile kt + 1 for the next step; tiles kt + 2 and kt + 3 stay in flight.
    if (kt + 1 < kt1) publish(kt + 1, min(kt1 - 1, kt + kStages - 1) - (kt + 1));
  }

  if (bad) atomicOr(w.err, 1);
  if (split_unit >= 0) {
    // Slot layout, in float pairs: O as [wave][n][v / 2][lane], then (m, l) as [wave][lane]; every
    // lane stores and later loads exactly its own registers.  The slots are written and read with
    // relaxed device-scope atomic accesses (coherent across the XCDs' L2 caches without the
    // whole-cache write-back and invalidation a device-scope fence costs every workgroup on the
    // XCD); a piece counts itself only once its stores have completed.
    constexpr size_t kSlotPairs = (size_t)kThreads * (D / 4 + 1);
    typedef unsigned long long u64;
    auto o_at = [&](int slot) {
      return reinterpret_cast<u64*>(w.ppart) + (size_t)slot * kSlotPairs + (size_t)wave * NO * 8 * 64 + lane;
    };
    auto ml_at = [&](int slot) {
      return reinterpret_cast<u64*>(w.ppart) + (size_t)slot * kSlotPairs + (size_t)kThreads * (D / 4) +
             (size_t)wave * 64 + lane;
    };
    auto pack = [](float x, float y) {
      return (u64)__float_as_uint(x) | ((u64)__float_as_uint(y) << 32);
    };
    auto lo = [](u64 v) { return __uint_as_float((unsigned)v); };
    auto hi = [](u64 v) { return __uint_as_float((unsigned)(v >> 32)); };
    {
      u64* o = o_at(su.x + piece);
#pragma unroll
      for (int n = 0; n < NO; ++n)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2)
          __hip_atomic_store(o + (n * 8 + v2) * 64, pack(oacc[n][2 * v2], oacc[n][2 * v2 + 1]), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(ml_at(su.x + piece), pack(m_ref, l_run), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's slot stores have completed
    __syncthreads();
    // The arrival flag reuses the page-id table's first word: no id is read after the key loop.
    if (tid == 0) {
      const int done = atomicAdd(w.pcount + split_unit, 1) + 1;
      ids[0] = done == n_pieces;
      if (done == n_pieces) atomicExch(w.pcount + split_unit, 0);  // ready for the next launch
    }
    __syncthreads();
    if (!ids[0]) return;
    // The last piece: combine the states in piece order (its own from registers, the others from
    // their slots), so the result does not depend on which piece finished last.
    f32x16 own[NO];
#pragma unroll
    for (int n = 0; n < NO; ++n) own[n] = oacc[n];
    const u64 own_ml = pack(m_ref, l_run);
    for (int pc = 0; pc < n_pieces; ++pc) {
      f32x16 op[NO];
      u64 ml;
      if (pc == piece) {
        ml = own_ml;
#pragma unroll
        for (int n = 0; n < NO; ++n) op[n] = own[n];
      } else {
        const u64* o = o_at(su.x + pc);
        ml = __hip_atomic_load(ml_at(su.x + pc), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int n = 0; n < NO; ++n)
#pragma unroll
          for (int v2 = 0; v2 < 8; ++v2) {
            const u64 v = __hip_atomic_load(o + (n * 8 + v2) * 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            op[n][2 * v2] = lo(v);
            op[n][2 * v2 + 1] = hi(v);
          }
      }
      if (pc == 0) {
        m_ref = lo(ml);
        l_run = hi(ml);
#pragma unroll
        for (int n = 0; n < NO; ++n) oacc[n] = op[n];
      } else {
        const float m_b = lo(ml);
        const float m_new = fmaxf(m_ref, m_b);
        const float fa = m_new == -INFINITY ? 1.f : fast_exp2(m_ref - m_new);
        const float fb = m_new == -INFINITY ? 0.f : fast_exp2(m_b - m_new);
        m_ref = m_new;
        l_run = l_run * fa + hi(ml) * fb;
#pragma unroll
        for (int n = 0; n < NO; ++n) oacc[n] = oacc[n] * fa + op[n] * fb;
      }
    }
  }
  const float l_tot = pair_sum(l_run);
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
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)PrefillSmem<D>::kMaxBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((prefill_bf16<D, NH>), dim3(w.n_pitems), dim3(kThreads), PrefillSmem<D>::bytes(w.prefill_id_cap),
                     s, a, w);
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
  // largest power of two <= min(group, waves per workgroup) that divides the group
  int nh = 1;
  while (nh * 2 <= kWaves && group % (nh * 2) == 0) nh *= 2;
  return nh;
}

int prefill_rows_per_unit(int group, int dtype) {
  return dtype == 0 ? 32 * kWaves / prefill_heads_per_unit(group) : kPrefillRows;
}

int prefill_piece_tiles_for(long long total_tiles) {
  const long long even = (total_tiles + kPrefillPieceFill - 1) / kPrefillPieceFill;
  return (int)std::max<long long>(kPrefillPieceMinTiles, even);
}

size_t prefill_slot_bytes(int head_dim) { return (size_t)kThreads * (head_dim / 2 + 2) * sizeof(float); }

hipError_t launch_prefill(const AttnArgs& a, const WorkArgs& w, hipStream_t s) {
  if (w.n_pitems == 0) return hipSuccess;
  if (a.dtype == 0) return a.head_dim == 128 ? launch_bf16_nh<128>(a, w, s) : launch_bf16_nh<64>(a, w, s);
  const dim3 grid(w.n_pitems);
  if (a.head_dim == 128) hipLaunchKernelGGL(prefill_f32<128>, grid, dim3(256), 0, s, a, w);
  else hipLaunchKernelGGL(prefill_f32<64>, grid, dim3(256), 0, s, a, w);
  return hipGetLastError();
}

}  // namespace duet
