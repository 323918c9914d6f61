// Runtime behind the C ABI: context, CU-masked stream pool, per-iteration work lists, the
// temporal (aggregated) and spatial (CU-split) launch of the two attention halves, the page
// gather export, probes and calibration.
//
// Spatial sharing (paper, Section 4.3): the decode half and the prefill half run on two streams
// bound to disjoint CU sets.  On MI355X a stream's CU set is fixed when it is created
// (hipExtStreamCreateWithCUMask), so the context keeps one stream per distinct CU set and reuses
// it; choosing a split costs a map lookup.  The decode half is enqueued first (Section 4.3:
// decode is dispatched ahead of prefill so it never waits behind prefill launches).  The
// caller's stream forks to both with one event and joins both with two.
//
// CU mask bits: the runtime assumes bit i of the mask selects a CU on XCD (i mod 8), so a run
// of 8 consecutive bits takes one CU from each of the 8 XCDs; decode takes bits from the low
// end, prefill from the high end.  The placement probe verifies this on the device.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

#include "duet_internal.h"
#include "gemm.h"
#include "kernels.h"

namespace {

using namespace duet;

constexpr int kStagingSlots = 4;
// Each CU-masked stream owns a hardware queue.  Only the current split's pair is kept: with more
// masked queues alive, the decode half of a pair created second in a process ran 20-30% slower
// and its reduce kernel 4-5x slower beside a running prefill (same CUs reached, measured with the
// placement probe), while a pair that reuses the freed queues runs at full speed.  Changing the
// split then recreates two streams, which a serving loop does only when Algorithm 1 switches.
constexpr size_t kMaxMaskedStreams = 2;
constexpr size_t kAlign = 256;
// Workspace head: the device error word at offset 0 and the decode queue counters from
// kCounterOffset on; the head is zeroed by every call's upload.
constexpr size_t kCounterOffset = 128;
constexpr int kMaxLayers = 1024;
constexpr int kMaxLookahead = 64;     // decode steps per look-ahead call
constexpr size_t kMaxGraphs = 128;    // cached decode-step graphs per context
// Scratch of duet_attn_mixed_batch_noalloc: the workspace of one call (work lists, decode queue
// counters, split-K partials) in a file-scope device array, for callers that cannot allocate.
// Each device the library runs on holds its own copy until the process ends.  In host code the
// array's name is not a device address: its address on a device comes from hipGetSymbolAddress
// (duet_init, with the device current) and is kept in the context.
constexpr size_t kScratchBytes = size_t(64) << 20;
// Pinned staging allocated up front for each slot, so that the no-allocation path never grows it.
constexpr size_t kStagingPrealloc = size_t(1) << 20;

inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

static __device__ __align__(256) char scratch[kScratchBytes];
static_assert(kScratchBytes == DUET_NOALLOC_SCRATCH_BYTES, "the header states the scratch size");

#define HIP_TRY(expr)                                                                       \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(DUET_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

struct StagingSlot {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t done = nullptr;
  bool pending = false;
};

// Decode work lists of one look-ahead step s >= 1 (its own metadata: decode request r becomes
// (decode, i, 1, cached_len + s), i = its index among the decode requests).
struct StepPlan {
  std::vector<int4> meta, dreq;
  std::vector<int4> ditems;
  int n_items = 0, max_split = 0;
  size_t off_meta = 0, off_dreq = 0, off_ditems = 0;
};

// Work lists of one iteration and where they live in the caller's workspace.
struct Plan {
  std::vector<int4> meta, pitems, dreq;
  std::vector<int2> psplit;  // per split prefill unit: (first partial slot, pieces | tiles per piece << 16)
  std::vector<int4> ditems;
  std::vector<StepPlan> ahead;  // look-ahead decode steps 1 .. steps - 1
  int steps = 1;
  int n_items_decode = 0, max_split = 0, pages_per_split = 0, group = 0, prefill_id_cap = 0;
  int prefill_piece_tiles = 0, n_split_units = 0, n_slots = 0;
  size_t off_meta = 0, off_pitems = 0, off_dreq = 0, off_ditems = 0, off_psplit = 0, off_pcount = 0, off_ppart = 0,
         upload_bytes = 0, total = 0;
  // Two buffers of split-K partials: consecutive layers of a call alternate between them, so a
  // layer's partials survive until the next layer's decode kernel has merged them.
  size_t off_pacc[2] = {0, 0}, off_pml[2] = {0, 0};
};

// Fixed per dtype, never per split or placement, so results are identical for every CU split.
int pages_per_split_for(const duet_shape* s) {
  return s->dtype == DUET_F32 ? kDecodePagesPerSplitF32 : kDecodePagesPerSplit;
}

// Decode work of the batch's decode requests when each holds `extra` more tokens than seq_meta
// states: per request (req, item_base, n_split, n_pages), and for bf16 the work items in
// execution order -- every full split first, then the shorter last splits, longest first -- as
// descriptors (q_start, req | kv head << 24, first page | (tokens - 1) << 22, row of the split's
// partial).  With step_rows (look-ahead steps), decode request i reads its query from row i.
// A (request, kv head) range of n_pages pages is cut into splits of pps pages from page 0, the
// last one short.
void decode_lists(const duet_shape* s, const duet_batch* b, int extra, bool step_rows, bool fill,
                  std::vector<int4>* dreq, std::vector<int4>* ditems, int64_t* n_dreq, int64_t* n_items,
                  int* max_split) {
  const int pps = pages_per_split_for(s);
  dreq->clear();
  ditems->clear();
  *n_dreq = 0;
  *n_items = 0;
  *max_split = 0;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& q = b->reqs[r];
    if (q.kind != DUET_KIND_DECODE) continue;
    const int64_t L = (int64_t)q.cached_len + q.q_len + extra;
    const int n_pages = (int)((L + 15) / 16);
    const int n_split = (n_pages + pps - 1) / pps;
    if (fill) dreq->push_back(make_int4(r, (int)*n_items, n_split, n_pages));
    *n_items += (int64_t)s->num_kv_heads * n_split;
    *max_split = std::max(*max_split, n_split);
    ++*n_dreq;
  }
  if (fill && s->dtype == DUET_BF16) {
    ditems->reserve(*n_items);
    struct Part {
      int pages;
      int4 item;
    };
    std::vector<Part> parts;
    for (size_t i = 0; i < dreq->size(); ++i) {
      const int4 d = (*dreq)[i];
      const duet_seq_meta& q = b->reqs[d.x];
      const int L = q.cached_len + q.q_len + extra;
      const int q_start = step_rows ? (int)i : q.q_start;
      for (int j = 0; j < s->num_kv_heads; ++j)
        for (int sp = 0; sp < d.z; ++sp) {
          const int first = sp * pps;
          const int tokens = std::min(16 * pps, L - 16 * first);
          const int pages = (tokens + 15) / 16;
          const int4 it = make_int4(q_start, d.x | (j << 24), first | ((tokens - 1) << 22), d.y + j * d.z + sp);
          if (pages == pps) ditems->push_back(it);
          else parts.push_back({pages, it});
        }
    }
    std::stable_sort(parts.begin(), parts.end(), [](const Part& x, const Part& y) { return x.pages > y.pages; });
    for (const Part& pt : parts) ditems->push_back(pt.item);
  }
}

// Work lists of a call over `layers` layers and `steps` decode steps (steps > 1: look-ahead),
// and their offsets in the workspace.
void plan_batch(const duet_shape* s, const duet_batch* b, int layers, int steps, Plan* p, bool fill) {
  const int g = s->num_q_heads / s->num_kv_heads;
  const int pps = pages_per_split_for(s);
  p->group = g;
  p->pages_per_split = pps;
  p->prefill_id_cap = 0;
  p->meta.clear();
  p->pitems.clear();
  p->steps = steps;
  p->psplit.clear();
  const bool bf16 = s->dtype == DUET_BF16;
  // bf16: a unit is nh heads of one group x rows queries; fp32: one head x rows queries.
  const int nh = bf16 ? prefill_heads_per_unit(g) : 1;
  const int rows = prefill_rows_per_unit(g, bf16 ? 0 : 1);
  const int units = s->num_q_heads / nh;
  // Key tiles of row block t of a request (the causal range of its last row).
  auto block_tiles = [&](const duet_seq_meta& q, int t) {
    return (int)(((int64_t)q.cached_len + std::min(q.q_len, (t + 1) * rows) - 1) / kPrefillKeys + 1);
  };
  int64_t total_tiles = 0;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& q = b->reqs[r];
    if (q.kind != DUET_KIND_PREFILL) continue;
    for (int t = 0; t * rows < q.q_len; ++t) total_tiles += (int64_t)block_tiles(q, t) * units;
  }
  const int P = bf16 && total_tiles > 0 ? prefill_piece_tiles_for(total_tiles) : 0;
  p->prefill_piece_tiles = P;
  // Units longer than 1.5 P: n pieces of equal length (the last may be shorter), none empty.
  auto pieces_of = [&](int nt) { return P > 0 && 2 * nt > 3 * P ? (nt + P - 1) / P : 1; };
  // Tail split: when the whole units (those the rule above leaves in one piece) number more than
  // two rounds of one workgroup per CU of the whole chip, the shortest round of them -- the last
  // dispatched -- runs as kPrefillTailPieces pieces each (of at least kPrefillTailMinTiles
  // tiles), so the final round is fine-grained on any CU share.  It depends on the batch only.
  std::vector<std::pair<int, int>> tail_blocks;  // (request, row block), sorted
  if (bf16 && P > 0) {
    struct Whole {
      int nt, r, t;
    };
    std::vector<Whole> whole;
    int64_t n_whole_units = 0;
    for (int r = 0; r < b->num_reqs; ++r) {
      const duet_seq_meta& q = b->reqs[r];
      if (q.kind != DUET_KIND_PREFILL) continue;
      for (int t = 0; t * rows < q.q_len; ++t) {
        const int nt = block_tiles(q, t);
        if (pieces_of(nt) == 1) {
          whole.push_back({nt, r, t});
          n_whole_units += units;
        }
      }
    }
    if (n_whole_units >= 2 * kPrefillPieceFill) {
      std::stable_sort(whole.begin(), whole.end(), [](const Whole& x, const Whole& y) { return x.nt < y.nt; });
      int64_t taken = 0;
      for (const Whole& w : whole) {
        if (taken >= kPrefillPieceFill) break;
        if (w.nt >= kPrefillTailPieces * kPrefillTailMinTiles) tail_blocks.emplace_back(w.r, w.t);
        taken += units;
      }
      std::sort(tail_blocks.begin(), tail_blocks.end());
    }
  }
  int64_t n_pitems = 0;
  int n_su = 0, n_slots = 0;
  struct Tile {
    int64_t keys;
    int4 item;
  };
  std::vector<Tile> tiles;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& q = b->reqs[r];
    if (fill) p->meta.push_back(make_int4(q.kind, q.q_start, q.q_len, q.cached_len));
    const int64_t L = (int64_t)q.cached_len + q.q_len;
    if (q.kind != DUET_KIND_PREFILL) continue;
    p->prefill_id_cap = std::max(p->prefill_id_cap, (int)((L + 15) / 16));
    for (int t = 0; t * rows < q.q_len; ++t) {
      const int nt = block_tiles(q, t);
      int pieces = pieces_of(nt);
      if (pieces == 1 && std::binary_search(tail_blocks.begin(), tail_blocks.end(), std::make_pair(r, t)))
        pieces = kPrefillTailPieces;
      const int len = (nt + pieces - 1) / pieces;
      pieces = (nt + len - 1) / len;
      n_pitems += (int64_t)pieces * units;
      if (pieces > 1) {
        if (fill)
          for (int u = 0; u < units; ++u) p->psplit.push_back(make_int2(n_slots + u * pieces, pieces | (len << 16)));
        n_su += units;
        n_slots += units * pieces;
      }
      if (!fill) continue;
      // Units ordered so that workgroup index mod 8 follows the kv head: the units sharing one kv
      // head land on one XCD and share its L2.  Piece pc of every unit of a block, then piece
      // pc + 1: pieces of equal length stay together through the sort below.
      for (int pc = 0; pc < pieces; ++pc) {
        const int64_t keys = pieces > 1 ? (int64_t)std::min(len, nt - pc * len) * kPrefillKeys
                                        : q.cached_len + std::min(q.q_len, (t + 1) * rows);
        for (int u = 0; u < units; ++u) {
          const int h = nh == 1 ? (u % s->num_kv_heads) * g + u / s->num_kv_heads : u * nh;
          const int su = pieces > 1 ? n_su - units + u : -1;
          tiles.push_back({keys, make_int4(r, h, t * rows, ((su + 1) << kPrefillPieceBits) | (pieces > 1 ? pc : 0))});
        }
      }
    }
  }
  p->n_split_units = n_su;
  p->n_slots = n_slots;
  if (fill) {
    std::stable_sort(tiles.begin(), tiles.end(), [](const Tile& x, const Tile& y) { return x.keys > y.keys; });
    p->pitems.reserve(tiles.size());
    for (const Tile& t : tiles) p->pitems.push_back(t.item);
  }
  int64_t n_dreq = 0, n_items = 0;
  int max_split = 0;
  decode_lists(s, b, 0, false, fill, &p->dreq, &p->ditems, &n_dreq, &n_items, &max_split);
  p->n_items_decode = (int)n_items;
  p->max_split = max_split;
  size_t off = align_up(kCounterOffset + (size_t)kDecodeCounterInts * sizeof(int32_t));
  p->off_meta = off;
  off = align_up(off + (size_t)b->num_reqs * sizeof(int4));
  p->off_pitems = off;
  off = align_up(off + (size_t)n_pitems * sizeof(int4));
  p->off_dreq = off;
  off = align_up(off + (size_t)n_dreq * sizeof(int4));
  p->off_ditems = off;
  off = align_up(off + (s->dtype == DUET_BF16 ? (size_t)n_items * sizeof(int4) : 0));
  p->off_psplit = off;
  off = align_up(off + (size_t)n_su * sizeof(int2));
  p->off_pcount = off;  // zeroed by the upload
  off = align_up(off + (size_t)n_su * sizeof(int32_t));
  // Look-ahead steps: each has its own metadata and decode lists; the split-K partials are
  // shared, since the steps run one after another on one stream.
  int64_t max_items = n_items;
  p->ahead.resize(steps - 1);
  for (int st = 1; st < steps; ++st) {
    StepPlan& sp = p->ahead[st - 1];
    sp.meta.clear();
    if (fill) {
      int i = 0;
      for (int r = 0; r < b->num_reqs; ++r) {
        const duet_seq_meta& q = b->reqs[r];
        if (q.kind == DUET_KIND_DECODE) sp.meta.push_back(make_int4(q.kind, i++, 1, q.cached_len + st));
        else sp.meta.push_back(make_int4(q.kind, q.q_start, q.q_len, q.cached_len));
      }
    }
    int64_t nd = 0, ni = 0;
    decode_lists(s, b, st, true, fill, &sp.dreq, &sp.ditems, &nd, &ni, &sp.max_split);
    sp.n_items = (int)ni;
    max_items = std::max(max_items, ni);
    sp.off_meta = off;
    off = align_up(off + (size_t)b->num_reqs * sizeof(int4));
    sp.off_dreq = off;
    off = align_up(off + (size_t)nd * sizeof(int4));
    sp.off_ditems = off;
    off = align_up(off + (s->dtype == DUET_BF16 ? (size_t)ni * sizeof(int4) : 0));
  }
  p->upload_bytes = off;
  for (int b = 0; b < 2; ++b) {
    p->off_pacc[b] = off;
    off = align_up(off + (size_t)max_items * g * s->head_dim * sizeof(float));
    p->off_pml[b] = off;
    off = align_up(off + (size_t)max_items * g * 2 * sizeof(float));
  }
  p->off_ppart = off;
  off = align_up(off + (size_t)n_slots * prefill_slot_bytes(s->head_dim));
  p->total = off;
}

// Prefill units on a CU share: the units are listed longest first in rounds of 8 (one per XCD,
// workgroup index mod 8), and each XCD's workgroups are dealt evenly to its shader engines, so a
// plain longest-first list gives one engine the longest unit of every round.  Reversing the rounds
// inside every other block of four balances the engines' work (the 2048-token chunk on 96 CUs:
// 126 vs 131 us); on all 256 CUs the plain order is kept (the long 70B chunk: 1% faster).  A
// permutation of whole rounds: every XCD keeps its units.
void snake_prefill_rounds(std::vector<int4>* items) {
  std::vector<int4>& v = *items;
  for (size_t b0 = 32; b0 + 32 <= v.size(); b0 += 64)
    for (int a = 0, z = 3; a < z; ++a, --z)
      for (int u = 0; u < 8; ++u) std::swap(v[b0 + 8 * a + u], v[b0 + 8 * z + u]);
}

// Fork and join of a profiled call on the caller's stream; A and B bracket probe kernels.
enum ProfEv { kEvFork, kEvJoin, kEvA, kEvB, kNumProfEv };

// One kernel launch of a decode step; a step's launches are what its graph captures.
struct DecodeLaunch {
  enum Kind { kAppend, kPartial, kReduce } kind;
  AttnArgs a;
  WorkArgs w;
  AppendArgs ap;
};

hipError_t run_launch(const DecodeLaunch& l, hipStream_t st) {
  switch (l.kind) {
    case DecodeLaunch::kAppend: return launch_kv_append(l.ap, l.w, st);
    case DecodeLaunch::kPartial: return launch_decode_partial(l.a, l.w, st);
    default: return launch_decode_reduce(l.a, l.w, st);
  }
}

template <typename T>
inline uint64_t bits(T x) {
  static_assert(sizeof(T) <= 8, "field wider than a key word");
  uint64_t u = 0;
  std::memcpy(&u, &x, sizeof x);
  return u;
}

// Every argument that reaches a kernel (and so fixes a launch's grid), field by field: two
// steps with equal keys launch identical kernels, so a graph captured for one replays the other.
void append_key(std::vector<uint64_t>* k, const DecodeLaunch& l) {
  const AttnArgs& a = l.a;
  const WorkArgs& w = l.w;
  const AppendArgs& p = l.ap;
  const uint64_t f[] = {(uint64_t)l.kind, bits(a.q), bits(a.k_cache), bits(a.v_cache), bits(a.page_table),
                        bits(a.out), bits(a.num_phys_pages), bits(a.max_pages), bits(a.h_q), bits(a.h_kv),
                        bits(a.group), bits(a.head_dim), bits(a.dtype), bits(a.scale_log2), bits(w.meta),
                        bits(w.pitems), bits(w.dreq), bits(w.pacc), bits(w.pml), bits(w.ditems), bits(w.err),
                        bits(w.work_counter), bits(w.clear_counter), bits(w.merge_pacc), bits(w.merge_pml),
                        bits(w.merge_out), bits(w.n_merge), bits(w.n_pitems), bits(w.n_dreq), bits(w.max_split),
                        bits(w.n_ditems), bits(w.pages_per_split), bits(w.decode_cus), bits(w.prefill_id_cap),
                        bits(w.ppart), bits(w.psplit), bits(w.pcount), bits(w.prefill_piece_tiles),
                        bits(p.k_cache), bits(p.v_cache), bits(p.k_new), bits(p.v_new), bits(p.page_table),
                        bits(p.num_phys_pages), bits(p.max_pages), bits(p.h_kv), bits(p.head_dim), bits(p.dtype)};
  k->insert(k->end(), std::begin(f), std::end(f));
}

// Word-wise multiply-xor hash (a lookup index only: a hit is confirmed by comparing the keys).
uint64_t hash_key(const std::vector<uint64_t>& k) {
  uint64_t h = 0x9e3779b97f4a7c15ull ^ k.size();
  for (uint64_t x : k) {
    h ^= x + 0x9e3779b97f4a7c15ull + (h << 6) + (h >> 2);
    h *= 0xff51afd7ed558ccdull;
  }
  return h ^ (h >> 33);
}

struct GraphEntry {
  std::vector<uint64_t> key;
  hipGraphExec_t exec = nullptr;
  uint64_t last_use = 0;
};

}  // namespace

struct duet_ctx {
  int device = 0;
  int num_cus = 0;
  duet_model model;
  std::mutex mu;
  std::map<std::pair<int, int>, hipStream_t> streams;  // (cus, high_end) -> masked stream
  std::map<std::pair<int, int>, uint64_t> last_use;    // for evicting the least recently used
  uint64_t use_clock = 0;
  hipEvent_t ev_fork = nullptr, ev_djoin = nullptr, ev_pjoin = nullptr;
  hipEvent_t prof[kNumProfEv] = {};
  int profiling = 0;  // 0 off, 1 iteration events only, 2 also per-kernel events
  bool prof_valid = false;
  bool prof_decode = false, prof_prefill = false, prof_kernels = false;
  bool prof_deferred = false;  // only the last layer of the profiled call launched a reduce kernel
  int prof_layers = 0;
  // Per-layer kernel brackets of a profiled call: decode layer l uses events 3l (before the
  // partial kernel), 3l+1 (between partial and reduce) and 3l+2 (after the reduce); prefill
  // layer l uses 2l (before) and 2l+1 (after).
  std::vector<hipEvent_t> ev_dec, ev_pre;
  StagingSlot slots[kStagingSlots];
  int next_slot = 0;
  int32_t* dev_flag = nullptr;  // gather error word
  unsigned* dev_sink = nullptr;  // probe sink
  Plan plan;                     // reused host vectors
  // Look-ahead decode: each step's kernels are captured once into a graph (on a private
  // capture stream) and replayed on the decode stream while its launch arguments recur.
  bool decode_graphs = true;
  hipStream_t capture = nullptr;
  std::unordered_map<uint64_t, GraphEntry> graphs;
  uint64_t graph_clock = 0;
  uint64_t graphs_captured = 0, graphs_replayed = 0;
  std::vector<hipEvent_t> ev_step;  // decode stream: before step 0, after each step
  int prof_steps = 0;               // decode steps of the last profiled call (0: not look-ahead)
  duet::GemmCache* gemm = nullptr;  // hipBLASLt handle and planned GEMMs of the block forward
  void* scratch_dev = nullptr;      // this device's copy of `scratch` (no-allocation path)
};

namespace {

int get_stream(duet_ctx* ctx, int cus, int high_end, hipStream_t* out) {
  if (cus < DUET_CU_STEP || cus > ctx->num_cus || cus % DUET_CU_STEP)
    return fail(DUET_EINVAL, "CU count %d must be a multiple of %d in [%d, %d]", cus, DUET_CU_STEP, DUET_CU_STEP,
                ctx->num_cus);
  const auto key = std::make_pair(cus, cus == ctx->num_cus ? 0 : high_end);
  auto it = ctx->streams.find(key);
  if (it != ctx->streams.end()) {
    ctx->last_use[key] = ++ctx->use_clock;
    *out = it->second;
    return DUET_OK;
  }
  if (ctx->streams.size() >= kMaxMaskedStreams) {
    auto victim = ctx->last_use.begin();
    for (auto u = ctx->last_use.begin(); u != ctx->last_use.end(); ++u)
      if (u->second < victim->second) victim = u;
    hipStream_t vs = ctx->streams[victim->first];
    HIP_TRY(hipStreamSynchronize(vs));
    HIP_TRY(hipStreamDestroy(vs));
    ctx->streams.erase(victim->first);
    ctx->last_use.erase(victim);
  }
  std::vector<uint32_t> mask((ctx->num_cus + 31) / 32, 0u);
  for (int i = 0; i < cus; ++i) {
    const int bit = key.second ? ctx->num_cus - 1 - i : i;
    mask[bit / 32] |= 1u << (bit % 32);
  }
  hipStream_t st = nullptr;
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(hipExtStreamCreateWithCUMask(&st, (uint32_t)mask.size(), mask.data()));
  ctx->streams[key] = st;
  ctx->last_use[key] = ++ctx->use_clock;
  *out = st;
  return DUET_OK;
}

int ensure_layer_events(duet_ctx* ctx, int layers) {
  while (ctx->ev_dec.size() < (size_t)(3 * layers)) {
    hipEvent_t e = nullptr;
    HIP_TRY(hipEventCreate(&e));
    ctx->ev_dec.push_back(e);
  }
  while (ctx->ev_pre.size() < (size_t)(2 * layers)) {
    hipEvent_t e = nullptr;
    HIP_TRY(hipEventCreate(&e));
    ctx->ev_pre.push_back(e);
  }
  return DUET_OK;
}

int stage_upload(duet_ctx* ctx, const Plan& p, char* ws, hipStream_t st, bool may_allocate = true) {
  StagingSlot& slot = ctx->slots[ctx->next_slot];
  if (!may_allocate && slot.cap < p.upload_bytes)
    return fail(DUET_EWORKSPACE, "work lists of %zu bytes exceed the %zu bytes of preallocated staging", p.upload_bytes,
                slot.cap);
  ctx->next_slot = (ctx->next_slot + 1) % kStagingSlots;
  if (slot.pending) {
    HIP_TRY(hipEventSynchronize(slot.done));
    slot.pending = false;
  }
  if (slot.cap < p.upload_bytes) {
    if (slot.host) HIP_TRY(hipHostFree(slot.host));
    slot.host = nullptr;
    slot.cap = 0;
    const size_t cap = std::max<size_t>(p.upload_bytes * 2, 1 << 16);
    if (hipHostMalloc(&slot.host, cap, hipHostMallocDefault) != hipSuccess)
      return fail(DUET_ENOMEM, "pinned staging allocation of %zu bytes failed", cap);
    slot.cap = cap;
  }
  char* h = static_cast<char*>(slot.host);
  std::memset(h, 0, p.off_meta);  // clears the error word and the decode work counters
  std::memcpy(h + p.off_meta, p.meta.data(), p.meta.size() * sizeof(int4));
  std::memcpy(h + p.off_pitems, p.pitems.data(), p.pitems.size() * sizeof(int4));
  std::memcpy(h + p.off_dreq, p.dreq.data(), p.dreq.size() * sizeof(int4));
  std::memcpy(h + p.off_ditems, p.ditems.data(), p.ditems.size() * sizeof(int4));
  std::memcpy(h + p.off_psplit, p.psplit.data(), p.psplit.size() * sizeof(int2));
  std::memset(h + p.off_pcount, 0, (size_t)p.n_split_units * sizeof(int32_t));
  for (const StepPlan& sp : p.ahead) {
    std::memcpy(h + sp.off_meta, sp.meta.data(), sp.meta.size() * sizeof(int4));
    std::memcpy(h + sp.off_dreq, sp.dreq.data(), sp.dreq.size() * sizeof(int4));
    std::memcpy(h + sp.off_ditems, sp.ditems.data(), sp.ditems.size() * sizeof(int4));
  }
  HIP_TRY(hipMemcpyAsync(ws, h, p.upload_bytes, hipMemcpyHostToDevice, st));
  HIP_TRY(hipEventRecord(slot.done, st));
  slot.pending = true;
  return DUET_OK;
}

int check_device_ptr(const void* p, const char* name) {
  if (!p) return fail(DUET_EINVAL, "%s is NULL", name);
  return DUET_OK;
}

// One call over `layers` layers that share the batch, its page table and its work lists.  Each
// half runs its kernels for every layer back to back on its own stream; one fork and one join
// per call.
// Host-side checks of an attention call, before anything is enqueued.  Decode requests must
// have pages for `extra` tokens past their stated length (look-ahead slots).
int check_call(duet_ctx* ctx, const duet_shape* shape, int layers, const void* const* q_l, const void* const* k_l,
               const void* const* v_l, int64_t num_phys_pages, const int32_t* page_table, int32_t max_pages_per_req,
               const duet_batch* batch, duet_cu_split split, const void* workspace, const void* const* out_l,
               int extra) {
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, true))) return rc;
  if (layers < 1 || layers > kMaxLayers) return fail(DUET_EINVAL, "num_layers %d not in [1, %d]", layers, kMaxLayers);
  if ((rc = check_device_ptr(page_table, "page_table")) || (rc = check_device_ptr(workspace, "workspace")))
    return rc;
  for (int l = 0; l < layers; ++l) {
    if ((rc = check_device_ptr(q_l[l], "q")) || (rc = check_device_ptr(k_l[l], "k_cache")) ||
        (rc = check_device_ptr(v_l[l], "v_cache")) || (rc = check_device_ptr(out_l[l], "out")))
      return rc;
    if (out_l[l] == q_l[l] || out_l[l] == k_l[l] || out_l[l] == v_l[l])
      return fail(DUET_EINVAL, "layer %d: out aliases an input", l);
  }
  if (num_phys_pages < 1 || num_phys_pages > (int64_t)INT32_MAX)
    return fail(DUET_EINVAL, "num_phys_pages %lld out of range", (long long)num_phys_pages);
  for (int r = 0; r < batch->num_reqs; ++r) {
    const duet_seq_meta& q = batch->reqs[r];
    const int64_t L = (int64_t)q.cached_len + q.q_len + (q.kind == DUET_KIND_DECODE ? extra : 0);
    if ((L + 15) / 16 > max_pages_per_req)
      return fail(DUET_EINVAL, "request %d needs %lld pages, page_table rows hold %d", r, (long long)((L + 15) / 16),
                  max_pages_per_req);
  }
  {
    int n_dec = 0;
    for (int r = 0; r < batch->num_reqs; ++r) {
      const duet_seq_meta& q = batch->reqs[r];
      const int64_t L = (int64_t)q.cached_len + q.q_len + (q.kind == DUET_KIND_DECODE ? extra : 0);
      if (q.kind == DUET_KIND_DECODE) ++n_dec;
      if (q.kind == DUET_KIND_PREFILL && L > kMaxPrefillKeys)
        return fail(DUET_EUNSUPPORTED, "request %d: prefill attends %lld keys, at most %d supported", r,
                    (long long)L, kMaxPrefillKeys);
      if (q.kind == DUET_KIND_DECODE && (L + 15) / 16 > kMaxDecodePages)
        return fail(DUET_EUNSUPPORTED, "request %d: decode context %lld too long", r, (long long)L);
    }
    if (n_dec > 65535) return fail(DUET_EUNSUPPORTED, "more than 65535 decode requests");
    if (batch->num_reqs >= (1 << 24)) return fail(DUET_EUNSUPPORTED, "more than %d requests", (1 << 24) - 1);
    if (shape->num_kv_heads > 63) return fail(DUET_EUNSUPPORTED, "more than 63 kv heads");
  }
  if (split.mode == DUET_SPLIT) {
    if (split.cus_prefill < DUET_CU_STEP || split.cus_decode < DUET_CU_STEP || split.cus_prefill % DUET_CU_STEP ||
        split.cus_decode % DUET_CU_STEP || split.cus_prefill + split.cus_decode > ctx->num_cus)
      return fail(DUET_EINVAL, "split %d/%d: CU shares must be multiples of %d summing to at most %d",
                  split.cus_prefill, split.cus_decode, DUET_CU_STEP, ctx->num_cus);
  } else if (split.mode != DUET_AGG && split.mode != DUET_CONCURRENT) {
    return fail(DUET_EINVAL, "split mode %d", split.mode);
  }

  return DUET_OK;
}

// Arguments common to every kernel of a call (step 0's work lists; no per-layer pointers).
void base_args(const duet_ctx* ctx, const duet_shape* shape, const Plan& p, char* ws, duet_cu_split split,
               const int32_t* page_table, int64_t num_phys_pages, int32_t max_pages_per_req, AttnArgs* a,
               WorkArgs* w) {
  *a = AttnArgs{};
  a->page_table = page_table;
  a->num_phys_pages = num_phys_pages;
  a->max_pages = max_pages_per_req;
  a->h_q = shape->num_q_heads;
  a->h_kv = shape->num_kv_heads;
  a->group = p.group;
  a->head_dim = shape->head_dim;
  a->dtype = shape->dtype;
  a->scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)shape->head_dim));
  *w = WorkArgs{};
  w->meta = reinterpret_cast<const int4*>(ws + p.off_meta);
  w->pitems = reinterpret_cast<const int4*>(ws + p.off_pitems);
  w->dreq = reinterpret_cast<const int4*>(ws + p.off_dreq);
  w->pacc = reinterpret_cast<float*>(ws + p.off_pacc[0]);
  w->pml = reinterpret_cast<float*>(ws + p.off_pml[0]);
  w->ditems = reinterpret_cast<const int4*>(ws + p.off_ditems);
  w->err = reinterpret_cast<int32_t*>(ws);
  w->work_counter = reinterpret_cast<int32_t*>(ws + kCounterOffset);
  w->n_ditems = (int)p.ditems.size();
  w->decode_cus = split.mode == DUET_SPLIT ? split.cus_decode : ctx->num_cus;
  w->n_pitems = (int)p.pitems.size();
  w->n_dreq = (int)p.dreq.size();
  w->max_split = p.max_split;
  w->pages_per_split = p.pages_per_split;
  w->prefill_id_cap = p.prefill_id_cap;
  w->ppart = reinterpret_cast<float*>(ws + p.off_ppart);
  w->psplit = reinterpret_cast<const int2*>(ws + p.off_psplit);
  w->pcount = reinterpret_cast<int32_t*>(ws + p.off_pcount);
  w->prefill_piece_tiles = p.prefill_piece_tiles;
}

// A masked stream the context already holds (no creation): the no-allocation path's lookup.
int find_stream(duet_ctx* ctx, int cus, int high_end, hipStream_t* out) {
  const auto key = std::make_pair(cus, cus == ctx->num_cus ? 0 : high_end);
  auto it = ctx->streams.find(key);
  if (it == ctx->streams.end())
    return fail(DUET_EINVAL, "no CU-masked stream for %d CUs (%s end) yet: the no-allocation path creates none; run "
                "one allocating call with this split first", cus, key.second ? "high" : "low");
  ctx->last_use[key] = ++ctx->use_clock;
  *out = it->second;
  return DUET_OK;
}

// no_alloc: the workspace is the context's scratch, streams must exist, staging never grows and
// no profiling events are created (profiling is ignored).
int attn_layers(duet_ctx* ctx, const duet_shape* shape, int layers, const void* const* q_l,
                const void* const* k_l, const void* const* v_l, int64_t num_phys_pages, const int32_t* page_table,
                int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                size_t workspace_bytes, void* const* out_l, void* stream, bool no_alloc = false) {
  int rc = check_call(ctx, shape, layers, q_l, k_l, v_l, num_phys_pages, page_table, max_pages_per_req, batch, split,
                      workspace, out_l, 0);
  if (rc) return rc;

  std::lock_guard<std::mutex> lock(ctx->mu);
  Plan& p = ctx->plan;
  plan_batch(shape, batch, layers, 1, &p, true);
  if (split.mode == DUET_SPLIT) snake_prefill_rounds(&p.pitems);
  if (workspace_bytes < p.total)
    return fail(DUET_EWORKSPACE, "%s %zu bytes, need %zu", no_alloc ? "scratch holds" : "workspace", workspace_bytes,
                p.total);

  hipStream_t order = static_cast<hipStream_t>(stream);
  hipStream_t sd = order, sp = order;
  HIP_TRY(hipSetDevice(ctx->device));
  auto stream_for = [&](int cus, int high_end, hipStream_t* out) {
    return no_alloc ? find_stream(ctx, cus, high_end, out) : get_stream(ctx, cus, high_end, out);
  };
  if (split.mode == DUET_SPLIT) {
    if ((rc = stream_for(split.cus_decode, 0, &sd))) return rc;
    if ((rc = stream_for(split.cus_prefill, 1, &sp))) return rc;
  } else if (split.mode == DUET_CONCURRENT) {
    // two streams whose masks both cover every CU
    if ((rc = stream_for(ctx->num_cus, 0, &sd))) return rc;
    if ((rc = stream_for(ctx->num_cus, 1, &sp))) return rc;
  }
  const bool forked = split.mode != DUET_AGG;

  char* ws = static_cast<char*>(workspace);
  AttnArgs a;
  WorkArgs w;
  base_args(ctx, shape, p, ws, split, page_table, num_phys_pages, max_pages_per_req, &a, &w);
  const bool prof_iter = ctx->profiling >= 1 && !no_alloc;
  const bool prof = ctx->profiling >= 2 && !no_alloc;
  const bool has_decode = w.n_dreq > 0, has_prefill = w.n_pitems > 0;

  if (prof_iter) HIP_TRY(hipEventRecord(ctx->prof[kEvFork], order));
  if ((rc = stage_upload(ctx, p, ws, order, !no_alloc))) return rc;
  auto layer_args = [&](int l) {
    AttnArgs al = a;
    al.q = q_l[l];
    al.k_cache = k_l[l];
    al.v_cache = v_l[l];
    al.out = out_l[l];
    return al;
  };
  if (prof && (rc = ensure_layer_events(ctx, layers))) return rc;
  // Aggregated execution runs each layer's decode kernels, then its prefill kernel, on the
  // caller's stream.  Spatial sharing forks both CU-masked streams off the caller's stream and
  // enqueues the two halves layer by layer, alternating, so neither half waits for the host to
  // finish enqueueing the other.
  if (forked) {
    HIP_TRY(hipEventRecord(ctx->ev_fork, order));
    if (has_decode) HIP_TRY(hipStreamWaitEvent(sd, ctx->ev_fork, 0));
    if (has_prefill) HIP_TRY(hipStreamWaitEvent(sp, ctx->ev_fork, 0));
  }
  // bf16 decode defers each layer's split merge into the next layer's partial kernel, whose waves
  // merge once their item queue is empty; partial buffers and counter sets alternate by layer,
  // and one reduce kernel merges the last layer.  The fp32 path merges every layer in its own
  // reduce kernel.
  const bool defer = has_decode && shape->dtype == DUET_BF16;
  for (int l = 0; l < layers; ++l) {
    const AttnArgs al = layer_args(l);
    if (has_decode) {
      WorkArgs wl = w;
      if (defer) {
        const int cur = l & 1, prev = cur ^ 1;
        wl.pacc = reinterpret_cast<float*>(ws + p.off_pacc[cur]);
        wl.pml = reinterpret_cast<float*>(ws + p.off_pml[cur]);
        wl.work_counter = w.work_counter + cur * kDecodeSetInts;
        wl.clear_counter = w.work_counter + prev * kDecodeSetInts;
        if (l > 0) {
          wl.merge_pacc = reinterpret_cast<const float*>(ws + p.off_pacc[prev]);
          wl.merge_pml = reinterpret_cast<const float*>(ws + p.off_pml[prev]);
          wl.merge_out = out_l[l - 1];
          wl.n_merge = w.n_dreq * a.h_q;
        }
      }
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_dec[3 * l], sd));
      HIP_TRY(launch_decode_partial(al, wl, sd));
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_dec[3 * l + 1], sd));
      if (!defer || l == layers - 1) {
        HIP_TRY(launch_decode_reduce(al, wl, sd));
        if (prof) HIP_TRY(hipEventRecord(ctx->ev_dec[3 * l + 2], sd));
      }
    }
    if (has_prefill) {
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_pre[2 * l], sp));
      HIP_TRY(launch_prefill(al, w, sp));
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_pre[2 * l + 1], sp));
    }
  }
  if (forked) {
    HIP_TRY(hipEventRecord(ctx->ev_djoin, sd));
    HIP_TRY(hipEventRecord(ctx->ev_pjoin, sp));
    HIP_TRY(hipStreamWaitEvent(order, ctx->ev_djoin, 0));
    HIP_TRY(hipStreamWaitEvent(order, ctx->ev_pjoin, 0));
  }
  if (prof_iter) HIP_TRY(hipEventRecord(ctx->prof[kEvJoin], order));
  if (no_alloc) return DUET_OK;  // the last profiled call's events stay valid
  ctx->prof_valid = prof_iter;
  ctx->prof_kernels = prof;
  ctx->prof_deferred = defer;
  ctx->prof_decode = has_decode;
  ctx->prof_prefill = has_prefill;
  ctx->prof_layers = layers;
  ctx->prof_steps = 0;
  return DUET_OK;
}

int ensure_step_events(duet_ctx* ctx, int steps) {
  while (ctx->ev_step.size() < (size_t)(steps + 1)) {
    hipEvent_t e = nullptr;
    HIP_TRY(hipEventCreate(&e));
    ctx->ev_step.push_back(e);
  }
  return DUET_OK;
}

void clear_graphs(duet_ctx* ctx) {
  for (auto& kv : ctx->graphs) (void)hipGraphExecDestroy(kv.second.exec);
  ctx->graphs.clear();
}

// Enqueues a run of decode launches on `st`: from its cached graph when one with the same launch
// arguments exists, else captured now (on the private capture stream, so `st` keeps its
// pending work and its CU mask governs the replay), or launched directly when graphs are off.
int run_decode_step(duet_ctx* ctx, const std::vector<DecodeLaunch>& launches, hipStream_t st) {
  if (!ctx->decode_graphs) {
    for (const DecodeLaunch& l : launches) HIP_TRY(run_launch(l, st));
    return DUET_OK;
  }
  std::vector<uint64_t> key;
  key.reserve(launches.size() * 40);
  for (const DecodeLaunch& l : launches) append_key(&key, l);
  const uint64_t h = hash_key(key);
  auto it = ctx->graphs.find(h);
  if (it == ctx->graphs.end() || it->second.key != key) {
    if (!ctx->capture) HIP_TRY(hipStreamCreateWithFlags(&ctx->capture, hipStreamNonBlocking));
    HIP_TRY(hipStreamBeginCapture(ctx->capture, hipStreamCaptureModeThreadLocal));
    hipError_t e = hipSuccess;
    for (const DecodeLaunch& l : launches)
      if ((e = run_launch(l, ctx->capture)) != hipSuccess) break;
    hipGraph_t g = nullptr;
    const hipError_t e_end = hipStreamEndCapture(ctx->capture, &g);
    if (e != hipSuccess || e_end != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return fail(DUET_EHIP, "capturing a decode step: %s",
                  hipGetErrorString(e != hipSuccess ? e : e_end));
    }
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) return fail(DUET_EHIP, "instantiating a decode step graph: %s", hipGetErrorString(e));
    if (it != ctx->graphs.end() || ctx->graphs.size() >= kMaxGraphs) {
      // A replaced or evicted graph may still be running: wait for the device first.
      HIP_TRY(hipDeviceSynchronize());
      auto victim = it;
      if (victim == ctx->graphs.end()) {  // evict the least recently used graph
        victim = ctx->graphs.begin();
        for (auto u = ctx->graphs.begin(); u != ctx->graphs.end(); ++u)
          if (u->second.last_use < victim->second.last_use) victim = u;
      }
      (void)hipGraphExecDestroy(victim->second.exec);
      ctx->graphs.erase(victim);
    }
    GraphEntry& g_new = ctx->graphs[h];
    g_new.key = std::move(key);
    g_new.exec = ex;
    it = ctx->graphs.find(h);
    ++ctx->graphs_captured;
  } else {
    ++ctx->graphs_replayed;
  }
  it->second.last_use = ++ctx->graph_clock;
  HIP_TRY(hipGraphLaunch(it->second.exec, st));
  return DUET_OK;
}

// Look-ahead decode (Section 4.3): the prefill half once over all layers and the decode half for
// k = split.k_decode_steps steps, step s >= 1 writing its token before attending.  SPLIT and
// CONCURRENT enqueue the first prefill layer, every decode step (one graph) on the decode stream,
// then the other prefill layers; AGG runs decode step 0, the prefill layers and decode steps
// 1 .. k - 1 in that order on the caller's stream.
int attn_lookahead(duet_ctx* ctx, const duet_shape* shape, const void* const* q_l, const void* const* q_ahead,
                   const void* const* k_ahead, const void* const* v_ahead, void* const* kc_l, void* const* vc_l,
                   int64_t num_phys_pages, const int32_t* page_table, int32_t max_pages_per_req,
                   const duet_batch* batch, duet_cu_split split, void* workspace, size_t workspace_bytes,
                   void* const* out_l, void* const* out_ahead, void* stream) {
  if (!shape) return fail(DUET_EINVAL, "shape is NULL");
  if (!q_l || !kc_l || !vc_l || !out_l) return fail(DUET_EINVAL, "per-layer pointer array is NULL");
  const int layers = shape->num_layers;
  const int k = split.k_decode_steps;
  if (k < 1 || k > kMaxLookahead) return fail(DUET_EINVAL, "k_decode_steps %d not in [1, %d]", k, kMaxLookahead);
  if (layers < 1 || layers > kMaxLayers) return fail(DUET_EINVAL, "num_layers %d not in [1, %d]", layers, kMaxLayers);
  const std::vector<const void*> kcc(kc_l, kc_l + layers), vcc(vc_l, vc_l + layers);
  int rc = check_call(ctx, shape, layers, q_l, kcc.data(), vcc.data(), num_phys_pages, page_table, max_pages_per_req,
                      batch, split, workspace, out_l, k - 1);
  if (rc) return rc;
  if ((int64_t)layers * k > 16384) return fail(DUET_EINVAL, "num_layers x k_decode_steps above 16384");
  int n_dec = 0;
  for (int r = 0; r < batch->num_reqs; ++r) n_dec += batch->reqs[r].kind == DUET_KIND_DECODE;
  if (k > 1 && n_dec > 0) {
    if (!q_ahead || !k_ahead || !v_ahead || !out_ahead)
      return fail(DUET_EINVAL, "look-ahead pointer array is NULL");
    for (int x = 0; x < (k - 1) * layers; ++x) {
      if ((rc = check_device_ptr(q_ahead[x], "q_ahead")) || (rc = check_device_ptr(k_ahead[x], "k_ahead")) ||
          (rc = check_device_ptr(v_ahead[x], "v_ahead")) || (rc = check_device_ptr(out_ahead[x], "out_ahead")))
        return rc;
      const int l = x % layers;
      if (out_ahead[x] == q_ahead[x] || out_ahead[x] == k_ahead[x] || out_ahead[x] == v_ahead[x] ||
          out_ahead[x] == kc_l[l] || out_ahead[x] == vc_l[l])
        return fail(DUET_EINVAL, "look-ahead output %d aliases an input", x);
    }
  }

  std::lock_guard<std::mutex> lock(ctx->mu);
  Plan& p = ctx->plan;
  plan_batch(shape, batch, layers, k, &p, true);
  if (split.mode == DUET_SPLIT) snake_prefill_rounds(&p.pitems);
  if (workspace_bytes < p.total)
    return fail(DUET_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, p.total);

  hipStream_t order = static_cast<hipStream_t>(stream);
  hipStream_t sd = order, sp = order;
  HIP_TRY(hipSetDevice(ctx->device));
  if (split.mode == DUET_SPLIT) {
    if ((rc = get_stream(ctx, split.cus_decode, 0, &sd))) return rc;
    if ((rc = get_stream(ctx, split.cus_prefill, 1, &sp))) return rc;
  } else if (split.mode == DUET_CONCURRENT) {
    if ((rc = get_stream(ctx, ctx->num_cus, 0, &sd))) return rc;
    if ((rc = get_stream(ctx, ctx->num_cus, 1, &sp))) return rc;
  }
  const bool forked = split.mode != DUET_AGG;
  char* ws = static_cast<char*>(workspace);
  AttnArgs a;
  WorkArgs w;
  base_args(ctx, shape, p, ws, split, page_table, num_phys_pages, max_pages_per_req, &a, &w);
  const bool prof_iter = ctx->profiling >= 1;
  const bool prof = ctx->profiling >= 2;
  const bool has_decode = n_dec > 0, has_prefill = w.n_pitems > 0;
  if (prof_iter && ((rc = ensure_step_events(ctx, k)) || (rc = ensure_layer_events(ctx, layers)))) return rc;

  if (prof_iter) HIP_TRY(hipEventRecord(ctx->prof[kEvFork], order));
  if ((rc = stage_upload(ctx, p, ws, order))) return rc;
  if (forked) {
    HIP_TRY(hipEventRecord(ctx->ev_fork, order));
    if (has_decode) HIP_TRY(hipStreamWaitEvent(sd, ctx->ev_fork, 0));
    if (has_prefill) HIP_TRY(hipStreamWaitEvent(sp, ctx->ev_fork, 0));
  }
  std::vector<DecodeLaunch> launches;
  // Appends decode step st's launches (every layer) to `launches`.
  auto add_step = [&](int st) {
    WorkArgs ws_w = w;
    if (st > 0) {
      const StepPlan& spl = p.ahead[st - 1];
      ws_w.meta = reinterpret_cast<const int4*>(ws + spl.off_meta);
      ws_w.dreq = reinterpret_cast<const int4*>(ws + spl.off_dreq);
      ws_w.ditems = reinterpret_cast<const int4*>(ws + spl.off_ditems);
      ws_w.n_dreq = (int)spl.dreq.size();
      ws_w.n_ditems = (int)spl.ditems.size();
      ws_w.max_split = spl.max_split;
    }
    for (int l = 0; l < layers; ++l) {
      const int x = (st - 1) * layers + l;
      DecodeLaunch dl;
      dl.a = a;
      dl.a.q = st == 0 ? q_l[l] : q_ahead[x];
      dl.a.k_cache = kc_l[l];
      dl.a.v_cache = vc_l[l];
      dl.a.out = st == 0 ? out_l[l] : out_ahead[x];
      dl.w = ws_w;
      dl.ap = AppendArgs{};
      if (st > 0) {
        dl.ap.k_cache = kc_l[l];
        dl.ap.v_cache = vc_l[l];
        dl.ap.k_new = k_ahead[x];
        dl.ap.v_new = v_ahead[x];
        dl.ap.page_table = page_table;
        dl.ap.num_phys_pages = num_phys_pages;
        dl.ap.max_pages = max_pages_per_req;
        dl.ap.h_kv = shape->num_kv_heads;
        dl.ap.head_dim = shape->head_dim;
        dl.ap.dtype = shape->dtype;
        dl.kind = DecodeLaunch::kAppend;
        launches.push_back(dl);
      }
      dl.kind = DecodeLaunch::kPartial;
      launches.push_back(dl);
      dl.kind = DecodeLaunch::kReduce;
      launches.push_back(dl);
    }
  };
  // Enqueues decode steps first .. last - 1 on the decode stream as one graph (one launch for the
  // whole run of steps).  Profiled, step 0 is a graph of its own, so that an event marks when its
  // tokens are ready; the other steps still run as one graph, as they do unprofiled (one graph per
  // step would add the launch gaps between graphs to every step it measures).
  auto decode_steps = [&](int first, int last) -> int {
    hipStream_t ds = forked ? sd : order;
    for (int st = first; st < last;) {
      const int end = prof_iter && st == 0 ? 1 : last;
      launches.clear();
      for (int x = st; x < end; ++x) add_step(x);
      int r2 = run_decode_step(ctx, launches, ds);
      if (r2) return r2;
      if (prof_iter) HIP_TRY(hipEventRecord(ctx->ev_step[end], ds));
      st = end;
    }
    return DUET_OK;
  };
  auto prefill_layers = [&](int l0, int l1) -> int {
    for (int l = l0; l < l1; ++l) {
      AttnArgs al = a;
      al.q = q_l[l];
      al.k_cache = kc_l[l];
      al.v_cache = vc_l[l];
      al.out = out_l[l];
      if (prof_iter && (prof || l == 0)) HIP_TRY(hipEventRecord(ctx->ev_pre[2 * l], sp));
      HIP_TRY(launch_prefill(al, w, sp));
      if (prof_iter && (prof || l == layers - 1)) HIP_TRY(hipEventRecord(ctx->ev_pre[2 * l + 1], sp));
    }
    return DUET_OK;
  };
  if (has_decode && prof_iter) HIP_TRY(hipEventRecord(ctx->ev_step[0], forked ? sd : order));
  if (forked) {
    // The first prefill layer is enqueued, then every decode step, then the other prefill layers:
    // the prefill stream starts at once (enqueueing the k steps first would hold it back by their
    // host-side launch time, up to a millisecond with one graph per step), and the decode
    // partition waits for one kernel launch only.
    if (has_prefill && (rc = prefill_layers(0, 1))) return rc;
    if (has_decode && (rc = decode_steps(0, k))) return rc;
    if (has_prefill && (rc = prefill_layers(1, layers))) return rc;
  } else {
    if (has_decode && (rc = decode_steps(0, 1))) return rc;
    if (has_prefill && (rc = prefill_layers(0, layers))) return rc;
    if (has_decode && k > 1 && (rc = decode_steps(1, k))) return rc;
  }
  if (forked) {
    HIP_TRY(hipEventRecord(ctx->ev_djoin, sd));
    HIP_TRY(hipEventRecord(ctx->ev_pjoin, sp));
    HIP_TRY(hipStreamWaitEvent(order, ctx->ev_djoin, 0));
    HIP_TRY(hipStreamWaitEvent(order, ctx->ev_pjoin, 0));
  }
  if (prof_iter) HIP_TRY(hipEventRecord(ctx->prof[kEvJoin], order));
  ctx->prof_valid = prof_iter;
  ctx->prof_kernels = prof;
  ctx->prof_deferred = false;
  ctx->prof_decode = has_decode;
  ctx->prof_prefill = has_prefill;
  ctx->prof_layers = layers;
  ctx->prof_steps = k;
  return DUET_OK;
}

// ---- the whole block: token-level operators around the attention kernels --------------------

// Byte offsets of the block forward's buffers after the attention workspace.
struct BlockLayout {
  size_t h = 0, qkv = 0, q = 0, attn = 0, gu = 0, act = 0, gemm_ws[2] = {0, 0}, total = 0;
};

BlockLayout block_layout(const duet_shape* s, const duet_block_shape* blk, int64_t T, size_t attn_total) {
  const size_t d = (size_t)s->num_q_heads * s->head_dim;
  const size_t d_qkv = (size_t)(s->num_q_heads + 2 * s->num_kv_heads) * s->head_dim;
  const size_t m = (size_t)blk->ffn_dim, b = 2;
  BlockLayout L;
  size_t off = align_up(attn_total);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.h = take(T * d * b);
  L.qkv = take(T * d_qkv * b);
  L.q = take(T * d * b);
  L.attn = take(T * d * b);
  L.gu = take(T * 2 * m * b);
  L.act = take(T * m * b);
  L.gemm_ws[0] = take(kGemmWorkspaceBytes);
  L.gemm_ws[1] = take(kGemmWorkspaceBytes);
  L.total = off;
  return L;
}

int check_block_exec(const duet_shape* s, const duet_block_shape* blk) {
  if (!blk) return fail(DUET_EINVAL, "block is NULL");
  if (s->dtype != DUET_BF16) return fail(DUET_EUNSUPPORTED, "the block forward runs bf16 only");
  if (blk->flags != (DUET_BLOCK_GQA_QKV | DUET_BLOCK_FUSED_GATE_UP))
    return fail(DUET_EUNSUPPORTED, "the block forward needs flags DUET_BLOCK_GQA_QKV | DUET_BLOCK_FUSED_GATE_UP");
  if (blk->ffn_dim < 8 || blk->ffn_dim % 8) return fail(DUET_EINVAL, "ffn_dim %d must be a positive multiple of 8", blk->ffn_dim);
  if (blk->ffn_dim > (1 << 20)) return fail(DUET_EINVAL, "ffn_dim %d too large", blk->ffn_dim);
  return DUET_OK;
}

// Rows [row0, row0 + rows) of the requests of one kind, or rows = -1 when they are not one
// contiguous range (rows = 0: none of that kind).
void kind_rows(const duet_batch* b, int kind, int* row0, int* rows) {
  int64_t lo = INT64_MAX, hi = -1, n = 0;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& q = b->reqs[r];
    if (q.kind != kind) continue;
    lo = std::min<int64_t>(lo, q.q_start);
    hi = std::max<int64_t>(hi, (int64_t)q.q_start + q.q_len);
    n += q.q_len;
  }
  *row0 = n ? (int)lo : 0;
  *rows = n == 0 ? 0 : (hi - lo == n ? (int)n : -1);
}

int block_forward(duet_ctx* ctx, const duet_shape* shape, const duet_block_shape* blk, const duet_block_weights* wts,
                  float eps, void* x, void* const* x_ahead, void* const* k_l, void* const* v_l, int64_t num_phys_pages,
                  const int32_t* page_table, int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split,
                  void* workspace, size_t workspace_bytes, void* stream) {
  if (!shape) return fail(DUET_EINVAL, "shape is NULL");
  const int layers = shape->num_layers;
  if (layers < 1 || layers > kMaxLayers) return fail(DUET_EINVAL, "num_layers %d not in [1, %d]", layers, kMaxLayers);
  const int k = split.k_decode_steps;
  if (k < 1 || k > kMaxLookahead) return fail(DUET_EINVAL, "k_decode_steps %d not in [1, %d]", k, kMaxLookahead);
  if (!wts || !k_l || !v_l) return fail(DUET_EINVAL, "per-layer array is NULL");
  int rc = check_device_ptr(x, "x");
  if (rc) return rc;
  if (!(eps > 0.0f)) return fail(DUET_EINVAL, "norm_eps must be > 0");
  // Attention reads q from the block's own buffer and writes another one: check_call sees x as q
  // and the workspace as the output (checked non-null and distinct from the caches).
  std::vector<const void*> xs(layers, x), kc(k_l, k_l + layers), vc(v_l, v_l + layers);
  std::vector<void*> outs(layers, workspace);
  for (int l = 0; l < layers; ++l) {
    const duet_block_weights& w = wts[l];
    if ((rc = check_device_ptr(w.attn_norm, "attn_norm")) || (rc = check_device_ptr(w.w_qkv, "w_qkv")) ||
        (rc = check_device_ptr(w.w_o, "w_o")) || (rc = check_device_ptr(w.ffn_norm, "ffn_norm")) ||
        (rc = check_device_ptr(w.w_gate_up, "w_gate_up")) || (rc = check_device_ptr(w.w_down, "w_down")))
      return rc;
    if (x == k_l[l] || x == v_l[l]) return fail(DUET_EINVAL, "layer %d: x aliases a cache", l);
  }
  if ((rc = check_call(ctx, shape, layers, xs.data(), kc.data(), vc.data(), num_phys_pages, page_table,
                       max_pages_per_req, batch, split, workspace, outs.data(), k - 1)))
    return rc;
  if ((rc = check_block_exec(shape, blk))) return rc;
  int dec0 = 0, n_dec = 0, pre0 = 0, n_pre = 0;
  kind_rows(batch, DUET_KIND_DECODE, &dec0, &n_dec);
  kind_rows(batch, DUET_KIND_PREFILL, &pre0, &n_pre);
  if ((split.mode != DUET_AGG || k > 1) && (n_dec < 0 || n_pre < 0))
    return fail(DUET_EUNSUPPORTED,
                "a split or look-ahead block forward needs each kind's rows to be one contiguous range");
  const int steps = n_dec > 0 ? k : 1;  // decode steps of this call
  if (steps > 1) {
    if (!x_ahead) return fail(DUET_EINVAL, "x_ahead is NULL with k_decode_steps > 1");
    for (int s = 0; s < steps - 1; ++s) {
      if ((rc = check_device_ptr(x_ahead[s], "x_ahead"))) return rc;
      if (x_ahead[s] == x) return fail(DUET_EINVAL, "x_ahead[%d] aliases x", s);
    }
  }

  std::lock_guard<std::mutex> lock(ctx->mu);
  Plan& p = ctx->plan;
  plan_batch(shape, batch, 1, steps, &p, true);
  if (split.mode == DUET_SPLIT) snake_prefill_rounds(&p.pitems);

  int64_t T = 0;
  for (int r = 0; r < batch->num_reqs; ++r) T += batch->reqs[r].q_len;
  const BlockLayout B = block_layout(shape, blk, T, p.total);
  if (workspace_bytes < B.total)
    return fail(DUET_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, B.total);
  if (!ctx->gemm && !(ctx->gemm = gemm_cache_create())) return fail(DUET_EHIP, "hipBLASLt initialisation failed");

  hipStream_t order = static_cast<hipStream_t>(stream);
  hipStream_t sd = order, sp = order;
  HIP_TRY(hipSetDevice(ctx->device));
  if (split.mode == DUET_SPLIT) {
    if ((rc = get_stream(ctx, split.cus_decode, 0, &sd))) return rc;
    if ((rc = get_stream(ctx, split.cus_prefill, 1, &sp))) return rc;
  } else if (split.mode == DUET_CONCURRENT) {
    if ((rc = get_stream(ctx, ctx->num_cus, 0, &sd))) return rc;
    if ((rc = get_stream(ctx, ctx->num_cus, 1, &sp))) return rc;
  }
  const bool forked = split.mode != DUET_AGG;
  char* ws = static_cast<char*>(workspace);
  AttnArgs a;
  WorkArgs w;
  base_args(ctx, shape, p, ws, split, page_table, num_phys_pages, max_pages_per_req, &a, &w);
  // Profiling brackets the call (fork to join) and, under a split, each partition's work: the
  // decode partition step by step (its tokens of step s are ready at the end of step s), the
  // prefill partition as one span.
  const bool prof = ctx->profiling >= 1;
  if (prof && ((rc = ensure_step_events(ctx, steps)) || (rc = ensure_layer_events(ctx, 1)))) return rc;
  if (prof) HIP_TRY(hipEventRecord(ctx->prof[kEvFork], order));
  if ((rc = stage_upload(ctx, p, ws, order))) return rc;

  // One partition: a stream, its token rows (of x and of the activation buffers) and its
  // attention kernels.
  struct Part {
    hipStream_t st;
    int row0, rows;
    bool decode, prefill;
    void* gemm_ws;
  };
  std::vector<Part> parts;
  if (!forked) {
    parts.push_back({order, 0, (int)T, w.n_dreq > 0, w.n_pitems > 0, ws + B.gemm_ws[0]});
  } else {
    if (n_dec > 0) parts.push_back({sd, dec0, n_dec, true, false, ws + B.gemm_ws[0]});
    if (n_pre > 0) parts.push_back({sp, pre0, n_pre, false, true, ws + B.gemm_ws[1]});
    HIP_TRY(hipEventRecord(ctx->ev_fork, order));
    for (const Part& pt : parts) {
      HIP_TRY(hipStreamWaitEvent(pt.st, ctx->ev_fork, 0));
      if (prof) HIP_TRY(hipEventRecord(pt.decode ? ctx->ev_step[0] : ctx->ev_pre[0], pt.st));
    }
  }
  const int d = shape->num_q_heads * shape->head_dim;
  const int d_qkv = (shape->num_q_heads + 2 * shape->num_kv_heads) * shape->head_dim;
  const int m = blk->ffn_dim;
  __bf16* hb = reinterpret_cast<__bf16*>(ws + B.h);
  __bf16* qkvb = reinterpret_cast<__bf16*>(ws + B.qkv);
  __bf16* qb = reinterpret_cast<__bf16*>(ws + B.q);
  __bf16* ab = reinterpret_cast<__bf16*>(ws + B.attn);
  __bf16* gub = reinterpret_cast<__bf16*>(ws + B.gu);
  __bf16* actb = reinterpret_cast<__bf16*>(ws + B.act);
  const char* msg = nullptr;
  // One layer of one partition over its rows: xr is its first residual row; the activation
  // buffers use rows [pt.row0, pt.row0 + pt.rows).  Look-ahead steps (dreq != null) index their
  // decode requests from 0, so their q / attention rows are addressed from the partition's first
  // row; step 0 addresses every row absolutely (its requests' q_start).
  auto run_layer = [&](const Part& pt, int l, __bf16* xr, const WorkArgs& wl, const int4* step_dreq) -> int {
    const duet_block_weights& wt = wts[l];
    const size_t r0 = (size_t)pt.row0;
    __bf16* h = hb + r0 * d;
    __bf16* qkv = qkvb + r0 * d_qkv;
    __bf16* gu = gub + r0 * 2 * m;
    __bf16* act = actb + r0 * m;
    auto gemm = [&](const __bf16* in, const void* wm, __bf16* out, int d_in, int d_out, bool acc) {
      return gemm_bf16(ctx->gemm, in, wm, out, pt.rows, d_in, d_out, acc, pt.gemm_ws, pt.st, &msg);
    };
    AttnArgs al = a;
    al.q = step_dreq ? qb + r0 * d : qb;
    al.k_cache = k_l[l];
    al.v_cache = v_l[l];
    al.out = step_dreq ? ab + r0 * d : ab;
    HIP_TRY(launch_rmsnorm(xr, static_cast<const __bf16*>(wt.attn_norm), h, pt.rows, d, eps, pt.st));
    if (gemm(h, wt.w_qkv, qkv, d, d_qkv, false)) return fail(DUET_EHIP, "QKV projection: %s", msg);
    QkvSplitArgs qs;
    qs.qkv = step_dreq ? qkv : qkvb;
    qs.q = static_cast<__bf16*>(const_cast<void*>(al.q));
    qs.k_cache = static_cast<__bf16*>(k_l[l]);
    qs.v_cache = static_cast<__bf16*>(v_l[l]);
    qs.meta = wl.meta;
    qs.dreq = step_dreq;
    qs.page_table = page_table;
    qs.num_phys_pages = num_phys_pages;
    qs.err = w.err;
    qs.num_reqs = batch->num_reqs;
    qs.max_pages = max_pages_per_req;
    qs.h_q = shape->num_q_heads;
    qs.h_kv = shape->num_kv_heads;
    qs.head_dim = shape->head_dim;
    qs.row0 = step_dreq ? 0 : pt.row0;
    HIP_TRY(launch_qkv_split(qs, pt.rows, pt.st));
    if (pt.decode) {
      HIP_TRY(launch_decode_partial(al, wl, pt.st));
      HIP_TRY(launch_decode_reduce(al, wl, pt.st));
    }
    if (pt.prefill) HIP_TRY(launch_prefill(al, wl, pt.st));
    const __bf16* attn_rows = ab + r0 * d;
    if (gemm(attn_rows, wt.w_o, xr, d, d, true)) return fail(DUET_EHIP, "output projection: %s", msg);
    HIP_TRY(launch_rmsnorm(xr, static_cast<const __bf16*>(wt.ffn_norm), h, pt.rows, d, eps, pt.st));
    if (gemm(h, wt.w_gate_up, gu, d, 2 * m, false)) return fail(DUET_EHIP, "gate-up projection: %s", msg);
    HIP_TRY(launch_swiglu(gu, act, pt.rows, m, pt.st));
    if (gemm(act, wt.w_down, xr, m, d, true)) return fail(DUET_EHIP, "down projection: %s", msg);
    return DUET_OK;
  };
  __bf16* xb = static_cast<__bf16*>(x);
  for (int l = 0; l < layers; ++l)
    for (const Part& pt : parts)
      if ((rc = run_layer(pt, l, xb + (size_t)pt.row0 * d, w, nullptr))) return rc;
  // Look-ahead decode steps 1 .. steps - 1 (Section 4.3): the decode partition runs every layer
  // again for its requests' next tokens, whose residual rows the caller passed in x_ahead; step s
  // writes its tokens' keys and values at position cached_len + s before attending.
  const Part dpart = forked ? parts[0] : Part{order, dec0, n_dec, true, false, ws + B.gemm_ws[0]};
  if (prof && steps > 1 && forked) HIP_TRY(hipEventRecord(ctx->ev_step[1], dpart.st));
  for (int st = 1; st < steps; ++st) {
    const StepPlan& spl = p.ahead[st - 1];
    WorkArgs wl = w;
    wl.meta = reinterpret_cast<const int4*>(ws + spl.off_meta);
    wl.dreq = reinterpret_cast<const int4*>(ws + spl.off_dreq);
    wl.ditems = reinterpret_cast<const int4*>(ws + spl.off_ditems);
    wl.n_dreq = (int)spl.dreq.size();
    wl.n_ditems = (int)spl.ditems.size();
    wl.max_split = spl.max_split;
    for (int l = 0; l < layers; ++l)
      if ((rc = run_layer(dpart, l, static_cast<__bf16*>(x_ahead[st - 1]), wl, wl.dreq))) return rc;
    if (prof && forked) HIP_TRY(hipEventRecord(ctx->ev_step[st + 1], dpart.st));
  }
  bool dec_part = false, pre_part = false;
  if (forked) {
    hipEvent_t joins[2] = {ctx->ev_djoin, ctx->ev_pjoin};
    for (size_t i = 0; i < parts.size(); ++i) {
      if (prof && (!parts[i].decode || steps == 1))
        HIP_TRY(hipEventRecord(parts[i].decode ? ctx->ev_step[1] : ctx->ev_pre[1], parts[i].st));
      dec_part |= parts[i].decode;
      pre_part |= parts[i].prefill;
      HIP_TRY(hipEventRecord(joins[i], parts[i].st));
      HIP_TRY(hipStreamWaitEvent(order, joins[i], 0));
    }
  }
  if (prof) HIP_TRY(hipEventRecord(ctx->prof[kEvJoin], order));
  ctx->prof_valid = prof;
  ctx->prof_kernels = false;
  ctx->prof_deferred = false;
  ctx->prof_decode = dec_part;
  ctx->prof_prefill = pre_part;
  ctx->prof_layers = 1;
  ctx->prof_steps = steps;
  return DUET_OK;
}

}  // namespace

extern "C" {

int duet_init(int device, duet_ctx** out) {
  clear_error();
  if (!out) return fail(DUET_EINVAL, "out is NULL");
  *out = nullptr;
  int n = 0;
  HIP_TRY(hipGetDeviceCount(&n));
  if (device < 0 || device >= n) return fail(DUET_EINVAL, "device %d not in [0, %d)", device, n);
  hipDeviceProp_t prop;
  HIP_TRY(hipGetDeviceProperties(&prop, device));
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(DUET_EUNSUPPORTED, "device %d is %s, the kernels are built for gfx950", device, prop.gcnArchName);
  if (prop.multiProcessorCount != DUET_TOTAL_CUS)
    return fail(DUET_EUNSUPPORTED, "device has %d CUs; CU splits assume %d (single-partition mode)",
                prop.multiProcessorCount, DUET_TOTAL_CUS);
  duet_ctx* ctx = new (std::nothrow) duet_ctx;
  if (!ctx) return fail(DUET_ENOMEM, "context allocation failed");
  ctx->device = device;
  ctx->num_cus = prop.multiProcessorCount;
  model_init_nominal(&ctx->model);
  auto cleanup = [&](int rc) {
    duet_destroy(ctx);
    return rc;
  };
  if (hipSetDevice(device) != hipSuccess) return cleanup(fail(DUET_EHIP, "hipSetDevice failed"));
  const unsigned ev_flags = hipEventDisableTiming;
  if (hipEventCreateWithFlags(&ctx->ev_fork, ev_flags) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_djoin, ev_flags) != hipSuccess ||
      hipEventCreateWithFlags(&ctx->ev_pjoin, ev_flags) != hipSuccess)
    return cleanup(fail(DUET_EHIP, "event creation failed"));
  for (auto& e : ctx->prof)
    if (hipEventCreate(&e) != hipSuccess) return cleanup(fail(DUET_EHIP, "event creation failed"));
  for (auto& s : ctx->slots)
    if (hipEventCreateWithFlags(&s.done, hipEventDisableTiming) != hipSuccess)
      return cleanup(fail(DUET_EHIP, "event creation failed"));
  if (hipMalloc(&ctx->dev_flag, 256) != hipSuccess || hipMemset(ctx->dev_flag, 0, 256) != hipSuccess)
    return cleanup(fail(DUET_EHIP, "device flag allocation failed"));
  // This device's copy of the no-allocation scratch (the device is current).
  {
    const hipError_t e = hipGetSymbolAddress(&ctx->scratch_dev, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ctx->scratch_dev)
      return cleanup(fail(DUET_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e)));
  }
  for (auto& sl : ctx->slots) {
    if (hipHostMalloc(&sl.host, kStagingPrealloc, hipHostMallocDefault) != hipSuccess)
      return cleanup(fail(DUET_ENOMEM, "pinned staging allocation of %zu bytes failed", kStagingPrealloc));
    sl.cap = kStagingPrealloc;
  }
  ctx->dev_sink = reinterpret_cast<unsigned*>(ctx->dev_flag) + 16;
  *out = ctx;
  return DUET_OK;
}

int duet_init_with_model(int device, const char* model_path, duet_ctx** out) {
  if (!out) return fail(DUET_EINVAL, "out is NULL");
  *out = nullptr;
  if (!model_path) return fail(DUET_EINVAL, "model_path is NULL");
  duet_ctx* ctx = nullptr;
  int rc = duet_init(device, &ctx);
  if (rc) return rc;
  if ((rc = duet_model_load(&ctx->model, model_path))) {
    duet_destroy(ctx);
    return rc;
  }
  *out = ctx;
  return DUET_OK;
}

int duet_destroy(duet_ctx* ctx) {
  if (!ctx) return DUET_OK;
  (void)hipSetDevice(ctx->device);
  if (ctx->gemm) {
    (void)hipDeviceSynchronize();
    duet::gemm_cache_destroy(ctx->gemm);
    ctx->gemm = nullptr;
  }
  for (auto& kv : ctx->streams) {
    (void)hipStreamSynchronize(kv.second);
    (void)hipStreamDestroy(kv.second);
  }
  for (auto& s : ctx->slots) {
    if (s.done) {
      if (s.pending) (void)hipEventSynchronize(s.done);
      (void)hipEventDestroy(s.done);
    }
    if (s.host) (void)hipHostFree(s.host);
  }
  for (auto& e : ctx->prof)
    if (e) (void)hipEventDestroy(e);
  for (auto& e : ctx->ev_dec) (void)hipEventDestroy(e);
  for (auto& e : ctx->ev_pre) (void)hipEventDestroy(e);
  for (auto& e : ctx->ev_step) (void)hipEventDestroy(e);
  if (!ctx->graphs.empty()) (void)hipDeviceSynchronize();
  clear_graphs(ctx);
  if (ctx->capture) (void)hipStreamDestroy(ctx->capture);
  if (ctx->ev_fork) (void)hipEventDestroy(ctx->ev_fork);
  if (ctx->ev_djoin) (void)hipEventDestroy(ctx->ev_djoin);
  if (ctx->ev_pjoin) (void)hipEventDestroy(ctx->ev_pjoin);
  if (ctx->dev_flag) (void)hipFree(ctx->dev_flag);
  delete ctx;
  return DUET_OK;
}

duet_model* duet_ctx_model(duet_ctx* ctx) { return ctx ? &ctx->model : nullptr; }

int duet_workspace_bytes(const duet_shape* shape, const duet_batch* batch, size_t* bytes) {
  clear_error();
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if (!bytes) return fail(DUET_EINVAL, "bytes is NULL");
  Plan p;
  plan_batch(shape, batch, shape->num_layers, 1, &p, false);
  *bytes = p.total;
  return DUET_OK;
}

int duet_block_workspace_bytes(const duet_shape* shape, const duet_block_shape* block, const duet_batch* batch,
                               int32_t k_decode_steps, size_t* bytes) {
  clear_error();
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if ((rc = check_block_exec(shape, block))) return rc;
  if (!bytes) return fail(DUET_EINVAL, "bytes is NULL");
  if (k_decode_steps < 1 || k_decode_steps > kMaxLookahead)
    return fail(DUET_EINVAL, "k_decode_steps %d not in [1, %d]", k_decode_steps, kMaxLookahead);
  Plan p;
  plan_batch(shape, batch, 1, k_decode_steps, &p, false);
  int64_t T = 0;
  for (int r = 0; r < batch->num_reqs; ++r) T += batch->reqs[r].q_len;
  *bytes = block_layout(shape, block, T, p.total).total;
  return DUET_OK;
}

int duet_block_buffers(const duet_shape* shape, const duet_block_shape* block, const duet_batch* batch,
                       int32_t k_decode_steps, size_t* offsets) {
  clear_error();
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if ((rc = check_block_exec(shape, block))) return rc;
  if (!offsets) return fail(DUET_EINVAL, "offsets is NULL");
  if (k_decode_steps < 1 || k_decode_steps > kMaxLookahead)
    return fail(DUET_EINVAL, "k_decode_steps %d not in [1, %d]", k_decode_steps, kMaxLookahead);
  Plan p;
  plan_batch(shape, batch, 1, k_decode_steps, &p, false);
  int64_t T = 0;
  for (int r = 0; r < batch->num_reqs; ++r) T += batch->reqs[r].q_len;
  const BlockLayout B = block_layout(shape, block, T, p.total);
  const size_t v[6] = {B.h, B.qkv, B.q, B.attn, B.gu, B.act};
  for (int i = 0; i < 6; ++i) offsets[i] = v[i];
  return DUET_OK;
}

int duet_rmsnorm(duet_ctx* ctx, const void* x, const void* weight, void* y, int32_t rows, int32_t d, float eps,
                 void* stream) {
  clear_error();
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  int rc;
  if ((rc = check_device_ptr(x, "x")) || (rc = check_device_ptr(weight, "weight")) || (rc = check_device_ptr(y, "y")))
    return rc;
  if (rows < 0 || d < 8 || d % 8 || d > (1 << 20)) return fail(DUET_EINVAL, "rows %d / d %d: d a multiple of 8", rows, d);
  if (!(eps > 0.0f)) return fail(DUET_EINVAL, "eps must be > 0");
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(launch_rmsnorm(static_cast<const __bf16*>(x), static_cast<const __bf16*>(weight), static_cast<__bf16*>(y),
                         rows, d, eps, static_cast<hipStream_t>(stream)));
  return DUET_OK;
}

int duet_swiglu(duet_ctx* ctx, const void* gate_up, void* act, int32_t rows, int32_t m, void* stream) {
  clear_error();
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  int rc;
  if ((rc = check_device_ptr(gate_up, "gate_up")) || (rc = check_device_ptr(act, "act"))) return rc;
  if (rows < 0 || m < 8 || m % 8 || m > (1 << 20)) return fail(DUET_EINVAL, "rows %d / m %d: m a multiple of 8", rows, m);
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(launch_swiglu(static_cast<const __bf16*>(gate_up), static_cast<__bf16*>(act), rows, m,
                        static_cast<hipStream_t>(stream)));
  return DUET_OK;
}

int duet_qkv_split(duet_ctx* ctx, const duet_shape* shape, const void* qkv, void* q, void* k_cache, void* v_cache,
                   int64_t num_phys_pages, const int32_t* page_table, int32_t max_pages_per_req,
                   const duet_batch* batch, void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  if (!shape) return fail(DUET_EINVAL, "shape is NULL");
  if (shape->dtype != DUET_BF16) return fail(DUET_EUNSUPPORTED, "the QKV split runs bf16 only");
  const void* q_l[1] = {qkv};
  const void* k_l[1] = {k_cache};
  const void* v_l[1] = {v_cache};
  const void* o_l[1] = {q};
  int rc = check_call(ctx, shape, 1, q_l, k_l, v_l, num_phys_pages, page_table, max_pages_per_req, batch,
                      duet_cu_split{DUET_AGG, DUET_TOTAL_CUS, 0, 1}, workspace, o_l, 0);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ctx->mu);
  Plan& p = ctx->plan;
  plan_batch(shape, batch, 1, 1, &p, true);
  if (workspace_bytes < p.total) return fail(DUET_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, p.total);
  hipStream_t st = static_cast<hipStream_t>(stream);
  HIP_TRY(hipSetDevice(ctx->device));
  char* ws = static_cast<char*>(workspace);
  if ((rc = stage_upload(ctx, p, ws, st))) return rc;
  int64_t T = 0;
  for (int r = 0; r < batch->num_reqs; ++r) T += batch->reqs[r].q_len;
  QkvSplitArgs a;
  a.qkv = static_cast<const __bf16*>(qkv);
  a.q = static_cast<__bf16*>(q);
  a.k_cache = static_cast<__bf16*>(k_cache);
  a.v_cache = static_cast<__bf16*>(v_cache);
  a.meta = reinterpret_cast<const int4*>(ws + p.off_meta);
  a.dreq = nullptr;
  a.page_table = page_table;
  a.num_phys_pages = num_phys_pages;
  a.err = reinterpret_cast<int32_t*>(ws);
  a.num_reqs = batch->num_reqs;
  a.max_pages = max_pages_per_req;
  a.h_q = shape->num_q_heads;
  a.h_kv = shape->num_kv_heads;
  a.head_dim = shape->head_dim;
  a.row0 = 0;
  HIP_TRY(launch_qkv_split(a, (int)T, st));
  return DUET_OK;
}

int duet_block_forward(duet_ctx* ctx, const duet_shape* shape, const duet_block_shape* block,
                       const duet_block_weights* weights, float norm_eps, void* x, void* const* x_ahead,
                       void* const* k_cache, void* const* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                       int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                       size_t workspace_bytes, void* stream) {
  clear_error();
  return block_forward(ctx, shape, block, weights, norm_eps, x, x_ahead, k_cache, v_cache, num_phys_pages,
                       page_table, max_pages_per_req, batch, split, workspace, workspace_bytes, stream);
}

int duet_attn_mixed_batch(duet_ctx* ctx, const duet_shape* shape, const void* q, const void* k_cache,
                          const void* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                          int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                          size_t workspace_bytes, void* out, void* stream) {
  clear_error();
  return attn_layers(ctx, shape, 1, &q, &k_cache, &v_cache, num_phys_pages, page_table, max_pages_per_req, batch,
                     split, workspace, workspace_bytes, &out, stream);
}

int duet_attn_mixed_batch_noalloc(duet_ctx* ctx, const duet_shape* shape, const void* q, const void* k_cache,
                                  const void* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                                  int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* out,
                                  void* stream) {
  clear_error();
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  if (!ctx->scratch_dev) return fail(DUET_EHIP, "the context holds no scratch address");
  return attn_layers(ctx, shape, 1, &q, &k_cache, &v_cache, num_phys_pages, page_table, max_pages_per_req, batch,
                     split, ctx->scratch_dev, kScratchBytes, &out, stream, true);
}

int duet_attn_iteration(duet_ctx* ctx, const duet_shape* shape, const void* const* q, const void* const* k_cache,
                        const void* const* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                        int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                        size_t workspace_bytes, void* const* out, void* stream) {
  clear_error();
  if (!shape) return fail(DUET_EINVAL, "shape is NULL");
  if (!q || !k_cache || !v_cache || !out) return fail(DUET_EINVAL, "per-layer pointer array is NULL");
  return attn_layers(ctx, shape, shape->num_layers, q, k_cache, v_cache, num_phys_pages, page_table,
                     max_pages_per_req, batch, split, workspace, workspace_bytes, out, stream);
}

int duet_lookahead_workspace_bytes(const duet_shape* shape, const duet_batch* batch, int32_t k_decode_steps,
                                   size_t* bytes) {
  clear_error();
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if (!bytes) return fail(DUET_EINVAL, "bytes is NULL");
  if (k_decode_steps < 1 || k_decode_steps > kMaxLookahead)
    return fail(DUET_EINVAL, "k_decode_steps %d not in [1, %d]", k_decode_steps, kMaxLookahead);
  Plan p;
  plan_batch(shape, batch, shape->num_layers, k_decode_steps, &p, false);
  *bytes = p.total;
  return DUET_OK;
}

int duet_attn_lookahead(duet_ctx* ctx, const duet_shape* shape, const void* const* q, const void* const* q_ahead,
                        const void* const* k_ahead, const void* const* v_ahead, void* const* k_cache,
                        void* const* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                        int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                        size_t workspace_bytes, void* const* out, void* const* out_ahead, void* stream) {
  clear_error();
  return attn_lookahead(ctx, shape, q, q_ahead, k_ahead, v_ahead, k_cache, v_cache, num_phys_pages, page_table,
                        max_pages_per_req, batch, split, workspace, workspace_bytes, out, out_ahead, stream);
}

int duet_set_decode_graphs(duet_ctx* ctx, int32_t enable) {
  clear_error();
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  std::lock_guard<std::mutex> lock(ctx->mu);
  ctx->decode_graphs = enable != 0;
  return DUET_OK;
}

int duet_decode_graph_stats(duet_ctx* ctx, int64_t* cached, int64_t* captured, int64_t* replayed) {
  clear_error();
  if (!ctx || !cached || !captured || !replayed) return fail(DUET_EINVAL, "NULL argument");
  std::lock_guard<std::mutex> lock(ctx->mu);
  *cached = (int64_t)ctx->graphs.size();
  *captured = (int64_t)ctx->graphs_captured;
  *replayed = (int64_t)ctx->graphs_replayed;
  return DUET_OK;
}

int duet_check_device_error(duet_ctx* ctx, void* workspace, void* stream) {
  clear_error();
  if (!ctx || !workspace) return fail(DUET_EINVAL, "NULL argument");
  int32_t word = 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(hipMemcpyAsync(&word, workspace, sizeof word, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  if (word) {
    const int32_t zero = 0;
    HIP_TRY(hipMemcpy(workspace, &zero, sizeof zero, hipMemcpyHostToDevice));
    return fail(DUET_EPAGE, "a kernel read a page id outside [0, num_phys_pages)");
  }
  return DUET_OK;
}

int duet_gather_kv(duet_ctx* ctx, const duet_shape* shape, int32_t which, const void* cache, int64_t num_phys_pages,
                   const int32_t* page_table, int32_t max_pages_per_req, int32_t req, int32_t kv_len, void* out_contig,
                   void* stream) {
  clear_error();
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  int rc = check_shape(shape);
  if (rc) return rc;
  if (which != 0 && which != 1) return fail(DUET_EINVAL, "which must be 0 (keys) or 1 (values)");
  if ((rc = check_device_ptr(cache, "cache")) || (rc = check_device_ptr(page_table, "page_table")) ||
      (rc = check_device_ptr(out_contig, "out_contig")))
    return rc;
  if (req < 0 || kv_len < 0 || num_phys_pages < 1) return fail(DUET_EINVAL, "negative request, length or pool");
  if ((kv_len + 15) / 16 > max_pages_per_req) return fail(DUET_EINVAL, "kv_len exceeds the page-table row");
  std::lock_guard<std::mutex> lock(ctx->mu);
  hipStream_t st = static_cast<hipStream_t>(stream);
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(hipMemsetAsync(ctx->dev_flag, 0, sizeof(int32_t), st));
  HIP_TRY(launch_gather(cache, which, shape->dtype == DUET_BF16 ? 2 : 4, shape->num_kv_heads, shape->head_dim,
                        page_table, max_pages_per_req, num_phys_pages, req, kv_len, out_contig, ctx->dev_flag, st));
  int32_t word = 0;
  HIP_TRY(hipMemcpyAsync(&word, ctx->dev_flag, sizeof word, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  return word ? fail(DUET_EPAGE, "page id out of range in the gathered request") : DUET_OK;
}

int duet_set_profiling(duet_ctx* ctx, int32_t enable) {
  if (!ctx) return fail(DUET_EINVAL, "ctx is NULL");
  std::lock_guard<std::mutex> lock(ctx->mu);
  ctx->profiling = enable < 0 ? 0 : (enable > 2 ? 2 : enable);
  return DUET_OK;
}

int duet_last_kernel_times(duet_ctx* ctx, duet_kernel_times* out) {
  clear_error();
  if (!ctx || !out) return fail(DUET_EINVAL, "NULL argument");
  std::lock_guard<std::mutex> lock(ctx->mu);
  if (!ctx->prof_valid) return fail(DUET_EINVAL, "no profiled call recorded");
  HIP_TRY(hipEventSynchronize(ctx->prof[kEvJoin]));
  float ms = 0.f;
  auto span_us = [&](hipEvent_t x, hipEvent_t y, double* us) -> int {
    HIP_TRY(hipEventElapsedTime(&ms, x, y));
    *us = ms * 1e3;
    return DUET_OK;
  };
  std::memset(out, 0, sizeof *out);
  const int L = ctx->prof_layers;
  out->layers = L;
  int rc;
  if (ctx->prof_steps > 0) {
    // look-ahead call: the decode partition's start, the end of step 0 and the end of its last step
    const int k = ctx->prof_steps;
    out->decode_steps = k;
    if (ctx->prof_decode) {
      const std::vector<hipEvent_t>& e = ctx->ev_step;
      if ((rc = span_us(e[0], e[k], &out->decode_total_us)) ||
          (rc = span_us(ctx->prof[kEvFork], e[0], &out->decode_start_us)) ||
          (rc = span_us(e[0], e[1], &out->decode_first_step_us)))
        return rc;
      out->decode_step_us = out->decode_total_us / k;
    }
    if (ctx->prof_prefill) {
      const std::vector<hipEvent_t>& e = ctx->ev_pre;
      if ((rc = span_us(e[0], e[2 * L - 1], &out->prefill_total_us)) ||
          (rc = span_us(ctx->prof[kEvFork], e[0], &out->prefill_start_us)))
        return rc;
      for (int l = 0; ctx->prof_kernels && l < L; ++l) {
        double t = 0.0;
        if ((rc = span_us(e[2 * l], e[2 * l + 1], &t))) return rc;
        out->prefill_us += t / L;
      }
    }
    return span_us(ctx->prof[kEvFork], ctx->prof[kEvJoin], &out->iteration_us);
  }
  if (ctx->prof_kernels && ctx->prof_decode) {
    const std::vector<hipEvent_t>& e = ctx->ev_dec;
    // Layers whose merge was deferred into the next layer's partial kernel launched no reduce.
    const int first_red = ctx->prof_deferred ? L - 1 : 0;
    for (int l = 0; l < L; ++l) {
      double part = 0.0, red = 0.0;
      if ((rc = span_us(e[3 * l], e[3 * l + 1], &part))) return rc;
      out->decode_partial_us += part / L;
      if (l < first_red) continue;
      if ((rc = span_us(e[3 * l + 1], e[3 * l + 2], &red))) return rc;
      out->decode_reduce_us += red / (L - first_red);
    }
    if ((rc = span_us(e[0], e[3 * L - 1], &out->decode_total_us)) ||
        (rc = span_us(ctx->prof[kEvFork], e[0], &out->decode_start_us)))
      return rc;
  }
  if (ctx->prof_kernels && ctx->prof_prefill) {
    const std::vector<hipEvent_t>& e = ctx->ev_pre;
    for (int l = 0; l < L; ++l) {
      double t = 0.0;
      if ((rc = span_us(e[2 * l], e[2 * l + 1], &t))) return rc;
      out->prefill_us += t / L;
    }
    if ((rc = span_us(e[0], e[2 * L - 1], &out->prefill_total_us)) ||
        (rc = span_us(ctx->prof[kEvFork], e[0], &out->prefill_start_us)))
      return rc;
  }
  return span_us(ctx->prof[kEvFork], ctx->prof[kEvJoin], &out->iteration_us);
}

int duet_probe_read_bw(duet_ctx* ctx, int32_t cus, const void* buf, size_t bytes, int32_t iters,
                       double* bytes_per_s) {
  clear_error();
  if (!ctx || !buf || !bytes_per_s) return fail(DUET_EINVAL, "NULL argument");
  if (bytes < (1u << 24) || iters < 1) return fail(DUET_EINVAL, "need >= 16 MiB and iters >= 1");
  std::lock_guard<std::mutex> lock(ctx->mu);
  hipStream_t st;
  int rc = get_stream(ctx, cus, 0, &st);
  if (rc) return rc;
  // The share's ceiling: the best of three grid sizes (8, 16 and 32 waves per CU), each warmed
  // up once and then timed over `iters` launches.
  double best = 0.0;
  for (int blocks_per_cu : {2, 4, 8}) {
    const int blocks = cus * blocks_per_cu;
    HIP_TRY(launch_read_probe(buf, bytes, blocks, ctx->dev_sink, st));
    HIP_TRY(hipEventRecord(ctx->prof[kEvA], st));
    for (int i = 0; i < iters; ++i) HIP_TRY(launch_read_probe(buf, bytes, blocks, ctx->dev_sink, st));
    HIP_TRY(hipEventRecord(ctx->prof[kEvB], st));
    HIP_TRY(hipEventSynchronize(ctx->prof[kEvB]));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, ctx->prof[kEvA], ctx->prof[kEvB]));
    best = std::max(best, (double)read_probe_bytes(bytes, blocks) * iters / (ms * 1e-3));
  }
  ctx->prof_valid = false;
  *bytes_per_s = best;
  return DUET_OK;
}

int duet_probe_mfma(duet_ctx* ctx, int32_t cus, int32_t iters, double* flops_per_s) {
  clear_error();
  if (!ctx || !flops_per_s) return fail(DUET_EINVAL, "NULL argument");
  if (iters < 1) return fail(DUET_EINVAL, "iters must be >= 1");
  std::lock_guard<std::mutex> lock(ctx->mu);
  hipStream_t st;
  int rc = get_stream(ctx, cus, 0, &st);
  if (rc) return rc;
  const int blocks = cus;  // one 8-wave workgroup per CU, two waves per SIMD
  float* sink = reinterpret_cast<float*>(ctx->dev_sink);
  // Clocks settle under sustained matrix load and drop in idle gaps: warm up with four launches,
  // then time three back-to-back launches per sample (no host wait between them) and keep the
  // best of three samples.
  for (int i = 0; i < 4; ++i) HIP_TRY(launch_mfma_probe(blocks, iters, sink, st));
  double best = 0.0;
  const double flops = 3.0 * blocks * 8 /*waves*/ * iters * 32 /*MFMAs per trip*/ * (16.0 * 16 * 32 * 2);
  for (int rep = 0; rep < 3; ++rep) {
    HIP_TRY(hipEventRecord(ctx->prof[kEvA], st));
    for (int l = 0; l < 3; ++l) HIP_TRY(launch_mfma_probe(blocks, iters, sink, st));
    HIP_TRY(hipEventRecord(ctx->prof[kEvB], st));
    HIP_TRY(hipEventSynchronize(ctx->prof[kEvB]));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, ctx->prof[kEvA], ctx->prof[kEvB]));
    best = std::max(best, flops / (ms * 1e-3));
  }
  ctx->prof_valid = false;
  *flops_per_s = best;
  return DUET_OK;
}

int duet_probe_placement(duet_ctx* ctx, int32_t cus, int32_t high_end, int32_t blocks, uint32_t* hw_ids_dev) {
  clear_error();
  if (!ctx || !hw_ids_dev) return fail(DUET_EINVAL, "NULL argument");
  if (blocks < 1 || blocks > 65536) return fail(DUET_EINVAL, "blocks must be in [1, 65536]");
  std::lock_guard<std::mutex> lock(ctx->mu);
  hipStream_t st;
  int rc = get_stream(ctx, cus, high_end ? 1 : 0, &st);
  if (rc) return rc;
  HIP_TRY(launch_placement_probe(blocks, hw_ids_dev, st));
  HIP_TRY(hipStreamSynchronize(st));
  return DUET_OK;
}

int duet_calibrate(duet_ctx* ctx, duet_model* m, const void* scratch, size_t scratch_bytes) {
  clear_error();
  if (!ctx || !m || !scratch) return fail(DUET_EINVAL, "NULL argument");
  std::vector<int32_t> cus(kNumCuSteps);
  std::vector<double> fl(kNumCuSteps), by(kNumCuSteps);
  for (int i = 0; i < kNumCuSteps; ++i) {
    cus[i] = DUET_CU_STEP * (i + 1);
    int rc = duet_probe_read_bw(ctx, cus[i], scratch, scratch_bytes, 3, &by[i]);
    if (rc) return rc;
    if ((rc = duet_probe_mfma(ctx, cus[i], 8192, &fl[i]))) return rc;
  }
  return duet_model_set_tables(m, kNumCuSteps, cus.data(), fl.data(), by.data());
}

}  // extern "C"
