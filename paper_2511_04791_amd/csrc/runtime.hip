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
#include <vector>

#include "duet_internal.h"
#include "kernels.h"

namespace {

using namespace duet;

constexpr int kStagingSlots = 4;
constexpr size_t kMaxMaskedStreams = 6;  // each CU-masked stream owns a hardware queue
constexpr size_t kAlign = 256;
// Workspace head: the device error word at offset 0, one decode work counter per layer from
// kCounterOffset on; the head is zeroed by every call's upload.
constexpr size_t kCounterOffset = 64;
constexpr int kMaxLayers = 1024;

inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

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

// Work lists of one iteration and where they live in the caller's workspace.
struct Plan {
  std::vector<int4> meta, pitems, dreq;
  std::vector<int32_t> ditems;
  int n_items_decode = 0, max_split = 0, pages_per_split = 0, group = 0, prefill_id_cap = 0;
  size_t off_meta = 0, off_pitems = 0, off_dreq = 0, off_ditems = 0, off_pacc = 0, off_pml = 0, upload_bytes = 0,
         total = 0;
};

// Fixed per dtype, never per split or placement, so results are identical for every CU split.
int pages_per_split_for(const duet_shape* s) {
  return s->dtype == DUET_F32 ? kDecodePagesPerSplitF32 : kDecodePagesPerSplit;
}

void plan_batch(const duet_shape* s, const duet_batch* b, int layers, Plan* p, bool fill) {
  const int g = s->num_q_heads / s->num_kv_heads;
  const int pps = pages_per_split_for(s);
  p->group = g;
  p->pages_per_split = pps;
  p->prefill_id_cap = 0;
  p->meta.clear();
  p->pitems.clear();
  p->dreq.clear();
  p->ditems.clear();
  int64_t n_pitems = 0, n_dreq = 0, n_items = 0;
  int max_split = 0;
  struct Tile {
    int64_t keys;
    int4 item;
  };
  std::vector<Tile> tiles;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& q = b->reqs[r];
    if (fill) p->meta.push_back(make_int4(q.kind, q.q_start, q.q_len, q.cached_len));
    const int64_t L = (int64_t)q.cached_len + q.q_len;
    if (q.kind == DUET_KIND_PREFILL) {
      p->prefill_id_cap = std::max(p->prefill_id_cap, (int)((L + 15) / 16));
      // bf16: a unit is nh heads of one group x rows queries; fp32: one head x rows queries.
      const int nh = s->dtype == DUET_BF16 ? prefill_heads_per_unit(g) : 1;
      const int rows = prefill_rows_per_unit(g, s->dtype == DUET_BF16 ? 0 : 1);
      const int n_tiles = (q.q_len + rows - 1) / rows;
      const int units = s->num_q_heads / nh;
      n_pitems += (int64_t)n_tiles * units;
      if (fill) {
        for (int t = 0; t < n_tiles; ++t) {
          const int64_t keys = q.cached_len + std::min(q.q_len, (t + 1) * rows);
          // Units ordered so that workgroup index mod 8 follows the kv head: the units sharing
          // one kv head land on one XCD and share its L2.
          for (int u = 0; u < units; ++u) {
            int h;
            if (nh == 1) h = (u % s->num_kv_heads) * g + u / s->num_kv_heads;
            else h = u * nh;
            tiles.push_back({keys, make_int4(r, h, t * rows, 0)});
          }
        }
      }
    } else {
      const int n_pages = (int)((L + 15) / 16);
      const int n_split = (n_pages + pps - 1) / pps;
      if (fill) p->dreq.push_back(make_int4(r, (int)n_items, n_split, n_pages));
      n_items += (int64_t)s->num_kv_heads * n_split;
      max_split = std::max(max_split, n_split);
      ++n_dreq;
    }
  }
  if (fill) {
    std::stable_sort(tiles.begin(), tiles.end(), [](const Tile& x, const Tile& y) { return x.keys > y.keys; });
    p->pitems.reserve(tiles.size());
    for (const Tile& t : tiles) p->pitems.push_back(t.item);
    // bf16 decode items in execution order: every full split first, then the shorter last
    // splits (longest first), packed as i | j << 16 | s << 22.
    if (s->dtype == DUET_BF16) {
      p->ditems.reserve(n_items);
      for (int pass = 0; pass < 2; ++pass)
        for (size_t i = 0; i < p->dreq.size(); ++i) {
          const int4 d = p->dreq[i];
          const bool full_last = d.w % pps == 0;
          for (int j = 0; j < s->num_kv_heads; ++j)
            for (int sp = 0; sp < d.z; ++sp) {
              const bool is_full = sp + 1 < d.z || full_last;
              if (is_full == (pass == 0)) p->ditems.push_back((int32_t)i | (j << 16) | (sp << 22));
            }
        }
    }
  }
  p->n_items_decode = (int)n_items;
  p->max_split = max_split;
  size_t off = align_up(kCounterOffset + (size_t)layers * sizeof(int32_t));
  p->off_meta = off;
  off = align_up(off + (size_t)b->num_reqs * sizeof(int4));
  p->off_pitems = off;
  off = align_up(off + (size_t)n_pitems * sizeof(int4));
  p->off_dreq = off;
  off = align_up(off + (size_t)n_dreq * sizeof(int4));
  p->off_ditems = off;
  off = align_up(off + (s->dtype == DUET_BF16 ? (size_t)n_items * sizeof(int32_t) : 0));
  p->upload_bytes = off;
  p->off_pacc = off;
  off = align_up(off + (size_t)n_items * g * s->head_dim * sizeof(float));
  p->off_pml = off;
  off = align_up(off + (size_t)n_items * g * 2 * sizeof(float));
  p->total = off;
}

// Fork and join of a profiled call on the caller's stream; A and B bracket probe kernels.
enum ProfEv { kEvFork, kEvJoin, kEvA, kEvB, kNumProfEv };

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

int stage_upload(duet_ctx* ctx, const Plan& p, char* ws, hipStream_t st) {
  StagingSlot& slot = ctx->slots[ctx->next_slot];
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
  std::memcpy(h + p.off_ditems, p.ditems.data(), p.ditems.size() * sizeof(int32_t));
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
int attn_layers(duet_ctx* ctx, const duet_shape* shape, int layers, const void* const* q_l,
                const void* const* k_l, const void* const* v_l, int64_t num_phys_pages, const int32_t* page_table,
                int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                size_t workspace_bytes, void* const* out_l, void* stream) {
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
    const int64_t L = (int64_t)batch->reqs[r].cached_len + batch->reqs[r].q_len;
    if ((L + 15) / 16 > max_pages_per_req)
      return fail(DUET_EINVAL, "request %d needs %lld pages, page_table rows hold %d", r, (long long)((L + 15) / 16),
                  max_pages_per_req);
  }
  {
    int n_dec = 0;
    for (int r = 0; r < batch->num_reqs; ++r) {
      const duet_seq_meta& q = batch->reqs[r];
      const int64_t L = (int64_t)q.cached_len + q.q_len;
      if (q.kind == DUET_KIND_DECODE) ++n_dec;
      if (q.kind == DUET_KIND_PREFILL && L > kMaxPrefillKeys)
        return fail(DUET_EUNSUPPORTED, "request %d: prefill attends %lld keys, at most %d supported", r,
                    (long long)L, kMaxPrefillKeys);
      if (q.kind == DUET_KIND_DECODE && (L + 15) / 16 > 1023LL * kDecodePagesPerSplit)
        return fail(DUET_EUNSUPPORTED, "request %d: decode context %lld too long", r, (long long)L);
    }
    if (n_dec > 65535) return fail(DUET_EUNSUPPORTED, "more than 65535 decode requests");
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

  std::lock_guard<std::mutex> lock(ctx->mu);
  Plan& p = ctx->plan;
  plan_batch(shape, batch, layers, &p, true);
  if (workspace_bytes < p.total)
    return fail(DUET_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, p.total);

  hipStream_t order = static_cast<hipStream_t>(stream);
  hipStream_t sd = order, sp = order;
  HIP_TRY(hipSetDevice(ctx->device));
  if (split.mode == DUET_SPLIT) {
    if ((rc = get_stream(ctx, split.cus_decode, 0, &sd))) return rc;
    if ((rc = get_stream(ctx, split.cus_prefill, 1, &sp))) return rc;
  } else if (split.mode == DUET_CONCURRENT) {
    // two streams whose masks both cover every CU
    if ((rc = get_stream(ctx, ctx->num_cus, 0, &sd))) return rc;
    if ((rc = get_stream(ctx, ctx->num_cus, 1, &sp))) return rc;
  }
  const bool forked = split.mode != DUET_AGG;

  char* ws = static_cast<char*>(workspace);
  AttnArgs a;
  a.page_table = page_table;
  a.num_phys_pages = num_phys_pages;
  a.max_pages = max_pages_per_req;
  a.h_q = shape->num_q_heads;
  a.h_kv = shape->num_kv_heads;
  a.group = p.group;
  a.head_dim = shape->head_dim;
  a.dtype = shape->dtype;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)shape->head_dim));
  WorkArgs w;
  w.meta = reinterpret_cast<const int4*>(ws + p.off_meta);
  w.pitems = reinterpret_cast<const int4*>(ws + p.off_pitems);
  w.dreq = reinterpret_cast<const int4*>(ws + p.off_dreq);
  w.pacc = reinterpret_cast<float*>(ws + p.off_pacc);
  w.pml = reinterpret_cast<float*>(ws + p.off_pml);
  w.ditems = reinterpret_cast<const int32_t*>(ws + p.off_ditems);
  w.err = reinterpret_cast<int32_t*>(ws);
  w.n_ditems = (int)p.ditems.size();
  w.decode_cus = split.mode == DUET_SPLIT ? split.cus_decode : ctx->num_cus;
  w.n_pitems = (int)p.pitems.size();
  w.n_dreq = (int)p.dreq.size();
  w.max_split = p.max_split;
  w.pages_per_split = p.pages_per_split;
  w.prefill_id_cap = p.prefill_id_cap;
  const bool prof_iter = ctx->profiling >= 1;
  const bool prof = ctx->profiling >= 2;
  const bool has_decode = w.n_dreq > 0, has_prefill = w.n_pitems > 0;

  if (prof_iter) HIP_TRY(hipEventRecord(ctx->prof[kEvFork], order));
  if ((rc = stage_upload(ctx, p, ws, order))) return rc;
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
  for (int l = 0; l < layers; ++l) {
    const AttnArgs al = layer_args(l);
    if (has_decode) {
      WorkArgs wl = w;
      wl.work_counter = reinterpret_cast<int32_t*>(ws + kCounterOffset) + l;
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_dec[3 * l], sd));
      HIP_TRY(launch_decode_partial(al, wl, sd));
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_dec[3 * l + 1], sd));
      HIP_TRY(launch_decode_reduce(al, wl, sd));
      if (prof) HIP_TRY(hipEventRecord(ctx->ev_dec[3 * l + 2], sd));
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
  ctx->prof_valid = prof_iter;
  ctx->prof_kernels = prof;
  ctx->prof_decode = has_decode;
  ctx->prof_prefill = has_prefill;
  ctx->prof_layers = layers;
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
  ctx->dev_sink = reinterpret_cast<unsigned*>(ctx->dev_flag) + 16;
  *out = ctx;
  return DUET_OK;
}

int duet_destroy(duet_ctx* ctx) {
  if (!ctx) return DUET_OK;
  (void)hipSetDevice(ctx->device);
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
  plan_batch(shape, batch, shape->num_layers, &p, false);
  *bytes = p.total;
  return DUET_OK;
}

int duet_attn_mixed_batch(duet_ctx* ctx, const duet_shape* shape, const void* q, const void* k_cache,
                          const void* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                          int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                          size_t workspace_bytes, void* out, void* stream) {
  clear_error();
  return attn_layers(ctx, shape, 1, &q, &k_cache, &v_cache, num_phys_pages, page_table, max_pages_per_req, batch,
                     split, workspace, workspace_bytes, &out, stream);
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
  if (ctx->prof_kernels && ctx->prof_decode) {
    const std::vector<hipEvent_t>& e = ctx->ev_dec;
    for (int l = 0; l < L; ++l) {
      double part = 0.0, red = 0.0;
      if ((rc = span_us(e[3 * l], e[3 * l + 1], &part)) || (rc = span_us(e[3 * l + 1], e[3 * l + 2], &red))) return rc;
      out->decode_partial_us += part / L;
      out->decode_reduce_us += red / L;
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
  if (bytes < (1u << 20) || iters < 1) return fail(DUET_EINVAL, "need >= 1 MiB and iters >= 1");
  std::lock_guard<std::mutex> lock(ctx->mu);
  hipStream_t st;
  int rc = get_stream(ctx, cus, 0, &st);
  if (rc) return rc;
  const int blocks = cus * 8;
  HIP_TRY(launch_read_probe(buf, bytes, blocks, ctx->dev_sink, st));  // warm-up
  HIP_TRY(hipEventRecord(ctx->prof[kEvA], st));
  for (int i = 0; i < iters; ++i) HIP_TRY(launch_read_probe(buf, bytes, blocks, ctx->dev_sink, st));
  HIP_TRY(hipEventRecord(ctx->prof[kEvB], st));
  HIP_TRY(hipEventSynchronize(ctx->prof[kEvB]));
  float ms = 0.f;
  HIP_TRY(hipEventElapsedTime(&ms, ctx->prof[kEvA], ctx->prof[kEvB]));
  ctx->prof_valid = false;
  *bytes_per_s = (double)(bytes / 16 * 16) * iters / (ms * 1e-3);
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
  const int blocks = cus * 2;  // 8 waves per CU, two per SIMD
  float* sink = reinterpret_cast<float*>(ctx->dev_sink);
  HIP_TRY(launch_mfma_probe(blocks, iters, sink, st));
  HIP_TRY(hipEventRecord(ctx->prof[kEvA], st));
  HIP_TRY(launch_mfma_probe(blocks, iters, sink, st));
  HIP_TRY(hipEventRecord(ctx->prof[kEvB], st));
  HIP_TRY(hipEventSynchronize(ctx->prof[kEvB]));
  float ms = 0.f;
  HIP_TRY(hipEventElapsedTime(&ms, ctx->prof[kEvA], ctx->prof[kEvB]));
  ctx->prof_valid = false;
  const double flops = (double)blocks * 4 /*waves*/ * iters * 4 /*chains*/ * (32.0 * 32 * 16 * 2);
  *flops_per_s = flops / (ms * 1e-3);
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
    if ((rc = duet_probe_mfma(ctx, cus[i], 2048, &fl[i]))) return rc;
  }
  return duet_model_set_tables(m, kNumCuSteps, cus.data(), fl.data(), by.data());
}

}  // extern "C"
