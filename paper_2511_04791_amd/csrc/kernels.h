// Launch interface between the runtime and the HIP kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace duet {

// Per-iteration tensors and shape, common to every attention kernel.
struct AttnArgs {
  const void* q;         // [T, h_q, d]
  const void* k_cache;   // [P, h_kv, 16, d]
  const void* v_cache;   // [P, h_kv, d, 16]
  const int32_t* page_table;
  void* out;             // [T, h_q, d]
  long long num_phys_pages;
  int32_t max_pages;     // row stride of page_table
  int32_t h_q, h_kv, group, head_dim, dtype;
  float scale_log2;      // log2(e) / sqrt(d): scores are kept in base-2 units
};

// Work lists and scratch that live in the caller's workspace.
struct WorkArgs {
  const int4* meta;     // [R]  (kind, q_start, q_len, cached_len)
  const int4* pitems;   // [NP] prefill tiles (req, q_head, q_row0, 0), heaviest first
  const int4* dreq;     // [RD] decode requests (req, item_base, n_split, n_pages)
  float* pacc;          // [ND, group, d]  unnormalised split-K partial outputs
  float* pml;           // [ND, group, 2]  (running max in base-2 units, softmax denominator)
  const int4* ditems;   // [ND] bf16 decode items in execution order: (q_start, req | kv head << 24,
                        //      first page | (tokens - 1) << 22, row of the item's partial)
  int32_t* err;         // error word: bit 0 = page id out of range
  int32_t* work_counter;  // kDecodeSetInts ints: this launch's counter set (see kDecodeQueues)
  int32_t* clear_counter; // counter set a bf16 partial kernel clears when it starts, or null
  // Deferred merge (bf16): the split-K partials of the layer before, merged by this partial
  // kernel's waves once its item queue is empty.  n_merge = 0: nothing to merge.
  const float* merge_pacc;
  const float* merge_pml;
  void* merge_out;        // that layer's output
  int32_t n_merge;        // (decode request, query head) pairs
  int32_t n_pitems, n_dreq, max_split, n_ditems;
  int32_t pages_per_split;
  int32_t decode_cus;   // CUs the decode stream may use (sizes the persistent grid)
  int32_t prefill_id_cap;  // most pages of any prefill request (sizes the LDS page-id table)
  // Prefill key split (bf16, see kPrefillPieceFill): a piece item carries
  // ((split unit + 1) << kPrefillPieceBits) | piece in its w field (0: a whole unit).
  float* ppart;               // [slots] partial state of every piece: unnormalised O, running max, denominator
  const int2* psplit;         // [split units] (first slot, pieces | key tiles per piece << 16)
  int32_t* pcount;            // [split units] pieces finished; zero before and after every launch
  int32_t prefill_piece_tiles;  // P of the rule below (0: no unit is split)
};

// One decode step's cache write (look-ahead decode): new key and value rows in, paged cache out.
struct AppendArgs {
  void* k_cache;         // [P, h_kv, 16, d], written
  void* v_cache;         // [P, h_kv, d, 16], written
  const void* k_new;     // [R_d, h_kv, d]: row = the request's q_start in the step's metadata
  const void* v_new;     // [R_d, h_kv, d]
  const int32_t* page_table;
  long long num_phys_pages;
  int32_t max_pages;
  int32_t h_kv, head_dim, dtype;
};

// Decode split length in pages (bf16); fixed, so results do not depend on the CU split.
constexpr int kDecodePagesPerSplit = 32;
constexpr int kDecodePagesPerSplitF32 = 2;
// Most logical pages of a bf16 decode request (an item's first page is a 22-bit field).
constexpr long long kMaxDecodePages = (1LL << 22) - 1;

// The persistent decode kernel's work queue is split into kDecodeQueues counters (items are dealt
// round-robin to them), each on its own 128-byte line: atomics on one line are serialised, at a
// few tens per microsecond.  A counter set is kDecodeQueues item queues followed by kDecodeQueues
// merge queues (the deferred merge of the layer before).  A call has two sets, which consecutive
// layers alternate: the upload zeroes both, a partial kernel clears the set the kernel before it
// on the stream used (that kernel has finished), and a reduce kernel clears the set of the
// partial kernel it follows.
constexpr int kDecodeQueues = 8;
constexpr int kDecodeQueueStride = 32;  // ints: one 128-byte line per counter
constexpr int kDecodeSetLines = 2 * kDecodeQueues;
constexpr int kDecodeSetInts = kDecodeSetLines * kDecodeQueueStride;
constexpr int kDecodeCounterInts = 2 * kDecodeSetInts;

// Keys a prefill request may attend (its page ids are staged in LDS: 8192 ids, 32 KB).
constexpr int kMaxPrefillKeys = 131072;

constexpr int kPrefillRows = 128;  // query rows per fp32 prefill item (4 waves x 32)
constexpr int kPrefillKeys = 64;   // keys per LDS stage (4 pages)

// bf16 prefill work unit: prefill_heads_per_unit(group) query heads of one GQA group times
// prefill_rows_per_unit(group, dtype) queries.  fp32 items are one head times kPrefillRows.
int prefill_heads_per_unit(int group);
int prefill_rows_per_unit(int group, int dtype);

// Prefill key split (bf16).  Let T be the batch's total key tiles (kPrefillKeys keys) over all
// units and P = max(kPrefillPieceMinTiles, ceil(T / kPrefillPieceFill)), an even share of the
// batch over one workgroup per CU of the whole chip.  A unit whose causal key range spans more
// than 1.5 P tiles runs as n = ceil(tiles / P) pieces of ceil(tiles / n) consecutive tiles (the
// last may be shorter; n is recounted so that none is empty), so a short chunk after a long
// cached prefix (few units, each long) still fills the CUs.  Every piece pays a fixed start-up
// cost and a partial-state round trip, so units within 1.5 P of the share stay whole.  P depends
// on the batch only, never on the CU split, so results are the same for every split.  Each piece
// writes its partial state to a slot; the piece that finishes last (an arrival counter per unit)
// merges the slots in piece order and writes the output.  Split units number at most
// T / P <= kPrefillPieceFill and their slots at most 2 T / P, plus the tail split's below
// (kPrefillPieceFill units, kPrefillTailPieces slots each).
constexpr int kPrefillPieceMinTiles = 8;
constexpr int kPrefillPieceFill = 256;
// Tail split (batch-only as well): when the whole units number at least 2 kPrefillPieceFill, the
// kPrefillPieceFill shortest of them (dispatched last) run as kPrefillTailPieces pieces, each of
// at least kPrefillTailMinTiles tiles, so the last round of workgroups is fine-grained on any share
// (one workgroup per CU leaves up to one unit's length idle at the end otherwise).
constexpr int kPrefillTailPieces = 4;
constexpr int kPrefillTailMinTiles = 16;
constexpr int kPrefillPieceBits = 12;  // piece index field of an item's w (pieces <= 4095)
int prefill_piece_tiles_for(long long total_tiles);
size_t prefill_slot_bytes(int head_dim);  // one piece's partial state

// The QKV-split step of a block (bf16): query rows out, new keys and values into the cache.
struct QkvSplitArgs {
  const __bf16* qkv;       // [T, (h_q + 2 h_kv) d] projection output
  __bf16* q;               // [T, h_q, d]
  __bf16* k_cache;         // [P, h_kv, 16, d]
  __bf16* v_cache;         // [P, h_kv, d, 16]
  const int4* meta;        // [R] (kind, q_start, q_len, cached_len), q_start rising
  const int4* dreq;        // null: a row's request is found by q_start; else row i is decode request i
                           //       (dreq[i].x) of a look-ahead step
  const int32_t* page_table;
  long long num_phys_pages;
  int32_t* err;
  int32_t num_reqs, max_pages, h_q, h_kv, head_dim;
  int32_t row0;            // first row of the launch
};

hipError_t launch_rmsnorm(const __bf16* x, const __bf16* w, __bf16* y, int rows, int d, float eps, hipStream_t s);
hipError_t launch_swiglu(const __bf16* gu, __bf16* a, int rows, int m, hipStream_t s);
hipError_t launch_qkv_split(const QkvSplitArgs& a, int rows, hipStream_t s);

hipError_t launch_decode_partial(const AttnArgs& a, const WorkArgs& w, hipStream_t s);
hipError_t launch_decode_reduce(const AttnArgs& a, const WorkArgs& w, hipStream_t s);
hipError_t launch_prefill(const AttnArgs& a, const WorkArgs& w, hipStream_t s);
// Writes the new token of every decode request in w.dreq (position = meta cached_len).
hipError_t launch_kv_append(const AppendArgs& a, const WorkArgs& w, hipStream_t s);

hipError_t launch_gather(const void* cache, int which, int elem_bytes, int h_kv, int d, const int32_t* page_table,
                         int max_pages, long long num_phys, int req, int kv_len, void* out, int32_t* err,
                         hipStream_t s);

hipError_t launch_read_probe(const void* buf, size_t bytes, int blocks, unsigned* sink, hipStream_t s);
size_t read_probe_bytes(size_t bytes, int blocks);
hipError_t launch_mfma_probe(int blocks, int iters, float* sink, hipStream_t s);
hipError_t launch_placement_probe(int blocks, uint32_t* out, hipStream_t s);

}  // namespace duet
