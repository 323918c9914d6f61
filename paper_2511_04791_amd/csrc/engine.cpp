// Serving engine: continuous batching with chunked prefill and a paged KV-cache allocator.
//
// The iterations the paper's scheduler forms (Section 3 and Section 4: a Sarathi-style batch
// former mixes the running decodes with chunks of prompts under a token budget; Section 2: each
// request's keys and values live in cache pages that persist for its lifetime).  Each step:
//   1. every running request whose prompt is fully prefilled decodes one token (its context so
//      far is cached), in admission order, while the budget lasts;
//   2. the rest of the budget goes to prompt tokens: first the requests already partly
//      prefilled, then the waiting ones in arrival order; the last one taken may be chunked;
//   3. the cache pages the scheduled tokens need are reserved from a free list (all or nothing).
// Completing the step advances the chunks, gives each decode its token, admits the requests
// whose first chunk ran, and releases the pages of the requests that have produced all their
// output tokens.  A look-ahead step (Section 4.3: k decode steps while one prefill step runs)
// reserves pages for k tokens of every decode and credits each decode min(k, its remaining
// output) tokens; the steps a finished request would not need are computed and dropped.  Host-only integer bookkeeping: the GPU work of a step is duet_block_forward
// or duet_attn_iteration on the returned rows and page table.
#include <algorithm>
#include <cstdint>
#include <deque>
#include <memory>
#include <new>
#include <vector>

#include "duet_internal.h"

using duet::fail;

namespace {

struct Req {
  int64_t id = 0;
  int prompt = 0, output = 0, prefilled = 0, generated = 0;
  std::vector<int32_t> pages;
};

}  // namespace

struct duet_engine {
  int budget = 0, page_size = 16, max_pages = 0;
  std::vector<int32_t> free_pages;  // a stack: the next page handed out is at the back
  std::deque<std::unique_ptr<Req>> waiting;
  std::vector<std::unique_ptr<Req>> running;
  // the step formed but not yet completed
  bool pending = false;
  int step_k = 1;  // decode steps of the pending step
  std::vector<Req*> step_decodes;
  std::vector<std::pair<Req*, int>> step_chunks;
  int64_t next_id = 0;
};

namespace {

int pages_for(int64_t tokens, int ps) { return (int)((tokens + ps - 1) / ps); }

// splitmix64 (Steele, Lea and Flood, 2014): the permutation of the initial free list.
uint64_t splitmix64(uint64_t* s) {
  uint64_t z = (*s += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

}  // namespace

extern "C" {

int duet_engine_create(int32_t token_budget, int32_t page_size, int64_t num_pages, int32_t max_pages_per_req,
                       uint64_t shuffle_seed, duet_engine** out) {
  duet::clear_error();
  if (!out) return fail(DUET_EINVAL, "out is NULL");
  *out = nullptr;
  if (token_budget < 1) return fail(DUET_EINVAL, "token_budget %d < 1", token_budget);
  if (page_size != 16) return fail(DUET_EUNSUPPORTED, "page_size %d (16 supported)", page_size);
  if (num_pages < 1 || num_pages > (int64_t)INT32_MAX) return fail(DUET_EINVAL, "num_pages %lld out of range", (long long)num_pages);
  if (max_pages_per_req < 1) return fail(DUET_EINVAL, "max_pages_per_req %d < 1", max_pages_per_req);
  duet_engine* e = new (std::nothrow) duet_engine;
  if (!e) return fail(DUET_ENOMEM, "engine allocation failed");
  e->budget = token_budget;
  e->page_size = page_size;
  e->max_pages = max_pages_per_req;
  e->free_pages.resize((size_t)num_pages);
  for (int64_t i = 0; i < num_pages; ++i) e->free_pages[(size_t)i] = (int32_t)(num_pages - 1 - i);  // hands out 0, 1, ...
  if (shuffle_seed) {  // Fisher-Yates
    uint64_t st = shuffle_seed;
    for (size_t i = e->free_pages.size() - 1; i > 0; --i)
      std::swap(e->free_pages[i], e->free_pages[splitmix64(&st) % (i + 1)]);
  }
  *out = e;
  return DUET_OK;
}

int duet_engine_destroy(duet_engine* e) {
  delete e;
  return DUET_OK;
}

int duet_engine_add_request(duet_engine* e, int32_t prompt_len, int32_t output_len, int64_t* id) {
  duet::clear_error();
  if (!e) return fail(DUET_EINVAL, "engine is NULL");
  if (prompt_len < 1 || output_len < 1) return fail(DUET_EINVAL, "prompt and output lengths must be >= 1");
  if (pages_for((int64_t)prompt_len + output_len, e->page_size) > e->max_pages)
    return fail(DUET_EINVAL, "a request of %d + %d tokens needs more than %d pages", prompt_len, output_len, e->max_pages);
  auto r = std::make_unique<Req>();
  r->id = e->next_id++;
  r->prompt = prompt_len;
  r->output = output_len;
  if (id) *id = r->id;
  e->waiting.push_back(std::move(r));
  return DUET_OK;
}

int duet_engine_step_lookahead(duet_engine* e, int32_t decode_steps, duet_seq_meta* meta, int32_t* page_table,
                               int64_t* req_ids, int32_t max_reqs, int32_t* num_reqs) {
  duet::clear_error();
  if (!e || !meta || !page_table || !num_reqs) return fail(DUET_EINVAL, "NULL argument");
  if (e->pending) return fail(DUET_EINVAL, "the previous step is not completed");
  if (decode_steps < 1) return fail(DUET_EINVAL, "decode_steps %d < 1", decode_steps);
  const int k = decode_steps;
  std::vector<Req*> decodes;
  std::vector<std::pair<Req*, int>> chunks;
  int budget = e->budget;
  for (auto& r : e->running)
    if (budget > 0 && r->prefilled >= r->prompt) {
      decodes.push_back(r.get());
      --budget;
    }
  auto take_chunk = [&](Req* r) {
    if (budget <= 0) return;
    const int take = std::min(budget, r->prompt - r->prefilled);
    chunks.emplace_back(r, take);
    budget -= take;
  };
  for (auto& r : e->running)
    if (r->prefilled < r->prompt) take_chunk(r.get());
  for (auto& r : e->waiting) take_chunk(r.get());
  const int n = (int)(decodes.size() + chunks.size());
  if (n > max_reqs) return fail(DUET_EINVAL, "the step holds %d requests, the arrays %d", n, max_reqs);
  // Pages: a decode's k tokens sit at positions prompt + generated .. + k - 1, a chunk's tokens
  // at prefilled .. prefilled + take - 1.
  int64_t need = 0;
  for (Req* r : decodes) {
    const int want = pages_for((int64_t)r->prompt + r->generated + k, e->page_size);
    if (want > e->max_pages)
      return fail(DUET_EINVAL, "request %lld: %d decode steps need %d pages, rows hold %d", (long long)r->id, k, want,
                  e->max_pages);
    need += std::max(0, want - (int)r->pages.size());
  }
  for (auto& c : chunks)
    need += std::max(0, pages_for((int64_t)c.first->prefilled + c.second, e->page_size) - (int)c.first->pages.size());
  if (need > (int64_t)e->free_pages.size())
    return fail(DUET_ENOMEM, "the step needs %lld cache pages, %zu are free", (long long)need, e->free_pages.size());
  auto reserve = [&](Req* r, int64_t tokens) {
    while ((int)r->pages.size() < pages_for(tokens, e->page_size)) {
      r->pages.push_back(e->free_pages.back());
      e->free_pages.pop_back();
    }
  };
  int row = 0, q_start = 0;
  auto emit = [&](Req* r, int kind, int q_len, int cached) {
    meta[row] = duet_seq_meta{kind, q_start, q_len, cached};
    int32_t* pt = page_table + (size_t)row * e->max_pages;
    for (int i = 0; i < e->max_pages; ++i) pt[i] = i < (int)r->pages.size() ? r->pages[i] : -1;
    if (req_ids) req_ids[row] = r->id;
    q_start += q_len;
    ++row;
  };
  for (Req* r : decodes) {
    reserve(r, (int64_t)r->prompt + r->generated + k);
    emit(r, DUET_KIND_DECODE, 1, r->prompt + r->generated);
  }
  for (auto& c : chunks) {
    reserve(c.first, (int64_t)c.first->prefilled + c.second);
    emit(c.first, DUET_KIND_PREFILL, c.second, c.first->prefilled);
  }
  *num_reqs = n;
  e->step_decodes = std::move(decodes);
  e->step_chunks = std::move(chunks);
  e->step_k = k;
  e->pending = true;
  return DUET_OK;
}

int duet_engine_step(duet_engine* e, duet_seq_meta* meta, int32_t* page_table, int64_t* req_ids, int32_t max_reqs,
                     int32_t* num_reqs) {
  return duet_engine_step_lookahead(e, 1, meta, page_table, req_ids, max_reqs, num_reqs);
}

int duet_engine_complete_lookahead(duet_engine* e, int32_t decode_steps_run) {
  duet::clear_error();
  if (!e) return fail(DUET_EINVAL, "engine is NULL");
  if (!e->pending) return fail(DUET_EINVAL, "no step to complete");
  if (decode_steps_run < 1 || decode_steps_run > e->step_k)
    return fail(DUET_EINVAL, "decode_steps_run %d not in [1, %d]", decode_steps_run, e->step_k);
  e->step_k = decode_steps_run;
  for (auto& c : e->step_chunks) {
    Req* r = c.first;
    auto it = std::find_if(e->waiting.begin(), e->waiting.end(), [&](const std::unique_ptr<Req>& w) { return w.get() == r; });
    if (it != e->waiting.end()) {
      e->running.push_back(std::move(*it));
      e->waiting.erase(it);
    }
    r->prefilled += c.second;
  }
  for (Req* r : e->step_decodes) r->generated = std::min(r->output, r->generated + e->step_k);
  std::vector<std::unique_ptr<Req>> keep;
  for (auto& r : e->running) {
    if (r->generated < r->output) {
      keep.push_back(std::move(r));
    } else {
      for (int32_t p : r->pages) e->free_pages.push_back(p);
    }
  }
  e->running = std::move(keep);
  e->step_decodes.clear();
  e->step_chunks.clear();
  e->pending = false;
  return DUET_OK;
}

int duet_engine_complete(duet_engine* e) {
  if (!e) {
    duet::clear_error();
    return fail(DUET_EINVAL, "engine is NULL");
  }
  return duet_engine_complete_lookahead(e, e->step_k);
}

int duet_engine_stats(const duet_engine* e, int64_t* waiting, int64_t* running, int64_t* free_pages) {
  duet::clear_error();
  if (!e) return fail(DUET_EINVAL, "engine is NULL");
  if (waiting) *waiting = (int64_t)e->waiting.size();
  if (running) *running = (int64_t)e->running.size();
  if (free_pages) *free_pages = (int64_t)e->free_pages.size();
  return DUET_OK;
}

}  // extern "C"
