// Host-side attention-aware roofline latency model and CU-split optimiser.
//
// Paper, Section 4.1 (sequence-level operators, overall estimation): per request with q
// scheduled and c cached tokens,
//   F(q, c) = 4 h_q q (q + c) d + 2 h_q q (q + c)        B(q, c) = 2 h_q q d b + 2 h_kv (q + c) d b
// and a set of requests on S CUs takes t = L * sum_r max(F_r / Pi(S), B_r / B(S)).
// Paper, Section 4.2 and Algorithm 1: temporal sharing when the whole-GPU estimate meets the
// TBT bound; otherwise the split (S_p, S_d, k) that maximises token throughput
// (k T_decode + T_prefill) / max(k t_d(S_d), t_p(S_p)) subject to t_d(S_d) <= tau.
//
// Tables hold S = 8, 16, ..., 256 (one CU per XCD per step); Algorithm 1 searches S_d in steps of
// 32 CUs (one CU per shader engine of every XCD), the shares on which work spreads evenly.
// Extension: a fixed latency per layer of each partition kind on S CUs (kernel launches, the
// decode kernel's tail), zero by default, added when the batch holds requests of that kind.
#include <cerrno>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "duet_internal.h"

namespace duet {

namespace {
thread_local std::string g_err;

constexpr double kNominalBf16Flops = 2.5e15;  // dense bf16 MFMA, 256 CUs at 2.4 GHz
constexpr double kNominalHbmBytes = 8.0e12;   // HBM3E

struct ReqCost {
  double flops, bytes;
};

inline ReqCost request_cost(const duet_shape* s, const duet_seq_meta& r) {
  const double q = r.q_len, c = r.cached_len, hq = s->num_q_heads, hkv = s->num_kv_heads;
  const double d = s->head_dim, b = (s->dtype == DUET_BF16) ? 2.0 : 4.0;
  ReqCost rc;
  rc.flops = 4.0 * hq * q * (q + c) * d + 2.0 * hq * q * (q + c);
  rc.bytes = 2.0 * hq * q * d * b + 2.0 * hkv * (q + c) * d * b;
  return rc;
}

inline int cu_index(int cus) { return cus / DUET_CU_STEP - 1; }

// Token-level operators of one layer on n tokens (Section 4.1): sum of max(F / pi, B / bw).
double token_level(double n, const duet_shape* s, const duet_block_shape* blk, double pi, double bw) {
  const double b = (s->dtype == DUET_BF16) ? 2.0 : 4.0;
  const double hq = s->num_q_heads, hkv = s->num_kv_heads, dh = s->head_dim;
  const double d = hq * dh, ffn = blk->ffn_dim;
  const double d_qkv = (blk->flags & DUET_BLOCK_GQA_QKV) ? (hq + 2.0 * hkv) * dh : d;
  const double d_gu = (blk->flags & DUET_BLOCK_FUSED_GATE_UP) ? 2.0 * ffn : ffn;
  auto op = [&](double f, double by) { return std::fmax(f / pi, by / bw); };
  auto linear = [&](double di, double dout) { return op(2.0 * n * di * dout, n * di * b + di * dout * b + n * dout * b); };
  const double norm = op(4.0 * n * d, 2.0 * n * d * b + d * b);
  const double add = op(1.0 * n * d, 3.0 * n * d * b);
  double t = norm;
  t += linear(d, d_qkv);
  t += linear(d, d);
  t += add;
  t += norm;
  t += linear(d, d_gu);
  t += op(5.0 * n * ffn, 3.0 * n * ffn * b);
  t += linear(ffn, d);
  t += add;
  return t;
}

// Seconds for `num_layers` layers of the requests whose kind matches `kind` (-1 = all) on `cus`
// CUs: attention only (blk NULL), or the full model with its token-level operators and classifier.
// `shared`: the half runs while the other half runs on the other CUs, so the spatial-sharing
// efficiencies apply.
double f_roofline(const duet_model* m, const duet_shape* s, const duet_batch* b, int kind, int cus,
                  bool shared = false, const duet_block_shape* blk = nullptr) {
  const int i = cu_index(cus);
  const bool tab = shared && m->has_shared;
  const double pi = (tab ? m->flops_shared[i] : m->flops[i]) * (shared ? m->prefill_eff : 1.0);
  const double bw = (tab ? m->bytes_shared[i] : m->bytes[i]) * (shared ? m->decode_eff : 1.0);
  double t = 0.0, n = 0.0;
  int n_req = 0;
  bool any_pre = false, any_dec = false;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& rq = b->reqs[r];
    if (kind >= 0 && rq.kind != kind) continue;
    const ReqCost rc = request_cost(s, rq);
    t += std::fmax(rc.flops / pi, rc.bytes / bw);
    n += rq.q_len;
    ++n_req;
    (rq.kind == DUET_KIND_DECODE ? any_dec : any_pre) = true;
  }
  t += (any_pre ? m->launch_prefill[i] : 0.0) + (any_dec ? m->launch_decode[i] : 0.0);
  if (!blk || n_req == 0) return s->num_layers * t;
  double total = s->num_layers * (token_level(n, s, blk, pi, bw) + t);
  if (blk->vocab_size > 0) {
    const double el = (s->dtype == DUET_BF16) ? 2.0 : 4.0;
    const double d = (double)s->num_q_heads * s->head_dim, v = blk->vocab_size, rows = n_req;
    total += std::fmax(2.0 * rows * d * v / pi, (rows * d * el + d * v * el + rows * v * el) / bw);
  }
  return total;
}

bool has_both_kinds(const duet_batch* b) {
  bool d = false, p = false;
  for (int r = 0; r < b->num_reqs; ++r) (b->reqs[r].kind == DUET_KIND_DECODE ? d : p) = true;
  return d && p;
}

const duet_model* model_or_nominal(const duet_model* m, duet_model* storage) {
  if (m) return m;
  model_init_nominal(storage);
  return storage;
}

bool check_split(const duet_cu_split& sp) {
  if (sp.mode == DUET_AGG) return true;
  if (sp.mode != DUET_SPLIT) return false;
  if (sp.cus_prefill < DUET_CU_STEP || sp.cus_decode < DUET_CU_STEP) return false;
  if (sp.cus_prefill % DUET_CU_STEP || sp.cus_decode % DUET_CU_STEP) return false;
  if (sp.cus_prefill + sp.cus_decode > DUET_TOTAL_CUS) return false;
  return sp.k_decode_steps >= 1;
}
}  // namespace

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

void clear_error() { g_err.clear(); }

const char* last_error_cstr() { return g_err.c_str(); }

int check_shape(const duet_shape* s) {
  if (!s) return fail(DUET_EINVAL, "shape is NULL");
  if (s->num_q_heads < 1 || s->num_kv_heads < 1 || s->num_layers < 1)
    return fail(DUET_EINVAL, "head counts and num_layers must be >= 1");
  if (s->num_q_heads % s->num_kv_heads)
    return fail(DUET_EUNSUPPORTED, "num_q_heads %d not a multiple of num_kv_heads %d", s->num_q_heads,
                s->num_kv_heads);
  if (s->num_q_heads / s->num_kv_heads > 16)
    return fail(DUET_EUNSUPPORTED, "query heads per kv head must be <= 16");
  if (s->head_dim != 64 && s->head_dim != 128) return fail(DUET_EUNSUPPORTED, "head_dim must be 64 or 128");
  if (s->page_size != 16) return fail(DUET_EUNSUPPORTED, "page_size must be 16");
  if (s->dtype != DUET_BF16 && s->dtype != DUET_F32) return fail(DUET_EUNSUPPORTED, "dtype must be bf16 or f32");
  return DUET_OK;
}

int check_batch(const duet_shape* s, const duet_batch* b, bool need_q_start) {
  if (!b) return fail(DUET_EINVAL, "batch is NULL");
  if (b->num_reqs < 0) return fail(DUET_EINVAL, "num_reqs < 0");
  if (b->num_reqs > 0 && !b->reqs) return fail(DUET_EINVAL, "batch.reqs is NULL");
  int64_t next = 0;
  for (int r = 0; r < b->num_reqs; ++r) {
    const duet_seq_meta& q = b->reqs[r];
    if (q.kind != DUET_KIND_PREFILL && q.kind != DUET_KIND_DECODE)
      return fail(DUET_EINVAL, "request %d: kind %d", r, q.kind);
    if (q.q_len < 1) return fail(DUET_EINVAL, "request %d: q_len %d < 1", r, q.q_len);
    if (q.cached_len < 0) return fail(DUET_EINVAL, "request %d: cached_len < 0", r);
    if (q.kind == DUET_KIND_DECODE && q.q_len != 1)
      return fail(DUET_EINVAL, "request %d: decode requests schedule exactly one token", r);
    if ((int64_t)q.cached_len + q.q_len > (int64_t)1 << 30) return fail(DUET_EINVAL, "request %d: too long", r);
    if (need_q_start) {
      if (q.q_start != next) return fail(DUET_EINVAL, "request %d: q_start %d, expected %lld", r, q.q_start,
                                         (long long)next);
      next += q.q_len;
    }
  }
  (void)s;
  return DUET_OK;
}

void model_init_nominal(duet_model* m) {
  for (int i = 0; i < kNumCuSteps; ++i) {
    const double frac = double(DUET_CU_STEP * (i + 1)) / DUET_TOTAL_CUS;
    m->flops[i] = kNominalBf16Flops * frac;
    m->bytes[i] = kNominalHbmBytes * frac;
  }
  m->has_shared = false;
  for (int i = 0; i < kNumCuSteps; ++i) m->launch_prefill[i] = m->launch_decode[i] = 0.0;
  m->prefill_eff = 1.0;
  m->decode_eff = 1.0;
  m->calibrated = false;
}

}  // namespace duet

using namespace duet;

extern "C" {

const char* duet_last_error(void) { return duet::last_error_cstr(); }

int duet_model_create(duet_model** out) {
  if (!out) return fail(DUET_EINVAL, "out is NULL");
  duet_model* m = new (std::nothrow) duet_model;
  if (!m) return fail(DUET_ENOMEM, "model allocation failed");
  model_init_nominal(m);
  *out = m;
  return DUET_OK;
}

int duet_model_destroy(duet_model* m) {
  delete m;
  return DUET_OK;
}

int duet_batch_work(const duet_shape* shape, const duet_batch* batch, int32_t kind, double* flops, double* bytes) {
  clear_error();
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if (!flops || !bytes) return fail(DUET_EINVAL, "NULL output");
  if (kind != -1 && kind != DUET_KIND_PREFILL && kind != DUET_KIND_DECODE) return fail(DUET_EINVAL, "kind %d", kind);
  double f = 0.0, b = 0.0;
  for (int r = 0; r < batch->num_reqs; ++r) {
    if (kind >= 0 && batch->reqs[r].kind != kind) continue;
    const ReqCost c = request_cost(shape, batch->reqs[r]);
    f += c.flops;
    b += c.bytes;
  }
  *flops = shape->num_layers * f;
  *bytes = shape->num_layers * b;
  return DUET_OK;
}

namespace {
int check_tables(int32_t n, const int32_t* cus, const double* flops_per_s, const double* bytes_per_s) {
  if (!cus || !flops_per_s || !bytes_per_s) return fail(DUET_EINVAL, "NULL argument");
  if (n != kNumCuSteps) return fail(DUET_EINVAL, "expected %d table entries, got %d", kNumCuSteps, n);
  for (int i = 0; i < n; ++i) {
    if (cus[i] != DUET_CU_STEP * (i + 1)) return fail(DUET_EINVAL, "cus[%d] = %d, expected %d", i, cus[i],
                                                       DUET_CU_STEP * (i + 1));
    if (!(flops_per_s[i] > 0) || !(bytes_per_s[i] > 0) || !std::isfinite(flops_per_s[i]) ||
        !std::isfinite(bytes_per_s[i]))
      return fail(DUET_EINVAL, "table entry %d not positive and finite", i);
  }
  return DUET_OK;
}
}  // namespace

int duet_model_set_tables(duet_model* m, int32_t n, const int32_t* cus, const double* flops_per_s,
                          const double* bytes_per_s) {
  if (!m) return fail(DUET_EINVAL, "model is NULL");
  int rc = check_tables(n, cus, flops_per_s, bytes_per_s);
  if (rc) return rc;
  for (int i = 0; i < n; ++i) {
    m->flops[i] = flops_per_s[i];
    m->bytes[i] = bytes_per_s[i];
  }
  m->has_shared = false;
  m->calibrated = true;
  return DUET_OK;
}

int duet_model_set_sharing_tables(duet_model* m, int32_t n, const int32_t* cus, const double* flops_per_s,
                                  const double* bytes_per_s) {
  if (!m) return fail(DUET_EINVAL, "model is NULL");
  int rc = check_tables(n, cus, flops_per_s, bytes_per_s);
  if (rc) return rc;
  for (int i = 0; i < n; ++i) {
    m->flops_shared[i] = flops_per_s[i];
    m->bytes_shared[i] = bytes_per_s[i];
  }
  m->has_shared = true;
  return DUET_OK;
}

int duet_model_get_sharing_tables(const duet_model* m, int32_t n, int32_t* cus, double* flops_per_s,
                                  double* bytes_per_s, int32_t* is_set) {
  if (!m || !cus || !flops_per_s || !bytes_per_s || !is_set) return fail(DUET_EINVAL, "NULL argument");
  if (n != kNumCuSteps) return fail(DUET_EINVAL, "expected %d table entries", kNumCuSteps);
  for (int i = 0; i < n; ++i) {
    cus[i] = DUET_CU_STEP * (i + 1);
    flops_per_s[i] = m->has_shared ? m->flops_shared[i] : m->flops[i];
    bytes_per_s[i] = m->has_shared ? m->bytes_shared[i] : m->bytes[i];
  }
  *is_set = m->has_shared ? 1 : 0;
  return DUET_OK;
}

int duet_model_get_tables(const duet_model* m, int32_t n, int32_t* cus, double* flops_per_s, double* bytes_per_s) {
  if (!m || !cus || !flops_per_s || !bytes_per_s) return fail(DUET_EINVAL, "NULL argument");
  if (n != kNumCuSteps) return fail(DUET_EINVAL, "expected %d table entries", kNumCuSteps);
  for (int i = 0; i < n; ++i) {
    cus[i] = DUET_CU_STEP * (i + 1);
    flops_per_s[i] = m->flops[i];
    bytes_per_s[i] = m->bytes[i];
  }
  return DUET_OK;
}

int duet_model_set_launch_tables(duet_model* m, int32_t n, const int32_t* cus, const double* prefill_s,
                                 const double* decode_s) {
  if (!m || !cus || !prefill_s || !decode_s) return fail(DUET_EINVAL, "NULL argument");
  if (n != kNumCuSteps) return fail(DUET_EINVAL, "expected %d table entries, got %d", kNumCuSteps, n);
  for (int i = 0; i < n; ++i) {
    if (cus[i] != DUET_CU_STEP * (i + 1))
      return fail(DUET_EINVAL, "cus[%d] = %d, expected %d", i, cus[i], DUET_CU_STEP * (i + 1));
    if (!(prefill_s[i] >= 0) || !(decode_s[i] >= 0) || !std::isfinite(prefill_s[i]) || !std::isfinite(decode_s[i]))
      return fail(DUET_EINVAL, "launch table entry %d not finite and >= 0", i);
  }
  for (int i = 0; i < n; ++i) {
    m->launch_prefill[i] = prefill_s[i];
    m->launch_decode[i] = decode_s[i];
  }
  return DUET_OK;
}

int duet_model_get_launch_tables(const duet_model* m, int32_t n, int32_t* cus, double* prefill_s, double* decode_s) {
  if (!m || !cus || !prefill_s || !decode_s) return fail(DUET_EINVAL, "NULL argument");
  if (n != kNumCuSteps) return fail(DUET_EINVAL, "expected %d table entries", kNumCuSteps);
  for (int i = 0; i < n; ++i) {
    cus[i] = DUET_CU_STEP * (i + 1);
    prefill_s[i] = m->launch_prefill[i];
    decode_s[i] = m->launch_decode[i];
  }
  return DUET_OK;
}

int duet_model_set_efficiency(duet_model* m, double prefill_eff, double decode_eff) {
  if (!m) return fail(DUET_EINVAL, "model is NULL");
  if (!(prefill_eff > 0 && prefill_eff <= 1) || !(decode_eff > 0 && decode_eff <= 1))
    return fail(DUET_EINVAL, "efficiencies must lie in (0, 1]");
  m->prefill_eff = prefill_eff;
  m->decode_eff = decode_eff;
  return DUET_OK;
}

int duet_model_save(const duet_model* m, const char* path) {
  if (!m || !path) return fail(DUET_EINVAL, "NULL argument");
  FILE* f = std::fopen(path, "w");
  if (!f) return fail(DUET_EIO, "cannot open %s for writing", path);
  std::fprintf(f, "{\"version\": 3, \"calibrated\": %d, \"prefill_eff\": %.17g, \"decode_eff\": %.17g,\n",
               m->calibrated ? 1 : 0, m->prefill_eff, m->decode_eff);
  const char* names[7] = {"cus", "flops_per_s", "bytes_per_s", "launch_prefill_s", "launch_decode_s",
                          "shared_flops_per_s", "shared_bytes_per_s"};
  const double* tabs[7] = {nullptr, m->flops, m->bytes, m->launch_prefill, m->launch_decode, m->flops_shared,
                           m->bytes_shared};
  const int n_arrays = m->has_shared ? 7 : 5;
  for (int k = 0; k < n_arrays; ++k) {
    std::fprintf(f, " \"%s\": [", names[k]);
    for (int i = 0; i < kNumCuSteps; ++i) {
      if (k == 0) std::fprintf(f, "%d", DUET_CU_STEP * (i + 1));
      else std::fprintf(f, "%.17g", tabs[k][i]);
      std::fprintf(f, i + 1 < kNumCuSteps ? ", " : "]");
    }
    std::fprintf(f, k + 1 < n_arrays ? ",\n" : "}\n");
  }
  const bool ok = std::fclose(f) == 0;
  return ok ? DUET_OK : fail(DUET_EIO, "write to %s failed", path);
}

namespace {
// Minimal reader for the file written above: finds "key" and parses a number or a number array.
bool find_key(const std::string& s, const char* key, size_t* pos) {
  const std::string k = std::string("\"") + key + "\"";
  size_t p = s.find(k);
  if (p == std::string::npos) return false;
  p = s.find(':', p + k.size());
  if (p == std::string::npos) return false;
  *pos = p + 1;
  return true;
}

bool read_number(const std::string& s, const char* key, double* v) {
  size_t p;
  if (!find_key(s, key, &p)) return false;
  const char* c = s.c_str() + p;
  char* end = nullptr;
  errno = 0;
  *v = std::strtod(c, &end);
  return end != c && errno == 0;
}

bool read_array(const std::string& s, const char* key, std::vector<double>* out) {
  size_t p;
  if (!find_key(s, key, &p)) return false;
  p = s.find('[', p);
  if (p == std::string::npos) return false;
  const size_t e = s.find(']', p);
  if (e == std::string::npos) return false;
  const char* c = s.c_str() + p + 1;
  const char* stop = s.c_str() + e;
  out->clear();
  while (c < stop) {
    while (c < stop && (*c == ' ' || *c == ',' || *c == '\n')) ++c;
    if (c >= stop) break;
    char* end = nullptr;
    const double v = std::strtod(c, &end);
    if (end == c) return false;
    out->push_back(v);
    c = end;
  }
  return true;
}
}  // namespace

int duet_model_load(duet_model* m, const char* path) {
  if (!m || !path) return fail(DUET_EINVAL, "NULL argument");
  FILE* f = std::fopen(path, "r");
  if (!f) return fail(DUET_EIO, "cannot open %s", path);
  std::string s;
  char buf[4096];
  size_t n;
  while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) s.append(buf, n);
  std::fclose(f);
  std::vector<double> cus, fl, by;
  double pe = 1.0, de = 1.0, cal = 1.0;
  if (!read_array(s, "cus", &cus) || !read_array(s, "flops_per_s", &fl) || !read_array(s, "bytes_per_s", &by))
    return fail(DUET_EIO, "%s: missing tables", path);
  read_number(s, "prefill_eff", &pe);
  read_number(s, "decode_eff", &de);
  read_number(s, "calibrated", &cal);
  if ((int)cus.size() != kNumCuSteps || fl.size() != cus.size() || by.size() != cus.size())
    return fail(DUET_EIO, "%s: tables must hold %d entries", path, kNumCuSteps);
  std::vector<int32_t> ci(cus.begin(), cus.end());
  duet_model tmp = *m;
  int rc = duet_model_set_tables(&tmp, kNumCuSteps, ci.data(), fl.data(), by.data());
  if (rc) return rc;
  std::vector<double> sfl, sby;
  if (read_array(s, "shared_flops_per_s", &sfl) && read_array(s, "shared_bytes_per_s", &sby)) {
    if (sfl.size() != cus.size() || sby.size() != cus.size())
      return fail(DUET_EIO, "%s: sharing tables must hold %d entries", path, kNumCuSteps);
    if ((rc = duet_model_set_sharing_tables(&tmp, kNumCuSteps, ci.data(), sfl.data(), sby.data()))) return rc;
  }
  std::vector<double> lp, ld;
  if (read_array(s, "launch_prefill_s", &lp) && read_array(s, "launch_decode_s", &ld)) {
    if (lp.size() != cus.size() || ld.size() != cus.size())
      return fail(DUET_EIO, "%s: launch tables must hold %d entries", path, kNumCuSteps);
    if ((rc = duet_model_set_launch_tables(&tmp, kNumCuSteps, ci.data(), lp.data(), ld.data()))) return rc;
  }
  rc = duet_model_set_efficiency(&tmp, pe, de);
  if (rc) return rc;
  tmp.calibrated = cal != 0.0;
  *m = tmp;
  return DUET_OK;
}

namespace {
int check_block(const duet_block_shape* blk) {
  if (!blk) return fail(DUET_EINVAL, "block is NULL");
  if (blk->ffn_dim < 1) return fail(DUET_EINVAL, "ffn_dim %d must be >= 1", blk->ffn_dim);
  if (blk->vocab_size < 0) return fail(DUET_EINVAL, "vocab_size %d must be >= 0", blk->vocab_size);
  if (blk->flags & ~(DUET_BLOCK_GQA_QKV | DUET_BLOCK_FUSED_GATE_UP))
    return fail(DUET_EINVAL, "unknown block flags 0x%x", (unsigned)blk->flags);
  return DUET_OK;
}

int predict_impl(const duet_model* m, const duet_shape* shape, const duet_block_shape* blk, const duet_batch* batch,
                 duet_cu_split split, double* us) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if (!us) return fail(DUET_EINVAL, "us is NULL");
  if (!check_split(split)) return fail(DUET_EINVAL, "invalid CU split");
  duet_model nominal;
  const duet_model* mm = model_or_nominal(m, &nominal);
  double t;
  if (split.mode == DUET_AGG) {
    t = f_roofline(mm, shape, batch, -1, DUET_TOTAL_CUS, false, blk);
  } else {
    const bool shared = has_both_kinds(batch);
    const double td = f_roofline(mm, shape, batch, DUET_KIND_DECODE, split.cus_decode, shared, blk);
    const double tp = f_roofline(mm, shape, batch, DUET_KIND_PREFILL, split.cus_prefill, shared, blk);
    t = std::fmax(split.k_decode_steps * td, tp);
  }
  *us = t * 1e6;
  return DUET_OK;
}

int choose_impl(const duet_model* m, const duet_shape* shape, const duet_block_shape* blk, const duet_batch* batch,
                double tbt_slo_us, int32_t max_decode_steps, duet_cu_split* out, double* predicted_us, double* rho,
                int32_t* status_flags) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if (!out) return fail(DUET_EINVAL, "out is NULL");
  if (!(tbt_slo_us > 0) || !std::isfinite(tbt_slo_us)) return fail(DUET_EINVAL, "tbt_slo_us must be > 0");
  duet_model nominal;
  const duet_model* mm = model_or_nominal(m, &nominal);
  const double tau = tbt_slo_us * 1e-6;
  int32_t flags = mm->calibrated ? 0 : DUET_STATUS_UNCALIBRATED;

  const double t_mixed = f_roofline(mm, shape, batch, -1, DUET_TOTAL_CUS, false, blk);
  duet_cu_split agg{DUET_AGG, DUET_TOTAL_CUS, 0, 1};
  if (t_mixed <= tau) {
    *out = agg;
    if (predicted_us) *predicted_us = t_mixed * 1e6;
    if (rho) *rho = 0.0;
    if (status_flags) *status_flags = flags;
    return DUET_OK;
  }
  double t_decode_tokens = 0.0, t_prefill_tokens = 0.0;
  for (int r = 0; r < batch->num_reqs; ++r) {
    if (batch->reqs[r].kind == DUET_KIND_DECODE) t_decode_tokens += 1.0;
    else t_prefill_tokens += batch->reqs[r].q_len;
  }
  double best_rho = 0.0, best_t = 0.0;
  duet_cu_split best{-1, 0, 0, 0};
  const bool shared = has_both_kinds(batch);
  for (int sd = DUET_SPLIT_STEP; sd < DUET_TOTAL_CUS; sd += DUET_SPLIT_STEP) {
    const double td = f_roofline(mm, shape, batch, DUET_KIND_DECODE, sd, shared, blk);
    if (td > tau) continue;
    const int sp = DUET_TOTAL_CUS - sd;
    const double tp = f_roofline(mm, shape, batch, DUET_KIND_PREFILL, sp, shared, blk);
    const double base = td > 0.0 ? std::floor(tp / td) : 1.0;
    // rho(k) rises up to k = base and falls from base + 1 on: under a cap on the decode steps
    // the candidates are clamped to it (the second is skipped when both clamp to the cap).
    for (int j = 0; j < 2; ++j) {
      double k = base + j;
      if (max_decode_steps > 0 && k > max_decode_steps) {
        if (j == 1 && base >= max_decode_steps) continue;
        k = max_decode_steps;
      }
      if (k < 1.0 || k > 1e9) continue;
      const double t = std::fmax(k * td, tp);
      const double r = (k * t_decode_tokens + t_prefill_tokens) / t;
      if (r > best_rho) {
        best_rho = r;
        best_t = t;
        best = duet_cu_split{DUET_SPLIT, sp, sd, (int32_t)k};
      }
    }
  }
  if (best.mode != DUET_SPLIT) {
    *out = agg;
    if (predicted_us) *predicted_us = t_mixed * 1e6;
    if (rho) *rho = 0.0;
    if (status_flags) *status_flags = flags | DUET_STATUS_SLO_INFEASIBLE;
    return DUET_OK;
  }
  *out = best;
  if (predicted_us) *predicted_us = best_t * 1e6;
  if (rho) *rho = best_rho;
  if (status_flags) *status_flags = flags;
  return DUET_OK;
}

}  // namespace

int duet_predict_iter_latency(const duet_model* m, const duet_shape* shape, const duet_batch* batch,
                              duet_cu_split split, double* us) {
  return predict_impl(m, shape, nullptr, batch, split, us);
}

int duet_predict_partition_latency(const duet_model* m, const duet_shape* shape, const duet_batch* batch,
                                   int32_t kind, int32_t cus, int32_t shared, double* us) {
  clear_error();
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_batch(shape, batch, false))) return rc;
  if (!us) return fail(DUET_EINVAL, "us is NULL");
  if (kind != DUET_KIND_PREFILL && kind != DUET_KIND_DECODE) return fail(DUET_EINVAL, "kind %d", kind);
  if (cus < DUET_CU_STEP || cus > DUET_TOTAL_CUS || cus % DUET_CU_STEP)
    return fail(DUET_EINVAL, "cus %d must be a multiple of %d in [%d, %d]", cus, DUET_CU_STEP, DUET_CU_STEP,
                DUET_TOTAL_CUS);
  duet_model nominal;
  const duet_model* mm = model_or_nominal(m, &nominal);
  *us = f_roofline(mm, shape, batch, kind, cus, shared != 0 && has_both_kinds(batch), nullptr) * 1e6;
  return DUET_OK;
}

int duet_choose_cu_split(const duet_model* m, const duet_shape* shape, const duet_batch* batch,
                         double tbt_slo_us, int32_t max_decode_steps, duet_cu_split* out,
                         double* predicted_us, double* rho, int32_t* status_flags) {
  return choose_impl(m, shape, nullptr, batch, tbt_slo_us, max_decode_steps, out, predicted_us, rho, status_flags);
}

int duet_predict_model_latency(const duet_model* m, const duet_shape* shape, const duet_block_shape* block,
                               const duet_batch* batch, duet_cu_split split, double* us) {
  clear_error();
  const int rc = check_block(block);
  return rc ? rc : predict_impl(m, shape, block, batch, split, us);
}

int duet_choose_cu_split_model(const duet_model* m, const duet_shape* shape, const duet_block_shape* block,
                               const duet_batch* batch, double tbt_slo_us, int32_t max_decode_steps,
                               duet_cu_split* out, double* predicted_us, double* rho, int32_t* status_flags) {
  clear_error();
  const int rc = check_block(block);
  return rc ? rc : choose_impl(m, shape, block, batch, tbt_slo_us, max_decode_steps, out, predicted_us, rho,
                               status_flags);
}

}  // extern "C"
