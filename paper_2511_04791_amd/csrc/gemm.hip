// bf16 GEMMs on hipBLASLt for the token-level operators (paper, Section 4.1: linear operators
// n x d_in by d_in x d_out).  hipBLASLt is column-major: the row-major product
// y[n, d_out] = x[n, d_in] w[d_in, d_out] is the column-major y^T = w^T x^T, i.e. A = w viewed as
// [d_out x d_in] (ld d_out), B = x viewed as [d_in x n] (ld d_in), C = D = y viewed as
// [d_out x n] (ld d_out), no transposes.  Each problem shape is planned once (heuristic query)
// and its algorithm reused.
#include "gemm.h"

#include <hipblaslt/hipblaslt.h>

#include <map>
#include <tuple>

namespace duet {

struct GemmPlan {
  hipblasLtMatmulDesc_t op = nullptr;
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
  hipblasLtMatmulAlgo_t algo{};
};

struct GemmCache {
  hipblasLtHandle_t handle = nullptr;
  std::map<std::tuple<int, int, int>, GemmPlan> plans;  // (n, d_in, d_out)
};

GemmCache* gemm_cache_create() {
  GemmCache* c = new (std::nothrow) GemmCache;
  if (!c) return nullptr;
  if (hipblasLtCreate(&c->handle) != HIPBLAS_STATUS_SUCCESS) {
    delete c;
    return nullptr;
  }
  return c;
}

static void destroy_plan(GemmPlan& p) {
  if (p.op) hipblasLtMatmulDescDestroy(p.op);
  if (p.a) hipblasLtMatrixLayoutDestroy(p.a);
  if (p.b) hipblasLtMatrixLayoutDestroy(p.b);
  if (p.c) hipblasLtMatrixLayoutDestroy(p.c);
}

void gemm_cache_destroy(GemmCache* c) {
  if (!c) return;
  for (auto& kv : c->plans) destroy_plan(kv.second);
  if (c->handle) hipblasLtDestroy(c->handle);
  delete c;
}

static int plan_for(GemmCache* c, int n, int d_in, int d_out, GemmPlan** out, const char** msg) {
  const auto key = std::make_tuple(n, d_in, d_out);
  auto it = c->plans.find(key);
  if (it != c->plans.end()) {
    *out = &it->second;
    return 0;
  }
  // A serving loop meets many row counts: keep the cache bounded (plans are cheap to re-make).
  constexpr size_t kMaxPlans = 512;
  if (c->plans.size() >= kMaxPlans) {
    for (auto& kv : c->plans) destroy_plan(kv.second);
    c->plans.clear();
  }
  GemmPlan p;
  const hipblasOperation_t no = HIPBLAS_OP_N;
  bool ok = hipblasLtMatmulDescCreate(&p.op, HIPBLAS_COMPUTE_32F, HIP_R_32F) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_TRANSA, &no, sizeof no) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_TRANSB, &no, sizeof no) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, d_out, d_in, d_out) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatrixLayoutCreate(&p.b, HIP_R_16BF, d_in, n, d_in) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatrixLayoutCreate(&p.c, HIP_R_16BF, d_out, n, d_out) == HIPBLAS_STATUS_SUCCESS;
  if (!ok) {
    destroy_plan(p);
    *msg = "hipBLASLt descriptor creation failed";
    return -1;
  }
  hipblasLtMatmulPreference_t pref = nullptr;
  uint64_t ws = kGemmWorkspaceBytes;
  hipblasLtMatmulHeuristicResult_t res[1];
  int found = 0;
  ok = hipblasLtMatmulPreferenceCreate(&pref) == HIPBLAS_STATUS_SUCCESS &&
       hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof ws) ==
           HIPBLAS_STATUS_SUCCESS &&
       hipblasLtMatmulAlgoGetHeuristic(c->handle, p.op, p.a, p.b, p.c, p.c, pref, 1, res, &found) ==
           HIPBLAS_STATUS_SUCCESS &&
       found > 0;
  if (pref) hipblasLtMatmulPreferenceDestroy(pref);
  if (!ok) {
    destroy_plan(p);
    *msg = "hipBLASLt found no algorithm for a bf16 GEMM of this shape";
    return -1;
  }
  p.algo = res[0].algo;
  *out = &(c->plans[key] = p);
  return 0;
}

int gemm_bf16(GemmCache* c, const void* x, const void* w, void* y, int n, int d_in, int d_out, bool accumulate,
              void* ws, hipStream_t s, const char** msg) {
  if (n <= 0) return 0;
  GemmPlan* p = nullptr;
  if (plan_for(c, n, d_in, d_out, &p, msg)) return -1;
  const float alpha = 1.0f, beta = accumulate ? 1.0f : 0.0f;
  if (hipblasLtMatmul(c->handle, p->op, &alpha, w, p->a, x, p->b, &beta, y, p->c, y, p->c, &p->algo, ws,
                      kGemmWorkspaceBytes, s) != HIPBLAS_STATUS_SUCCESS) {
    *msg = "hipblasLtMatmul failed";
    return -1;
  }
  return 0;
}

}  // namespace duet
