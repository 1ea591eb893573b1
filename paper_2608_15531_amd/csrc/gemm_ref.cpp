// bf16 GEMM comparator on hipBLASLt: the C ABI of include/fq_gemm_ref.h.
//
// Row-major Y[M][N] = X[M][K] * W is handed to hipBLASLt, which is
// column-major, as the column-major product Y^T (N x M) = W^T (N x K) * X^T
// (K x M): a row-major matrix read column-major is its transpose, so no data
// moves.  A = W (op N for the [K][N] layout, op T for [N][K]), B = X, C = D = Y.

#include "fq_gemm_ref.h"

#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt-ext.hpp>
#include <hipblaslt/hipblaslt.h>

#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

namespace {

enum : int { kOk = 0, kBadArg = 1, kNotPrepared = 2, kLibFail = 3 };

thread_local std::string t_error;

int fail(int code, const std::string& what) {
  t_error = what;
  return code;
}

struct Problem {
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
  std::vector<hipblasLtMatmulHeuristicResult_t> cands;
  ~Problem() {
    if (a) hipblasLtMatrixLayoutDestroy(a);
    if (b) hipblasLtMatrixLayoutDestroy(b);
    if (c) hipblasLtMatrixLayoutDestroy(c);
    if (desc) hipblasLtMatmulDescDestroy(desc);
  }
};

using Key = std::tuple<int, int32_t, int32_t, int32_t, int32_t>;

std::mutex g_mu;
std::map<int, hipblasLtHandle_t> g_handles;             // one handle per device
std::map<Key, std::shared_ptr<Problem>> g_problems;

const float kAlpha = 1.0f, kBeta = 0.0f;

bool shape_ok(int32_t M, int32_t K, int32_t N, int32_t layout) {
  const int32_t lim = 1 << 20;
  return M >= 1 && K >= 1 && N >= 1 && M <= lim && K <= lim && N <= lim &&
         (layout == FQ_REF_W_KN || layout == FQ_REF_W_NK);
}

int current_device(int* dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return fail(kLibFail, std::string("hipGetDevice: ") + hipGetErrorString(e));
  return kOk;
}

// handle of the current device (created on first use); caller holds g_mu
int handle_for(int dev, hipblasLtHandle_t* h) {
  auto it = g_handles.find(dev);
  if (it != g_handles.end()) {
    *h = it->second;
    return kOk;
  }
  hipblasStatus_t s = hipblasLtCreate(h);
  if (s != HIPBLAS_STATUS_SUCCESS) return fail(kLibFail, "hipblasLtCreate failed: " + std::to_string(int(s)));
  g_handles[dev] = *h;
  return kOk;
}

#define LT_CHECK(call)                                                              \
  do {                                                                              \
    hipblasStatus_t s_ = (call);                                                    \
    if (s_ != HIPBLAS_STATUS_SUCCESS)                                               \
      return fail(kLibFail, std::string(#call) + " failed: " + std::to_string(int(s_))); \
  } while (0)

int build_descriptors(Problem& p, int32_t M, int32_t K, int32_t N, int32_t layout) {
  const hipblasOperation_t op_a = layout == FQ_REF_W_KN ? HIPBLAS_OP_N : HIPBLAS_OP_T;
  const hipblasOperation_t op_b = HIPBLAS_OP_N;
  LT_CHECK(hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F));
  LT_CHECK(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &op_a, sizeof(op_a)));
  LT_CHECK(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &op_b, sizeof(op_b)));
  if (layout == FQ_REF_W_KN)
    LT_CHECK(hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, uint64_t(N), uint64_t(K), int64_t(N)));
  else
    LT_CHECK(hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, uint64_t(K), uint64_t(N), int64_t(K)));
  LT_CHECK(hipblasLtMatrixLayoutCreate(&p.b, HIP_R_16BF, uint64_t(K), uint64_t(M), int64_t(K)));
  LT_CHECK(hipblasLtMatrixLayoutCreate(&p.c, HIP_R_16BF, uint64_t(N), uint64_t(M), int64_t(N)));
  return kOk;
}

int heuristic(hipblasLtHandle_t h, Problem& p, int32_t max_c, uint64_t max_ws) {
  hipblasLtMatmulPreference_t pref = nullptr;
  LT_CHECK(hipblasLtMatmulPreferenceCreate(&pref));
  std::unique_ptr<std::remove_pointer<hipblasLtMatmulPreference_t>::type,
                  hipblasStatus_t (*)(hipblasLtMatmulPreference_t)>
      guard(pref, hipblasLtMatmulPreferenceDestroy);
  LT_CHECK(hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES,
                                                 &max_ws, sizeof(max_ws)));
  std::vector<hipblasLtMatmulHeuristicResult_t> res(max_c);
  int got = 0;
  LT_CHECK(hipblasLtMatmulAlgoGetHeuristic(h, p.desc, p.a, p.b, p.c, p.c, pref, max_c, res.data(), &got));
  for (int i = 0; i < got; ++i)
    if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= max_ws) p.cands.push_back(res[i]);
  return kOk;
}

int exhaustive(hipblasLtHandle_t h, Problem& p, int32_t layout, int32_t max_c, uint64_t max_ws) {
  const hipblasOperation_t op_a = layout == FQ_REF_W_KN ? HIPBLAS_OP_N : HIPBLAS_OP_T;
  std::vector<hipblasLtMatmulHeuristicResult_t> all;
  LT_CHECK(hipblaslt_ext::getAllAlgos(h, hipblaslt_ext::GemmType::HIPBLASLT_GEMM, op_a, HIPBLAS_OP_N,
                                      HIP_R_16BF, HIP_R_16BF, HIP_R_16BF, HIP_R_16BF,
                                      HIPBLAS_COMPUTE_32F, all));
  for (auto& r : all) {
    if (int32_t(p.cands.size()) >= max_c) break;
    size_t ws = 0;
    if (hipblaslt_ext::matmulIsAlgoSupported(h, p.desc, &kAlpha, p.a, p.b, &kBeta, p.c, p.c, r.algo, ws) !=
        HIPBLAS_STATUS_SUCCESS)
      continue;
    if (ws > max_ws) continue;
    hipblasLtMatmulHeuristicResult_t c = r;
    c.workspaceSize = ws;
    c.state = HIPBLAS_STATUS_SUCCESS;
    p.cands.push_back(c);
  }
  return kOk;
}

// the problem of the current device, or nullptr; caller holds g_mu
std::shared_ptr<Problem> find_problem(int dev, int32_t M, int32_t K, int32_t N, int32_t layout) {
  auto it = g_problems.find(Key{dev, M, K, N, layout});
  return it == g_problems.end() ? nullptr : it->second;
}

}  // namespace

extern "C" {

int fq_ref_gemm_bf16_prepare(int32_t M, int32_t K, int32_t N, int32_t layout, int32_t source,
                             int32_t max_candidates, uint64_t max_workspace,
                             int32_t* n_candidates) {
  t_error.clear();
  if (!shape_ok(M, K, N, layout)) return fail(kBadArg, "shape or layout out of range");
  if (source != FQ_REF_HEURISTIC && source != FQ_REF_EXHAUSTIVE) return fail(kBadArg, "unknown source");
  if (max_candidates < 1 || max_candidates > 4096) return fail(kBadArg, "max_candidates out of range");
  if (!n_candidates) return fail(kBadArg, "n_candidates is NULL");
  int dev = 0;
  if (int rc = current_device(&dev)) return rc;
  std::lock_guard<std::mutex> lk(g_mu);
  hipblasLtHandle_t h = nullptr;
  if (int rc = handle_for(dev, &h)) return rc;
  auto p = std::make_shared<Problem>();
  if (int rc = build_descriptors(*p, M, K, N, layout)) return rc;
  int rc = source == FQ_REF_HEURISTIC ? heuristic(h, *p, max_candidates, max_workspace)
                                      : exhaustive(h, *p, layout, max_candidates, max_workspace);
  if (rc) return rc;
  if (p->cands.empty()) return fail(kLibFail, "hipBLASLt offers no algorithm for this problem");
  g_problems[Key{dev, M, K, N, layout}] = p;
  *n_candidates = int32_t(p->cands.size());
  return kOk;
}

int fq_ref_gemm_bf16_candidate(int32_t M, int32_t K, int32_t N, int32_t layout,
                               int32_t candidate, uint64_t* workspace_bytes, char* name,
                               size_t name_len) {
  t_error.clear();
  if (!shape_ok(M, K, N, layout)) return fail(kBadArg, "shape or layout out of range");
  int dev = 0;
  if (int rc = current_device(&dev)) return rc;
  std::lock_guard<std::mutex> lk(g_mu);
  auto p = find_problem(dev, M, K, N, layout);
  if (!p) return fail(kNotPrepared, "problem not prepared on this device");
  if (candidate < 0 || candidate >= int32_t(p->cands.size()))
    return fail(kNotPrepared, "candidate index out of range");
  auto& c = p->cands[candidate];
  if (workspace_bytes) *workspace_bytes = c.workspaceSize;
  if (name && name_len > 0) {
    const std::string s = hipblaslt_ext::getKernelNameFromAlgo(g_handles[dev], c.algo);
    const size_t n = s.size() < name_len - 1 ? s.size() : name_len - 1;
    std::memcpy(name, s.data(), n);
    name[n] = '\0';
  }
  return kOk;
}

int fq_ref_gemm_bf16(const void* X, const void* W, void* Y, int32_t M, int32_t K, int32_t N,
                     int32_t layout, int32_t candidate, void* workspace,
                     uint64_t workspace_bytes, void* stream) {
  t_error.clear();
  if (!shape_ok(M, K, N, layout)) return fail(kBadArg, "shape or layout out of range");
  if (!X || !W || !Y) return fail(kBadArg, "X, W and Y must be device pointers");
  int dev = 0;
  if (int rc = current_device(&dev)) return rc;
  std::shared_ptr<Problem> p;
  hipblasLtHandle_t h = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    p = find_problem(dev, M, K, N, layout);
    h = g_handles.count(dev) ? g_handles[dev] : nullptr;
  }
  if (!p || !h) return fail(kNotPrepared, "problem not prepared on this device");
  if (candidate < 0 || candidate >= int32_t(p->cands.size()))
    return fail(kNotPrepared, "candidate index out of range");
  const auto& c = p->cands[candidate];
  if (c.workspaceSize > 0 && (!workspace || workspace_bytes < c.workspaceSize))
    return fail(kBadArg, "workspace smaller than the candidate needs (" + std::to_string(c.workspaceSize) +
                             " bytes)");
  LT_CHECK(hipblasLtMatmul(h, p->desc, &kAlpha, W, p->a, X, p->b, &kBeta, Y, p->c, Y, p->c, &c.algo,
                           workspace, c.workspaceSize, hipStream_t(stream)));
  return kOk;
}

const char* fq_ref_gemm_last_error(void) { return t_error.c_str(); }

}  // extern "C"
