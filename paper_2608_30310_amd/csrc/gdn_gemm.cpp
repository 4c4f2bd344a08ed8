// hipBLASLt-backed projections for the layer block (interface in gdn_gemm.h).
#include "gdn_gemm.h"

#include <hipblaslt/hipblaslt.h>

#include <map>
#include <memory>
#include <mutex>
#include <tuple>

namespace gdn {
namespace {

struct Problem {
  int device;
  int64_t m, n, k, lda, ldb, ldd;
  int32_t d_dtype;
  size_t ws_cap;
  bool operator<(const Problem& o) const {
    return std::tie(device, m, n, k, lda, ldb, ldd, d_dtype, ws_cap) <
           std::tie(o.device, o.m, o.n, o.k, o.lda, o.ldb, o.ldd, o.d_dtype, o.ws_cap);
  }
};

// Descriptors and the chosen algorithm for one problem; built once, then only
// read (by any number of threads), destroyed with the last reference.
struct Prepared {
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, ld = nullptr;
  hipblasLtMatmulAlgo_t algo{};
  size_t ws = 0;
  ~Prepared() {
    if (ld) hipblasLtMatrixLayoutDestroy(ld);
    if (lb) hipblasLtMatrixLayoutDestroy(lb);
    if (la) hipblasLtMatrixLayoutDestroy(la);
    if (desc) hipblasLtMatmulDescDestroy(desc);
  }
};

// A serving process sees many token counts; past this many problems new ones
// are prepared per call instead of cached.
constexpr size_t kMaxCached = 512;

std::mutex g_mutex;
std::map<int, hipblasLtHandle_t> g_handles;
std::map<Problem, std::shared_ptr<const Prepared>> g_prepared;

gdn_status lt_fail(std::string* err, const char* what, hipblasStatus_t s) {
  *err = std::string("hipBLASLt ") + what + " failed (status " + std::to_string(static_cast<int>(s)) + ")";
  return GDN_ERR_HIP;
}

#define LT_CHECK(call, what)                                         \
  do {                                                               \
    const hipblasStatus_t s_ = (call);                               \
    if (s_ != HIPBLAS_STATUS_SUCCESS) return lt_fail(err, what, s_); \
  } while (0)

gdn_status handle_for(int device, hipblasLtHandle_t* h, std::string* err) {
  auto it = g_handles.find(device);
  if (it != g_handles.end()) { *h = it->second; return GDN_OK; }
  hipblasLtHandle_t nh = nullptr;
  LT_CHECK(hipblasLtCreate(&nh), "handle creation");
  g_handles[device] = nh;
  *h = nh;
  return GDN_OK;
}

gdn_status prepare(hipblasLtHandle_t h, const Problem& p, std::shared_ptr<const Prepared>* out,
                   std::string* err) {
  auto r = std::make_shared<Prepared>();   // releases whatever was created on any early return
  const hipDataType dt = p.d_dtype == GDN_F32 ? HIP_R_32F : HIP_R_16BF;
  LT_CHECK(hipblasLtMatmulDescCreate(&r->desc, HIPBLAS_COMPUTE_32F, HIP_R_32F), "matmul descriptor");
  const hipblasOperation_t opT = HIPBLAS_OP_T, opN = HIPBLAS_OP_N;
  LT_CHECK(hipblasLtMatmulDescSetAttribute(r->desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opT, sizeof(opT)), "transa");
  LT_CHECK(hipblasLtMatmulDescSetAttribute(r->desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opN, sizeof(opN)), "transb");
  // column-major views: A^T stored k x m (ld lda), B^T k x n (ld ldb), D^T m x n (ld ldd)
  LT_CHECK(hipblasLtMatrixLayoutCreate(&r->la, HIP_R_16BF, p.k, p.m, p.lda), "layout A");
  LT_CHECK(hipblasLtMatrixLayoutCreate(&r->lb, HIP_R_16BF, p.k, p.n, p.ldb), "layout B");
  LT_CHECK(hipblasLtMatrixLayoutCreate(&r->ld, dt, p.m, p.n, p.ldd), "layout D");
  hipblasLtMatmulPreference_t pref = nullptr;
  LT_CHECK(hipblasLtMatmulPreferenceCreate(&pref), "preference");
  const uint64_t cap = p.ws_cap;
  hipblasStatus_t s = hipblasLtMatmulPreferenceSetAttribute(
      pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &cap, sizeof(cap));
  hipblasLtMatmulHeuristicResult_t res[8];
  int found = 0;
  if (s == HIPBLAS_STATUS_SUCCESS)
    s = hipblasLtMatmulAlgoGetHeuristic(h, r->desc, r->la, r->lb, r->ld, r->ld, pref, 8, res, &found);
  hipblasLtMatmulPreferenceDestroy(pref);
  if (s != HIPBLAS_STATUS_SUCCESS) return lt_fail(err, "heuristic query", s);
  for (int i = 0; i < found; ++i) {
    if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= p.ws_cap) {
      r->algo = res[i].algo;
      r->ws = res[i].workspaceSize;
      *out = std::move(r);
      return GDN_OK;
    }
  }
  *err = "hipBLASLt offers no algorithm for a " + std::to_string(p.m) + " x " + std::to_string(p.n) +
         " x " + std::to_string(p.k) + " bf16 projection";
  return GDN_ERR_HIP;
}

}  // namespace

gdn_status gemm_tn(int64_t m, int64_t n, int64_t k, const void* a, int64_t lda, const void* b,
                   int64_t ldb, void* d, int64_t ldd, int32_t d_dtype, void* workspace,
                   size_t workspace_bytes, hipStream_t stream, std::string* err) {
  if (m == 0 || n == 0) return GDN_OK;
  int device = 0;
  const hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) { *err = std::string("hipGetDevice: ") + hipGetErrorString(e); return GDN_ERR_HIP; }
  const Problem p{device, m, n, k, lda, ldb, ldd, d_dtype, workspace_bytes};
  hipblasLtHandle_t h = nullptr;
  std::shared_ptr<const Prepared> prep;
  {
    std::lock_guard<std::mutex> lock(g_mutex);
    gdn_status st = handle_for(device, &h, err);
    if (st != GDN_OK) return st;
    auto it = g_prepared.find(p);
    if (it != g_prepared.end()) {
      prep = it->second;
    } else {
      st = prepare(h, p, &prep, err);
      if (st != GDN_OK) return st;
      if (g_prepared.size() < kMaxCached) g_prepared[p] = prep;
    }
  }
  const float alpha = 1.0f, beta = 0.0f;
  LT_CHECK(hipblasLtMatmul(h, prep->desc, &alpha, a, prep->la, b, prep->lb, &beta, d, prep->ld, d, prep->ld,
                           &prep->algo, prep->ws ? workspace : nullptr, prep->ws, stream),
           "matmul");
  return GDN_OK;
}

}  // namespace gdn
