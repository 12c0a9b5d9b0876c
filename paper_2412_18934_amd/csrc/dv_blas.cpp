// Plain GEMMs of the large-M prefill through hipBLASLt.
//
// Every prefill projection is D = B A^T with A the weight matrix [m][k]
// (row-major bf16, the caller's own layout), B the activations [n][k] (the
// bf16 hi rows of the tokens followed by their lo rows) and D [n][m] fp32.
// In hipBLASLt's column-major terms that is D^T (m x n) = op_T(A^T) B^T with
// both operands k-contiguous ("TN").  Descriptors, layouts and the chosen
// algorithm are cached per (m, n, k, ldb); the first algorithm of the heuristic is
// used, so a shape always runs the same kernel.
#include <hip/hip_runtime_api.h>
#include <hipblaslt/hipblaslt.h>

#include <map>
#include <tuple>

#include "dv_internal.h"

struct BlasCtx {
    hipblasLtHandle_t lt = nullptr;
    void *ws = nullptr;
    size_t ws_bytes = 0;
    struct Plan {
        hipblasLtMatmulDesc_t desc = nullptr;
        hipblasLtMatrixLayout_t a = nullptr, b = nullptr, d = nullptr;
        hipblasLtMatmulAlgo_t algo;
        bool ok = false;
    };
    std::map<std::tuple<int, int, int, int>, Plan> plans;
};

namespace {

constexpr size_t kWorkspace = 64u << 20;

BlasCtx::Plan *get_plan(BlasCtx *c, int m, int n, int k, int ldb)
{
    auto key = std::make_tuple(m, n, k, ldb);
    auto it = c->plans.find(key);
    if (it != c->plans.end()) return it->second.ok ? &it->second : nullptr;
    BlasCtx::Plan &p = c->plans[key];
    const hipblasOperation_t opT = HIPBLAS_OP_T, opN = HIPBLAS_OP_N;
    if (hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS) return nullptr;
    hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opT, sizeof opT);
    hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opN, sizeof opN);
    // A^T stored k x m (ld k), B^T stored k x n (ld ldb), D^T m x n (ld m)
    if (hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, k, m, k) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutCreate(&p.b, HIP_R_16BF, k, n, ldb) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutCreate(&p.d, HIP_R_32F, m, n, m) != HIPBLAS_STATUS_SUCCESS)
        return nullptr;
    hipblasLtMatmulPreference_t pref = nullptr;
    if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS) return nullptr;
    const uint64_t wsb = c->ws_bytes;
    hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsb, sizeof wsb);
    hipblasLtMatmulHeuristicResult_t res[1];
    int found = 0;
    const hipblasStatus_t st =
        hipblasLtMatmulAlgoGetHeuristic(c->lt, p.desc, p.a, p.b, p.d, p.d, pref, 1, res, &found);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (st != HIPBLAS_STATUS_SUCCESS || found < 1 || res[0].workspaceSize > c->ws_bytes) return nullptr;
    p.algo = res[0].algo;
    p.ok = true;
    return &p;
}

}  // namespace

BlasCtx *blas_create()
{
    BlasCtx *c = new BlasCtx;
    if (hipblasLtCreate(&c->lt) != HIPBLAS_STATUS_SUCCESS || hipMalloc(&c->ws, kWorkspace) != hipSuccess) {
        blas_destroy(c);
        return nullptr;
    }
    c->ws_bytes = kWorkspace;
    return c;
}

void blas_destroy(BlasCtx *c)
{
    if (!c) return;
    for (auto &kv : c->plans) {
        BlasCtx::Plan &p = kv.second;
        if (p.a) hipblasLtMatrixLayoutDestroy(p.a);
        if (p.b) hipblasLtMatrixLayoutDestroy(p.b);
        if (p.d) hipblasLtMatrixLayoutDestroy(p.d);
        if (p.desc) hipblasLtMatmulDescDestroy(p.desc);
    }
    if (c->ws) (void)hipFree(c->ws);
    if (c->lt) hipblasLtDestroy(c->lt);
    delete c;
}

int blas_gemm_tn(BlasCtx *c, int m, int n, int k, const uint16_t *A, const uint16_t *B, int ldb, float *D,
                 hipStream_t s)
{
    BlasCtx::Plan *p = get_plan(c, m, n, k, ldb);
    if (!p) return -1;
    const float alpha = 1.f, beta = 0.f;
    const hipblasStatus_t st = hipblasLtMatmul(c->lt, p->desc, &alpha, A, p->a, B, p->b, &beta, D, p->d, D, p->d,
                                               &p->algo, c->ws, c->ws_bytes, s);
    return st == HIPBLAS_STATUS_SUCCESS ? 0 : -1;
}
