// The layer's Q/K/V/O projections (Algorithm 1: Q = u W_Q, ..., out = O W_O)
// are plain GEMMs and run through hipBLASLt (fp32 accumulation, 16-bit in and
// out).  C (M, N) is row-major; A is given either as (M, K) row-major ("K
// contiguous") or as (K, M) row-major, and B either as (N, K) row-major or as
// (K, N) row-major.  hipBLASLt is column-major, so the call computes
// D = C^T (N x M, leading dimension N) = B^T . A^T:
//   its matrix "A" is our B:  (N, K) row-major = K x N column-major, op T;
//                             (K, N) row-major = N x K column-major, op N;
//   its matrix "B" is our A:  (M, K) row-major = K x M column-major, op N;
//                             (K, M) row-major = M x K column-major, op T.
// Batched over `batch` with element strides sa, sb, sc (0 = shared operand).
//
// Host-side state: one hipBLASLt handle per device and one plan (descriptors
// and the heuristic's first algorithm) per shape, created on first use under a
// mutex that also serialises the enqueue.  No device memory is allocated here:
// the algorithm's workspace is a slice of the caller's workspace.
#include <hipblaslt/hipblaslt.h>

#include <map>
#include <mutex>
#include <tuple>

#include "common.h"
#include "internal.h"

namespace h3 {
namespace {

struct LtPlan {
    bool ok = false;
    hipblasLtMatmulDesc_t desc{};
    hipblasLtMatrixLayout_t la{}, lb{}, lc{};
    hipblasLtMatmulAlgo_t algo{};
    size_t ws = 0;
};

std::mutex g_lt_mu;
std::map<int, hipblasLtHandle_t> g_lt_handles;
using LtKey = std::tuple<int, int, int, int, int, int, long, long, long, size_t, bool, bool>;
std::map<LtKey, LtPlan> g_lt_plans;

bool make_plan(hipblasLtHandle_t h, hipDataType t, int M, int N, int K, bool a_kc, bool b_kc, int batch, long sa,
               long sb, long sc, size_t ws_bytes, LtPlan &p) {
    if (hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS) return false;
    const hipblasOperation_t ta = b_kc ? HIPBLAS_OP_T : HIPBLAS_OP_N;
    const hipblasOperation_t tb = a_kc ? HIPBLAS_OP_N : HIPBLAS_OP_T;
    hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof(ta));
    hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof(tb));
    const hipblasStatus_t s1 = b_kc ? hipblasLtMatrixLayoutCreate(&p.la, t, K, N, K)    // our B
                                    : hipblasLtMatrixLayoutCreate(&p.la, t, N, K, N);
    if (s1 != HIPBLAS_STATUS_SUCCESS) return false;
    const hipblasStatus_t s2 = a_kc ? hipblasLtMatrixLayoutCreate(&p.lb, t, K, M, K)    // our A
                                    : hipblasLtMatrixLayoutCreate(&p.lb, t, M, K, M);
    if (s2 != HIPBLAS_STATUS_SUCCESS) return false;
    if (hipblasLtMatrixLayoutCreate(&p.lc, t, N, M, N) != HIPBLAS_STATUS_SUCCESS) return false;   // C = D
    if (batch > 1) {
        const int32_t bc = batch;
        const int64_t s_la = sb, s_lb = sa, s_lc = sc;
        hipblasLtMatrixLayoutSetAttribute(p.la, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &bc, sizeof(bc));
        hipblasLtMatrixLayoutSetAttribute(p.lb, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &bc, sizeof(bc));
        hipblasLtMatrixLayoutSetAttribute(p.lc, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &bc, sizeof(bc));
        hipblasLtMatrixLayoutSetAttribute(p.la, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &s_la, sizeof(s_la));
        hipblasLtMatrixLayoutSetAttribute(p.lb, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &s_lb, sizeof(s_lb));
        hipblasLtMatrixLayoutSetAttribute(p.lc, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &s_lc, sizeof(s_lc));
    }
    hipblasLtMatmulPreference_t pref;
    if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS) return false;
    const uint64_t maxws = ws_bytes;
    hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &maxws, sizeof(maxws));
    hipblasLtMatmulHeuristicResult_t res[4];
    int n = 0;
    const hipblasStatus_t st =
        hipblasLtMatmulAlgoGetHeuristic(h, p.desc, p.la, p.lb, p.lc, p.lc, pref, 4, res, &n);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (st != HIPBLAS_STATUS_SUCCESS || n < 1 || res[0].state != HIPBLAS_STATUS_SUCCESS) return false;
    if (res[0].workspaceSize > ws_bytes) return false;
    p.algo = res[0].algo;
    p.ws = res[0].workspaceSize;
    return true;
}

}  // namespace

hipError_t launch_gemm_lt(const void *A, bool a_kc, const void *B, bool b_kc, void *C, int M, int N, int K, int batch,
                          long sa, long sb, long sc, int dtype, void *ws, size_t ws_bytes, hipStream_t s) {
    if (dtype != F16 && dtype != BF16) return hipErrorNotSupported;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return hipErrorNotSupported;
    const hipDataType t = dtype == BF16 ? HIP_R_16BF : HIP_R_16F;
    std::lock_guard<std::mutex> lock(g_lt_mu);
    auto hit = g_lt_handles.find(dev);
    if (hit == g_lt_handles.end()) {
        hipblasLtHandle_t h;
        if (hipblasLtCreate(&h) != HIPBLAS_STATUS_SUCCESS) return hipErrorNotSupported;
        hit = g_lt_handles.emplace(dev, h).first;
    }
    const LtKey key{dev, dtype, M, N, K, batch, sa, sb, sc, ws_bytes, a_kc, b_kc};
    auto pit = g_lt_plans.find(key);
    if (pit == g_lt_plans.end()) {
        LtPlan p;
        p.ok = make_plan(hit->second, t, M, N, K, a_kc, b_kc, batch, sa, sb, sc, ws_bytes, p);
        pit = g_lt_plans.emplace(key, p).first;
    }
    const LtPlan &p = pit->second;
    if (!p.ok) return hipErrorNotSupported;
    const float alpha = 1.f, beta = 0.f;
    const hipblasStatus_t st = hipblasLtMatmul(hit->second, p.desc, &alpha, B, p.la, A, p.lb, &beta, C, p.lc, C,
                                               p.lc, &p.algo, p.ws ? ws : nullptr, p.ws, s);
    return st == HIPBLAS_STATUS_SUCCESS ? hipSuccess : hipErrorLaunchFailure;
}

}  // namespace h3
