// usp_dense_ref.cpp -- the dense baseline the benchmark compares the sparse
// product against: Y = W X as one hipBLASLt fp16 GEMM (fp16 A, B and C, fp32
// compute), called through hipBLASLt's C API. Not part of the product path
// (libusp_denseref.so, loaded by the benchmark only).
//
// Layout: hipBLASLt is column-major. W (row-major M x K) is the column-major
// K x M matrix A used transposed; X (token-major [N][K]) is the column-major
// K x N matrix B; Y (token-major [N][M]) is the column-major M x N matrix C.
// So C = A^T B, the "TN" layout.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt-ext.hpp>
#include <hipblaslt/hipblaslt.h>

#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

namespace {

struct DenseGemm {
    hipblasLtHandle_t handle = nullptr;
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
    hipblasLtMatmulPreference_t pref = nullptr;
    std::vector<hipblasLtMatmulHeuristicResult_t> algos;
};

void destroy(DenseGemm *g) {
    if (!g) return;
    if (g->pref) hipblasLtMatmulPreferenceDestroy(g->pref);
    if (g->c) hipblasLtMatrixLayoutDestroy(g->c);
    if (g->b) hipblasLtMatrixLayoutDestroy(g->b);
    if (g->a) hipblasLtMatrixLayoutDestroy(g->a);
    if (g->desc) hipblasLtMatmulDescDestroy(g->desc);
    if (g->handle) hipblasLtDestroy(g->handle);
    delete g;
}

}  // namespace

extern "C" {

// Sets up the GEMM for (M, K, N) and asks hipBLASLt's heuristic for up to
// max_algos algorithms allowed at most ws_bytes of workspace. Returns 0 and a
// context in *out (with *n_algos algorithms), or a nonzero hipBLAS status.
int usp_dense_plan(int64_t M, int64_t K, int64_t N, int max_algos, size_t ws_bytes, void **out, int *n_algos) {
    *out = nullptr;
    *n_algos = 0;
    DenseGemm *g = new DenseGemm();
    hipblasStatus_t st = hipblasLtCreate(&g->handle);
    if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatmulDescCreate(&g->desc, HIPBLAS_COMPUTE_32F, HIP_R_32F);
    const hipblasOperation_t opA = HIPBLAS_OP_T, opB = HIPBLAS_OP_N;
    if (st == HIPBLAS_STATUS_SUCCESS)
        st = hipblasLtMatmulDescSetAttribute(g->desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opA, sizeof(opA));
    if (st == HIPBLAS_STATUS_SUCCESS)
        st = hipblasLtMatmulDescSetAttribute(g->desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opB, sizeof(opB));
    if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatrixLayoutCreate(&g->a, HIP_R_16F, K, M, K);
    if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatrixLayoutCreate(&g->b, HIP_R_16F, K, N, K);
    if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatrixLayoutCreate(&g->c, HIP_R_16F, M, N, M);
    if (st == HIPBLAS_STATUS_SUCCESS) st = hipblasLtMatmulPreferenceCreate(&g->pref);
    uint64_t ws = ws_bytes;
    if (st == HIPBLAS_STATUS_SUCCESS)
        st = hipblasLtMatmulPreferenceSetAttribute(g->pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof(ws));
    if (st == HIPBLAS_STATUS_SUCCESS) {
        g->algos.resize(max_algos > 0 ? max_algos : 1);
        int n = 0;
        st = hipblasLtMatmulAlgoGetHeuristic(g->handle, g->desc, g->a, g->b, g->c, g->c, g->pref, (int)g->algos.size(),
                                             g->algos.data(), &n);
        g->algos.resize(st == HIPBLAS_STATUS_SUCCESS ? n : 0);
    }
    if (st != HIPBLAS_STATUS_SUCCESS || g->algos.empty()) {
        destroy(g);
        return st != HIPBLAS_STATUS_SUCCESS ? (int)st : -1;
    }
    *out = g;
    *n_algos = (int)g->algos.size();
    return 0;
}

// Workspace bytes algorithm i needs.
size_t usp_dense_workspace(void *ctx, int i) {
    DenseGemm *g = static_cast<DenseGemm *>(ctx);
    return (g && i >= 0 && i < (int)g->algos.size()) ? g->algos[i].workspaceSize : 0;
}

// hipBLASLt's solution index of algorithm i and its solution name (into buf).
int usp_dense_algo_info(void *ctx, int i, char *buf, size_t len) {
    DenseGemm *g = static_cast<DenseGemm *>(ctx);
    if (!g || i < 0 || i >= (int)g->algos.size()) return -1;
    const int index = hipblaslt_ext::getIndexFromAlgo(g->algos[i].algo);
    const std::string name = hipblaslt_ext::getSolutionNameFromAlgo(g->handle, g->algos[i].algo);
    if (buf && len) {
        const size_t n = name.size() < len - 1 ? name.size() : len - 1;
        std::memcpy(buf, name.data(), n);
        buf[n] = '\0';
    }
    return index;
}

// Y = W X with algorithm i on `stream` (asynchronous).
int usp_dense_run(void *ctx, int i, const void *W, const void *X, void *Y, void *ws, size_t ws_bytes, void *stream) {
    DenseGemm *g = static_cast<DenseGemm *>(ctx);
    if (!g || i < 0 || i >= (int)g->algos.size()) return -1;
    const float alpha = 1.0f, beta = 0.0f;
    return (int)hipblasLtMatmul(g->handle, g->desc, &alpha, W, g->a, X, g->b, &beta, Y, g->c, Y, g->c,
                                &g->algos[i].algo, ws, ws_bytes, reinterpret_cast<hipStream_t>(stream));
}

void usp_dense_free(void *ctx) { destroy(static_cast<DenseGemm *>(ctx)); }

}  // extern "C"
