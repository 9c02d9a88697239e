// usp_abi.cpp -- the extern "C" entry points declared in include/usp.h:
// argument checking, handle lifetime, host<->device transfers, error strings.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>

#include "usp_internal.h"

namespace {

thread_local std::string g_last_error;

// Makes `dev` current for the scope and restores the caller's device after.
struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) return;
        ok = (prev == dev) || hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

// Every handle usp_encode returned and usp_free has not released. A handle is
// checked against this set before it is dereferenced, so a freed (or never
// issued) pointer is reported instead of read.
std::mutex g_live_mu;
std::unordered_set<const usp_matrix *> g_live;

bool alive(const usp_matrix *A) {
    if (!A) return false;
    std::lock_guard<std::mutex> lk(g_live_mu);
    return g_live.count(A) != 0;
}

// Releases a handle's device memory and the handle itself (registered or not).
void release(usp_matrix *A) {
    {
        DeviceGuard g(A->device);
        if (A->d_stream) (void)hipFree(A->d_stream);
        if (A->d_off) (void)hipFree(A->d_off);
    }
    delete A;
}

usp_status hip_fail(hipError_t e, const char *what) {
    return usp::fail(USP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace

namespace usp {
usp_status fail(usp_status st, const std::string &msg) {
    g_last_error = msg;
    return st;
}
}  // namespace usp

extern "C" {

const char *usp_last_error(void) { return g_last_error.c_str(); }

usp_status usp_encode(const uint16_t *W, int64_t ldw, const uint8_t *mask, int64_t ldm, int64_t M, int64_t K,
                      int device, usp_matrix **out) {
    if (out) *out = nullptr;
    if (!out || !W || !mask) return usp::fail(USP_ERR_INVALID_ARG, "usp_encode: null pointer");
    if (M < 1 || K < 1) return usp::fail(USP_ERR_INVALID_ARG, "usp_encode: M and K must be >= 1");
    if (ldw < K || ldm < K) return usp::fail(USP_ERR_INVALID_ARG, "usp_encode: ldw and ldm must be >= K");
    if (M > usp::kMaxRows)
        return usp::fail(USP_ERR_UNSUPPORTED, "usp_encode: M above 2^20 rows (the workspace's arrival counters)");
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess) return hip_fail(e, "usp_encode: hipGetDeviceCount");
    if (device < 0 || device >= ndev) return usp::fail(USP_ERR_INVALID_ARG, "usp_encode: no such device");

    usp::HostEncoding enc;
    try {
        usp::encode_host(W, ldw, mask, ldm, M, K, enc);
    } catch (const std::bad_alloc &) {
        return usp::fail(USP_ERR_OOM, "usp_encode: host allocation failed (or encoding exceeds 64 GiB)");
    }
    DeviceGuard g(device);
    if (!g.ok) return usp::fail(USP_ERR_HIP, "usp_encode: cannot select device");
    usp_matrix *A = new (std::nothrow) usp_matrix();
    if (!A) return usp::fail(USP_ERR_OOM, "usp_encode: host allocation failed");
    A->device = device;
    A->M = M;
    A->K = K;
    A->RB = enc.RB;
    A->KT = enc.KT;
    A->nnz = enc.nnz;
    A->max_chunks = enc.max_chunks;
    A->stream_bytes = enc.stream.size();
    A->d_stream = nullptr;
    A->d_off = nullptr;
    A->num_cus = 0;
    if (hipDeviceGetAttribute(&A->num_cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess)
        A->num_cus = 0;
    // The kernels' last load of a record may read up to 1 KB past it.
    e = hipMalloc(&A->d_stream, A->stream_bytes + usp::kStreamPad);
    if (e == hipSuccess) e = hipMemset(A->d_stream, 0, A->stream_bytes + usp::kStreamPad);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&A->d_off), enc.off.size() * sizeof(uint32_t));
    if (e != hipSuccess) {
        release(A);
        return usp::fail(USP_ERR_OOM, std::string("usp_encode: hipMalloc: ") + hipGetErrorString(e));
    }
    // One-time set-up of this device's scratch for usp_spmm_noalloc (outside
    // any graph capture: encoding precedes every product).
    if (e == hipSuccess) e = (hipError_t)usp::noalloc_setup(device);
    if (e != hipSuccess) {
        release(A);
        return hip_fail(e, "usp_encode: device scratch set-up");
    }
    e = hipMemcpy(A->d_stream, enc.stream.data(), A->stream_bytes, hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(A->d_off, enc.off.data(), enc.off.size() * sizeof(uint32_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        release(A);
        return hip_fail(e, "usp_encode: hipMemcpy");
    }
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        g_live.insert(A);
    }
    *out = A;
    return USP_OK;
}

size_t usp_workspace_size(const usp_matrix *A, int64_t N) {
    if (!alive(A) || N < 1) return 0;
    return usp::spmm_workspace_bytes(A, N);
}

usp_status usp_plan(const usp_matrix *A, int64_t N, char *buf, size_t len) {
    if (!alive(A)) return usp::fail(USP_ERR_INVALID_ARG, "usp_plan: invalid or freed handle");
    if (N < 1 || !buf || len == 0) return usp::fail(USP_ERR_INVALID_ARG, "usp_plan: need N >= 1 and a buffer");
    DeviceGuard g(A->device);
    if (!g.ok) return usp::fail(USP_ERR_HIP, "usp_plan: cannot select device");
    const std::string d = usp::describe_plan(A, N);
    const size_t n = d.size() < len - 1 ? d.size() : len - 1;
    std::memcpy(buf, d.data(), n);
    buf[n] = '\0';
    return USP_OK;
}

static usp_status spmm_common(const char *fn, const usp_matrix *A, const void *X, int64_t ldx, void *Y,
                              int64_t ldy, int64_t N, const usp::Epilogue &ep, void *workspace, size_t ws_bytes,
                              void *stream) {
    const std::string f(fn);
    if (!alive(A)) return usp::fail(USP_ERR_INVALID_ARG, f + ": invalid or freed handle");
    if (!X || !Y) return usp::fail(USP_ERR_INVALID_ARG, f + ": null X or Y");
    if (N < 1) return usp::fail(USP_ERR_INVALID_ARG, f + ": N must be >= 1");
    if (N > (int64_t)1 << 20) return usp::fail(USP_ERR_UNSUPPORTED, f + ": N too large");
    if (ldx < A->K) return usp::fail(USP_ERR_INVALID_ARG, f + ": ldx must be >= K");
    if (ldy < A->M) return usp::fail(USP_ERR_INVALID_ARG, f + ": ldy must be >= M");
    if ((reinterpret_cast<uintptr_t>(X) & 1) || (reinterpret_cast<uintptr_t>(Y) & 1))
        return usp::fail(USP_ERR_INVALID_ARG, f + ": X and Y must be 2-byte aligned");
    if (ep.act < USP_ACT_NONE || ep.act > USP_ACT_SILU)
        return usp::fail(USP_ERR_INVALID_ARG, f + ": unknown activation");
    if (reinterpret_cast<uintptr_t>(ep.bias) & 1) return usp::fail(USP_ERR_INVALID_ARG, f + ": bias must be 2-byte aligned");
    if (ep.res && ((reinterpret_cast<uintptr_t>(ep.res) & 1) || ep.ldr < A->M))
        return usp::fail(USP_ERR_INVALID_ARG, f + ": residual must be 2-byte aligned with ldr >= M");
    const size_t need = usp::spmm_workspace_bytes(A, N);
    if (need && (!workspace || ws_bytes < need))
        return usp::fail(USP_ERR_INVALID_ARG, f + ": workspace too small (see usp_workspace_size)");
    if (need && (reinterpret_cast<uintptr_t>(workspace) & 15))
        return usp::fail(USP_ERR_INVALID_ARG, f + ": workspace must be 16-byte aligned");
    DeviceGuard g(A->device);
    if (!g.ok) return usp::fail(USP_ERR_HIP, f + ": cannot select device");
    const int rc = usp::launch_spmm(A, X, ldx, Y, ldy, N, ep, workspace, stream);
    if (rc != 0) return hip_fail((hipError_t)rc, (f + ": launch").c_str());
    return USP_OK;
}

usp_status usp_spmm(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                    void *workspace, size_t ws_bytes, void *stream) {
    return spmm_common("usp_spmm", A, X, ldx, Y, ldy, N, usp::Epilogue(), workspace, ws_bytes, stream);
}

usp_status usp_spmm_ex(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                       const void *bias, const void *residual, int64_t ldr, int activation, void *workspace,
                       size_t ws_bytes, void *stream) {
    usp::Epilogue ep;
    ep.bias = reinterpret_cast<const uint16_t *>(bias);
    ep.res = reinterpret_cast<const uint16_t *>(residual);
    ep.ldr = ldr;
    ep.act = activation;
    return spmm_common("usp_spmm_ex", A, X, ldx, Y, ldy, N, ep, workspace, ws_bytes, stream);
}

usp_status usp_spmm_noalloc(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                            void *stream) {
    if (!alive(A)) return usp::fail(USP_ERR_INVALID_ARG, "usp_spmm_noalloc: invalid or freed handle");
    if (N < 1) return usp::fail(USP_ERR_INVALID_ARG, "usp_spmm_noalloc: N must be >= 1");
    const size_t need = usp::spmm_workspace_bytes(A, N);
    if (need > USP_NOALLOC_SCRATCH_BYTES)
        return usp::fail(USP_ERR_UNSUPPORTED, "usp_spmm_noalloc: this product needs " + std::to_string(need) +
                                                  " bytes of workspace, above the " +
                                                  std::to_string((size_t)USP_NOALLOC_SCRATCH_BYTES) +
                                                  "-byte device scratch (use usp_spmm with a workspace)");
    void *ws = usp::noalloc_scratch(A->device);
    if (!ws) return usp::fail(USP_ERR_INTERNAL, "usp_spmm_noalloc: device scratch not set up");
    return spmm_common("usp_spmm_noalloc", A, X, ldx, Y, ldy, N, usp::Epilogue(), ws, USP_NOALLOC_SCRATCH_BYTES,
                       stream);
}

usp_status usp_densify(const usp_matrix *A, void *Wd, int64_t ldw, void *stream) {
    if (!alive(A)) return usp::fail(USP_ERR_INVALID_ARG, "usp_densify: invalid or freed handle");
    if (!Wd) return usp::fail(USP_ERR_INVALID_ARG, "usp_densify: null output");
    if (ldw < A->K) return usp::fail(USP_ERR_INVALID_ARG, "usp_densify: ldw must be >= K");
    if (reinterpret_cast<uintptr_t>(Wd) & 1) return usp::fail(USP_ERR_INVALID_ARG, "usp_densify: misaligned output");
    DeviceGuard g(A->device);
    if (!g.ok) return usp::fail(USP_ERR_HIP, "usp_densify: cannot select device");
    const int rc = usp::launch_densify(A, Wd, ldw, stream);
    if (rc != 0) return hip_fail((hipError_t)rc, "usp_densify: launch");
    return USP_OK;
}

usp_status usp_decode(const usp_matrix *A, uint16_t *W_out, uint8_t *mask_out) {
    if (!alive(A)) return usp::fail(USP_ERR_INVALID_ARG, "usp_decode: invalid or freed handle");
    if (!W_out || !mask_out) return usp::fail(USP_ERR_INVALID_ARG, "usp_decode: null output");
    usp::HostEncoding enc;
    try {
        enc.M = A->M;
        enc.K = A->K;
        enc.RB = A->RB;
        enc.KT = A->KT;
        enc.nnz = A->nnz;
        enc.off.resize(A->RB * A->KT + 1);
        enc.stream.resize(A->stream_bytes);
    } catch (const std::bad_alloc &) {
        return usp::fail(USP_ERR_OOM, "usp_decode: host allocation failed");
    }
    DeviceGuard g(A->device);
    if (!g.ok) return usp::fail(USP_ERR_HIP, "usp_decode: cannot select device");
    hipError_t e = hipMemcpy(enc.stream.data(), A->d_stream, A->stream_bytes, hipMemcpyDeviceToHost);
    if (e == hipSuccess)
        e = hipMemcpy(enc.off.data(), A->d_off, enc.off.size() * sizeof(uint32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "usp_decode: hipMemcpy");
    if (!usp::decode_host(enc, W_out, mask_out))
        return usp::fail(USP_ERR_INTERNAL, "usp_decode: encoding is inconsistent");
    return USP_OK;
}

usp_status usp_info(const usp_matrix *A, usp_info_t *info) {
    if (!alive(A)) return usp::fail(USP_ERR_INVALID_ARG, "usp_info: invalid or freed handle");
    if (!info) return usp::fail(USP_ERR_INVALID_ARG, "usp_info: null output");
    std::memset(info, 0, sizeof(*info));
    info->M = A->M;
    info->K = A->K;
    info->nnz = A->nnz;
    info->device_bytes = A->stream_bytes;
    info->table_bytes = (size_t)(A->RB * A->KT + 1) * sizeof(uint32_t);
    info->format_version = USP_FORMAT_VERSION;
    info->tile_rows = usp::kTileRows;
    info->tile_k = usp::kTileK;
    info->device = A->device;
    return USP_OK;
}

usp_status usp_free(usp_matrix *A) {
    if (!A) return USP_OK;
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        if (g_live.erase(A) == 0) return usp::fail(USP_ERR_INVALID_ARG, "usp_free: invalid or already freed handle");
    }
    release(A);
    return USP_OK;
}

}  // extern "C"
