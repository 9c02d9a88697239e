/*
 * usp.h -- C ABI of the unstructured-sparse fp16 SpMM library (libusp.so).
 *
 * The library computes Y = W X for a weight matrix W (M x K, fp16) pruned to
 * moderate unstructured sparsity and a skinny dense input X (K x N, fp16, N the
 * number of tokens of a decode step), with fp32 accumulation and fp16 output.
 * This is the sparse matrix multiplication of Section 5.1 of the paper
 * (weight M x K sparse, input K x N dense, output M x N dense), the operation its
 * storage format (Section 3) and kernel (Section 4) exist to accelerate.
 *
 * W is first converted once, on the host, into a compressed device-resident
 * format (the one-time conversion of Section 5.3, "Storage Format Conversion");
 * every product then streams that format from HBM and decodes it on chip.
 *
 * Layout conventions (all strides in elements):
 *   W     row-major M x K: row m at W + m*ldw (the nn.Linear weight layout)
 *   mask  row-major M x K bytes: row m at mask + m*ldm; nonzero = kept
 *   X     token-major: column n of the logical K x N matrix at X + n*ldx,
 *         i.e. a contiguous [N, K] activation when ldx == K
 *   Y     token-major: column n of the logical M x N matrix at Y + n*ldy
 *
 * Errors: every entry point returns a usp_status; no exception crosses the
 * ABI. usp_last_error() returns a message for the calling thread's most recent
 * failure. Kernel faults surface at the caller's next synchronisation.
 * Thread safety: a handle is immutable after usp_encode; concurrent usp_spmm
 * calls on one handle are safe when each uses its own workspace.
 */
#ifndef USP_H
#define USP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct usp_matrix usp_matrix; /* opaque; owns the device memory of one encoded W */

typedef enum {
    USP_OK = 0,
    USP_ERR_INVALID_ARG = 1, /* null pointer, bad size or stride, freed handle */
    USP_ERR_UNSUPPORTED = 2, /* valid request this build does not serve (alignment, N range) */
    USP_ERR_OOM = 3,         /* host or device allocation failed */
    USP_ERR_HIP = 4,         /* a HIP runtime call failed (message has the HIP error) */
    USP_ERR_INTERNAL = 5
} usp_status;

/* Format version written by usp_encode and reported by usp_info. */
#define USP_FORMAT_VERSION 2

/*
 * usp_encode -- one-time conversion of W and its keep-mask into the compressed
 * device format (Section 3.2 defines the paper's own format; ours is described
 * with the library). Blocking.
 *   W     host pointer, M x K fp16 bit patterns, row stride ldw >= K
 *   mask  host pointer, M x K bytes, row stride ldm >= K; nonzero = keep
 *   M, K  >= 1, M <= 2^20 (USP_ERR_UNSUPPORTED above: the workspace keeps one
 *         arrival counter per 16 rows in a fixed 256 KB region)
 *   device  HIP device ordinal that will hold the encoding
 *   out   receives the new handle; set to NULL on any error
 * Kept values are stored as opaque 16-bit words (signed zeros, subnormals,
 * NaN payloads and kept exact zeros survive bit for bit); values where the
 * mask is zero are ignored. The caller keeps ownership of W and mask.
 */
usp_status usp_encode(const uint16_t *W, int64_t ldw, const uint8_t *mask, int64_t ldm,
                      int64_t M, int64_t K, int device, usp_matrix **out);

/*
 * usp_workspace_size -- bytes of device workspace usp_spmm needs for this
 * handle and this N (0 when none). Returns 0 for a NULL handle. The
 * workspace holds the split rows' arrival counters and fp32 partials and,
 * where the shared-decode kernel serves the call (33 to 256 tokens on large
 * layers), a copy of X rearranged into the order its products read it
 * (KT x 8 x ceil(N / 16) KB), rewritten by every such call.
 */
size_t usp_workspace_size(const usp_matrix *A, int64_t N);

/*
 * usp_spmm -- Y = W X on the handle's device, enqueued on `stream`
 * (a hipStream_t; NULL = the default stream). Asynchronous: returns after the
 * launch. Y is overwritten (no accumulation into it).
 *   X   device pointer, fp16, token-major with stride ldx >= K
 *   Y   device pointer, fp16, token-major with stride ldy >= M; must not alias X
 *   N   number of tokens, 1 <= N
 *   workspace  device pointer, 16-byte aligned, to >= usp_workspace_size(A, N)
 *       bytes (may be NULL when that size is 0); owned by the caller; must not be
 *       used by another in-flight call. It must be zero-filled before its first
 *       use; every completed call leaves it ready for the next one (with any
 *       handle and any N), so it is cleared once, not per call.
 * Accumulation is fp32 in a fixed order: results are bitwise reproducible run
 * to run. The output is rounded to fp16 with round-to-nearest-even.
 * Inputs with X not 16-byte aligned or ldx not a multiple of 8 take a slower
 * element-wise path. No allocation and no synchronisation happens inside, and
 * the call only enqueues kernels on `stream` (no memory-set or copy operations),
 * so it may be captured into a HIP graph and the graph replayed; each replay
 * leaves the workspace ready for the next, as each call does.
 */
usp_status usp_spmm(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy,
                    int64_t N, void *workspace, size_t ws_bytes, void *stream);

/* Activation of usp_spmm_ex, applied after the bias. */
typedef enum {
    USP_ACT_NONE = 0,
    USP_ACT_RELU = 1,      /* max(v, 0) */
    USP_ACT_GELU_TANH = 2, /* 0.5 v (1 + tanh(sqrt(2/pi) (v + 0.044715 v^3))) */
    USP_ACT_SILU = 3       /* v / (1 + exp(-v)) */
} usp_activation;

/*
 * usp_spmm_ex -- usp_spmm with a linear layer's epilogue fused into the output
 * store: Y = act(W X + bias) + residual. The decode-step linear layers the
 * paper's sparse product replaces (Section 2.1; its models' projections carry a
 * bias, the FFN an activation, the block a residual add) need nothing else.
 * Per output, in fp32: the sum, + bias, the activation, + residual, then the
 * one rounding to fp16 (round to nearest even).
 *   bias       device fp16 [M] (2-byte aligned), or NULL for none
 *   residual   device fp16, logical M x N, column n at residual + n * ldr with
 *              ldr >= M (2-byte aligned), or NULL for none. It may be Y itself
 *              with ldr == ldy (an in-place add: each output reads its residual
 *              before it is written, by the same thread); otherwise it must not
 *              overlap Y.
 *   activation a usp_activation
 * Everything else -- arguments, workspace, asynchrony, reproducibility -- as
 * usp_spmm; usp_spmm(...) equals usp_spmm_ex(..., NULL, NULL, 0, USP_ACT_NONE, ...).
 * An activation outside usp_activation is USP_ERR_INVALID_ARG.
 */
usp_status usp_spmm_ex(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                       const void *bias, const void *residual, int64_t ldr, int activation,
                       void *workspace, size_t ws_bytes, void *stream);

/* Bytes of the device scratch usp_spmm_noalloc uses on each GPU (32 MiB). */
#define USP_NOALLOC_SCRATCH_BYTES (32u << 20)

/*
 * usp_spmm_noalloc -- for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. The same product as usp_spmm (same kernels, same bits), with no
 * workspace argument: its workspace is a USP_NOALLOC_SCRATCH_BYTES device array
 * the library holds on each GPU until the process ends (looked up and cleared
 * once per device inside usp_encode, so the handle's device is set up by the
 * time any product runs). This call allocates nothing and calls no allocating
 * routine.
 *   A, X, ldx, Y, ldy, N, stream   as usp_spmm
 * Every call on a GPU shares that GPU's scratch, which keeps the last call's
 * contents; each completed call leaves its arrival counters at zero, as the
 * next call needs them. Calls that overlap in time on one GPU (other streams,
 * other host threads) race on the scratch and give wrong results: serialize
 * them. Returns USP_ERR_UNSUPPORTED, enqueueing nothing, when the product needs
 * more workspace than the scratch holds (usp_workspace_size(A, N) >
 * USP_NOALLOC_SCRATCH_BYTES; every configured layer up to 64 tokens fits).
 */
usp_status usp_spmm_noalloc(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy,
                            int64_t N, void *stream);

/*
 * usp_plan -- which kernel usp_spmm runs for this handle and N when X is 16-byte
 * aligned with ldx = K, as a short text ("row W=8", "chunk S=5 W=8 nb=1 grid=200",
 * "dma nb=4 tg=1 grid=1024", "fourwave passes=1 nt=2 grid=768"), written to
 * buf (at most len bytes with the terminating NUL, truncated if longer). For
 * tests and tuning; enqueues nothing. USP_ERR_INVALID_ARG for a NULL handle,
 * N < 1, or no buffer.
 */
usp_status usp_plan(const usp_matrix *A, int64_t N, char *buf, size_t len);

/*
 * usp_densify -- writes W with the mask applied (pruned entries as +0) into a
 * dense row-major M x K fp16 device buffer Wd with row stride ldw >= K, by the
 * same on-chip decode the product uses. Asynchronous on `stream`. For checks.
 */
usp_status usp_densify(const usp_matrix *A, void *Wd, int64_t ldw, void *stream);

/*
 * usp_decode -- host-side inverse of usp_encode: copies the encoding back and
 * rebuilds W (masked entries as 0x0000) and the mask (0/1) into the caller's
 * host buffers of M x K entries each (contiguous rows). Blocking.
 */
usp_status usp_decode(const usp_matrix *A, uint16_t *W_out, uint8_t *mask_out);

typedef struct {
    int64_t M, K;           /* logical shape */
    int64_t nnz;            /* kept entries */
    size_t device_bytes;    /* bytes of the encoding the product streams from HBM */
    size_t table_bytes;     /* bytes of the per-tile offset table (also streamed) */
    int32_t format_version; /* USP_FORMAT_VERSION */
    int32_t tile_rows, tile_k; /* tile geometry of the encoding */
    int32_t device;
} usp_info_t;

/* usp_info -- shape, size and geometry of an encoding. */
usp_status usp_info(const usp_matrix *A, usp_info_t *info);

/* usp_free -- releases the handle and its device memory. NULL is accepted.
 * The caller guarantees no usp_spmm/usp_densify on it is still in flight.
 * Handles are looked up among the live ones before use, never dereferenced
 * blindly: passing a freed handle (or any pointer usp_encode did not return)
 * to any entry point gives USP_ERR_INVALID_ARG, unless a later usp_encode
 * happened to return the same address. */
usp_status usp_free(usp_matrix *A);

/* usp_last_error -- message of the calling thread's most recent failure ("" if none). */
const char *usp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* USP_H */
