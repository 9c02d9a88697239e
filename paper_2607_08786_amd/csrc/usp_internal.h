// usp_internal.h -- handle layout and helpers shared by the library's sources.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "usp.h"
#include "usp_format.h"

struct usp_matrix {
    int device;
    int64_t M, K;            // logical shape
    int64_t RB, KT;          // row blocks (16 rows) and column tiles (256 columns)
    int64_t nnz;
    int64_t max_chunks;      // most 16-byte value chunks in one tile record
    size_t stream_bytes;     // bytes of all tile records
    void *d_stream;          // device: tile records
    uint32_t *d_off;         // device: RB*KT + 1 offsets in 16-byte units
    int num_cus;             // compute units of the device
};

namespace usp {

// Most rows an encoding may have: the workspace's arrival counters (one
// 32-bit word per row block, rounded up to sets of 4) occupy a fixed 256 KB
// region at its start whatever the handle.
constexpr int64_t kMaxRows = int64_t(1) << 20;

// Host-side encoding result (before upload).
struct HostEncoding {
    int64_t M = 0, K = 0, RB = 0, KT = 0, nnz = 0;
    int64_t max_chunks = 0;        // most 16-byte value chunks in one record
    std::vector<uint32_t> off;     // RB*KT + 1 entries, 16-byte units
    std::vector<uint8_t> stream;   // 16 * off.back() bytes
};

// Encoder / decoder (usp_encode.cpp). encode_host throws std::bad_alloc on OOM.
void encode_host(const uint16_t *W, int64_t ldw, const uint8_t *mask, int64_t ldm,
                 int64_t M, int64_t K, HostEncoding &out);
// Returns false when the records are inconsistent with the shape.
bool decode_host(const HostEncoding &enc, uint16_t *W_out, uint8_t *mask_out);

// Error reporting (usp_abi.cpp).
usp_status fail(usp_status st, const std::string &msg);

// Launchers (usp_kernels.hip). They return hipSuccess or the launch error code.
struct SpmmPlan {
    int64_t row_groups;  // groups of 4 row blocks
    int64_t units;       // row groups * column tiles
    int64_t grid;        // persistent workgroups
    int64_t maxseg;      // most workgroups sharing one row group
    bool split;          // some row group is shared by several workgroups
};
SpmmPlan plan_spmm(const usp_matrix *A, int64_t N);
size_t spmm_workspace_bytes(const usp_matrix *A, int64_t N);
// The kernel usp_spmm runs for A and N (X 16-byte aligned, ldx = K), as text.
std::string describe_plan(const usp_matrix *A, int64_t N);
// Fused output epilogue: Y = act(W X + bias) + residual (all optional).
struct Epilogue {
    const uint16_t *bias = nullptr;  // fp16 [M]
    const uint16_t *res = nullptr;   // fp16, column n at res + n * ldr
    int64_t ldr = 0;
    int act = 0;                     // usp_activation
};
int launch_spmm(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                const Epilogue &ep, void *workspace, void *stream);
int launch_densify(const usp_matrix *A, void *Wd, int64_t ldw, void *stream);
// Device scratch of usp_spmm_noalloc: noalloc_setup looks up and clears the
// calling thread's current device's copy once (returns a HIP error code);
// noalloc_scratch returns its device address, or null before the set-up.
int noalloc_setup(int device);
void *noalloc_scratch(int device);

}  // namespace usp
