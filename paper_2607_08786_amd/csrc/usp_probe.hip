// usp_probe.hip -- measurement references the benchmark reports beside the
// sparse product, not part of the product path (libusp_probe.so, loaded by the
// benchmark only):
//   * usp_probe_read: a plain streaming read, how long reading a buffer of the
//     same size as an encoded matrix takes on this GPU, launch and ramp
//     included;
//   * usp_probe_mfma: the issue rate of the dense matrix-core product
//     v_mfma_f32_16x16x32_f16 and of the sparse one v_smfmac_f32_16x16x64_f16
//     (a 2:4 A operand: 2 kept entries of every 4 consecutive k), the numbers
//     behind the choice of dense MFMA for the contraction.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
constexpr int kLanes = 64;
constexpr int kInFlight = 8;  // 1 KB loads in flight per wavefront

// Wavefront w reads its contiguous share of the buffer in 1 KB loads (16 bytes
// per lane), kInFlight at a time, through a buffer resource that ends at the
// share's end (loads past it return zeros and fetch nothing). The xor of the
// data is stored only if it equals a value it practically never takes, so the
// loads are not optimised away and nothing is written.
__global__ __launch_bounds__(kLanes) void read_kernel(const uint8_t *__restrict__ buf, int64_t kb, uint32_t *sink) {
    const int lane = threadIdx.x;
    const int64_t w = blockIdx.x, G = gridDim.x;
    const int64_t q0 = w * kb / G, q1 = (w + 1) * kb / G;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(buf + q0 * 1024), (short)0, (int)((q1 - q0) * 1024), 0x00020000);
    v4u32 acc = {0u, 0u, 0u, 0u};
    for (int64_t q = 0; q < q1 - q0; q += kInFlight) {
        v4u32 v[kInFlight];
#pragma unroll
        for (int d = 0; d < kInFlight; ++d)
            v[d] = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)((q + d) * 1024 + lane * 16), 0, 0);
#pragma unroll
        for (int d = 0; d < kInFlight; ++d) acc ^= v[d];
    }
    if (acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u) sink[w] = acc.z;
}

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Every wavefront issues `iters` rounds of 8 independent products (8
// accumulators, so no product waits for another). Inline assembly keeps the
// loop to the products alone (the compiler otherwise moves accumulators between
// register files every round). The sums go to `sink`.
template <bool SPARSE>
__global__ __launch_bounds__(256) void mfma_rate_kernel(int iters, floatx4 *sink) {
    const int lane = threadIdx.x & 63;
    half8 a;
    half16 b;
    for (int i = 0; i < 8; ++i) a[i] = (_Float16)((lane + i) & 7);
    for (int i = 0; i < 16; ++i) b[i] = (_Float16)((lane * 3 + i) & 7);
    const half8 b8 = {b[0], b[1], b[2], b[3], b[4], b[5], b[6], b[7]};
    const int idx = 0x4E4E4E4E;  // 2-bit positions of the kept entries within their windows
    floatx4 c[8];
    for (int q = 0; q < 8; ++q) c[q] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (SPARSE)
                asm volatile("v_smfmac_f32_16x16x64_f16 %0, %1, %2, %3" : "+v"(c[q]) : "v"(a), "v"(b), "v"(idx));
            else
                asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(c[q]) : "v"(a), "v"(b8));
        }
    }
    floatx4 t = c[0];
    for (int q = 1; q < 8; ++q) t += c[q];
    sink[blockIdx.x * 256 + threadIdx.x] = t;
}

}  // namespace

// Issues `iters` rounds of 8 independent matrix-core products per wavefront in
// `blocks` workgroups of 4 wavefronts: v_smfmac_f32_16x16x64_f16 when `sparse`,
// else v_mfma_f32_16x16x32_f16. `sink` holds blocks * 256 float4. Time the call
// with events: products per second = blocks * 4 * iters * 8 / seconds. Returns
// 0, or the HIP error code.
extern "C" int usp_probe_mfma(int sparse, int blocks, int iters, void *sink, void *stream) {
    if (blocks < 1 || iters < 1 || !sink) return (int)hipErrorInvalidValue;
    if (sparse)
        hipLaunchKernelGGL(mfma_rate_kernel<true>, dim3((unsigned)blocks), dim3(256), 0,
                           reinterpret_cast<hipStream_t>(stream), iters, reinterpret_cast<floatx4 *>(sink));
    else
        hipLaunchKernelGGL(mfma_rate_kernel<false>, dim3((unsigned)blocks), dim3(256), 0,
                           reinterpret_cast<hipStream_t>(stream), iters, reinterpret_cast<floatx4 *>(sink));
    return (int)hipGetLastError();
}

// Reads the first `bytes` (rounded down to whole KB, at most 2^31 per
// wavefront share) of the device buffer `buf` with `waves` single-wavefront
// workgroups on `stream`; `sink` is a device buffer of at least `waves` uint32
// that is (practically) never written. Returns 0, or the HIP error code.
extern "C" int usp_probe_read(const void *buf, size_t bytes, int waves, void *sink, void *stream) {
    if (!buf || !sink || waves < 1 || bytes / 1024 / (size_t)waves >= ((size_t)1 << 21)) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)waves), dim3(kLanes), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint8_t *>(buf), (int64_t)(bytes / 1024), reinterpret_cast<uint32_t *>(sink));
    return (int)hipGetLastError();
}
