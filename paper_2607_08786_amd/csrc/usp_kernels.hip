// usp_kernels.hip -- gfx950 kernels of the sparse product and their launchers.
//
// Five kernels share one decode; the planner (wave_kind, plan_wave, plan_pass)
// picks one by shape and token count:
//   * spmm_dma_kernel (large layers, up to 32 tokens; beyond, only records too
//     large for the next kernel's slots): one wavefront per workgroup streams
//     a contiguous range of units (4 row blocks x 1 column tile), records moved
//     straight into a ring of LDS slots, X in registers; more than 4 blocks of
//     16 tokens are split into token groups;
//   * spmm_share_kernel and its pipelined variant spmm_pipe_kernel (large
//     layers, 33 to 256 tokens): four wavefronts stream a range of units, each
//     decodes one row block's record into a shared LDS buffer of A operands and
//     multiplies all four by its quarter of the tokens, reading X packed in
//     product order by pack_x_kernel;
//   * spmm_chunk_kernel (small layers, up to 32 tokens): 4 or 8 row blocks x a
//     chunk of 4 column tiles per workgroup, every record requested at once;
//   * spmm_row_kernel (few row blocks, up to 16 tokens): one row block per
//     workgroup, its column tiles split over the wavefronts and summed in LDS;
//   * spmm_kernel (everything else, any token count in passes): a workgroup of
//     4 wavefronts walks the column tiles of one row group (64 rows) at a time,
//     the X tile staged in LDS once per tile for all 4, one tile in flight.
// Per record, whatever the kernel:
//   * a wavefront prefix sum of the lanes' kept counts gives each lane the start
//     of its packed values at every 32-column step (the decode is a prefix sum
//     over the metadata, as the paper's PDD decode in Section 4.3 is); three
//     packed DPP scans cover all 8 steps;
//   * each lane expands its 8 positions of the step into the 16 x 32 fp16 A
//     operand: two nibble expansions, each a funnel shift (v_alignbyte) of three
//     LDS dwords plus two byte permutes (v_perm) driven by a 16-entry selector
//     table;
//   * v_mfma_f32_16x16x32_f16 accumulates in fp32 (the dense-contraction part,
//     Section 4.3).
// Epilogue: fp32 -> optional bias, activation and residual -> fp16 with round
// to nearest even. A row block (or row group) whose columns were split over
// several wavefronts or workgroups is finished by whichever arrives last: each
// writes its fp32 partial sums with device-coherent stores and bumps a counter;
// the last reads every partial with device-coherent loads, sums them in a fixed
// order (bitwise reproducible, no floating-point atomics), stores Y and resets
// the counter to zero for the next call. No workgroup waits on another.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdio>
#include <mutex>
#include <string>
#include <utility>

#include "usp_internal.h"

namespace usp {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer resource on gfx9-class targets (untyped 32-bit data).
constexpr int kBufferRsrcWord3 = 0x00020000;
// Cache policy of loads whose data is used once (the non-temporal bit): tile
// records read by a single wavefront. They then no longer push X, which every
// unit re-reads, out of L2: the 70B FFN layer at 16 tokens takes 57.2 instead of
// 59.2 us, 13B attention 12.6 instead of 13.2. Records that several token
// groups read in turn keep the default policy, which lets the later groups find
// them in L2 (128 tokens: 166 against 170 us with the bit set).
constexpr int kCachePolicyStream = 2;
// Cache policy with the device-scope bit (sc1): coherent across the XCDs' L2s.
constexpr int kCachePolicyDevice = 16;

constexpr int kWaves = 4;                              // row blocks per workgroup
constexpr int kThreads = kWaves * kLanes;              // 256
constexpr int kGroupRows = kWaves * kTileRows;         // rows of a row group (64)
constexpr int kWRegionBytes = kMaxValBytes;            // 8 KB per wavefront (8 KB aligned)
constexpr int kXRowBytes = kTileK * 2 + 16;            // 528: padded token row of the X tile
constexpr int kMaxNT = 8;                              // 16-token blocks per pass (N <= 128)

struct SpmmArgs {
    const uint8_t *stream;
    const uint32_t *off;
    int64_t M, K, RB, KT;
    const uint16_t *X;
    int64_t ldx;
    uint16_t *Y;
    int64_t ldy;
    int N;            // tokens of this pass (<= 16 * NT)
    int64_t units;    // row groups * KT
    int64_t maxseg;   // partial slots per row group
    float *ws;        // partials [row group][slot][N][64], or null when no row group is split
    uint32_t *cnt;    // arrival counters, one per row group (zero between calls)
    int x_vec;        // X chunks may be read as 16-byte vectors
    int y_vec;        // Y may be written as 8-byte vectors
    const uint16_t *bias;  // fused epilogue (Epilogue): fp16 [M] or null
    const uint16_t *res;   // fp16 residual, token n at res + n * ldr, or null
    int64_t ldr;
    int act;               // usp_activation
};

// The fused epilogue of one output (row m, token n), in fp32: + bias, the
// activation, + residual. Arguments are uniform, so the branches are too.
template <class Args>
__device__ inline float epilogue(const Args &a, int n, int64_t m, float v) {
    if (a.bias) v += (float)__builtin_bit_cast(_Float16, a.bias[m]);
    if (a.act == 1) {
        v = v > 0.f ? v : 0.f;
    } else if (a.act == 2) {  // tanh form of GELU; sqrt(2 / pi) = 0.7978845608...
        v = 0.5f * v * (1.f + tanhf(0.7978845608028654f * (v + 0.044715f * v * v * v)));
    } else if (a.act == 3) {
        v = v / (1.f + expf(-v));
    }
    if (a.res) v += (float)__builtin_bit_cast(_Float16, a.res[(int64_t)n * a.ldr + m]);
    return v;
}

// Selector pair for expanding nibble `n` (positions 0..3) from the 4 packed
// halfs (c0,c1 | c2,c3) held in x0 | x1: output half j takes c_rank(j) when bit
// j is set and zero (selector byte 0x0c) otherwise.
__device__ inline uint2 nibble_selectors(uint32_t n) {
    uint32_t sel[2] = {0x0c0c0c0cu, 0x0c0c0c0cu};
    uint32_t r = 0;
    for (int j = 0; j < 4; ++j) {
        if (n & (1u << j)) {
            const uint32_t pair = (2 * r) | ((2 * r + 1) << 8);
            const int sh = 16 * (j & 1);
            sel[j >> 1] = (sel[j >> 1] & ~(0xFFFFu << sh)) | (pair << sh);
            ++r;
        }
    }
    return make_uint2(sel[0], sel[1]);
}

// The LDS words one step's decode needs: for each of the two nibbles, the three
// dwords holding its packed values and its selector pair, plus the byte
// offsets of both starts. Reading them for step s + 1 before finishing step s
// hides the LDS latency.
struct StepWords {
    uint32_t e[6];
    uint2 sel[2];
    uint32_t hb[2];
};

typedef const __attribute__((address_space(3))) uint32_t lds_u32;

// An LDS array seen as 32-bit words. Indexing the array itself (rather than an
// integer address) lets the compiler tell LDS arrays apart, which its waits for
// direct-to-LDS loads rely on.
__device__ inline lds_u32 *as_lds(const void *p) {
    return (lds_u32 *)(const __attribute__((address_space(3))) void *)p;
}

// region: the staged values. hb is the nibble's first byte (even); the three
// dwords from its dword hold its up to 4 values whatever its alignment. A read
// may run up to 12 bytes past the record's values, which every region leaves
// room for.
__device__ inline void read_nibble(lds_u32 *region, uint32_t hb, uint32_t idx8, const uint8_t *lut,
                                   uint32_t *e, uint2 &sel) {
    typedef const __attribute__((address_space(3))) uint8_t lds_u8;
    typedef volatile const __attribute__((address_space(3))) uint32_t lds_vu32;
    lds_vu32 *d = (lds_vu32 *)((lds_u8 *)region + (hb & ~3u));
    e[0] = d[0];
    e[1] = d[1];
    e[2] = d[2];
    sel = *reinterpret_cast<const uint2 *>(lut + idx8);
}

// Expands one nibble whose packed values start at byte hb (even) from its three
// dwords: a funnel shift aligns the 4 candidate halfs, then two byte permutes
// place them (or zeros) at the nibble's 4 positions.
__device__ inline void finish_nibble(const uint32_t *e, uint2 sel, uint32_t hb, uint32_t &o0, uint32_t &o1) {
    const uint32_t x0 = __builtin_amdgcn_alignbyte(e[1], e[0], hb);  // uses hb & 3 (0 or 2)
    const uint32_t x1 = __builtin_amdgcn_alignbyte(e[2], e[1], hb);
    o0 = __builtin_amdgcn_perm(x1, x0, sel.x);
    o1 = __builtin_amdgcn_perm(x1, x0, sel.y);
}

// Inclusive prefix sum over the 64 lanes of a wavefront (DPP row shifts and
// row broadcasts, 6 adds).
__device__ inline uint32_t wave_inclusive_scan(uint32_t v) {
    v += __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xF, 0xF, true);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xF, 0xF, true);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xF, 0xF, true);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xF, 0xF, true);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0u, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0u, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return v;
}

// Number of set bits of each 4-bit nibble of x, one count per nibble.
__device__ inline uint32_t nibble_popcounts(uint32_t x) {
    x = x - ((x >> 1) & 0x55555555u);
    return (x & 0x33333333u) + ((x >> 2) & 0x33333333u);
}

// Per-record decode state of one lane, from its mask word (byte s = step s).
// The record's values are 16 blocks, b = 2 s + h for step s and nibble half h
// (h = 0: positions 0-3, h = 1: positions 4-7), each holding the 64 lanes'
// values of that nibble in lane order. A lane's nibble (s, h) therefore starts
// at the block's start plus the lane's exclusive prefix of the block's kept
// counts: four DPP scans over 8-bit fields give every lane its prefix for all
// 16 blocks (at most 63 x 4 = 252, so the fields never carry), and lane 63's
// prefix plus its own count gives each block's size.
struct RecState {
    uint32_t excl[4];            // prefixes: [2 (s / 4) + h], field s % 4
    uint32_t base2[2 * kSteps];  // byte offset of block b (wavefront-uniform)
    uint32_t t[4];               // selector-table offsets (nibble x 8): [2 (s / 4) + h], byte s % 4
};

__device__ inline RecState rec_state(uint2 msk) {
    const uint32_t nx = nibble_popcounts(msk.x), ny = nibble_popcounts(msk.y);
    const uint32_t w[4] = {nx & 0x0F0F0F0Fu, (nx >> 4) & 0x0F0F0F0Fu, ny & 0x0F0F0F0Fu, (ny >> 4) & 0x0F0F0F0Fu};
    RecState o;
    uint32_t tot[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t inc = wave_inclusive_scan(w[i]);
        asm("" : "+v"(inc));     // keeps the scan's last add a DPP add (the optimizer would split it)
        o.excl[i] = inc - w[i];  // exact: lane 63's inclusive sum may carry, the difference does not
        // Block sizes: lane 63's prefix plus its own count, per field (up to 256), in 16-bit halves.
        const uint32_t x = __builtin_amdgcn_readlane(o.excl[i], 63), c = __builtin_amdgcn_readlane(w[i], 63);
        const uint32_t even = (x & 0x00FF00FFu) + (c & 0x00FF00FFu), odd = ((x >> 8) & 0x00FF00FFu) + ((c >> 8) & 0x00FF00FFu);
        tot[i][0] = even & 0xFFFFu;
        tot[i][1] = odd & 0xFFFFu;
        tot[i][2] = even >> 16;
        tot[i][3] = odd >> 16;
    }
    uint32_t run = 0;
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            o.base2[2 * st + h] = 2 * run;
            run += tot[2 * (st >> 2) + h][st & 3];
        }
    }
    uint32_t t0 = (msk.x << 3) & 0x78787878u, t1 = (msk.x >> 1) & 0x78787878u;
    uint32_t t2 = (msk.y << 3) & 0x78787878u, t3 = (msk.y >> 1) & 0x78787878u;
    // Opaque to the optimizer: a step's selector index is then one bit-field
    // extract of these words instead of a shift and a mask of the raw mask.
    asm("" : "+v"(t0), "+v"(t1), "+v"(t2), "+v"(t3));
    o.t[0] = t0;
    o.t[1] = t1;
    o.t[2] = t2;
    o.t[3] = t3;
    return o;
}

// Issues the LDS reads of step s of the staged record.
__device__ inline StepWords read_step(lds_u32 *region, const uint8_t *lut, const RecState &rs, int s) {
    StepWords w;
    const int f = 8 * (s & 3), q = 2 * (s >> 2);
    w.hb[0] = 2 * ((rs.excl[q] >> f) & 0xFFu) + rs.base2[2 * s];
    w.hb[1] = 2 * ((rs.excl[q + 1] >> f) & 0xFFu) + rs.base2[2 * s + 1];
    read_nibble(region, w.hb[0], (rs.t[q] >> f) & 0xFFu, lut, w.e, w.sel[0]);
    read_nibble(region, w.hb[1], (rs.t[q + 1] >> f) & 0xFFu, lut, w.e + 3, w.sel[1]);
    return w;
}

// The A operand (8 halfs) of a step from its LDS words.
__device__ inline half8 finish_step(const StepWords &w) {
    uint4 a;
    finish_nibble(w.e, w.sel[0], w.hb[0], a.x, a.y);
    finish_nibble(w.e + 3, w.sel[1], w.hb[1], a.z, a.w);
    return __builtin_bit_cast(half8, a);
}

__device__ inline half8 decode_step(lds_u32 *region, const uint8_t *lut, const RecState &rs, int s) {
    return finish_step(read_step(region, lut, rs, s));
}

// One 16-byte chunk X[n][k..k+7] of the X tile, zero outside N x K.
// XFAST: X is 16-byte aligned, ldx and K are multiples of 8, so a chunk is
// either entirely inside or entirely outside; the load is issued
// unconditionally (from a valid address) and zeroed afterwards, which keeps
// the number of loads per tile fixed. Otherwise element-wise guarded loads.
template <bool XFAST>
__device__ inline uint4 load_x_chunk(const SpmmArgs &a, int n, int64_t k) {
    const bool inside = n < a.N && k < a.K;
    if (XFAST) {
        const uint16_t *p = a.X + (inside ? (int64_t)n * a.ldx + k : 0);
        const uint4 v = *reinterpret_cast<const uint4 *>(p);
        return inside ? v : make_uint4(0, 0, 0, 0);
    }
    uint4 v = make_uint4(0, 0, 0, 0);
    if (!inside) return v;
    const uint16_t *p = a.X + (int64_t)n * a.ldx + k;
    uint16_t h[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = (k + j < a.K) ? p[j] : (uint16_t)0;
    v.x = h[0] | ((uint32_t)h[1] << 16);
    v.y = h[2] | ((uint32_t)h[3] << 16);
    v.z = h[4] | ((uint32_t)h[5] << 16);
    v.w = h[6] | ((uint32_t)h[7] << 16);
    return v;
}

// Rounds four consecutive rows m..m+3 of token n to fp16 (after the fused
// epilogue, if any) and stores those < M.
__device__ inline void store_y4(const SpmmArgs &a, int n, int64_t m, float v0, float v1, float v2, float v3) {
    if (a.bias || a.res || a.act) {
        if (m < a.M) v0 = epilogue(a, n, m, v0);
        if (m + 1 < a.M) v1 = epilogue(a, n, m + 1, v1);
        if (m + 2 < a.M) v2 = epilogue(a, n, m + 2, v2);
        if (m + 3 < a.M) v3 = epilogue(a, n, m + 3, v3);
    }
    const uint16_t h0 = __builtin_bit_cast(uint16_t, (_Float16)v0);
    const uint16_t h1 = __builtin_bit_cast(uint16_t, (_Float16)v1);
    const uint16_t h2 = __builtin_bit_cast(uint16_t, (_Float16)v2);
    const uint16_t h3 = __builtin_bit_cast(uint16_t, (_Float16)v3);
    uint16_t *dst = a.Y + (int64_t)n * a.ldy + m;
    if (a.y_vec && m + 4 <= a.M) {
        *reinterpret_cast<uint2 *>(dst) = make_uint2(h0 | ((uint32_t)h1 << 16), h2 | ((uint32_t)h3 << 16));
    } else {
        if (m < a.M) dst[0] = h0;
        if (m + 1 < a.M) dst[1] = h1;
        if (m + 2 < a.M) dst[2] = h2;
        if (m + 3 < a.M) dst[3] = h3;
    }
}

// Registers holding one prefetched tile: this lane's share of the X tile and of
// the wavefront's tile record.
// 16-byte chunks of an X tile of NT blocks of 16 tokens per thread.
template <int NT>
constexpr int kXTileChunks = NT * 16 * 32 / kThreads;

template <int NT>
struct TileRegs {
    uint4 x[kXTileChunks<NT>];
    uint4 w[8];
    uint2 msk;
    int nch;  // 16-byte chunks of packed values (wavefront-uniform)
};

// Issues the loads of tile (rb, kt) into r: this lane's X chunks, its mask
// word and the tile's packed values in 1 KB wavefront loads (as many as the
// record needs; lanes past the record's end read the bytes that follow it,
// which the device allocation pads, and those chunks are never used). The
// record offsets come from read-only memory through the scalar path.
template <int NT, bool XFAST>
__device__ inline void fetch_tile(const SpmmArgs &a, const uint32_t *__restrict__ off,
                                  const uint8_t *__restrict__ stream, int64_t rb, bool rb_ok, int64_t kt, int tid,
                                  int lane, TileRegs<NT> &r) {
#pragma unroll
    for (int i = 0; i < kXTileChunks<NT>; ++i) {
        const int c = tid + kThreads * i;
        r.x[i] = load_x_chunk<XFAST>(a, c >> 5, kt * kTileK + 8 * (c & 31));
    }
    const int64_t t = (rb_ok ? rb : 0) * a.KT + kt;
    const uint32_t o0 = off[t], o1 = off[t + 1];
    const uint8_t *rec = stream + (size_t)o0 * 16;
    r.msk = reinterpret_cast<const uint2 *>(rec)[lane];  // only used when rb_ok
    r.nch = rb_ok ? (int)(o1 - o0) - kMaskChunks : 0;
    const uint4 *vp = reinterpret_cast<const uint4 *>(rec + kMaskBytes);
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (kLanes * i < r.nch) r.w[i] = vp[lane + kLanes * i];
}

// Workgroup holding unit x when G workgroups split U units evenly: the largest
// w with floor(w U / G) <= x.
__device__ inline int64_t unit_owner(int64_t x, int64_t U, int64_t G) { return ((x + 1) * G - 1) / U; }

template <int NT>
__device__ inline void stage_tile(const TileRegs<NT> &r, uint8_t *xs, uint8_t *region, int tid, int lane) {
#pragma unroll
    for (int i = 0; i < kXTileChunks<NT>; ++i) {
        const int c = tid + kThreads * i;
        *reinterpret_cast<uint4 *>(xs + (c >> 5) * kXRowBytes + 16 * (c & 31)) = r.x[i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (kLanes * i < r.nch) reinterpret_cast<uint4 *>(region)[lane + kLanes * i] = r.w[i];
}

template <int NT>
__device__ inline void compute_tile(lds_u32 *region, const uint8_t *xs, const uint8_t *lut, uint2 msk, int lane,
                                    floatx4 (&acc)[NT]) {
    const RecState rs = rec_state(msk);
    const uint8_t *xb = xs + (lane & 15) * kXRowBytes + 16 * (lane >> 4);
    StepWords cur = read_step(region, lut, rs, 0);
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
        StepWords nxt;
        if (s + 1 < kSteps) nxt = read_step(region, lut, rs, s + 1);
        half8 bv[NT];
#pragma unroll
        for (int nb = 0; nb < NT; ++nb) bv[nb] = *reinterpret_cast<const half8 *>(xb + nb * 16 * kXRowBytes + 64 * s);
        const half8 av = finish_step(cur);
#pragma unroll
        for (int nb = 0; nb < NT; ++nb) acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv[nb], acc[nb], 0, 0, 0);
        if (s + 1 < kSteps) cur = nxt;
    }
}

// Finishes row group rg for the columns this workgroup accumulated in acc.
// Lane holds D[4*(lane/16) + i][lane % 16]: rows m0..m0+3 of token 16 nb + lane % 16.
template <int NT>
__device__ inline void flush_row_group(const SpmmArgs &a, int64_t rg, int64_t wg, int64_t G, int tid, int lane,
                                       int wave, const floatx4 (&acc)[NT], uint32_t *last_flag) {
    const int64_t rb = rg * kWaves + wave;
    const int64_t m0 = rb * kTileRows + 4 * (lane >> 4);
    const int64_t w_first = unit_owner(rg * a.KT, a.units, G);
    const int64_t w_last = unit_owner(rg * a.KT + a.KT - 1, a.units, G);
    if (w_first == w_last) {  // this workgroup covered every column of the row group
        if (rb >= a.RB) return;
#pragma unroll
        for (int nb = 0; nb < NT; ++nb) {
            const int n = 16 * nb + (lane & 15);
            if (n < a.N) store_y4(a, n, m0, acc[nb][0], acc[nb][1], acc[nb][2], acc[nb][3]);
        }
        return;
    }
    const int64_t nseg = w_last - w_first + 1;
    // Partials of this row group: [slot][token][kGroupRows rows] fp32, accessed through a
    // buffer resource with device-scope (sc1) cache policy: stores are written
    // through to the device-coherent level, loads read it.
    const int64_t slot_floats = (int64_t)a.N * kGroupRows;
    float *slot0 = a.ws + rg * a.maxseg * slot_floats;
    const __amdgpu_buffer_rsrc_t part =
        __builtin_amdgcn_make_buffer_rsrc(slot0, (short)0, (int)(nseg * slot_floats * 4), kBufferRsrcWord3);
    const int mine = (int)((wg - w_first) * slot_floats * 4);
    const int r0 = wave * kTileRows + 4 * (lane >> 4);  // row within the group
#pragma unroll
    for (int nb = 0; nb < NT; ++nb) {
        const int n = 16 * nb + (lane & 15);
        if (n >= a.N) continue;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, acc[nb]), part, mine + (n * kGroupRows + r0) * 4, 0,
                                               kCachePolicyDevice);
    }
    __builtin_amdgcn_s_waitcnt(0);  // every partial store acknowledged before the arrival is counted
    __syncthreads();
    if (tid == 0) {
        const uint32_t old = __hip_atomic_fetch_add(a.cnt + rg, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *last_flag = (old == (uint32_t)nseg - 1u);
    }
    __syncthreads();
    const bool last = *last_flag != 0;
    __syncthreads();  // the flag may be reused by the next flush
    if (!last) return;
    const int64_t row0 = rg * kWaves * kTileRows;
    constexpr int kItems = kGroupRows / 4;  // items of 4 consecutive rows per token
    for (int e = tid; e < kItems * a.N; e += kThreads) {
        const int n = e / kItems;
        const int r = 4 * (e % kItems);
        if (row0 + r >= a.RB * kTileRows) continue;
        floatx4 sum = {0.f, 0.f, 0.f, 0.f};
        for (int64_t j0 = 0; j0 < nseg; j0 += 8) {
            // Issue a batch of loads before adding, then add in slot order (fixed order:
            // bitwise reproducible).
            v4u32 v[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                v[jj] = j0 + jj < nseg ? __builtin_amdgcn_raw_buffer_load_b128(
                                             part, (int)((j0 + jj) * slot_floats * 4) + (n * kGroupRows + r) * 4, 0,
                                             kCachePolicyDevice)
                                       : v4u32{0u, 0u, 0u, 0u};
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                if (j0 + jj < nseg) sum += __builtin_bit_cast(floatx4, v[jj]);
        }
        store_y4(a, n, row0 + r, sum[0], sum[1], sum[2], sum[3]);
    }
    if (tid == 0) __hip_atomic_store(a.cnt + rg, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int NT, bool XFAST>
__global__ __launch_bounds__(kThreads, 8 / kWaves) void spmm_kernel(SpmmArgs a, const uint32_t *__restrict__ off,
                                                                   const uint8_t *__restrict__ stream) {
    // Wavefront regions first, 8 KB each, so a region offset can be masked; the
    // last region gets 16 bytes of read slack.
    __shared__ __attribute__((aligned(kWRegionBytes))) uint8_t wsm[kWaves * kWRegionBytes + 16];
    __shared__ __attribute__((aligned(16))) uint8_t xs[NT * 16 * kXRowBytes];
    __shared__ __attribute__((aligned(16))) uint8_t lut[16 * 8];
    __shared__ uint32_t last_flag;

    const int tid = threadIdx.x, lane = tid & 63;
    // Wavefront-uniform by construction; saying so lets the tile-offset lookups
    // be scalar loads, which do not wait on the vector loads in flight.
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t wg = blockIdx.x, G = gridDim.x;
    const int64_t u0 = wg * a.units / G, u1 = (wg + 1) * a.units / G;
    if (u0 >= u1) return;
    uint8_t *region = wsm + wave * kWRegionBytes;
    if (tid < 16) reinterpret_cast<uint2 *>(lut)[tid] = nibble_selectors((uint32_t)tid);

    floatx4 acc[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};

    // One tile in flight: while tile u is decoded from LDS, tile u + 1 is being
    // loaded into registers. (row group, column tile) advance incrementally.
    int64_t rg = u0 / a.KT;
    int64_t kt = u0 % a.KT;
    TileRegs<NT> buf;
    fetch_tile<NT, XFAST>(a, off, stream, rg * kWaves + wave, rg * kWaves + wave < a.RB, kt, tid, lane, buf);
    for (int64_t u = u0; u < u1; ++u) {
        const int64_t rb = rg * kWaves + wave;
        int64_t rgn = rg, ktn = kt + 1;
        if (ktn == a.KT) {
            ktn = 0;
            ++rgn;
        }
        const bool more = u + 1 < u1;
        const bool flush_now = !more || ktn == 0;
        const int64_t rbn = rgn * kWaves + wave;
        __syncthreads();  // every wavefront is done reading the previous tile
        stage_tile<NT>(buf, xs, region, tid, lane);
        const uint2 msk = buf.msk;
        __syncthreads();
        if (more && !flush_now) fetch_tile<NT, XFAST>(a, off, stream, rbn, rbn < a.RB, ktn, tid, lane, buf);
        if (rb < a.RB) compute_tile<NT>(as_lds(region), xs, lut, msk, lane, acc);
        if (flush_now) {
            // The flush waits for its own stores; fetching after it keeps that
            // wait from covering the next tile's loads as well.
            flush_row_group<NT>(a, rg, wg, G, tid, lane, wave, acc, &last_flag);
#pragma unroll
            for (int i = 0; i < NT; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
            if (more) fetch_tile<NT, XFAST>(a, off, stream, rbn, rbn < a.RB, ktn, tid, lane, buf);
        }
        rg = rgn;
        kt = ktn;
    }
}

// ---------------------------------------------------------------------------
// Shared parts of the single-pass kernels (up to 128 tokens): the column-chunk,
// direct-to-LDS and row-block kernels.
//
// All loads go through buffer resources (SGPR base, constant lane offsets,
// hardware zero-fill out of range). A record is read with L 1 KB loads, L
// being the smallest count that covers every record of the matrix; the
// resource ends at the record's own end, so the loads past it fetch nothing.
// The count per record is fixed, so the compiler's waits are exact.
// A row set whose column tiles are split over several wavefronts (or
// workgroups) is finished by the last to arrive: each stores its fp32 partial
// with device-coherent stores, counts its arrival once they are acknowledged,
// and the last arrival sums the partials in slot order.
// ---------------------------------------------------------------------------

struct WaveArgs {
    int64_t M, K, RB, KT;
    int64_t sets, units, maxseg;  // row sets; sets * KT; partial slots per row set
    const uint16_t *X;
    int64_t ldx;
    uint32_t x_bytes;             // readable bytes of X from its base
    uint16_t *Y;
    int64_t ldy;
    int N;
    float *ws;                    // partials [set][slot][token][16 R rows], or null
    uint32_t *cnt;                // arrival counters per row set and token group (zero between calls)
    int y_vec;
    int tg;                       // token groups: wavefronts that stream the same units
    const uint16_t *bias;         // fused epilogue (Epilogue): fp16 [M] or null
    const uint16_t *res;          // fp16 residual, token n at res + n * ldr, or null
    int64_t ldr;
    int act;                      // usp_activation
    const uint8_t *xp;            // X packed in product order (pack_x_kernel), or null
    uint32_t xp_bytes;
    int tb;                       // blocks of 16 tokens in xp: ceil(N / 16)
};

// Rows m..m+3 of token n (a lane's MFMA outputs), rounded to fp16 after the
// fused epilogue (if any), those < M.
__device__ inline void store_rows4(const WaveArgs &a, int n, int64_t m, const floatx4 &acc) {
    floatx4 v = acc;
    if (a.bias || a.res || a.act) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (m + i < a.M) v[i] = epilogue(a, n, m + i, v[i]);
    }
    const uint16_t h0 = __builtin_bit_cast(uint16_t, (_Float16)v[0]);
    const uint16_t h1 = __builtin_bit_cast(uint16_t, (_Float16)v[1]);
    const uint16_t h2 = __builtin_bit_cast(uint16_t, (_Float16)v[2]);
    const uint16_t h3 = __builtin_bit_cast(uint16_t, (_Float16)v[3]);
    uint16_t *dst = a.Y + (int64_t)n * a.ldy + m;
    if (a.y_vec && m + 4 <= a.M) {
        *reinterpret_cast<uint2 *>(dst) = make_uint2(h0 | ((uint32_t)h1 << 16), h2 | ((uint32_t)h3 << 16));
    } else {
        if (m < a.M) dst[0] = h0;
        if (m + 1 < a.M) dst[1] = h1;
        if (m + 2 < a.M) dst[2] = h2;
        if (m + 3 < a.M) dst[3] = h3;
    }
}

// Counts this wavefront's arrival at row set `set` for token group g (its
// partial must already be acknowledged); returns the counter's previous value
// (in lane 0).
__device__ inline uint32_t arrive_count(const WaveArgs &a, int64_t set, int lane, int g = 0) {
    uint32_t old = 0;
    if (lane == 0)
        old = __hip_atomic_fetch_add(a.cnt + set * a.tg + g, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return old;
}

// With the counter's previous value: the last of the nseg arrivals sums every
// slot in order for token group g's NB blocks of 16 tokens, stores Y and resets
// the counter.
template <int R, int NB = 1>
__device__ inline void arrive_finish(const WaveArgs &a, int64_t set, int64_t nseg, uint32_t old, int lane,
                                     int g = 0) {
    old = __builtin_amdgcn_readfirstlane(old);
    if (old != (uint32_t)nseg - 1u) return;
    const int64_t slot_floats = (int64_t)a.N * kTileRows * R;
    float *slot0 = a.ws + set * a.maxseg * slot_floats;
    const __amdgpu_buffer_rsrc_t part =
        __builtin_amdgcn_make_buffer_rsrc(slot0, (short)0, (int)(nseg * slot_floats * 4), kBufferRsrcWord3);
    const int g4 = 4 * (lane >> 4);
#pragma unroll 1
    for (int nb = 0; nb < NB; ++nb) {
        const int n = 16 * (NB * g + nb) + (lane & 15);
        if (n < a.N) {
            // Batches of B slots x R row blocks (16 loads), issued together, then
            // added in slot order per row block: one round trip for up to B slots.
            constexpr int B = R >= 16 ? 1 : 16 / R;
            floatx4 sum[R];
#pragma unroll
            for (int r = 0; r < R; ++r) sum[r] = floatx4{0.f, 0.f, 0.f, 0.f};
            const int lofs = (n * kTileRows * R + g4) * 4;
            for (int64_t j0 = 0; j0 < nseg; j0 += B) {
                v4u32 v[B][R];
#pragma unroll
                for (int jj = 0; jj < B; ++jj)
#pragma unroll
                    for (int r = 0; r < R; ++r)
                        v[jj][r] = j0 + jj < nseg ? __builtin_amdgcn_raw_buffer_load_b128(
                                                        part, (int)((j0 + jj) * slot_floats * 4) + lofs + 64 * r, 0,
                                                        kCachePolicyDevice)
                                                  : v4u32{0u, 0u, 0u, 0u};
#pragma unroll
                for (int jj = 0; jj < B; ++jj)
#pragma unroll
                    for (int r = 0; r < R; ++r)
                        if (j0 + jj < nseg) sum[r] += __builtin_bit_cast(floatx4, v[jj][r]);
            }
#pragma unroll
            for (int r = 0; r < R; ++r) store_rows4(a, n, (set * R + r) * kTileRows + g4, sum[r]);
        }
    }
    if (lane == 0) __hip_atomic_store(a.cnt + set * a.tg + g, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int R, int NB = 1>
__device__ inline void arrive_row_set(const WaveArgs &a, int64_t set, int64_t nseg, int lane, int g = 0) {
    arrive_finish<R, NB>(a, set, nseg, arrive_count(a, set, lane, g), lane, g);
}

// One tile record in registers: this lane's mask word and L KB of the packed
// values (16 bytes per lane per load).
template <int L>
struct WaveRec {
    v4u32 w[L];
    uint2 msk;
};

// Loads the record at 16-byte units [o0, o1) into registers.
template <int L>
__device__ inline void fetch_rec(const uint8_t *__restrict__ stream, uint32_t o0, uint32_t o1, int lane,
                                 WaveRec<L> &r) {
    const __amdgpu_buffer_rsrc_t rec = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(stream + (uint64_t)o0 * 16), (short)0, (int)((o1 - o0) * 16), kBufferRsrcWord3);
    r.msk = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rec, lane * 8, 0, kCachePolicyStream));
#pragma unroll
    for (int i = 0; i < L; ++i)
        r.w[i] = __builtin_amdgcn_raw_buffer_load_b128(rec, kMaskBytes + 1024 * i + lane * 16, 0, kCachePolicyStream);
}

// B operands of one tile: step s, lane (g = lane / 16, n = lane % 16) holds
// X[n][256 kt + 32 s + 8 g .. + 7]; zero for n >= N and for columns >= K, both
// by reading at or past the end of the X resource (the hardware returns
// zeros). Zeroing loaded registers instead would make the compiler wait for
// the newest loads on that path, and its waits on every path stricter.
__device__ inline void fetch_x(const WaveArgs &a, __amdgpu_buffer_rsrc_t xr, int xoff, int64_t kt, int lane,
                               v4u32 (&xb)[kSteps]) {
    const int base = xoff + (int)(kt * kTileK * 2);
    int at[kSteps];
#pragma unroll
    for (int s = 0; s < kSteps; ++s) at[s] = base + 64 * s;
    if ((kt + 1) * kTileK > a.K) {  // last, partial column tile
#pragma unroll
        for (int s = 0; s < kSteps; ++s)
            if (kt * kTileK + 32 * s + 8 * (lane >> 4) >= a.K) at[s] = (int)a.x_bytes;
    }
#pragma unroll
    for (int s = 0; s < kSteps; ++s) xb[s] = __builtin_amdgcn_raw_buffer_load_b128(xr, at[s], 0, 0);
}

// Issue the LDS reads of all 8 steps of a record before expanding any (more
// registers, shorter chain) instead of one step ahead: for 3 or more token
// blocks, where the direct-to-LDS kernel runs one wavefront per SIMD and
// nothing else hides the LDS latency (1-2% faster there, ~1% slower at one
// block).
constexpr int kDecodeAheadMinBlocks = 3;

// Decodes the record in `slot` (mask msk) against the tile's B operands.
template <int NB>
__device__ inline void decode_record(lds_u32 *slot, const uint8_t *lut, uint2 msk, const v4u32 (&xb)[NB][kSteps],
                                     floatx4 (&acc)[NB]) {
    const RecState rs = rec_state(msk);
    if (NB >= kDecodeAheadMinBlocks) {  // every step's LDS reads first: a short dependency chain per record
        StepWords all[kSteps];
#pragma unroll
        for (int s = 0; s < kSteps; ++s) all[s] = read_step(slot, lut, rs, s);
#pragma unroll
        for (int s = 0; s < kSteps; ++s) {
            const half8 av = finish_step(all[s]);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, __builtin_bit_cast(half8, xb[nb][s]), acc[nb], 0, 0, 0);
        }
        return;
    }
    StepWords sw = read_step(slot, lut, rs, 0);
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
        StepWords nx;
        if (s + 1 < kSteps) nx = read_step(slot, lut, rs, s + 1);
        const half8 av = finish_step(sw);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, __builtin_bit_cast(half8, xb[nb][s]), acc[nb], 0, 0, 0);
        if (s + 1 < kSteps) sw = nx;
    }
}

// ---------------------------------------------------------------------------
// Column-chunk kernel for small matrices (up to 32 tokens).
//
// A workgroup of W wavefronts (4 or 8) takes W consecutive row blocks and a
// chunk of C consecutive column tiles. The chunk's X columns (NB blocks of 16
// tokens x 256 C halfs) are staged in LDS once, behind the kernel's only
// barrier; every decoded step feeds NB MFMAs. Each
// wavefront reads the offsets of its C records with one vector load and issues
// the loads of all C records before decoding the first: on layers this small a
// wavefront has only a few records, and their round trips, not the HBM rate,
// set the time, so the wavefront waits about one record's latency instead of
// one per record (plus one per offset-table entry). The records stay in
// registers until their turn, then are staged in the wavefront's own LDS region
// and decoded. The chunks of a row block are summed through the workspace by
// the last to arrive, in chunk order.
// ---------------------------------------------------------------------------

constexpr int kChunkTiles = 4;                             // C
constexpr int kMaxChunkTokenBlocks = 2;                    // NB
constexpr int kChunkXRow = kChunkTiles * kTileK * 2 + 16;  // padded token row of the chunk's X (bytes)

template <int L, int W, int NB>
__global__ __launch_bounds__(W * kLanes) void spmm_chunk_kernel(WaveArgs a, const uint32_t *__restrict__ off,
                                                                 const uint8_t *__restrict__ stream) {
    constexpr int C = kChunkTiles;
    constexpr int kRegion = 1024 * L + 16;  // staged values + the decode's 12-byte overread
    constexpr int kXLoads = NB * 16 * 32 * C / (W * kLanes);  // 16-byte X chunks per thread
    // One LDS array: the selector table at its start and the wavefronts'
    // regions right after it, so that both addresses fit the offset fields of
    // the decode's LDS reads and cost no instruction per read; the chunk's X
    // last.
    __shared__ __attribute__((aligned(16))) uint8_t smem[16 * 8 + W * kRegion + NB * 16 * kChunkXRow];
    uint8_t *const lut = smem;
    uint8_t *const regions = smem + 16 * 8;
    uint8_t *const xs = regions + W * kRegion;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int64_t S = a.maxseg;  // chunks per row block
    const int64_t rg = blockIdx.x / S, seg = blockIdx.x % S;
    const int64_t rb = rg * W + wave, kt0 = seg * C;
    const int nct = (int)(a.KT - kt0 < C ? a.KT - kt0 : C);

    // X of the chunk: token n, 16-byte chunk c of its C * 256 columns; zero for
    // tokens >= N and columns >= K (read at the resource's end).
    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.X, (short)0, (int)a.x_bytes, kBufferRsrcWord3);
    v4u32 xv[kXLoads];
#pragma unroll
    for (int i = 0; i < kXLoads; ++i) {
        const int q = tid + W * kLanes * i, n = q / (32 * C), c = q % (32 * C);
        const int64_t col = kt0 * kTileK + 8 * c;
        const int at = (n < a.N && col < a.K) ? (int)((n * a.ldx + col) * 2) : (int)a.x_bytes;
        xv[i] = __builtin_amdgcn_raw_buffer_load_b128(xr, at, 0, 0);
    }
    // Lane j <= nct: offset-table entry j of the wavefront's records.
    const __amdgpu_buffer_rsrc_t offr =
        __builtin_amdgcn_make_buffer_rsrc((void *)off, (short)0, (int)((a.RB * a.KT + 1) * 4), kBufferRsrcWord3);
    const bool real = rb < a.RB && lane <= nct;
    const uint32_t ov =
        __builtin_amdgcn_raw_buffer_load_b32(offr, real ? (int)((rb * a.KT + kt0 + lane) * 4) : 0x7FFFFFF0, 0, 0);
#pragma unroll
    for (int i = 0; i < kXLoads; ++i) {
        const int q = tid + W * kLanes * i, n = q / (32 * C), c = q % (32 * C);
        *reinterpret_cast<v4u32 *>(xs + n * kChunkXRow + 16 * c) = xv[i];
    }
    if (tid < 16) reinterpret_cast<uint2 *>(lut)[tid] = nibble_selectors((uint32_t)tid);
    // The barrier comes before the records are requested: a wavefront issuing
    // its record loads can stall for microseconds while the memory system
    // drains, and its workgroup would wait for that at the barrier.
    __syncthreads();
    if (rb >= a.RB) return;
    WaveRec<L> rec[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const uint32_t o0 = __builtin_amdgcn_readlane(ov, j);
        const uint32_t o1 = j < nct ? __builtin_amdgcn_readlane(ov, j + 1) : o0;  // past the chunk: empty
        fetch_rec<L>(stream, o0, o1, lane, rec[j]);
    }

    uint8_t *const region = regions + wave * kRegion;
    lds_u32 *const rbase = as_lds(region);
    const int n_lane = lane & 15, g4 = 4 * (lane >> 4);
    const uint8_t *const xrow = xs + n_lane * kChunkXRow + 2 * 8 * (lane >> 4);
    floatx4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < C; ++j) {
        if (j < nct) {
            // In-order LDS: the previous decode's reads of the region are done.
#pragma unroll
            for (int i = 0; i < L; ++i) reinterpret_cast<v4u32 *>(region)[lane + kLanes * i] = rec[j].w[i];
            v4u32 xb[NB][kSteps];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int s = 0; s < kSteps; ++s)
                    xb[nb][s] = *reinterpret_cast<const v4u32 *>(xrow + nb * 16 * kChunkXRow + 2 * (j * kTileK + 32 * s));
            decode_record<NB>(rbase, lut, rec[j].msk, xb, acc);
        }
    }
    if (S == 1) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            if (16 * nb + n_lane < a.N) store_rows4(a, 16 * nb + n_lane, rb * kTileRows + g4, acc[nb]);
        return;
    }
    const int64_t slot_floats = (int64_t)a.N * kTileRows;
    float *slot = a.ws + (rb * S + seg) * slot_floats;
    const __amdgpu_buffer_rsrc_t part =
        __builtin_amdgcn_make_buffer_rsrc(slot, (short)0, (int)(slot_floats * 4), kBufferRsrcWord3);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int n = 16 * nb + n_lane;
        if (n < a.N)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, acc[nb]), part, (n * kTileRows + g4) * 4,
                                                   0, kCachePolicyDevice);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the partials are acknowledged before the arrival counts
    arrive_row_set<1, NB>(a, rb, S, lane);
}

// ---------------------------------------------------------------------------
// Direct-to-LDS kernel (4 row blocks per unit).
//
// Records are loaded by buffer-to-LDS transfers into a ring of four LDS slots,
// one per row block of the unit, so three records are in flight while one is
// decoded and no VGPRs hold them. Each slot is its own LDS array: the compiler
// waits for exactly the transfers into the slot a decode reads. The next unit's
// X operands are loaded into a second register buffer during the unit (except
// at 2 token blocks, see below).
// More tokens than one wavefront's registers hold X for are split into token
// groups: tg wavefronts stream the same units, each for its own NB blocks of 16
// tokens, and decode every record. Workgroups are dispatched to the eight XCDs
// in turn, so the group's wavefronts are placed 8 blocks apart: they share one
// XCD's L2, and the records they all read come from HBM about once.
// ---------------------------------------------------------------------------

constexpr int kDmaRows = 4;  // row blocks per unit = LDS slots

// Whether records travel into LDS whole, mask bytes included (one and two
// token blocks, two wavefronts per SIMD), or the mask word of each lane comes
// by its own load into registers (three and four blocks, one wavefront per
// SIMD, where reading the mask from LDS would put one more LDS round trip in
// front of every record's decode: 107.6 against 104.1 us on the 70B FFN layer
// at 64 tokens).
__host__ __device__ constexpr bool dma_mask_in_lds(int nb) { return nb <= 2; }

// Encoding of s_waitcnt that waits until at most n vector memory operations
// are outstanding and ignores the other counters.
__device__ constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

// Record extents (16-byte units) of the R row blocks of unit (set, kt): lane r
// (r < R) holds the start of row block r's record and lane R + r its end; a
// row block past the matrix gets an empty extent. One vector load per unit,
// issued a unit before use, so its latency never stalls the stream (a scalar
// load here waited on the scalar cache for every record).
__device__ inline uint32_t unit_offsets(const WaveArgs &a, __amdgpu_buffer_rsrc_t offr, int64_t set, int64_t kt,
                                        int lane, bool valid = true) {
    const int64_t rb = set * kDmaRows + lane % kDmaRows;
    const bool real = valid && lane < 2 * kDmaRows && rb < a.RB;
    const int byte = real ? (int)((rb * a.KT + kt + (lane >= kDmaRows)) * 4) : 0x7FFFFFF0;  // out of range: 0
    return __builtin_amdgcn_raw_buffer_load_b32(offr, byte, 0, 0);
}

// Loads the whole record at 16-byte units [o0, o1), mask bytes and values,
// into an LDS slot: L transfers of 16 bytes per lane. The mask comes with the
// values rather than by a separate load into registers: the compiler's wait
// for such a load at the top of the unit loop (merged over the loop's entry
// and back edge) also waited for the next record, which cost ~6% on the 70B
// FFN layer.
// Without MASK_IN_LDS the slot receives the values only and msk this lane's
// mask word. The whole-record form serves one and two token blocks, where each
// record is read by one wavefront: it streams (kCachePolicyStream).
template <int L, bool MASK_IN_LDS>
__device__ inline void dma_rec(const uint8_t *__restrict__ stream, uint32_t o0, uint32_t o1, int lane,
                               uint8_t *slot, uint2 &msk) {
    const __amdgpu_buffer_rsrc_t rec = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(stream + (uint64_t)o0 * 16), (short)0, (int)((o1 - o0) * 16), kBufferRsrcWord3);
    constexpr int first = MASK_IN_LDS ? 0 : kMaskBytes;
    constexpr int policy = MASK_IN_LDS ? kCachePolicyStream : 0;
    if (!MASK_IN_LDS) msk = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rec, lane * 8, 0, 0));
#pragma unroll
    for (int i = 0; i < L; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rec, (__attribute__((address_space(3))) void *)(slot + 1024 * i), 16,
                                                 first + 1024 * i + lane * 16, 0, 0, policy);
}

// This lane's mask word of the record staged in `slot`.
__device__ inline uint2 slot_mask(const uint8_t *slot, int lane) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    typedef const __attribute__((address_space(3))) u32x2 lds_u32x2;
    const u32x2 m = ((lds_u32x2 *)(const __attribute__((address_space(3))) void *)slot)[lane];
    return make_uint2(m.x, m.y);
}


// NB blocks of 16 tokens: each decoded step feeds NB MFMAs.
template <int L, int NB>
__global__ __launch_bounds__(kLanes) void spmm_dma_kernel(WaveArgs a, const uint32_t *__restrict__ off,
                                                         const uint8_t *__restrict__ stream) {
    constexpr int R = kDmaRows;
    constexpr bool kMaskInLds = dma_mask_in_lds(NB);
    constexpr int kValues = kMaskInLds ? kMaskBytes : 0;  // where the values start in a slot
    constexpr int kSlot = 1024 * L + 16;  // (mask bytes,) values and the decode's 12-byte overread
    __shared__ __attribute__((aligned(16))) uint8_t slot0[kSlot];
    __shared__ __attribute__((aligned(16))) uint8_t slot1[kSlot];
    __shared__ __attribute__((aligned(16))) uint8_t slot2[kSlot];
    __shared__ __attribute__((aligned(16))) uint8_t slot3[kSlot];
    __shared__ __attribute__((aligned(16))) uint8_t lut[16 * 8];
    uint8_t *const slots[4] = {slot0, slot1, slot2, slot3};  // indexed by constants < R only
    const int lane = threadIdx.x;
    // Block b: unit range w of G, token group g (the grid is a multiple of 8 tg).
    const int64_t b = blockIdx.x, G = gridDim.x / a.tg;
    const int g = (int)((b >> 3) % a.tg);
    const int64_t w = (b / (8 * a.tg)) * 8 + (b & 7);
    const int64_t u0 = w * a.units / G, u1 = (w + 1) * a.units / G;
    if (u0 >= u1) return;
    if (lane < 16) reinterpret_cast<uint2 *>(lut)[lane] = nibble_selectors((uint32_t)lane);

    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.X, (short)0, (int)a.x_bytes, kBufferRsrcWord3);
    const int n_lane = lane & 15, g4 = 4 * (lane >> 4);
    // Lanes of tokens >= N start at the resource's end: their loads return zeros.
    const int tok0 = 16 * NB * g;  // first token of this wavefront's group
    int xoff[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int tok = tok0 + 16 * nb + n_lane;
        xoff[nb] = tok < a.N ? (int)(tok * a.ldx * 2) + 16 * (lane >> 4) : (int)a.x_bytes;
    }

    floatx4 acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    int64_t set = u0 / a.KT, kt = u0 % a.KT;
    int64_t pend_set = -1, pend_nseg = 0;  // partial stored, arrival not yet counted
    uint2 msk[R];  // mask words, when they come by their own loads
    const __amdgpu_buffer_rsrc_t offr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)off, (short)0, (int)((a.RB * a.KT + 1) * 4), kBufferRsrcWord3);
    // The first unit's records 0..R-2 and X; record R-1 is requested while record 0
    // is decoded, and from then on the next unit's record r - 1 while record r is.
    uint32_t oc = unit_offsets(a, offr, set, kt, lane);
    uint32_t on;  // the next unit's extents (empty past the range's end)
    {
        int64_t s1 = set, k1 = kt + 1;
        if (k1 == a.KT) {
            k1 = 0;
            ++s1;
        }
        on = unit_offsets(a, offr, s1, k1, lane, u0 + 1 < u1);
    }
    // With whole records in LDS, X first: the compiler's wait counts at the
    // loop head merge this path with the loop's own, where X is older than
    // every record in flight. With separate mask loads (3-4 token blocks, 32 KB
    // of X per wavefront) the records first: 104 against 107 us on the 70B FFN
    // layer at 64 tokens.
    v4u32 xb[NB][kSteps];
    if (kMaskInLds) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) fetch_x(a, xr, xoff[nb], kt, lane, xb[nb]);
    }
#pragma unroll
    for (int r = 0; r < R - 1; ++r)
        dma_rec<L, kMaskInLds>(stream, __builtin_amdgcn_readlane(oc, r), __builtin_amdgcn_readlane(oc, R + r), lane,
                               slots[r], msk[r]);
    if (!kMaskInLds) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) fetch_x(a, xr, xoff[nb], kt, lane, xb[nb]);
    }
    for (int64_t u = u0; u < u1; ++u) {
        // Two wavefronts share most SIMDs, and issue arbitration favours the
        // older: with equal ranges the younger finished ~5 us after it (70B FFN
        // layer, 16 tokens). Raising the priority on every other unit gives both
        // about the same share of issue slots.
        if (NB <= 2) {
            if (u & 1)
                __builtin_amdgcn_s_setprio(1);
            else
                __builtin_amdgcn_s_setprio(0);
        }
        int64_t setn = set, ktn = kt + 1;
        if (ktn == a.KT) {
            ktn = 0;
            ++setn;
        }
        const bool more = u + 1 < u1;
        const int64_t kp = more ? ktn : kt;  // X of the next unit (past the range's end: this one's, unused)
        // The next unit's X is loaded into a second buffer while this unit is
        // decoded, except at two token blocks: there the second buffer would
        // cost the second wavefront per SIMD, so the one buffer is reloaded
        // after the unit's last decode and the next unit waits for it. (At 3 and
        // 4 blocks the kernel runs one wavefront per SIMD anyway, and the second
        // buffer fits the 512 registers: 404 and 490, no spills.)
        constexpr bool kXAhead = NB != 2;
        v4u32 xn[kXAhead ? NB : 1][kSteps];
        uint32_t old = 0;
        // Extents of the unit after next: loaded a whole unit before use.
        uint32_t onn;
        {
            int64_t s2 = setn, k2 = ktn + 1;
            if (k2 == a.KT) {
                k2 = 0;
                ++s2;
            }
            onn = unit_offsets(a, offr, s2, k2, lane, u + 2 < u1);  // past the range: empty extents
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            // The next unit's X is requested first in the unit, ahead of every
            // record it will be used with: loads complete in issue order, so a
            // later request would make the next unit's first decode wait for the
            // records issued before it as well.
            if (kXAhead && r == 0) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) fetch_x(a, xr, xoff[nb], kp, lane, xn[kXAhead ? nb : 0]);
            }
            // Arrival at the row set finished by the previous unit: its partial's
            // stores were followed by the offsets load, the next unit's X (8 loads
            // per token block, when prefetched) and record R-1's L (+ 1 for a
            // separate mask) loads; the counter's answer is read a record or two
            // later, so waiting for it stalls nothing.
            if (r == 1 && pend_set >= 0) {
                __builtin_amdgcn_s_waitcnt(vmcnt_only(kXAhead ? L + (kMaskInLds ? 1 : 2) + kSteps * NB : L + 1));
                old = arrive_count(a, pend_set, lane, g);
            }
            if (r == R - 1 && pend_set >= 0) {
                arrive_finish<R, NB>(a, pend_set, pend_nseg, old, lane, g);
                pend_set = -1;
            }
            if (r == 0)
                dma_rec<L, kMaskInLds>(stream, __builtin_amdgcn_readlane(oc, R - 1),
                                       __builtin_amdgcn_readlane(oc, 2 * R - 1), lane, slots[R - 1], msk[R - 1]);
            else
                dma_rec<L, kMaskInLds>(stream, __builtin_amdgcn_readlane(on, r - 1),
                                       __builtin_amdgcn_readlane(on, R + r - 1), lane, slots[r - 1], msk[r - 1]);
            decode_record<NB>(as_lds(slots[r] + kValues), lut, kMaskInLds ? slot_mask(slots[r], lane) : msk[r], xb,
                              acc[r]);
        }
        if (!kXAhead) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) fetch_x(a, xr, xoff[nb], kp, lane, xb[nb]);
        }

        if (!more || ktn == 0) {  // end of this wavefront's segment of the row set
            const int64_t w_first = unit_owner(set * a.KT, a.units, G);
            const int64_t w_last = unit_owner(set * a.KT + a.KT - 1, a.units, G);
            if (w_first == w_last) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int tok = tok0 + 16 * nb + n_lane;
                    if (tok < a.N) {
#pragma unroll
                        for (int r = 0; r < R; ++r) store_rows4(a, tok, (set * R + r) * kTileRows + g4, acc[r][nb]);
                    }
                }
            } else {
                const int64_t slot_floats = (int64_t)a.N * kTileRows * R;
                float *part_slot = a.ws + (set * a.maxseg + (w - w_first)) * slot_floats;
                const __amdgpu_buffer_rsrc_t part = __builtin_amdgcn_make_buffer_rsrc(
                    part_slot, (short)0, (int)(slot_floats * 4), kBufferRsrcWord3);
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int tok = tok0 + 16 * nb + n_lane;
                    if (tok < a.N) {
#pragma unroll
                        for (int r = 0; r < R; ++r)
                            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, acc[r][nb]), part,
                                                                   (tok * kTileRows * R + kTileRows * r + g4) * 4, 0,
                                                                   kCachePolicyDevice);
                    }
                }
                pend_set = set;
                pend_nseg = w_last - w_first + 1;
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
        if (kXAhead) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int i = 0; i < kSteps; ++i) xb[nb][i] = xn[kXAhead ? nb : 0][i];
        }
        oc = on;
        on = onn;
        set = setn;
        kt = ktn;
    }
    __builtin_amdgcn_s_waitcnt(0);  // also drains the unused prefetches of the range's end
    if (pend_set >= 0) arrive_row_set<R, NB>(a, pend_set, pend_nseg, lane, g);
}

// ---------------------------------------------------------------------------
// Shared-decode kernel (33 to 256 tokens on large layers).
//
// A workgroup of four wavefronts streams a contiguous range of units (4 row
// blocks x 1 column tile). Wavefront j owns row block j of every unit: it
// moves that record into its own two LDS ring slots (the transfer of unit
// u + 2 is issued at the end of unit u), decodes it once into the 8 A operands
// of its steps and writes them to a shared LDS buffer; after a barrier every
// wavefront multiplies all four records' operands with the X of its own slice
// of tokens (NB blocks of 16, up to 64 tokens, held in registers; X read from
// the packed copy). Each record is decoded once however many tokens there
// are: the direct-to-LDS kernel's token groups decoded every record once per
// group (2 at 128 tokens, 4 at 256). The steps run outermost, so each step's X
// operands are reloaded for the next unit as soon as its last MFMA has been
// issued, 7 steps of MFMAs ahead of their use. Split row sets are finished per
// wavefront through the token-group arrival protocol (counter and partial
// slices per wavefront).
// ---------------------------------------------------------------------------

constexpr int kShareWaves = 4;  // wavefronts per workgroup = row blocks per unit

// Workgroup barrier ordering LDS reads and writes only. __syncthreads() is a
// workgroup fence, and a fence that covers LDS also waits for every
// direct-to-LDS transfer in flight, which would drain the record ring at every
// barrier; here this wavefront's LDS instructions complete (lgkmcnt) before
// the barrier, and the clobber keeps the compiler from moving memory accesses
// across it. Transfers into a ring slot are only ever read by the wavefront
// that issued them, behind its own hand-counted wait.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ---------------------------------------------------------------------------
// X packed in the order the shared-decode kernel's products read it. Read in
// place, each B-operand load of 64 lanes x 16 bytes touches 16 token rows (64
// bytes of each, at the row stride of X); the memory pipeline handles such a
// load at a quarter of the rate of one contiguous kilobyte, and at 64 and more
// tokens those loads, not the decode or the products, set the shared-decode
// kernel's pace (measured: the same kernel with contiguous loads of the same
// count, 152.6 -> 112.9 us on the 70B FFN layer at 128 tokens). One pass
// before the product rewrites X as blocks of 1 KB: block ((kt * 8 + s) * TB +
// tb), lane l = 16 g + n, holds X[16 tb + n][256 kt + 32 s + 8 g .. + 7]
// (zeros past N and K), so every load in the product reads one block.
// ---------------------------------------------------------------------------

constexpr size_t kPackBlockBytes = 1024;
static size_t packed_x_bytes(int64_t KT, int64_t N) {
    return (size_t)KT * kSteps * (size_t)((N + 15) / 16) * kPackBlockBytes;
}

// One wavefront per (column tile, token block): its 8 steps' blocks. Needs
// K % 8 == 0, ldx % 8 == 0 and X 16-byte aligned (the single-pass kernels'
// conditions).
__global__ __launch_bounds__(kLanes) void pack_x_kernel(const uint16_t *__restrict__ X, int64_t ldx, int N, int64_t K,
                                                       int TB, uint8_t *__restrict__ xp) {
    const int lane = threadIdx.x;
    const int64_t kt = blockIdx.x / TB, tb = blockIdx.x % TB;
    const int64_t n = 16 * tb + (lane & 15);
    const int64_t k0 = kt * kTileK + 8 * (lane >> 4);
    v4u32 v[kSteps];
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
        const int64_t k = k0 + 32 * st;
        v[st] = n < N && k < K ? *reinterpret_cast<const v4u32 *>(X + n * ldx + k) : v4u32{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int st = 0; st < kSteps; ++st)
        reinterpret_cast<v4u32 *>(xp + ((kt * kSteps + st) * TB + tb) * kPackBlockBytes)[lane] = v[st];
}

// Loads the whole record at 16-byte units [o0, o1) into LDS at byte address
// `lds` (L transfers of 16 bytes per lane, non-temporal), issued from inline
// assembly: the compiler neither sees these loads nor waits for them, so the
// caller waits for them itself (s_waitcnt vmcnt, counting every vector memory
// instruction issued after them). The compiler's own waits for transfers into
// LDS arrays it can tell apart are exact only while at most 8 such arrays are in
// play and their index is a constant; a ring shared by the wavefronts of a
// workgroup, indexed by wavefront, made it wait for every transfer in flight.
typedef int v4i32 __attribute__((ext_vector_type(4)));
template <int L>
__device__ inline void dma_rec_asm(const uint8_t *__restrict__ stream, uint32_t o0, uint32_t o1, int lane,
                                   uint32_t lds) {
    const uint64_t base = reinterpret_cast<uint64_t>(stream) + (uint64_t)o0 * 16;
    const v4i32 rsrc = {(int)(uint32_t)base, (int)((uint32_t)(base >> 32) & 0xFFFFu), (int)((o1 - o0) * 16),
                        kBufferRsrcWord3};
#pragma unroll
    for (int i = 0; i < L; ++i)
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
                     :
                     : "s"(lds + 1024u * i), "v"(1024 * i + lane * 16), "s"(rsrc)
                     : "memory", "m0");
}

// Calls f(std::integral_constant<int, P>{}) for P = 0, 1, ...: an unrolled loop
// whose index is a constant in every copy, however large the body.
template <class F, int... P>
__device__ __attribute__((always_inline)) inline void static_for(F &&f, std::integer_sequence<int, P...>) {
    (f(std::integral_constant<int, P>{}), ...);
}

// Ring depth of the shared-decode kernel: two slots per wavefront (one unit
// in flight while one is decoded).
constexpr int kShareSlots = 2;

// Up to 2 token blocks the launch bound asks for two workgroups per CU (at most
// 256 registers: 238 at 2 blocks, no spills; 272 without the bound, one
// workgroup per CU, 174 against 154 us on the 70B FFN at 128 tokens).
template <int L, int NB>
__global__ __launch_bounds__(kShareWaves *kLanes, NB <= 2 ? 2 : 1) void spmm_share_kernel(
    WaveArgs a, const uint32_t *__restrict__ off, const uint8_t *__restrict__ stream) {
    constexpr int R = kShareWaves;
    constexpr int S = kShareSlots;
    constexpr int kSlot = 1024 * L + 16;  // mask bytes, values and the decode's 12-byte overread
    // One LDS object per ring position: the compiler then waits only for the
    // transfers into the slot a decode reads.
    __shared__ __attribute__((aligned(16))) uint8_t ring0[R][kSlot];
    __shared__ __attribute__((aligned(16))) uint8_t ring1[R][kSlot];
    __shared__ __attribute__((aligned(16))) uint4 abuf[R][kSteps][kLanes];  // decoded A operands of the unit
    __shared__ __attribute__((aligned(16))) uint8_t lut[16 * 8];
    uint8_t *const ring[2] = {ring0[0], ring1[0]};
    const int lane = threadIdx.x & (kLanes - 1);
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    const int64_t w = blockIdx.x, G = gridDim.x;
    const int64_t u0 = w * a.units / G, u1 = (w + 1) * a.units / G;
    if (u0 >= u1) return;  // the whole workgroup
    if (threadIdx.x < 16) reinterpret_cast<uint2 *>(lut)[threadIdx.x] = nibble_selectors((uint32_t)threadIdx.x);

    // X packed in product order: this wavefront's blocks of step st of column
    // tile kt start at ((kt * kSteps + st) * TB + NB j) KB (blocks past the
    // tokens are only read by wavefronts that issue no products).
    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.xp, (short)0, (int)a.xp_bytes, kBufferRsrcWord3);
    const __amdgpu_buffer_rsrc_t offr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)off, (short)0, (int)((a.RB * a.KT + 1) * 4), kBufferRsrcWord3);
    const int n_lane = lane & 15, g4 = 4 * (lane >> 4);
    const int tok0 = 16 * NB * j;  // first token of this wavefront's slice
    const bool has_tokens = tok0 < a.N;
    const int xlane = (NB * j * 64 + lane) * 16;
    auto x_at = [&](int64_t kx, int st, int nb) -> int {
        return (int)((kx * kSteps + st) * a.tb + nb) * (int)kPackBlockBytes + xlane;
    };
    // Extents of this wavefront's record of the unit at (set, kt): lane 0 its
    // start, lane 1 its end; empty past the range (real false) or the matrix.
    auto rec_offsets = [&](int64_t set, int64_t kt, bool real) -> uint32_t {
        const int64_t rb = set * R + j;
        const bool ok = real && lane < 2 && rb < a.RB;
        return __builtin_amdgcn_raw_buffer_load_b32(offr, ok ? (int)((rb * a.KT + kt + lane) * 4) : 0x7FFFFFF0, 0, 0);
    };
    auto advance = [&](int64_t &set, int64_t &kt) {
        if (++kt == a.KT) {
            kt = 0;
            ++set;
        }
    };
    auto dma = [&](uint8_t *slot, uint32_t o) {
        const uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t *)slot);
        dma_rec_asm<L>(stream, __builtin_amdgcn_readlane(o, 0), __builtin_amdgcn_readlane(o, 1), lane, lds);
    };
    // Vector memory instructions issued after this wavefront's transfer of a
    // unit's record and before its decode, on the path with the fewest: the
    // transfer is issued at the end of the unit two before; then the next unit's
    // offset load (1), its X loads (kSteps NB) and its own transfer (L), and this
    // unit's offset load (1). Waiting until at most one fewer remain outstanding
    // finishes the transfer (in-order completion); partial stores and arrivals
    // add instructions, which only makes the wait stricter. In the first unit
    // the prologue's second transfer, X and the offset load follow it:
    // L + kSteps NB + 1, the same count.
    constexpr int kRecWait = kSteps * NB + L + 1 < 63 ? kSteps * NB + L + 1 : 63;

    floatx4 acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    // Prologue: the offsets of units u0 .. u0 + 2, the records of u0 and u0 + 1,
    // then X (the order kRecWait counts). onext: the unit requested at the end
    // of the current one (two ahead).
    int64_t set = u0 / a.KT, kt = u0 % a.KT;
    int64_t la_set = set, la_kt = kt;  // the unit whose offsets are loaded next
    const uint32_t oa = rec_offsets(la_set, la_kt, true);
    advance(la_set, la_kt);
    const uint32_t ob = rec_offsets(la_set, la_kt, u0 + 1 < u1);
    advance(la_set, la_kt);
    uint32_t onext = rec_offsets(la_set, la_kt, u0 + 2 < u1);
    advance(la_set, la_kt);
    dma(ring[0] + j * kSlot, oa);
    dma(ring[1] + j * kSlot, ob);
    // X of the first unit, step by step as the loop loads it (the compiler's
    // waits at the loop head assume the loop's order on both paths).
    v4u32 xb[NB][kSteps];
    {
#pragma unroll
        for (int st = 0; st < kSteps; ++st)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) xb[nb][st] = __builtin_amdgcn_raw_buffer_load_b128(xr, x_at(kt, st, nb), 0, 0);
    }
    lds_barrier();  // the selector table

    // A split row set's partial is stored at the end of the unit that finishes
    // this workgroup's segment; the arrival is counted at the end of the next
    // unit, once the stores are acknowledged, and the counter's answer used at
    // the end of the unit after that (the last arrival then sums the partials):
    // neither wait then stalls. Whatever is pending is settled after the loop.
    int64_t pend_set = -1, pend_nseg = 0;  // stored, not yet counted
    int64_t cnt_set = -1, cnt_nseg = 0;    // counted, answer in cnt_old
    uint32_t cnt_old = 0;
    // Vector memory instructions issued after a partial's stores and before
    // its arrival: the transfer at the end of that unit (L), the next unit's
    // offset load (1) and its X loads (kSteps NB).
    constexpr int kPartWait = kSteps * NB + L + 1 < 63 ? kSteps * NB + L + 1 : 63;
    // One unit: par = (uu - u0) mod S is its ring position (a constant in every
    // unrolled copy).
    auto unit = [&](int64_t uu, auto parc) __attribute__((always_inline)) {
        constexpr int par = decltype(parc)::value;
        uint8_t *const slot = ring[par] + j * kSlot;
        const uint32_t onn = rec_offsets(la_set, la_kt, uu + 3 < u1);  // requested at the end of the next unit
        advance(la_set, la_kt);
        // Decode this wavefront's record of the unit into registers.
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kRecWait) : "memory");
        half8 af[kSteps];
        {
            const RecState rs = rec_state(slot_mask(slot, lane));
            lds_u32 *const vals = as_lds(slot + kMaskBytes);
            StepWords sw = read_step(vals, lut, rs, 0);
#pragma unroll
            for (int st = 0; st < kSteps; ++st) {
                StepWords nx;
                if (st + 1 < kSteps) nx = read_step(vals, lut, rs, st + 1);
                af[st] = finish_step(sw);
                if (st + 1 < kSteps) sw = nx;
            }
        }
        lds_barrier();  // every wavefront has read the previous unit's operands
#pragma unroll
        for (int st = 0; st < kSteps; ++st) abuf[j][st][lane] = __builtin_bit_cast(uint4, af[st]);
        lds_barrier();
        int64_t setn = set, ktn = kt + 1;
        if (ktn == a.KT) {
            ktn = 0;
            ++setn;
        }
        const bool more = uu + 1 < u1;
        const int64_t kx = more ? ktn : kt;  // X of the next unit (past the range's end: this one's, unused)
        // The X loads are issued whatever the wavefront's tokens or the range:
        // a path with fewer loads would make the compiler's merged waits drain
        // the record ring. The A operands of step st + 1 are requested before
        // step st's products issue (kept there by a scheduling barrier): read
        // one at a time just before use, their LDS latency set the pace.
        half8 av[2][R];
#pragma unroll
        for (int r = 0; r < R; ++r) av[0][r] = __builtin_bit_cast(half8, abuf[r][0][lane]);
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            if (st + 1 < kSteps) {
#pragma unroll
                for (int r = 0; r < R; ++r) av[(st + 1) & 1][r] = __builtin_bit_cast(half8, abuf[r][st + 1][lane]);
            }
            __builtin_amdgcn_sched_barrier(0);
            if (has_tokens) {
#pragma unroll
                for (int r = 0; r < R; ++r)
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        acc[r][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                            av[st & 1][r], __builtin_bit_cast(half8, xb[nb][st]), acc[r][nb], 0, 0, 0);
            }
            // This step's X for the next unit, as soon as its last MFMA is issued.
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) xb[nb][st] = __builtin_amdgcn_raw_buffer_load_b128(xr, x_at(kx, st, nb), 0, 0);
        }
        if (cnt_set >= 0) {
            const WaveArgs ac = a;
            arrive_finish<R, NB>(ac, cnt_set, cnt_nseg, cnt_old, lane, j);
            cnt_set = -1;
        }
        if (pend_set >= 0) {  // the partial stored at the end of the previous unit
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kPartWait) : "memory");
            cnt_old = arrive_count(a, pend_set, lane, j);
            cnt_set = pend_set;
            cnt_nseg = pend_nseg;
            pend_set = -1;
        }
        if (!more || ktn == 0) {  // end of this workgroup's segment of the row set
            const int64_t w_first = unit_owner(set * a.KT, a.units, G);
            const int64_t w_last = unit_owner(set * a.KT + a.KT - 1, a.units, G);
            if (has_tokens) {
                const WaveArgs ac = a;
                if (w_first == w_last) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const int tok = tok0 + 16 * nb + n_lane;
                        if (tok < a.N) {
#pragma unroll
                            for (int r = 0; r < R; ++r) store_rows4(ac, tok, (set * R + r) * kTileRows + g4, acc[r][nb]);
                        }
                    }
                } else {
                    const int64_t slot_floats = (int64_t)a.N * kTileRows * R;
                    float *part_slot = a.ws + (set * a.maxseg + (w - w_first)) * slot_floats;
                    const __amdgpu_buffer_rsrc_t part = __builtin_amdgcn_make_buffer_rsrc(
                        part_slot, (short)0, (int)(slot_floats * 4), kBufferRsrcWord3);
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const int tok = tok0 + 16 * nb + n_lane;
                        if (tok < a.N) {
#pragma unroll
                            for (int r = 0; r < R; ++r)
                                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, acc[r][nb]), part,
                                                                       (tok * kTileRows * R + kTileRows * r + g4) * 4,
                                                                       0, kCachePolicyDevice);
                        }
                    }
                    pend_set = set;
                    pend_nseg = w_last - w_first + 1;
                }
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
        dma(slot, onext);  // unit uu + 2, into the slot this unit's decode freed
        onext = onn;
        set = setn;
        kt = ktn;
    };
    // Whole rounds of S units, then the rest: no path through the main loop
    // skips a unit's loads, so the compiler's waits there stay exact.
    int64_t u = u0;
    for (; u + S <= u1; u += S) static_for([&](auto pc) { unit(u + pc.value, pc); }, std::make_integer_sequence<int, S>{});
    static_for(
        [&](auto pc) {
            if (pc.value < S - 1 && u + pc.value < u1) unit(u + pc.value, pc);
        },
        std::make_integer_sequence<int, S>{});
    __builtin_amdgcn_s_waitcnt(0);  // the transfers past the range's end, the last partial's stores
    if (cnt_set >= 0) arrive_finish<R, NB>(a, cnt_set, cnt_nseg, cnt_old, lane, j);
    if (pend_set >= 0) arrive_row_set<R, NB>(a, pend_set, pend_nseg, lane, j);
}

// The shared-decode kernel with the decode of unit u + 1 interleaved with the
// products of unit u. With 3-4 token blocks a wavefront needs more than 256
// registers, so each SIMD holds one wavefront and the kernel above alternates a
// decode (VALU and LDS) with the products (MFMA), overlapping neither. Here the
// A operands are double-buffered in LDS: in each step of unit u a wavefront
// issues that step's products from buffer u mod 2 and decodes the same step of
// its record of unit u + 1 into the other buffer, and one barrier per unit
// (instead of two) both publishes the new buffer and frees the old one. The
// record of unit u + 1 must be in its ring slot when unit u starts; the
// transfer of unit v + 2 goes into the slot freed by decoding unit v, at the end
// of unit v - 1 (two units of slack). LDS: two 2-slot rings, two 32 KB operand
// buffers (105 KB at 5 KB records): one workgroup per CU.
template <int L, int NB>
__global__ __launch_bounds__(kShareWaves *kLanes, 1) void spmm_pipe_kernel(WaveArgs a, const uint32_t *__restrict__ off,
                                                                          const uint8_t *__restrict__ stream) {
    constexpr int R = kShareWaves;
    constexpr int kSlot = 1024 * L + 16;
    __shared__ __attribute__((aligned(16))) uint8_t ring0[R][kSlot];
    __shared__ __attribute__((aligned(16))) uint8_t ring1[R][kSlot];
    __shared__ __attribute__((aligned(16))) uint4 abuf0[R][kSteps][kLanes];
    __shared__ __attribute__((aligned(16))) uint4 abuf1[R][kSteps][kLanes];
    __shared__ __attribute__((aligned(16))) uint8_t lut[16 * 8];
    uint8_t *const ring[2] = {ring0[0], ring1[0]};
    const int lane = threadIdx.x & (kLanes - 1);
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    const int64_t w = blockIdx.x, G = gridDim.x;
    const int64_t u0 = w * a.units / G, u1 = (w + 1) * a.units / G;
    if (u0 >= u1) return;  // the whole workgroup
    if (threadIdx.x < 16) reinterpret_cast<uint2 *>(lut)[threadIdx.x] = nibble_selectors((uint32_t)threadIdx.x);

    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.xp, (short)0, (int)a.xp_bytes, kBufferRsrcWord3);
    const __amdgpu_buffer_rsrc_t offr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)off, (short)0, (int)((a.RB * a.KT + 1) * 4), kBufferRsrcWord3);
    const int n_lane = lane & 15, g4 = 4 * (lane >> 4);
    const int tok0 = 16 * NB * j;
    const bool has_tokens = tok0 < a.N;
    const int xlane = (NB * j * 64 + lane) * 16;
    auto x_at = [&](int64_t kx, int st, int nb) -> int {
        return (int)((kx * kSteps + st) * a.tb + nb) * (int)kPackBlockBytes + xlane;
    };
    auto rec_offsets = [&](int64_t set, int64_t kt, bool real) -> uint32_t {
        const int64_t rb = set * R + j;
        const bool ok = real && lane < 2 && rb < a.RB;
        return __builtin_amdgcn_raw_buffer_load_b32(offr, ok ? (int)((rb * a.KT + kt + lane) * 4) : 0x7FFFFFF0, 0, 0);
    };
    auto advance = [&](int64_t &set, int64_t &kt) {
        if (++kt == a.KT) {
            kt = 0;
            ++set;
        }
    };
    auto dma = [&](uint8_t *slot, uint32_t o) {
        const uint32_t lds = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t *)slot);
        dma_rec_asm<L>(stream, __builtin_amdgcn_readlane(o, 0), __builtin_amdgcn_readlane(o, 1), lane, lds);
    };
    // Decodes this wavefront's record in `slot` straight into row block j of
    // the operand buffer `dst` (the prologue's whole-record decode).
    auto decode_to = [&](const uint8_t *slot, uint4 (*dst)[kSteps][kLanes]) {
        const RecState rs = rec_state(slot_mask(slot, lane));
        lds_u32 *const vals = as_lds(slot + kMaskBytes);
        StepWords sw = read_step(vals, lut, rs, 0);
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            StepWords nx;
            if (st + 1 < kSteps) nx = read_step(vals, lut, rs, st + 1);
            dst[j][st][lane] = __builtin_bit_cast(uint4, finish_step(sw));
            if (st + 1 < kSteps) sw = nx;
        }
    };
    // Vector memory instructions issued after the transfer of the record a
    // unit decodes (that of the next unit) and before that decode, on the path
    // with the fewest: the transfer is issued at the end of the unit two before;
    // then the previous unit's offset load (1), its X loads (kSteps NB) and its
    // transfer (L), and this unit's offset load (1). One fewer is waited for.
    // The first unit's record (the prologue's second transfer) is followed by
    // X (kSteps NB), the third transfer (L) and the offset load (1): the same.
    constexpr int kRecWait = kSteps * NB + L + 1 < 63 ? kSteps * NB + L + 1 : 63;
    // The prologue decodes the first record once X and the second transfer
    // follow it: kSteps NB + L instructions.
    constexpr int kFirstWait = kSteps * NB + L < 63 ? kSteps * NB + L : 63;
    constexpr int kPartWait = kSteps * NB + L + 1 < 63 ? kSteps * NB + L + 1 : 63;

    floatx4 acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    int64_t set = u0 / a.KT, kt = u0 % a.KT;
    int64_t la_set = set, la_kt = kt;
    const uint32_t oa = rec_offsets(la_set, la_kt, true);
    advance(la_set, la_kt);
    const uint32_t ob = rec_offsets(la_set, la_kt, u0 + 1 < u1);
    advance(la_set, la_kt);
    const uint32_t oc = rec_offsets(la_set, la_kt, u0 + 2 < u1);
    advance(la_set, la_kt);
    uint32_t onext = rec_offsets(la_set, la_kt, u0 + 3 < u1);  // requested at the end of the first unit
    advance(la_set, la_kt);
    dma(ring[0] + j * kSlot, oa);
    dma(ring[1] + j * kSlot, ob);
    v4u32 xb[NB][kSteps];
#pragma unroll
    for (int st = 0; st < kSteps; ++st)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) xb[nb][st] = __builtin_amdgcn_raw_buffer_load_b128(xr, x_at(kt, st, nb), 0, 0);
    lds_barrier();  // the selector table
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kFirstWait) : "memory");
    decode_to(ring[0] + j * kSlot, abuf0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    dma(ring[0] + j * kSlot, oc);  // unit u0 + 2 into the slot just decoded
    lds_barrier();                 // the first unit's operands

    int64_t pend_set = -1, pend_nseg = 0;
    int64_t cnt_set = -1, cnt_nseg = 0;
    uint32_t cnt_old = 0;
    // One unit: par = (uu - u0) mod 2 selects its operand buffer (the next
    // unit's record sits in ring slot 1 - par).
    auto unit = [&](int64_t uu, auto parc) __attribute__((always_inline)) {
        constexpr int par = decltype(parc)::value;
        uint4 (*const acur)[kSteps][kLanes] = par ? abuf1 : abuf0;
        uint4 (*const anext)[kSteps][kLanes] = par ? abuf0 : abuf1;
        uint8_t *const slot = ring[1 - par] + j * kSlot;  // the next unit's record
        const uint32_t onn = rec_offsets(la_set, la_kt, uu + 4 < u1);
        advance(la_set, la_kt);
        int64_t setn = set, ktn = kt + 1;
        if (ktn == a.KT) {
            ktn = 0;
            ++setn;
        }
        const bool more = uu + 1 < u1;
        const int64_t kx = more ? ktn : kt;
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kRecWait) : "memory");
        const RecState rs = rec_state(slot_mask(slot, lane));
        lds_u32 *const vals = as_lds(slot + kMaskBytes);
        // The products are issued whether or not this wavefront has tokens
        // (without tokens its results are never stored): a branch around them
        // would keep the scheduler from interleaving them with the decode.
        StepWords sw = read_step(vals, lut, rs, 0);
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            StepWords nx;
            if (st + 1 < kSteps) nx = read_step(vals, lut, rs, st + 1);
            half8 av[R];
#pragma unroll
            for (int r = 0; r < R; ++r) av[r] = __builtin_bit_cast(half8, acur[r][st][lane]);
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[r][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[r], __builtin_bit_cast(half8, xb[nb][st]),
                                                                      acc[r][nb], 0, 0, 0);
            anext[j][st][lane] = __builtin_bit_cast(uint4, finish_step(sw));
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) xb[nb][st] = __builtin_amdgcn_raw_buffer_load_b128(xr, x_at(kx, st, nb), 0, 0);
            if (st + 1 < kSteps) sw = nx;
        }
        if (cnt_set >= 0) {
            const WaveArgs ac = a;
            arrive_finish<R, NB>(ac, cnt_set, cnt_nseg, cnt_old, lane, j);
            cnt_set = -1;
        }
        if (pend_set >= 0) {
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kPartWait) : "memory");
            cnt_old = arrive_count(a, pend_set, lane, j);
            cnt_set = pend_set;
            cnt_nseg = pend_nseg;
            pend_set = -1;
        }
        if (!more || ktn == 0) {
            const int64_t w_first = unit_owner(set * a.KT, a.units, G);
            const int64_t w_last = unit_owner(set * a.KT + a.KT - 1, a.units, G);
            if (has_tokens) {
                const WaveArgs ac = a;
                if (w_first == w_last) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const int tok = tok0 + 16 * nb + n_lane;
                        if (tok < a.N) {
#pragma unroll
                            for (int r = 0; r < R; ++r) store_rows4(ac, tok, (set * R + r) * kTileRows + g4, acc[r][nb]);
                        }
                    }
                } else {
                    const int64_t slot_floats = (int64_t)a.N * kTileRows * R;
                    float *part_slot = a.ws + (set * a.maxseg + (w - w_first)) * slot_floats;
                    const __amdgpu_buffer_rsrc_t part = __builtin_amdgcn_make_buffer_rsrc(
                        part_slot, (short)0, (int)(slot_floats * 4), kBufferRsrcWord3);
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const int tok = tok0 + 16 * nb + n_lane;
                        if (tok < a.N) {
#pragma unroll
                            for (int r = 0; r < R; ++r)
                                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, acc[r][nb]), part,
                                                                       (tok * kTileRows * R + kTileRows * r + g4) * 4,
                                                                       0, kCachePolicyDevice);
                        }
                    }
                    pend_set = set;
                    pend_nseg = w_last - w_first + 1;
                }
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[r][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the decode's reads of the slot are done
        dma(slot, onext);  // unit uu + 3, into the slot just decoded
        onext = onn;
        set = setn;
        kt = ktn;
        lds_barrier();  // the next unit's operands are complete, this unit's free
    };
    int64_t u = u0;
    for (; u + 2 <= u1; u += 2) static_for([&](auto pc) { unit(u + pc.value, pc); }, std::make_integer_sequence<int, 2>{});
    if (u < u1) unit(u, std::integral_constant<int, 0>{});
    __builtin_amdgcn_s_waitcnt(0);
    if (cnt_set >= 0) arrive_finish<R, NB>(a, cnt_set, cnt_nseg, cnt_old, lane, j);
    if (pend_set >= 0) arrive_row_set<R, NB>(a, pend_set, pend_nseg, lane, j);
}

// ---------------------------------------------------------------------------
// Row-block kernel for small matrices (up to 16 tokens).
//
// One workgroup per row block: its W wavefronts split the row block's column
// tiles and sum their partials through LDS behind one barrier, in a fixed order.
// Small matrices cannot keep every CU busy without splitting K, and a split
// across workgroups costs device-coherent partial stores, an atomic arrival and
// a reduction at the very end of the kernel, where nothing hides it; inside a
// workgroup the split is almost free. Each wavefront keeps its next two
// records in flight in a register ring (one is staged in LDS and decoded) and
// loads the next record's X operands one record ahead. The first record's
// extent comes through the scalar cache; the others from one vector load of the
// wavefront's stretch of the offset table, issued at the start.
// ---------------------------------------------------------------------------

template <int L, int W>
__global__ __launch_bounds__(kLanes * W) void spmm_row_kernel(WaveArgs a, const uint32_t *__restrict__ off,
                                                             const uint8_t *__restrict__ stream) {
    constexpr int kRegion = 1024 * L + 16;  // staged values + the decode's 12-byte overread
    __shared__ __attribute__((aligned(16))) uint8_t regions[W][kRegion];
    __shared__ __attribute__((aligned(16))) uint8_t luts[W][16 * 8];
    __shared__ floatx4 parts[W][kLanes];
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    const int64_t rb = blockIdx.x;
    const int64_t t0 = wave * a.KT / W, t1 = (wave + 1) * a.KT / W;  // this wavefront's column tiles
    uint8_t *const region = regions[wave];
    uint8_t *const lut = luts[wave];
    if (lane < 16) reinterpret_cast<uint2 *>(lut)[lane] = nibble_selectors((uint32_t)lane);
    const int n_lane = lane & 15, g4 = 4 * (lane >> 4);

    floatx4 acc[1] = {floatx4{0.f, 0.f, 0.f, 0.f}};
    if (t0 < t1) {
        const int64_t n = t1 - t0;
        const __amdgpu_buffer_rsrc_t xr =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.X, (short)0, (int)a.x_bytes, kBufferRsrcWord3);
        // Lanes of tokens >= N start at the resource's end: their loads return zeros.
        const int xoff = n_lane < a.N ? (int)(n_lane * a.ldx * 2) + 16 * (lane >> 4) : (int)a.x_bytes;
        const int64_t e0 = rb * a.KT + t0;  // first offset-table entry of the stretch
        const __amdgpu_buffer_rsrc_t offr = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(off + e0), (short)0, (int)((n + 1) * 4), kBufferRsrcWord3);
        const uint32_t offv = __builtin_amdgcn_raw_buffer_load_b32(offr, lane * 4, 0, 0);  // lanes > n: 0
        WaveRec<L> ring[2];
        fetch_rec<L>(stream, off[e0], off[e0 + 1], lane, ring[0]);
        {
            uint32_t o0 = 0, o1 = 0;  // past the stretch: an empty extent, same load count
            if (n > 1) {
                o0 = __builtin_amdgcn_readlane(offv, 1);
                o1 = __builtin_amdgcn_readlane(offv, 2);
            }
            fetch_rec<L>(stream, o0, o1, lane, ring[1]);
        }
        v4u32 xb[2][1][kSteps];
        fetch_x(a, xr, xoff, t0, lane, xb[0][0]);
        for (int64_t i0 = 0; i0 < n; i0 += 2) {
#pragma unroll
            for (int d = 0; d < 2; ++d) {
                const int64_t i = i0 + d;
                if (i < n) {
                    // Stage record i (in-order LDS: the previous decode's reads are done).
#pragma unroll
                    for (int k = 0; k < L; ++k) reinterpret_cast<v4u32 *>(region)[lane + kLanes * k] = ring[d].w[k];
                    const uint2 msk = ring[d].msk;
                    {
                        uint32_t o0 = 0, o1 = 0;
                        if (i + 2 < n) {
                            o0 = __builtin_amdgcn_readlane(offv, (int)(i + 2));
                            o1 = __builtin_amdgcn_readlane(offv, (int)(i + 3));
                        }
                        fetch_rec<L>(stream, o0, o1, lane, ring[d]);
                    }
                    fetch_x(a, xr, xoff, t0 + (i + 1 < n ? i + 1 : i), lane, xb[d ^ 1][0]);
                    decode_record<1>(as_lds(region), lut, msk, xb[d], acc);
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(0);  // also drains the empty loads past the stretch
    }
    parts[wave][lane] = acc[0];
    __syncthreads();
    if (wave == 0 && n_lane < a.N) {
        floatx4 sum = parts[0][lane];
#pragma unroll
        for (int w = 1; w < W; ++w) sum += parts[w][lane];  // fixed order: bitwise reproducible
        store_rows4(a, n_lane, rb * kTileRows + g4, sum);
    }
}

// One wavefront per tile: decode every lane-step and store it densely.
__global__ __launch_bounds__(64) void densify_kernel(const uint8_t *stream, const uint32_t *off, int64_t M,
                                                     int64_t K, int64_t KT, uint16_t *Wd, int64_t ldw) {
    __shared__ __attribute__((aligned(kWRegionBytes))) uint8_t region[kWRegionBytes + 16];
    __shared__ __attribute__((aligned(16))) uint8_t lut[16 * 8];
    const int lane = threadIdx.x;
    const int64_t t = blockIdx.x;
    const int64_t rb = t / KT, kt = t % KT;
    if (lane < 16) reinterpret_cast<uint2 *>(lut)[lane] = nibble_selectors((uint32_t)lane);
    const uint32_t o0 = off[t], o1 = off[t + 1];
    const uint8_t *rec = stream + (size_t)o0 * 16;
    const uint2 msk = reinterpret_cast<const uint2 *>(rec)[lane];
    const int nch = (int)(o1 - o0) - kMaskChunks;
    const uint4 *vp = reinterpret_cast<const uint4 *>(rec + kMaskBytes);
    for (int c = lane; c < nch; c += kLanes) reinterpret_cast<uint4 *>(region)[c] = vp[c];
    __syncthreads();
    const RecState rs = rec_state(msk);
    const int64_t row = rb * kTileRows + (lane & 15);
    if (row >= M) return;
    for (int s = 0; s < kSteps; ++s) {
        const half8 av = decode_step(as_lds(region), lut, rs, s);
        const uint4 u = __builtin_bit_cast(uint4, av);
        const int64_t col = kt * kTileK + tile_col(lane >> 4, s, 0);
        uint16_t *dst = Wd + row * ldw + col;
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
        for (int j = 0; j < 8; ++j)
            if (col + j < K) dst[j] = (uint16_t)(w[j >> 1] >> (16 * (j & 1)));
    }
}

}  // namespace

// Resident workgroups per CU of a kernel, queried from the runtime once and kept
// in `slot`. Host threads planning calls at the same time may both query; they
// store the same value, and the slot is atomic, so that is not a data race.
static int cached_occupancy(std::atomic<int> &slot, const void *kernel, int threads) {
    int c = slot.load(std::memory_order_relaxed);
    if (c == 0) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1) n = 1;
        slot.store(n, std::memory_order_relaxed);
        c = n;
    }
    return c;
}

// Workgroups of spmm_kernel<NT, XFAST> resident per CU (queried once per instance).
template <int NT, bool XFAST>
static int resident_wgs() {
    static std::atomic<int> cached{0};
    return cached_occupancy(cached, reinterpret_cast<const void *>(spmm_kernel<NT, XFAST>), kThreads);
}

// Token blocks the four-wavefront kernel is built for: 1-4, and 8 for 5-8.
static int kernel_nt(int nt) { return nt <= 4 ? nt : kMaxNT; }

static int resident_wgs(int nt, bool xfast) {
    switch (kernel_nt(nt)) {
        case 1: return xfast ? resident_wgs<1, true>() : resident_wgs<1, false>();
        case 2: return xfast ? resident_wgs<2, true>() : resident_wgs<2, false>();
        case 3: return xfast ? resident_wgs<3, true>() : resident_wgs<3, false>();
        case 4: return xfast ? resident_wgs<4, true>() : resident_wgs<4, false>();
        default: return xfast ? resident_wgs<kMaxNT, true>() : resident_wgs<kMaxNT, false>();
    }
}

// Plan of one pass over nt 16-token blocks: the persistent grid fills every CU
// with as many workgroups as can be resident (at least the slowest variant's
// count, so the plan does not depend on X's alignment).
static SpmmPlan plan_pass(const usp_matrix *A, int nt) {
    SpmmPlan p;
    p.row_groups = ceil_div(A->RB, kWaves);
    p.units = p.row_groups * A->KT;
    const int per_cu = std::min(resident_wgs(nt, true), resident_wgs(nt, false));
    const int64_t slots = (int64_t)(A->num_cus > 0 ? A->num_cus : 256) * per_cu;
    p.grid = p.units < slots ? p.units : slots;
    // A range of KT units meets at most ceil(KT / shortest range) + 1 workgroups.
    const int64_t shortest = p.units / p.grid;
    p.maxseg = ceil_div(A->KT, shortest) + 1;
    // Is any row group split over several workgroups?
    p.split = (p.units % p.grid != 0) || ((p.units / p.grid) % A->KT != 0);
    return p;
}

// Tokens per pass of the four-wavefront kernel (measured on MI355X): 128 for
// small matrices (at most 8192 tiles; 13B attention at 128 tokens: 39.6 us
// against 46.3 in two passes of 64), 64 otherwise (the 70B FFN layer at 128
// tokens: 211 us in one pass, 204 in two: with one workgroup per CU the larger
// pass is bound by its SIMDs).
constexpr int64_t kSmallMatrixTiles = 8192;
static int64_t pass_tokens(const usp_matrix *A) {
    return A->RB * A->KT <= kSmallMatrixTiles ? 16 * kMaxNT : 64;
}

static int pass_nt(const usp_matrix *A, int64_t N, int64_t n0) {
    const int64_t P = pass_tokens(A);
    const int64_t nb = (N - n0) < P ? (N - n0) : P;
    return (int)((nb + 15) / 16);
}

// ---------------------------------------------------------------------------
// Plans of the single-pass kernels (up to 128 tokens).
// ---------------------------------------------------------------------------

enum WaveKind { kWaveNone = 0, kWaveDma4 = 1, kWaveRow = 2, kWaveChunk = 3, kWaveShare = 4 };

constexpr int kMinWaveLoads = 2;  // record load groups instantiated: 2..8
// The fewest units a direct-to-LDS wavefront streams before a split costs it a
// partial.
constexpr int64_t kMinUnitsPerDmaWave = 2;

// Record load groups (1 KB each) that cover the values of every record of A.
static int wave_loads(const usp_matrix *A) {
    const int l = (int)ceil_div(A->max_chunks, kLanes);
    return l < kMinWaveLoads ? kMinWaveLoads : l;
}

// Load groups of the direct-to-LDS kernel: at one or two token blocks it moves
// whole records (mask bytes and values) into LDS, otherwise the values only;
// more than kMaxWaveLoads (records of nearly dense tiles) leaves the kernel out.
constexpr int kMaxWaveLoads = 8;
static int dma_loads(const usp_matrix *A, int nb) {
    const int l = (int)ceil_div((dma_mask_in_lds(nb) ? kMaskChunks : 0) + A->max_chunks, kLanes);
    return l < kMinWaveLoads ? kMinWaveLoads : l;
}

typedef void (*WaveKernelFn)(WaveArgs, const uint32_t *, const uint8_t *);

// Token blocks of 16 a wavefront of the direct-to-LDS kernel serves (X for all
// of them stays in registers): 1 to 4 (3 and 4 leave one wavefront per SIMD);
// and the most token groups (wavefronts streaming the same units for different
// tokens).
constexpr int kMaxDmaTokenBlocks = 4;
constexpr int kMaxDmaTokenGroups = 4;

// Token groups and token blocks per wavefront of the direct-to-LDS kernel: as
// few groups as hold every block, the blocks spread evenly over them.
static void dma_tokens(int64_t N, int &nbw, int &tg) {
    const int nb = (int)ceil_div(N, 16);
    tg = (int)ceil_div(nb, kMaxDmaTokenBlocks);
    nbw = (int)ceil_div(nb, tg);
}

// Wavefronts per workgroup of the row-block kernel: 2, 4, 5 or 8.
static WaveKernelFn row_kernel(int loads, int wpg) {
#define USP_ROW(WV)                                   \
    switch (loads) {                                  \
        case 2: return spmm_row_kernel<2, WV>;        \
        case 3: return spmm_row_kernel<3, WV>;        \
        case 4: return spmm_row_kernel<4, WV>;        \
        case 5: return spmm_row_kernel<5, WV>;        \
        case 6: return spmm_row_kernel<6, WV>;        \
        case 7: return spmm_row_kernel<7, WV>;        \
        default: return spmm_row_kernel<8, WV>;       \
    }
    if (wpg <= 2) {
        USP_ROW(2)
    }
    if (wpg <= 4) {
        USP_ROW(4)
    }
    if (wpg <= 5) {
        USP_ROW(5)
    }
    USP_ROW(8)
#undef USP_ROW
}

// Workgroups of the row-block kernel resident per CU.
static int resident_row_groups(int loads, int wpg) {
    static std::atomic<int> cached[9][9];
    return cached_occupancy(cached[loads][wpg], reinterpret_cast<const void *>(row_kernel(loads, wpg)), kLanes * wpg);
}

// The most wavefronts per row block (2, 4, 5 or 8, at most KT) for which every
// row block's workgroup is resident at once.
static int row_wpg(const usp_matrix *A, int loads) {
    const int64_t cus = A->num_cus > 0 ? A->num_cus : 256;
    for (int wpg : {8, 5, 4})
        if (wpg <= A->KT && A->RB <= cus * resident_row_groups(loads, wpg)) return wpg;
    return 2;
}

static WaveKernelFn dma_kernel(int loads, int nb) {
#define USP_BY_LOADS(NB)                            \
    switch (loads) {                                \
        case 2: return spmm_dma_kernel<2, NB>;      \
        case 3: return spmm_dma_kernel<3, NB>;      \
        case 4: return spmm_dma_kernel<4, NB>;      \
        case 5: return spmm_dma_kernel<5, NB>;      \
        case 6: return spmm_dma_kernel<6, NB>;      \
        case 7: return spmm_dma_kernel<7, NB>;      \
        default: return spmm_dma_kernel<8, NB>;     \
    }
    if (nb == 1) {
        USP_BY_LOADS(1)
    }
    if (nb == 2) {
        USP_BY_LOADS(2)
    }
    if (nb == 3) {
        USP_BY_LOADS(3)
    }
    USP_BY_LOADS(4)
#undef USP_BY_LOADS
}

static WaveKernelFn chunk_kernel(int loads, int wpg, int nb) {
#define USP_CHUNK(WV, NBV)                                 \
    switch (loads) {                                       \
        case 2: return spmm_chunk_kernel<2, WV, NBV>;      \
        case 3: return spmm_chunk_kernel<3, WV, NBV>;      \
        case 4: return spmm_chunk_kernel<4, WV, NBV>;      \
        case 5: return spmm_chunk_kernel<5, WV, NBV>;      \
        case 6: return spmm_chunk_kernel<6, WV, NBV>;      \
        case 7: return spmm_chunk_kernel<7, WV, NBV>;      \
        default: return spmm_chunk_kernel<8, WV, NBV>;     \
    }
    if (nb == 1) {
        if (wpg == 8) {
            USP_CHUNK(8, 1)
        }
        USP_CHUNK(4, 1)
    }
    if (wpg == 8) {
        USP_CHUNK(8, 2)
    }
    USP_CHUNK(4, 2)
#undef USP_CHUNK
}

// Workgroups of the column-chunk kernel resident per CU.
static int resident_chunk_groups(int loads, int wpg, int nb) {
    static std::atomic<int> cached[9][9][kMaxChunkTokenBlocks + 1];
    return cached_occupancy(cached[loads][wpg][nb], reinterpret_cast<const void *>(chunk_kernel(loads, wpg, nb)),
                            kLanes * wpg);
}

// Wavefronts of the direct-to-LDS kernel resident per CU (queried once per
// variant).
// The direct-to-LDS kernel's wavefronts per CU, at most kMaxDmaWavesPerCu. With
// records of 3-4 KB (60-70% sparsity) up to 13 fit a CU's LDS, but then a
// layer of 14336 units no longer gives every wavefront 8 units and the planner
// fell back to the four-wavefront kernel; at 7 per CU the 70B FFN takes 52.4
// us at 60% and 50.1 at 70% (16 tokens) against 61.3 and 57.6 there, 67.6 and
// 65.0 against 78.8 and 75.9 at 32 tokens.
constexpr int kMaxDmaWavesPerCu = 7;
static int resident_waves(int loads, int nb) {
    static std::atomic<int> cached[9][kMaxDmaTokenBlocks + 1];
    const int r = cached_occupancy(cached[loads][nb], reinterpret_cast<const void *>(dma_kernel(loads, nb)), kLanes);
    return r < kMaxDmaWavesPerCu ? r : kMaxDmaWavesPerCu;
}

static WaveKernelFn share_kernel(int loads, int nb) {
#define USP_SHARE(NB)                                 \
    switch (loads) {                                  \
        case 2: return spmm_share_kernel<2, NB>;      \
        case 3: return spmm_share_kernel<3, NB>;      \
        case 4: return spmm_share_kernel<4, NB>;      \
        case 5: return spmm_share_kernel<5, NB>;      \
        case 6: return spmm_share_kernel<6, NB>;      \
        case 7: return spmm_share_kernel<7, NB>;      \
        default: return spmm_share_kernel<8, NB>;     \
    }
    // 1 or 2 token blocks: from 3 the planner always takes the pipelined variant.
    if (nb == 1) {
        USP_SHARE(1)
    }
    USP_SHARE(2)
#undef USP_SHARE
}

static WaveKernelFn pipe_kernel(int loads, int nb) {
#define USP_PIPE(NB)                                  \
    switch (loads) {                                  \
        case 2: return spmm_pipe_kernel<2, NB>;       \
        case 3: return spmm_pipe_kernel<3, NB>;       \
        case 4: return spmm_pipe_kernel<4, NB>;       \
        case 5: return spmm_pipe_kernel<5, NB>;       \
        case 6: return spmm_pipe_kernel<6, NB>;       \
        case 7: return spmm_pipe_kernel<7, NB>;       \
        default: return spmm_pipe_kernel<8, NB>;      \
    }
    if (nb == 2) {
        USP_PIPE(2)
    }
    if (nb == 3) {
        USP_PIPE(3)
    }
    USP_PIPE(4)
#undef USP_PIPE
}

// Whether the shared-decode kernel overlaps the next unit's decode with the
// products (spmm_pipe_kernel, one workgroup per CU) for `units` units: always
// at 3-4 token blocks per wavefront, where either way a SIMD holds one
// wavefront (70B FFN at 256 tokens 174.5 against 191.4 us, 66B FFN 241.7
// against 265.8, 13B FFN up 68.7 against 71.9); at 2 blocks only on layers of
// fewer than 32 units per CU, where two unpipelined workgroups per CU have too
// few units to hide each other (13B attention at 128 tokens 32.4 against 36.6,
// 13B FFN down 55.1 against 58.8; the 70B FFN, 56 units per CU, 131.8 against
// 109.5).
constexpr int kPipeMinBlocks = 3;
constexpr int64_t kPipeMaxUnitsPerCuAt2 = 32;
static bool share_pipelined(int nb, int64_t units, int64_t cus) {
    return nb >= kPipeMinBlocks || (nb == 2 && units < kPipeMaxUnitsPerCuAt2 * cus);
}

// Workgroups of the shared-decode kernel (pipelined or not) resident per CU.
static int resident_share_wgs(int loads, int nb, bool pipe = false) {
    if (pipe) {
        static std::atomic<int> cached_pipe[9][kMaxDmaTokenBlocks + 1];
        return cached_occupancy(cached_pipe[loads][nb], reinterpret_cast<const void *>(pipe_kernel(loads, nb)),
                                kShareWaves * kLanes);
    }
    static std::atomic<int> cached[9][kMaxDmaTokenBlocks + 1];
    return cached_occupancy(cached[loads][nb], reinterpret_cast<const void *>(share_kernel(loads, nb)),
                            kShareWaves * kLanes);
}

// Token blocks per wavefront of the shared-decode kernel (its four wavefronts
// split the tokens).
static int share_nb(int64_t N) { return (int)ceil_div(ceil_div(N, 16), kShareWaves); }

// The fewest units a shared-decode workgroup streams.
constexpr int64_t kMinUnitsPerShareWg = 4;
// Token blocks from which the shared-decode kernel serves a call (measured,
// packed X included): 70B FFN 84.2 against 89.4 us on the direct-to-LDS kernel
// at 48 tokens, 87.3 against 104.9 at 64; 13B FFN up 37.2 against 37.7 on the
// four-wavefront kernel at 48, 38.7 against 41.4 at 64. At 32 tokens two of
// its four wavefronts would have no tokens.
constexpr int kShareMinBlocks = 3;

struct WavePlan {
    WaveKind kind;
    int loads, rows, nb, tg;  // record load groups; row blocks per unit; token blocks per wavefront; groups
    int wpg;                  // column-chunk kernel: wavefronts (row blocks) per workgroup
    int64_t sets, units, ranges, grid, maxseg;  // ranges of units; workgroups = ranges * tg
    bool split;
    bool pipe = false;        // shared-decode kernel: the pipelined variant
};

// Which kernel suits A for N tokens (measured on MI355X): the direct-to-LDS
// kernel once every range gets at least 8 units of 4 row blocks (70B- and
// 66B-class FFN layers, up to 128 tokens); for small matrices and up to 16
// tokens, the row-block kernel when there are no more row blocks than CUs (its
// workgroups then spread evenly) and otherwise the column-chunk kernel (13B
// attention, 13B FFN up) unless a row block would be split into more than 8
// chunks (13B FFN down: 14 chunks, 29.0 against 27.7 us); the column-chunk
// kernel also at 17 to 32 tokens on the conditions below; everything else goes
// to the four-wavefront kernel, which shares X through LDS.
constexpr int64_t kDmaUnitsPerSlot = 8;
constexpr int64_t kMaxDmaWideSplit = 4;
constexpr int64_t kSmallMaxTiles = 8192;
constexpr int64_t kRowMaxTiles = 16;  // column tiles per row block
constexpr int64_t kChunkMaxTiles = 20480;
constexpr int64_t kChunkMaxSplit = 8;
static WaveKind wave_kind(const usp_matrix *A, int loads, int64_t N) {
    const int nb = (int)ceil_div(N, 16);
    // More than 32 tokens: the shared-decode kernel (each record decoded once,
    // X packed) on matrices with at least kMinUnitsPerShareWg units for every
    // resident workgroup, and above 64 tokens for one workgroup per CU. Between
    // the two, at 33-64 tokens, the kernels are within 7% either way: 13B
    // attention (1600 units) 21.4 us on the four-wavefront kernel against 22.9
    // at 48 tokens, 24.0 against 25.2 at 64; one GPU's share of the 70B FFN
    // (1792 units) 26.0 against 24.8 and 29.8 against 28.1. At 128 tokens 13B
    // attention takes 36.6 us on the shared-decode kernel against 40.9.
    if (nb >= kShareMinBlocks && nb <= kMaxDmaTokenBlocks * kShareWaves && dma_loads(A, 1) <= kMaxWaveLoads) {
        const int64_t cus = A->num_cus > 0 ? A->num_cus : 256;
        const int64_t per = nb > kShareWaves ? 1 : resident_share_wgs(dma_loads(A, 1), share_nb(N));
        if (ceil_div(A->RB, kShareWaves) * A->KT >= kMinUnitsPerShareWg * cus * per) return kWaveShare;
    }
    if (nb <= kMaxDmaTokenBlocks * kMaxDmaTokenGroups) {
        int nbw, tg;
        dma_tokens(N, nbw, tg);
        const int dl = dma_loads(A, nbw);
        const int64_t slots = dl > kMaxWaveLoads ? 0 : (int64_t)(A->num_cus > 0 ? A->num_cus : 256) * resident_waves(dl, nbw);
        const int64_t sets = ceil_div(A->RB, kDmaRows);
        // At 3-4 blocks (one wavefront per SIMD, 16 KB partials per row set at
        // 64 tokens) a row set split over more than 4 wavefronts costs more than
        // the four-wavefront kernel: the 70B FFN down projection (8192 x 28672,
        // 128 row sets over 1024 wavefronts) takes 107.9 us against 101.3 at 64
        // tokens, while the up projection (448 row sets) gains.
        const bool split_ok = nbw < 3 || sets * kMaxDmaWideSplit >= slots / tg;
        if (slots > 0 && split_ok && sets * A->KT >= kDmaUnitsPerSlot * (slots / tg)) return kWaveDma4;
    }
    // The row-block kernel for few long row blocks only while each has few
    // column tiles or the tokens are few: one GPU's share of the 70B FFN
    // (224 row blocks x 32 tiles) takes 16.8 us on it at 16 tokens against 14.8
    // on the column-chunk kernel, but 13.6 against 14.5 at 8 tokens; the tiny
    // layer (4 tiles) 4.5 against 6.6.
    // A wavefront of the row-block kernel reads its stretch of the offset table
    // (up to ceil(KT / 2) tiles at its fewest 2 wavefronts, plus one end entry)
    // with one 64-lane load, so the stretch is limited to 63 tiles.
    if (nb == 1 && A->RB * A->KT <= kSmallMaxTiles && A->RB <= (A->num_cus > 0 ? A->num_cus : 256) &&
        (A->KT <= kRowMaxTiles || N <= 8) && ceil_div(A->KT, 2) <= kLanes - 1)
        return kWaveRow;
    if (nb <= kMaxChunkTokenBlocks && A->RB * A->KT <= kChunkMaxTiles && ceil_div(A->KT, kChunkTiles) <= kChunkMaxSplit) {
        if (nb == 1) return kWaveChunk;
        // Two token blocks (one workgroup per CU: X for 32 tokens in LDS) only
        // in a single round of workgroups of 8 row blocks that covers at least
        // half the CUs: 13B attention 15.8 against 18.4 us at 32 tokens, one
        // GPU's share of the 70B FFN 16.5 against 22.0; the 13B FFN up (1080
        // workgroups of 4) 49.8 against 33.2, the tiny layer (8) 10.2 against 7.8.
        const int64_t cus = A->num_cus > 0 ? A->num_cus : 256;
        const int64_t wgs = ceil_div(A->RB, 8) * ceil_div(A->KT, kChunkTiles);
        if (2 * wgs >= cus && wgs <= cus * resident_chunk_groups(loads, 8, nb)) return kWaveChunk;
    }
    return kWaveNone;
}

static WavePlan plan_wave(const usp_matrix *A, int64_t N) {
    WavePlan p;
    p.loads = wave_loads(A);
    p.kind = wave_kind(A, p.loads, N);
    p.wpg = 0;
    if (p.kind == kWaveChunk) {  // workgroups of wpg row blocks x kChunkTiles column tiles
        p.rows = 1;
        p.nb = (int)ceil_div(N, 16);
        p.tg = 1;
        p.sets = A->RB;
        p.units = A->RB * A->KT;
        p.maxseg = ceil_div(A->KT, kChunkTiles);
        // 8 row blocks per workgroup when every workgroup is resident at once
        // (the chunk's X is staged once for twice the records; 13B attention at
        // 16 tokens: 13.1 against 13.6 us), else 4 (13B FFN up: 540 workgroups
        // of 8 need two rounds, 28.5 against 24.5 us).
        const int64_t cus = A->num_cus > 0 ? A->num_cus : 256;
        p.wpg = ceil_div(A->RB, 8) * p.maxseg <= cus * resident_chunk_groups(p.loads, 8, p.nb) ? 8 : 4;
        p.ranges = ceil_div(A->RB, p.wpg) * p.maxseg;
        p.grid = p.ranges;
        p.split = p.maxseg > 1;
        return p;
    }
    if (p.kind == kWaveShare) {
        p.nb = share_nb(N);
        p.tg = kShareWaves;  // one arrival counter per wavefront (token slice)
        p.loads = dma_loads(A, 1);
        p.rows = kShareWaves;
        p.sets = ceil_div(A->RB, p.rows);
        p.units = p.sets * A->KT;
        const int64_t cus = A->num_cus > 0 ? A->num_cus : 256;
        p.pipe = share_pipelined(p.nb, p.units, cus);
        const int64_t wgs = cus * resident_share_wgs(p.loads, p.nb, p.pipe);
        const int64_t want = ceil_div(p.units, kMinUnitsPerShareWg);
        p.ranges = want < wgs ? want : wgs;
        // One whole row set per workgroup when the sets fill at least 7/8 of
        // the resident workgroups: no partials, no arrivals (70B FFN, 448 sets,
        // 512 resident at 128 tokens: 112.9 against 117.7 us, 86.8 against 87.4
        // at 64; with fewer sets per slot it lost: 66B FFN at 128 tokens on 288
        // workgroups 223.0 against 155.4).
        if (p.sets <= wgs && 8 * p.sets >= 7 * wgs) p.ranges = p.sets;
        // At one block, half a set per workgroup when that fills at least 4/5
        // of them: every split set then has exactly two pieces (13B FFN up,
        // 216 sets: 432 workgroups, 36.6 against 38.3 us at 64 tokens, 35.3
        // against 36.5 at 48).
        else if (p.nb == 1 && 2 * p.sets <= wgs && 10 * p.sets >= 4 * wgs) p.ranges = 2 * p.sets;
        p.grid = p.ranges;
        const int64_t shortest = p.units / p.ranges;
        p.maxseg = ceil_div(A->KT, shortest) + 1;
        p.split = (p.units % p.ranges != 0) || ((p.units / p.ranges) % A->KT != 0);
        return p;
    }
    p.nb = 1;
    p.tg = 1;
    if (p.kind != kWaveDma4) {  // the row-block kernel (or none): no partials in the workspace
        p.rows = 1;
        p.sets = p.units = p.ranges = p.grid = p.maxseg = 0;
        p.split = false;
        return p;
    }
    dma_tokens(N, p.nb, p.tg);
    p.loads = dma_loads(A, p.nb);
    p.rows = kDmaRows;
    p.sets = ceil_div(A->RB, p.rows);
    p.units = p.sets * A->KT;
    const int64_t slots = (int64_t)(A->num_cus > 0 ? A->num_cus : 256) * resident_waves(p.loads, p.nb) / p.tg;
    const int64_t want = ceil_div(p.units, kMinUnitsPerDmaWave);
    p.ranges = want < slots ? want : slots;
    if (p.tg > 1) p.ranges = std::max<int64_t>(8, p.ranges / 8 * 8);  // whole groups of 8 ranges x tg
    p.grid = p.ranges * p.tg;
    // A range of KT units meets at most ceil(KT / shortest range) + 1 ranges.
    const int64_t shortest = p.units / p.ranges;
    p.maxseg = ceil_div(A->KT, shortest) + 1;
    p.split = (p.units % p.ranges != 0) || ((p.units / p.ranges) % A->KT != 0);
    return p;
}

// The single-pass kernels serve up to 256 tokens with X 16-byte
// aligned, ldx and K multiples of 8, and X's extent and the offset table
// addressable by 32-bit offsets.
constexpr int64_t kMaxWaveTokens = 16 * kMaxDmaTokenBlocks * kMaxDmaTokenGroups;
static bool use_wave_kernel(const usp_matrix *A, const void *X, int64_t ldx, int64_t N) {
    if (N > kMaxWaveTokens || (reinterpret_cast<uintptr_t>(X) & 15) || ldx % 8 || A->K % 8) return false;
    const int64_t x_bytes = ((N - 1) * ldx + A->K) * 2;
    if (x_bytes + 2 * A->KT * kTileK >= ((int64_t)1 << 31) || (A->RB * A->KT + 1) * 4 >= ((int64_t)1 << 31) ||
        packed_x_bytes(A->KT, N) + 16 * kPackBlockBytes >= ((size_t)1 << 31))
        return false;
    return wave_kind(A, wave_loads(A), N) != kWaveNone;
}

SpmmPlan plan_spmm(const usp_matrix *A, int64_t N) { return plan_pass(A, pass_nt(A, N, 0)); }

std::string describe_plan(const usp_matrix *A, int64_t N) {
    char buf[128];
    // As launch_spmm decides for X 16-byte aligned with ldx = K.
    if (use_wave_kernel(A, reinterpret_cast<const void *>(uintptr_t{256}), A->K, N)) {
        const int loads = wave_loads(A);
        const WaveKind kind = wave_kind(A, loads, N);
        if (kind == kWaveRow) {
            snprintf(buf, sizeof buf, "row W=%d", row_wpg(A, loads));
        } else {
            const WavePlan p = plan_wave(A, N);
            if (kind == kWaveChunk)
                snprintf(buf, sizeof buf, "chunk S=%lld W=%d nb=%d grid=%lld", (long long)p.maxseg, p.wpg, p.nb,
                         (long long)p.grid);
            else if (kind == kWaveShare)
                snprintf(buf, sizeof buf, "share nb=%d grid=%lld%s", p.nb, (long long)p.grid,
                         p.pipe ? " pipelined" : "");
            else
                snprintf(buf, sizeof buf, "dma nb=%d tg=%d grid=%lld", p.nb, p.tg, (long long)p.grid);
        }
        return buf;
    }
    const int64_t P = pass_tokens(A);
    const SpmmPlan p = plan_pass(A, pass_nt(A, N, 0));
    snprintf(buf, sizeof buf, "fourwave passes=%lld nt=%d grid=%lld", (long long)ceil_div(N, P), pass_nt(A, N, 0),
             (long long)p.grid);
    return buf;
}

// Workspace: the arrival counters at offset 0 (zero between calls), then the
// fp32 partials of the current pass.
// The counters take the first kCounterRegionBytes of every workspace whatever
// the handle (one word per row block, rounded up to whole sets of 4, for up to
// kMaxRows rows, which usp_encode enforces; the four-wavefront kernel's one per
// row group and the direct-to-LDS kernel's one per row set and token group fit
// the same region), and the partials start after it: partials a call leaves
// behind never sit where another handle's counters are, so one zero-filled
// workspace serves calls with any handle and any N.
constexpr size_t kCounterRegionBytes = 256 * 1024;
static_assert(kMaxRows / kTileRows * sizeof(uint32_t) <= kCounterRegionBytes, "counter region too small");
static size_t counters_bytes(const usp_matrix *) { return kCounterRegionBytes; }

static size_t partials_bytes(const SpmmPlan &p, int64_t nb) {
    return (size_t)p.row_groups * (size_t)p.maxseg * (size_t)nb * kGroupRows * sizeof(float);
}

static size_t wave_partials_bytes(const usp_matrix *A, int64_t N) {
    const WavePlan p = plan_wave(A, N);
    if (!p.split) return 0;
    return (size_t)p.sets * (size_t)p.maxseg * (size_t)N * kTileRows * p.rows * sizeof(float);
}

// Where the shared-decode kernel's packed X starts: after the counters and
// the partials (256-byte aligned).
static size_t packed_x_offset(const usp_matrix *A, int64_t N) {
    return counters_bytes(A) + (wave_partials_bytes(A, N) + 255) / 256 * 256;
}

size_t spmm_workspace_bytes(const usp_matrix *A, int64_t N) {
    // Layout: counters, then the partials of whichever pass runs. Passes run one
    // after another and reuse the workspace: full passes of pass_tokens(A)
    // tokens, then one pass over the remainder; up to 256 tokens may take a wave
    // kernel (sized here too, whichever needs more; a call whose X the wave
    // kernels cannot read goes to the passes). The shared-decode kernel also
    // keeps packed X after its partials.
    size_t need = N <= kMaxWaveTokens ? wave_partials_bytes(A, N) : 0;
    if (N <= kMaxWaveTokens && wave_kind(A, wave_loads(A), N) == kWaveShare)
        need = packed_x_offset(A, N) - counters_bytes(A) + packed_x_bytes(A->KT, N);
    auto add = [&](int64_t nb) {
        const SpmmPlan p = plan_pass(A, (int)((nb + 15) / 16));
        if (p.split) need = std::max(need, partials_bytes(p, nb));
    };
    const int64_t P = pass_tokens(A);
    if (N >= P) add(P);
    if (N % P) add(N % P);
    return need ? counters_bytes(A) + need : 0;
}

static void set_epilogue(WaveArgs &a, const Epilogue &ep) {
    a.bias = ep.bias;
    a.res = ep.res;
    a.ldr = ep.ldr;
    a.act = ep.act;
}

static int launch_row(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                      const Epilogue &ep, hipStream_t st) {
    const int loads = wave_loads(A);
    const int wpg = row_wpg(A, loads);
    WaveArgs a = {};
    a.M = A->M;
    a.K = A->K;
    a.RB = A->RB;
    a.KT = A->KT;
    a.X = reinterpret_cast<const uint16_t *>(X);
    a.ldx = ldx;
    a.x_bytes = (uint32_t)(((N - 1) * ldx + A->K) * 2);
    a.Y = reinterpret_cast<uint16_t *>(Y);
    a.ldy = ldy;
    a.N = (int)N;
    a.y_vec = ((reinterpret_cast<uintptr_t>(Y) & 7) == 0) && (ldy % 4 == 0);
    set_epilogue(a, ep);
    hipLaunchKernelGGL(row_kernel(loads, wpg), dim3((unsigned)A->RB), dim3(kLanes * wpg), 0, st, a, A->d_off,
                       reinterpret_cast<const uint8_t *>(A->d_stream));
    return (int)hipGetLastError();
}

static int launch_wave(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                       const Epilogue &ep, void *workspace, hipStream_t st) {
    if (wave_kind(A, wave_loads(A), N) == kWaveRow) return launch_row(A, X, ldx, Y, ldy, N, ep, st);
    const WavePlan p = plan_wave(A, N);
    WaveArgs a = {};
    a.M = A->M;
    a.K = A->K;
    a.RB = A->RB;
    a.KT = A->KT;
    a.sets = p.sets;
    a.units = p.units;
    a.maxseg = p.maxseg;
    a.X = reinterpret_cast<const uint16_t *>(X);
    a.ldx = ldx;
    a.x_bytes = (uint32_t)(((N - 1) * ldx + A->K) * 2);
    a.Y = reinterpret_cast<uint16_t *>(Y);
    a.ldy = ldy;
    a.N = (int)N;
    a.cnt = p.split ? reinterpret_cast<uint32_t *>(workspace) : nullptr;
    a.ws = p.split ? reinterpret_cast<float *>(reinterpret_cast<uint8_t *>(workspace) + counters_bytes(A)) : nullptr;
    a.y_vec = ((reinterpret_cast<uintptr_t>(Y) & 7) == 0) && (ldy % 4 == 0);
    a.tg = p.tg;
    set_epilogue(a, ep);
    if (p.kind == kWaveChunk)
        hipLaunchKernelGGL(chunk_kernel(p.loads, p.wpg, p.nb), dim3((unsigned)p.grid), dim3(kLanes * p.wpg), 0, st, a,
                           A->d_off, reinterpret_cast<const uint8_t *>(A->d_stream));
    else if (p.kind == kWaveShare) {
        uint8_t *xp = reinterpret_cast<uint8_t *>(workspace) + packed_x_offset(A, N);
        a.tb = (int)ceil_div(N, 16);
        a.xp = xp;
        a.xp_bytes = (uint32_t)packed_x_bytes(A->KT, N);
        hipLaunchKernelGGL(pack_x_kernel, dim3((unsigned)(A->KT * a.tb)), dim3(kLanes), 0, st,
                           reinterpret_cast<const uint16_t *>(X), ldx, (int)N, A->K, a.tb, xp);
        hipLaunchKernelGGL(p.pipe ? pipe_kernel(p.loads, p.nb) : share_kernel(p.loads, p.nb),
                           dim3((unsigned)p.grid), dim3(kShareWaves * kLanes), 0, st, a, A->d_off,
                           reinterpret_cast<const uint8_t *>(A->d_stream));
    }
    else
        hipLaunchKernelGGL(dma_kernel(p.loads, p.nb), dim3((unsigned)p.grid), dim3(kLanes), 0, st, a, A->d_off,
                           reinterpret_cast<const uint8_t *>(A->d_stream));
    return (int)hipGetLastError();
}

int launch_spmm(const usp_matrix *A, const void *X, int64_t ldx, void *Y, int64_t ldy, int64_t N,
                const Epilogue &ep, void *workspace, void *stream) {
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (use_wave_kernel(A, X, ldx, N)) return launch_wave(A, X, ldx, Y, ldy, N, ep, workspace, st);
    const int64_t P = pass_tokens(A);
    for (int64_t n0 = 0; n0 < N; n0 += P) {
        const int nb = (int)((N - n0) < P ? (N - n0) : P);
        const int nt = (nb + 15) / 16;
        const SpmmPlan p = plan_pass(A, nt);
        float *ws = p.split ? reinterpret_cast<float *>(reinterpret_cast<uint8_t *>(workspace) + counters_bytes(A))
                            : nullptr;
        SpmmArgs a;
        a.stream = reinterpret_cast<const uint8_t *>(A->d_stream);
        a.off = A->d_off;
        a.M = A->M;
        a.K = A->K;
        a.RB = A->RB;
        a.KT = A->KT;
        a.X = reinterpret_cast<const uint16_t *>(X) + n0 * ldx;
        a.ldx = ldx;
        a.Y = reinterpret_cast<uint16_t *>(Y) + n0 * ldy;
        a.ldy = ldy;
        a.N = nb;
        a.units = p.units;
        a.maxseg = p.maxseg;
        a.ws = ws;
        a.cnt = ws ? reinterpret_cast<uint32_t *>(workspace) : nullptr;
        a.x_vec = ((reinterpret_cast<uintptr_t>(a.X) & 15) == 0) && (ldx % 8 == 0);
        a.y_vec = ((reinterpret_cast<uintptr_t>(a.Y) & 7) == 0) && (ldy % 4 == 0);
        a.bias = ep.bias;
        a.res = ep.res ? ep.res + n0 * ep.ldr : nullptr;
        a.ldr = ep.ldr;
        a.act = ep.act;
        const dim3 grid((unsigned)p.grid), block(kThreads);
        const bool xfast = a.x_vec && (A->K % 8 == 0);
#define USP_LAUNCH(NTV)                                                                              \
    if (xfast) hipLaunchKernelGGL((spmm_kernel<NTV, true>), grid, block, 0, st, a, a.off, a.stream); \
    else hipLaunchKernelGGL((spmm_kernel<NTV, false>), grid, block, 0, st, a, a.off, a.stream);
        switch (kernel_nt(nt)) {
            case 1: USP_LAUNCH(1) break;
            case 2: USP_LAUNCH(2) break;
            case 3: USP_LAUNCH(3) break;
            case 4: USP_LAUNCH(4) break;
            default: USP_LAUNCH(kMaxNT) break;
        }
#undef USP_LAUNCH
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return (int)e;
    }
    return 0;
}

// ---------------------------------------------------------------------------
// Device scratch of usp_spmm_noalloc: the workspace (arrival counters, then
// partials) of callers that cannot allocate. One copy per GPU, held until the
// process ends. In host code `scratch` names a host-side stand-in, not device
// memory: its device address on each GPU is looked up once (with that GPU
// current) and only that address is used.
// ---------------------------------------------------------------------------

static __device__ __align__(256) uint8_t scratch[USP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::atomic<void *> g_scratch[kMaxDevices];
static std::mutex g_scratch_mu;

int noalloc_setup(int device) {
    if (device < 0 || device >= kMaxDevices) return (int)hipErrorInvalidDevice;
    if (g_scratch[device].load(std::memory_order_acquire)) return 0;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch[device].load(std::memory_order_relaxed)) return 0;
    void *ptr = nullptr;  // the caller made `device` current
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    // The arrival counters must start at zero; every completed product leaves
    // them at zero again.
    e = hipMemsetAsync(ptr, 0, kCounterRegionBytes, nullptr);
    if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
    if (e != hipSuccess) return (int)e;
    g_scratch[device].store(ptr, std::memory_order_release);
    return 0;
}

void *noalloc_scratch(int device) {
    return device >= 0 && device < kMaxDevices ? g_scratch[device].load(std::memory_order_acquire) : nullptr;
}

int launch_densify(const usp_matrix *A, void *Wd, int64_t ldw, void *stream) {
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    const int64_t T = A->RB * A->KT;
    hipLaunchKernelGGL(densify_kernel, dim3((unsigned)T), dim3(64), 0, st,
                       reinterpret_cast<const uint8_t *>(A->d_stream), A->d_off, A->M, A->K, A->KT,
                       reinterpret_cast<uint16_t *>(Wd), ldw);
    return (int)hipGetLastError();
}

}  // namespace usp
