// usp_encode.cpp -- one-time host conversion of (W, mask) into tile records,
// and its inverse. This plays the role of the paper's dense-to-format
// conversion (Section 5.3, "Storage Format Conversion"), for the bitmap-class
// format described in usp_format.h.
#include <algorithm>
#include <cstring>
#include <thread>

#include "usp_internal.h"

namespace usp {
namespace {

template <class F>
void parallel_rows(int64_t n, F &&fn) {
    unsigned hw = std::thread::hardware_concurrency();
    int64_t nt = std::max<int64_t>(1, std::min<int64_t>(hw ? hw : 1, 64));
    nt = std::min(nt, n);
    if (nt <= 1) {
        for (int64_t i = 0; i < n; ++i) fn(i);
        return;
    }
    std::vector<std::thread> th;
    th.reserve(nt);
    for (int64_t t = 0; t < nt; ++t) {
        th.emplace_back([&, t] {
            for (int64_t i = t; i < n; i += nt) fn(i);
        });
    }
    for (auto &x : th) x.join();
}

// Kept bits of one tile lane-step (8 positions), bit j = column 32 s + 8 g + j.
inline uint8_t lane_step_bits(const uint8_t *mask, int64_t ldm, int64_t M, int64_t K,
                              int64_t row, int64_t col0) {
    if (row >= M) return 0;
    uint8_t b = 0;
    const uint8_t *mr = mask + row * ldm;
    for (int j = 0; j < 8; ++j) {
        int64_t c = col0 + j;
        if (c < K && mr[c]) b |= (uint8_t)(1u << j);
    }
    return b;
}

}  // namespace

void encode_host(const uint16_t *W, int64_t ldw, const uint8_t *mask, int64_t ldm,
                 int64_t M, int64_t K, HostEncoding &out) {
    out.M = M;
    out.K = K;
    out.RB = ceil_div(M, kTileRows);
    out.KT = ceil_div(K, kTileK);
    const int64_t T = out.RB * out.KT;

    // Pass 1: kept count per tile -> record sizes.
    std::vector<int64_t> tile_nnz(T, 0);
    parallel_rows(out.RB, [&](int64_t rb) {
        for (int64_t kt = 0; kt < out.KT; ++kt) {
            int64_t cnt = 0;
            for (int r = 0; r < kTileRows; ++r) {
                int64_t row = rb * kTileRows + r;
                if (row >= M) break;
                const uint8_t *mr = mask + row * ldm;
                int64_t c0 = kt * kTileK, c1 = std::min<int64_t>(K, c0 + kTileK);
                for (int64_t c = c0; c < c1; ++c) cnt += mr[c] != 0;
            }
            tile_nnz[rb * out.KT + kt] = cnt;
        }
    });
    out.off.assign(T + 1, 0);
    int64_t total = 0, nnz = 0, max_chunks = 0;
    for (int64_t t = 0; t < T; ++t) {
        out.off[t] = (uint32_t)total;
        const int64_t chunks = ceil_div(2 * tile_nnz[t], 16);
        total += kMaskChunks + chunks;
        max_chunks = std::max(max_chunks, chunks);
        nnz += tile_nnz[t];
        if (total >= (int64_t(1) << 32)) throw std::bad_alloc();
    }
    out.off[T] = (uint32_t)total;
    out.nnz = nnz;
    out.max_chunks = max_chunks;
    out.stream.assign((size_t)total * 16, 0);

    // Pass 2: fill records.
    parallel_rows(out.RB, [&](int64_t rb) {
        for (int64_t kt = 0; kt < out.KT; ++kt) {
            uint8_t *rec = out.stream.data() + (size_t)out.off[rb * out.KT + kt] * 16;
            uint16_t *vals = reinterpret_cast<uint16_t *>(rec + kMaskBytes);
            int64_t v = 0;
            for (int s = 0; s < kSteps; ++s) {
                for (int l = 0; l < kLanes; ++l) {
                    const int r = l % kTileRows, g = l / kTileRows;
                    rec[8 * l + s] = lane_step_bits(mask, ldm, M, K, rb * kTileRows + r, kt * kTileK + tile_col(g, s, 0));
                }
                // Values of step s: block (s, low nibble), then block (s, high nibble);
                // within a block lane 0's values first, in column order.
                for (int h = 0; h < 2; ++h) {
                    for (int l = 0; l < kLanes; ++l) {
                        const uint8_t b = rec[8 * l + s];
                        const int r = l % kTileRows, g = l / kTileRows;
                        const int64_t row = rb * kTileRows + r;
                        const int64_t col0 = kt * kTileK + tile_col(g, s, 0);
                        for (int j = 4 * h; j < 4 * h + 4; ++j)
                            if (b & (1u << j)) vals[v++] = W[row * ldw + col0 + j];
                    }
                }
            }
        }
    });
}

bool decode_host(const HostEncoding &enc, uint16_t *W_out, uint8_t *mask_out) {
    const int64_t M = enc.M, K = enc.K;
    const int64_t T = enc.RB * enc.KT;
    if ((int64_t)enc.off.size() != T + 1) return false;
    if ((size_t)enc.off[T] * 16 != enc.stream.size()) return false;
    std::memset(W_out, 0, sizeof(uint16_t) * (size_t)(M * K));
    std::memset(mask_out, 0, (size_t)(M * K));
    bool ok = true;
    for (int64_t rb = 0; rb < enc.RB && ok; ++rb) {
        for (int64_t kt = 0; kt < enc.KT && ok; ++kt) {
            const int64_t t = rb * enc.KT + kt;
            const uint8_t *rec = enc.stream.data() + (size_t)enc.off[t] * 16;
            const int64_t cap = ((int64_t)enc.off[t + 1] - enc.off[t] - kMaskChunks) * 8;  // halfs
            const uint16_t *vals = reinterpret_cast<const uint16_t *>(rec + kMaskBytes);
            int64_t v = 0;
            for (int sh = 0; sh < 2 * kSteps && ok; ++sh) {
                const int s = sh / 2, h = sh % 2;  // block (step s, nibble half h)
                for (int l = 0; l < kLanes; ++l) {
                    const int r = l % kTileRows, g = l / kTileRows;
                    const int64_t row = rb * kTileRows + r;
                    const uint8_t b = rec[8 * l + s];
                    for (int j = 4 * h; j < 4 * h + 4; ++j) {
                        if (!(b & (1u << j))) continue;
                        const int64_t col = kt * kTileK + tile_col(g, s, j);
                        if (row >= M || col >= K || v >= cap) { ok = false; break; }
                        W_out[row * K + col] = vals[v++];
                        mask_out[row * K + col] = 1;
                    }
                }
            }
        }
    }
    return ok;
}

}  // namespace usp
