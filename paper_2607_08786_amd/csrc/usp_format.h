// usp_format.h -- geometry of the compressed weight format (version 2).
//
// The paper stores a pruned weight matrix in three layers (Section 3.2): a 2:4
// part for sparse tensor cores, a slot-filling part with differential position
// codes, and a CSR residual. This library uses one bitmap-class layer instead
// (1 bit per weight position plus the packed kept values), laid out so that one
// 64-lane wavefront decodes it straight into the A operand of
// v_mfma_f32_16x16x32_f16.
//
// Tiles. W is cut into tiles of TILE_ROWS x TILE_K (16 rows x 256 columns);
// M and K are padded up to tile multiples with pruned (mask 0) entries.
// Tile t = rb * KT + kt covers rows [16 rb, 16 rb + 16) and columns
// [256 kt, 256 kt + 256). Within a tile, lane l (0..63) of the decoding
// wavefront owns row r = l % 16 and column group g = l / 16; at step s (0..7)
// it owns the 8 positions
//     row 16 rb + r, columns 256 kt + 32 s + 8 g + j,  j = 0..7,
// which is exactly the slice of a 16 x 32 MFMA A operand lane l holds.
//
// Tile record (starts on a 16-byte boundary, byte offset 16 * off[t]):
//   [0, 512)            mask: lane l's 8 bytes at 8 l; byte s bit j = position
//                       (s, j) above is kept.
//   [512, 512 + 2 nnz)  kept values as fp16 bit patterns in 16 blocks, block
//                       b = 2 s + h holding nibble h of step s (h = 0: positions
//                       j = 0..3, h = 1: j = 4..7) of every lane: lane 0's kept
//                       values of that nibble (j ascending), then lane 1's, ...,
//                       then lane 63's; blocks in order b = 0..15, unpadded.
//                       A lane's nibble has 0-4 values, so the 64 lanes reading
//                       their nibble of one block read words about one dword
//                       apart (32 lanes span about the 32 LDS banks).
//   zero padding to a multiple of 16 bytes.
// off[] holds T + 1 uint32 entries in 16-byte units; off[T] is the total size.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define USP_HD __host__ __device__
#else
#define USP_HD
#endif

namespace usp {

constexpr int kTileRows = 16;
constexpr int kTileK = 256;
constexpr int kLanes = 64;
constexpr int kSteps = 8;                    // k-steps of 32 columns per tile
constexpr int kMaskBytes = kLanes * kSteps;  // 512
constexpr int kMaskChunks = kMaskBytes / 16; // 32 sixteen-byte units
constexpr int kMaxValBytes = kTileRows * kTileK * 2;  // 8192 (a fully dense tile)
constexpr int kStreamPad = 1024;  // device bytes after the last record (read, never used)

USP_HD inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Column of position (g, s, j) inside a tile.
USP_HD inline int tile_col(int g, int s, int j) { return 32 * s + 8 * g + j; }

}  // namespace usp
