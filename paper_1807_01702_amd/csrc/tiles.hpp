// tiles.hpp -- tile shapes shared by the launchers and the kernels, so that
// grid sizes, workspace sizes and kernel indexing agree by construction.
#pragma once
#include <stdint.h>

namespace bnr {

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };

// ---- standalone per-channel reductions (BN statistics, BN-backward sums) --
// One workgroup covers up to kStatsMaxCh channels of a block of rows; the
// partial sums of every (row block, channel) go to workspace and a separate
// combine kernel adds them in float64.
constexpr int kStatsMaxVec = 32;           // 16-byte vectors per row a workgroup covers
inline int stats_vec(int dtype) { return dtype == DT_BF16 ? 8 : 4; }
inline int stats_ch_per_block(int dtype) { return kStatsMaxVec * stats_vec(dtype); }
inline int64_t stats_row_blocks(int64_t m, int c, int dtype) {
    int64_t cb = (c + stats_ch_per_block(dtype) - 1) / stats_ch_per_block(dtype);
    int64_t target = 512 / cb;             // about two workgroups per CU
    if (target < 1) target = 1;
    int64_t minrows = 64;
    int64_t rb = (m + minrows - 1) / minrows;
    return rb < target ? rb : target;
}

// ---- implicit-GEMM CONV over pixel rows (forward and data gradient) -------
// Tile: BM pixel rows x BN output channels, K consumed in chunks of 32 input
// channels (all taps of a chunk resident in LDS).
constexpr int kRowsBK = 32;
constexpr int kRowsMaxW3 = 64;             // largest image width for 3x3 (halo = W+1 rows)
struct RowsTile { int bm, bn; };
inline RowsTile rows_tile(int dtype, int taps, int n_out) {
    if (dtype == DT_F32) return RowsTile{64, n_out <= 32 ? 32 : 64};
    if (taps == 1) return RowsTile{128, n_out <= 64 ? (n_out <= 32 ? 32 : 64) : 128};
    return RowsTile{128, n_out <= 32 ? 32 : 64};
}

// ---- weight gradient (reduction over pixels, split-K) ----------------------
// Workgroup tile: 64 input channels x (1 or 3 taps) x COT output channels,
// pixels in chunks of kWgBKP; S pixel splits write float32 partial tiles.
constexpr int kWgBKP = 64;
constexpr int kWgCIT = 64;
inline int wgrad_cot(int n_out) { return n_out <= 32 ? 32 : (n_out <= 64 ? 64 : 128); }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct WgradPlan {
    int ci_tiles, kh_tiles, co_tiles, cot, taps_per_wg;
    int64_t splits, chunks_per_split;
};
inline WgradPlan wgrad_plan(int64_t m, int c_in, int c_out, int k, int elem_bytes) {
    WgradPlan p;
    p.cot = wgrad_cot(c_out);
    p.ci_tiles = (int)ceil_div(c_in, kWgCIT);
    p.kh_tiles = k == 3 ? 3 : 1;
    p.taps_per_wg = k == 3 ? 3 : 1;
    p.co_tiles = (int)ceil_div(c_out, p.cot);
    int64_t n_out = (int64_t)p.ci_tiles * p.kh_tiles * p.co_tiles;
    int64_t chunks = ceil_div(m, kWgBKP);
    int64_t s = ceil_div(512, n_out);
    // keep the partial tiles (S * |dW| floats) small next to the operand bytes
    int64_t dw_bytes = (int64_t)k * k * c_in * c_out * 4;
    int64_t in_bytes = m * (int64_t)(c_in + c_out) * elem_bytes;
    int64_t cap = (in_bytes / 12) / (dw_bytes > 0 ? dw_bytes : 1);
    if (cap < 1) cap = 1;
    if (s > cap) s = cap;
    if (s > chunks) s = chunks;
    if (s < 1) s = 1;
    p.chunks_per_split = ceil_div(chunks, s);
    p.splits = ceil_div(chunks, p.chunks_per_split);
    return p;
}

}  // namespace bnr
