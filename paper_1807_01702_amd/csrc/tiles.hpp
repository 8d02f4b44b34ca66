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
// Row blocks of a sweep over m rows: the launched grid.  A block covers
// ceil(m / target) rows, so the grid is ceil(m / rows-per-block), which can be
// smaller than the target (m = 62720, target 512: 123 rows per block, 510
// blocks).  Workspace sizing, the sweep launch and the combine all use this
// count, so the combine never reads a partial row the sweep did not write.
inline int64_t stats_row_blocks(int64_t m, int c, int dtype) {
    int64_t cb = (c + stats_ch_per_block(dtype) - 1) / stats_ch_per_block(dtype);
    int64_t target = 512 / cb;             // about two workgroups per CU
    if (target < 1) target = 1;
    int64_t minrows = 64;
    int64_t rb = (m + minrows - 1) / minrows;
    const int64_t want = rb < target ? rb : target;
    if (m <= 0) return want;
    const int64_t rpb = (m + want - 1) / want;
    return (m + rpb - 1) / rpb;
}

// ---- implicit-GEMM CONV over pixel rows (forward and data gradient) -------
// Tile: BM pixel rows x BN output channels, K consumed in chunks of 32 input
// channels (all taps of a chunk resident in LDS).
constexpr int kRowsBK = 32;
constexpr int kRowsMaxW3 = 62;             // largest image width for 3x3 (halo = W+1 rows)
struct RowsTile { int bm, bn; };
// m > 0: a bf16 1x1 grid of 128-row tiles that would leave CUs idle (the
// late DenseNet blocks: 14x14 and 7x7 images) takes 64-row tiles instead,
// and 32-row tiles below 128 tiles of 64 rows (7x7 images at batch 128)
inline RowsTile rows_tile(int dtype, int taps, int n_out, int64_t m = 0) {
    if (dtype == DT_F32) return RowsTile{64, n_out <= 32 ? 32 : 64};
    if (taps == 1) {
        const int bn = n_out <= 64 ? (n_out <= 32 ? 32 : 64) : 128;
        const int64_t nt = (n_out + bn - 1) / bn;
        const int64_t tiles128 = (m + 127) / 128 * nt, tiles64 = (m + 63) / 64 * nt;
        if (bn != 128 || m <= 0 || tiles128 >= 256) return RowsTile{128, bn};
        return RowsTile{tiles64 >= 128 ? 64 : 32, bn};
    }
    return RowsTile{128, n_out <= 32 ? 32 : 64};
}

// ---- weight gradient (reduction over pixels, split-K) ----------------------
// Workgroup tile: 64 input channels x (1x1: the tap; 3x3: the 3 taps of one
// filter row) x COT output channels; K (pixels) in chunks of 64 positions.
// 3x3 chunks are R whole image rows laid out with a zero column on the left
// and zero padding to a width PW in {16, 32, 64}, so R * PW = 64.  The chunk
// range is split S ways; each split writes a float32 partial tile.
constexpr int kWgKC = 64;                  // K positions per chunk
constexpr int kWgCIT = 64;                 // input channels per tile
constexpr int kWgMaxW3 = 62;               // widest 3x3 image row (PW <= 64)
constexpr int kWgTrKQ1 = 64;               // pixels per chunk of the bf16 1x1 weight gradient (128: slower)
constexpr int64_t kWgTrSmallPartBytes = 32ll << 20;   // partial-tile budget of small bf16 weight gradients
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct WgradPlan {
    int k, cot, ci_tiles, kh_tiles, co_tiles;
    int R, PW;                             // 3x3 only
    int64_t chunks_per_image, nchunks, splits, chunks_per_split;
};
inline WgradPlan wgrad_plan(int64_t m, int n, int h, int w, int c_in, int c_out, int k, int elem_bytes)
{
    WgradPlan p;
    p.k = k;
    p.cot = c_out <= 32 ? 32 : (c_out <= 64 || k == 3 ? 64 : 128);
    p.ci_tiles = (int)ceil_div(c_in, kWgCIT);
    p.kh_tiles = k == 3 ? 3 : 1;
    p.co_tiles = (int)ceil_div(c_out, p.cot);
    if (k == 3) {
        p.PW = w + 2 <= 16 ? 16 : (w + 2 <= 32 ? 32 : 64);
        p.R = kWgKC / p.PW;
        p.chunks_per_image = ceil_div(h, p.R);
        p.nchunks = (int64_t)n * p.chunks_per_image;
    } else {
        p.PW = 0;
        p.R = 0;
        p.chunks_per_image = 0;
        p.nchunks = ceil_div(m, kWgKC);
    }
    const int64_t n_out = (int64_t)p.ci_tiles * p.kh_tiles * p.co_tiles;
    int64_t s = ceil_div(512, n_out);
    // partial tiles (S * |dW| float32, written and read once) kept below a
    // third of the operand bytes
    const int64_t dw_bytes = (int64_t)k * k * c_in * c_out * 4;
    const int64_t in_bytes = m * (int64_t)(c_in + c_out) * elem_bytes;
    int64_t cap = (in_bytes / 3) / (dw_bytes > 0 ? dw_bytes : 1);
    if (cap < 1) cap = 1;
    if (s > cap) s = cap;
    if (s > p.nchunks) s = p.nchunks;
    if (s < 1) s = 1;
    p.chunks_per_split = ceil_div(p.nchunks, s);
    p.splits = ceil_div(p.nchunks, p.chunks_per_split);
    return p;
}

// ---- bf16 weight gradient with transposing LDS reads --------------------
// Both operands are staged row-major (one row per K position, channels
// contiguous) and the matrix-core fragments are read transposed.  A
// workgroup owns CIT input channels x COT output channels (x all nine taps
// for 3x3).  K positions come in chunks of KQ: 1x1, 64 consecutive pixels;
// 3x3, R image rows of PW = W + 2 padded positions (a zero column at each
// end) rounded up to a multiple of 32, with the Z operand staged for the
// positions [-(PW + 1), KQ + PW + 1) so that tap (kh, kw) reads Z rows
// q + kh PW + kw (zero padding is the zero positions).
struct WgTrPlan {
    int k, cit, cot, ci_tiles, co_tiles;
    int R, PW, KQ, zrows;
    int64_t chunks_per_image, nchunks, splits, chunks_per_split;
};
inline WgTrPlan wgrad_tr_plan(int64_t m, int n, int h, int w, int c_in, int c_out, int k)
{
    WgTrPlan p;
    p.k = k;
    p.cot = c_out <= 32 ? 32 : (c_out <= 64 ? 64 : 128);
    if (k == 3 && p.cot > 64) p.cot = 64;
    p.cit = (k == 1 && c_in > 64) ? 128 : 64;
    p.ci_tiles = (int)ceil_div(c_in, p.cit);
    p.co_tiles = (int)ceil_div(c_out, p.cot);
    if (k == 3) {
        p.PW = w + 2;
        p.R = 128 / p.PW < 1 ? 1 : 128 / p.PW;
        if (p.R > h) p.R = h;
        p.KQ = (int)ceil_div((int64_t)p.R * p.PW, 32) * 32;
        p.zrows = p.KQ + 2 * p.PW + 2;
        p.chunks_per_image = ceil_div(h, p.R);
        p.nchunks = (int64_t)n * p.chunks_per_image;
    } else {
        p.PW = 0;
        p.R = 0;
        p.KQ = kWgTrKQ1;
        p.zrows = kWgTrKQ1;
        p.chunks_per_image = 0;
        p.nchunks = ceil_div(m, kWgTrKQ1);
    }
    const int64_t n_out = (int64_t)p.ci_tiles * p.co_tiles;
    int64_t s = ceil_div(512, n_out);                 // two workgroups per CU
    // partial tiles (S * |dW| float32, written and read once) kept below the
    // operand bytes, or below kWgTrSmallPartBytes for small operands (late
    // DenseNet blocks: a launch of a few dozen workgroups is latency-bound,
    // and a few MB more of partial tiles cost less than the idle CUs)
    const int64_t dw_bytes = (int64_t)k * k * c_in * c_out * 4;
    int64_t in_bytes = m * (int64_t)(c_in + c_out) * 2;
    if (in_bytes < kWgTrSmallPartBytes) in_bytes = kWgTrSmallPartBytes;
    int64_t cap = in_bytes / (dw_bytes > 0 ? dw_bytes : 1);
    if (cap < 1) cap = 1;
    if (s > cap) s = cap;
    if (s > p.nchunks) s = p.nchunks;
    if (s < 1) s = 1;
    p.chunks_per_split = ceil_div(p.nchunks, s);
    p.splits = ceil_div(p.nchunks, p.chunks_per_split);
    return p;
}

}  // namespace bnr
