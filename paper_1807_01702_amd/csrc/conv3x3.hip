// conv3x3.hip -- persistent 3x3 CONV (stride 1, zero padding 1), forward and
// data gradient, on the gfx950 matrix cores with the BN fission/fusion
// prologues and epilogues.
//
// The GEMM rows are the positions of the zero-padded image grid,
// P = (img (H + 2) + hp) (W + 2) + wp: a 3x3 tap is then the constant row
// offset (dh (W + 2) + dw) for every output row, padding taps read zero rows,
// and an A fragment is one LDS read at a wave-uniform row plus a fixed lane
// offset (no per-lane masks or address arithmetic in the matrix-core loop).
// Outputs at padding positions are computed and discarded (2 (H + W + 2) of
// every (H + 2)(W + 2) positions).
// One 512-thread workgroup per CU owns a contiguous range of positions
// [P0, P1).
//   * Weights: each of the 8 waves owns a 32-channel slice of the GEMM K
//     (input channels) and a 32-column slice of the outputs, and keeps the
//     matrix-core fragments of that slice for all nine taps in registers
//     (72 VGPRs), loaded once through LDS from [kh][kw][ci][co] (transposed for
//     the forward GEMM, taps flipped for the data gradient).  The remaining
//     8 / (K slices x N slices) waves split the 128 rows of a tile.
//   * Inputs: a ring buffer of position rows in LDS.  A 128-row output tile
//     at p0 needs the rows [p0 - (W+3), p0 + 128 + W + 3); consecutive tiles
//     share all but 128 of them, so each input pixel is read from HBM and
//     transformed by the prologue once (no halo re-reads inside a workgroup);
//     padding positions are written as zeros.
// The 128 new rows of the next tile are loaded into registers while the
// matrix cores work on the current tile, together with the epilogue operand
// of the current tile.  Two waves per SIMD let one wave's prologue / epilogue
// arithmetic overlap the other's matrix-core work.  Zero padding applies to
// the CONV input, i.e. after BN and ReLU.  The float32 partial tiles of the K
// slices are added in LDS in a fixed order.
//
// The epilogue reads whole 16-byte channel vectors of one pixel row, so every
// global access is coalesced, and keeps the per-channel statistics of the
// workgroup's rows in registers: one partial row per workgroup.  Prologue /
// epilogue modes are those of conv_rows.hip.
#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

constexpr int kP3Threads = 512;
constexpr int kP3BM = 128;          // output rows per tile
constexpr int kP3MaxW = 61;         // widest image row (ring = 128 + 2 (W + 3) rows: fill = two batches)
constexpr int kP3MaxH = 896;        // tallest image (exact multiply-shift row quotients)

// LDS layout (bytes): [ring: ring rows, then copies of its first 16 rows (so
// a 16-row fragment starting anywhere in the ring is contiguous), then one
// junk row for masked writes; lda bf16 per row]
// [stage: weights Ws[9][NP][ldw] bf16 at the start; afterwards the float32
// K-slice partial tiles red[WK][128][ldr] and finally the statistics scratch]
// [coefficients: 3 KP + 4 NP floats].
struct P3Geom {
    int KP, NP, lda, ldw, ldr, ring;
    int PW, PH, MP;                 // padded row length W + 2, image height H + 2, positions n PH PW
    int grid, mp_q, mp_r;           // workgroups and MP = mp_q grid + mp_r (set by the launcher)
    double inv_pw, inv_ph;
    uint32_t rpw, rph;              // ceil(2^20 / PW), ceil(2^20 / PH): multiply-shift quotients
    size_t ring_bytes, stage_bytes, lds;
};

static P3Geom p3_geom(int K, int N, int W)
{
    P3Geom g;
    g.KP = (K + 31) / 32 * 32;
    g.NP = N <= 32 ? 32 : (N <= 64 ? 64 : 128);
    g.lda = g.KP + 8;
    g.ldw = g.KP + 8;
    g.ldr = g.NP + 4;
    g.ring = kP3BM + 2 * (W + 3);
    g.ring_bytes = (size_t)(g.ring + 17) * g.lda * 2;   // + copies of the first 16 rows + a junk row
    g.PW = W + 2;
    g.PH = 0; g.MP = 0; g.inv_pw = 1.0 / g.PW; g.inv_ph = 0.0;   // set by the launcher
    g.grid = 1; g.mp_q = 0; g.mp_r = 0;
    const size_t wst = (size_t)9 * g.NP * g.ldw * 2;
    const size_t red = (size_t)(g.KP / 32) * kP3BM * g.ldr * 4;
    const size_t stats = (size_t)2 * (kP3Threads / (g.NP / 8)) * g.NP * 4;
    g.stage_bytes = wst > red ? wst : red;
    if (stats > g.stage_bytes) g.stage_bytes = stats;
    g.lds = g.ring_bytes + g.stage_bytes + (size_t)(3 * g.KP + 4 * g.NP) * 4;
    return g;
}

// Position -> pixel in two steps for the loops: a batch's first position
// (wave-uniform) is split once, then each lane's offset from it with 24-bit
// multiply-shift quotients, exact while x d < 2^20 for the dividend x and
// divisor d (x < PW + 256 against PW <= 64; y < PH + 86 against PH <= kP3MaxH + 2).
struct P3Base { int img, hp, wp, P; };
__device__ __forceinline__ P3Base p3_base(int q0, const P3Geom &g)
{
    P3Base b;
    b.P = q0 > 0 ? q0 : 0;
    const int t = b.P / g.PW;
    b.wp = b.P - t * g.PW;
    b.img = t / g.PH;
    b.hp = t - b.img * g.PH;
    return b;
}
__device__ __forceinline__ int p3_pixel_at(const P3Base &b, int P, const P3Geom &g, int H, int W)
{
    const int o = P - b.P;                                    // < 256 (negative only for P < 0)
    const int x = b.wp + (o > 0 ? o : 0);
    const int t = (int)(__umul24((uint32_t)x, g.rpw) >> 20);
    const int wp = x - __mul24(t, g.PW);
    const int y = b.hp + t;
    const int u = (int)(__umul24((uint32_t)y, g.rph) >> 20);
    const int hp = y - __mul24(u, g.PH);
    const int img = b.img + u;
    const bool ok = (P >= 0) & (P < g.MP) & (wp > 0) & (wp <= W) & (hp > 0) & (hp <= H);
    return ok ? (img * H + hp - 1) * W + wp - 1 : -1;
}

// Pixel of padded position P, or -1 for a padding position or one outside
// [0, MP).  The float64 quotient is within one of the exact one (|P| < 2^30).
// Branch-free (selects only): the persistent loops keep their loads in
// flight across it.
__device__ __forceinline__ int p3_pixel(int P, const P3Geom &g, int H, int W)
{
    int t = (int)((double)P * g.inv_pw);
    int wp = P - t * g.PW;
    t = wp < 0 ? t - 1 : (wp >= g.PW ? t + 1 : t);
    wp = P - t * g.PW;
    int img = (int)((double)t * g.inv_ph);
    int hp = t - img * g.PH;
    img = hp < 0 ? img - 1 : (hp >= g.PH ? img + 1 : img);
    hp = t - img * g.PH;
    const bool ok = P >= 0 && P < g.MP && wp > 0 && wp <= W && hp > 0 && hp <= H;
    return ok ? (img * H + hp - 1) * W + wp - 1 : -1;
}

// WK x WN: 32-channel K slices x 32-column N slices (one per wave); the
// other 8 / (WK WN) waves split the tile rows.  The epilogue kind EK and
// whether the prologue reads a second operand (PRO_BNGRAD) are compile-time,
// so the epilogue is straight-line code and the compiler can keep the next
// tile's loads in flight while it waits for the epilogue operand (a runtime
// mode switch makes it wait for every outstanding load at each branch).
// PC: the prologue, compile-time where it pays: PC3_BNGRAD (the deferred
// BN input gradient, which reads a second operand), PC3_BNRELU (the forward
// BN+ReLU with the statistics epilogue), PC3_RUNTIME (PRO_NONE / PRO_BNRELU /
// PRO_RELU chosen at run time).
// PC3_BNRELU_SAVE: BN+ReLU whose result z is also stored (the materialised
// O2' sweep; each workgroup stores the positions of its own range once).
enum { PC3_RUNTIME = 0, PC3_BNGRAD = 1, PC3_BNRELU = 2, PC3_BNRELU_SAVE = 3 };
// The BN-backward epilogue reading the stored z (p.e_zsrc) is an epilogue kind
// of its own, so the plain BN-backward epilogue carries none of its code.
constexpr int EK3_BNBWD_Z = 7;

template <int WK, int WN, int EK, int PC>
__global__ __launch_bounds__(kP3Threads) void k_conv3x3(RowsParams p, P3Geom g)
{
    constexpr bool BNG = PC == PC3_BNGRAD;
    constexpr bool ZK = EK == EK3_BNBWD_Z;                        // BN backward from the stored z
    constexpr bool BNB = EK == EK_BNBWD || ZK;                    // BN-backward epilogue
    constexpr bool SAVE = PC == PC3_BNRELU_SAVE;
    const int pro = PC == PC3_BNRELU || SAVE ? PRO_BNRELU : (PC == PC3_BNGRAD ? PRO_BNGRAD : p.pro);
    using T = bf16_t;
    using M = Mfma<T>;
    constexpr int VEC = 8;
    constexpr int KPC = 32 * WK, NPC = 32 * WN;
    constexpr int WR = 8 / (WK * WN);                            // row groups
    constexpr int RB = kP3BM / (16 * WR);                        // 16-row blocks per wave
    constexpr int VPRO = NPC / VEC, RSTEP = kP3Threads / VPRO;
    constexpr int RPT = kP3BM / RSTEP;                           // epilogue rows per thread
    constexpr bool READS = EK == EK_STORE_ACC || EK == EK_RELUMASK || BNB;
    constexpr int NVA = (kP3BM * (KPC / VEC) + kP3Threads - 1) / kP3Threads;
    constexpr int NVB = BNG ? NVA : 1, NVX = READS ? RPT : 1;
    // batches in flight: one (a second register buffer is merged back into
    // the first by the compiler, with copies that wait for its loads)
    constexpr int AHEAD = 1;
    static_assert(WR * WK * WN == 8 && RPT >= 1, "wave layout");
    extern __shared__ __align__(16) unsigned char smem[];
    T *ring = reinterpret_cast<T *>(smem);                       // [ring + 16][lda]
    unsigned char *stage = smem + g.ring_bytes;
    T *Ws = reinterpret_cast<T *>(stage);                        // [9][NP][ldw] (start only)
    float *red = reinterpret_cast<float *>(stage);               // [WK][BM][ldr]
    float *coef = reinterpret_cast<float *>(stage + g.stage_bytes);
    float *epi = coef + 3 * KPC;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave % WR, wk = (wave / WR) % WK, wn = wave / (WR * WK);
    const int K = p.K, N = p.N, RING = g.ring, lda = g.lda, ldr = g.ldr;
    const int m = (int)p.m;                                      // launcher: m < 2^30
    const int H = p.h, W = p.w, PW = g.PW;
    // range [floor(b MP / G), floor((b + 1) MP / G)) in 32-bit arithmetic
    // (b mp_q <= MP < 2^30, b mp_r < G^2): no 64-bit division, whose branches
    // would serialise the kernel-argument loads around it
    const int bid = blockIdx.x;
    const int P0 = bid * g.mp_q + (int)((uint32_t)(bid * g.mp_r) / (uint32_t)g.grid);
    const int P1 = (bid + 1) * g.mp_q + (int)((uint32_t)((bid + 1) * g.mp_r) / (uint32_t)g.grid);
    const T *wsrc = reinterpret_cast<const T *>(p.wraw);
    constexpr uint32_t ES = sizeof(T);
    // operand views as raw buffers (launcher guarantees each spans < 2^31 bytes)
    const int a_ldc = (int)p.a_ldc, a2_ldc = (int)p.a2_ldc, y_ldc = (int)p.y_ldc, ex_ldc = (int)p.ex_ldc;
    const __amdgpu_buffer_rsrc_t abuf = buf_view(p.a, (uint32_t)(((int64_t)(m - 1) * a_ldc + K) * ES));
    const __amdgpu_buffer_rsrc_t a2buf = buf_view(BNG ? p.a2 : p.a, BNG ? (uint32_t)(((int64_t)(m - 1) * a2_ldc + K) * ES) : 0u);
    const __amdgpu_buffer_rsrc_t ybuf = buf_view(p.y, (uint32_t)(((int64_t)(m - 1) * y_ldc + N) * ES));
    const int side_ldc = (int)p.side_ldc, ex2_ldc = (int)p.ex2_ldc;
    const __amdgpu_buffer_rsrc_t sbuf = buf_view(SAVE ? p.side : p.a,
                                                 SAVE ? (uint32_t)(((int64_t)(m - 1) * side_ldc + K) * ES) : 0u);
    const __amdgpu_buffer_rsrc_t xbuf = buf_view(p.ex ? p.ex : p.y,
                                                 p.ex ? (uint32_t)(((int64_t)(m - 1) * ex_ldc + N) * ES) : 0u);

    // ---- input batches: up to 128 consecutive positions, loaded to registers ----
    // This thread loads and transforms row tid / 4 of a batch, channel vectors
    // 4 j + (tid & 3): 4 consecutive lanes cover 64 contiguous bytes of one
    // pixel, 16 lane groups 16 rows (4 distinct coefficient addresses per
    // wave: LDS broadcast).  Batch t (positions from P0 + 128 (t + 1) + H1)
    // replaces ring rows in phase B of tile t; it is loaded AHEAD tiles
    // earlier into one of two register buffers, so its loads are in flight
    // for AHEAD tile periods.
    // own: the position lies in this workgroup's range (SAVE stores it)
    struct Batch { vec16 a[NVA]; vec16 b[NVB]; int pix; bool own; };
    auto load_rows = [&](int q0, int cnt, Batch &bt) __attribute__((always_inline)) {
        const int arow = tid >> 2;
        const P3Base b = p3_base(q0, g);
        const int pp = p3_pixel_at(b, q0 + arow, g, H, W);
        bt.pix = arow < cnt ? pp : -1;
        bt.own = q0 + arow >= P0 && q0 + arow < P1;
        #pragma unroll
        for (int j = 0; j < NVA; j++) {
            const int c = (4 * j + (tid & 3)) * VEC;
            const bool ok = bt.pix >= 0 && c < K;
            bt.a[j] = bld16(abuf, ok ? (uint32_t)(bt.pix * a_ldc + c) * ES : kBufOff);
            if (BNG) bt.b[j < NVB ? j : 0] = bld16(a2buf, ok ? (uint32_t)(bt.pix * a2_ldc + c) * ES : kBufOff);
        }
    };
    // ---- prologue loads, in the order they are needed: the per-channel
    // parameters (thread c holds channel c; KPC, NPC <= 128), the weights,
    // then the ring fill (the first tile's window, positions
    // [P0 - H1, P0 + 128 + H1) = RING rows in two batches).  Loads complete
    // in issue order for the wait counter, so the weight staging waits only
    // for the parameters and the weights, and the fill stays in flight.
    //   BNRELU: z = max(x * c0 + c1, 0) with c0 = gamma*rstd, c1 = beta - mean*gamma*rstd
    //   BNGRAD: d = c0 * dy + c1 * x + c2  (the deferred BN input gradient: deferred_coef_of)
    float q0 = 0.f, q1 = 0.f, q2 = 0.f, q3 = 0.f, q4 = 0.f;
    if (tid < K && pro == PRO_BNRELU) {
        q0 = p.p_gamma[tid]; q1 = p.p_beta[tid]; q2 = p.p_mean[tid]; q3 = p.p_rstd[tid];
    } else if (tid < K && pro == PRO_BNGRAD) {
        q1 = p.p_mean[tid]; q2 = p.p_rstd[tid];
        if (p.p_split) { q0 = p.p_alpha[tid]; q3 = p.p_betap[tid]; }
        else { q0 = p.p_gamma[tid]; q3 = p.p_dgamma[tid]; q4 = p.p_dbeta[tid]; }
    }
    float ep0 = 0.f, ep1 = 1.f, epg = 0.f, epb = 0.f;
    if (tid < N && BNB) { ep0 = p.e_mean[tid]; ep1 = p.e_rstd[tid]; epg = p.e_gamma[tid]; epb = p.e_beta[tid]; }
    if (tid < N && EK == EK_STATS && p.e_shift) ep0 = p.e_shift[tid];     // statistics of y - shift

    // weights -> LDS stage as Ws[tap][n][k] (zero outside K x N), in batches
    // of kWB vectors per thread whose loads are all in flight before any write
    constexpr int kWB = 16;
    const __amdgpu_buffer_rsrc_t wbuf = buf_view(wsrc, (uint32_t)(9 * K * N * ES));
    constexpr int wtotal = 9 * KPC * NPC / VEC;
    constexpr int VPK = KPC / VEC;
    vec16 wv[kWB];
    auto load_w = [&](int base) __attribute__((always_inline)) {
        #pragma unroll
        for (int u = 0; u < kWB; u++) {
            if (base + u * kP3Threads >= wtotal) break;      // (uniform: no empty loads issued)
            const int i = base + u * kP3Threads + tid;
            int off;
            if (!p.wtrans) {  // forward: W[tap][k][n] (k = c_in, n = c_out); consecutive lanes take consecutive k
                const int tap = i / (KPC * VPRO), rem = i % (KPC * VPRO);
                const int n0 = (rem / KPC) * VEC, k = rem % KPC;
                off = i < wtotal && k < K && n0 < N ? ((tap * K + k) * N + n0) * (int)ES : (int)kBufOff;
            } else {          // data gradient: W[8 - tap][n][k] (n = c_in, k = c_out), rows of k
                const int tap = i / (NPC * VPK), rem = i % (NPC * VPK);
                const int n = rem / VPK, k0 = (rem % VPK) * VEC;
                off = i < wtotal && n < N && k0 < K ? (((8 - tap) * N + n) * K + k0) * (int)ES : (int)kBufOff;
            }
            wv[u] = bld16(wbuf, (uint32_t)off);
        }
    };
    auto write_w = [&](int base) __attribute__((always_inline)) {
        #pragma unroll
        for (int u = 0; u < kWB; u++) {
            const int i = base + u * kP3Threads + tid;
            if (i >= wtotal) break;
            if (!p.wtrans) {  // scatter the n row to columns (a wave writes 64 consecutive k of a column)
                const int tap = i / (KPC * VPRO), rem = i % (KPC * VPRO);
                const int n0 = (rem / KPC) * VEC, k = rem % KPC;
                #pragma unroll
                for (int e = 0; e < VEC; e++)
                    Ws[(tap * NPC + n0 + e) * g.ldw + k] =
                        (T)((e & 1) ? (wv[u].u[e >> 1] >> 16) : (wv[u].u[e >> 1] & 0xffffu));
            } else {          // rows copy straight
                const int tap = i / (NPC * VPK), rem = i % (NPC * VPK);
                const int n = rem / VPK, k0 = (rem % VPK) * VEC;
                *reinterpret_cast<vec16 *>(Ws + (tap * NPC + n) * g.ldw + k0) = wv[u];
            }
        }
    };
    load_w(0);
    const int H1 = g.PW + 1;
    Batch bt0, bt1;
    load_rows(P0 - H1, kP3BM, bt0);
    load_rows(P0 - H1 + kP3BM, RING - kP3BM, bt1);
    write_w(0);
    for (int base = kWB * kP3Threads; base < wtotal; base += kWB * kP3Threads) {
        load_w(base);
        write_w(base);
    }
    // ---- per-channel prologue / epilogue parameters -> LDS ----
    if (tid < KPC) {
        const int c = tid;
        float c0 = 0.f, c1 = 0.f, c2 = 0.f;
        if (c < K && pro == PRO_BNRELU) bn_coef(q0, q1, q2, q3, c0, c1);
        else if (c < K && pro == PRO_BNGRAD) deferred_coef_of(p.p_split, 1.0f / (float)m, q0, q1, q2, q3, q4, c0, c1, c2);
        coef[c] = c0; coef[KPC + c] = c1; coef[2 * KPC + c] = c2;
    }
    if (tid < NPC) {
        const int c = tid;
        float e0 = ep0, e1 = ep1, e2 = 0.f, e3 = 0.f;
        if (c < N && BNB) {      // mean, rstd and the forward's y = x c0 + c1
            bn_coef(epg, epb, e0, e1, e2, e3);
            // e_zsrc: the operand is the stored z = relu(y): mask [z > 0] as
            // fma(z, 1, 0) > 0, xhat = (z - beta) / gamma, unless the channel's
            // vector holds a gamma = 0 channel (its threads read x: ex2)
            bool zv = ZK;
            if (zv) {                              // (the eight loads together, then the test)
                float ga[VEC];
                #pragma unroll
                for (int i = 0; i < VEC; i++) ga[i] = p.e_gamma[(c & ~(VEC - 1)) + i];
                #pragma unroll
                for (int i = 0; i < VEC; i++) zv = zv && ga[i] != 0.f;
            }
            if (zv) { e0 = p.e_beta[c]; e1 = 1.0f / p.e_gamma[c]; e2 = 1.f; e3 = 0.f; }
        }
        epi[c] = e0; epi[NPC + c] = e1; epi[2 * NPC + c] = e2; epi[3 * NPC + c] = e3;
    }
    __syncthreads();
    // this wave's weight fragments: K slice wk, columns wn*32 + {0, 16}, nine taps
    typename M::frag bfr[9][2];
    #pragma unroll
    for (int tap = 0; tap < 9; tap++)
        #pragma unroll
        for (int cb = 0; cb < 2; cb++)
            bfr[tap][cb] = M::load(Ws + (tap * NPC + wn * 32 + cb * 16 + (lane & 15)) * g.ldw + wk * 32 +
                                   (lane >> 4) * M::KPL);
    // epilogue channels of this thread are fixed (their BN parameters are
    // read from LDS per tile: registers are the occupancy limit)
    const int v = tid % VPRO, r0 = tid / VPRO;
    const int n = v * VEC;
    const bool col_ok = n < N;
    constexpr bool zsrc = ZK;
    bool zs = zsrc && col_ok;                      // this thread's vector reads z (else x)
    if (zsrc) {                                    // (the eight loads together, then the test)
        float ga[VEC];
        #pragma unroll
        for (int e = 0; e < VEC; e++) ga[e] = p.e_gamma[col_ok ? n + e : 0];
        #pragma unroll
        for (int e = 0; e < VEC; e++) zs = zs && ga[e] != 0.f;
    }
    const T *zsrc_col = reinterpret_cast<const T *>(zs ? p.ex : (p.ex2 ? p.ex2 : p.ex)) + (col_ok ? n : 0);
    const int zsrc_ldc = zs ? ex_ldc : ex2_ldc;

    // ---- prologue transform of a batch, then the ring writes.  The mode
    // switch is wave-uniform and outside the vector loop; invalid rows are
    // zeroed on the packed words and rows past the batch go to a junk row, so
    // each mode's vectors are straight-line code; only the copies of the first
    // 16 ring rows are written under a branch (around stores, no loads).
    // 32 NVA = KPC: every channel vector is in range. ----
    static_assert(32 * NVA == KPC, "batch vectors");
    auto store_rows = [&](int cnt, int slot0, Batch &bt) __attribute__((always_inline)) {
        const int arow = tid >> 2;
        const vec16 *ra = bt.a, *rb = bt.b;
        int s = slot0 + arow;
        s = s >= RING ? s - RING : s;
        const bool live = arow < cnt;
        const int s1 = live ? s : RING + 16;
        const int s2 = live && s < 16 ? s + RING : RING + 16;
        const uint32_t keep = bt.pix >= 0 ? 0xffffffffu : 0u;    // padding rows: zeros
        vec16 outv[NVA];
        if (BNG) {                                        // PRO_BNGRAD: d = c0 dy + c1 x + c2
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                const int c = (4 * j + (tid & 3)) * VEC;
                float f[VEC], x[VEC], c0[VEC], c1[VEC], c2[VEC];
                Elem<T>::unpack(ra[j], f);
                Elem<T>::unpack(rb[j < NVB ? j : 0], x);
                lds_f8(coef + c, c0);
                lds_f8(coef + KPC + c, c1);
                lds_f8(coef + 2 * KPC + c, c2);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = __builtin_fmaf(c0[e], f[e], __builtin_fmaf(c1[e], x[e], c2[e]));
                outv[j] = Elem<T>::pack(f);
                #pragma unroll
                for (int i = 0; i < 4; i++) outv[j].u[i] &= keep;
            }
        } else if (pro == PRO_BNRELU) {                   // z = max(x c0 + c1, 0)
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                const int c = (4 * j + (tid & 3)) * VEC;
                float f[VEC], ca[VEC], cb[VEC];
                Elem<T>::unpack(ra[j], f);
                lds_f8(coef + c, ca);
                lds_f8(coef + KPC + c, cb);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = __builtin_fmaxf(bn_lin(f[e], ca[e], cb[e]), 0.f);
                outv[j] = Elem<T>::pack(f);
                #pragma unroll
                for (int i = 0; i < 4; i++) outv[j].u[i] &= keep;
                if (SAVE)
                    bst16(sbuf, live && bt.own && bt.pix >= 0 && c < K ? (uint32_t)(bt.pix * side_ldc + c) * ES : kBufOff,
                          outv[j]);
            }
        } else if (pro == PRO_RELU) {                     // (padding rows load zeros)
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float f[VEC];
                Elem<T>::unpack(ra[j], f);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = __builtin_fmaxf(f[e], 0.f);
                outv[j] = Elem<T>::pack(f);
            }
        } else {
            #pragma unroll
            for (int j = 0; j < NVA; j++) outv[j] = ra[j];     // out-of-range loads read zero
        }
        #pragma unroll
        for (int j = 0; j < NVA; j++) {
            const int c = (4 * j + (tid & 3)) * VEC;
            *reinterpret_cast<vec16 *>(ring + s1 * lda + c) = outv[j];
        }
        // the copies of the first 16 ring rows: a branch around stores only
        // (most waves hold none of those rows and skip the writes)
        if (s2 != RING + 16)
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                const int c = (4 * j + (tid & 3)) * VEC;
                *reinterpret_cast<vec16 *>(ring + s2 * lda + c) = outv[j];
            }
    };

    // ---- epilogue operand: thread = one channel vector of rows r0, r0+RSTEP, ... ----
    vec16 rx[NVX];
    int epix[RPT];                  // pixels of this thread's epilogue rows (-1: padding / past the end)
    float s1[VEC], s2[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) { s1[e] = 0.f; s2[e] = 0.f; }
    auto load_epi = [&](int p0, int nrows) __attribute__((always_inline)) {
        const P3Base eb = p3_base(p0, g);
        #pragma unroll
        for (int j = 0; j < RPT; j++) {
            const int r = r0 + j * RSTEP;
            const int pp = p3_pixel_at(eb, p0 + r, g, H, W);
            epix[j] = col_ok && r < nrows ? pp : -1;
        }
        if (!READS) return;
        #pragma unroll
        for (int j = 0; j < NVX; j++) {
            const int pp = epix[j];
            const bool ok = pp >= 0;
            if (EK == EK_STORE_ACC) {
                rx[j] = bld16(ybuf, ok ? (uint32_t)(pp * y_ldc + n) * ES : kBufOff);
            } else if (ZK) {   // z, or x (gamma = 0 in the vector): one load from this thread's
                // source at a clamped pixel (a padding or past-the-end row is not used)
                rx[j] = ldg16(zsrc_col + (int64_t)(ok ? pp : 0) * zsrc_ldc);
            } else {
                rx[j] = bld16(xbuf, ok ? (uint32_t)(pp * ex_ldc + n) * ES : kBufOff);
            }
        }
    };

    // ---- ring fill (slots 0 .. RING-1), then the first AHEAD batches and
    // the first tile's epilogue operand (issued first: a wait for it then
    // leaves the batches in flight) ----
    store_rows(kP3BM, 0, bt0);
    store_rows(RING - kP3BM, kP3BM, bt1);
    auto batch_rows = [&](int t) __attribute__((always_inline)) -> int {
        const int c = P1 + H1 - (P0 + kP3BM + H1 + t * kP3BM);
        return c < 0 ? 0 : (c > kP3BM ? kP3BM : c);
    };
    load_epi(P0, P1 - P0 < kP3BM ? P1 - P0 : kP3BM);
    if (batch_rows(0) > 0) load_rows(P0 + kP3BM + H1, batch_rows(0), bt0);
    if (AHEAD == 2 && batch_rows(1) > 0) load_rows(P0 + 2 * kP3BM + H1, batch_rows(1), bt1);
    int sb = H1;                    // ring slot of the first row of the current tile
    __syncthreads();

    // Per tile two phases separated by barriers: (A) matrix cores on the
    // tile's ring window, partial tiles to LDS; (B) the ring rows of the tile
    // after next's window replace the rows only this tile needed, the
    // epilogue of this tile runs, and the next batch and epilogue operand are
    // loaded.
    auto tile = [&](int p0, Batch &bt) __attribute__((always_inline)) {
        const int tt = (p0 - P0) / kP3BM;

        // ---- (A) matrix cores: 16 RB rows x 32 columns x 32 K per wave, nine taps ----
        f32x4 acc[RB][2];               // set by the first tap's products
        // A fragment = ring row u (wave-uniform) + this lane's fixed offset;
        // the next tap's fragments are read while this tap's are multiplied
        const int lane_off = (lane & 15) * lda + wk * 32 + (lane >> 4) * M::KPL;
        const int ubase = sb + __builtin_amdgcn_readfirstlane(wr) * 16 * RB;
        // (double-buffered unless the 128-column variants' registers cannot hold it)
        constexpr int NB = WN == 4 ? 1 : 2;
        typename M::frag af[NB][RB];
        auto load_tap = [&](int tap, typename M::frag *dst) __attribute__((always_inline)) {
            const int off = (tap / 3 - 1) * PW + (tap % 3 - 1);
            #pragma unroll
            for (int ib = 0; ib < RB; ib++) {
                int u = ubase + ib * 16 + off;           // in [-(PW + 1), 2 RING)
                u = u < 0 ? u + RING : (u >= RING ? u - RING : u);
                dst[ib] = M::load(ring + u * lda + lane_off);
            }
        };
        if (NB == 2) load_tap(0, af[0]);
        #pragma unroll
        for (int tap = 0; tap < 9; tap++) {
            if (NB == 1) load_tap(tap, af[0]);
            else if (tap + 1 < 9) load_tap(tap + 1, af[(tap + 1) % NB]);
            #pragma unroll
            for (int ib = 0; ib < RB; ib++) {
                if (tap == 0) {
                    M::mma0(acc[ib][0], bfr[0][0], af[0][ib]);
                    M::mma0(acc[ib][1], bfr[0][1], af[0][ib]);
                } else {
                    M::mma(acc[ib][0], bfr[tap][0], af[tap % NB][ib]);
                    M::mma(acc[ib][1], bfr[tap][1], af[tap % NB][ib]);
                }
            }
        }
        // ---- float32 partial tile of this K slice -> LDS (the weights are
        // the matrix cores' first operand, so a lane holds four consecutive
        // channels of one position: one 16-byte write) ----
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < 2; cb++) {
                const int row = wr * 16 * RB + ib * 16 + (lane & 15);
                const int col = wn * 32 + cb * 16 + (lane >> 4) * 4;
                *reinterpret_cast<f32x4 *>(red + (wk * kP3BM + row) * ldr + col) = acc[ib][cb];
            }
        __syncthreads();
        // ---- (B) ring rows of the tile after next, then this tile's epilogue ----
        store_rows(batch_rows(tt), (tt * kP3BM) % RING, bt);
        // ---- epilogue row pass: sum of the K slices (fixed order), rounded to
        // the storage type; all outputs of this thread first (no branch,
        // invalid rows contribute zeros), then the stores back to back ----
        {
            vec16 vo[RPT];
            float eM[VEC], eR[VEC], eC0[VEC], eC1[VEC];
            if (EK == EK_STATS) lds_f8(epi + n, eM);                  // shift
            if (BNB) {
                lds_f8(epi + n, eM);
                lds_f8(epi + NPC + n, eR);
                lds_f8(epi + 2 * NPC + n, eC0);
                lds_f8(epi + 3 * NPC + n, eC1);
            }
            #pragma unroll
            for (int j = 0; j < RPT; j++) {
                const int r = r0 + j * RSTEP;
                const bool ok = epix[j] >= 0;
                float f[VEC];
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = 0.f;
                #pragma unroll
                for (int q = 0; q < WK; q++) {
                    const float4 *src = reinterpret_cast<const float4 *>(red + (q * kP3BM + r) * ldr + n);
                    const float4 lo = src[0], hi = src[1];
                    f[0] += lo.x; f[1] += lo.y; f[2] += lo.z; f[3] += lo.w;
                    f[4] += hi.x; f[5] += hi.y; f[6] += hi.z; f[7] += hi.w;
                }
                const vec16 cv = Elem<T>::pack(f);
                Elem<T>::unpack(cv, f);
                vo[j] = cv;
                if (EK == EK_STORE_ACC) {
                    float old[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], old);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] += old[e];
                    vo[j] = Elem<T>::pack(f);
                } else if (EK == EK_STATS) {
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float fv = ok ? f[e] - eM[e] : 0.f;
                        s1[e] += fv;
                        s2[e] += fv * fv;
                    }
                } else if (EK == EK_RELUMASK) {
                    float yv[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], yv);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] = yv[e] > 0.f ? f[e] : 0.f;
                    vo[j] = Elem<T>::pack(f);
                } else if (BNB) {
                    float x[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], x);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float xh = (x[e] - eM[e]) * eR[e];
                        const float d = ok && bn_lin(x[e], eC0[e], eC1[e]) > 0.f ? f[e] : 0.f;
                        f[e] = d;
                        s1[e] += d;
                        s2[e] += d * xh;
                    }
                    vo[j] = Elem<T>::pack(f);
                }
            }
            #pragma unroll
            for (int j = 0; j < RPT; j++)
                bst16(ybuf, epix[j] >= 0 ? (uint32_t)(epix[j] * y_ldc + n) * ES : kBufOff, vo[j]);
        }
        // unconditional (past the end: zero rows, out-of-range offsets), so the
        // compiler's memory counters stay exact across the loop
        load_epi(p0 + kP3BM, P1 - p0 - kP3BM < kP3BM ? (P1 - p0 - kP3BM > 0 ? P1 - p0 - kP3BM : 0) : kP3BM);
        load_rows(P0 + kP3BM + H1 + (tt + AHEAD) * kP3BM, batch_rows(tt + AHEAD), bt);
        sb += kP3BM;
        if (sb >= RING) sb -= RING;
        __syncthreads();
    };
    for (int p0 = P0; p0 < P1; p0 += 2 * kP3BM) {
        tile(p0, bt0);
        if (p0 + kP3BM >= P1) break;
        tile(p0 + kP3BM, AHEAD == 2 ? bt1 : bt0);
    }

    // ---- per-workgroup statistics partial row ----
    if (EK == EK_STATS || BNB) {
        #pragma unroll
        for (int e = 0; e < VEC; e++) {
            red[r0 * NPC + n + e] = s1[e];
            red[(RSTEP + r0) * NPC + n + e] = s2[e];
        }
        lds_colsum2(red, RSTEP, NPC, NPC, kP3Threads, tid, p.part + (int64_t)blockIdx.x * 2 * N,
                    p.part + (int64_t)blockIdx.x * 2 * N + N, N);
    }
}

// ------------------------------------------------------------- launchers ---
static int p3_cus()
{
    static int cus = 0;
    if (!cus) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
    }
    return cus;
}

bool conv3x3_supported(int dtype, int K, int N, int H, int W)
{
    if (dtype != DT_BF16 || K > 128 || N > 128 || W > kP3MaxW || W < 1 || H > kP3MaxH || H < 1) return false;
    const P3Geom g = p3_geom(K, N, W);
    const int wk = g.KP / 32, wn = g.NP / 32;
    if (wk == 3 || wk * wn > 4) return false;      // at most 64 rows x 2 column blocks of accumulators per wave
    return g.lds <= 160 * 1024;
}

// One workgroup per 32 pixels, at most one per CU: a small image (14 x 14,
// 7 x 7) would otherwise leave most CUs idle, and each workgroup's launch
// prologue (weights, parameters, ring fill) is a fixed cost that more
// workgroups share out; a range shorter than a tile is a masked tile.
int64_t conv3x3_partial_rows(int64_t m)
{
    const int64_t tiles = ceil_div(m, 32);
    const int64_t g = p3_cus();
    return tiles < g ? tiles : g;
}

template <int WK, int WN, int EK, int PC>
static hipError_t run_p3(const RowsParams &p, const P3Geom &g0, hipStream_t s)
{
    constexpr bool BNG = PC == PC3_BNGRAD;
    auto kern = k_conv3x3<WK, WN, EK, PC>;
    static bool attr_set = false;
    if (!attr_set) {
        const hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int grid = (int)conv3x3_partial_rows(p.m);
    P3Geom g = g0;
    g.grid = grid;
    g.mp_q = g.MP / grid;
    g.mp_r = g.MP % grid;
    const double e = 2.0, m = (double)p.m;
    double a = m * p.K;
    if (BNG || PC == PC3_BNRELU_SAVE) a *= 2.0;     // second operand read / z written
    double out = m * p.N;
    if (EK == EK_STORE_ACC || EK == EK_RELUMASK || EK == EK_BNBWD || EK == EK3_BNBWD_Z) out += m * p.N;
    TraceScope tr(KC_CONV, KID_CONV_3X3, s, e * (a + out + 9.0 * p.K * p.N), 2.0 * m * 9.0 * p.K * p.N);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kP3Threads), g.lds, s, p, g);
    return hipGetLastError();
}

// (K slices, N slices) with WK * WN <= 4, WK in {1, 2, 4}
template <int EK, int PC>
static hipError_t run_p3_shape(const RowsParams &p, const P3Geom &g, hipStream_t s)
{
    const int wk = g.KP / 32, wn = g.NP / 32;
    switch (wk * 8 + wn) {
    case 1 * 8 + 1: return run_p3<1, 1, EK, PC>(p, g, s);
    case 1 * 8 + 2: return run_p3<1, 2, EK, PC>(p, g, s);
    case 1 * 8 + 4: return run_p3<1, 4, EK, PC>(p, g, s);
    case 2 * 8 + 1: return run_p3<2, 1, EK, PC>(p, g, s);
    case 2 * 8 + 2: return run_p3<2, 2, EK, PC>(p, g, s);
    case 4 * 8 + 1: return run_p3<4, 1, EK, PC>(p, g, s);
    default: return hipErrorInvalidValue;
    }
}

template <int PC>
static hipError_t run_p3_ek(const RowsParams &p, const P3Geom &g, int ek, hipStream_t s)
{
    switch (ek) {
    case EK_STORE: return run_p3_shape<EK_STORE, PC>(p, g, s);
    case EK_STORE_ACC: return run_p3_shape<EK_STORE_ACC, PC>(p, g, s);
    case EK_STATS: return run_p3_shape<EK_STATS, PC>(p, g, s);
    case EK_RELUMASK: return run_p3_shape<EK_RELUMASK, PC>(p, g, s);
    default: return p.e_zsrc ? run_p3_shape<EK3_BNBWD_Z, PC>(p, g, s) : run_p3_shape<EK_BNBWD, PC>(p, g, s);
    }
}

hipError_t launch_conv3x3(const RowsParams &p, hipStream_t s)
{
    if (!p.a || !p.wraw || !p.y || p.taps != 9 || p.pro == PRO_POOLUP || !conv3x3_supported(p.dtype, p.K, p.N, p.h, p.w))
        return hipErrorInvalidValue;
    if (p.pro == PRO_BNRELU && (!p.p_mean || !p.p_gamma || !p.p_rstd || !p.p_beta)) return hipErrorInvalidValue;
    if (p.pro == PRO_BNGRAD && (!p.a2 || !p.p_mean || !p.p_rstd ||
                                (p.p_split ? (!p.p_alpha || !p.p_betap) : (!p.p_gamma || !p.p_dbeta || !p.p_dgamma))))
        return hipErrorInvalidValue;
    if ((p.epi == EPI_STATS || p.epi == EPI_BNBWD) && !p.part) return hipErrorInvalidValue;
    if (p.epi == EPI_BNBWD && p.e_scale) return hipErrorInvalidValue;     // summed-gradient form: conv_rows
    if (p.epi == EPI_BNBWD && (!p.ex || !p.e_mean || !p.e_rstd || !p.e_gamma || !p.e_beta)) return hipErrorInvalidValue;
    if (p.epi == EPI_RELUMASK && !p.ex) return hipErrorInvalidValue;
    if ((int64_t)p.n * p.h * p.w != p.m || p.m < 1) return hipErrorInvalidValue;
    const bool save = p.pro == PRO_BNRELU && p.side;
    if (p.side && (!save || p.wtrans || (p.epi != EPI_STORE && p.epi != EPI_STATS) || p.accumulate))
        return hipErrorInvalidValue;
    if (p.e_zsrc && (p.epi != EPI_BNBWD || !p.ex2)) return hipErrorInvalidValue;
    // 32-bit pixel indices and raw-buffer operand views: every span below 2^31 bytes
    const int64_t lim = (int64_t)1 << 31;
    if (p.m >= (lim >> 1) || (p.m * p.a_ldc + p.K) * 2 >= lim || (p.m * p.y_ldc + p.N) * 2 >= lim ||
        (p.a2 && (p.m * p.a2_ldc + p.K) * 2 >= lim) || (p.ex && (p.m * p.ex_ldc + p.N) * 2 >= lim) ||
        (save && (p.m * p.side_ldc + p.K) * 2 >= lim) || (p.ex2 && (p.m * p.ex2_ldc + p.N) * 2 >= lim))
        return hipErrorInvalidValue;
    P3Geom g = p3_geom(p.K, p.N, p.w);
    g.PH = p.h + 2;
    g.inv_ph = 1.0 / g.PH;
    g.rpw = (uint32_t)(((1u << 20) + g.PW - 1) / g.PW);
    g.rph = (uint32_t)(((1u << 20) + g.PH - 1) / g.PH);
    const int64_t mp = (int64_t)p.n * g.PH * g.PW;                // padded positions
    if (mp >= (lim >> 1)) return hipErrorInvalidValue;
    g.MP = (int)mp;
    const int ek = epilogue_kind(p.epi, p.accumulate, 0);
    if (save) return ek == EK_STATS ? run_p3_shape<EK_STATS, PC3_BNRELU_SAVE>(p, g, s)
                                    : run_p3_shape<EK_STORE, PC3_BNRELU_SAVE>(p, g, s);
    if (p.pro == PRO_BNGRAD) return run_p3_ek<PC3_BNGRAD>(p, g, ek, s);
    if (p.pro == PRO_BNRELU && ek == EK_STATS) return run_p3_shape<EK_STATS, PC3_BNRELU>(p, g, s);
    return run_p3_ek<PC3_RUNTIME>(p, g, ek, s);
}

}  // namespace bnr
