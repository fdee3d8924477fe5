// Training gradients of OctreeNCA (Sec. 3.2, efficient training; supplement
// S7): the backward of one NCA step for fp32 states, the adjoint of the
// upsample + inject, and a readout-channel MSE as the synthetic loss.
//
// One step S -> S' = S + m * u (hidden channels, Sec. 3.1) is taken back,
// for G' = dL/dS', by recomputing its activations from S (nothing of the
// forward but the states is kept):
//   gu = m G' (hidden channels), dW2 += gu h^T, ga = (W2^T gu) * [a > 0],
//   dW1 += ga f^T, db1 += ga, [gS, gP] = W1^T ga, dconv_b += gP,
//   dK[c][t] += gP[p][c] S[p + o_t][c], dL/dS = G' + gS + conv^T(gP).
// Three kernels:
//   1. bwd_cell: four lanes per cell, blocks of 64 cells (halo tile of S in
//      LDS): perception, then the hidden units streamed once, a quarter per
//      lane, each giving a, h, gh and ga; writes G' + gS and gP to memory and
//      keeps the cells' records [f | h | ga | gu | gP] in LDS, from which the
//      block forms its sums of every weight-gradient entry (4 x 4 register
//      blocks of the outer-product sums) and stores them as one row;
//   2. bwd_conv_t: dL/dS = (G' + gS) + the transposed depthwise convolution of
//      gP (halo tile of gP in LDS);
//   3. wgrad_reduce: per 64 entries, 16 waves add the block rows in fp64
//      (wave w takes rows w, w + 16, ... in order, then the waves' sums in
//      wave order) to the caller's gradients (accumulated, so the steps of a
//      level sum up).
// One step (octree_nca_step_backward) runs the three.  A level of a training
// step runs bwd_cell once per step, each after the first forming its G' from
// the previous one's (G' + gS, gP) with the transposed convolution fused and
// adding to its block's partial row, then bwd_conv_t and wgrad_reduce once.
#include "launch.h"

namespace octnca {

namespace {

constexpr int kBwdThreads = 256;
constexpr int kWgCells = 64;   // cells per block of the weight-gradient partial sums

template <int NDIM> struct BwdTile;
template <> struct BwdTile<2> { static constexpr int TZ = 1, TY = 8, TX = 32; };
template <> struct BwdTile<3> { static constexpr int TZ = 4, TY = 8, TX = 8; };

// Record of a cell: f (2C) | h (H) | ga (H) | gu (C) | gP (C), stored field
// by field (entry k of cell p at rec[k * cells + p]) so that neighbouring
// cells' entries are neighbouring words.
template <int C, int H> struct Rec {
    static constexpr int F = 0, Hh = 2 * C, GA = 2 * C + H, GU = 2 * C + 2 * H,
                         GP = 3 * C + 2 * H, N = 4 * C + 2 * H;
};

// Number of weight-gradient entries: dW1 (H x 2C), dW2 (C x H), db1 (H),
// dconv_b (C), dconv_w (C x taps), in that order.
template <int C, int H, int TAPS> struct WG {
    static constexpr int W1 = 0, W2 = 2 * C * H, B1 = 3 * C * H, CB = 3 * C * H + H,
                         CW = 3 * C * H + H + C, N = 3 * C * H + H + C + C * TAPS;
};

// LDS staging of TOTAL words by the block: word i = load(i), stored by
// store(i, value).  The loads go out in batches of BATCH per thread before
// their stores, so that a thread's loads are in flight together (a plain
// strided loop waits for each load before the next).
template <int TOTAL, int BATCH, class Load, class Store>
__device__ __forceinline__ void stage(Load load, Store store) {
    constexpr int ITERS = (TOTAL + kBwdThreads - 1) / kBwdThreads;
#pragma unroll 1
    for (int it0 = 0; it0 < ITERS; it0 += BATCH) {
        float v[BATCH];
#pragma unroll
        for (int j = 0; j < BATCH; ++j) {
            const int i = (int)threadIdx.x + (it0 + j) * kBwdThreads;
            v[j] = load(min(i, TOTAL - 1));
        }
#pragma unroll
        for (int j = 0; j < BATCH; ++j) {
            const int i = (int)threadIdx.x + (it0 + j) * kBwdThreads;
            if (it0 + j < ITERS && i < TOTAL) store(i, v[j]);
        }
    }
}

// Sums over kWgCells cells of every weight-gradient entry, from the cells'
// records in LDS (a row of RS = R::N + 4 words per cell, zero rows for cells
// outside the grid).  Each thread takes jobs of entries that share operands:
// a 4 x 4 block of dW1 (ga[j..j+3] x f[k..k+3]) or of dW2 (gu[c..c+3] x
// h[j..j+3]), four entries of db1 or dconv_b, or one tap of dconv_w for four
// channels (state(p, t, c) gives channel c of the tap-t neighbour of cell p);
// per cell a job reads two 16-byte words and does up to 16 FMAs, in cell
// order.  out receives the G::N sums (one block-major row).
template <int NDIM, int C, int H, class State>
__device__ __forceinline__ void wgrad_block(const float *recs, State state, float *out,
                                            bool accumulate) {
    // the sums start from the block's row (accumulate: the steps of a level,
    // in order) or from zero
    auto start = [&](int o) { return accumulate ? out[o] : 0.f; };
    using R = Rec<C, H>;
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    using G = WG<C, H, TAPS>;
    static_assert(C % 4 == 0 && H % 4 == 0, "entries in blocks of 4");
    constexpr int RS = R::N + 4;
    auto quad = [&](int cell, int e) {
        return *reinterpret_cast<const float4 *>(&recs[cell * RS + e]);
    };
    constexpr int J1 = (H / 4) * (2 * C / 4);    // dW1 blocks
    constexpr int J2 = (C / 4) * (H / 4);        // dW2 blocks
    constexpr int JB = H / 4, JC = C / 4;        // db1, dconv_b quads
    constexpr int JK = (C / 4) * TAPS;           // dconv_w (channel quad, tap)
    constexpr int NJ = J1 + J2 + JB + JC + JK;
    for (int job = threadIdx.x; job < NJ; job += kBwdThreads) {
        if (job < J1 + J2) {
            int ea, eb, o0, os;
            if (job < J1) {                      // dW1[j][k] = sum ga[j] f[k]
                const int jb = job / (2 * C / 4), kb = job % (2 * C / 4);
                ea = R::GA + 4 * jb; eb = R::F + 4 * kb;
                o0 = G::W1 + 4 * jb * 2 * C + 4 * kb; os = 2 * C;
            } else {                             // dW2[c][j] = sum gu[c] h[j]
                const int jj = job - J1, cb = jj / (H / 4), jb = jj % (H / 4);
                ea = R::GU + 4 * cb; eb = R::Hh + 4 * jb;
                o0 = G::W2 + 4 * cb * H + 4 * jb; os = H;
            }
            float acc[4][4];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[r][c] = start(o0 + r * os + c);
#pragma unroll 4
            for (int i = 0; i < kWgCells; ++i) {
                const float4 av = quad(i, ea), bv = quad(i, eb);
                const float ar[4] = {av.x, av.y, av.z, av.w}, br[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(ar[r], br[c], acc[r][c]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) out[o0 + r * os + c] = acc[r][c];
        } else if (job < J1 + J2 + JB + JC) {    // db1[j] = sum ga[j]; dconv_b[c] = sum gP[c]
            const int jj = job - J1 - J2;
            const int e = jj < JB ? R::GA + 4 * jj : R::GP + 4 * (jj - JB);
            const int o0 = jj < JB ? G::B1 + 4 * jj : G::CB + 4 * (jj - JB);
            float sum[4] = {start(o0), start(o0 + 1), start(o0 + 2), start(o0 + 3)};
            for (int i = 0; i < kWgCells; ++i) {
                const float4 v = quad(i, e);
                sum[0] += v.x; sum[1] += v.y; sum[2] += v.z; sum[3] += v.w;
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) out[o0 + r] = sum[r];
        } else {                                 // dconv_w[c][t] = sum gP[c] S[p + o_t][c]
            const int jj = job - J1 - J2 - JB - JC;
            const int cq = jj / TAPS, t = jj % TAPS;
            float sum[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) sum[r] = start(G::CW + (4 * cq + r) * TAPS + t);
#pragma unroll 4
            for (int i = 0; i < kWgCells; ++i) {
                const float4 gpv = quad(i, R::GP + 4 * cq);
                sum[0] = fmaf(gpv.x, state(i, t, 4 * cq + 0), sum[0]);
                sum[1] = fmaf(gpv.y, state(i, t, 4 * cq + 1), sum[1]);
                sum[2] = fmaf(gpv.z, state(i, t, 4 * cq + 2), sum[2]);
                sum[3] = fmaf(gpv.w, state(i, t, 4 * cq + 3), sum[3]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) out[G::CW + (4 * cq + r) * TAPS + t] = sum[r];
        }
    }
}

// bwd_cell: a quad of lanes per cell (lane = 4 * cell + part); part p takes
// hidden units j = 4 i + p, and the four partial feature gradients W1^T ga
// are summed across the quad.  Blocks of 64 cells.  W1 and W2^T sit in LDS
// with rows padded by 4 words, so the quad's four rows fall in different
// banks.  The cells' records stay in LDS, and the block then forms its sums of
// every weight-gradient entry from them (see wgrad_block) and stores one
// block-major row of partial sums; only G' + gS and gP go to memory.
constexpr int kParts = 4;
template <int NDIM> struct BwdCellTile;
template <> struct BwdCellTile<2> { static constexpr int TZ = 1, TY = 2, TX = 32; };
template <> struct BwdCellTile<3> { static constexpr int TZ = 2, TY = 4, TX = 8; };

// G' (dL/dS' of the step) comes from gout, or, when gp_prev is not null,
// from the previous backward step (the step after this one in the forward)
// as gout + conv^T(gp_prev): its pass-through part and the transposed
// convolution of its perception gradient, formed here for the block's cells
// (the tile of gp_prev with a one-cell halo in LDS), so that no separate
// launch has to write dL/dS between the steps of a level.  accumulate: the
// block's weight-gradient sums are added to its partial row (the steps of a
// level, in order) instead of replacing it.
template <int NDIM, int NIN, int C, int H>
__global__ __launch_bounds__(kBwdThreads) void bwd_cell(
    const float *__restrict__ src, const float *__restrict__ gout,
    const float *__restrict__ gp_prev, int dd, int dh, int dw,
    int tiles_x, int tiles_y, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold,
    float *__restrict__ gpart, float *__restrict__ gp, float *__restrict__ partial,
    int64_t cells, int accumulate) {
    using T = BwdCellTile<NDIM>;
    using R = Rec<C, H>;
    constexpr int HZ = NDIM == 3 ? T::TZ + 2 : 1, HY = T::TY + 2, HX = T::TX + 2;
    constexpr int NCELL = HZ * HY * HX;
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    constexpr int HP = H / kParts;   // hidden units per lane
    static_assert(T::TZ * T::TY * T::TX * kParts == kBwdThreads, "a quad of lanes per tile cell");
    static_assert(H % kParts == 0 && C % kParts == 0, "parts of equal size");
    __shared__ float tile[C][NCELL];   // channel-major: neighbouring cells, neighbouring words
    __shared__ __align__(16) float sw1[H][2 * C + 4];   // W1
    __shared__ __align__(16) float sw2[H][C + 4];       // W2^T
    __shared__ float sb1[H];
    constexpr int RS = R::N + 4;   // words per record row (16-byte aligned rows)
    __shared__ __align__(16) float recs[kWgCells * RS];   // [cell][entry]
    // gp_prev of the tile and its halo ([c][cell], for the fused G'), in the
    // record rows' space: read before the first record is written
    static_assert(C * NCELL <= kWgCells * RS, "gp_prev tile fits the record rows");
    float *const gtile = recs;

    int b = blockIdx.x;
    const int bx = b % tiles_x;
    b /= tiles_x;
    const int by = b % tiles_y;
    const int bz = b / tiles_y;
    const int x0 = bx * T::TX, y0 = by * T::TY, z0 = bz * T::TZ;
    stage<NCELL * C, 8>(
        [&](int i) {
            const int c = i / NCELL, cell = i % NCELL;
            const int lx = cell % HX, ly = (cell / HX) % HY, lz = cell / (HX * HY);
            const int gx = x0 + lx - 1, gy = y0 + ly - 1, gz = NDIM == 3 ? z0 + lz - 1 : 0;
            const bool in = gx >= 0 && gx < dw && gy >= 0 && gy < dh && gz >= 0 && gz < dd;
            const int cx = min(max(gx, 0), dw - 1), cy = min(max(gy, 0), dh - 1),
                      cz = min(max(gz, 0), dd - 1);
            const float v = src[(((int64_t)cz * dh + cy) * dw + cx) * C + c];
            return in ? v : 0.f;
        },
        [&](int i, float v) { tile[i / NCELL][i % NCELL] = v; });
    if (gp_prev != nullptr)
        stage<NCELL * C, 8>(
            [&](int i) {
                const int c = i / NCELL, cell = i % NCELL;
                const int lx = cell % HX, ly = (cell / HX) % HY, lz = cell / (HX * HY);
                const int gx = x0 + lx - 1, gy = y0 + ly - 1, gz = NDIM == 3 ? z0 + lz - 1 : 0;
                const bool in = gx >= 0 && gx < dw && gy >= 0 && gy < dh && gz >= 0 && gz < dd;
                const int cx = min(max(gx, 0), dw - 1), cy = min(max(gy, 0), dh - 1),
                          cz = min(max(gz, 0), dd - 1);
                const float v = gp_prev[c * cells + ((int64_t)cz * dh + cy) * dw + cx];
                return in ? v : 0.f;
            },
            [&](int i, float v) { gtile[i] = v; });
    stage<H * 2 * C, 8>([&](int i) { return w1[i]; },
                        [&](int i, float v) { sw1[i / (2 * C)][i % (2 * C)] = v; });
    stage<C * H, 8>([&](int i) { return w2[i]; },
                    [&](int i, float v) { sw2[i % H][i / H] = v; });
    for (int i = threadIdx.x; i < H; i += kBwdThreads) sb1[i] = b1[i];
    __syncthreads();

    const int part = threadIdx.x % kParts, cl = threadIdx.x / kParts;
    const int tx = cl % T::TX, ty = (cl / T::TX) % T::TY, tz = cl / (T::TX * T::TY);
    const int x = x0 + tx, y = y0 + ty, z = z0 + tz;
    // a quad outside the grid computes on a clamped cell and stores nothing
    // (no early return: the quad's lanes exchange values below)
    const bool valid = x < dw && y < dh && z < dd;
    const int centre = ((tz + (NDIM == 3 ? 1 : 0)) * HY + ty + 1) * HX + tx + 1;
    const int64_t idx =
        ((int64_t)min(z, dd - 1) * dh + min(y, dh - 1)) * dw + min(x, dw - 1);

    float f[2 * C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        f[c] = tile[c][centre];
        f[C + c] = conv_b[c];
    }
#pragma unroll 1
    for (int t = 0; t < TAPS; ++t) {
        const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
        const int nb = centre + (dz * HY + dy) * HX + dx;
#pragma unroll
        for (int c = 0; c < C; ++c) f[C + c] = fmaf(conv_w[c * TAPS + t], tile[c][nb], f[C + c]);
    }
    const bool fire = cell_fires(seed, level, step, batch, (uint64_t)idx, threshold);
    constexpr int FP = 2 * C / kParts, CP = C / kParts;
    // G' = dL/dS' of this cell, the quad's part: channels part * CP + k
    float gq[CP];
#pragma unroll
    for (int k = 0; k < CP; ++k) gq[k] = gout[idx * C + part * CP + k];
    if (gp_prev != nullptr) {
        // cell p receives K[c][t] gP[p - o_t] from each tap t
#pragma unroll
        for (int t = 0; t < TAPS; ++t) {
            const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
            const int nb = centre - (dz * HY + dy) * HX - dx;
#pragma unroll
            for (int k = 0; k < CP; ++k) {
                const int c = part * CP + k;
                gq[k] = fmaf(conv_w[c * TAPS + t], gtile[c * NCELL + nb], gq[k]);
            }
        }
        __syncthreads();   // every lane has read gtile before the records overwrite it
    }
    float *r = recs + cl * RS;   // this cell's record row
    // the quad's parts share gu = m G' (hidden channels) through the record
    // row; the four lanes of a cell are in one wave, whose LDS accesses
    // complete in order
#pragma unroll
    for (int k = 0; k < CP; ++k) {
        const int c = part * CP + k;
        r[R::GU + c] = (c >= NIN && fire) ? gq[k] : 0.f;
    }
    __builtin_amdgcn_wave_barrier();
    float gu[C];
#pragma unroll
    for (int c = 0; c < C; ++c) gu[c] = r[R::GU + c];
    __builtin_amdgcn_wave_barrier();

    float gf[2 * C];
#pragma unroll
    for (int k = 0; k < 2 * C; ++k) gf[k] = 0.f;
#pragma unroll 2
    for (int jj = 0; jj < HP; ++jj) {
        const int j = jj * kParts + part;
        float a = sb1[j];
#pragma unroll
        for (int k = 0; k < 2 * C; ++k) a = fmaf(sw1[j][k], f[k], a);
        float gh = 0.f;
#pragma unroll
        for (int c = NIN; c < C; ++c) gh = fmaf(sw2[j][c], gu[c], gh);
        const float ga = a > 0.f ? gh : 0.f;
#pragma unroll
        for (int k = 0; k < 2 * C; ++k) gf[k] = fmaf(sw1[j][k], ga, gf[k]);
        r[R::Hh + j] = valid ? fmaxf(a, 0.f) : 0.f;   // a cell outside the grid adds 0
        r[R::GA + j] = valid ? ga : 0.f;
    }
    // sum of the quad's four partial W1^T ga (the same order in every lane)
#pragma unroll
    for (int k = 0; k < 2 * C; ++k) {
        gf[k] += __shfl_xor(gf[k], 1);
        gf[k] += __shfl_xor(gf[k], 2);
    }
#pragma unroll
    for (int k = 0; k < 2 * C; ++k)
        if (k / FP == part) r[R::F + k] = valid ? f[k] : 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
        if (c / CP == part) {
            r[R::GU + c] = valid ? gu[c] : 0.f;
            r[R::GP + c] = valid ? gf[C + c] : 0.f;
            if (valid) {
                gp[c * cells + idx] = gf[C + c];
                gpart[idx * C + c] = gq[c - part * CP] + gf[c];
            }
        }
    __syncthreads();
    // dconv_w needs S at the neighbours of cell p: tile word of p's centre
    // plus the tap's offset (zero outside the grid, as staged)
    wgrad_block<NDIM, C, H>(recs, [&](int p, int t, int c) {
        const int px = p % T::TX, py = (p / T::TX) % T::TY, pz = p / (T::TX * T::TY);
        const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
        const int nb = ((pz + (NDIM == 3 ? 1 : 0) + dz) * HY + py + 1 + dy) * HX + px + 1 + dx;
        return tile[c][nb];
    }, partial + (int64_t)blockIdx.x * WG<C, H, TAPS>::N, accumulate != 0);
}

// bwd_cell on the matrix cores, for C = 16, H = 64: the same results as
// bwd_cell (fp32 products, fp32 sums), with every contraction on
// v_mfma_f32_16x16x4_f32.  A wave takes 16 cells of the block's 64 (lane l:
// cell n = l % 16, lane group g = l / 16, which owns channel quad g), in the
// lane layout of the forward step kernels:
//   * features: the lane's 8 K slots are state channels 4g..4g+3 and
//     perception channels 4g..4g+3 of its cell; layer 1 recomputed as 4
//     hidden tiles x 8 K chunks, leaving a = W1 f + b1 of hidden unit
//     16 t + 4 g + i in register i of tile t;
//   * gh = W2^T gu: K chunk i holds channel 4 g + i in lane group g, which is
//     the lane's own G' value i, so 4 tiles x 4 chunks with A = W2 gathered;
//     gh lands in the layout of a, and ga = gh [a > 0] is elementwise;
//   * W1^T ga: K chunk (t, i) holds hidden unit 16 t + 4 g + i in lane group
//     g (the lane's own ga), 2 output tiles of 16 features x 16 chunks; tile
//     0 gives gS and tile 1 gP of channels 4g..4g+3: the lane's own quad, so
//     G' + gS and gP are stored without exchange;
//   * the block's outer-product sums dW1 = sum ga f^T and dW2 = sum gu h^T
//     take the cells as K: the cells' records [f | h | ga | gu | gP] go to
//     LDS, and each wave reads them back as MFMA operands (4 cells per K
//     chunk, 16 chunks per output tile; wave w takes dW1 tiles 2w, 2w+1 and
//     dW2 tile w); db1, dconv_b and dconv_w are summed on the VALU.
// Record rows are padded so that the 4 rows a wave reads at once start 16
// banks apart.
template <int NDIM, int NIN>
__global__ __launch_bounds__(kBwdThreads, 2) void bwd_cell_mfma(
    const float *__restrict__ src, const float *__restrict__ gout,
    const float *__restrict__ gp_prev, int dd, int dh, int dw, int tiles_x, int tiles_y,
    const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold,
    float *__restrict__ gpart, float *__restrict__ gp, float *__restrict__ partial,
    int64_t cells, int accumulate) {
    constexpr int C = 16, H = 64;
    using T = BwdCellTile<NDIM>;
    using G = WG<C, H, NDIM == 3 ? 27 : 9>;
    constexpr int HZ = NDIM == 3 ? T::TZ + 2 : 1, HY = T::TY + 2, HX = T::TX + 2;
    constexpr int NCELL = HZ * HY * HX;
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    constexpr int SF = 48, SH = 80, SQ = 16;   // record row strides (floats)
    static_assert(T::TZ * T::TY * T::TX == kWgCells, "64 cells per block");
    typedef float v4 __attribute__((ext_vector_type(4)));

    __shared__ float4 tile[4][NCELL];       // S, channel quads
    __shared__ float4 kw[TAPS][4];          // [tap][quad] conv weights of channels 4q..4q+3
    __shared__ float4 kb[4];                // conv bias of channel quad q
    // records: f [64][SF], h and ga [64][SH], gu and gP [64][SQ]; the gp_prev
    // tile (fused G') lives in the same space before the records are written
    __shared__ __align__(16) float recs[kWgCells * (SF + 2 * SH + 2 * SQ)];
    float *const rf = recs;
    float *const rh = rf + kWgCells * SF;
    float *const rga = rh + kWgCells * SH;
    float *const rgu = rga + kWgCells * SH;
    float *const rgp = rgu + kWgCells * SQ;
    float4 *const gtile = reinterpret_cast<float4 *>(recs);   // [4][NCELL]
    static_assert(4 * NCELL * 4 <= kWgCells * (SF + 2 * SH + 2 * SQ), "gp_prev tile fits");

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, g = lane >> 4;
    int b = blockIdx.x;
    const int bx = b % tiles_x;
    b /= tiles_x;
    const int by = b % tiles_y;
    const int bz = b / tiles_y;
    const int x0 = bx * T::TX, y0 = by * T::TY, z0 = bz * T::TZ;

    // The wave's 16 cells (one per lane n; lane group g owns channels
    // 4g..4g+3).  Their G' entries and fire bits do not depend on the tiles
    // below: the load is issued and the fire bit computed first, so both
    // overlap the tile loads instead of stalling the cell's chain later.
    const int cl = 16 * wave + n;
    const int tx = cl % T::TX, ty = (cl / T::TX) % T::TY, tz = cl / (T::TX * T::TY);
    const int x = x0 + tx, y = y0 + ty, z = z0 + tz;
    const bool valid = x < dw && y < dh && z < dd;
    const int64_t idx = ((int64_t)min(z, dd - 1) * dh + min(y, dh - 1)) * dw + min(x, dw - 1);
    const float4 go = *reinterpret_cast<const float4 *>(gout + idx * C + 4 * g);
    const bool fire = cell_fires(seed, level, step, batch, (uint64_t)idx, threshold);

    // S (and gp_prev) tiles with a one-cell halo, zero outside the grid
    auto halo_cell = [&](int cell, int64_t &gidx) {
        const int lx = cell % HX, ly = (cell / HX) % HY, lz = cell / (HX * HY);
        const int gx = x0 + lx - 1, gy = y0 + ly - 1, gz = NDIM == 3 ? z0 + lz - 1 : 0;
        gidx = ((int64_t)gz * dh + gy) * dw + gx;
        return gx >= 0 && gx < dw && gy >= 0 && gy < dh && gz >= 0 && gz < dd;
    };
    // Every thread loads its elements from clamped in-grid addresses and zeroes
    // the values outside afterwards, and all tile loads are issued before the
    // first LDS write: the tiles then cost one memory round trip (a load
    // behind the cell's condition became a branch and a wait per element).
    constexpr int LPT = (4 * NCELL + kBwdThreads - 1) / kBwdThreads;
    // v with every bit cleared where m is 0 (an exact +0 whatever v holds)
    auto masked = [](float4 v, uint32_t m) {
        return make_float4(__uint_as_float(__float_as_uint(v.x) & m),
                           __uint_as_float(__float_as_uint(v.y) & m),
                           __uint_as_float(__float_as_uint(v.z) & m),
                           __uint_as_float(__float_as_uint(v.w) & m));
    };
    float4 sv[LPT], gv[LPT];
    uint32_t s_m[LPT], g_m[LPT];
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
        const int i = min((int)threadIdx.x + j * kBwdThreads, 4 * NCELL - 1);
        const int q = i % 4, cell = i / 4;
        int64_t gi;
        const bool ok = halo_cell(cell, gi);
        s_m[j] = ok ? 0xffffffffu : 0u;
        sv[j] = *reinterpret_cast<const float4 *>(src + (ok ? gi : 0) * C + 4 * q);
    }
    if (gp_prev != nullptr) {
#pragma unroll
        for (int j = 0; j < LPT; ++j) {
            const int i = min((int)threadIdx.x + j * kBwdThreads, 4 * NCELL - 1);
            const int cell = i % NCELL, q = i / NCELL;
            int64_t gi;
            const bool ok = halo_cell(cell, gi);
            g_m[j] = ok ? 0xffffffffu : 0u;
            const int64_t gc = ok ? gi : 0;
            gv[j] = make_float4(gp_prev[(4 * q + 0) * cells + gc], gp_prev[(4 * q + 1) * cells + gc],
                                gp_prev[(4 * q + 2) * cells + gc], gp_prev[(4 * q + 3) * cells + gc]);
        }
    }
    // conv weights and bias for LDS (a tap's weights are one 16-byte read per
    // lane there, instead of four global reads inside the tap loops); thread
    // i < 4 TAPS holds [tap i / 4][quad i % 4], thread i < 4 the bias of quad
    // i, loaded from clamped indices by every thread
    static_assert(TAPS * 4 <= kBwdThreads, "one conv weight quad per thread");
    float4 kwv, kbv;
    {
        const int i = min((int)threadIdx.x, TAPS * 4 - 1);
        const int t = i / 4, q = i % 4;
        kwv = make_float4(conv_w[(4 * q + 0) * TAPS + t], conv_w[(4 * q + 1) * TAPS + t],
                          conv_w[(4 * q + 2) * TAPS + t], conv_w[(4 * q + 3) * TAPS + t]);
        const int qb = min((int)threadIdx.x, 3);
        kbv = make_float4(conv_b[4 * qb + 0], conv_b[4 * qb + 1], conv_b[4 * qb + 2],
                          conv_b[4 * qb + 3]);
    }
    // weights in the lane's operand layouts
    float w1a[4][8];    // [t][kc] = W1[16t + n][feature(kc, g)]
    float w1t[2][4][4]; // [ft][t][i] = W1[16t + 4g + i][16 ft + n]
    float w2t[4][4];    // [t][i] = W2[4g + i][16t + n] (0 for input channels)
    v4 bias[4];         // [t][i] = b1[16t + 4g + i]
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int kc = 0; kc < 8; ++kc)
            w1a[t][kc] = w1[(16 * t + n) * 2 * C + (kc < 4 ? 4 * g + kc : C + 4 * g + kc - 4)];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            w1t[0][t][i] = w1[(16 * t + 4 * g + i) * 2 * C + n];
            w1t[1][t][i] = w1[(16 * t + 4 * g + i) * 2 * C + C + n];
            const float v2 = w2[(4 * g + i) * H + 16 * t + n];   // loaded for every row
            w2t[t][i] = 4 * g + i < NIN ? 0.f : v2;
            bias[t][i] = b1[16 * t + 4 * g + i];
        }
    }
    // LDS writes, after every load of the block's set-up has been issued
    if (threadIdx.x < TAPS * 4) kw[threadIdx.x / 4][threadIdx.x % 4] = kwv;
    if (threadIdx.x < 4) kb[threadIdx.x] = kbv;
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
        const int i = (int)threadIdx.x + j * kBwdThreads;
        if (i < 4 * NCELL) tile[i % 4][i / 4] = masked(sv[j], s_m[j]);
    }
    if (gp_prev != nullptr) {
#pragma unroll
        for (int j = 0; j < LPT; ++j) {
            const int i = (int)threadIdx.x + j * kBwdThreads;
            if (i < 4 * NCELL) gtile[i] = masked(gv[j], g_m[j]);
        }
    }
    __syncthreads();

    // ---- the wave's 16 cells ----
    const int centre = ((tz + (NDIM == 3 ? 1 : 0)) * HY + ty + 1) * HX + tx + 1;

    const float4 sq = tile[g][centre];
    float f[8] = {sq.x, sq.y, sq.z, sq.w};
    {
        const float4 cb = kb[g];
        float pc[4] = {cb.x, cb.y, cb.z, cb.w};
#pragma unroll
        for (int t = 0; t < TAPS; ++t) {
            const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
            const float4 v = tile[g][centre + (dz * HY + dy) * HX + dx];
            const float4 w = kw[t][g];
            pc[0] = fmaf(w.x, v.x, pc[0]);
            pc[1] = fmaf(w.y, v.y, pc[1]);
            pc[2] = fmaf(w.z, v.z, pc[2]);
            pc[3] = fmaf(w.w, v.w, pc[3]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) f[4 + i] = pc[i];
    }
    // layer 1, recomputed
    v4 a[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = bias[t];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc)
#pragma unroll
        for (int t = 0; t < 4; ++t)
            a[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1a[t][kc], f[kc], a[t], 0, 0, 0);
    // G' of channels 4g..4g+3 of the cell
    float gq[4] = {go.x, go.y, go.z, go.w};
    if (gp_prev != nullptr) {
        // cell p receives K[c][t] gP[p - o_t] from each tap t
#pragma unroll
        for (int t = 0; t < TAPS; ++t) {
            const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
            const float4 v = gtile[g * NCELL + centre - (dz * HY + dy) * HX - dx];
            const float4 w = kw[t][g];
            gq[0] = fmaf(w.x, v.x, gq[0]);
            gq[1] = fmaf(w.y, v.y, gq[1]);
            gq[2] = fmaf(w.z, v.z, gq[2]);
            gq[3] = fmaf(w.w, v.w, gq[3]);
        }
    }
    float gu[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) gu[i] = (4 * g + i >= NIN && fire) ? gq[i] : 0.f;
    // gh = W2^T gu, ga = gh [a > 0]
    v4 ga[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        ga[t] = v4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i)
            ga[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(w2t[t][i], gu[i], ga[t], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) ga[t][i] = a[t][i] > 0.f ? ga[t][i] : 0.f;
    // [gS, gP] = W1^T ga
    v4 gsp[2];
#pragma unroll
    for (int ft = 0; ft < 2; ++ft) {
        gsp[ft] = v4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                gsp[ft] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1t[ft][t][i], ga[t][i], gsp[ft], 0, 0, 0);
    }
    if (valid) {
        *reinterpret_cast<float4 *>(gpart + idx * C + 4 * g) =
            make_float4(gq[0] + gsp[0][0], gq[1] + gsp[0][1], gq[2] + gsp[0][2], gq[3] + gsp[0][3]);
#pragma unroll
        for (int i = 0; i < 4; ++i) gp[(4 * g + i) * cells + idx] = gsp[1][i];
    }
    if (gp_prev != nullptr) __syncthreads();   // every lane has read gtile
    // records (zero for cells outside the grid: they add nothing to the sums)
    const float vm = valid ? 1.f : 0.f;
    *reinterpret_cast<float4 *>(rf + cl * SF + 4 * g) =
        make_float4(vm * f[0], vm * f[1], vm * f[2], vm * f[3]);
    *reinterpret_cast<float4 *>(rf + cl * SF + C + 4 * g) =
        make_float4(vm * f[4], vm * f[5], vm * f[6], vm * f[7]);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        *reinterpret_cast<float4 *>(rh + cl * SH + 16 * t + 4 * g) =
            make_float4(vm * fmaxf(a[t][0], 0.f), vm * fmaxf(a[t][1], 0.f), vm * fmaxf(a[t][2], 0.f),
                        vm * fmaxf(a[t][3], 0.f));
        *reinterpret_cast<float4 *>(rga + cl * SH + 16 * t + 4 * g) =
            make_float4(vm * ga[t][0], vm * ga[t][1], vm * ga[t][2], vm * ga[t][3]);
    }
    *reinterpret_cast<float4 *>(rgu + cl * SQ + 4 * g) =
        make_float4(vm * gu[0], vm * gu[1], vm * gu[2], vm * gu[3]);
    *reinterpret_cast<float4 *>(rgp + cl * SQ + 4 * g) =
        make_float4(vm * gsp[1][0], vm * gsp[1][1], vm * gsp[1][2], vm * gsp[1][3]);
    __syncthreads();

    // ---- the block's weight-gradient sums ----
    float *out = partial + (int64_t)blockIdx.x * G::N;
    auto start = [&](int o) { return accumulate ? out[o] : 0.f; };
    // dW1 tiles (t, ft) = (wave, 0), (wave, 1): D[i][j] = sum_cells ga[16t + i] f[16ft + j]
#pragma unroll
    for (int ft = 0; ft < 2; ++ft) {
        const int t = wave;
        // two interleaved chains (even and odd K chunks), added at the end
        v4 acc, acc2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = start(G::W1 + (16 * t + 4 * g + i) * 2 * C + 16 * ft + n);
#pragma unroll 4
        for (int k4 = 0; k4 < kWgCells / 4; k4 += 2) {
            const int c = 4 * k4 + g;
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(rga[c * SH + 16 * t + n], rf[c * SF + 16 * ft + n],
                                                       acc, 0, 0, 0);
            acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(rga[(c + 4) * SH + 16 * t + n],
                                                        rf[(c + 4) * SF + 16 * ft + n], acc2, 0, 0, 0);
        }
        acc += acc2;
#pragma unroll
        for (int i = 0; i < 4; ++i) out[G::W1 + (16 * t + 4 * g + i) * 2 * C + 16 * ft + n] = acc[i];
    }
    // dW2 tile t = wave: D[c][j] = sum_cells gu[c] h[16t + j]
    {
        const int t = wave;
        v4 acc, acc2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = start(G::W2 + (4 * g + i) * H + 16 * t + n);
#pragma unroll 4
        for (int k4 = 0; k4 < kWgCells / 4; k4 += 2) {
            const int c = 4 * k4 + g;
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(rgu[c * SQ + n], rh[c * SH + 16 * t + n], acc,
                                                       0, 0, 0);
            acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(rgu[(c + 4) * SQ + n],
                                                        rh[(c + 4) * SH + 16 * t + n], acc2, 0, 0, 0);
        }
        acc += acc2;
#pragma unroll
        for (int i = 0; i < 4; ++i) out[G::W2 + (4 * g + i) * H + 16 * t + n] = acc[i];
    }
    // db1, dconv_b (a quad of entries per job) and dconv_w (a channel quad of
    // one tap): four consecutive lanes per job, each summing a quarter of the
    // cells, then the quarters added across the four lanes
    constexpr int JB = H / 4, JC = C / 4, JK = (C / 4) * TAPS;
    constexpr int NJ = JB + JC + JK;
    constexpr int QC = kWgCells / 4;
    for (int base = 0; base < 4 * NJ; base += kBwdThreads) {
        const int slot = base + (int)threadIdx.x;
        const int job = min(slot / 4, NJ - 1), qtr = slot % 4;
        float sum[4] = {0.f, 0.f, 0.f, 0.f};
        int o[4];
        if (job < JB + JC) {
            const bool isb = job < JB;
            const float *src4 = isb ? rga + 4 * job : rgp + 4 * (job - JB);
            const int stride = isb ? SH : SQ;
            const int o0 = isb ? G::B1 + 4 * job : G::CB + 4 * (job - JB);
#pragma unroll
            for (int r = 0; r < 4; ++r) o[r] = o0 + r;
            for (int c = qtr * QC; c < (qtr + 1) * QC; ++c) {
                const float4 v = *reinterpret_cast<const float4 *>(src4 + c * stride);
                sum[0] += v.x; sum[1] += v.y; sum[2] += v.z; sum[3] += v.w;
            }
        } else {
            const int jj = job - JB - JC;
            const int cq = jj / TAPS, t = jj % TAPS;
            const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
#pragma unroll
            for (int r = 0; r < 4; ++r) o[r] = G::CW + (4 * cq + r) * TAPS + t;
#pragma unroll 4
            for (int c = qtr * QC; c < (qtr + 1) * QC; ++c) {
                const int px = c % T::TX, py = (c / T::TX) % T::TY, pz = c / (T::TX * T::TY);
                const int nb = ((pz + (NDIM == 3 ? 1 : 0) + dz) * HY + py + 1 + dy) * HX + px + 1 + dx;
                const float4 gpv = *reinterpret_cast<const float4 *>(rgp + c * SQ + 4 * cq);
                const float4 sv = tile[cq][nb];
                sum[0] = fmaf(gpv.x, sv.x, sum[0]);
                sum[1] = fmaf(gpv.y, sv.y, sum[1]);
                sum[2] = fmaf(gpv.z, sv.z, sum[2]);
                sum[3] = fmaf(gpv.w, sv.w, sum[3]);
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            sum[r] += __shfl_xor(sum[r], 1);
            sum[r] += __shfl_xor(sum[r], 2);
        }
        if (qtr == 0 && slot / 4 < NJ)
#pragma unroll
            for (int r = 0; r < 4; ++r) out[o[r]] = start(o[r]) + sum[r];
    }
}

template <int NDIM, int C, int H>
__global__ __launch_bounds__(kBwdThreads) void bwd_conv_t(
    const float *__restrict__ gpart, const float *__restrict__ gp, int dd, int dh, int dw,
    int tiles_x, int tiles_y, const float *__restrict__ conv_w, float *__restrict__ gin,
    int64_t cells) {
    using T = BwdTile<NDIM>;
    constexpr int HZ = NDIM == 3 ? T::TZ + 2 : 1, HY = T::TY + 2, HX = T::TX + 2;
    constexpr int NCELL = HZ * HY * HX;
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    __shared__ float tile[C][NCELL];   // gP of the tile and its halo

    int b = blockIdx.x;
    const int bx = b % tiles_x;
    b /= tiles_x;
    const int by = b % tiles_y;
    const int bz = b / tiles_y;
    const int x0 = bx * T::TX, y0 = by * T::TY, z0 = bz * T::TZ;
    stage<NCELL * C, 8>(
        [&](int i) {
            const int c = i / NCELL, cell = i % NCELL;
            const int lx = cell % HX, ly = (cell / HX) % HY, lz = cell / (HX * HY);
            const int gx = x0 + lx - 1, gy = y0 + ly - 1, gz = NDIM == 3 ? z0 + lz - 1 : 0;
            const bool in = gx >= 0 && gx < dw && gy >= 0 && gy < dh && gz >= 0 && gz < dd;
            const int cx = min(max(gx, 0), dw - 1), cy = min(max(gy, 0), dh - 1),
                      cz = min(max(gz, 0), dd - 1);
            const float v = gp[c * cells + ((int64_t)cz * dh + cy) * dw + cx];
            return in ? v : 0.f;
        },
        [&](int i, float v) { tile[i / NCELL][i % NCELL] = v; });
    __syncthreads();

    const int tx = threadIdx.x % T::TX, ty = (threadIdx.x / T::TX) % T::TY,
              tz = threadIdx.x / (T::TX * T::TY);
    const int x = x0 + tx, y = y0 + ty, z = z0 + tz;
    if (x >= dw || y >= dh || z >= dd) return;
    const int centre = ((tz + (NDIM == 3 ? 1 : 0)) * HY + ty + 1) * HX + tx + 1;
    const int64_t idx = ((int64_t)z * dh + y) * dw + x;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        float v = gpart[idx * C + c];
#pragma unroll
        for (int t = 0; t < TAPS; ++t) {
            // cell q receives K[c][t] gP[q - o_t]
            const int dz = NDIM == 3 ? t / 9 - 1 : 0, dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
            v = fmaf(conv_w[c * TAPS + t], tile[c][centre - (dz * HY + dy) * HX - dx], v);
        }
        gin[idx * C + c] = v;
    }
}

// grads += the sum of the block partial sums of each entry.  A block of
// kRedWaves waves takes 64 consecutive entries; wave w sums block rows w,
// w + kRedWaves, ... in order in fp64 (lane = entry, so each row read is one
// coalesced 256-byte segment), and the waves' sums are added in wave order
// (deterministic).
constexpr int kRedWaves = 16;
template <int C, int H, int TAPS>
__global__ __launch_bounds__(64 * kRedWaves) void wgrad_reduce(const float *__restrict__ partial,
                                                               int64_t blocks, LevelGradsDev g,
                                                               int overwrite) {
    using G = WG<C, H, TAPS>;
    __shared__ double red[kRedWaves][64];
    const int lane = threadIdx.x & 63, w = (int)(threadIdx.x >> 6);
    const int o = blockIdx.x * 64 + lane;
    const int oc = min(o, G::N - 1);
    double s = 0.0;
#pragma unroll 8
    for (int64_t b = w; b < blocks; b += kRedWaves) s += (double)partial[b * G::N + oc];
    red[w][lane] = s;
    __syncthreads();
    if (w != 0 || o >= G::N) return;
    double t = red[0][lane];
#pragma unroll
    for (int k = 1; k < kRedWaves; ++k) t += red[k][lane];
    float *dst;
    if (o < G::W2) dst = g.w1 + o;
    else if (o < G::B1) dst = g.w2 + (o - G::W2);
    else if (o < G::CB) dst = g.b1 + (o - G::B1);
    else if (o < G::CW) dst = g.conv_b + (o - G::CB);
    else dst = g.conv_w + (o - G::CW);
    *dst = overwrite ? (float)t : (float)((double)*dst + t);
}

// Block counts of the two backward tilings of a level.
template <int NDIM>
struct BwdGrid {
    int tiles_x, tiles_y, ctiles_x, ctiles_y;
    int64_t blocks, cblocks;
    explicit BwdGrid(const Extent3 &e) {
        using T = BwdTile<NDIM>;
        using TC = BwdCellTile<NDIM>;
        tiles_x = (int)((e.w + T::TX - 1) / T::TX);
        tiles_y = (int)((e.h + T::TY - 1) / T::TY);
        blocks = (int64_t)tiles_x * tiles_y * ((e.d + T::TZ - 1) / T::TZ);
        ctiles_x = (int)((e.w + TC::TX - 1) / TC::TX);
        ctiles_y = (int)((e.h + TC::TY - 1) / TC::TY);
        cblocks = (int64_t)ctiles_x * ctiles_y * ((e.d + TC::TZ - 1) / TC::TZ);
    }
};

template <int NDIM, int NIN, int C, int H>
void enqueue_bwd_cell(const StepArgs &a, const BwdGrid<NDIM> &gr, const float *src,
                      const float *gout, const float *gp_prev, float *gpart, float *gp,
                      float *partial, bool accumulate, hipStream_t stream) {
    if constexpr (C == 16 && H == 64) {
        bwd_cell_mfma<NDIM, NIN><<<(unsigned)gr.cblocks, kBwdThreads, 0, stream>>>(
            src, gout, gp_prev, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, gr.ctiles_x,
            gr.ctiles_y, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch,
            a.seed, a.threshold, gpart, gp, partial, a.ext.cells(), accumulate ? 1 : 0);
        return;
    }
    bwd_cell<NDIM, NIN, C, H><<<(unsigned)gr.cblocks, kBwdThreads, 0, stream>>>(
        src, gout, gp_prev, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, gr.ctiles_x, gr.ctiles_y,
        a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch, a.seed,
        a.threshold, gpart, gp, partial, a.ext.cells(), accumulate ? 1 : 0);
}

template <int NDIM, int C, int H>
void enqueue_tail(const StepArgs &a, const BwdGrid<NDIM> &gr, const float *gpart, const float *gp,
                  float *gin, const float *partial, LevelGradsDev g, bool overwrite,
                  hipStream_t stream) {
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    bwd_conv_t<NDIM, C, H><<<(unsigned)gr.blocks, kBwdThreads, 0, stream>>>(
        gpart, gp, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, gr.tiles_x, gr.tiles_y, a.w.conv_w,
        gin, a.ext.cells());
    wgrad_reduce<C, H, TAPS><<<(WG<C, H, TAPS>::N + 63) / 64, 64 * kRedWaves, 0, stream>>>(
        partial, gr.cblocks, g, overwrite ? 1 : 0);
}

// One step: bwd_cell, bwd_conv_t, wgrad_reduce.
template <int NDIM, int NIN, int C, int H>
hipError_t launch_bwd(const StepArgs &a, const float *src, const float *gout, float *gin,
                      LevelGradsDev g, float *ws, hipStream_t stream) {
    const int64_t cells = a.ext.cells();
    if (cells == 0) return hipSuccess;
    const BwdGrid<NDIM> gr(a.ext);
    float *gpart = ws;                 // G' + gS
    float *gp = gpart + cells * C;     // gP, [C][cells]
    float *partial = gp + cells * C;   // [cblocks][entries]
    enqueue_bwd_cell<NDIM, NIN, C, H>(a, gr, src, gout, nullptr, gpart, gp, partial, false,
                                      stream);
    enqueue_tail<NDIM, C, H>(a, gr, gpart, gp, gin, partial, g, false, stream);
    return hipGetLastError();
}

// All steps of a level, last step first: each bwd_cell after the first takes
// G' from the previous one's (G' + gS, gP) with the transposed convolution
// fused, the weight-gradient sums accumulate in the blocks' partial rows, and
// one bwd_conv_t and one wgrad_reduce finish the level.
template <int NDIM, int NIN, int C, int H>
hipError_t launch_bwd_level(const StepArgs &a0, int32_t steps, const float *states,
                            const float *gout, float *gin, LevelGradsDev g, float *ws,
                            hipStream_t stream) {
    const int64_t cells = a0.ext.cells();
    if (cells == 0 || steps <= 0) return hipSuccess;
    const BwdGrid<NDIM> gr(a0.ext);
    float *gpart[2] = {ws, ws + cells * C};
    float *gp[2] = {ws + 2 * cells * C, ws + 3 * cells * C};
    float *partial = ws + 4 * cells * C;
    StepArgs a = a0;
    int cur = 0;
    for (int32_t t = steps - 1; t >= 0; --t) {
        a.step = (uint32_t)t;
        const bool first = t == steps - 1;
        enqueue_bwd_cell<NDIM, NIN, C, H>(a, gr, states + (size_t)t * cells * C,
                                          first ? gout : gpart[cur ^ 1],
                                          first ? nullptr : gp[cur ^ 1], gpart[cur], gp[cur],
                                          partial, !first, stream);
        cur ^= 1;
    }
    enqueue_tail<NDIM, C, H>(a, gr, gpart[cur ^ 1], gp[cur ^ 1], gin, partial, g, true, stream);
    return hipGetLastError();
}

template <int NDIM, int C, int H>
hipError_t bwd_nin(const StepArgs &a, const float *src, const float *gout, float *gin,
                   LevelGradsDev g, float *ws, hipStream_t stream, int32_t level_steps) {
    if (level_steps >= 0) {
        if (a.n_in == 1)
            return launch_bwd_level<NDIM, 1, C, H>(a, level_steps, src, gout, gin, g, ws, stream);
        if (a.n_in == 3)
            return launch_bwd_level<NDIM, 3, C, H>(a, level_steps, src, gout, gin, g, ws, stream);
        return hipErrorInvalidValue;
    }
    if (a.n_in == 1) return launch_bwd<NDIM, 1, C, H>(a, src, gout, gin, g, ws, stream);
    if (a.n_in == 3) return launch_bwd<NDIM, 3, C, H>(a, src, gout, gin, g, ws, stream);
    return hipErrorInvalidValue;
}

template <int NDIM>
hipError_t bwd_size(const StepArgs &a, const float *src, const float *gout, float *gin,
                    LevelGradsDev g, float *ws, hipStream_t stream, int32_t level_steps) {
    if (a.channels == 16 && a.hidden == 64)
        return bwd_nin<NDIM, 16, 64>(a, src, gout, gin, g, ws, stream, level_steps);
    if (a.channels == 12 && a.hidden == 48)
        return bwd_nin<NDIM, 12, 48>(a, src, gout, gin, g, ws, stream, level_steps);
    if (a.channels == 20 && a.hidden == 100)
        return bwd_nin<NDIM, 20, 100>(a, src, gout, gin, g, ws, stream, level_steps);
    return hipErrorInvalidValue;
}

// Adjoint of the upsample + inject: one thread per coarse cell and channel.
__global__ __launch_bounds__(256) void upsample_adjoint(const float *__restrict__ gfine,
                                                        Extent3 cext, int fz, int fy, int fx,
                                                        int n_in, int channels,
                                                        float *__restrict__ gcoarse) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t total = cext.d * cext.h * cext.w * channels;
    if (i >= total) return;
    const int c = (int)(i % channels);
    const int64_t q = i / channels;
    const int64_t cx = q % cext.w, cy = (q / cext.w) % cext.h, cz = q / (cext.w * cext.h);
    const int64_t fh = cext.h * fy, fw = cext.w * fx;
    double s = 0.0;
    if (c >= n_in)
        for (int a = 0; a < fz; ++a)
            for (int b = 0; b < fy; ++b)
                for (int d = 0; d < fx; ++d)
                    s += gfine[(((cz * fz + a) * fh + cy * fy + b) * fw + cx * fx + d) * channels + c];
    gcoarse[i] = (float)s;
}

// Readout MSE: grad (all channels, zero but the last two) and per-block loss
// partials (fp64); then loss = their sum in block order.
__global__ __launch_bounds__(256) void mse_grad(const float *__restrict__ state,
                                                const float *__restrict__ target, int64_t cells,
                                                int channels, float *__restrict__ grad,
                                                double *__restrict__ block_loss) {
    __shared__ double part[256];
    const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
    double l = 0.0;
    if (p < cells) {
        for (int c = 0; c < channels - 2; ++c) grad[p * channels + c] = 0.f;
        for (int k = 0; k < 2; ++k) {
            // the difference of two fp32 values is exact in fp64; the gradient
            // is its correctly rounded fp32 value
            const double d = (double)state[p * channels + channels - 2 + k] - (double)target[p * 2 + k];
            grad[p * channels + channels - 2 + k] = (float)d;
            l += 0.5 * d * d;
        }
    }
    part[threadIdx.x] = l;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) block_loss[blockIdx.x] = part[0];
}

// Sum of the block partials in a fixed order (thread t sums partials t,
// t + 256, ...; then a tree over the threads), so the loss is deterministic.
__global__ __launch_bounds__(256) void sum_losses(const double *__restrict__ block_loss,
                                                  int64_t blocks, double *__restrict__ loss) {
    __shared__ double part[256];
    double s = 0.0;
    for (int64_t b = threadIdx.x; b < blocks; b += 256) s += block_loss[b];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int k = 128; k > 0; k >>= 1) {
        if ((int)threadIdx.x < k) part[threadIdx.x] += part[threadIdx.x + k];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = part[0];
}

__global__ __launch_bounds__(256) void fill_zero(float *__restrict__ p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

}  // namespace

size_t step_backward_workspace_floats(int ndim, int channels, int hidden, Extent3 e) {
    const int taps = ndim == 3 ? 27 : 9;
    const int64_t cells = e.cells();
    const int64_t wg_n = 3 * channels * hidden + hidden + channels + channels * taps;
    // bwd_cell blocks: 2 x 32 cells (2D), 2 x 4 x 8 (3D)
    const int64_t tz = ndim == 3 ? 2 : 1, ty = ndim == 3 ? 4 : 2, tx = ndim == 3 ? 8 : 32;
    const int64_t cblocks =
        ((e.d + tz - 1) / tz) * ((e.h + ty - 1) / ty) * ((e.w + tx - 1) / tx);
    return (size_t)(2 * cells * channels + cblocks * wg_n);
}

size_t level_backward_workspace_floats(int ndim, int channels, int hidden, Extent3 e) {
    // two more cell-sized buffers than one step: (G' + gS, gP) of the step
    // read and of the step written
    return step_backward_workspace_floats(ndim, channels, hidden, e) +
           (size_t)(2 * e.cells() * channels);
}

hipError_t launch_step_backward(const StepArgs &a, const float *src, const float *gout,
                                float *gin, LevelGradsDev g, float *ws, hipStream_t stream) {
    return a.ndim == 2 ? bwd_size<2>(a, src, gout, gin, g, ws, stream, -1)
                       : bwd_size<3>(a, src, gout, gin, g, ws, stream, -1);
}

hipError_t launch_level_backward(const StepArgs &a, int32_t steps, const float *states,
                                 const float *gout, float *gin, LevelGradsDev g, float *ws,
                                 hipStream_t stream) {
    if (steps <= 0) return hipSuccess;
    return a.ndim == 2 ? bwd_size<2>(a, states, gout, gin, g, ws, stream, steps)
                       : bwd_size<3>(a, states, gout, gin, g, ws, stream, steps);
}

hipError_t launch_upsample_adjoint(const float *gfine, Extent3 coarse, int fz, int fy, int fx,
                                   int n_in, int channels, float *gcoarse, hipStream_t stream) {
    const int64_t total = coarse.cells() * channels;
    if (total == 0) return hipSuccess;
    upsample_adjoint<<<(unsigned)((total + 255) / 256), 256, 0, stream>>>(
        gfine, coarse, fz, fy, fx, n_in, channels, gcoarse);
    return hipGetLastError();
}

size_t mse_workspace_doubles(int64_t cells) { return (size_t)((cells + 255) / 256); }

hipError_t launch_readout_mse(const float *state, const float *target, int64_t cells, int channels,
                              float *grad, double *loss, double *ws, hipStream_t stream) {
    const int64_t blocks = (cells + 255) / 256;
    if (blocks > 0)
        mse_grad<<<(unsigned)blocks, 256, 0, stream>>>(state, target, cells, channels, grad, ws);
    sum_losses<<<1, 256, 0, stream>>>(ws, blocks, loss);
    return hipGetLastError();
}

hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    fill_zero<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(p, n);
    return hipGetLastError();
}

}  // namespace octnca
