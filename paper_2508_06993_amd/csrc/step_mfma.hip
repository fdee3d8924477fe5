// Fused NCA step on the matrix cores (Sec. 3.1; supplement S3, Listing 1).
//
// The per-cell MLP 2C -> H -> C is a dense contraction over a batch of
// cells, so it runs on MFMA; perception, ReLU, the fire gate and the
// residual stay on the VALU.
//
// Lane mapping (wave64, one "group" = 16 cells handled by one MFMA chain):
//   lane l -> cell n = l % 16 of the group, channel quad g = l / 16, i.e. the
//   lane owns channels 4g .. 4g+3 of its cell.
//   * it computes the perception of those 4 channels (depthwise taps read
//     from an LDS tile with a one-cell halo, zero padding outside the grid);
//   * layer 1, H[j][n] = b1[j] + sum_k W1[j][k] F[n][k], runs as
//     v_mfma_f32_16x16x4_f32 with A = W1 tile (16 hidden units x 4
//     features), B = features (4 x 16 cells).  The B operand of lane l is
//     feature row k = l / 16 of its cell, so feature chunk kc is taken as
//     state channel 4g + kc (kc < 4) or perception channel 4g + kc - 4;
//     W1's columns are gathered in the same order.  4 hidden tiles x 8
//     feature chunks = 32 MFMAs per group;
//   * the accumulator of hidden tile jt leaves hidden unit jt*16 + 4g + i of
//     cell n in register i of lane l, which is exactly the B operand layout
//     of the second layer with K index g; so after ReLU the registers feed
//     layer 2 (U[c][n] = sum_j W2[c][j] H[j][n]) directly, 16 MFMAs, with
//     W2's columns gathered to match.  No hidden value leaves the registers;
//   * layer 2's accumulator holds channels 4g .. 4g+3 of cell n in lane l:
//     the channels whose state the lane already holds, so the residual
//     update and the 16-byte store need no data exchange.
// Fire bits: each wave evaluates Philox4x64-10 once per lane for up to 64
// quads of cells (the rows it owns), spreads the bits with four ballots and
// every lane picks its cell's bit.
//
// 2D: a persistent grid loops over 16 x 32 tiles; the 18 x 34 halo tile is
// staged in LDS as fp32 in four channel-quad planes (conflict-free 16-byte
// reads).  3D: a block owns an 8 x 32 column of the (y, x) plane and a run
// of z planes, keeping three halo planes in an LDS ring (each plane is read
// from HBM once per run).
#include <algorithm>

#include "launch.h"

namespace octnca {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v8f __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;   // 4 waves

// Feature order seen by lane (g, n): slot s < 4 is state channel 4g + s,
// slot s >= 4 is perception channel 4g + s - 4.
__device__ __forceinline__ int feature_of(int slot, int g) {
    return slot < 4 ? 4 * g + slot : kC + 4 * g + (slot - 4);
}

// ---------------------------------------------------------------------------
// MLP policies.  Each gathers its weights into lane registers once per block
// (load) and computes the update of channels 4g..4g+3 of the lane's cell from
// its 8 features (update).  All accumulate in fp32.
// ---------------------------------------------------------------------------

// fp32 operands: v_mfma_f32_16x16x4_f32, 32 + 16 MFMAs per 16 cells.
struct MlpF32 {
    float w1[4][8];   // [jt][kc] = W1[jt*16 + n][feature(kc, g)]
    v4f b1[4];        // [jt][i]  = b1[jt*16 + 4g + i]
    float w2[4][4];   // [jt][i]  = W2[n][jt*16 + 4g + i]   (n = output channel)

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g) {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
            for (int kc = 0; kc < 8; ++kc) w1[jt][kc] = W1[(jt * 16 + n) * 2 * kC + feature_of(kc, g)];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                b1[jt][i] = B1[jt * 16 + 4 * g + i];
                w2[jt][i] = W2[n * kH + jt * 16 + 4 * g + i];
            }
        }
    }

    __device__ __forceinline__ v4f update(const float f[8]) const {
        v4f acc[4];
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[jt][0], f[0], b1[jt], 0, 0, 0);
#pragma unroll
        for (int kc = 1; kc < 8; ++kc)
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
                acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[jt][kc], f[kc], acc[jt], 0, 0, 0);
        v4f u0 = {0.f, 0.f, 0.f, 0.f}, u1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float h = fmaxf(acc[jt][i], 0.f);
                if ((jt * 4 + i) & 1)
                    u1 = __builtin_amdgcn_mfma_f32_16x16x4f32(w2[jt][i], h, u1, 0, 0, 0);
                else
                    u0 = __builtin_amdgcn_mfma_f32_16x16x4f32(w2[jt][i], h, u0, 0, 0, 0);
            }
        return u0 + u1;
    }
};

// Split-precision bf16: every fp32 operand x is written as hi + lo with
// hi = bf16(x), lo = bf16(x - hi); a product a*b is taken as
// hi_a*hi_b + hi_a*lo_b + lo_a*hi_b (the dropped lo*lo term is below 2^-16
// relative), on v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  The K = 32
// operand of a lane is 8 consecutive K slots, so one MFMA covers all 32
// features of layer 1 and two cover the 64 hidden units of layer 2:
// 12 + 6 MFMAs per 16 cells.  A and B use the same (lane group, slot) -> K
// correspondence, so the feature / hidden order only has to agree between
// the weights gathered here and the activations.
__device__ __forceinline__ void split_bf16(const v8f &x, v8bf &hi, v8bf &lo) {
    hi = __builtin_convertvector(x, v8bf);
    const v8f back = __builtin_convertvector(hi, v8f);
    lo = __builtin_convertvector(x - back, v8bf);
}

struct MlpBf16x3 {
    v8bf w1h[4], w1l[4];   // [jt] slot s: W1[jt*16 + n][feature(s, g)]
    v4f b1[4];
    v8bf w2h[2], w2l[2];   // [p] slot s: W2[n][hidden(p, s, g)]

    // hidden unit in K slot s of layer-2 MFMA p for lane group g: it is the
    // layer-1 accumulator register (jt = 2p + s/4, i = s%4) of the lane.
    __device__ static __forceinline__ int hidden_of(int p, int s, int g) {
        return (2 * p + s / 4) * 16 + 4 * g + (s % 4);
    }

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g) {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = W1[(jt * 16 + n) * 2 * kC + feature_of(s, g)];
            split_bf16(x, w1h[jt], w1l[jt]);
#pragma unroll
            for (int i = 0; i < 4; ++i) b1[jt][i] = B1[jt * 16 + 4 * g + i];
        }
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = W2[n * kH + hidden_of(p, s, g)];
            split_bf16(x, w2h[p], w2l[p]);
        }
    }

    __device__ __forceinline__ v4f update(const float f[8]) const {
        v8f fx;
#pragma unroll
        for (int s = 0; s < 8; ++s) fx[s] = f[s];
        v8bf fh, fl;
        split_bf16(fx, fh, fl);
        v4f acc[4];
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1l[jt], fh, b1[jt], 0, 0, 0);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1h[jt], fl, acc[jt], 0, 0, 0);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1h[jt], fh, acc[jt], 0, 0, 0);
        v8bf hh[2], hl[2];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = fmaxf(acc[2 * p + s / 4][s % 4], 0.f);
            split_bf16(x, hh[p], hl[p]);
        }
        v4f u[2];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            u[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w2l[p], hh[p], v4f{0.f, 0.f, 0.f, 0.f},
                                                           0, 0, 0);
            u[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w2h[p], hl[p], u[p], 0, 0, 0);
        }
#pragma unroll
        for (int p = 0; p < 2; ++p)
            u[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w2h[p], hh[p], u[p], 0, 0, 0);
        return u[0] + u[1];
    }
};

// fp16 operands, single pass (for fp16 state storage): weights, features and
// hidden activations rounded to fp16, products accumulated in fp32 on
// v_mfma_f32_16x16x32_f16; 4 + 2 MFMAs per 16 cells.
struct MlpF16 {
    v8h w1[4];
    v4f b1[4];
    v8h w2[2];

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g) {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = W1[(jt * 16 + n) * 2 * kC + feature_of(s, g)];
            w1[jt] = __builtin_convertvector(x, v8h);
#pragma unroll
            for (int i = 0; i < 4; ++i) b1[jt][i] = B1[jt * 16 + 4 * g + i];
        }
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = W2[n * kH + MlpBf16x3::hidden_of(p, s, g)];
            w2[p] = __builtin_convertvector(x, v8h);
        }
    }

    __device__ __forceinline__ v4f update(const float f[8]) const {
        v8f fx;
#pragma unroll
        for (int s = 0; s < 8; ++s) fx[s] = f[s];
        const v8h fh = __builtin_convertvector(fx, v8h);
        v4f acc[4];
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(w1[jt], fh, b1[jt], 0, 0, 0);
        v4f u = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = fmaxf(acc[2 * p + s / 4][s % 4], 0.f);
            u = __builtin_amdgcn_mfma_f32_16x16x32_f16(w2[p], __builtin_convertvector(x, v8h), u,
                                                       0, 0, 0);
        }
        return u;
    }
};

// Fire bits for the quads of up to four rows of cells (16 quads per row).
// Lane L evaluates quad q0[L / 16] + L % 16; bit (word k, quad offset o of
// row r) is bit 16 r + o of ballot k.
struct FireBallots {
    uint64_t w[4];
};

__device__ __forceinline__ FireBallots fire_ballots(uint64_t quad, uint32_t step, uint32_t level,
                                                    uint64_t seed, uint64_t threshold) {
    const Philox4x64Out r = philox4x64_10(quad, step, level, 0, seed, 0);
    FireBallots b;
    b.w[0] = __ballot((r.w[0] >> 32) < threshold);
    b.w[1] = __ballot((r.w[1] >> 32) < threshold);
    b.w[2] = __ballot((r.w[2] >> 32) < threshold);
    b.w[3] = __ballot((r.w[3] >> 32) < threshold);
    return b;
}

__device__ __forceinline__ bool fire_bit(const FireBallots &b, int row_slot, uint64_t idx,
                                         uint64_t row_quad0) {
    const int o = (int)((idx >> 2) - row_quad0);
    const int k = (int)(idx & 3);
    const uint64_t w = k == 0 ? b.w[0] : k == 1 ? b.w[1] : k == 2 ? b.w[2] : b.w[3];
    return (w >> (16 * row_slot + o)) & 1;
}

// Store 4 channels (fp32 values) of one cell in the storage type.
__device__ __forceinline__ void store_quad(float *dst, int64_t cell, int g, v4f v) {
    *reinterpret_cast<float4 *>(dst + cell * kC + 4 * g) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store_quad(__half *dst, int64_t cell, int g, v4f v) {
    const uint32_t lo = Storage<__half>::pack_pair(v[0], v[1]);
    const uint32_t hi = Storage<__half>::pack_pair(v[2], v[3]);
    *reinterpret_cast<uint2 *>(dst + cell * kC + 4 * g) = make_uint2(lo, hi);
}

// Load one cell (all C channels, 16 bytes per thread-chunk) into 4 fp32 quad
// planes of LDS.  For fp32 storage chunk q is quad q; for fp16 storage chunk q
// holds quads 2q and 2q+1.
template <typename T> struct CellChunks;
template <> struct CellChunks<float> { static constexpr int N = 4; };
template <> struct CellChunks<__half> { static constexpr int N = 2; };

template <typename T>
__device__ __forceinline__ void stage_chunk(float4 *planes, int plane_stride, int cell, int q,
                                            const T *src_cell, bool valid);

template <>
__device__ __forceinline__ void stage_chunk<float>(float4 *planes, int ps, int cell, int q,
                                                   const float *src_cell, bool valid) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (valid) v = reinterpret_cast<const float4 *>(src_cell)[q];
    planes[q * ps + cell] = v;
}

template <>
__device__ __forceinline__ void stage_chunk<__half>(float4 *planes, int ps, int cell, int q,
                                                    const __half *src_cell, bool valid) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (valid) v = reinterpret_cast<const uint4 *>(src_cell)[q];
    float f[8];
    Storage<__half>::unpack(v, f);
    planes[(2 * q) * ps + cell] = make_float4(f[0], f[1], f[2], f[3]);
    planes[(2 * q + 1) * ps + cell] = make_float4(f[4], f[5], f[6], f[7]);
}

// Plane stride (in float4) with stride % 8 == 2: the four planes start in
// different bank groups, so 16-byte LDS writes of consecutive chunks do not
// collide.
constexpr int plane_stride(int cells) { return (cells + 7) / 8 * 8 + 2; }

// ---------------------------------------------------------------------------
// 2D
// ---------------------------------------------------------------------------
constexpr int k2TY = 16, k2TX = 32;
constexpr int k2HY = k2TY + 2, k2HX = k2TX + 2;
constexpr int k2Cells = k2HY * k2HX;
constexpr int k2PS = plane_stride(k2Cells);

template <typename T, int NIN, class Mlp>
__global__ __launch_bounds__(kThreads, 2) void nca_step_mfma_2d(
    const T *__restrict__ src, T *__restrict__ dst, int dh, int dw, int tiles_x, int tiles,
    const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint64_t seed, uint64_t threshold) {
    __shared__ float4 planes[4 * k2PS];
    constexpr int NQ = CellChunks<T>::N;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int n = lane & 15;
    const int g = lane >> 4;

    Mlp mlp;
    mlp.load(w1, b1, w2, n, g);
    float cw[9][4];
    float cb[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        cb[k] = conv_b[4 * g + k];
#pragma unroll
        for (int t = 0; t < 9; ++t) cw[t][k] = conv_w[(4 * g + k) * 9 + t];
    }
    // channels < NIN are copied, never updated
    float upd[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) upd[k] = (4 * g + k) >= NIN ? 1.f : 0.f;

    for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int ty = tile / tiles_x, tx = tile - (tile / tiles_x) * tiles_x;
        const int y0 = ty * k2TY, x0 = tx * k2TX;

        for (int i = threadIdx.x; i < k2Cells * NQ; i += kThreads) {
            const int q = i % NQ;
            const int cell = i / NQ;
            const int ly = cell / k2HX, lx = cell - (cell / k2HX) * k2HX;
            const int gy = y0 + ly - 1, gx = x0 + lx - 1;
            const bool valid = gy >= 0 && gy < dh && gx >= 0 && gx < dw;
            const int64_t gcell = valid ? (int64_t)gy * dw + gx : 0;
            stage_chunk<T>(planes, k2PS, cell, q, src + gcell * kC, valid);
        }

        // fire bits of the wave's 4 rows (rows 4*wave .. 4*wave+3 of the tile)
        const int brow = lane >> 4;
        const uint64_t brow_idx = (uint64_t)(y0 + 4 * wave + brow) * dw + x0;
        const FireBallots fb =
            fire_ballots((brow_idx >> 2) + (lane & 15), step, level, seed, threshold);
        __syncthreads();

#pragma unroll 1
        for (int grp = 0; grp < 8; ++grp) {
            const int r = grp >> 1;                 // row slot within the wave
            const int cx = (grp & 1) * 16 + n;      // column within the tile
            const int ly = 4 * wave + r;
            const int centre = (ly + 1) * k2HX + cx + 1;
            const float4 *pl = planes + g * k2PS;

            float f[8];
            const float4 s = pl[centre];
            f[0] = s.x; f[1] = s.y; f[2] = s.z; f[3] = s.w;
            float p[4] = {cb[0], cb[1], cb[2], cb[3]};
#pragma unroll
            for (int t = 0; t < 9; ++t) {
                const int off = (t / 3 - 1) * k2HX + (t % 3 - 1);
                const float4 v = pl[centre + off];
                p[0] = fmaf(cw[t][0], v.x, p[0]);
                p[1] = fmaf(cw[t][1], v.y, p[1]);
                p[2] = fmaf(cw[t][2], v.z, p[2]);
                p[3] = fmaf(cw[t][3], v.w, p[3]);
            }
            f[4] = p[0]; f[5] = p[1]; f[6] = p[2]; f[7] = p[3];

            const v4f u = mlp.update(f);

            const int y = y0 + ly, x = x0 + cx;
            if (y < dh && x < dw) {
                const uint64_t idx = (uint64_t)y * dw + x;
                const uint64_t row_q0 = ((uint64_t)y * dw + x0) >> 2;
                const float m = fire_bit(fb, r, idx, row_q0) ? 1.f : 0.f;
                v4f out;
                out[0] = fmaf(m * upd[0], u[0], f[0]);
                out[1] = fmaf(m * upd[1], u[1], f[1]);
                out[2] = fmaf(m * upd[2], u[2], f[2]);
                out[3] = fmaf(m * upd[3], u[3], f[3]);
                store_quad(dst, (int64_t)idx, g, out);
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// 3D: 8 x 32 (y, x) column, z planes streamed through a ring of 3 halo planes
// ---------------------------------------------------------------------------
constexpr int k3TY = 8, k3TX = 32;
constexpr int k3HY = k3TY + 2, k3HX = k3TX + 2;
constexpr int k3Cells = k3HY * k3HX;
constexpr int k3PS = plane_stride(k3Cells);
constexpr int k3ZRun = 16;    // z planes per work item

template <typename T>
__device__ __forceinline__ void stage_plane_3d(float4 *ring_slot, const T *__restrict__ src,
                                               int z, int dd, int dh, int dw, int y0, int x0) {
    constexpr int NQ = CellChunks<T>::N;
    const bool zin = z >= 0 && z < dd;
    for (int i = threadIdx.x; i < k3Cells * NQ; i += kThreads) {
        const int q = i % NQ;
        const int cell = i / NQ;
        const int ly = cell / k3HX, lx = cell - (cell / k3HX) * k3HX;
        const int gy = y0 + ly - 1, gx = x0 + lx - 1;
        const bool valid = zin && gy >= 0 && gy < dh && gx >= 0 && gx < dw;
        const int64_t gcell = valid ? ((int64_t)z * dh + gy) * dw + gx : 0;
        stage_chunk<T>(ring_slot, k3PS, cell, q, src + gcell * kC, valid);
    }
}

template <typename T, int NIN, class Mlp>
__global__ __launch_bounds__(kThreads, 2) void nca_step_mfma_3d(
    const T *__restrict__ src, T *__restrict__ dst, int dd, int dh, int dw, int tiles_x,
    int tiles_y, int items, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint64_t seed, uint64_t threshold) {
    __shared__ float4 ring[3][4 * k3PS];
    __shared__ float4 tapw[27][4];      // [tap][quad] conv weights of channels 4q..4q+3
    constexpr int NQ = CellChunks<T>::N;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int n = lane & 15;
    const int g = lane >> 4;

    for (int i = threadIdx.x; i < 27 * 4; i += kThreads) {
        const int t = i / 4, q = i % 4;
        tapw[t][q] = make_float4(conv_w[(4 * q + 0) * 27 + t], conv_w[(4 * q + 1) * 27 + t],
                                 conv_w[(4 * q + 2) * 27 + t], conv_w[(4 * q + 3) * 27 + t]);
    }
    Mlp mlp;
    mlp.load(w1, b1, w2, n, g);
    float cb[4];
    float upd[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        cb[k] = conv_b[4 * g + k];
        upd[k] = (4 * g + k) >= NIN ? 1.f : 0.f;
    }
    const int zruns = (dd + k3ZRun - 1) / k3ZRun;

    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        int rest = item;
        const int zr = rest % zruns;
        rest /= zruns;
        const int tx = rest % tiles_x;
        const int ty = rest / tiles_x;
        const int y0 = ty * k3TY, x0 = tx * k3TX;
        const int z_begin = zr * k3ZRun;
        const int z_end = min(dd, z_begin + k3ZRun);

        __syncthreads();   // previous item's readers are done with the ring
        stage_plane_3d<T>(ring[(z_begin + 2) % 3], src, z_begin - 1, dd, dh, dw, y0, x0);
        stage_plane_3d<T>(ring[z_begin % 3], src, z_begin, dd, dh, dw, y0, x0);

        for (int z = z_begin; z < z_end; ++z) {
            stage_plane_3d<T>(ring[(z + 1) % 3], src, z + 1, dd, dh, dw, y0, x0);
            // fire bits of the wave's 2 rows of this plane
            const int brow = (lane >> 4) & 1;
            const uint64_t brow_idx = ((uint64_t)z * dh + (y0 + 2 * wave + brow)) * dw + x0;
            const FireBallots fb =
                fire_ballots((brow_idx >> 2) + (lane & 15), step, level, seed, threshold);
            __syncthreads();

            const float4 *pm = ring[(z + 2) % 3] + g * k3PS;   // plane z - 1
            const float4 *pc = ring[z % 3] + g * k3PS;         // plane z
            const float4 *pp = ring[(z + 1) % 3] + g * k3PS;   // plane z + 1
#pragma unroll 1
            for (int grp = 0; grp < 4; ++grp) {
                const int r = grp >> 1;
                const int cx = (grp & 1) * 16 + n;
                const int ly = 2 * wave + r;
                const int centre = (ly + 1) * k3HX + cx + 1;
                float f[8];
                const float4 s = pc[centre];
                f[0] = s.x; f[1] = s.y; f[2] = s.z; f[3] = s.w;
                float p[4] = {cb[0], cb[1], cb[2], cb[3]};
#pragma unroll
                for (int t = 0; t < 27; ++t) {
                    const float4 *pl = t < 9 ? pm : t < 18 ? pc : pp;
                    const int tt = t % 9;
                    const int off = (tt / 3 - 1) * k3HX + (tt % 3 - 1);
                    const float4 v = pl[centre + off];
                    const float4 w = tapw[t][g];
                    p[0] = fmaf(w.x, v.x, p[0]);
                    p[1] = fmaf(w.y, v.y, p[1]);
                    p[2] = fmaf(w.z, v.z, p[2]);
                    p[3] = fmaf(w.w, v.w, p[3]);
                }
                f[4] = p[0]; f[5] = p[1]; f[6] = p[2]; f[7] = p[3];

                const v4f u = mlp.update(f);

                const int y = y0 + ly, x = x0 + cx;
                if (y < dh && x < dw) {
                    const uint64_t idx = ((uint64_t)z * dh + y) * dw + x;
                    const uint64_t row_q0 = (((uint64_t)z * dh + y) * dw + x0) >> 2;
                    const float m = fire_bit(fb, r, idx, row_q0) ? 1.f : 0.f;
                    v4f out;
                    out[0] = fmaf(m * upd[0], u[0], f[0]);
                    out[1] = fmaf(m * upd[1], u[1], f[1]);
                    out[2] = fmaf(m * upd[2], u[2], f[2]);
                    out[3] = fmaf(m * upd[3], u[3], f[3]);
                    store_quad(dst, (int64_t)idx, g, out);
                }
            }
            __syncthreads();   // plane z - 1's slot is refilled next
        }
    }
}

int device_cus() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cached[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

constexpr int kBlocksPerCu = 2;

template <typename T, int NIN, class Mlp>
hipError_t launch_2d(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    const int tiles_x = (int)((a.ext.w + k2TX - 1) / k2TX);
    const int tiles_y = (int)((a.ext.h + k2TY - 1) / k2TY);
    const int64_t tiles = (int64_t)tiles_x * tiles_y;
    if (tiles == 0) return hipSuccess;
    if (tiles > INT32_MAX) return hipErrorInvalidValue;
    const int grid = (int)std::min<int64_t>(tiles, (int64_t)device_cus() * kBlocksPerCu);
    nca_step_mfma_2d<T, NIN, Mlp><<<grid, kThreads, 0, stream>>>(
        (const T *)src, (T *)dst, (int)a.ext.h, (int)a.ext.w, tiles_x, (int)tiles, a.w.conv_w,
        a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.seed, a.threshold);
    return hipGetLastError();
}

template <typename T, int NIN, class Mlp>
hipError_t launch_3d(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    const int tiles_x = (int)((a.ext.w + k3TX - 1) / k3TX);
    const int tiles_y = (int)((a.ext.h + k3TY - 1) / k3TY);
    const int64_t zruns = (a.ext.d + k3ZRun - 1) / k3ZRun;
    const int64_t items = (int64_t)tiles_x * tiles_y * zruns;
    if (items == 0) return hipSuccess;
    if (items > INT32_MAX) return hipErrorInvalidValue;
    const int grid = (int)std::min<int64_t>(items, (int64_t)device_cus() * kBlocksPerCu);
    nca_step_mfma_3d<T, NIN, Mlp><<<grid, kThreads, 0, stream>>>(
        (const T *)src, (T *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, tiles_x, tiles_y,
        (int)items, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.seed,
        a.threshold);
    return hipGetLastError();
}

template <typename T, class Mlp>
hipError_t dispatch(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.ndim == 2) {
        if (a.n_in == 1) return launch_2d<T, 1, Mlp>(a, src, dst, stream);
        if (a.n_in == 3) return launch_2d<T, 3, Mlp>(a, src, dst, stream);
    } else {
        if (a.n_in == 1) return launch_3d<T, 1, Mlp>(a, src, dst, stream);
        if (a.n_in == 3) return launch_3d<T, 3, Mlp>(a, src, dst, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_step_mfma(const StepArgs &a, MfmaMlp mlp, const void *src, void *dst,
                            hipStream_t stream) {
    if (mlp == MfmaMlp::Default)
        mlp = a.dtype == Dtype::F32 ? MfmaMlp::Bf16x3 : MfmaMlp::F16;
    if (a.dtype == Dtype::F32) {
        switch (mlp) {
            case MfmaMlp::F32: return dispatch<float, MlpF32>(a, src, dst, stream);
            case MfmaMlp::Bf16x3: return dispatch<float, MlpBf16x3>(a, src, dst, stream);
            default: return hipErrorInvalidValue;   // fp16 operands are too coarse for fp32 states
        }
    }
    switch (mlp) {
        case MfmaMlp::F32: return dispatch<__half, MlpF32>(a, src, dst, stream);
        case MfmaMlp::Bf16x3: return dispatch<__half, MlpBf16x3>(a, src, dst, stream);
        case MfmaMlp::F16: return dispatch<__half, MlpF16>(a, src, dst, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace octnca
