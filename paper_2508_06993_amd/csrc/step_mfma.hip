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

// ReLU as an integer max on the float's bits: negative floats (sign bit set)
// are negative integers and become +0; one instruction, no NaN quieting.
__device__ __forceinline__ float relu(float x) {
    return __int_as_float(max(__float_as_int(x), 0));
}

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
                const float h = relu(acc[jt][i]);
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
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// hi = bf16(x) (round to nearest even, two values per conversion), hi read
// back as fp32 by bit shifts, lo = bf16(x - hi).
__device__ __forceinline__ void split_bf16(const v8f &x, v8bf &hi, v8bf &lo) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const v2bf hp = __builtin_convertvector(v2f{x[2 * p], x[2 * p + 1]}, v2bf);
        h[p] = __builtin_bit_cast(uint32_t, hp);
        const float back0 = __uint_as_float(h[p] << 16);
        const float back1 = __uint_as_float(h[p] & 0xffff0000u);
        const v2bf lp = __builtin_convertvector(v2f{x[2 * p] - back0, x[2 * p + 1] - back1}, v2bf);
        l[p] = __builtin_bit_cast(uint32_t, lp);
    }
    hi = __builtin_bit_cast(v8bf, h);
    lo = __builtin_bit_cast(v8bf, l);
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
            for (int s = 0; s < 8; ++s) x[s] = relu(acc[2 * p + s / 4][s % 4]);
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
            for (int s = 0; s < 8; ++s) x[s] = relu(acc[2 * p + s / 4][s % 4]);
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

// ---------------------------------------------------------------------------
// Halo tiles: a tile of cells (plus a one-cell halo) is read from HBM in
// 16-byte chunks, consecutive threads taking consecutive chunks (coalesced),
// and kept in LDS as fp32 in four channel-quad planes, so that the 16 lanes
// of a quad read 16 consecutive 16-byte words (no bank conflicts).  The plane
// stride is 2 mod 8 (in 16-byte words) so the four planes of one cell sit in
// different bank groups.  Loads go through registers: the next tile's loads
// are issued before the current tile is computed and written to LDS after it
// (software pipelining), so HBM latency overlaps the compute.
// ---------------------------------------------------------------------------
template <typename T> struct CellChunks;
template <> struct CellChunks<float> { static constexpr int N = 4; };    // 16 B = 4 channels
template <> struct CellChunks<__half> { static constexpr int N = 2; };   // 16 B = 8 channels

constexpr int plane_stride(int cells) { return (cells + 7) / 8 * 8 + 2; }

template <typename T, int HY, int HX>
struct HaloLoader {
    static constexpr int kCells = HY * HX;
    static constexpr int NQ = CellChunks<T>::N;
    static constexpr int kChunks = kCells * NQ;
    static constexpr int NCH = (kChunks + kThreads - 1) / kThreads;
    static constexpr int PS = plane_stride(kCells);
    uint4 v[NCH];

    // Halo plane z (ignored for 2D: pass z = 0, dd = 1) of the tile whose
    // interior starts at (y0, x0); cells outside the grid read as zero.
    __device__ __forceinline__ void issue(const T *__restrict__ src, int z, int dd, int dh, int dw,
                                          int y0, int x0) {
        const bool zin = z >= 0 && z < dd;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int i = (int)threadIdx.x + c * kThreads;
            const int q = i % NQ;
            const int cell = i / NQ;
            const int ly = cell / HX, lx = cell - (cell / HX) * HX;
            const int gy = y0 + ly - 1, gx = x0 + lx - 1;
            const bool valid = i < kChunks && zin && gy >= 0 && gy < dh && gx >= 0 && gx < dw;
            v[c] = make_uint4(0u, 0u, 0u, 0u);
            if (valid) {
                const int64_t gcell = ((int64_t)z * dh + gy) * dw + gx;
                v[c] = reinterpret_cast<const uint4 *>(src + gcell * kC)[q];
            }
        }
    }

    __device__ __forceinline__ void commit(float4 *planes) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int i = (int)threadIdx.x + c * kThreads;
            if (i < kChunks) {
                const int q = i % NQ;
                const int cell = i / NQ;
                if constexpr (NQ == 4) {
                    planes[q * PS + cell] = make_float4(__uint_as_float(v[c].x),
                                                        __uint_as_float(v[c].y),
                                                        __uint_as_float(v[c].z),
                                                        __uint_as_float(v[c].w));
                } else {
                    float f[8];
                    Storage<__half>::unpack(v[c], f);
                    planes[(2 * q) * PS + cell] = make_float4(f[0], f[1], f[2], f[3]);
                    planes[(2 * q + 1) * PS + cell] = make_float4(f[4], f[5], f[6], f[7]);
                }
            }
        }
    }
};

// Residual update and store of the lane's 4 channels (fp32 values, stored in
// the storage type).  upd[k] is 0 for input channels, 1 otherwise; with
// m * upd = 0 the fma returns the state bit for bit (u is finite).
__device__ __forceinline__ void store_quad(float *dst, int64_t cell, int g, v4f v) {
    *reinterpret_cast<float4 *>(dst + cell * kC + 4 * g) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store_quad(__half *dst, int64_t cell, int g, v4f v) {
    const uint32_t lo = Storage<__half>::pack_pair(v[0], v[1]);
    const uint32_t hi = Storage<__half>::pack_pair(v[2], v[3]);
    *reinterpret_cast<uint2 *>(dst + cell * kC + 4 * g) = make_uint2(lo, hi);
}

template <typename T>
__device__ __forceinline__ void update_store(T *dst, int64_t idx, int g, const float f[8],
                                             const v4f &u, const float upd[4], bool fire) {
    const float m = fire ? 1.f : 0.f;
    v4f out;
    out[0] = fmaf(m * upd[0], u[0], f[0]);
    out[1] = fmaf(m * upd[1], u[1], f[1]);
    out[2] = fmaf(m * upd[2], u[2], f[2]);
    out[3] = fmaf(m * upd[3], u[3], f[3]);
    store_quad(dst, idx, g, out);
}

// ---------------------------------------------------------------------------
// 2D: persistent blocks loop over 16 x 32 tiles (tile index row-major).
// ---------------------------------------------------------------------------
constexpr int k2TY = 16, k2TX = 32;
constexpr int k2HY = k2TY + 2, k2HX = k2TX + 2;

template <typename T, int NIN, class Mlp>
__global__ __launch_bounds__(kThreads, 2) void nca_step_mfma_2d(
    const T *__restrict__ src, T *__restrict__ dst, int dh, int dw, int tiles_x, int tiles,
    const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint64_t seed, uint64_t threshold) {
    using Loader = HaloLoader<T, k2HY, k2HX>;
    __shared__ float4 planes[4 * Loader::PS];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int n = lane & 15;
    const int g = lane >> 4;

    Mlp mlp;
    mlp.load(w1, b1, w2, n, g);
    float cw[9][4];
    float cb[4];
    float upd[4];   // channels < NIN are copied, never updated
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        cb[k] = conv_b[4 * g + k];
        upd[k] = (4 * g + k) >= NIN ? 1.f : 0.f;
#pragma unroll
        for (int t = 0; t < 9; ++t) cw[t][k] = conv_w[(4 * g + k) * 9 + t];
    }

    Loader ld;
    int tile = blockIdx.x;
    if (tile < tiles) {
        const int ty = tile / tiles_x;
        ld.issue(src, 0, 1, dh, dw, ty * k2TY, (tile - ty * tiles_x) * k2TX);
    }
    for (; tile < tiles; tile += gridDim.x) {
        const int ty = tile / tiles_x;
        const int y0 = ty * k2TY, x0 = (tile - ty * tiles_x) * k2TX;
        ld.commit(planes);
        // fire bits of the wave's 4 rows (rows 4*wave .. 4*wave+3 of the tile)
        const uint64_t brow_idx = (uint64_t)(y0 + 4 * wave + (lane >> 4)) * dw + x0;
        const FireBallots fb =
            fire_ballots((brow_idx >> 2) + (lane & 15), step, level, seed, threshold);
        __syncthreads();
        const int next = tile + (int)gridDim.x;
        if (next < tiles) {
            const int nty = next / tiles_x;
            ld.issue(src, 0, 1, dh, dw, nty * k2TY, (next - nty * tiles_x) * k2TX);
        }

        const float4 *pl = planes + g * Loader::PS;
#pragma unroll 1
        for (int grp = 0; grp < 8; ++grp) {
            const int r = grp >> 1;                 // row slot within the wave
            const int cx = (grp & 1) * 16 + n;      // column within the tile
            const int ly = 4 * wave + r;
            const int centre = (ly + 1) * k2HX + cx + 1;

            float f[8];
            const float4 sv = pl[centre];
            f[0] = sv.x; f[1] = sv.y; f[2] = sv.z; f[3] = sv.w;
            float p[4] = {cb[0], cb[1], cb[2], cb[3]};
#pragma unroll
            for (int t = 0; t < 9; ++t) {
                const float4 v = pl[centre + (t / 3 - 1) * k2HX + (t % 3 - 1)];
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
                update_store(dst, (int64_t)idx, g, f, u, upd, fire_bit(fb, r, idx, row_q0));
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// 3D: a work item is an 8 x 32 (y, x) column and a run of z planes; planes
// stream through a ring of three halo planes in LDS, the plane after next
// being loaded while the current one is computed.
// ---------------------------------------------------------------------------
constexpr int k3TY = 8, k3TX = 32;
constexpr int k3HY = k3TY + 2, k3HX = k3TX + 2;
constexpr int k3ZRun = 16;    // z planes per work item

template <typename T, int NIN, class Mlp>
__global__ __launch_bounds__(kThreads, 2) void nca_step_mfma_3d(
    const T *__restrict__ src, T *__restrict__ dst, int dd, int dh, int dw, int tiles_x,
    int tiles_y, int items, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint64_t seed, uint64_t threshold) {
    using Loader = HaloLoader<T, k3HY, k3HX>;
    __shared__ float4 ring[3][4 * Loader::PS];
    __shared__ float4 tapw[27][4];      // [tap][quad] conv weights of channels 4q..4q+3

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
    Loader ld;

    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        int rest = item;
        const int zr = rest % zruns;
        rest /= zruns;
        const int tx = rest % tiles_x;
        const int ty = rest / tiles_x;
        const int y0 = ty * k3TY, x0 = tx * k3TX;
        const int z_begin = zr * k3ZRun;
        const int z_end = min(dd, z_begin + k3ZRun);

        __syncthreads();   // the previous item's readers are done with the ring
        ld.issue(src, z_begin - 1, dd, dh, dw, y0, x0);
        ld.commit(ring[(z_begin + 2) % 3]);
        ld.issue(src, z_begin, dd, dh, dw, y0, x0);
        ld.commit(ring[z_begin % 3]);
        ld.issue(src, z_begin + 1, dd, dh, dw, y0, x0);

        for (int z = z_begin; z < z_end; ++z) {
            ld.commit(ring[(z + 1) % 3]);
            // fire bits of the wave's 2 rows of this plane
            const uint64_t brow_idx =
                ((uint64_t)z * dh + (y0 + 2 * wave + ((lane >> 4) & 1))) * dw + x0;
            const FireBallots fb =
                fire_ballots((brow_idx >> 2) + (lane & 15), step, level, seed, threshold);
            __syncthreads();
            if (z + 2 <= z_end) ld.issue(src, z + 2, dd, dh, dw, y0, x0);

            const float4 *pm = ring[(z + 2) % 3] + g * Loader::PS;   // plane z - 1
            const float4 *pc = ring[z % 3] + g * Loader::PS;         // plane z
            const float4 *pp = ring[(z + 1) % 3] + g * Loader::PS;   // plane z + 1
#pragma unroll 1
            for (int grp = 0; grp < 4; ++grp) {
                const int r = grp >> 1;
                const int cx = (grp & 1) * 16 + n;
                const int ly = 2 * wave + r;
                const int centre = (ly + 1) * k3HX + cx + 1;
                float f[8];
                const float4 sv = pc[centre];
                f[0] = sv.x; f[1] = sv.y; f[2] = sv.z; f[3] = sv.w;
                float p[4] = {cb[0], cb[1], cb[2], cb[3]};
                // taps in order (dz, dy, dx); one plane at a time keeps the
                // number of LDS values in flight (and registers) bounded
#pragma unroll 1
                for (int pz = 0; pz < 3; ++pz) {
                    const float4 *pl = pz == 0 ? pm : pz == 1 ? pc : pp;
#pragma unroll
                    for (int tt = 0; tt < 9; ++tt) {
                        const float4 v = pl[centre + (tt / 3 - 1) * k3HX + (tt % 3 - 1)];
                        const float4 w = tapw[pz * 9 + tt][g];
                        p[0] = fmaf(w.x, v.x, p[0]);
                        p[1] = fmaf(w.y, v.y, p[1]);
                        p[2] = fmaf(w.z, v.z, p[2]);
                        p[3] = fmaf(w.w, v.w, p[3]);
                    }
                }
                f[4] = p[0]; f[5] = p[1]; f[6] = p[2]; f[7] = p[3];

                const v4f u = mlp.update(f);

                const int y = y0 + ly, x = x0 + cx;
                if (y < dh && x < dw) {
                    const uint64_t idx = ((uint64_t)z * dh + y) * dw + x;
                    const uint64_t row_q0 = (((uint64_t)z * dh + y) * dw + x0) >> 2;
                    update_store(dst, (int64_t)idx, g, f, u, upd, fire_bit(fb, r, idx, row_q0));
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
