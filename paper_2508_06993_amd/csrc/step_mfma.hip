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
// Fire bits: each lane evaluates Philox4x64-10 for one block of 8 cells of
// the rows its wave owns (covering several tiles or planes ahead), the bits
// are spread with eight ballots and every lane picks its cell's bit.
//
// 2D: a persistent grid loops over 16 x 32 tiles; the 18 x 34 halo tile is
// staged in LDS as fp32 in four channel-quad planes (conflict-free 16-byte
// reads).  3D: a block owns an 8 x 32 column of the (y, x) plane and a run
// of z planes, keeping three halo planes in an LDS ring (each plane is read
// from HBM once per run).
#include <atomic>
#include <algorithm>
#include <type_traits>

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

// Marks a register value as produced here (an empty asm that reads and
// rewrites it): loads of kernel-wide constants then complete in the prologue
// instead of being sunk into the tile loop, where the compiler would have to
// wait for all outstanding memory operations at their first use.
template <typename V>
__device__ __forceinline__ void pin(V &x) {
    asm volatile("" : "+v"(x));
}

// ---------------------------------------------------------------------------
// MLP policies.  Each gathers its weights into lane registers once per block
// (load) and computes the update of channels 4g..4g+3 of the lane's cell from
// its 8 features in two halves: layer1 (features -> hidden accumulators, all
// MFMA) and layer2 (ReLU, hidden -> update).  Splitting them lets a wave
// issue the next group's perception while layer 1's MFMAs run.  All
// accumulate in fp32.  The second layer has outputs for the hidden channels
// only (Sec. 3.1): load() gathers the W2 rows of the nin input channels as
// zeros, so their update is exactly +0 and the residual needs no per-channel
// mask.  Those rows are loaded like the others and then replaced by zero: a
// load behind the lane condition became a branch and a full memory wait per
// element (16 round trips, about 5 us per launch, measured).
// kPerceptionScale: the factor the kernel applies to the perception weights
// and bias (features 4..7 arrive multiplied by it).
// ---------------------------------------------------------------------------

// ReLU as an integer max on the float's bits: negative floats (sign bit set)
// are negative integers and become +0; one instruction, no NaN quieting.
__device__ __forceinline__ float relu(float x) {
    return __int_as_float(max(__float_as_int(x), 0));
}

// fp32 operands: v_mfma_f32_16x16x4_f32, 32 + 16 MFMAs per 16 cells.
struct MlpF32 {
    static constexpr int kChannels = kC, kHidden = kH;
    static constexpr float kPerceptionScale = 1.f;
    float w1[4][8];   // [jt][kc] = W1[jt*16 + n][feature(kc, g)]
    v4f b1[4];        // [jt][i]  = b1[jt*16 + 4g + i]
    float w2[4][4];   // [jt][i]  = W2[n][jt*16 + 4g + i]   (n = output channel)

    __device__ __forceinline__ void pin_all() {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
            for (int k = 0; k < 8; ++k) pin(w1[jt][k]);
#pragma unroll
            for (int i = 0; i < 4; ++i) pin(w2[jt][i]);
            pin(b1[jt]);
        }
    }

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g, int nin) {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
            for (int kc = 0; kc < 8; ++kc) w1[jt][kc] = W1[(jt * 16 + n) * 2 * kC + feature_of(kc, g)];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                b1[jt][i] = B1[jt * 16 + 4 * g + i];
                const float v = W2[n * kH + jt * 16 + 4 * g + i];   // loaded for every n
                w2[jt][i] = n < nin ? 0.f : v;
            }
        }
    }

    __device__ __forceinline__ void layer1(const float f[8], v4f acc[4]) const {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[jt][0], f[0], b1[jt], 0, 0, 0);
#pragma unroll
        for (int kc = 1; kc < 8; ++kc)
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
                acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[jt][kc], f[kc], acc[jt], 0, 0, 0);
    }

    __device__ __forceinline__ v4f layer2(const v4f acc[4]) const {
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
    static constexpr int kChannels = kC, kHidden = kH;
    static constexpr float kPerceptionScale = 1.f;
    v8bf w1h[4], w1l[4];   // [jt] slot s: W1[jt*16 + n][feature(s, g)]
    v4f b1[4];
    v8bf w2h[2], w2l[2];   // [p] slot s: W2[n][hidden(p, s, g)]

    __device__ __forceinline__ void pin_all() {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            pin(w1h[jt]);
            pin(w1l[jt]);
            pin(b1[jt]);
        }
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            pin(w2h[p]);
            pin(w2l[p]);
        }
    }

    // hidden unit in K slot s of layer-2 MFMA p for lane group g: it is the
    // layer-1 accumulator register (jt = 2p + s/4, i = s%4) of the lane.
    __device__ static __forceinline__ int hidden_of(int p, int s, int g) {
        return (2 * p + s / 4) * 16 + 4 * g + (s % 4);
    }

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g, int nin) {
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
            for (int s = 0; s < 8; ++s) {
                const float v = W2[n * kH + hidden_of(p, s, g)];   // loaded for every n
                x[s] = n < nin ? 0.f : v;
            }
            split_bf16(x, w2h[p], w2l[p]);
        }
    }

    __device__ __forceinline__ void layer1(const float f[8], v4f acc[4]) const {
        v8f fx;
#pragma unroll
        for (int s = 0; s < 8; ++s) fx[s] = f[s];
        v8bf fh, fl;
        split_bf16(fx, fh, fl);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1l[jt], fh, b1[jt], 0, 0, 0);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1h[jt], fl, acc[jt], 0, 0, 0);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1h[jt], fh, acc[jt], 0, 0, 0);
    }

    __device__ __forceinline__ v4f layer2(const v4f acc[4]) const {
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
    static constexpr int kChannels = kC, kHidden = kH;
    static constexpr float kPerceptionScale = 1.f;
    v8h w1[4];
    v4f b1[4];
    v8h w2[2];

    __device__ __forceinline__ void pin_all() {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            pin(w1[jt]);
            pin(b1[jt]);
        }
        pin(w2[0]);
        pin(w2[1]);
    }

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g, int nin) {
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
            for (int s = 0; s < 8; ++s) {
                const float v = W2[n * kH + MlpBf16x3::hidden_of(p, s, g)];   // loaded for every n
                x[s] = n < nin ? 0.f : v;
            }
            w2[p] = __builtin_convertvector(x, v8h);
        }
    }

    __device__ __forceinline__ void layer1(const float f[8], v4f acc[4]) const {
        v8f fx;
#pragma unroll
        for (int s = 0; s < 8; ++s) fx[s] = f[s];
        layer1_h(__builtin_convertvector(fx, v8h), acc);
    }

    // features already in fp16 (slot s = feature_of(s, g))
    __device__ __forceinline__ void layer1_h(const v8h &fh, v4f acc[4]) const {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(w1[jt], fh, b1[jt], 0, 0, 0);
    }

    // ReLU after the rounding to fp16, as packed fp16 max (half the
    // instructions of an fp32 max; rounding is monotonic and keeps 0, so the
    // operand is the same fp16 value).
    __device__ __forceinline__ v4f layer2(const v4f acc[4]) const {
        v4f u = {0.f, 0.f, 0.f, 0.f};
        const v8h zero = {};
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = acc[2 * p + s / 4][s % 4];
            const v8h h = __builtin_elementwise_max(__builtin_convertvector(x, v8h), zero);
            u = __builtin_amdgcn_mfma_f32_16x16x32_f16(w2[p], h, u, 0, 0, 0);
        }
        return u;
    }
};

// Scaled fp16 activations with split fp16 weights (for fp32 states).  The
// features and the hidden units are rounded to fp16 after a scaling by 2^-8
// (a power of two: exact), which keeps fp32 states of magnitude up to
// 65504 * 2^8 in fp16 range; the weights are hi + lo fp16 pairs (W1 as is,
// b1 times 2^-8 as the accumulator start, W2 times 2^8 so that u comes out
// unscaled), two products per weight: 8 + 4 MFMAs per 16 cells and no
// activation split.  The activations keep fp16's 2^-12 relative rounding,
// the weights about 2^-22.
constexpr float kF16ActScale = 1.f / 256.f;

// Feature order of a model with C channels (C <= 16, a multiple of 4): slot
// s < 4 of lane group g is state channel 4g + s, slot s >= 4 perception
// channel 4g + s - 4; lane groups g >= C / 4 hold no channel.
template <int C>
__device__ __forceinline__ int feature_of_c(int slot, int g) {
    return slot < 4 ? 4 * g + slot : C + 4 * g + (slot - 4);
}

// C / H: the model's size.  The lane layout is that of C = 16, H = 64; a
// smaller model (C = 12, H = 48 of the paper's ablation, supplement S10)
// leaves channel quad 3 and hidden tile 3 empty.  Their weights are gathered
// as zeros (loaded from clamped indices and then replaced), hidden tile 3 is
// not computed, and the update of channels >= C is +0.
template <int C, int H>
struct MlpF16SM {
    static_assert(C % 4 == 0 && C <= kC && H % 16 == 0 && H <= kH, "fits the 16 / 64 lanes");
    static constexpr int kChannels = C, kHidden = H;
    static constexpr int NT = H / 16;   // hidden tiles computed
    static constexpr float kPerceptionScale = kF16ActScale;
    v8h w1h[NT], w1l[NT];   // [jt] slot s: W1[jt*16 + n][feature(s, g)], hi + lo
    v4f b1[NT];             // b1 * 2^-8
    v8h w2h[2], w2l[2];     // [p] slot s: 2^8 W2[n][hidden(p, s, g)], hi + lo

    __device__ __forceinline__ void pin_all() {
#pragma unroll
        for (int jt = 0; jt < NT; ++jt) {
            pin(w1h[jt]);
            pin(w1l[jt]);
            pin(b1[jt]);
        }
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            pin(w2h[p]);
            pin(w2l[p]);
        }
    }

    __device__ static __forceinline__ void split(const v8f &x, v8h &hi, v8h &lo) {
        hi = __builtin_convertvector(x, v8h);
        lo = __builtin_convertvector(x - __builtin_convertvector(hi, v8f), v8h);
    }

    __device__ __forceinline__ void load(const float *__restrict__ W1, const float *__restrict__ B1,
                                         const float *__restrict__ W2, int n, int g, int nin) {
        const bool g_ok = g < C / 4;
        const int gc = g_ok ? g : 0;
#pragma unroll
        for (int jt = 0; jt < NT; ++jt) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const float v = W1[(jt * 16 + n) * 2 * C + feature_of_c<C>(s, gc)];
                x[s] = g_ok ? v : 0.f;
            }
            split(x, w1h[jt], w1l[jt]);
#pragma unroll
            for (int i = 0; i < 4; ++i) b1[jt][i] = B1[jt * 16 + 4 * g + i] * kF16ActScale;
        }
        // rows of the input channels and of channels >= C are zero
        const bool row_ok = n >= nin && n < C;
        const int nc = n < C ? n : 0;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const int hid = MlpBf16x3::hidden_of(p, s, g);
                const float v = W2[nc * H + (hid < H ? hid : 0)];   // loaded for every n
                x[s] = row_ok && hid < H ? v * (1.f / kF16ActScale) : 0.f;
            }
            split(x, w2h[p], w2l[p]);
        }
    }

    __device__ __forceinline__ void layer1(const float f[8], v4f acc[4]) const {
        v8f fx;   // state features scaled here, the perception arrives scaled
#pragma unroll
        for (int s = 0; s < 8; ++s) fx[s] = s < 4 ? f[s] * kF16ActScale : f[s];
        const v8h fh = __builtin_convertvector(fx, v8h);
#pragma unroll
        for (int jt = 0; jt < NT; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(w1l[jt], fh, b1[jt], 0, 0, 0);
#pragma unroll
        for (int jt = 0; jt < NT; ++jt)
            acc[jt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(w1h[jt], fh, acc[jt], 0, 0, 0);
    }

    // ReLU as packed fp16 max after the rounding (as in MlpF16); hidden tiles
    // that are not computed enter as zeros
    __device__ __forceinline__ v4f layer2(const v4f acc[4]) const {
        v4f u = {0.f, 0.f, 0.f, 0.f};
        const v8h zero = {};
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            v8f x;
#pragma unroll
            for (int s = 0; s < 8; ++s) x[s] = 2 * p + s / 4 < NT ? acc[2 * p + s / 4][s % 4] : 0.f;
            const v8h h = __builtin_elementwise_max(__builtin_convertvector(x, v8h), zero);
            u = __builtin_amdgcn_mfma_f32_16x16x32_f16(w2l[p], h, u, 0, 0, 0);
            u = __builtin_amdgcn_mfma_f32_16x16x32_f16(w2h[p], h, u, 0, 0, 0);
        }
        return u;
    }
};
using MlpF16S = MlpF16SM<kC, kH>;

// The MLP policy of fp32 states when none is asked for.
using MlpF32State = MlpF16S;

// Fire bits.  One Philox4x64-10 evaluation gives the draws of a block of 8
// consecutive cells, so a wave evaluates one block per lane and spreads the
// bits with eight ballots (ballot b holds the bit of cell b of each lane's
// block).  Lanes are assigned to row slots of `opr` blocks each: bit
// (slot * opr + o) of ballot b is the bit of cell 8 * (b0(slot) + o) + b,
// where b0(slot) = (canonical index of the slot's first cell) >> 3.
// When rows start on an 8-cell boundary (w % 8 == 0) a 32-cell tile row is
// exactly 4 blocks (opr = 4) and a lane's cells always take the same ballot
// (cell n of a 16-cell group has b = n % 8), so each lane selects its ballot
// once per evaluation; otherwise a row uses opr = 8 and the ballot is
// selected per cell.  The 2D step selects in registers (FireBits below); the
// 3D steps keep the 8 ballots in a small per-wave LDS array and read ballot
// (idx & 7) by address, because there the register select was lowered to a
// private array whose loads the stores then had to wait for.
struct FireBallots {
    uint64_t w[8];
};

__device__ __forceinline__ FireBallots fire_ballots(uint64_t block, uint32_t step, uint32_t level,
                                                    uint32_t batch, uint64_t seed,
                                                    uint64_t threshold) {
    const Philox4x64Out r = philox4x64_10(block, step, level, batch, seed, 0);
    FireBallots f;
#pragma unroll
    for (int b = 0; b < 8; ++b) f.w[b] = __ballot((uint64_t)draw_of(r, (uint32_t)b) < threshold);
    return f;
}

// Ballot b of the set, selected without branches.
__device__ __forceinline__ uint64_t select_ballot(const FireBallots &f, uint32_t b) {
    const uint64_t w01 = (b & 1u) ? f.w[1] : f.w[0];
    const uint64_t w23 = (b & 1u) ? f.w[3] : f.w[2];
    const uint64_t w45 = (b & 1u) ? f.w[5] : f.w[4];
    const uint64_t w67 = (b & 1u) ? f.w[7] : f.w[6];
    const uint64_t w03 = (b & 2u) ? w23 : w01;
    const uint64_t w47 = (b & 2u) ? w67 : w45;
    return (b & 4u) ? w47 : w03;
}

// Per-lane view of one evaluation: `mine` is the ballot of the lane's cells
// when rows are 8-aligned.
struct FireBits {
    FireBallots f;
    uint64_t mine;
    bool aligned;
    int opr;

    // Bit of cell idx in row slot `slot` whose first block is row_b0.
    __device__ __forceinline__ bool bit(int slot, uint64_t idx, uint64_t row_b0) const {
        const int o = (int)((idx >> 3) - row_b0);
        const uint64_t w = aligned ? mine : select_ballot(f, (uint32_t)idx & 7u);
        return (w >> (slot * opr + o)) & 1;
    }

};

// ---------------------------------------------------------------------------
// Halo tiles: HY rows of 34 cells (a 32-cell-wide interior plus one halo cell
// on each side) of one z plane.  In LDS they are kept as fp32 in four
// channel-quad planes, so that the 16 lanes of a quad read 16 consecutive
// 16-byte words (no bank conflicts); the plane stride is 2 mod 8 (16-byte
// words, see plane_stride).
// Loads are whole 16-byte chunks: a "body" load moves the 64 chunks of a row
// segment (16 cells in fp32, 32 in fp16) from one wave-uniform address, a
// "side" load moves the left and right halo cells of several rows.  The loads are spread over the 4 waves
// and go through registers: the next tile's loads are issued before the
// current tile is computed and written to LDS after it (software
// pipelining), so HBM latency overlaps the compute.
// ---------------------------------------------------------------------------
template <typename T> struct CellChunks;
template <> struct CellChunks<float> { static constexpr int N = 4; };    // 16 B = 4 channels
template <> struct CellChunks<__half> { static constexpr int N = 2; };   // 16 B = 8 channels

// Plane stride rounded up to 16 words (256 B): measured on gfx950, strides of
// 2, 4 and 12 words mod 16 left the 16-lane plane reads with ~20x more LDS
// bank-conflict cycles than this choice.
constexpr int plane_stride(int cells) { return (cells + 15) / 16 * 16; }
constexpr int kTileW = 32;
constexpr int kHaloW = kTileW + 2;

// Buffer resources: every global access of the step kernel goes through a
// raw buffer descriptor whose range covers only the rows a tile may touch;
// an out-of-range offset (0xffffffff is used for cells outside the grid)
// reads 0 and drops a store.  So no load or store sits behind a branch, the
// compiler sees a fixed sequence of vector-memory operations per tile, and
// waits for the prefetched loads without draining the stores (loads and
// stores share one completion counter).
typedef __amdgpu_buffer_rsrc_t Rsrc;
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
constexpr uint32_t kOut = 0xffffffffu;      // offset that is always out of range
constexpr int kRsrcWord3 = 0x00020000;      // raw buffer, 32-bit data format

__device__ __forceinline__ Rsrc make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, kRsrcWord3);
}

// Workgroups go to the eight XCDs in turn (blockIdx % 8) and each XCD has an
// L2 of its own.  The grid-stride loops of the 3D step kernels map their index
// u to a work item such that the workgroups of one XCD that run at the same
// time take consecutive items (neighbouring tiles of one z run), which then
// find each other's halo rows and columns in that L2 instead of fetching the
// same lines again (measured: 1% off the video step; the 2D row kernel, where
// it measured 2% slower, keeps the plain order).  A bijection of
// [0, rounds * grid) when grid % 8 == 0, the identity otherwise.
constexpr int kXcds = 8;
__device__ __forceinline__ int64_t xcd_item(int64_t u, int grid) {
    if (grid % kXcds) return u;
    const int64_t r = u / grid;
    const int b = (int)(u - r * grid);
    return (r * kXcds + b % kXcds) * (grid / kXcds) + b / kXcds;
}

// C: channels of a cell; a cell fills kChunks of the NQ 16-byte chunks, the
// loads of the others (channel quad 3 when C = 12) take the out-of-range
// offset and read as zero.
template <typename T, int HY, int C = kC>
struct RowLoader {
    static constexpr int NQ = CellChunks<T>::N;
    static constexpr int kCellBytes = C * (int)sizeof(T);
    static constexpr int kChunks = kCellBytes / 16;
    static_assert(kCellBytes % 16 == 0 && kChunks <= NQ, "whole 16-byte chunks");
    static constexpr int kCellsPerBody = 64 / NQ;            // cells per body load
    static constexpr int kBodyPerRow = kTileW / kCellsPerBody;
    static constexpr int kRowsPerSide = 64 / (2 * NQ);       // rows per side load
    static constexpr int kBody = HY * kBodyPerRow;
    static constexpr int kSide = (HY + kRowsPerSide - 1) / kRowsPerSide;
    static constexpr int kBodySlots = (kBody + 3) / 4;       // body loads per wave (max)
    static_assert(kSide <= 4, "one side load per wave at most");
    static constexpr int PS = plane_stride(HY * kHaloW);
    // Body load J (0 <= J < kBody) is slot J / 4 of wave J % 4: every wave
    // runs the same instruction sequence.  Side load s is done by wave 3 - s,
    // in one extra slot.
    uint4 v[kBodySlots + 1];

    // A body load moves the kCellsPerBody cells x NQ chunks of a row segment.
    // Lane i takes chunk i / kCellsPerBody of cell i % kCellsPerBody: the
    // wave still reads one contiguous 1 KB, and each group of consecutive
    // lanes writes consecutive 16-byte words of one LDS plane (no bank
    // conflicts on the commit).
    __device__ static __forceinline__ int body_cell(int lane) { return lane % kCellsPerBody; }
    __device__ static __forceinline__ int body_chunk(int lane) { return lane / kCellsPerBody; }

    // Per-lane byte offsets of a tile's loads within its rows (kOut for
    // unused slots and for cells left of x = 0, above y = 0 or right of the
    // grid; rows below the grid fall outside the descriptor).  They depend on
    // the tile only, so a plane loop computes them once per work item and
    // issue_at() changes only the descriptor from plane to plane.
    struct Offsets {
        uint32_t o[kBodySlots + 1];
    };
    __device__ __forceinline__ static Offsets offsets(int dw, int y0, int x0) {
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int gy0 = y0 - 1;
        const int base_row = gy0 > 0 ? gy0 : 0;
        const uint32_t row_bytes = (uint32_t)dw * kCellBytes;
        const int cell = body_cell(lane);
        const uint32_t lane_off = (uint32_t)(cell * kCellBytes + body_chunk(lane) * 16);
        Offsets r;
#pragma unroll
        for (int k = 0; k < kBodySlots; ++k) {
            const int J = wave + 4 * k;                       // wave-uniform
            const int gy = gy0 + J / kBodyPerRow;
            const int cx0 = x0 + (J % kBodyPerRow) * kCellsPerBody;
            const bool ok = J < kBody && gy >= 0 && cx0 + cell < dw && body_chunk(lane) < kChunks;
            const uint32_t off = (uint32_t)(gy - base_row) * row_bytes +
                                 (uint32_t)cx0 * kCellBytes + lane_off;
            r.o[k] = ok ? off : kOut;
        }
        const int s = 3 - wave;
        const int row = s * kRowsPerSide + lane / (2 * NQ);
        const int gy = gy0 + row;
        const int gx = ((lane / NQ) & 1) ? x0 + kTileW : x0 - 1;
        const bool ok =
            s < kSide && row < HY && gy >= 0 && gx >= 0 && gx < dw && lane % NQ < kChunks;
        const uint32_t off = (uint32_t)(gy - base_row) * row_bytes + (uint32_t)gx * kCellBytes +
                             (uint32_t)(lane % NQ) * 16;
        r.o[kBodySlots] = ok ? off : kOut;
        return r;
    }

    // Tile whose interior starts at (y0, x0) in plane z (lane offsets `of`
    // from offsets()); cells outside the grid (or z outside [0, dd)) read as
    // zero.  The grid must satisfy HY * dw * kCellBytes < 2^32 (checked by
    // the launcher).  With active = false nothing is read (the descriptor is
    // empty) and the registers are zero: the next-tile prefetch is issued
    // unconditionally.
    __device__ __forceinline__ void issue_at(const T *__restrict__ src, const Offsets &of, int z,
                                             int dd, int dh, int dw, int y0, bool active = true) {
        const int gy0 = y0 - 1;
        const int base_row = gy0 > 0 ? gy0 : 0;
        const int rows =
            (active && z >= 0 && z < dd) ? max(0, min(gy0 + HY, dh) - base_row) : 0;
        const uint32_t row_bytes = (uint32_t)dw * kCellBytes;
        const Rsrc r = make_rsrc(src + ((int64_t)max(z, 0) * dh + base_row) * dw * C,
                                 (uint32_t)rows * row_bytes);
#pragma unroll
        for (int k = 0; k <= kBodySlots; ++k) {
            const v4u x = __builtin_amdgcn_raw_buffer_load_b128(r, of.o[k], 0, 0);
            v[k] = make_uint4(x[0], x[1], x[2], x[3]);
        }
    }
    __device__ __forceinline__ void issue(const T *__restrict__ src, int z, int dd, int dh, int dw,
                                          int y0, int x0, bool active = true) {
        issue_at(src, offsets(dw, y0, x0), z, dd, dh, dw, y0, active);
    }

__device__ __forceinline__ static void put(float4 *planes, int q, int cell, const uint4 &c) {
        if constexpr (NQ == 4) {
            planes[q * PS + cell] = make_float4(__uint_as_float(c.x), __uint_as_float(c.y),
                                                __uint_as_float(c.z), __uint_as_float(c.w));
        } else {
            float f[8];
            Storage<__half>::unpack(c, f);
            planes[(2 * q) * PS + cell] = make_float4(f[0], f[1], f[2], f[3]);
            planes[(2 * q + 1) * PS + cell] = make_float4(f[4], f[5], f[6], f[7]);
        }
    }

    // LDS slot that is never read (plane padding): target of the writes of
    // unused load slots, so the commit has no branches either.
    static constexpr int kDummyCell = HY * kHaloW;
    static_assert(kDummyCell < PS, "plane padding holds the dummy slot");

    __device__ __forceinline__ void commit(float4 *planes) const {
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int cell = body_cell(lane), chunk = body_chunk(lane);
#pragma unroll
        for (int k = 0; k < kBodySlots; ++k) {
            const int J = wave + 4 * k;
            const int slot =
                (J / kBodyPerRow) * kHaloW + 1 + (J % kBodyPerRow) * kCellsPerBody + cell;
            put(planes, chunk, J < kBody ? slot : kDummyCell, v[k]);
        }
        const int s = 3 - wave;
        const int row = s * kRowsPerSide + lane / (2 * NQ);
        const int slot = row * kHaloW + (((lane / NQ) & 1) ? kHaloW - 1 : 0);
        put(planes, lane % NQ, (s < kSide && row < HY) ? slot : kDummyCell, v[kBodySlots]);
    }

    // fp16 rows kept as fp16 in LDS: four channel-quad planes of 8-byte words
    // (channels 4q..4q+3 of a cell); a 16-byte chunk c (channels 8c..8c+7)
    // is split between quad planes 2c and 2c+1.  Same slots as commit().
    // Quad plane stride of the fp16 planes (8-byte words): 16 mod 32, so the
    // planes of lane groups g and g + 1 start 128 bytes apart modulo 256 (the
    // 8-byte reads of one wave then hit disjoint banks; measured 8.8x fewer
    // bank-conflict cycles than a multiple of 32).
    static constexpr int PS16 = (HY * kHaloW + 1 + 15) / 32 * 32 + 16;
    static_assert(PS16 > kDummyCell, "fp16 plane padding holds the dummy slot");
    __device__ static __forceinline__ void put_raw(uint2 *planes, int c, int cell, const uint4 &x) {
        planes[(2 * c) * PS16 + cell] = make_uint2(x.x, x.y);
        planes[(2 * c + 1) * PS16 + cell] = make_uint2(x.z, x.w);
    }

    // Image elements of a tile's rows for the fused upsample (one per thread
    // and load).
    static constexpr int kThreadsPerBlock = 256;
    template <int NIN>
    struct Image {
        static constexpr int kElems = HY * kHaloW * NIN;
        static constexpr int kImg = (kElems + kThreadsPerBlock - 1) / kThreadsPerBlock;
        uint32_t e[kImg];
    };

    // Per-lane byte offsets of the fused-upsample loads within the coarse rows
    // and the image rows a tile may touch (kOut for unused slots and cells
    // outside the grid): like offsets(), they depend on the tile only and are
    // computed once per work item (the per-lane divisions by fx and fy no
    // longer run per plane).
    template <int NIN>
    struct UpOffsets {
        uint32_t o[kBodySlots + 1];
        uint32_t img[Image<NIN>::kImg];
    };
    template <int NIN>
    __device__ __forceinline__ static UpOffsets<NIN> up_offsets(int cdw, int fy, int fx, int dw,
                                                                int y0, int x0) {
        static_assert(C == kC, "the fused upsample serves C = 16");
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int gy0 = y0 - 1;
        const int base_row = gy0 > 0 ? gy0 : 0;
        const int cbase = base_row / fy;
        const uint32_t crow_bytes = (uint32_t)cdw * kCellBytes;
        const int cell = body_cell(lane);
        const uint32_t chunk_off = (uint32_t)body_chunk(lane) * 16;
        UpOffsets<NIN> r;
#pragma unroll
        for (int k = 0; k < kBodySlots; ++k) {
            const int J = wave + 4 * k;
            const int gy = gy0 + J / kBodyPerRow;
            const int cx = x0 + (J % kBodyPerRow) * kCellsPerBody + cell;
            const bool ok = J < kBody && gy >= 0 && cx < dw;
            const uint32_t off = (uint32_t)(gy / fy - cbase) * crow_bytes +
                                 (uint32_t)(cx / fx) * kCellBytes + chunk_off;
            r.o[k] = ok ? off : kOut;
        }
        {
            const int s = 3 - wave;
            const int row = s * kRowsPerSide + lane / (2 * NQ);
            const int gy = gy0 + row;
            const int gx = ((lane / NQ) & 1) ? x0 + kTileW : x0 - 1;
            const bool ok = s < kSide && row < HY && gy >= 0 && gx >= 0 && gx < dw;
            const uint32_t off = (uint32_t)(gy / fy - cbase) * crow_bytes +
                                 (uint32_t)(gx / fx) * kCellBytes + (uint32_t)(lane % NQ) * 16;
            r.o[kBodySlots] = ok ? off : kOut;
        }
        const uint32_t irow_bytes = (uint32_t)dw * NIN * (uint32_t)sizeof(T);
#pragma unroll
        for (int j = 0; j < Image<NIN>::kImg; ++j) {
            const int e = (int)threadIdx.x + kThreadsPerBlock * j;
            const int row = e / (kHaloW * NIN);
            const int rem = e - row * (kHaloW * NIN);
            const int gy = gy0 + row;
            const int gx = x0 - 1 + rem / NIN;
            const bool ok = e < Image<NIN>::kElems && gy >= 0 && gx >= 0 && gx < dw;
            const uint32_t off = (uint32_t)(gy - base_row) * irow_bytes +
                                 (uint32_t)(gx * NIN + rem % NIN) * (uint32_t)sizeof(T);
            r.img[j] = ok ? off : kOut;
        }
        return r;
    }

    // Upsample + inject fused into the load (3D first step of a level; fp16
    // planes): plane z, row gy and cell gx of the fine level come from the
    // coarse state's plane z / fz, row gy / fy and cell gx / fx; the NIN input
    // channels from the fine image, one element per thread and load, written
    // over channel quad 0 by commit_up_raw.  `of` holds the lane offsets of the
    // tile whose interior starts at (y0, x0) (from up_offsets()); rows outside
    // the grid and z outside [0, dd) read as zero through the descriptors'
    // ranges (the fine height is a multiple of fy, so a row below the grid
    // maps past the coarse rows covered).
    template <int NIN>
    __device__ __forceinline__ void issue_up(const T *__restrict__ coarse, int cdh, int cdw,
                                             int fz, int fy, const T *__restrict__ img,
                                             const UpOffsets<NIN> &of, Image<NIN> &im, int z,
                                             int dd, int dh, int dw, int y0, bool active = true) {
        const int gy0 = y0 - 1;
        const int base_row = gy0 > 0 ? gy0 : 0;
        const int rows =
            (active && z >= 0 && z < dd) ? max(0, min(gy0 + HY, dh) - base_row) : 0;
        // coarse rows base_row / fy .. (base_row + rows - 1) / fy of plane z / fz
        const int cbase = base_row / fy;
        const int crows = rows > 0 ? (base_row + rows - 1) / fy - cbase + 1 : 0;
        const uint32_t crow_bytes = (uint32_t)cdw * kCellBytes;
        const Rsrc r = make_rsrc(coarse + ((int64_t)(max(z, 0) / fz) * cdh + cbase) * cdw * C,
                                 (uint32_t)crows * crow_bytes);
#pragma unroll
        for (int k = 0; k <= kBodySlots; ++k) {
            const v4u x = __builtin_amdgcn_raw_buffer_load_b128(r, of.o[k], 0, 0);
            v[k] = make_uint4(x[0], x[1], x[2], x[3]);
        }
        const uint32_t irow_bytes = (uint32_t)dw * NIN * (uint32_t)sizeof(T);
        const Rsrc ri = make_rsrc(img + ((int64_t)max(z, 0) * dh + base_row) * dw * NIN,
                                  (uint32_t)rows * irow_bytes);
#pragma unroll
        for (int j = 0; j < Image<NIN>::kImg; ++j)
            im.e[j] = __builtin_amdgcn_raw_buffer_load_b16(ri, of.img[j], 0, 0);
    }

    // Called by every thread of the block: the coarse words of a cell and its
    // image channels are written by different waves, so a barrier orders them.
    template <int NIN>
    __device__ __forceinline__ void commit_up_raw(uint2 *planes, const Image<NIN> &im) const {
        commit_raw(planes);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < Image<NIN>::kImg; ++j) {
            const int e = (int)threadIdx.x + kThreadsPerBlock * j;
            const int row = e / (kHaloW * NIN);
            const int rem = e - row * (kHaloW * NIN);
            const int slot = e < Image<NIN>::kElems ? row * kHaloW + rem / NIN : kDummyCell;
            reinterpret_cast<unsigned short *>(planes + slot)[rem % NIN] =
                (unsigned short)im.e[j];   // channel quad plane 0
        }
    }

    __device__ __forceinline__ void commit_raw(uint2 *planes) const {
        static_assert(NQ == 2, "raw fp16 planes");
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int cell = body_cell(lane), chunk = body_chunk(lane);
#pragma unroll
        for (int k = 0; k < kBodySlots; ++k) {
            const int J = wave + 4 * k;
            const int slot =
                (J / kBodyPerRow) * kHaloW + 1 + (J % kBodyPerRow) * kCellsPerBody + cell;
            put_raw(planes, chunk, J < kBody ? slot : kDummyCell, v[k]);
        }
        const int s = 3 - wave;
        const int row = s * kRowsPerSide + lane / (2 * NQ);
        const int slot = row * kHaloW + (((lane / NQ) & 1) ? kHaloW - 1 : 0);
        put_raw(planes, lane % NQ, (s < kSide && row < HY) ? slot : kDummyCell, v[kBodySlots]);
    }
};

// Residual update and store of the lane's 4 channels (fp32 values, stored in
// the storage type) through the tile's store descriptor; `off` is the byte
// offset of the cell in it, or kOut for a cell outside the grid.  u is +0 for
// the input channels (zero W2 rows) and m is 0 for a cell that does not
// fire: then the fma returns the state bit for bit (u finite).
__device__ __forceinline__ void store_quad(float *, Rsrc w, uint32_t off, int g, const v4f &v) {
    const v4u x = {__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                   __float_as_uint(v[3])};
    __builtin_amdgcn_raw_buffer_store_b128(x, w, off == kOut ? kOut : off + 16u * g, 0, 0);
}
__device__ __forceinline__ void store_quad(__half *, Rsrc w, uint32_t off, int g, const v4f &v) {
    const v2u x = {Storage<__half>::pack_pair(v[0], v[1]), Storage<__half>::pack_pair(v[2], v[3])};
    __builtin_amdgcn_raw_buffer_store_b64(x, w, off == kOut ? kOut : off + 8u * g, 0, 0);
}

template <typename T>
__device__ __forceinline__ void update_store(T *tag, Rsrc w, uint32_t off, int g, const float f[8],
                                             const v4f &u, float m) {   // m: 1 fires, 0 keeps
    v4f out;
    out[0] = fmaf(m, u[0], f[0]);
    out[1] = fmaf(m, u[1], f[1]);
    out[2] = fmaf(m, u[2], f[2]);
    out[3] = fmaf(m, u[3], f[3]);
    store_quad(tag, w, off, g, out);
}

// Perception of channels 4g..4g+3 of the cell at LDS slot `centre`: the
// cell's own state in f[0..4), bias + taps in f[4..8).  `pl` points at the
// lane's channel-quad plane(s); tapw holds the conv weights as [tap][quad].
__device__ __forceinline__ void perceive_2d(const float4 *pl, const float4 (*tapw)[4], int g,
                                            int centre, const float cb[4], float f[8]) {
    const float4 sv = pl[centre];
    f[0] = sv.x; f[1] = sv.y; f[2] = sv.z; f[3] = sv.w;
    float p[4] = {cb[0], cb[1], cb[2], cb[3]};
#pragma unroll
    for (int t = 0; t < 9; ++t) {
        const float4 v = pl[centre + (t / 3 - 1) * kHaloW + (t % 3 - 1)];
        const float4 w = tapw[t][g];
        p[0] = fmaf(w.x, v.x, p[0]);
        p[1] = fmaf(w.y, v.y, p[1]);
        p[2] = fmaf(w.z, v.z, p[2]);
        p[3] = fmaf(w.w, v.w, p[3]);
    }
    f[4] = p[0]; f[5] = p[1]; f[6] = p[2]; f[7] = p[3];
}

// 3D: planes z-1, z, z+1 of the ring; taps in order (dz, dy, dx), one plane
// at a time (bounds the LDS values in flight and the registers).
__device__ __forceinline__ void perceive_3d(const float4 *pm, const float4 *pc, const float4 *pp,
                                            const float4 (*tapw)[4], int g, int centre,
                                            const float cb[4], float f[8]) {
    const float4 sv = pc[centre];
    f[0] = sv.x; f[1] = sv.y; f[2] = sv.z; f[3] = sv.w;
    float p[4] = {cb[0], cb[1], cb[2], cb[3]};
#pragma unroll 1
    for (int pz = 0; pz < 3; ++pz) {
        const float4 *pl = pz == 0 ? pm : pz == 1 ? pc : pp;
#pragma unroll
        for (int tt = 0; tt < 9; ++tt) {
            const float4 v = pl[centre + (tt / 3 - 1) * kHaloW + (tt % 3 - 1)];
            const float4 w = tapw[pz * 9 + tt][g];
            p[0] = fmaf(w.x, v.x, p[0]);
            p[1] = fmaf(w.y, v.y, p[1]);
            p[2] = fmaf(w.z, v.z, p[2]);
            p[3] = fmaf(w.w, v.w, p[3]);
        }
    }
    f[4] = p[0]; f[5] = p[1]; f[6] = p[2]; f[7] = p[3];
}

// ---------------------------------------------------------------------------
// 2D: persistent blocks loop over 16 x 32 tiles (tile index row-major); wave
// w computes rows 4w .. 4w+3 of the tile, 8 groups of 16 cells.
// ---------------------------------------------------------------------------
constexpr int k2TY = 16;
constexpr int k2BlocksPerCu = 2;   // 2 waves per SIMD: <= 256 VGPRs

template <typename T, int NIN, class Mlp>
__global__ __launch_bounds__(kThreads, k2BlocksPerCu) void nca_step_mfma_2d(
    const T *__restrict__ src, T *__restrict__ dst, int dh, int dw, int tiles_x, int tiles,
    const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold) {
    static_assert(Mlp::kChannels == kC && Mlp::kHidden == kH, "built for C = 16, H = 64");
    using Loader = RowLoader<T, k2TY + 2>;
    __shared__ float4 planes[4 * Loader::PS];
    __shared__ float4 tapw[9][4];       // [tap][quad] conv weights of channels 4q..4q+3

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int g = lane >> 4;

    {
        const int i = (int)threadIdx.x % (9 * 4);
        const int t = i / 4, q = i % 4;
        constexpr float ps = Mlp::kPerceptionScale;
        const float4 tw = make_float4(ps * conv_w[(4 * q + 0) * 9 + t], ps * conv_w[(4 * q + 1) * 9 + t],
                                      ps * conv_w[(4 * q + 2) * 9 + t], ps * conv_w[(4 * q + 3) * 9 + t]);
        tapw[t][q] = tw;   // threads >= 36 rewrite an entry (same value): no branch
    }
    Mlp mlp;
    mlp.load(w1, b1, w2, n, g, NIN);
    float cb[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) cb[k] = Mlp::kPerceptionScale * conv_b[4 * g + k];
    // all weight loads done before the tile loop (keeps the compiler's
    // vector-memory counting exact inside it)
    mlp.pin_all();
#pragma unroll
    for (int k = 0; k < 4; ++k) pin(cb[k]);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // Fire evaluations: a tile's 4 rows per wave take 4 * opr lanes, so one
    // evaluation serves 64 / (4 opr) consecutive tiles of this block (4 when
    // rows are 8-aligned, else 2).
    FireBits fire;
    fire.aligned = (dw & 7) == 0;
    fire.opr = fire.aligned ? 4 : 8;
    const int lg_opr = fire.aligned ? 2 : 3;
    const int tiles_per_eval = 64 / (4 * fire.opr);
    const int stride = (int)gridDim.x;
    constexpr int kCellBytes = Loader::kCellBytes;
    const uint32_t row_bytes = (uint32_t)dw * kCellBytes;

    // The tile's halo is in LDS when an iteration starts: the first tile is
    // staged here, each later one is loaded during the previous iteration's
    // compute and written to LDS at its end (so every wait for those loads
    // sees the same history of memory operations).
    Loader ld;
    int tile = blockIdx.x;
    if (tile < tiles) {
        const int ty = tile / tiles_x;
        ld.issue(src, 0, 1, dh, dw, ty * k2TY, (tile - ty * tiles_x) * kTileW);
        ld.commit(planes);
    }
    for (int iter = 0; tile < tiles; tile += stride, ++iter) {
        const int ty = tile / tiles_x;
        const int y0 = ty * k2TY, x0 = (tile - ty * tiles_x) * kTileW;
        const int phase = iter & (tiles_per_eval - 1);
        if (phase == 0) {
            // lane -> (tile offset, row r of the wave's 4, block o of the row)
            const int tt = lane >> (lg_opr + 2);
            int t2 = tile + tt * stride;
            t2 = t2 < tiles ? t2 : tile;
            const int ty2 = t2 / tiles_x;
            const uint64_t row = (uint64_t)(ty2 * k2TY + 4 * wave + ((lane >> lg_opr) & 3));
            const uint64_t b0 = (row * dw + (uint64_t)(t2 - ty2 * tiles_x) * kTileW) >> 3;
            fire.f = fire_ballots(b0 + (lane & (fire.opr - 1)), step, level, batch, seed, threshold);
            fire.mine = select_ballot(fire.f, (uint32_t)n & 7u);
        }
        const int slot0 = phase * 4;
        __syncthreads();
        {
            const int next = tile + stride;
            const bool more = next < tiles;
            const int nt = more ? next : tile;
            const int nty = nt / tiles_x;
            ld.issue(src, 0, 1, dh, dw, nty * k2TY, (nt - nty * tiles_x) * kTileW, more);
        }

        // stores of this tile: rows y0 .. y0 + k2TY - 1 (clipped to the grid)
        const Rsrc wr = make_rsrc(dst + (int64_t)y0 * dw * kC,
                                  (uint32_t)min(k2TY, dh - y0) * row_bytes);
        // groups are software-pipelined: group grp + 1's perception is issued
        // while group grp's first-layer MFMAs run
        const float4 *pl = planes + g * Loader::PS;
        auto centre_of = [&](int grp) {
            return (4 * wave + (grp >> 1) + 1) * kHaloW + (grp & 1) * 16 + n + 1;
        };
        float f[8];
        perceive_2d(pl, tapw, g, centre_of(0), cb, f);
        // fully unrolled: with a counted sequence of stores the compiler can
        // wait for the prefetched loads alone (stores share the vector-memory
        // counter), instead of draining every store of the tile
#pragma unroll
        for (int grp = 0; grp < 8; ++grp) {
            v4f acc[4];
            mlp.layer1(f, acc);
            float fn[8];
            if (grp < 7) perceive_2d(pl, tapw, g, centre_of(grp + 1), cb, fn);
            const v4f u = mlp.layer2(acc);

            const int r = grp >> 1;                 // row slot within the wave
            const int ly = 4 * wave + r;
            const int y = y0 + ly, x = x0 + (grp & 1) * 16 + n;
            const uint64_t idx = (uint64_t)y * dw + x;
            const uint64_t row_b0 = ((uint64_t)y * dw + x0) >> 3;
            const uint32_t off = x < dw ? (uint32_t)ly * row_bytes + (uint32_t)x * kCellBytes : kOut;
            update_store(dst, wr, off, g, f, u, fire.bit(slot0 + r, idx, row_b0));
#pragma unroll
            for (int k = 0; k < 8; ++k) f[k] = fn[k];
            // keep the scheduler from interleaving whole groups (register pressure)
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
        ld.commit(planes);   // the next tile (zeros when there is none)
    }
}

// ---------------------------------------------------------------------------
// 2D, row streaming: a block is one wave, and a work item is a 32-cell-wide
// strip of a run of rows.  The wave streams the strip's halo rows (34 cells)
// through a private ring of four LDS row slots, so no block barrier is
// needed (LDS accesses of one wave complete in order).  Each input row q is
// read once: its 3 taps along x feed three rolling perception sums per
// 16-cell group, for outputs q + 1 (the dy = -1 weights), q (dy = 0) and
// q - 1 (dy = +1).  After row q the sum of output q - 1 is complete and that
// row's MLP, fire gate and store run, with the cell's own state re-read from
// the ring.  An iteration takes two input rows; the loads of the next two are
// issued at its start and written to LDS at its end.
// ---------------------------------------------------------------------------
constexpr int k2RunRows = 128;      // output rows per work item
constexpr int k2WavesPerSimd = 2;   // 255 VGPRs with the split-bf16 MLP

// The row kernels' conv weights: tapw[t][q] = the tap-t weights of channels
// 4q..4q+3 and cb = the bias of the lane's channel quad, both times the MLP's
// perception scale (Sec. 3.1: one 3x3 filter and bias per channel).  Quads
// >= C / 4 (quad 3 of a C = 12 model) are zero; their indices are clamped and
// the values replaced, so every lane loads.
template <int C>
__device__ __forceinline__ void load_conv_2d(const float *__restrict__ conv_w,
                                             const float *__restrict__ conv_b, float ps,
                                             float4 (*tapw)[4], float cb[4]) {
    const int lane = threadIdx.x & 63;
    const int i = lane % (9 * 4);
    const int t = i / 4, q = i % 4;
    const bool q_ok = q < C / 4;
    const int qc = q_ok ? q : 0;
    const float4 tw = make_float4(ps * conv_w[(4 * qc + 0) * 9 + t], ps * conv_w[(4 * qc + 1) * 9 + t],
                                  ps * conv_w[(4 * qc + 2) * 9 + t], ps * conv_w[(4 * qc + 3) * 9 + t]);
    const int g = lane >> 4;
    const bool g_ok = g < C / 4;
    const int gc = g_ok ? g : 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) cb[k] = g_ok ? ps * conv_b[4 * gc + k] : 0.f;
    // lanes >= 36 write an entry again with the same value: no branch, so the
    // loads above are not sunk behind one and wait once together
    tapw[t][q] = q_ok ? tw : make_float4(0.f, 0.f, 0.f, 0.f);
}

// One halo row of a strip: kBody body loads (16 cells x 4 chunks in fp32,
// 32 cells x 2 chunks in fp16, lane i -> cell i % cells-per-load, chunk
// i / cells-per-load) and one side load whose first 2 NQ lanes take the left
// and right halo cells.  Cells outside the grid and rows outside [0, h) read
// as zero through an out-of-range offset or an empty descriptor.  A cell of C
// channels fills kChunks of the NQ chunks; the others (channel quad 3 when
// C = 12) read as zero the same way, so the ring holds the cell padded to 16
// channels with zeros.
template <typename T, int C = kC>
struct RowStream {
    static constexpr int NQ = CellChunks<T>::N;
    static constexpr int kCellBytes = C * (int)sizeof(T);
    static constexpr int kChunks = kCellBytes / 16;
    static_assert(kCellBytes % 16 == 0 && kChunks <= NQ, "whole 16-byte chunks");
    static constexpr int kCellsPerBody = 64 / NQ;
    static constexpr int kBody = kTileW / kCellsPerBody;
    static constexpr int kDummy = kHaloW;                 // never-read slot
    static constexpr int PS = plane_stride(kHaloW + 1);   // quad plane stride (16-byte words)
    static constexpr int kSlotWords = 4 * PS;             // one ring slot
    uint4 v[kBody + 1];

    __device__ __forceinline__ void issue(const T *__restrict__ src, int y, int dh, int dw, int x0) {
        const int lane = threadIdx.x & 63;
        const bool row_ok = y >= 0 && y < dh;
        const Rsrc r = make_rsrc(src + (int64_t)(row_ok ? y : 0) * dw * C,
                                 row_ok ? (uint32_t)dw * kCellBytes : 0u);
        const int cell = lane % kCellsPerBody, chunk = lane / kCellsPerBody;
#pragma unroll
        for (int k = 0; k < kBody; ++k) {
            const int cx = x0 + k * kCellsPerBody + cell;
            const uint32_t off = chunk < kChunks && cx >= 0 && cx < dw
                                     ? (uint32_t)cx * kCellBytes + (uint32_t)chunk * 16
                                     : kOut;
            const v4u x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
            v[k] = make_uint4(x[0], x[1], x[2], x[3]);
        }
        const int cx = lane < NQ ? x0 - 1 : x0 + kTileW;
        const bool ok = lane < 2 * NQ && lane % NQ < kChunks && cx >= 0 && cx < dw;
        const uint32_t off = ok ? (uint32_t)cx * kCellBytes + (uint32_t)(lane % NQ) * 16 : kOut;
        const v4u x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
        v[kBody] = make_uint4(x[0], x[1], x[2], x[3]);
    }

    // LDS: four channel-quad planes of PS 16-byte words, fp32; slot 0 is the
    // left halo cell, 1..32 the strip, 33 the right halo cell.
    __device__ static __forceinline__ void put(float4 *planes, int q, int slot, const uint4 &c) {
        if constexpr (NQ == 4) {
            planes[q * PS + slot] = make_float4(__uint_as_float(c.x), __uint_as_float(c.y),
                                                __uint_as_float(c.z), __uint_as_float(c.w));
        } else {
            float f[8];
            Storage<__half>::unpack(c, f);
            planes[(2 * q) * PS + slot] = make_float4(f[0], f[1], f[2], f[3]);
            planes[(2 * q + 1) * PS + slot] = make_float4(f[4], f[5], f[6], f[7]);
        }
    }

    __device__ __forceinline__ void commit(float4 *planes) const {
        const int lane = threadIdx.x & 63;
        const int cell = lane % kCellsPerBody, chunk = lane / kCellsPerBody;
#pragma unroll
        for (int k = 0; k < kBody; ++k) put(planes, chunk, 1 + k * kCellsPerBody + cell, v[k]);
        const int slot = lane < NQ ? 0 : (lane < 2 * NQ ? kHaloW - 1 : kDummy);
        put(planes, lane % NQ, slot, v[kBody]);
    }

    // Upsample + inject fused into the load (Sec. 3.2; supplement S6): fine row
    // y comes from the coarse state's row y / fy, cell x from coarse cell x / fx,
    // and the NIN input channels from the fine image's row y (one image element
    // per lane, kImg loads).  commit_up writes the coarse cells like commit()
    // and then overwrites the input channels (all in channel quad 0) with the
    // image values, so the ring holds exactly the upsampled fine state.
    template <int NIN>
    struct Image {
        static constexpr int kElems = kHaloW * NIN;
        static constexpr int kImg = (kElems + 63) / 64;
        uint32_t e[kImg];
    };

    template <int NIN>
    __device__ __forceinline__ void issue_up(const T *__restrict__ coarse, int cdw, int fy,
                                             int fx, const T *__restrict__ img, Image<NIN> &im,
                                             int y, int dh, int dw, int x0) {
        const int lane = threadIdx.x & 63;
        const bool row_ok = y >= 0 && y < dh;
        const Rsrc r = make_rsrc(coarse + (int64_t)(row_ok ? y / fy : 0) * cdw * C,
                                 row_ok ? (uint32_t)cdw * kCellBytes : 0u);
        const int cell = lane % kCellsPerBody, chunk = lane / kCellsPerBody;
#pragma unroll
        for (int k = 0; k < kBody; ++k) {
            const int cx = x0 + k * kCellsPerBody + cell;
            const uint32_t off = chunk < kChunks && cx >= 0 && cx < dw
                                     ? (uint32_t)(cx / fx) * kCellBytes + (uint32_t)chunk * 16
                                     : kOut;
            const v4u x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
            v[k] = make_uint4(x[0], x[1], x[2], x[3]);
        }
        {
            const int cx = lane < NQ ? x0 - 1 : x0 + kTileW;
            const bool ok = lane < 2 * NQ && lane % NQ < kChunks && cx >= 0 && cx < dw;
            const uint32_t off =
                ok ? (uint32_t)(cx / fx) * kCellBytes + (uint32_t)(lane % NQ) * 16 : kOut;
            const v4u x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
            v[kBody] = make_uint4(x[0], x[1], x[2], x[3]);
        }
        const Rsrc ri = make_rsrc(img + (int64_t)(row_ok ? y : 0) * dw * NIN,
                                  row_ok ? (uint32_t)dw * NIN * (uint32_t)sizeof(T) : 0u);
#pragma unroll
        for (int j = 0; j < Image<NIN>::kImg; ++j) {
            const int e = lane + 64 * j;
            const int fc = x0 - 1 + e / NIN;
            const bool ok = e < Image<NIN>::kElems && fc >= 0 && fc < dw;
            const uint32_t off = ok ? (uint32_t)(fc * NIN + e % NIN) * (uint32_t)sizeof(T) : kOut;
            if constexpr (sizeof(T) == 4)
                im.e[j] = __builtin_amdgcn_raw_buffer_load_b32(ri, off, 0, 0);
            else
                im.e[j] = __builtin_amdgcn_raw_buffer_load_b16(ri, off, 0, 0);
        }
    }

    template <int NIN>
    __device__ __forceinline__ void commit_up(float4 *planes, const Image<NIN> &im) const {
        commit(planes);
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int j = 0; j < Image<NIN>::kImg; ++j) {
            const int e = lane + 64 * j;
            const int slot = e < Image<NIN>::kElems ? e / NIN : kDummy;
            float val;
            if constexpr (sizeof(T) == 4)
                val = __uint_as_float(im.e[j]);
            else
                val = __half2float(__ushort_as_half((unsigned short)im.e[j]));
            reinterpret_cast<float *>(planes + slot)[e % NIN] = val;   // quad plane 0
        }
    }
};

// UP: the step's input is not a state of this level but the next coarser
// level's state (src, width up_cdw) upsampled by (up_fy, up_fx) with the input
// channels taken from up_img (the first step of a level, fused with the
// upsample + inject).
template <typename T, int NIN, class Mlp, bool ALIGNED, bool UP>
__global__ __launch_bounds__(64, k2WavesPerSimd) void nca_step_mfma_2d_rows(
    const T *__restrict__ src, T *__restrict__ dst, int dh, int dw, int strips, int runs,
    int run_rows, int items, const float *__restrict__ conv_w,
    const float *__restrict__ conv_b, const float *__restrict__ w1, const float *__restrict__ b1,
    const float *__restrict__ w2, uint32_t level, uint32_t step, uint32_t batch, uint64_t seed,
    uint64_t threshold, const T *__restrict__ up_img, int up_cdw, int up_fy, int up_fx) {
    constexpr int C = Mlp::kChannels;
    using RS = RowStream<T, C>;
    __shared__ float4 ring[4][RS::kSlotWords];   // row y in slot y & 3
    __shared__ float4 tapw[9][4];                // [tap][quad] conv weights of channels 4q..4q+3

    const int lane = threadIdx.x & 63;
    const int n = lane & 15;
    const int g = lane >> 4;

    Mlp mlp;
    mlp.load(w1, b1, w2, n, g, NIN);
    float cb[4];
    load_conv_2d<C>(conv_w, conv_b, Mlp::kPerceptionScale, tapw, cb);
    mlp.pin_all();
#pragma unroll
    for (int k = 0; k < 4; ++k) pin(cb[k]);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // Fire evaluations: a row takes opr lanes, so one evaluation serves
    // 64 / opr consecutive output rows (16 when rows are 8-aligned, else 8).
    // ALIGNED (w % 8 == 0): a lane's cells always take ballot n % 8 at bit
    // offset 2 grp + n / 8 within their row's slot.
    FireBits fire;
    fire.aligned = ALIGNED;
    fire.opr = ALIGNED ? 4 : 8;
    constexpr int lg_opr = ALIGNED ? 2 : 3;
    constexpr int rows_per_eval = ALIGNED ? 16 : 8;
    constexpr int kCellBytes = RS::kCellBytes;
    const uint32_t row_bytes = (uint32_t)dw * kCellBytes;
    int gq = g;
    RS ra, rb;
    typename RS::template Image<NIN> ia, ib;   // used by UP only
    // Rows at or beyond y_lim (the run's last input row + 1, or the grid's
    // height) read as zero through an empty descriptor, without a memory access.
    int y_lim = dh;
    auto issue = [&](RS &rs, typename RS::template Image<NIN> &im, int y, int x0) {
        if constexpr (UP)
            rs.template issue_up<NIN>(src, up_cdw, up_fy, up_fx, up_img, im, y, y_lim, dw, x0);
        else
            rs.issue(src, y, y_lim, dw, x0);
    };
    auto commit = [&](const RS &rs, const typename RS::template Image<NIN> &im, float4 *slot) {
        if constexpr (UP)
            rs.template commit_up<NIN>(slot, im);
        else
            rs.commit(slot);
    };

    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        const int sx = item % strips;
        const int ry = item / strips;
        const int x0 = sx * kTileW;
        const int y_begin = ry * run_rows;
        const int y_end = min(dh, y_begin + run_rows);
        y_lim = min(dh, y_end + 1);   // input rows y_begin - 1 .. y_end feed the run

        // rolling perception sums (bias included) of outputs q - 1, q, q + 1
        float acc_p[2][4], acc_c[2][4], acc_n[2][4];
#pragma unroll
        for (int grp = 0; grp < 2; ++grp)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                acc_p[grp][k] = cb[k];
                acc_c[grp][k] = cb[k];
                acc_n[grp][k] = cb[k];
            }

        // Input row q with its x taps: output q + 1 takes the dy = -1 weights,
        // q the dy = 0 ones and q - 1 the dy = +1 ones.
        auto fold_row = [&](int q) {
            const float4 *pl = ring[q & 3] + g * RS::PS;
            pin(gq);   // re-read the tap weights every row instead of keeping 36 registers
#pragma unroll
            for (int dx = 0; dx < 3; ++dx) {
                const float4 wm = tapw[dx][gq];
                const float4 w0 = tapw[3 + dx][gq];
                const float4 wp = tapw[6 + dx][gq];
                const float a_m[4] = {wm.x, wm.y, wm.z, wm.w};
                const float a_0[4] = {w0.x, w0.y, w0.z, w0.w};
                const float a_p[4] = {wp.x, wp.y, wp.z, wp.w};
#pragma unroll
                for (int grp = 0; grp < 2; ++grp) {
                    const float4 v = pl[grp * 16 + n + dx];
                    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        acc_n[grp][k] = fmaf(a_m[k], vv[k], acc_n[grp][k]);
                        acc_c[grp][k] = fmaf(a_0[k], vv[k], acc_c[grp][k]);
                        acc_p[grp][k] = fmaf(a_p[k], vv[k], acc_p[grp][k]);
                    }
                }
            }
        };

        // Fire bits of output rows yo .. yo + rows_per_eval - 1.
        auto evaluate_fire = [&](int yo) {
            const int yy = min(yo + (lane >> lg_opr), dh - 1);
            const uint64_t b0 = ((uint64_t)yy * dw + x0) >> 3;
            fire.f = fire_ballots(b0 + (lane & (fire.opr - 1)), step, level, batch, seed, threshold);
            fire.mine = select_ballot(fire.f, (uint32_t)n & 7u);
        };

        // The sums shift by one row: output q + 1 becomes the next to finish.
        auto shift = [&]() {
#pragma unroll
            for (int grp = 0; grp < 2; ++grp)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    acc_p[grp][k] = acc_c[grp][k];
                    acc_c[grp][k] = acc_n[grp][k];
                    acc_n[grp][k] = cb[k];
                }
        };

        // Output row yo (complete in acc_p): MLP, fire gate and store of its
        // two groups; stores of rows outside [y_begin, y_end) are dropped by an
        // empty descriptor.  Then the sums shift by one row.
        auto finish_row = [&](int yo) {
            const bool out_ok = yo >= y_begin && yo < y_end;
            const int phase = (yo - y_begin) & (rows_per_eval - 1);
            if (out_ok && phase == 0 && yo != y_begin) evaluate_fire(yo);
            const int yc = max(yo, 0);
            const Rsrc wr = make_rsrc(dst + (int64_t)yc * dw * C, out_ok ? row_bytes : 0u);
            const float4 *own = ring[yo & 3] + g * RS::PS;
            const uint64_t row_b0 = ((uint64_t)yc * dw + x0) >> 3;
            v4f acc[2][4];
            float f[2][8];
#pragma unroll
            for (int grp = 0; grp < 2; ++grp) {
                const float4 sp = own[1 + grp * 16 + n];
                f[grp][0] = sp.x; f[grp][1] = sp.y; f[grp][2] = sp.z; f[grp][3] = sp.w;
#pragma unroll
                for (int k = 0; k < 4; ++k) f[grp][4 + k] = acc_p[grp][k];
                mlp.layer1(f[grp], acc[grp]);
            }
#pragma unroll
            for (int grp = 0; grp < 2; ++grp) {
                const v4f u = mlp.layer2(acc[grp]);
                const int x = x0 + grp * 16 + n;
                const uint32_t off = x < dw && g < C / 4 ? (uint32_t)x * kCellBytes : kOut;
                bool fires;
                if constexpr (ALIGNED) {
                    fires = (fire.mine >> (phase * 4 + 2 * grp + (n >> 3))) & 1;
                } else {
                    const uint64_t idx = (uint64_t)yc * dw + x;
                    fires = fire.bit(phase, idx, row_b0);
                }
                update_store(dst, wr, off, g, f[grp], u, fires);
            }
            shift();
        };

        // Rows y_begin - 1 and y_begin into the ring, y_begin + 1 and
        // y_begin + 2 in flight while they are folded; outputs y_begin - 2 and
        // y_begin - 1, which they complete, are outside the run (not computed).
        // The run's first fire evaluation runs while the first rows load.
        issue(ra, ia, y_begin - 1, x0);
        issue(rb, ib, y_begin, x0);
        evaluate_fire(y_begin);
        commit(ra, ia, ring[(y_begin - 1) & 3]);
        commit(rb, ib, ring[y_begin & 3]);
        issue(ra, ia, y_begin + 1, x0);
        issue(rb, ib, y_begin + 2, x0);
        fold_row(y_begin - 1);
        shift();
        fold_row(y_begin);
        shift();
        commit(ra, ia, ring[(y_begin + 1) & 3]);
        commit(rb, ib, ring[(y_begin + 2) & 3]);

        // input rows q, q + 1 per iteration, from y_begin + 1 through y_end
        // (plus one padding row when the count is odd)
        for (int q = y_begin + 1; q <= y_end; q += 2) {
            issue(ra, ia, q + 2, x0);
            issue(rb, ib, q + 3, x0);
            fold_row(q);
            finish_row(q - 1);
            __builtin_amdgcn_sched_barrier(0);
            fold_row(q + 1);
            finish_row(q);
            __builtin_amdgcn_sched_barrier(0);
            commit(ra, ia, ring[(q + 2) & 3]);
            commit(rb, ib, ring[(q + 3) & 3]);
        }
    }
}

// ---------------------------------------------------------------------------
// 2D, two steps per launch (temporal fusion).  The fire mask is a function of
// (seed, level, step, cell) alone, so a wave can run step t + 1 on its own
// copy of step t's result.  Same row streaming as nca_step_mfma_2d_rows, with
// the strip narrowed to 30 output cells: the wave loads 34-cell halo rows
// (cells x0 - 2 .. x0 + 31), runs step t on the 32 cells x0 - 1 .. x0 + 30 and
// writes each finished row into a second LDS ring of two slots (cells and
// rows outside the grid as 0: the zero padding of step t + 1's perception).
// Step t + 1 folds those rows into its own rolling sums and finishes cells
// x0 .. x0 + 31, of which x0 .. x0 + 29 are stored (the last two lack their
// right neighbours).  Per input row q: step t folds q and finishes q - 1, then
// step t + 1 folds q - 1; its row q - 2, complete then, is finished in the
// next row's body, next to step t's fold.  The state between the two steps
// never reaches HBM, so HBM sees one read and one write of the state per two
// steps, for 32/30 of the MLP work and 2 halo rows of step t per run; the
// results equal two single-step launches bit for bit (the same operations in
// the same order).
// ---------------------------------------------------------------------------
constexpr int k2PairW = kTileW - 2;   // output cells per strip

// UP: step t is a level's first step, fused with the upsample + inject as in
// nca_step_mfma_2d_rows (src is the next coarser state, width up_cdw, factors
// up_fy, up_fx; the input channels come from up_img).  SEG: the launch also
// writes the two-class readout of its result (Sec. 3.2) to seg: the lanes of
// channel quad 3 hold channels 12..15 of their cell, and its byte is 1 iff
// channel C - 1 > channel C - 2 (ties and NaNs give 0), the readout kernel's
// rule; the finest level's last launch uses it.
template <typename T, int NIN, class Mlp, bool UP, bool SEG>
__global__ __launch_bounds__(64, k2WavesPerSimd) void nca_step2_mfma_2d_rows(
    const T *__restrict__ src, T *__restrict__ dst, int dh, int dw, int strips, int run_rows,
    int items, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold,
    const T *__restrict__ up_img, int up_cdw, int up_fy, int up_fx, uint8_t *__restrict__ seg) {
    static_assert(std::is_same_v<T, float>, "the intermediate ring holds fp32 states");
    constexpr int C = Mlp::kChannels;
    using RS = RowStream<T, C>;
    // Row r of a work item (first input row `base`) lives in slot
    // (r - base) % 3 of the input ring and (r - base) % 2 of the ring of step
    // t's output rows.
    __shared__ float4 ring[3][RS::kSlotWords];
    __shared__ float4 mid[2][RS::kSlotWords];
    __shared__ float4 tapw[9][4];                // [tap][quad] conv weights of channels 4q..4q+3
    // Fire bits of the work item, [step t / t + 1][row]: byte o of a row's
    // word holds the 8 draws of the o-th block of 8 cells from the block that
    // contains the row's first strip cell.
    constexpr int kOpr = 5, kEvalRows = 12;
    constexpr int kEvalBlocks = (k2RunRows + 2 + kEvalRows - 1) / kEvalRows;
    constexpr int kMaskRows = kEvalBlocks * kEvalRows;
    __shared__ uint64_t fire_rows[2][kMaskRows];
    // The same words shifted once per work item so that bit c is the draw of
    // strip cell c (x0 - 1 + c for step t, x0 + c for step t + 1): a lane's
    // bit is then one bit-field extract.
    __shared__ uint32_t fire_bits[2][kMaskRows];

    const int lane = threadIdx.x & 63;
    const int n = lane & 15;
    const int g = lane >> 4;

    // Slots 32 and 33 of the step-t ring are never written: the two cells
    // per quad that step t + 1 computes but does not store read them.
    if (lane < 16) mid[lane >> 3][((lane >> 1) & 3) * RS::PS + 32 + (lane & 1)] = make_float4(0.f, 0.f, 0.f, 0.f);
    Mlp mlp;
    mlp.load(w1, b1, w2, n, g, NIN);
    float cb[4];
    load_conv_2d<C>(conv_w, conv_b, Mlp::kPerceptionScale, tapw, cb);
    mlp.pin_all();
#pragma unroll
    for (int k = 0; k < 4; ++k) pin(cb[k]);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // Fire evaluations: a strip row spans at most 5 blocks of 8 cells (it may
    // start anywhere within a block), so an evaluation gives 5 lanes to each of
    // 12 rows of one step (lanes 60..63 repeat row 11).  All evaluations of a
    // work item run at its start, where few registers are live; each lane
    // writes the 8 fire bits of its block as one byte of its row's word.
    const int ev_row = min(lane / kOpr, kEvalRows - 1), ev_blk = lane % kOpr;
    auto evaluate = [&](int s, int blk, uint32_t st, int y_first, uint32_t xs) {
        const int yy = min(max(y_first + ev_row, 0), dh - 1);
        const uint64_t b0 = (((uint64_t)yy * dw + xs) >> 3) + ev_blk;
        const Philox4x64Out r = philox4x64_10(b0, st, level, batch, seed, 0);
        uint32_t bits = 0;
#pragma unroll
        for (int c = 0; c < 8; ++c) bits |= ((uint64_t)draw_of(r, (uint32_t)c) < threshold ? 1u : 0u) << c;
        reinterpret_cast<uint8_t *>(&fire_rows[s][blk * kEvalRows + ev_row])[ev_blk] = (uint8_t)bits;
    };
    // Fire bit of strip cell c (c = x - xs >= 0) in row `rel` (rows from the
    // step's first row) of step s, whose row starts at canonical index rowc:
    // bit c + ((rowc + xs) & 7) of the row's word in fire_rows, bit c of its
    // word in fire_bits.  2D cell indices fit 32 bits (two fp32 states of
    // 2^32 cells would need 512 GB).  Rows outside the step's range read some
    // in-range word.
    auto row_bits = [&](int s, int rel) {
        return fire_bits[s][min(max(rel, 0), kMaskRows - 1)];
    };
    constexpr int kCellBytes = RS::kCellBytes;
    const uint32_t row_bytes = (uint32_t)dw * kCellBytes;
    int gq = g;
    RS ra, rb;
    using Img = typename RS::template Image<NIN>;
    Img ia, ib;   // used by UP only
    // UP: the lane's byte offsets within a coarse row and an image row, the
    // same for every row of a work item (computed once per item).
    struct UpCols {
        uint32_t body[RS::kBody], side, img[Img::kImg];
    } uc;
    auto up_cols = [&](int x) {
        const int lane = threadIdx.x & 63;
        const int cell = lane % RS::kCellsPerBody, chunk = lane / RS::kCellsPerBody;
#pragma unroll
        for (int kk = 0; kk < RS::kBody; ++kk) {
            const int cx = x + kk * RS::kCellsPerBody + cell;
            uc.body[kk] = chunk < RS::kChunks && cx >= 0 && cx < dw
                              ? (uint32_t)(cx / up_fx) * kCellBytes + (uint32_t)chunk * 16 : kOut;
        }
        const int cx = lane < RS::NQ ? x - 1 : x + kTileW;
        uc.side = lane < 2 * RS::NQ && lane % RS::NQ < RS::kChunks && cx >= 0 && cx < dw
                      ? (uint32_t)(cx / up_fx) * kCellBytes + (uint32_t)(lane % RS::NQ) * 16 : kOut;
#pragma unroll
        for (int j = 0; j < Img::kImg; ++j) {
            const int e = lane + 64 * j;
            const int fc = x - 1 + e / NIN;
            uc.img[j] = e < Img::kElems && fc >= 0 && fc < dw
                            ? (uint32_t)(fc * NIN + e % NIN) * (uint32_t)sizeof(T) : kOut;
        }
    };
    // Fine row y of the upsampled state: coarse row cy = y / fy, image row y.
    // The loop passes cy kept by counting (a division per row in the unrolled
    // loop made the compiler spill).
    auto issue = [&](RS &rs, Img &im, int y, int cy, int x) {
        if constexpr (UP) {
            const bool row_ok = y >= 0 && y < dh;
            const Rsrc r = make_rsrc(src + (int64_t)(row_ok ? cy : 0) * up_cdw * C,
                                     row_ok ? (uint32_t)up_cdw * kCellBytes : 0u);
#pragma unroll
            for (int kk = 0; kk < RS::kBody; ++kk) {
                const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, uc.body[kk], 0, 0);
                rs.v[kk] = make_uint4(v[0], v[1], v[2], v[3]);
            }
            const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, uc.side, 0, 0);
            rs.v[RS::kBody] = make_uint4(v[0], v[1], v[2], v[3]);
            const Rsrc ri = make_rsrc(up_img + (int64_t)(row_ok ? y : 0) * dw * NIN,
                                      row_ok ? (uint32_t)dw * NIN * (uint32_t)sizeof(T) : 0u);
#pragma unroll
            for (int j = 0; j < Img::kImg; ++j)
                im.e[j] = __builtin_amdgcn_raw_buffer_load_b32(ri, uc.img[j], 0, 0);
        } else {
            rs.issue(src, y, dh, dw, x);
        }
    };
    auto commit = [&](const RS &rs, const Img &im, float4 *slot) {
        if constexpr (UP)
            rs.template commit_up<NIN>(slot, im);
        else
            rs.commit(slot);
    };

    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        const int sx = item % strips;
        const int ry = item / strips;
        const int x0 = sx * k2PairW;
        const int x1 = x0 - 1;             // first cell of step t's strip
        const uint32_t xs1 = (uint32_t)max(x1, 0);
        const int y_begin = ry * run_rows;
        const int y_end = min(dh, y_begin + run_rows);
        const int x_stop = min(dw, x0 + k2PairW);
        const int base = y_begin - 2;      // first input row

        // Rolling perception sums (bias included): A[(r - base) % 3] holds
        // step t's sum of output row r, B[(r - base) % 3] step t + 1's.  The
        // loop body is unrolled three times, so the three sums of a step
        // rotate roles without register moves.
        float A[3][2][4], B[3][2][4];

        if constexpr (UP) up_cols(x1);
        issue(ra, ia, base, base >= 0 ? base / up_fy : 0, x1);
        issue(rb, ib, base + 1, base + 1 >= 0 ? (base + 1) / up_fy : 0, x1);
        // coarse row and remainder of the next row the loop loads (y_begin >= 0)
        int up_cy = y_begin / up_fy, up_ry = y_begin - up_cy * up_fy;
        // step t's rows y_begin - 1 .. y_end, step t + 1's y_begin .. y_end - 1
        for (int e = 0; e < 2 * kEvalBlocks; ++e) {
            const int st = e >= kEvalBlocks ? 1 : 0;
            const int blk = e - st * kEvalBlocks;
            const int y_first = y_begin - 1 + st + blk * kEvalRows;
            if (y_first <= y_end - st)
                evaluate(st, blk, step + st, y_first, st ? (uint32_t)x0 : xs1);
        }
        // Align each row's word to the strip: step t's strip starts at x1
        // (x1 = -1 on the first strip, whose cell 0 is outside the grid and
        // gets bit 0, unused), step t + 1's at x0.  A word spans the 5 blocks
        // of 8 cells that hold cells xs .. xs + 31, so bits sh .. sh + 31 with
        // sh <= 7 are inside it.
        for (int i = lane; i < 2 * kMaskRows; i += 64) {
            const int s = i >= kMaskRows ? 1 : 0;
            const int rel = i - s * kMaskRows;
            const int yo = y_begin - 1 + s + rel;
            const uint32_t rowc = (uint32_t)min(max(yo, 0), dh - 1) * (uint32_t)dw;
            const int sh = s ? (int)((rowc + (uint32_t)x0) & 7u)
                             : (int)((rowc + xs1) & 7u) + (x1 - (int)xs1);
            fire_bits[s][rel] = (uint32_t)((fire_rows[s][rel] << 1) >> (sh + 1));
        }
        commit(ra, ia, ring[0]);
        commit(rb, ib, ring[1]);

        // Row r of a plane set with its x taps: output r + 1 takes the dy = -1
        // weights (its first contribution, started from the bias), r the
        // dy = 0 ones and r - 1 the dy = +1 ones (its last).
        auto fold = [&](const float4 *pl, float (&first)[2][4], float (&second)[2][4],
                        float (&last)[2][4]) {
            pin(gq);   // re-read the tap weights every row instead of keeping 36 registers
#pragma unroll
            for (int dx = 0; dx < 3; ++dx) {
                const float4 wm = tapw[dx][gq];
                const float4 w0 = tapw[3 + dx][gq];
                const float4 wp = tapw[6 + dx][gq];
                const float a_m[4] = {wm.x, wm.y, wm.z, wm.w};
                const float a_0[4] = {w0.x, w0.y, w0.z, w0.w};
                const float a_p[4] = {wp.x, wp.y, wp.z, wp.w};
#pragma unroll
                for (int grp = 0; grp < 2; ++grp) {
                    const float4 v = pl[grp * 16 + n + dx];
                    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        first[grp][k] = fmaf(a_m[k], vv[k], dx == 0 ? cb[k] : first[grp][k]);
                        second[grp][k] = fmaf(a_0[k], vv[k], second[grp][k]);
                        last[grp][k] = fmaf(a_p[k], vv[k], last[grp][k]);
                    }
                }
            }
        };

        // Step t, row yo (complete in p) -> mid ring.  Rows y_begin - 1 ..
        // y_end are the ones step t + 1 reads; earlier rows are pipeline
        // start-up whose values are never used.
        auto finish_a = [&](int yo, int slot, const float (&p)[2][4]) {
            const bool row_in = yo >= 0 && yo < dh;
            const uint32_t fl = row_bits(0, yo - (y_begin - 1)) >> n;   // bits 0, 16: cells n, 16 + n
            const float4 *own = ring[slot] + g * RS::PS;
            float4 *out = mid[(yo - base) & 1] + g * RS::PS;
            v4f acc[2][4];
            float f[2][8];
#pragma unroll
            for (int grp = 0; grp < 2; ++grp) {
                const float4 sv = own[1 + grp * 16 + n];
                f[grp][0] = sv.x; f[grp][1] = sv.y; f[grp][2] = sv.z; f[grp][3] = sv.w;
#pragma unroll
                for (int k = 0; k < 4; ++k) f[grp][4 + k] = p[grp][k];
                mlp.layer1(f[grp], acc[grp]);
            }
#pragma unroll
            for (int grp = 0; grp < 2; ++grp) {
                const v4f u = mlp.layer2(acc[grp]);
                const int x = x1 + grp * 16 + n;
                const bool in = row_in && x >= 0 && x < dw;
                const float m = (float)__builtin_amdgcn_ubfe(fl, grp * 16u, 1u);
                float v[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = in ? fmaf(m, u[k], f[grp][k]) : 0.f;
                out[grp * 16 + n] = make_float4(v[0], v[1], v[2], v[3]);
            }
        };

        // Step t + 1, row yo (complete in p): MLP, fire gate and store; rows
        // outside [y_begin, y_end) are dropped by an empty descriptor.
        auto finish_b = [&](int yo, const float (&p)[2][4]) {
            const bool out_ok = yo >= y_begin && yo < y_end;
            const int yc = min(max(yo, 0), dh - 1);
            const uint32_t fl = row_bits(1, yo - y_begin) >> n;   // bits 0, 16: cells n, 16 + n
            const Rsrc wr = make_rsrc(dst + (int64_t)yc * dw * C, out_ok ? row_bytes : 0u);
            const float4 *own = mid[(yo - base) & 1] + g * RS::PS;
            v4f acc[2][4];
            float f[2][8];
#pragma unroll
            for (int grp = 0; grp < 2; ++grp) {
                const float4 sv = own[1 + grp * 16 + n];
                f[grp][0] = sv.x; f[grp][1] = sv.y; f[grp][2] = sv.z; f[grp][3] = sv.w;
#pragma unroll
                for (int k = 0; k < 4; ++k) f[grp][4 + k] = p[grp][k];
                mlp.layer1(f[grp], acc[grp]);
            }
#pragma unroll
            for (int grp = 0; grp < 2; ++grp) {
                const v4f u = mlp.layer2(acc[grp]);
                const int x = x0 + grp * 16 + n;
                const uint32_t off = x < x_stop && g < C / 4 ? (uint32_t)x * kCellBytes : kOut;
                const float m = (float)__builtin_amdgcn_ubfe(fl, grp * 16u, 1u);
                if constexpr (SEG) {
                    v4f o;
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) o[kk] = fmaf(m, u[kk], f[grp][kk]);
                    store_quad(dst, wr, off, g, o);
                    const Rsrc sr = make_rsrc(seg + (int64_t)yc * dw, out_ok ? (uint32_t)dw : 0u);
                    const uint32_t so = g == C / 4 - 1 && x < x_stop ? (uint32_t)x : kOut;
                    __builtin_amdgcn_raw_buffer_store_b8((unsigned char)(o[3] > o[2] ? 1 : 0), sr,
                                                         so, 0, 0);
                } else {
                    update_store(dst, wr, off, g, f[grp], u, m);
                }
            }
        };

        // One input row q per body, from base through y_end + 1 (rounded up
        // to whole groups of three): step t finishes row q - 1, step t + 1 row
        // q - 2.  Row q + 2 is loaded during the body and written to the slot
        // of row q - 1 at its end.
        auto body = [&](int q, auto jc) {
            constexpr int j = decltype(jc)::value;   // (q - base) % 3
            constexpr int jm = (j + 2) % 3, jp = (j + 1) % 3;   // rows q - 1, q + 1 (= q - 2)
            issue(ra, ia, q + 2, up_cy, x1);
            if constexpr (UP) {
                up_cy += ++up_ry == up_fy ? 1 : 0;
                up_ry = up_ry == up_fy ? 0 : up_ry;
            }
            // input row q: outputs q + 1, q, q - 1 of step t; next to it
            // (independent, so the matrix cores overlap the fold's FMAs) step
            // t + 1's row q - 3, whose sum the previous body completed (B[j]
            // is restarted by this body's second fold)
            fold(ring[j] + g * RS::PS, A[jp], A[j], A[jm]);
            finish_b(q - 3, B[j]);
            finish_a(q - 1, jm, A[jm]);
            __builtin_amdgcn_sched_barrier(0);
            // step t's row q - 1: outputs q, q - 1, q - 2 of step t + 1
            fold(mid[(q - 1 - base) & 1] + g * RS::PS, B[j], B[jm], B[jp]);
            __builtin_amdgcn_sched_barrier(0);
            commit(ra, ia, ring[jm]);
        };
        // The first bodies see sums that were never started (rows before
        // base); they only feed rows that are not used.
#pragma unroll
        for (int i = 0; i < 3; ++i)
#pragma unroll
            for (int grp = 0; grp < 2; ++grp)
#pragma unroll
                for (int k = 0; k < 4; ++k) A[i][grp][k] = B[i][grp][k] = cb[k];
        int q0 = base;
        for (; q0 <= y_end + 1; q0 += 3) {
            body(q0, std::integral_constant<int, 0>{});
            body(q0 + 1, std::integral_constant<int, 1>{});
            body(q0 + 2, std::integral_constant<int, 2>{});
        }
        finish_b(q0 - 3, B[0]);   // the last body's deferred row
    }
}

// ---------------------------------------------------------------------------
// 3D: a work item is an 8 x 32 (y, x) column and a run of `zrun` output
// planes (up to k3ZRun; the launch picks it with a load model).  Input planes
// stream through a ring of three LDS plane slots
// (planes p - 1 and p are in use while p + 1 is written).  Each input plane p
// is read once: its 9 in-plane taps feed three rolling perception sums, for
// outputs p + 1 (the dz = -1 weights), p (dz = 0) and p - 1 (dz = +1).  After
// plane p the sum of output p - 1 is complete and that plane's MLP, fire gate
// and store run, with the cell's own state re-read from the ring.  Wave w
// owns rows 2w, 2w+1 (4 groups of 16 cells); the conv weights of a tap are
// read once per wave and applied to all 4 groups.
// ---------------------------------------------------------------------------
constexpr int k3TY = 8;
// Longest run of output planes per work item.  A run re-reads two halo planes,
// so long runs on deep levels stream less; its fire words (one evaluation per
// 4 or 8 planes) take k3ZRun / 4 x 64 B of LDS per wave.  128 keeps the fp16
// step at 3 blocks per CU (44 KB each) and the fp32 one at 2 (78 KB); against
// 32 it took the video pass 89.0 -> 85.3 ms (64: 86.9 ms).  The fp16 step
// takes runs of up to 256 planes (16 KB of fire words per block: 52 KB, still
// 3 blocks per CU).
constexpr int k3ZRun = 128;
constexpr int k3hZRun = 256;
// Work item i of a 3D step is tile (tx, ty) of z run zr, with
// i = (zr * tiles_y + ty) * tiles_x + tx.


// ALIGNED: rows start on an 8-cell boundary (w % 8 == 0), which makes the
// ballot and the bit offset of a lane's cells lane constants.
template <typename T, int NIN, class Mlp, bool ALIGNED>
__global__ __launch_bounds__(kThreads, 2) void nca_step_mfma_3d(
    const T *__restrict__ src, T *__restrict__ dst, int dd, int dh, int dw, int tiles_x,
    int tiles_y, int items, int zrun, const float *__restrict__ conv_w,
    const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold) {
    // C = 16 (H = 64) or the ablation's C = 12 (H = 48): channel quad 3 idle
    constexpr int C = Mlp::kChannels;
    using Loader = RowLoader<T, k3TY + 2, C>;
    __shared__ float4 ring[3][4 * Loader::PS];
    __shared__ float4 tapw[27][4];      // [tap][quad] conv weights of channels 4q..4q+3
    // [wave][evaluation of the work item][b]: ballot b (k3ZRun / 4 evaluations
    // at most: one per 4 or 8 planes)
    __shared__ uint64_t fire_words[4][k3ZRun / 4][8];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int g = lane >> 4;

    {
        const int i = min((int)threadIdx.x, 27 * 4 - 1);
        const int t = i / 4, q = i % 4;
        const int qc = q < C / 4 ? q : 0;   // quads >= C / 4: zero weights
        constexpr float ps = Mlp::kPerceptionScale;
        const float4 tw = make_float4(ps * conv_w[(4 * qc + 0) * 27 + t], ps * conv_w[(4 * qc + 1) * 27 + t],
                                      ps * conv_w[(4 * qc + 2) * 27 + t], ps * conv_w[(4 * qc + 3) * 27 + t]);
        if (threadIdx.x < 27 * 4) tapw[t][q] = q < C / 4 ? tw : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    Mlp mlp;
    mlp.load(w1, b1, w2, n, g, NIN);
    float cb[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
        cb[k] = g < C / 4 ? Mlp::kPerceptionScale * conv_b[4 * (g < C / 4 ? g : 0) + k] : 0.f;
    mlp.pin_all();
#pragma unroll
    for (int k = 0; k < 4; ++k) pin(cb[k]);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // Fire evaluations: a plane's 2 rows per wave take 2 * opr lanes, so one
    // evaluation serves 64 / (2 opr) consecutive output planes (8 when rows
    // are 8-aligned, else 4).  The 8 ballots go to a per-wave LDS array and a
    // cell reads the one it needs by address: selecting among them by a
    // per-lane value in registers makes the compiler build a private
    // (scratch) array, whose loads would be waited for with the stores.
    constexpr int opr = ALIGNED ? 4 : 8;
    constexpr int lg_opr = ALIGNED ? 2 : 3;
    constexpr int planes_per_eval = 64 / (2 * opr);
    constexpr int kCellBytes = Loader::kCellBytes;
    const uint32_t row_bytes = (uint32_t)dw * kCellBytes;
    Loader ld;
    // LDS word of group grp's cell (row 2 wave + grp / 2, column 16 (grp % 2) + n)
    // in the quad plane of this lane, relative to a plane slot.
    int centre[4];
#pragma unroll
    for (int grp = 0; grp < 4; ++grp)
        centre[grp] = g * Loader::PS + (2 * wave + (grp >> 1) + 1) * kHaloW + (grp & 1) * 16 + n + 1;

    const int64_t span = ((int64_t)items + gridDim.x - 1) / gridDim.x * gridDim.x;
    for (int64_t u = blockIdx.x; u < span; u += gridDim.x) {
        const int64_t it = xcd_item(u, (int)gridDim.x);
        if (it >= items) continue;                       // uniform over the block
        const int tiles = tiles_x * tiles_y;
        const int zr = (int)it / tiles;
        const int rest = (int)it - zr * tiles;
        const int tx = rest % tiles_x;
        const int ty = rest / tiles_x;
        const int y0 = ty * k3TY, x0 = tx * kTileW;
        const int z_begin = zr * zrun;
        const int z_end = min(dd, z_begin + zrun);
        // store offsets of the lane's 4 cells within an output plane's tile rows
        uint32_t offs[4];
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
            const int x = x0 + (grp & 1) * 16 + n;
            offs[grp] = x < dw && g < C / 4
                            ? (uint32_t)(2 * wave + (grp >> 1)) * row_bytes + (uint32_t)x * kCellBytes
                            : kOut;
        }

        // Rolling perception sums (bias included): A[(r - z_begin + 1) % 3]
        // holds the sum of output plane r.  The plane loop is unrolled three
        // times, so the sums rotate roles instead of being moved; a run is
        // padded to whole groups of three planes (padding planes load and
        // store nothing).
        float A[3][4][4];
#pragma unroll
        for (int i = 0; i < 3; ++i)
#pragma unroll
            for (int grp = 0; grp < 4; ++grp)
#pragma unroll
                for (int k = 0; k < 4; ++k) A[i][grp][k] = cb[k];

        __syncthreads();   // the previous item's readers are done with the ring
        const typename Loader::Offsets lofs = Loader::offsets(dw, y0, x0);
        ld.issue_at(src, lofs, z_begin - 1, dd, dh, dw, y0);
        // All fire evaluations of the work item, before the plane loop:
        // evaluation e covers output planes z_begin + e * planes_per_eval onwards.
        for (int e = 0; z_begin + e * planes_per_eval < z_end; ++e) {
            const int zo = z_begin + e * planes_per_eval;
            const int zz = min(zo + (lane >> (lg_opr + 1)), dd - 1);
            const uint64_t row =
                (uint64_t)zz * dh + (uint64_t)(y0 + 2 * wave + ((lane >> lg_opr) & 1));
            const FireBallots fb = fire_ballots(((row * dw + x0) >> 3) + (lane & (opr - 1)), step,
                                                level, batch, seed, threshold);
            uint64_t word = fb.w[0];
#pragma unroll
            for (int b = 1; b < 8; ++b) word = (lane & 7) == b ? fb.w[b] : word;
            fire_words[wave][e][lane & 7] = word;   // 8 lanes per address, same value
        }
        ld.commit(ring[0]);
        ld.issue_at(src, lofs, z_begin, dd, dh, dw, y0);
        __syncthreads();

        // Plane p (j = (p - z_begin + 1) % 3) is in ring slot j, plane p - 1 in
        // slot (j + 2) % 3, and plane p + 1 goes to slot (j + 1) % 3.
        auto body = [&](int p, auto jc) {
            constexpr int j = decltype(jc)::value;
            constexpr int jm = (j + 2) % 3, jp = (j + 1) % 3;
            float (&first)[4][4] = A[jp];    // output p + 1 (dz = -1 weights)
            float (&second)[4][4] = A[j];    // output p (dz = 0)
            float (&last)[4][4] = A[jm];     // output p - 1 (dz = +1), complete after
            const float4 *pl = ring[j];
            // Taps are software-pipelined: the LDS reads of tap t + 1 are issued
            // before the FMAs of tap t, and pinning the sums after each tap keeps
            // the compiler from hoisting every read of the plane at once.
            int gq = g;
            pin(gq);   // re-read the tap weights every plane rather than keep 27 in registers
            float4 sv[2][4], wv[2][3];
            auto read_tap = [&](int t, float4 (&s4)[4], float4 (&w3)[3]) {
                const int off = (t / 3 - 1) * kHaloW + (t % 3 - 1);
                w3[0] = tapw[t][gq];        // dz = -1: output p + 1
                w3[1] = tapw[9 + t][gq];    // dz =  0: output p
                w3[2] = tapw[18 + t][gq];   // dz = +1: output p - 1
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) s4[grp] = pl[centre[grp] + off];
            };
            read_tap(0, sv[0], wv[0]);
#pragma unroll
            for (int t = 0; t < 9; ++t) {
                if (t + 1 < 9) read_tap(t + 1, sv[(t + 1) & 1], wv[(t + 1) & 1]);
                const float4 *w3 = wv[t & 1];
                const float a_m[4] = {w3[0].x, w3[0].y, w3[0].z, w3[0].w};
                const float a_0[4] = {w3[1].x, w3[1].y, w3[1].z, w3[1].w};
                const float a_p[4] = {w3[2].x, w3[2].y, w3[2].z, w3[2].w};
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    const float4 v = sv[t & 1][grp];
                    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        first[grp][k] = fmaf(a_m[k], vv[k], t == 0 ? cb[k] : first[grp][k]);
                        second[grp][k] = fmaf(a_0[k], vv[k], second[grp][k]);
                        last[grp][k] = fmaf(a_p[k], vv[k], last[grp][k]);
                    }
                }
#pragma unroll
                for (int grp = 0; grp < 4; ++grp)
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        pin(first[grp][k]);
                        pin(second[grp][k]);
                        pin(last[grp][k]);
                    }
            }
            __builtin_amdgcn_sched_barrier(0);

            // output plane zo = p - 1: MLP, fire gate, store (stores of planes
            // outside [z_begin, z_end) are dropped by an empty descriptor)
            const int zo = p - 1;
            const bool out_ok = zo >= z_begin && zo < z_end;
            const int zrel = min(max(zo - z_begin, 0), k3ZRun - 1);   // in range for any plane
            const int phase = zrel & (planes_per_eval - 1);
            const uint64_t *fwe = fire_words[wave][zrel / planes_per_eval];
            const int slot0 = 2 * phase;
            const Rsrc wr = make_rsrc(dst + ((int64_t)max(zo, 0) * dh + y0) * dw * C,
                                      out_ok ? (uint32_t)min(k3TY, dh - y0) * row_bytes : 0u);
            const float4 *own = ring[jm];
            // ALIGNED: the bits of the lane's 4 cells of this plane, at 2 grp
            // (cell n of group grp is cell n % 8 of block 2 (grp % 2) + n / 8
            // of row grp / 2: bit (slot0 + grp / 2) * 4 + 2 (grp % 2) + n / 8)
            uint32_t fw_lane = 0;
            if constexpr (ALIGNED) fw_lane = (uint32_t)(fwe[n & 7] >> (slot0 * opr + (n >> 3)));
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const float4 sp = own[centre[grp]];
                float f[8] = {sp.x, sp.y, sp.z, sp.w};
#pragma unroll
                for (int k = 0; k < 4; ++k) f[4 + k] = last[grp][k];
                // The MLP of a plane outside the run (the first two bodies of a
                // work item and its padding) is skipped: a uniform branch with
                // no memory operation inside, so the store below and the wait
                // counts around it are the same on both paths.  That store is
                // dropped, so u may hold anything there (left unspecified: no
                // register moves to merge the two paths).
                v4f u = __builtin_nondeterministic_value(u);
                if (out_ok) {
                    v4f acc[4];
                    mlp.layer1(f, acc);
                    u = mlp.layer2(acc);
                }
                float m;
                if constexpr (ALIGNED) {
                    m = (float)__builtin_amdgcn_ubfe(fw_lane, 2u * grp, 1u);
                } else {
                    const int r = grp >> 1;
                    const int y = y0 + 2 * wave + r, x = x0 + (grp & 1) * 16 + n;
                    const uint64_t idx = ((uint64_t)max(zo, 0) * dh + y) * dw + x;
                    const uint64_t row_b0 = (((uint64_t)max(zo, 0) * dh + y) * dw + x0) >> 3;
                    const uint64_t fw = fwe[idx & 7];
                    m = (fw >> ((slot0 + r) * opr + (int)((idx >> 3) - row_b0))) & 1 ? 1.f : 0.f;
                }
                update_store(dst, wr, offs[grp], g, f, u, m);
                __builtin_amdgcn_sched_barrier(0);
            }

            // plane p + 1 into the free slot, then start loading p + 2
            ld.commit(ring[jp]);
            ld.issue_at(src, lofs, p + 2, dd, dh, dw, y0, p + 2 <= z_end);
            __syncthreads();
        };
        for (int p0 = z_begin - 1; p0 <= z_end; p0 += 3) {
            body(p0, std::integral_constant<int, 0>{});
            body(p0 + 1, std::integral_constant<int, 1>{});
            body(p0 + 2, std::integral_constant<int, 2>{});
        }
    }
}

// ---------------------------------------------------------------------------
// 3D step for fp16 states with the fp16 MLP: the same z streaming as
// nca_step_mfma_3d, but the ring holds the planes as fp16 (8-byte channel
// quads, half the LDS) and the perception sums are packed fp16 FMAs
// (v_pk_fma_f16: two channels per instruction, half the VALU work of fp32
// sums).  The features go to the fp16 MFMAs without conversion.  The sums
// are rounded to fp16 after every tap; with fp16 storage this changes the
// result by far less than the fp16 rounding of the stored state itself.
// ---------------------------------------------------------------------------
typedef _Float16 h2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
// (mask & a) | (~mask & b) in one instruction (the compiler builds it from
// two ands, an and-or and the mask's complement)
__device__ __forceinline__ uint32_t bfi(uint32_t mask, uint32_t a, uint32_t b) {
    uint32_t r;
    asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(mask), "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ uint32_t as_u32(h2 v) { return __builtin_bit_cast(uint32_t, v); }

constexpr int k3hBlocksPerCu = 3;
// the upsample-fused variant: its extra set-up registers spill a few words
// outside the plane loop at 3 blocks per CU
constexpr int k3hUpBlocksPerCu = 3;

// UP: the first step of a level fused with the upsample + inject: src is the
// next coarser level's state (extent up_cdh x up_cdw per plane), upsampled by
// (up_fz, up_fy, up_fx), with the input channels from up_img.
// (The UP variant runs one step per level and needs more registers for its
// extra loads: it is built for 2 blocks per CU, the plain one for 3.)
// SEG: the launch also writes the two-class readout of the state it stores
// (channel C - 1 > channel C - 2 in the stored fp16 values, ties and NaNs 0)
// to seg; the finest level's last launch uses it.
template <int NIN, bool ALIGNED, bool UP, bool SEG = false>
__global__ __launch_bounds__(kThreads, UP ? k3hUpBlocksPerCu : k3hBlocksPerCu) void nca_step_mfma_3d_f16(
    const __half *__restrict__ src, __half *__restrict__ dst, int dd, int dh, int dw,
    int tiles_x, int tiles_y, int items, int zrun, const float *__restrict__ conv_w,
    const float *__restrict__ conv_b, const float *__restrict__ w1, const float *__restrict__ b1,
    const float *__restrict__ w2, uint32_t level, uint32_t step, uint32_t batch, uint64_t seed,
    uint64_t threshold, const __half *__restrict__ up_img, int up_cdh, int up_cdw, int up_fz,
    int up_fy, int up_fx, uint8_t *__restrict__ seg) {
    using Loader = RowLoader<__half, k3TY + 2>;
    __shared__ uint2 ring[3][4 * Loader::PS16];
    __shared__ uint2 tapw[27][4];           // [tap][quad] fp16 conv weights of channels 4q..4q+3
    // [wave][evaluation of the work item][b]: ballot b (k3hZRun / 4 evaluations
    // at most: one per 4 or 8 planes)
    __shared__ uint64_t fire_words[4][k3hZRun / 4][8];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int g = lane >> 4;

    {
        const int i = min((int)threadIdx.x, 27 * 4 - 1);
        const int t = i / 4, q = i % 4;
        const h2 lo = {(_Float16)conv_w[(4 * q + 0) * 27 + t], (_Float16)conv_w[(4 * q + 1) * 27 + t]};
        const h2 hi = {(_Float16)conv_w[(4 * q + 2) * 27 + t], (_Float16)conv_w[(4 * q + 3) * 27 + t]};
        if (threadIdx.x < 27 * 4) tapw[t][q] = make_uint2(as_u32(lo), as_u32(hi));
    }
    MlpF16 mlp;
    mlp.load(w1, b1, w2, n, g, NIN);
    h2 cb[2];
    cb[0] = h2{(_Float16)conv_b[4 * g + 0], (_Float16)conv_b[4 * g + 1]};
    cb[1] = h2{(_Float16)conv_b[4 * g + 2], (_Float16)conv_b[4 * g + 3]};
    float one = 1.f;
    mlp.pin_all();
    pin(cb[0]);
    pin(cb[1]);
    pin(one);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // fire evaluations as in nca_step_mfma_3d; ALIGNED (w % 8 == 0) makes the
    // ballot and bit offsets of a lane's cells lane constants
    constexpr int opr = ALIGNED ? 4 : 8;
    constexpr int lg_opr = ALIGNED ? 2 : 3;
    constexpr int planes_per_eval = 64 / (2 * opr);
    constexpr int kCellBytes = Loader::kCellBytes;
    const uint32_t row_bytes = (uint32_t)dw * kCellBytes;
    int y0_cur = 0;   // the current item's first tile row (for the loads)
    typename Loader::Offsets lofs;  // and its lane offsets (plain loads)
    typename Loader::template UpOffsets<NIN> uofs;   // (fused upsample loads)
    Loader ld;
    typename Loader::template Image<NIN> im;   // used by UP only
    auto issue = [&](int z, bool active) {
        if constexpr (UP)
            ld.template issue_up<NIN>(src, up_cdh, up_cdw, up_fz, up_fy, up_img, uofs, im, z,
                                      dd, dh, dw, y0_cur, active);
        else
            ld.issue_at(src, lofs, z, dd, dh, dw, y0_cur, active);
    };
    auto commit = [&](uint2 *slot) {
        if constexpr (UP)
            ld.template commit_up_raw<NIN>(slot, im);
        else
            ld.commit_raw(slot);
    };
    int centre[4];
#pragma unroll
    for (int grp = 0; grp < 4; ++grp)
        centre[grp] = g * Loader::PS16 + (2 * wave + (grp >> 1) + 1) * kHaloW + (grp & 1) * 16 + n + 1;

    const int64_t span = ((int64_t)items + gridDim.x - 1) / gridDim.x * gridDim.x;
    for (int64_t u = blockIdx.x; u < span; u += gridDim.x) {
        const int64_t it = xcd_item(u, (int)gridDim.x);
        if (it >= items) continue;                       // uniform over the block
        const int tiles = tiles_x * tiles_y;
        const int zr = (int)it / tiles;
        const int rest = (int)it - zr * tiles;
        const int tx = rest % tiles_x;
        const int ty = rest / tiles_x;
        const int y0 = ty * k3TY, x0 = tx * kTileW;
        y0_cur = y0;
        if constexpr (UP)
            uofs = Loader::template up_offsets<NIN>(up_cdw, up_fy, up_fx, dw, y0, x0);
        else
            lofs = Loader::offsets(dw, y0, x0);
        const int z_begin = zr * zrun;
        const int z_end = min(dd, z_begin + zrun);
        // store offsets of the lane's 4 cells within an output plane's tile rows
        uint32_t offs[4];
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
            const int x = x0 + (grp & 1) * 16 + n;
            offs[grp] = x < dw ? (uint32_t)(2 * wave + (grp >> 1)) * row_bytes +
                                     (uint32_t)x * kCellBytes + 8u * g
                               : kOut;
        }

        // Rolling perception sums (bias included), channels (4g, 4g+1) in
        // [.][0] and (4g+2, 4g+3) in [.][1]: A[(r - z_begin + 1) % 3] holds the
        // sum of output plane r.  The plane loop is unrolled three times, so
        // the three sums rotate roles instead of being moved; a run is padded
        // to whole groups of three planes (the padding planes load nothing and
        // store nothing).
        h2 A[3][4][2];
#pragma unroll
        for (int i = 0; i < 3; ++i)
#pragma unroll
            for (int grp = 0; grp < 4; ++grp)
#pragma unroll
                for (int k = 0; k < 2; ++k) A[i][grp][k] = cb[k];

        __syncthreads();
        issue(z_begin - 1, true);
        // All fire evaluations of the work item, before the plane loop (inside
        // it they cost the loop registers): evaluation e covers output planes
        // z_begin + e * planes_per_eval onwards.
        for (int e = 0; z_begin + e * planes_per_eval < z_end; ++e) {
            const int zo = z_begin + e * planes_per_eval;
            const int zz = min(zo + (lane >> (lg_opr + 1)), dd - 1);
            const uint64_t row =
                (uint64_t)zz * dh + (uint64_t)(y0 + 2 * wave + ((lane >> lg_opr) & 1));
            const FireBallots fb = fire_ballots(((row * dw + x0) >> 3) + (lane & (opr - 1)), step,
                                                level, batch, seed, threshold);
            uint64_t word = fb.w[0];
#pragma unroll
            for (int b = 1; b < 8; ++b) word = (lane & 7) == b ? fb.w[b] : word;
            fire_words[wave][e][lane & 7] = word;
        }
        commit(ring[0]);
        issue(z_begin, true);
        __syncthreads();

        // Plane p (j = (p - z_begin + 1) % 3) is in ring slot j, plane p - 1 in
        // slot (j + 2) % 3, and plane p + 1 goes to slot (j + 1) % 3.
        auto body = [&](int p, auto jc) {
            constexpr int j = decltype(jc)::value;
            constexpr int jm = (j + 2) % 3, jp = (j + 1) % 3;
            h2 (&first)[4][2] = A[jp];    // output p + 1 (dz = -1 weights)
            h2 (&second)[4][2] = A[j];    // output p (dz = 0)
            h2 (&last)[4][2] = A[jm];     // output p - 1 (dz = +1), complete after
            const uint2 *pl = ring[j];
            int gq = g;
            pin(gq);
            uint2 sv[2][4], wv[2][3];
            auto read_tap = [&](int t, uint2 (&s4)[4], uint2 (&w3)[3]) {
                const int off = (t / 3 - 1) * kHaloW + (t % 3 - 1);
                w3[0] = tapw[t][gq];
                w3[1] = tapw[9 + t][gq];
                w3[2] = tapw[18 + t][gq];
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) s4[grp] = pl[centre[grp] + off];
            };
            read_tap(0, sv[0], wv[0]);
#pragma unroll
            for (int t = 0; t < 9; ++t) {
                if (t + 1 < 9) read_tap(t + 1, sv[(t + 1) & 1], wv[(t + 1) & 1]);
                const uint2 *w3 = wv[t & 1];
                const h2 a_m[2] = {as_h2(w3[0].x), as_h2(w3[0].y)};
                const h2 a_0[2] = {as_h2(w3[1].x), as_h2(w3[1].y)};
                const h2 a_p[2] = {as_h2(w3[2].x), as_h2(w3[2].y)};
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    const h2 v[2] = {as_h2(sv[t & 1][grp].x), as_h2(sv[t & 1][grp].y)};
#pragma unroll
                    for (int k = 0; k < 2; ++k) {
                        first[grp][k] = __builtin_elementwise_fma(a_m[k], v[k],
                                                                  t == 0 ? cb[k] : first[grp][k]);
                        second[grp][k] = __builtin_elementwise_fma(a_0[k], v[k], second[grp][k]);
                        last[grp][k] = __builtin_elementwise_fma(a_p[k], v[k], last[grp][k]);
                    }
                }
#pragma unroll
                for (int grp = 0; grp < 4; ++grp)
#pragma unroll
                    for (int k = 0; k < 2; ++k) {
                        pin(first[grp][k]);
                        pin(second[grp][k]);
                        pin(last[grp][k]);
                    }
            }
            __builtin_amdgcn_sched_barrier(0);

            const int zo = p - 1;
            const bool out_ok = zo >= z_begin && zo < z_end;
            const int zrel = min(max(zo - z_begin, 0), k3hZRun - 1);   // in range for any plane
            const int phase = zrel & (planes_per_eval - 1);
            const uint64_t *fwe = fire_words[wave][zrel / planes_per_eval];
            const int slot0 = 2 * phase;
            const Rsrc wr = make_rsrc(dst + ((int64_t)max(zo, 0) * dh + y0) * dw * kC,
                                      out_ok ? (uint32_t)min(k3TY, dh - y0) * row_bytes : 0u);
            const uint2 *own = ring[jm];
            // ALIGNED: the bits of the lane's 4 cells of this plane, at 2 grp
            uint32_t fw_lane = 0;
            if constexpr (ALIGNED) fw_lane = (uint32_t)(fwe[n & 7] >> (slot0 * opr + (n >> 3)));
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const uint2 sp = own[centre[grp]];
                const h2 s01 = as_h2(sp.x), s23 = as_h2(sp.y);
                const v8h fh = {s01[0], s01[1], s23[0], s23[1], last[grp][0][0], last[grp][0][1],
                                last[grp][1][0], last[grp][1][1]};
                v4f acc[4];
                mlp.layer1_h(fh, acc);
                const v4f u = mlp.layer2(acc);
                const int r = grp >> 1;
                // all ones when the cell fires, else zero
                uint32_t keep_new;
                if constexpr (ALIGNED) {
                    // cell n of the group is cell n % 8 of block (grp & 1) * 2 + n / 8 of its
                    // row: bit (r * opr + (grp & 1) * 2) of fw_lane, i.e. bit 2 grp
                    keep_new = (uint32_t)__builtin_amdgcn_sbfe((int)fw_lane, 2 * grp, 1);
                } else {
                    const int y = y0 + 2 * wave + r, x = x0 + (grp & 1) * 16 + n;
                    const uint64_t idx = ((uint64_t)max(zo, 0) * dh + y) * dw + x;
                    const uint64_t row_b0 = (((uint64_t)max(zo, 0) * dh + y) * dw + x0) >> 3;
                    const uint64_t fw = fwe[idx & 7];
                    keep_new = (fw >> ((slot0 + r) * opr + (int)((idx >> 3) - row_b0))) & 1 ? ~0u : 0u;
                }
                const uint32_t off = offs[grp];
                // state + update in fp32, rounded once to fp16 (u = +0 keeps an
                // input channel exactly); a cell that does not fire keeps its
                // stored bits
                // (as fmas with a register 1.0: one mixed-precision fma per value)
                const h2 n01 = {(_Float16)fmaf(one, u[0], (float)s01[0]),
                                (_Float16)fmaf(one, u[1], (float)s01[1])};
                const h2 n23 = {(_Float16)fmaf(one, u[2], (float)s23[0]),
                                (_Float16)fmaf(one, u[3], (float)s23[1])};
                const v2u out = {bfi(keep_new, as_u32(n01), sp.x), bfi(keep_new, as_u32(n23), sp.y)};
                __builtin_amdgcn_raw_buffer_store_b64(out, wr, off, 0, 0);
                if constexpr (SEG) {
                    // lanes of quad 3: out[1] holds channels 14 (low) and 15 (high)
                    const h2 c1415 = as_h2(out[1]);
                    const int x = x0 + (grp & 1) * 16 + n;
                    const Rsrc sr = make_rsrc(seg + ((int64_t)max(zo, 0) * dh + y0) * dw,
                                              out_ok ? (uint32_t)min(k3TY, dh - y0) * dw : 0u);
                    const uint32_t so =
                        g == 3 && x < dw ? (uint32_t)(2 * wave + (grp >> 1)) * dw + x : kOut;
                    __builtin_amdgcn_raw_buffer_store_b8(
                        (unsigned char)((float)c1415[1] > (float)c1415[0] ? 1 : 0), sr, so, 0, 0);
                }
            }

            commit(ring[jp]);
            issue(p + 2, p + 2 <= z_end);
            __syncthreads();
        };
        for (int p0 = z_begin - 1; p0 <= z_end; p0 += 3) {
            body(p0, std::integral_constant<int, 0>{});
            body(p0 + 1, std::integral_constant<int, 1>{});
            body(p0 + 2, std::integral_constant<int, 2>{});
        }
    }
}

// ==== host side: launch plans and dispatch ====

// Compute units of the current device, cached per device.  Host threads may
// call this concurrently: racing first calls store the same value.
int device_cus() {
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

constexpr int kBlocksPerCu = 2;

// Work layout of a 2D level: row streaming over strips of 32 cells (the 16 x
// 32 tile kernel only when asked for).  A work item is a run of k2RunRows
// rows where the level has at least one such run per SIMD of a full MI355X
// (256 CUs x 4 SIMDs); smaller levels take shorter runs (down to 2 rows) so
// that they still spread over about that many waves: they are bound by the
// latency of a wave's rows, not by throughput, and the extra halo rows of
// short runs cost less than idle SIMDs.  Measured against 16 x 32 tiles:
// medium 2D pass 1.43 -> 1.25 ms, tiny 2D 0.285 -> 0.22 ms, training step
// 3.20 -> 3.07 ms; aiming at one run per wave slot (2 per SIMD) or at half a
// run per SIMD was slower.  The row kernel sums the taps in the tile
// kernel's order, so the results are the same bits.  Two steps per launch
// need at least one two-step run per wave slot (kPlanSlots).  Both counts are
// those of a full MI355X, not the device's, so the launch sequence (and with
// it the buffer that holds a result) is the same on every device; only grid
// sizes follow the device.
constexpr int64_t kPlanSlots = 256 * 4 * k2WavesPerSimd;
constexpr int64_t kRowRuns = 256 * 4;

struct RowsPlan {
    int tiles_x;
    int run;                      // rows per work item
    int64_t runs, items, slots;   // slots: wave slots of this device (grid size)
};

RowsPlan rows_plan(const StepArgs &a) {
    RowsPlan r;
    r.tiles_x = (int)((a.ext.w + kTileW - 1) / kTileW);
    r.slots = (int64_t)device_cus() * 4 * k2WavesPerSimd;
    r.run = (int)std::min<int64_t>(
        k2RunRows, std::max<int64_t>(2, (a.ext.h * r.tiles_x + kRowRuns - 1) / kRowRuns));
    r.runs = (a.ext.h + r.run - 1) / r.run;
    r.items = (int64_t)r.tiles_x * r.runs;
    return r;
}

bool uses_rows(const StepArgs &, Layout2d layout) { return layout != Layout2d::Tiles; }

// Row kernel launch; UP: the first step of a level fused with the upsample
// from the coarse state src (width cdw) by (fy, fx) and the image img.
template <typename T, int NIN, class Mlp, bool UP>
hipError_t launch_rows(const StepArgs &a, const void *src, void *dst, const void *img, int cdw,
                       int fy, int fx, hipStream_t stream) {
    const RowsPlan r = rows_plan(a);
    if (r.items == 0) return hipSuccess;
    if (r.items > INT32_MAX) return hipErrorInvalidValue;
    const int grid = (int)std::min<int64_t>(r.items, r.slots);
    auto kern = a.ext.w % 8 == 0 ? nca_step_mfma_2d_rows<T, NIN, Mlp, true, UP>
                                 : nca_step_mfma_2d_rows<T, NIN, Mlp, false, UP>;
    kern<<<grid, 64, 0, stream>>>(
        (const T *)src, (T *)dst, (int)a.ext.h, (int)a.ext.w, r.tiles_x, (int)r.runs, r.run,
        (int)r.items, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch,
        a.seed, a.threshold, (const T *)img, cdw, fy, fx);
    return hipGetLastError();
}

// Two-step row kernel: strips of 30 output cells; used where the single-step
// kernel would use the row layout (fp32 states, default MLP).
RowsPlan pair_plan(const StepArgs &a) {
    RowsPlan r;
    r.tiles_x = (int)((a.ext.w + k2PairW - 1) / k2PairW);
    r.slots = (int64_t)device_cus() * 4 * k2WavesPerSimd;
    r.runs = (a.ext.h + k2RunRows - 1) / k2RunRows;
    r.items = (int64_t)r.tiles_x * r.runs;
    return r;
}

// The ablation's C = 12, H = 48 model (supplement S10) on the kernels of
// C = 16: fp32 states (the 2D row kernels and the 3D step), scaled fp16 MLP,
// the lanes of channel quad 3 and hidden tile 3 idle.
using MlpC12 = MlpF16SM<12, 48>;
bool is_c12(const StepArgs &a) { return a.channels == 12 && a.hidden == 48; }
bool is_c16(const StepArgs &a) { return a.channels == kC && a.hidden == kH; }

bool uses_pairs(const StepArgs &a, MfmaMlp mlp, Layout2d layout) {
    return a.ndim == 2 && a.dtype == Dtype::F32 && (is_c16(a) || is_c12(a)) &&
           a.ext.h * a.ext.w < (int64_t(1) << 32) &&   // 32-bit cell indices in the kernel
           (mlp == MfmaMlp::Default || mlp == MfmaMlp::F16S) &&
           (layout == Layout2d::Rows ||
            (layout == Layout2d::Auto && pair_plan(a).items >= kPlanSlots));
}

// UP: src is the coarse state (width cdw) upsampled by (fy, fx), img the
// level's image; steps a.step and a.step + 1.
template <class Mlp, int NIN, bool UP>
hipError_t launch_rows_pair(const StepArgs &a, const void *src, void *dst, const void *img,
                            int cdw, int fy, int fx, hipStream_t stream) {
    const RowsPlan r = pair_plan(a);
    if (r.items == 0) return hipSuccess;
    if (r.items > INT32_MAX) return hipErrorInvalidValue;
    const int grid = (int)std::min<int64_t>(r.items, r.slots);
    auto kern = a.seg != nullptr ? nca_step2_mfma_2d_rows<float, NIN, Mlp, UP, true>
                                 : nca_step2_mfma_2d_rows<float, NIN, Mlp, UP, false>;
    kern<<<grid, 64, 0, stream>>>(
        (const float *)src, (float *)dst, (int)a.ext.h, (int)a.ext.w, r.tiles_x, k2RunRows,
        (int)r.items, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch,
        a.seed, a.threshold, (const float *)img, cdw, fy, fx, a.seg);
    return hipGetLastError();
}

template <typename T, int NIN, class Mlp>
hipError_t launch_2d(const StepArgs &a, Layout2d layout, const void *src, void *dst,
                     hipStream_t stream) {
    const int tiles_x = (int)((a.ext.w + kTileW - 1) / kTileW);
    const int tiles_y = (int)((a.ext.h + k2TY - 1) / k2TY);
    const int64_t tiles = (int64_t)tiles_x * tiles_y;
    if (tiles == 0) return hipSuccess;
    if (tiles > INT32_MAX) return hipErrorInvalidValue;
    if (uses_rows(a, layout))
        return launch_rows<T, NIN, Mlp, false>(a, src, dst, nullptr, 0, 1, 1, stream);
    if constexpr (Mlp::kChannels != kC) {
        return hipErrorInvalidValue;   // other model sizes: rows only
    } else {
        const int grid = (int)std::min<int64_t>(tiles, (int64_t)device_cus() * k2BlocksPerCu);
        nca_step_mfma_2d<T, NIN, Mlp><<<grid, kThreads, 0, stream>>>(
            (const T *)src, (T *)dst, (int)a.ext.h, (int)a.ext.w, tiles_x, (int)tiles,
            a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch, a.seed,
            a.threshold);
        return hipGetLastError();
    }
}

// Output planes per 3D work item, chosen per launch: the run length r in
// 1 .. max_run that minimises ceil(items(r) / slots) * (planes(r) + 2), the work
// of the most loaded block slot (grid-stride rounds times the planes a work
// item streams, its two halo planes included); ties go to the longer run.
// Short runs spread small levels over the chip at the cost of reading their
// halo planes again; long runs stream large levels with little re-reading.
// With groups of 3 (the fp16 kernel's plane loop is unrolled three times),
// a work item streams its planes in whole groups of three.
int pick_zrun(int64_t tiles, int64_t depth, int64_t slots, bool groups_of_3, int max_run) {
    int best = 1;
    int64_t best_cost = INT64_MAX;
    for (int r = 1; r <= max_run; ++r) {
        const int64_t items = tiles * ((depth + r - 1) / r);
        int64_t planes = std::min<int64_t>(r, depth) + 2;
        if (groups_of_3) planes = (planes + 2) / 3 * 3;
        const int64_t cost = (items + slots - 1) / slots * planes;
        if (cost <= best_cost) {
            best_cost = cost;
            best = r;
        }
    }
    return best;
}

template <typename T, int NIN, class Mlp>
hipError_t launch_3d(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    constexpr bool kF16 = std::is_same_v<T, __half> && std::is_same_v<Mlp, MlpF16>;
    const int tiles_x = (int)((a.ext.w + kTileW - 1) / kTileW);
    const int tiles_y = (int)((a.ext.h + k3TY - 1) / k3TY);
    const int64_t slots = (int64_t)device_cus() * (kF16 ? k3hBlocksPerCu : kBlocksPerCu);
    const int zrun =
        pick_zrun((int64_t)tiles_x * tiles_y, a.ext.d, slots, true, kF16 ? k3hZRun : k3ZRun);
    const int64_t zruns = (a.ext.d + zrun - 1) / zrun;
    const int64_t items = (int64_t)tiles_x * tiles_y * zruns;
    if (items == 0) return hipSuccess;
    if (items > INT32_MAX) return hipErrorInvalidValue;
    if constexpr (kF16) {
        const int grid = (int)std::min<int64_t>(items, slots);
        auto kern = a.seg != nullptr
                        ? (a.ext.w % 8 == 0 ? nca_step_mfma_3d_f16<NIN, true, false, true>
                                            : nca_step_mfma_3d_f16<NIN, false, false, true>)
                        : (a.ext.w % 8 == 0 ? nca_step_mfma_3d_f16<NIN, true, false>
                                            : nca_step_mfma_3d_f16<NIN, false, false>);
        kern<<<grid, kThreads, 0, stream>>>(
            (const __half *)src, (__half *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, tiles_x,
            tiles_y, (int)items, zrun, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level,
            a.step, a.batch, a.seed, a.threshold, nullptr, 0, 0, 1, 1, 1, a.seg);
    } else {
        const int grid = (int)std::min<int64_t>(items, slots);
        auto kern = a.ext.w % 8 == 0 ? nca_step_mfma_3d<T, NIN, Mlp, true>
                                     : nca_step_mfma_3d<T, NIN, Mlp, false>;
        kern<<<grid, kThreads, 0, stream>>>(
            (const T *)src, (T *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, tiles_x, tiles_y,
            (int)items, zrun, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step,
            a.batch, a.seed, a.threshold);
    }
    return hipGetLastError();
}

// fp16 3D first step fused with the upsample from the coarse state (planes of
// cdh x cdw cells, factors fz, fy, fx) and the level's image img.
template <int NIN>
hipError_t launch_3d_f16_up(const StepArgs &a, const void *coarse, int cdh, int cdw, int fz,
                            int fy, int fx, const void *img, void *dst, hipStream_t stream) {
    const int tiles_x = (int)((a.ext.w + kTileW - 1) / kTileW);
    const int tiles_y = (int)((a.ext.h + k3TY - 1) / k3TY);
    const int64_t slots = (int64_t)device_cus() * k3hUpBlocksPerCu;
    const int zrun = pick_zrun((int64_t)tiles_x * tiles_y, a.ext.d, slots, true, k3hZRun);
    const int64_t zruns = (a.ext.d + zrun - 1) / zrun;
    const int64_t items = (int64_t)tiles_x * tiles_y * zruns;
    if (items == 0) return hipSuccess;
    if (items > INT32_MAX) return hipErrorInvalidValue;
    const int grid = (int)std::min<int64_t>(items, slots);
    auto kern = a.ext.w % 8 == 0 ? nca_step_mfma_3d_f16<NIN, true, true>
                                 : nca_step_mfma_3d_f16<NIN, false, true>;
    kern<<<grid, kThreads, 0, stream>>>(
        (const __half *)coarse, (__half *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, tiles_x,
        tiles_y, (int)items, zrun, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level,
        a.step, a.batch, a.seed, a.threshold, (const __half *)img, cdh, cdw, fz, fy, fx, nullptr);
    return hipGetLastError();
}

template <typename T, class Mlp>
hipError_t dispatch(const StepArgs &a, Layout2d layout, const void *src, void *dst,
                    hipStream_t stream) {
    if (a.ndim == 2) {
        if (a.n_in == 1) return launch_2d<T, 1, Mlp>(a, layout, src, dst, stream);
        if (a.n_in == 3) return launch_2d<T, 3, Mlp>(a, layout, src, dst, stream);
    } else if constexpr (Mlp::kChannels == kC || std::is_same_v<T, float>) {
        // 3D: C = 16, H = 64, or fp32 states of C = 12, H = 48
        if (a.n_in == 1) return launch_3d<T, 1, Mlp>(a, src, dst, stream);
        if (a.n_in == 3) return launch_3d<T, 3, Mlp>(a, src, dst, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool mfma_fits(const StepArgs &a) {
    // Buffer descriptors address a tile's rows with 32-bit offsets: rows of
    // more than (2^32 / 18 rows) bytes go to the vector kernel instead.
    const int64_t cell_bytes = (int64_t)kC * (a.dtype == Dtype::F32 ? 4 : 2);
    return (int64_t)(k2TY + 2) * a.ext.w * cell_bytes < (int64_t(1) << 32);
}

bool step_mfma_single_readout(const StepArgs &a, MfmaMlp mlp) {
    return a.ndim == 3 && a.dtype == Dtype::F16 && a.channels == kC && a.hidden == kH &&
           (mlp == MfmaMlp::Default || mlp == MfmaMlp::F16) && mfma_fits(a);
}

bool step_mfma_pairs(const StepArgs &a, MfmaMlp mlp, Layout2d layout) {
    return mfma_fits(a) && uses_pairs(a, mlp, layout);
}

template <class Mlp>
hipError_t launch_pair_size(const StepArgs &a, const void *src, void *dst, const void *img,
                            int cdw, int fy, int fx, bool up, hipStream_t stream) {
    if (a.n_in == 1)
        return up ? launch_rows_pair<Mlp, 1, true>(a, src, dst, img, cdw, fy, fx, stream)
                  : launch_rows_pair<Mlp, 1, false>(a, src, dst, nullptr, 0, 1, 1, stream);
    if (a.n_in == 3)
        return up ? launch_rows_pair<Mlp, 3, true>(a, src, dst, img, cdw, fy, fx, stream)
                  : launch_rows_pair<Mlp, 3, false>(a, src, dst, nullptr, 0, 1, 1, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_step2_mfma(const StepArgs &a, MfmaMlp mlp, Layout2d layout, const void *src,
                             void *dst, hipStream_t stream) {
    if (!step_mfma_pairs(a, mlp, layout)) return hipErrorInvalidValue;
    return is_c12(a) ? launch_pair_size<MlpC12>(a, src, dst, nullptr, 0, 1, 1, false, stream)
                     : launch_pair_size<MlpF32State>(a, src, dst, nullptr, 0, 1, 1, false, stream);
}

hipError_t launch_step2_mfma_up(const StepArgs &a, MfmaMlp mlp, Layout2d layout,
                                const void *coarse, int coarse_w, int fy, int fx, const void *img,
                                void *dst, hipStream_t stream) {
    if (!step_mfma_pairs(a, mlp, layout)) return hipErrorInvalidValue;
    return is_c12(a)
               ? launch_pair_size<MlpC12>(a, coarse, dst, img, coarse_w, fy, fx, true, stream)
               : launch_pair_size<MlpF32State>(a, coarse, dst, img, coarse_w, fy, fx, true, stream);
}

bool step_mfma_serves(const StepArgs &a, Layout2d layout) {
    if (is_c16(a)) return true;
    return is_c12(a) && a.dtype == Dtype::F32 && (a.ndim == 3 || uses_rows(a, layout)) &&
           mfma_fits(a);
}

bool step_mfma_fuses_upsample(const StepArgs &a, MfmaMlp mlp, Layout2d layout) {
    if (mlp != MfmaMlp::Default || !mfma_fits(a)) return false;
    if (is_c12(a)) return a.ndim == 2 && step_mfma_serves(a, layout);
    if (!is_c16(a)) return false;
    if (a.ndim == 2) return uses_rows(a, layout);
    return a.dtype == Dtype::F16;   // the fp16 3D step
}

hipError_t launch_step_mfma_up(const StepArgs &a, Layout2d layout, const void *coarse,
                               int coarse_h, int coarse_w, int fz, int fy, int fx,
                               const void *img, void *dst, hipStream_t stream) {
    if (!step_mfma_fuses_upsample(a, MfmaMlp::Default, layout)) return hipErrorInvalidValue;
    if (a.ndim == 3) {
        if (a.n_in == 1)
            return launch_3d_f16_up<1>(a, coarse, coarse_h, coarse_w, fz, fy, fx, img, dst,
                                       stream);
        if (a.n_in == 3)
            return launch_3d_f16_up<3>(a, coarse, coarse_h, coarse_w, fz, fy, fx, img, dst,
                                       stream);
        return hipErrorInvalidValue;
    }
    if (is_c12(a)) {
        if (a.n_in == 1)
            return launch_rows<float, 1, MlpC12, true>(a, coarse, dst, img, coarse_w, fy, fx,
                                                       stream);
        if (a.n_in == 3)
            return launch_rows<float, 3, MlpC12, true>(a, coarse, dst, img, coarse_w, fy, fx,
                                                       stream);
        return hipErrorInvalidValue;
    }
    if (a.dtype == Dtype::F32) {
        if (a.n_in == 1)
            return launch_rows<float, 1, MlpF32State, true>(a, coarse, dst, img, coarse_w, fy, fx,
                                                            stream);
        if (a.n_in == 3)
            return launch_rows<float, 3, MlpF32State, true>(a, coarse, dst, img, coarse_w, fy, fx,
                                                            stream);
    } else {
        if (a.n_in == 1)
            return launch_rows<__half, 1, MlpF16, true>(a, coarse, dst, img, coarse_w, fy, fx,
                                                        stream);
        if (a.n_in == 3)
            return launch_rows<__half, 3, MlpF16, true>(a, coarse, dst, img, coarse_w, fy, fx,
                                                        stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_step_mfma(const StepArgs &a, MfmaMlp mlp, Layout2d layout, const void *src,
                            void *dst, hipStream_t stream) {
    if (!mfma_fits(a)) return launch_step_valu(a, src, dst, stream);
    if (is_c12(a)) {
        if (!step_mfma_serves(a, layout) || mlp != MfmaMlp::Default) return hipErrorInvalidValue;
        return dispatch<float, MlpC12>(a, layout, src, dst, stream);
    }
    if (!is_c16(a)) return hipErrorInvalidValue;
    if (mlp == MfmaMlp::Default)
        mlp = a.dtype == Dtype::F32 ? MfmaMlp::F16S : MfmaMlp::F16;
    if (a.dtype == Dtype::F32) {
        switch (mlp) {
            case MfmaMlp::F32: return dispatch<float, MlpF32>(a, layout, src, dst, stream);
            case MfmaMlp::Bf16x3: return dispatch<float, MlpBf16x3>(a, layout, src, dst, stream);
            case MfmaMlp::F16S: return dispatch<float, MlpF32State>(a, layout, src, dst, stream);
            default: return hipErrorInvalidValue;   // fp16 operands are too coarse for fp32 states
        }
    }
    switch (mlp) {
        case MfmaMlp::F32: return dispatch<__half, MlpF32>(a, layout, src, dst, stream);
        case MfmaMlp::Bf16x3: return dispatch<__half, MlpBf16x3>(a, layout, src, dst, stream);
        case MfmaMlp::F16: return dispatch<__half, MlpF16>(a, layout, src, dst, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace octnca
