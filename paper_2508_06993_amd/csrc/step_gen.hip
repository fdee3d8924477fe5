// Fused NCA step on the matrix cores for any model size C / H with C a
// multiple of 4 (Sec. 3.1; supplement S3, Listing 1).  It serves the other
// sizes of the paper's ablation (supplement S10: C / H = 12 / 48 and
// 20 / 100); the C = 16, H = 64 model has its own specialised kernels.
//
// Layout (generalising the 16 / 64 kernels' lane mapping):
//   lane l of a wave -> cell n = l % 16 of a 16-cell group and lane group
//   g = l / 16.  The 2C features of a cell are taken in K chunks of 32: chunk
//   k holds channel quads q = 4k .. 4k+3, lane group g the quad q = 4k + g as
//   eight K slots (its 4 state channels, then its 4 perception channels).
//   Quads beyond C / 4 are zero slots.  So a lane forms the perception of the
//   channels it owns, and
//   * layer 1, H[j][n] = b1[j] + sum_k W1[j][k] F[k][n], is
//     v_mfma_f32_16x16x32_f16 with A = a 16-unit tile of W1's rows (columns
//     gathered in the slot order above) and B = the lane's 8 features; its
//     accumulator leaves hidden unit 16t + 4g + i of cell n in register i;
//   * two hidden tiles (2p, 2p+1) together are the 8 K slots of lane group g
//     in layer 2's chunk p: slot s <-> hidden unit (2p + s/4) 16 + 4g + s%4,
//     W2's columns gathered to match, so ReLU'd accumulators feed layer 2
//     directly (no hidden activation leaves the registers);
//   * layer 2's output tile k holds channels 16k + 4g + i of cell n, which is
//     the lane's own quad of chunk k: the residual and the store need no
//     exchange.
// Hidden tiles are padded to an even count with zero weights; W2's rows of
// the input channels (and of channels >= C) are zero, so their update is +0.
// MLP arithmetic: fp32 states take the scaled-fp16 form of the 16 / 64
// kernels (activations times 2^-8 rounded to fp16, weights as fp16 hi + lo,
// two products per weight, fp32 accumulation); fp16 states take fp16
// weights and activations, fp32 accumulation.
//
// Work: a persistent grid loops over tiles of 8 x 32 cells (2D) or
// 2 x 4 x 32 (3D).  A tile and its one-cell halo are staged in LDS as fp32 in
// channel-quad planes (16 consecutive lanes read 16 consecutive 16-byte
// words); the block's weights are converted once into LDS in lane order, and
// each wave reads an MFMA's weight operand once for its four groups.  Fire
// bits: one Philox4x64-10 evaluation per block of 8 consecutive cells of a
// tile row, kept as a byte in LDS.
#include <algorithm>
#include <type_traits>

#include "launch.h"

namespace octnca {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v8f __attribute__((ext_vector_type(8)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int kGenThreads = 256;   // 4 waves, 4 groups of 16 cells each
constexpr float kGenScale = 1.f / 256.f;

template <int C, int H>
struct GenDims {
    static_assert(C % 4 == 0, "channels in whole quads");
    static constexpr int NQ = C / 4;              // channel quads
    static constexpr int NK = (NQ + 3) / 4;       // layer-1 K chunks = layer-2 output tiles
    static constexpr int NT = (H + 15) / 16;      // hidden tiles
    static constexpr int NT2 = (NT + 1) / 2 * 2;  // padded to whole pairs
    static constexpr int NP = NT2 / 2;            // layer-2 K chunks
};

template <int NDIM> struct GenTile;
template <> struct GenTile<2> { static constexpr int TZ = 1, TY = 8, TX = 32; };
template <> struct GenTile<3> { static constexpr int TZ = 2, TY = 4, TX = 32; };

struct WPair {
    v8h hi, lo;
};

__device__ __forceinline__ float4 load_quad(const float *p) {
    return *reinterpret_cast<const float4 *>(p);
}
__device__ __forceinline__ float4 load_quad(const __half *p) {
    const uint2 v = *reinterpret_cast<const uint2 *>(p);
    float4 r;
    Storage<__half>::unpack_pair(v.x, r.x, r.y);
    Storage<__half>::unpack_pair(v.y, r.z, r.w);
    return r;
}
__device__ __forceinline__ void store_quad(float *p, float4 v) {
    *reinterpret_cast<float4 *>(p) = v;
}
__device__ __forceinline__ void store_quad(__half *p, float4 v) {
    *reinterpret_cast<uint2 *>(p) =
        make_uint2(Storage<__half>::pack_pair(v.x, v.y), Storage<__half>::pack_pair(v.z, v.w));
}

// An empty asm that reads and rewrites the value: work before it stays before it.
__device__ __forceinline__ void pin4(float4 &v) {
    asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
}

__device__ __forceinline__ float4 fma4(float4 a, float4 b, float4 c) {
    return make_float4(fmaf(a.x, b.x, c.x), fmaf(a.y, b.y, c.y), fmaf(a.z, b.z, c.z),
                       fmaf(a.w, b.w, c.w));
}

// Feature column of W1 for K slot s of lane group g in chunk k (-1: zero slot).
template <int C>
__device__ __forceinline__ int gen_feature(int k, int g, int s) {
    const int q = 4 * k + g;
    if (q >= C / 4) return -1;
    return s < 4 ? 4 * q + s : C + 4 * q + (s - 4);
}

// Hidden unit of layer 2's K slot s of lane group g in chunk p.
__device__ __forceinline__ int gen_hidden(int p, int g, int s) {
    return (2 * p + s / 4) * 16 + 4 * g + s % 4;
}

// Blocks per CU (4 waves each) that LDS (160 KB per CU) and registers allow:
// 2D C = 12 three (about 32 KB of LDS each), 2D C = 20 and 3D C = 12 two
// (79 KB and 55 KB), 3D C = 20 one (115 KB).
template <int NDIM, int C>
constexpr int kGenBlocksPerCu = NDIM == 2 ? (C <= 12 ? 3 : 2) : (C <= 12 ? 2 : 1);

template <typename T, int NDIM, int NIN, int C, int H>
__global__ __launch_bounds__(kGenThreads, (kGenBlocksPerCu<NDIM, C>)) void nca_step_gen(
    const T *__restrict__ src, T *__restrict__ dst, int dd, int dh, int dw, int tiles_x,
    int tiles_y, int tiles, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold) {
    using D = GenDims<C, H>;
    constexpr bool kSplit = std::is_same_v<T, float>;   // fp32 states: split weights, scaled
    constexpr float kScale = kSplit ? kGenScale : 1.f;
    constexpr int TZ = GenTile<NDIM>::TZ, TY = GenTile<NDIM>::TY, TX = GenTile<NDIM>::TX;
    constexpr int HZ = NDIM == 3 ? TZ + 2 : 1, HY = TY + 2, HX = TX + 2;
    constexpr int NCELL = HZ * HY * HX;
    constexpr int PS = (NCELL + 15) / 16 * 16;          // quad-plane stride (float4s)
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    constexpr int ROWS = TZ * TY;                        // tile rows of TX cells
    constexpr int BPR = TX / 8 + 1;                      // 8-cell blocks a tile row can touch

    __shared__ float4 halo[D::NQ * PS];
    __shared__ float4 tapw[TAPS][D::NQ];                 // conv weights of quad q, times kScale
    __shared__ float4 cbias[D::NQ];                      // conv bias, times kScale
    __shared__ WPair w1s[D::NT2][D::NK][64];             // layer-1 A operands in lane order
    __shared__ float4 b1s[D::NT2][4];                    // [t][g]: b1[16t + 4g + i] * kScale
    __shared__ WPair w2s[D::NP][D::NK][64];              // layer-2 A operands in lane order
    __shared__ uint32_t fire_bytes[ROWS][BPR];           // 8 fire bits per block (low byte)

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int n = lane & 15;
    const int g = lane >> 4;

    // ---- weights into LDS (once per block) ----
    for (int i = tid; i < TAPS * D::NQ; i += kGenThreads) {
        const int t = i / D::NQ, q = i % D::NQ;
        tapw[t][q] = make_float4(kScale * conv_w[(4 * q + 0) * TAPS + t],
                                 kScale * conv_w[(4 * q + 1) * TAPS + t],
                                 kScale * conv_w[(4 * q + 2) * TAPS + t],
                                 kScale * conv_w[(4 * q + 3) * TAPS + t]);
    }
    for (int q = tid; q < D::NQ; q += kGenThreads)
        cbias[q] = make_float4(kScale * conv_b[4 * q + 0], kScale * conv_b[4 * q + 1],
                               kScale * conv_b[4 * q + 2], kScale * conv_b[4 * q + 3]);
    for (int i = tid; i < D::NT2 * D::NK * 64; i += kGenThreads) {
        const int l = i % 64, k = (i / 64) % D::NK, t = i / (64 * D::NK);
        const int row = 16 * t + (l & 15), lg = l >> 4;
        v8f x;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const int f = gen_feature<C>(k, lg, s);
            // load a valid element for every slot, then zero the padding (a
            // load behind the condition costs a branch and a memory wait)
            const float v = w1[min(row, H - 1) * 2 * C + max(f, 0)];
            x[s] = (row < H && f >= 0) ? v : 0.f;
        }
        WPair wp;
        wp.hi = __builtin_convertvector(x, v8h);
        wp.lo = __builtin_convertvector(x - __builtin_convertvector(wp.hi, v8f), v8h);
        w1s[t][k][l] = wp;
    }
    for (int i = tid; i < D::NT2 * 4; i += kGenThreads) {
        const int t = i / 4, lg = i % 4;
        float b[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int j = 16 * t + 4 * lg + r;
            const float v = b1[min(j, H - 1)];
            b[r] = j < H ? kScale * v : 0.f;
        }
        b1s[t][lg] = make_float4(b[0], b[1], b[2], b[3]);
    }
    for (int i = tid; i < D::NP * D::NK * 64; i += kGenThreads) {
        const int l = i % 64, k = (i / 64) % D::NK, p = i / (64 * D::NK);
        const int ch = 16 * k + (l & 15), lg = l >> 4;
        v8f x;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const int j = gen_hidden(p, lg, s);
            const float v = w2[min(ch, C - 1) * H + min(j, H - 1)];
            x[s] = (ch >= NIN && ch < C && j < H) ? v * (1.f / kScale) : 0.f;
        }
        WPair wp;
        wp.hi = __builtin_convertvector(x, v8h);
        wp.lo = __builtin_convertvector(x - __builtin_convertvector(wp.hi, v8f), v8h);
        w2s[p][k][l] = wp;
    }

    // LDS index of group grp's cell (relative to a quad plane), and its
    // position in the tile: 2D rows 2 wave + grp / 2; 3D plane wave / 2,
    // rows 2 (wave % 2) + grp / 2; columns 16 (grp % 2) + n.
    int lz[4], ly[4], lx[4], centre[4];
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
        lz[grp] = NDIM == 3 ? wave / 2 : 0;
        ly[grp] = NDIM == 3 ? 2 * (wave % 2) + grp / 2 : 2 * wave + grp / 2;
        lx[grp] = 16 * (grp % 2) + n;
        centre[grp] = ((NDIM == 3 ? lz[grp] + 1 : 0) * HY + ly[grp] + 1) * HX + lx[grp] + 1;
    }

    // The next tile's halo chunks are loaded into registers while the current
    // tile is computed (LPT 16-byte chunks per thread) and written to LDS
    // after it, so the loads' latency overlaps the compute.
    constexpr int LPT = (NCELL * D::NQ + kGenThreads - 1) / kGenThreads;
    float4 pre[LPT];
    auto issue = [&](int tile) {
        const int x0 = (tile % tiles_x) * TX, y0 = ((tile / tiles_x) % tiles_y) * TY;
        const int z0 = (tile / (tiles_x * tiles_y)) * TZ;
#pragma unroll
        for (int j = 0; j < LPT; ++j) {
            const int i = tid + j * kGenThreads;
            const int q = i % D::NQ, cell = i / D::NQ;
            const int hx = cell % HX, hy = (cell / HX) % HY, hz = cell / (HX * HY);
            const int x = x0 - 1 + hx, y = y0 - 1 + hy, z = NDIM == 3 ? z0 - 1 + hz : z0;
            pre[j] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (tile < tiles && i < NCELL * D::NQ && x >= 0 && x < dw && y >= 0 && y < dh &&
                z >= 0 && z < dd)
                pre[j] = load_quad(src + (((int64_t)z * dh + y) * dw + x) * C + 4 * q);
        }
    };
    issue(blockIdx.x);

    for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int tx = tile % tiles_x;
        const int ty = (tile / tiles_x) % tiles_y;
        const int tz = tile / (tiles_x * tiles_y);
        const int x0 = tx * TX, y0 = ty * TY, z0 = tz * TZ;

        __syncthreads();   // weights written / the previous tile's readers are done
        // ---- halo tile: fp32 channel-quad planes, zero outside the grid ----
#pragma unroll
        for (int j = 0; j < LPT; ++j) {
            const int i = tid + j * kGenThreads;
            if (i < NCELL * D::NQ) halo[(i % D::NQ) * PS + i / D::NQ] = pre[j];
        }
        // ---- fire bits: block b0(row) + k of each tile row ----
        for (int i = tid; i < ROWS * BPR; i += kGenThreads) {
            const int r = i / BPR, k = i % BPR;
            const int z = z0 + r / TY, y = y0 + r % TY;
            uint32_t byte = 0;
            if (z < dd && y < dh) {
                const uint64_t idx0 = ((uint64_t)z * dh + y) * dw + x0;
                const Philox4x64Out o =
                    philox4x64_10((idx0 >> 3) + k, step, level, batch, seed, 0);
#pragma unroll
                for (int b = 0; b < 8; ++b) byte |= ((uint64_t)draw_of(o, b) < threshold ? 1u : 0u) << b;
            }
            fire_bytes[r][k] = byte;
        }
        __syncthreads();
        issue(tile + gridDim.x);   // the next tile's loads, in flight during the compute

        // ---- features: chunk k of group grp = quad 4k + g of its cell; a
        // tap's weights are read once and applied to the four groups ----
        v8h fe[4][D::NK];
        float4 st[4][D::NK];   // the lane's state quads (for the residual)
#pragma unroll
        for (int k = 0; k < D::NK; ++k) {
            const int q = 4 * k + g;
            const bool qv = q < D::NQ;
            const int qc = qv ? q : D::NQ - 1;
            const float4 *pl = halo + qc * PS;
            float4 p[4];
            const float4 cb = cbias[qc];
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) p[grp] = cb;
#pragma unroll
            for (int t = 0; t < TAPS; ++t) {
                const int dz = NDIM == 3 ? t / 9 - 1 : 0;
                const int dy = (t / 3) % 3 - 1, dx = t % 3 - 1;
                const float4 w = tapw[t][qc];
#pragma unroll
                for (int grp = 0; grp < 4; ++grp)
                    p[grp] = fma4(w, pl[centre[grp] + (dz * HY + dy) * HX + dx], p[grp]);
                // keep the compiler from hoisting every tap's reads at once
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) pin4(p[grp]);
            }
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const float4 sv = pl[centre[grp]];
                st[grp][k] = sv;
                v8f x = {sv.x * kScale, sv.y * kScale, sv.z * kScale, sv.w * kScale,
                         p[grp].x, p[grp].y, p[grp].z, p[grp].w};
                if (!qv) x = v8f{};
                fe[grp][k] = __builtin_convertvector(x, v8h);
            }
        }

        // ---- MLP: per hidden-tile pair, layer 1 then its share of layer 2 ----
        v4f u[4][D::NK];
#pragma unroll
        for (int grp = 0; grp < 4; ++grp)
#pragma unroll
            for (int k = 0; k < D::NK; ++k) u[grp][k] = v4f{0.f, 0.f, 0.f, 0.f};
        const v8h zero = {};
#pragma unroll
        for (int pr = 0; pr < D::NP; ++pr) {
            v4f acc[4][2];
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int t = 2 * pr + h2;
                const float4 bb = b1s[t][g];
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) acc[grp][h2] = v4f{bb.x, bb.y, bb.z, bb.w};
#pragma unroll
                for (int k = 0; k < D::NK; ++k) {
                    const WPair w = w1s[t][k][lane];
#pragma unroll
                    for (int grp = 0; grp < 4; ++grp) {
                        if constexpr (kSplit)
                            acc[grp][h2] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                                w.lo, fe[grp][k], acc[grp][h2], 0, 0, 0);
                        acc[grp][h2] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                            w.hi, fe[grp][k], acc[grp][h2], 0, 0, 0);
                    }
                }
            }
            v8h hh[4];
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                v8f x;
#pragma unroll
                for (int s = 0; s < 8; ++s) x[s] = acc[grp][s / 4][s % 4];
                // ReLU after the rounding to fp16 (monotonic, keeps zero)
                hh[grp] = __builtin_elementwise_max(__builtin_convertvector(x, v8h), zero);
            }
#pragma unroll
            for (int k = 0; k < D::NK; ++k) {
                const WPair w = w2s[pr][k][lane];
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    if constexpr (kSplit)
                        u[grp][k] =
                            __builtin_amdgcn_mfma_f32_16x16x32_f16(w.lo, hh[grp], u[grp][k], 0, 0, 0);
                    u[grp][k] =
                        __builtin_amdgcn_mfma_f32_16x16x32_f16(w.hi, hh[grp], u[grp][k], 0, 0, 0);
                }
            }
        }

        // ---- fire gate, residual, store (out of place) ----
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
            const int z = z0 + lz[grp], y = y0 + ly[grp], x = x0 + lx[grp];
            if (z >= dd || y >= dh || x >= dw) continue;
            const int r = lz[grp] * TY + ly[grp];
            const uint64_t idx0 = ((uint64_t)z * dh + y) * dw + x0;
            const uint64_t off = idx0 + (uint64_t)lx[grp];
            const int k8 = (int)((off >> 3) - (idx0 >> 3));
            const bool fires = (fire_bytes[r][k8] >> (off & 7)) & 1u;
            T *cell = dst + (((int64_t)z * dh + y) * dw + x) * C;
#pragma unroll
            for (int k = 0; k < D::NK; ++k) {
                const int q = 4 * k + g;
                if (q >= D::NQ) continue;
                const float4 s = st[grp][k];
                const v4f du = u[grp][k];
                const float4 out = fires ? make_float4(s.x + du[0], s.y + du[1], s.z + du[2],
                                                       s.w + du[3])
                                         : s;
                store_quad(cell + 4 * q, out);
            }
        }
    }
}

template <typename T, int NDIM, int NIN, int C, int H>
hipError_t launch_gen_t(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    constexpr int TZ = GenTile<NDIM>::TZ, TY = GenTile<NDIM>::TY, TX = GenTile<NDIM>::TX;
    const int64_t tiles_x = (a.ext.w + TX - 1) / TX;
    const int64_t tiles_y = (a.ext.h + TY - 1) / TY;
    const int64_t tiles_z = (a.ext.d + TZ - 1) / TZ;
    const int64_t tiles = tiles_x * tiles_y * tiles_z;
    if (tiles == 0) return hipSuccess;
    if (tiles > INT32_MAX || tiles_x * tiles_y > INT32_MAX) return hipErrorInvalidValue;
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int grid =
        (int)std::min<int64_t>(tiles, (int64_t)std::max(cus, 1) * kGenBlocksPerCu<NDIM, C>);
    nca_step_gen<T, NDIM, NIN, C, H><<<grid, kGenThreads, 0, stream>>>(
        (const T *)src, (T *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, (int)tiles_x,
        (int)tiles_y, (int)tiles, a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step,
        a.batch, a.seed, a.threshold);
    return hipGetLastError();
}

template <typename T, int C, int H>
hipError_t launch_gen_size(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.ndim == 2) {
        if (a.n_in == 1) return launch_gen_t<T, 2, 1, C, H>(a, src, dst, stream);
        if (a.n_in == 3) return launch_gen_t<T, 2, 3, C, H>(a, src, dst, stream);
    } else if (a.ndim == 3) {
        if (a.n_in == 1) return launch_gen_t<T, 3, 1, C, H>(a, src, dst, stream);
        if (a.n_in == 3) return launch_gen_t<T, 3, 3, C, H>(a, src, dst, stream);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_gen_dtype(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.channels == 12 && a.hidden == 48) return launch_gen_size<T, 12, 48>(a, src, dst, stream);
    if (a.channels == 20 && a.hidden == 100) return launch_gen_size<T, 20, 100>(a, src, dst, stream);
    return hipErrorInvalidValue;
}

}  // namespace

bool step_gen_serves(const StepArgs &a) {
    return (a.channels == 12 && a.hidden == 48) || (a.channels == 20 && a.hidden == 100);
}

hipError_t launch_step_gen(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (!step_gen_serves(a)) return hipErrorInvalidValue;
    return a.dtype == Dtype::F32 ? launch_gen_dtype<float>(a, src, dst, stream)
                                 : launch_gen_dtype<__half>(a, src, dst, stream);
}

}  // namespace octnca
