// Fused NCA step, plain VALU version (Sec. 3.1; supplement S3, Listing 1):
// one thread per cell.  The block's cells plus a one-cell halo are staged in
// LDS once; each thread then forms its 2C features (own state, depthwise
// perception with zero padding), runs the MLP 2C -> H -> C in registers with
// the hidden units streamed one at a time (no hidden activation ever leaves
// the thread), applies its fire bit and writes the new state to the other
// buffer (out of place, supplement S3).  Weights are wave-uniform and are
// read through the scalar data cache.
#include <type_traits>

#include "launch.h"

namespace octnca {

namespace {

// A cell's C channels move in chunks of 16 bytes, or of 8 bytes when C
// channels of T are not a whole number of 16-byte chunks (fp16 with C = 12 or
// 20).  Chunk values are converted to fp32 element by element.
template <typename T, int C>
struct CellIO {
    using Chunk = std::conditional_t<(C * sizeof(T)) % 16 == 0, uint4, uint2>;
    static constexpr int K = (int)(sizeof(Chunk) / sizeof(T));   // channels per chunk
    static constexpr int NQ = C / K;                              // chunks per cell
    static_assert(NQ * K == C, "whole chunks per cell");
    __device__ static __forceinline__ void unpack(const Chunk &c, float *out) {
        T v[K];
        __builtin_memcpy(v, &c, sizeof(c));
#pragma unroll
        for (int k = 0; k < K; ++k) out[k] = Storage<T>::to_float(v[k]);
    }
    __device__ static __forceinline__ Chunk pack(const float *in) {
        T v[K];
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = Storage<T>::from_float(in[k]);
        Chunk c;
        __builtin_memcpy(&c, v, sizeof(c));
        return c;
    }
};

template <int NDIM> struct ValuTile;
template <> struct ValuTile<2> { static constexpr int TZ = 1, TY = 8, TX = 32; };
template <> struct ValuTile<3> { static constexpr int TZ = 4, TY = 8, TX = 8; };

constexpr int kValuThreads = 256;

template <typename T, int NDIM, int NIN, int C, int H>
__global__ __launch_bounds__(kValuThreads) void nca_step_valu(
    const T *__restrict__ src, T *__restrict__ dst, int dd, int dh, int dw, int tiles_x,
    int tiles_y, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold) {
    using IO = CellIO<T, C>;
    using Chunk = typename IO::Chunk;
    constexpr int K = IO::K;                        // channels per chunk
    constexpr int NQ = IO::NQ;                      // chunks per cell
    constexpr int TZ = ValuTile<NDIM>::TZ, TY = ValuTile<NDIM>::TY, TX = ValuTile<NDIM>::TX;
    constexpr int HZ = NDIM == 3 ? TZ + 2 : 1, HY = TY + 2, HX = TX + 2;
    constexpr int NCELL = HZ * HY * HX;
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    static_assert(TZ * TY * TX == kValuThreads, "one thread per tile cell");

    // Halo'd tile, one plane per chunk so that neighbouring threads read
    // neighbouring 16-byte words (no bank conflicts).
    __shared__ Chunk tile[NQ][NCELL];

    int b = blockIdx.x;
    const int bx = b % tiles_x;
    b /= tiles_x;
    const int by = b % tiles_y;
    const int bz = b / tiles_y;
    const int x0 = bx * TX, y0 = by * TY, z0 = bz * TZ;

    for (int i = threadIdx.x; i < NCELL * NQ; i += kValuThreads) {
        const int q = i % NQ;
        const int cell = i / NQ;
        const int lx = cell % HX;
        const int ly = (cell / HX) % HY;
        const int lz = cell / (HX * HY);
        const int gx = x0 + lx - 1, gy = y0 + ly - 1;
        const int gz = NDIM == 3 ? z0 + lz - 1 : 0;
        Chunk v = {};
        if (gx >= 0 && gx < dw && gy >= 0 && gy < dh && gz >= 0 && gz < dd) {
            const int64_t g = ((int64_t)gz * dh + gy) * dw + gx;
            v = reinterpret_cast<const Chunk *>(src + g * C)[q];
        }
        tile[q][cell] = v;
    }
    __syncthreads();

    const int tx = threadIdx.x % TX;
    const int ty = (threadIdx.x / TX) % TY;
    const int tz = threadIdx.x / (TX * TY);
    const int x = x0 + tx, y = y0 + ty, z = z0 + tz;
    if (x >= dw || y >= dh || z >= dd) return;

    const int centre = ((tz + (NDIM == 3 ? 1 : 0)) * HY + ty + 1) * HX + tx + 1;

    // features: f[0..C) = own state, f[C..2C) = perception
    float f[2 * C];
#pragma unroll
    for (int q = 0; q < NQ; ++q) IO::unpack(tile[q][centre], f + q * K);
#pragma unroll
    for (int c = 0; c < C; ++c) f[C + c] = conv_b[c];
#pragma unroll
    for (int t = 0; t < TAPS; ++t) {
        const int dz = NDIM == 3 ? t / 9 - 1 : 0;
        const int dy = (t / 3) % 3 - 1;
        const int dx = t % 3 - 1;
        const int nb = centre + (dz * HY + dy) * HX + dx;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            float v[K];
            IO::unpack(tile[q][nb], v);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int c = q * K + k;
                f[C + c] = fmaf(conv_w[c * TAPS + t], v[k], f[C + c]);
            }
        }
    }

    // MLP 2C -> H (bias, ReLU) -> C (no bias), hidden units streamed
    float u[C];
#pragma unroll
    for (int c = 0; c < C; ++c) u[c] = 0.f;
#pragma unroll 4
    for (int j = 0; j < H; ++j) {
        float a = b1[j];
#pragma unroll
        for (int k = 0; k < 2 * C; ++k) a = fmaf(w1[j * 2 * C + k], f[k], a);
        a = fmaxf(a, 0.f);
#pragma unroll
        for (int c = NIN; c < C; ++c) u[c] = fmaf(w2[c * H + j], a, u[c]);
    }

    const int64_t idx = ((int64_t)z * dh + y) * dw + x;
    const bool fire = cell_fires(seed, level, step, batch, (uint64_t)idx, threshold);
    float out[C];
#pragma unroll
    for (int c = 0; c < C; ++c) out[c] = (c >= NIN && fire) ? f[c] + u[c] : f[c];
#pragma unroll
    for (int q = 0; q < NQ; ++q)
        reinterpret_cast<Chunk *>(dst + idx * C)[q] = IO::pack(out + q * K);
}

template <typename T, int NDIM, int NIN, int C, int H>
hipError_t launch_valu(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    using Tile = ValuTile<NDIM>;
    const int tiles_x = (int)((a.ext.w + Tile::TX - 1) / Tile::TX);
    const int tiles_y = (int)((a.ext.h + Tile::TY - 1) / Tile::TY);
    const int tiles_z = (int)((a.ext.d + Tile::TZ - 1) / Tile::TZ);
    const int64_t blocks = (int64_t)tiles_x * tiles_y * tiles_z;
    if (blocks == 0) return hipSuccess;
    nca_step_valu<T, NDIM, NIN, C, H><<<(unsigned)blocks, kValuThreads, 0, stream>>>(
        (const T *)src, (T *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, tiles_x, tiles_y,
        a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch, a.seed,
        a.threshold);
    return hipGetLastError();
}

template <typename T, int NDIM, int C, int H>
hipError_t dispatch_nin(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    switch (a.n_in) {
        case 1: return launch_valu<T, NDIM, 1, C, H>(a, src, dst, stream);
        case 3: return launch_valu<T, NDIM, 3, C, H>(a, src, dst, stream);
        default: return hipErrorInvalidValue;
    }
}

// model sizes: the paper's 16/64 and the two of its ablation (supplement S10)
template <typename T, int NDIM>
hipError_t dispatch_size(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.channels == 16 && a.hidden == 64) return dispatch_nin<T, NDIM, 16, 64>(a, src, dst, stream);
    if (a.channels == 12 && a.hidden == 48) return dispatch_nin<T, NDIM, 12, 48>(a, src, dst, stream);
    if (a.channels == 20 && a.hidden == 100)
        return dispatch_nin<T, NDIM, 20, 100>(a, src, dst, stream);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_step_valu(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.dtype == Dtype::F32)
        return a.ndim == 2 ? dispatch_size<float, 2>(a, src, dst, stream)
                           : dispatch_size<float, 3>(a, src, dst, stream);
    return a.ndim == 2 ? dispatch_size<__half, 2>(a, src, dst, stream)
                       : dispatch_size<__half, 3>(a, src, dst, stream);
}

}  // namespace octnca
