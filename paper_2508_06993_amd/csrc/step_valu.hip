// Fused NCA step, plain VALU version (Sec. 3.1; supplement S3, Listing 1):
// one thread per cell.  The block's cells plus a one-cell halo are staged in
// LDS once; each thread then forms its 2C features (own state, depthwise
// perception with zero padding), runs the MLP 2C -> H -> C in registers with
// the hidden units streamed one at a time (no hidden activation ever leaves
// the thread), applies its fire bit and writes the new state to the other
// buffer (out of place, supplement S3).  Weights are wave-uniform and are
// read through the scalar data cache.
#include "launch.h"

namespace octnca {

namespace {

template <int NDIM> struct ValuTile;
template <> struct ValuTile<2> { static constexpr int TZ = 1, TY = 8, TX = 32; };
template <> struct ValuTile<3> { static constexpr int TZ = 4, TY = 8, TX = 8; };

constexpr int kValuThreads = 256;

template <typename T, int NDIM, int NIN>
__global__ __launch_bounds__(kValuThreads) void nca_step_valu(
    const T *__restrict__ src, T *__restrict__ dst, int dd, int dh, int dw, int tiles_x,
    int tiles_y, const float *__restrict__ conv_w, const float *__restrict__ conv_b,
    const float *__restrict__ w1, const float *__restrict__ b1, const float *__restrict__ w2,
    uint32_t level, uint32_t step, uint32_t batch, uint64_t seed, uint64_t threshold) {
    using S = Storage<T>;
    constexpr int K = S::kPerChunk;                 // channels per 16-byte chunk
    constexpr int NQ = kC / K;                      // chunks per cell
    constexpr int TZ = ValuTile<NDIM>::TZ, TY = ValuTile<NDIM>::TY, TX = ValuTile<NDIM>::TX;
    constexpr int HZ = NDIM == 3 ? TZ + 2 : 1, HY = TY + 2, HX = TX + 2;
    constexpr int NCELL = HZ * HY * HX;
    constexpr int TAPS = NDIM == 3 ? 27 : 9;
    static_assert(TZ * TY * TX == kValuThreads, "one thread per tile cell");

    // Halo'd tile, one plane per chunk so that neighbouring threads read
    // neighbouring 16-byte words (no bank conflicts).
    __shared__ uint4 tile[NQ][NCELL];

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
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (gx >= 0 && gx < dw && gy >= 0 && gy < dh && gz >= 0 && gz < dd) {
            const int64_t g = ((int64_t)gz * dh + gy) * dw + gx;
            v = reinterpret_cast<const uint4 *>(src + g * kC)[q];
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
    float f[2 * kC];
#pragma unroll
    for (int q = 0; q < NQ; ++q) S::unpack(tile[q][centre], f + q * K);
#pragma unroll
    for (int c = 0; c < kC; ++c) f[kC + c] = conv_b[c];
#pragma unroll
    for (int t = 0; t < TAPS; ++t) {
        const int dz = NDIM == 3 ? t / 9 - 1 : 0;
        const int dy = (t / 3) % 3 - 1;
        const int dx = t % 3 - 1;
        const int nb = centre + (dz * HY + dy) * HX + dx;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            float v[K];
            S::unpack(tile[q][nb], v);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int c = q * K + k;
                f[kC + c] = fmaf(conv_w[c * TAPS + t], v[k], f[kC + c]);
            }
        }
    }

    // MLP 2C -> H (bias, ReLU) -> C (no bias), hidden units streamed
    float u[kC];
#pragma unroll
    for (int c = 0; c < kC; ++c) u[c] = 0.f;
#pragma unroll 4
    for (int j = 0; j < kH; ++j) {
        float a = b1[j];
#pragma unroll
        for (int k = 0; k < 2 * kC; ++k) a = fmaf(w1[j * 2 * kC + k], f[k], a);
        a = fmaxf(a, 0.f);
#pragma unroll
        for (int c = NIN; c < kC; ++c) u[c] = fmaf(w2[c * kH + j], a, u[c]);
    }

    const int64_t idx = ((int64_t)z * dh + y) * dw + x;
    const bool fire = cell_fires(seed, level, step, batch, (uint64_t)idx, threshold);
    float out[kC];
#pragma unroll
    for (int c = 0; c < kC; ++c) out[c] = (c >= NIN && fire) ? f[c] + u[c] : f[c];
#pragma unroll
    for (int q = 0; q < NQ; ++q)
        reinterpret_cast<uint4 *>(dst + idx * kC)[q] = S::pack(out + q * K);
}

template <typename T, int NDIM, int NIN>
hipError_t launch_valu(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    using Tile = ValuTile<NDIM>;
    const int tiles_x = (int)((a.ext.w + Tile::TX - 1) / Tile::TX);
    const int tiles_y = (int)((a.ext.h + Tile::TY - 1) / Tile::TY);
    const int tiles_z = (int)((a.ext.d + Tile::TZ - 1) / Tile::TZ);
    const int64_t blocks = (int64_t)tiles_x * tiles_y * tiles_z;
    if (blocks == 0) return hipSuccess;
    nca_step_valu<T, NDIM, NIN><<<(unsigned)blocks, kValuThreads, 0, stream>>>(
        (const T *)src, (T *)dst, (int)a.ext.d, (int)a.ext.h, (int)a.ext.w, tiles_x, tiles_y,
        a.w.conv_w, a.w.conv_b, a.w.w1, a.w.b1, a.w.w2, a.level, a.step, a.batch, a.seed, a.threshold);
    return hipGetLastError();
}

template <typename T, int NDIM>
hipError_t dispatch_nin(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    switch (a.n_in) {
        case 1: return launch_valu<T, NDIM, 1>(a, src, dst, stream);
        case 3: return launch_valu<T, NDIM, 3>(a, src, dst, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_step_valu(const StepArgs &a, const void *src, void *dst, hipStream_t stream) {
    if (a.dtype == Dtype::F32)
        return a.ndim == 2 ? dispatch_nin<float, 2>(a, src, dst, stream)
                           : dispatch_nin<float, 3>(a, src, dst, stream);
    return a.ndim == 2 ? dispatch_nin<__half, 2>(a, src, dst, stream)
                       : dispatch_nin<__half, 3>(a, src, dst, stream);
}

}  // namespace octnca
