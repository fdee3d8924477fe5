// Memory-bound kernels around the NCA step: image pyramid (node averaging),
// upsample + image injection between levels, two-class readout, fire-mask
// export.  All are single passes over HBM with coalesced 16-byte accesses
// where the layout allows it.
#include "launch.h"

namespace octnca {

namespace {

constexpr int kBlock = 256;

inline unsigned grid_for(int64_t n) { return (unsigned)((n + kBlock - 1) / kBlock); }

// ---------------------------------------------------------------------------
// Pyramid (Sec. 3.2; supplement S7): one thread per output element (cell, c).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kBlock) void pool_kernel(const T *__restrict__ src,
                                                      T *__restrict__ dst, int64_t dd, int64_t dh,
                                                      int64_t dw, int fz, int fy, int fx,
                                                      int n_in) {
    const int64_t total = dd * dh * dw * n_in;
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= total) return;
    const int c = (int)(i % n_in);
    const int64_t cell = i / n_in;
    const int64_t x = cell % dw;
    const int64_t y = (cell / dw) % dh;
    const int64_t z = cell / (dw * dh);
    const int64_t sh = dh * fy, sw = dw * fx;
    float acc = 0.f;
    for (int a = 0; a < fz; ++a)
        for (int b = 0; b < fy; ++b)
            for (int e = 0; e < fx; ++e) {
                const int64_t s = ((z * fz + a) * sh + (y * fy + b)) * sw + (x * fx + e);
                acc += Storage<T>::to_float(src[s * n_in + c]);
            }
    dst[i] = Storage<T>::from_float(acc / (float)(fz * fy * fx));
}

// ---------------------------------------------------------------------------
// Upsample + inject (Sec. 3.2; supplement S6, Listings 2 and 3): one thread
// per 16-byte chunk of a fine cell.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kBlock) void upsample_kernel(const T *__restrict__ coarse,
                                                          int64_t fd, int64_t fh, int64_t fw,
                                                          int fz, int fy, int fx,
                                                          const T *__restrict__ img,
                                                          T *__restrict__ fine, int n_in) {
    constexpr int K = Storage<T>::kPerChunk;
    constexpr int NQ = kC / K;
    const int64_t total = fd * fh * fw * NQ;
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= total) return;
    const int q = (int)(i % NQ);
    const int64_t cell = i / NQ;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (coarse != nullptr) {
        const int64_t x = cell % fw;
        const int64_t y = (cell / fw) % fh;
        const int64_t z = cell / (fw * fh);
        const int64_t ch = fh / fy, cw = fw / fx;
        const int64_t parent = ((z / fz) * ch + (y / fy)) * cw + (x / fx);
        v = reinterpret_cast<const uint4 *>(coarse + parent * kC)[q];
    }
    if (q * K < n_in) {
        // this chunk holds input channels: overwrite them with the level's image
        T vals[K];
        __builtin_memcpy(vals, &v, sizeof(v));
        for (int k = 0; k < K && q * K + k < n_in; ++k) vals[k] = img[cell * n_in + q * K + k];
        __builtin_memcpy(&v, vals, sizeof(v));
    }
    reinterpret_cast<uint4 *>(fine + cell * kC)[q] = v;
}

// ---------------------------------------------------------------------------
// Readout (Sec. 3.2): seg = state[C-1] > state[C-2].
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kBlock) void readout_kernel(const T *__restrict__ state,
                                                         int64_t cells,
                                                         uint8_t *__restrict__ seg) {
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= cells) return;
    const float a = Storage<T>::to_float(state[p * kC + kC - 2]);
    const float b = Storage<T>::to_float(state[p * kC + kC - 1]);
    seg[p] = (b > a) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void fire_mask_kernel(uint64_t seed, uint32_t level,
                                                           uint32_t step, int64_t cells,
                                                           uint64_t threshold,
                                                           uint8_t *__restrict__ mask) {
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= cells) return;
    mask[p] = cell_fires(seed, level, step, (uint64_t)p, threshold) ? 1 : 0;
}

}  // namespace

hipError_t launch_pool(Dtype dt, const void *src, Extent3 e, void *dst, int fz, int fy, int fx,
                       int n_in, hipStream_t stream) {
    const int64_t n = e.cells() * n_in;
    if (n == 0) return hipSuccess;
    if (dt == Dtype::F32)
        pool_kernel<float><<<grid_for(n), kBlock, 0, stream>>>(
            (const float *)src, (float *)dst, e.d, e.h, e.w, fz, fy, fx, n_in);
    else
        pool_kernel<__half><<<grid_for(n), kBlock, 0, stream>>>(
            (const __half *)src, (__half *)dst, e.d, e.h, e.w, fz, fy, fx, n_in);
    return hipGetLastError();
}

hipError_t launch_upsample(Dtype dt, const void *coarse, Extent3 e, int fz, int fy, int fx,
                           const void *img, void *fine, int n_in, hipStream_t stream) {
    const int nq = dt == Dtype::F32 ? kC / 4 : kC / 8;
    const int64_t n = e.cells() * nq;
    if (n == 0) return hipSuccess;
    if (dt == Dtype::F32)
        upsample_kernel<float><<<grid_for(n), kBlock, 0, stream>>>(
            (const float *)coarse, e.d, e.h, e.w, fz, fy, fx, (const float *)img, (float *)fine,
            n_in);
    else
        upsample_kernel<__half><<<grid_for(n), kBlock, 0, stream>>>(
            (const __half *)coarse, e.d, e.h, e.w, fz, fy, fx, (const __half *)img,
            (__half *)fine, n_in);
    return hipGetLastError();
}

hipError_t launch_readout(Dtype dt, const void *state, int64_t cells, uint8_t *seg,
                          hipStream_t stream) {
    if (cells == 0) return hipSuccess;
    if (dt == Dtype::F32)
        readout_kernel<float><<<grid_for(cells), kBlock, 0, stream>>>((const float *)state,
                                                                      cells, seg);
    else
        readout_kernel<__half><<<grid_for(cells), kBlock, 0, stream>>>((const __half *)state,
                                                                       cells, seg);
    return hipGetLastError();
}

hipError_t launch_fire_mask(uint64_t seed, uint32_t level, uint32_t step, int64_t cells,
                            uint64_t threshold, uint8_t *mask, hipStream_t stream) {
    if (cells == 0) return hipSuccess;
    fire_mask_kernel<<<grid_for(cells), kBlock, 0, stream>>>(seed, level, step, cells, threshold,
                                                              mask);
    return hipGetLastError();
}

}  // namespace octnca
