// Memory-bound kernels around the NCA step: image pyramid (node averaging),
// upsample + image injection between levels, two-class readout, fire-mask
// export.  All are single passes over HBM with coalesced 16-byte accesses
// where the layout allows it.
#include <algorithm>
#include <type_traits>

#include "launch.h"

namespace octnca {

namespace {

constexpr int kBlock = 256;

inline unsigned grid_for(int64_t n) { return (unsigned)((n + kBlock - 1) / kBlock); }

// Grids of the pyramid and upsample kernels: x covers the elements of one
// row, y the rows and z the planes (each clamped to the hardware limit of
// those grid dimensions, with the kernels looping over the rest).  The row
// and plane come from the block index, so a thread's index arithmetic is a
// few 32-bit operations (64-bit division per element made these kernels
// instruction-bound).
constexpr int64_t kMaxGridYZ = 65535;

inline dim3 row_grid(int64_t row_elems, int64_t rows, int64_t planes) {
    return dim3((unsigned)((row_elems + kBlock - 1) / kBlock),
                (unsigned)std::min<int64_t>(rows, kMaxGridYZ),
                (unsigned)std::min<int64_t>(planes, kMaxGridYZ));
}

// ---------------------------------------------------------------------------
// Pyramid (Sec. 3.2; supplement S7): one thread per output element (cell, c)
// of a row; the fz*fy*fx inputs are summed in fp32 in (dz, dy, dx) order and
// the sum is divided by their count.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kBlock) void pool_kernel(const T *__restrict__ src,
                                                      T *__restrict__ dst, int dd, int dh, int dw,
                                                      int fz, int fy, int fx, int n_in) {
    const uint32_t i = blockIdx.x * (uint32_t)kBlock + threadIdx.x;   // element in the row
    if ((uint64_t)i >= (uint64_t)dw * n_in) return;
    const uint32_t x = i / (uint32_t)n_in;
    const uint32_t c = i - x * (uint32_t)n_in;
    const int64_t sh = (int64_t)dh * fy, sw = (int64_t)dw * fx;
    const float inv = (float)(fz * fy * fx);
    for (int z = blockIdx.z; z < dd; z += gridDim.z) {
        for (int y = blockIdx.y; y < dh; y += gridDim.y) {
            float acc = 0.f;
            for (int a = 0; a < fz; ++a)
                for (int b = 0; b < fy; ++b) {
                    const int64_t srow = (((int64_t)z * fz + a) * sh + ((int64_t)y * fy + b)) * sw;
                    for (int e = 0; e < fx; ++e) {
                        const int64_t s = srow + (int64_t)x * fx + e;
                        acc += Storage<T>::to_float(src[s * n_in + c]);
                    }
                }
            dst[((int64_t)z * dh + y) * dw * n_in + i] = Storage<T>::from_float(acc / inv);
        }
    }
}

// The same for the common factors (1, 2, 2): one thread per output cell of a
// row, whose 2 x 2 x NIN inputs are 2 NIN consecutive values in each of its
// two input rows (fewer, wider loads than one thread per channel); the sums
// are taken in the same (dy, dx) order, so the results are the same bits.
template <typename T, int NIN>
__global__ __launch_bounds__(kBlock) void pool22_kernel(const T *__restrict__ src,
                                                        T *__restrict__ dst, int dd, int dh,
                                                        int dw) {
    const uint32_t x = blockIdx.x * (uint32_t)kBlock + threadIdx.x;   // output cell in the row
    if (x >= (uint32_t)dw) return;
    const int64_t sw = (int64_t)dw * 2 * NIN;   // values per input row
    for (int z = blockIdx.z; z < dd; z += gridDim.z) {
        for (int y = blockIdx.y; y < dh; y += gridDim.y) {
            const T *r0 = src + ((int64_t)z * dh * 2 + 2 * y) * sw + (int64_t)x * 2 * NIN;
            const T *r1 = r0 + sw;
            float v0[2 * NIN], v1[2 * NIN];
#pragma unroll
            for (int k = 0; k < 2 * NIN; ++k) {
                v0[k] = Storage<T>::to_float(r0[k]);
                v1[k] = Storage<T>::to_float(r1[k]);
            }
            T *out = dst + ((int64_t)z * dh + y) * dw * NIN + (int64_t)x * NIN;
#pragma unroll
            for (int c = 0; c < NIN; ++c) {
                float acc = 0.f;
                acc += v0[c];
                acc += v0[NIN + c];
                acc += v1[c];
                acc += v1[NIN + c];
                out[c] = Storage<T>::from_float(acc / 4.f);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Upsample + inject (Sec. 3.2; supplement S6, Listings 2 and 3): one thread
// per 16-byte chunk of a fine cell of a row (consecutive threads write
// consecutive chunks).
// ---------------------------------------------------------------------------
template <typename T, typename Chunk>
__global__ __launch_bounds__(kBlock) void upsample_kernel(const T *__restrict__ coarse, int fd,
                                                          int fh, int fw, int fz, int fy, int fx,
                                                          const T *__restrict__ img,
                                                          T *__restrict__ fine, int n_in,
                                                          int channels) {
    constexpr int K = (int)(sizeof(Chunk) / sizeof(T));   // channels per chunk
    const int nq = channels / K;                           // chunks per cell
    const uint32_t i = blockIdx.x * (uint32_t)kBlock + threadIdx.x;   // chunk in the row
    if ((uint64_t)i >= (uint64_t)fw * nq) return;
    const uint32_t x = i / (uint32_t)nq;
    const int q = (int)(i - x * (uint32_t)nq);
    const int64_t ch = fh / fy, cw = fw / fx;
    const uint32_t px = x / (uint32_t)fx;
    for (int z = blockIdx.z; z < fd; z += gridDim.z) {
        for (int y = blockIdx.y; y < fh; y += gridDim.y) {
            const int64_t cell = ((int64_t)z * fh + y) * fw + x;
            Chunk v = {};
            if (coarse != nullptr) {
                const int64_t parent = ((int64_t)(z / fz) * ch + y / fy) * cw + px;
                v = reinterpret_cast<const Chunk *>(coarse + parent * channels)[q];
            }
            if (q * K < n_in) {
                // this chunk holds input channels: overwrite them with the level's image
                T vals[K];
                __builtin_memcpy(vals, &v, sizeof(v));
                for (int k = 0; k < K && q * K + k < n_in; ++k) vals[k] = img[cell * n_in + q * K + k];
                __builtin_memcpy(&v, vals, sizeof(v));
            }
            reinterpret_cast<Chunk *>(fine + cell * channels)[q] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// K-class readout (several classes, as in the paper's surgery data, Sec. 4):
// seg = index k in [0, K) of the largest of state[C-K+k], scanning k upwards
// and moving only on a strictly greater value (ties to the lower class; a NaN
// never replaces an earlier channel).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kBlock) void readout_classes_kernel(const T *__restrict__ state,
                                                                 int64_t cells, int channels,
                                                                 int classes,
                                                                 uint8_t *__restrict__ seg) {
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= cells) return;
    const T *s = state + p * channels + (channels - classes);
    float best = Storage<T>::to_float(s[0]);
    int best_k = 0;
    for (int k = 1; k < classes; ++k) {
        const float v = Storage<T>::to_float(s[k]);
        if (v > best) {
            best = v;
            best_k = k;
        }
    }
    seg[p] = (uint8_t)best_k;
}

// ---------------------------------------------------------------------------
// Readout (Sec. 3.2): seg = state[C-1] > state[C-2].
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kBlock) void readout_kernel(const T *__restrict__ state,
                                                         int64_t cells, int channels,
                                                         uint8_t *__restrict__ seg) {
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= cells) return;
    const float a = Storage<T>::to_float(state[p * channels + channels - 2]);
    const float b = Storage<T>::to_float(state[p * channels + channels - 1]);
    seg[p] = (b > a) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void fire_mask_kernel(uint64_t seed, uint32_t level,
                                                           uint32_t step, int64_t cells,
                                                           uint64_t threshold,
                                                           uint8_t *__restrict__ mask) {
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= cells) return;
    mask[p] = cell_fires(seed, level, step, 0, (uint64_t)p, threshold) ? 1 : 0;
}

}  // namespace

hipError_t launch_pool(Dtype dt, const void *src, Extent3 e, void *dst, int fz, int fy, int fx,
                       int n_in, hipStream_t stream) {
    if (e.cells() == 0) return hipSuccess;
    if (fz == 1 && fy == 2 && fx == 2 && (n_in == 1 || n_in == 3)) {
        const dim3 g22 = row_grid(e.w, e.h, e.d);
        auto go = [&](auto tag, auto nin) {
            using T = decltype(tag);
            pool22_kernel<T, decltype(nin)::value><<<g22, kBlock, 0, stream>>>(
                (const T *)src, (T *)dst, (int)e.d, (int)e.h, (int)e.w);
        };
        if (dt == Dtype::F32) {
            if (n_in == 1) go(float{}, std::integral_constant<int, 1>{});
            else go(float{}, std::integral_constant<int, 3>{});
        } else {
            if (n_in == 1) go(__half{}, std::integral_constant<int, 1>{});
            else go(__half{}, std::integral_constant<int, 3>{});
        }
        return hipGetLastError();
    }
    const dim3 grid = row_grid(e.w * n_in, e.h, e.d);
    if (dt == Dtype::F32)
        pool_kernel<float><<<grid, kBlock, 0, stream>>>((const float *)src, (float *)dst,
                                                         (int)e.d, (int)e.h, (int)e.w, fz, fy, fx,
                                                         n_in);
    else
        pool_kernel<__half><<<grid, kBlock, 0, stream>>>((const __half *)src, (__half *)dst,
                                                          (int)e.d, (int)e.h, (int)e.w, fz, fy,
                                                          fx, n_in);
    return hipGetLastError();
}

hipError_t launch_upsample(Dtype dt, const void *coarse, Extent3 e, int fz, int fy, int fx,
                           const void *img, void *fine, int n_in, int channels,
                           hipStream_t stream) {
    if (e.cells() == 0) return hipSuccess;
    const int esize = dt == Dtype::F32 ? 4 : 2;
    const bool wide = (channels * esize) % 16 == 0;         // 16-byte chunks, else 8-byte
    const int nq = channels * esize / (wide ? 16 : 8);
    const dim3 grid = row_grid(e.w * nq, e.h, e.d);
    auto go = [&](auto tag, auto chunk) -> hipError_t {
        using T = decltype(tag);
        using Chunk = decltype(chunk);
        upsample_kernel<T, Chunk><<<grid, kBlock, 0, stream>>>(
            (const T *)coarse, (int)e.d, (int)e.h, (int)e.w, fz, fy, fx, (const T *)img,
            (T *)fine, n_in, channels);
        return hipGetLastError();
    };
    if (dt == Dtype::F32) return wide ? go(float{}, uint4{}) : go(float{}, uint2{});
    return wide ? go(__half{}, uint4{}) : go(__half{}, uint2{});
}

hipError_t launch_readout(Dtype dt, const void *state, int64_t cells, int channels, uint8_t *seg,
                          hipStream_t stream) {
    if (cells == 0) return hipSuccess;
    if (dt == Dtype::F32)
        readout_kernel<float><<<grid_for(cells), kBlock, 0, stream>>>((const float *)state,
                                                                      cells, channels, seg);
    else
        readout_kernel<__half><<<grid_for(cells), kBlock, 0, stream>>>((const __half *)state,
                                                                       cells, channels, seg);
    return hipGetLastError();
}

hipError_t launch_readout_classes(Dtype dt, const void *state, int64_t cells, int channels,
                                  int classes, uint8_t *seg, hipStream_t stream) {
    if (cells == 0) return hipSuccess;
    if (dt == Dtype::F32)
        readout_classes_kernel<float><<<grid_for(cells), kBlock, 0, stream>>>(
            (const float *)state, cells, channels, classes, seg);
    else
        readout_classes_kernel<__half><<<grid_for(cells), kBlock, 0, stream>>>(
            (const __half *)state, cells, channels, classes, seg);
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
