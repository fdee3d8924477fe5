// Device-side building blocks shared by the OctreeNCA kernels: the fire-mask
// generator and the storage-type traits.  Internal header (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace octnca {

constexpr int kC = 16;   // state channels (supplement S3: fixed at compile time)
constexpr int kH = 64;   // hidden units of the per-cell MLP

// ---------------------------------------------------------------------------
// Fire mask: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random
// Numbers: As Easy as 1, 2, 3", SC 2011).  The paper only asks for a 50%
// Bernoulli gate per cell and step (Sec. 3.1); a counter-based generator makes
// the gate a pure function of (seed, level, step, cell), independent of launch
// shape.  Counter (idx >> 3, step, level, batch), key (seed, 0): one call
// covers 8 consecutive cells, cell idx takes the upper (odd idx) or lower
// (even idx) 32 bits of output word (idx >> 1) & 3 and fires iff that draw is
// below the threshold T = min(2^32, floor(rate * 2^32)).  batch is the image's
// index in a batch (0 for a single image).
// ---------------------------------------------------------------------------
struct Philox4x64Out {
    uint64_t w[4];
};

// 64 x 64 -> 128-bit product as (hi, lo), from four 32 x 32 -> 64-bit
// products with 64-bit addends (one multiply-add each; no partial sum
// overflows: (2^32 - 1)^2 + 2 (2^32 - 1) < 2^64).
__device__ __forceinline__ void mul_wide_u64(uint64_t a, uint64_t b, uint64_t &hi, uint64_t &lo) {
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t p0 = (uint64_t)a0 * b0;
    const uint64_t t1 = (uint64_t)a0 * b1 + (p0 >> 32);
    const uint64_t t2 = (uint64_t)a1 * b0 + (uint32_t)t1;
    lo = (t2 << 32) | (uint32_t)p0;
    hi = (uint64_t)a1 * b1 + (t1 >> 32) + (t2 >> 32);
}

__device__ __forceinline__ Philox4x64Out philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                                       uint64_t c3, uint64_t k0, uint64_t k1) {
    // Round multipliers and key increments of the 4x64 variant (SC 2011, Table 2).
    const uint64_t mul_a = 0xD2E7470EE14C6C93ull;   // applied to word 0
    const uint64_t mul_b = 0xCA5A826395121157ull;   // applied to word 2
    const uint64_t bump_a = 0x9E3779B97F4A7C15ull;  // golden ratio
    const uint64_t bump_b = 0xBB67AE8584CAA73Bull;  // sqrt(3) - 1
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        uint64_t hi_a, lo_a, hi_b, lo_b;
        mul_wide_u64(mul_a, c0, hi_a, lo_a);
        mul_wide_u64(mul_b, c2, hi_b, lo_b);
        const uint64_t n0 = hi_b ^ c1 ^ k0;
        const uint64_t n2 = hi_a ^ c3 ^ k1;
        c0 = n0;
        c1 = lo_b;
        c2 = n2;
        c3 = lo_a;
        k0 += bump_a;
        k1 += bump_b;
    }
    return Philox4x64Out{{c0, c1, c2, c3}};
}

// Fire bit of the cell with canonical index `idx` = (z*h + y)*w + x: block
// (idx >> 3), word (idx >> 1) & 3, upper 32 bits for odd idx, lower for even.
__device__ __forceinline__ uint32_t draw_of(const Philox4x64Out &r, uint32_t cell_in_block) {
    const uint32_t k = (cell_in_block >> 1) & 3u;
    const uint64_t lo = (k & 1u) ? r.w[1] : r.w[0];
    const uint64_t hi = (k & 1u) ? r.w[3] : r.w[2];
    const uint64_t w = (k & 2u) ? hi : lo;
    return (cell_in_block & 1u) ? (uint32_t)(w >> 32) : (uint32_t)w;
}

__device__ __forceinline__ bool cell_fires(uint64_t seed, uint32_t level, uint32_t step,
                                           uint32_t batch, uint64_t idx, uint64_t threshold) {
    const Philox4x64Out r = philox4x64_10(idx >> 3, step, level, batch, seed, 0);
    return (uint64_t)draw_of(r, (uint32_t)idx & 7u) < threshold;
}

// ---------------------------------------------------------------------------
// Storage traits: a cell's C channels are moved in 16-byte chunks.
// ---------------------------------------------------------------------------
template <typename T> struct Storage;

template <> struct Storage<float> {
    static constexpr int kPerChunk = 4;               // channels per 16-byte chunk
    __device__ static inline void unpack(const uint4 &v, float *out) {
        out[0] = __uint_as_float(v.x);
        out[1] = __uint_as_float(v.y);
        out[2] = __uint_as_float(v.z);
        out[3] = __uint_as_float(v.w);
    }
    __device__ static inline uint4 pack(const float *in) {
        return make_uint4(__float_as_uint(in[0]), __float_as_uint(in[1]),
                          __float_as_uint(in[2]), __float_as_uint(in[3]));
    }
    __device__ static inline float to_float(float v) { return v; }
    __device__ static inline float from_float(float v) { return v; }
};

template <> struct Storage<__half> {
    static constexpr int kPerChunk = 8;
    __device__ static inline void unpack_pair(uint32_t u, float &a, float &b) {
        a = __half2float(__ushort_as_half((unsigned short)(u & 0xffffu)));
        b = __half2float(__ushort_as_half((unsigned short)(u >> 16)));
    }
    __device__ static inline uint32_t pack_pair(float a, float b) {
        const uint32_t lo = __half_as_ushort(__float2half_rn(a));
        const uint32_t hi = __half_as_ushort(__float2half_rn(b));
        return lo | (hi << 16);
    }
    __device__ static inline void unpack(const uint4 &v, float *out) {
        unpack_pair(v.x, out[0], out[1]);
        unpack_pair(v.y, out[2], out[3]);
        unpack_pair(v.z, out[4], out[5]);
        unpack_pair(v.w, out[6], out[7]);
    }
    __device__ static inline uint4 pack(const float *in) {
        return make_uint4(pack_pair(in[0], in[1]), pack_pair(in[2], in[3]),
                          pack_pair(in[4], in[5]), pack_pair(in[6], in[7]));
    }
    __device__ static inline float to_float(__half v) { return __half2float(v); }
    __device__ static inline __half from_float(float v) { return __float2half_rn(v); }
};

// Kernel-argument view of one level's weights (device pointers, fp32).
struct LevelWeightsDev {
    const float *conv_w;   // [C][taps]
    const float *conv_b;   // [C]
    const float *w1;       // [H][2C]
    const float *b1;       // [H]
    const float *w2;       // [C][H]
};

// Gradients of one level's weights (same layouts), accumulated by the backward.
struct LevelGradsDev {
    float *conv_w;
    float *conv_b;
    float *w1;
    float *b1;
    float *w2;
};

}  // namespace octnca
