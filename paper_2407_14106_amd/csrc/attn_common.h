// Helpers shared by the attention kernels: per-lane feature slices of bf16 or
// fp32 rows, dot products with fp32 accumulation, and the (dtype, d, H)
// dispatch.
#pragma once

#include "common.h"

namespace gt {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Lane layout of the edge kernels: each (node, head) is owned by L = D / F
// consecutive lanes, each holding F consecutive features (32 bytes of bf16, 64
// of fp32), which keeps the per-lane register footprint small enough for
// several resident wavefronts per SIMD to overlap their gathers.
template <typename T, int D, int H>
struct EdgeCfg {
    static constexpr int F = 16;                        // features per lane
    static constexpr int L = D / F;                     // lanes per (node, head)
    static constexpr int G = H * L;                     // lanes per node
    static constexpr int NPW = kWave / G;               // nodes per wavefront
    static_assert(D % F == 0 && G <= kWave && kWave % G == 0, "unsupported (d, H)");
};

// F features of one row slice, stored packed as loaded.
template <typename T, int F>
struct Slice;

template <int F>
struct Slice<uint16_t, F> {
    uint32_t w[F / 2];
    __device__ __forceinline__ void load(const uint16_t* p) {
        const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
        for (int i = 0; i < F / 8; ++i) {
            uint4 v = q[i];
            w[4 * i + 0] = v.x;
            w[4 * i + 1] = v.y;
            w[4 * i + 2] = v.z;
            w[4 * i + 3] = v.w;
        }
    }
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int i = 0; i < F / 2; ++i) w[i] = 0;
    }
    __device__ __forceinline__ float f(int i) const { return (i & 1) ? bf16hi(w[i >> 1]) : bf16lo(w[i >> 1]); }
    __device__ __forceinline__ float dot(const Slice& o) const {
        float a0 = 0.f, a1 = 0.f;
#pragma unroll
        for (int i = 0; i < F / 2; i += 2) {
            a0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[i]),
                                                 __builtin_bit_cast(bf16x2_t, o.w[i]), a0, false);
            a1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[i + 1]),
                                                 __builtin_bit_cast(bf16x2_t, o.w[i + 1]), a1, false);
        }
        return a0 + a1;
    }
    // acc[2i] += p * lo(w[i]), acc[2i+1] += p * hi(w[i]) with p given as the
    // bf16 pairs (p, 0) and (0, p): one dot2 per element, no conversion.
    __device__ __forceinline__ void axpy_w(float (&acc)[F], uint32_t p_lo, uint32_t p_hi) const {
#pragma unroll
        for (int i = 0; i < F / 2; ++i) {
            const bf16x2_t x = __builtin_bit_cast(bf16x2_t, w[i]);
            acc[2 * i] = __builtin_amdgcn_fdot2_f32_bf16(x, __builtin_bit_cast(bf16x2_t, p_lo), acc[2 * i], false);
            acc[2 * i + 1] =
                __builtin_amdgcn_fdot2_f32_bf16(x, __builtin_bit_cast(bf16x2_t, p_hi), acc[2 * i + 1], false);
        }
    }
};

template <int F>
struct Slice<float, F> {
    float w[F];
    __device__ __forceinline__ void load(const float* p) {
        const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
        for (int i = 0; i < F / 4; ++i) {
            float4 v = q[i];
            w[4 * i + 0] = v.x;
            w[4 * i + 1] = v.y;
            w[4 * i + 2] = v.z;
            w[4 * i + 3] = v.w;
        }
    }
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int i = 0; i < F; ++i) w[i] = 0.f;
    }
    __device__ __forceinline__ float f(int i) const { return w[i]; }
    __device__ __forceinline__ float dot(const Slice& o) const {
        float a0 = 0.f, a1 = 0.f;
#pragma unroll
        for (int i = 0; i < F; i += 2) {
            a0 = fmaf(w[i], o.w[i], a0);
            a1 = fmaf(w[i + 1], o.w[i + 1], a1);
        }
        return a0 + a1;
    }
};

// acc[i] += p * x[i]
template <typename T, int F>
__device__ __forceinline__ void axpy(float (&acc)[F], float p, const Slice<T, F>& x) {
#pragma unroll
    for (int i = 0; i < F; ++i) acc[i] = fmaf(p, x.f(i), acc[i]);
}

// Store F fp32 values, times scale, as T (bf16: round to nearest even).
template <typename T, int F>
__device__ __forceinline__ void store_slice(T* p, const float (&v)[F], float scale) {
    if constexpr (sizeof(T) == 2) {
        static_assert(F % 8 == 0, "bf16 slices are stored 16 bytes at a time");
        uint4* q = reinterpret_cast<uint4*>(p);
#pragma unroll
        for (int i = 0; i < F / 8; ++i) {
            uint4 o;
            o.x = pack_bf16x2(v[8 * i + 0] * scale, v[8 * i + 1] * scale);
            o.y = pack_bf16x2(v[8 * i + 2] * scale, v[8 * i + 3] * scale);
            o.z = pack_bf16x2(v[8 * i + 4] * scale, v[8 * i + 5] * scale);
            o.w = pack_bf16x2(v[8 * i + 6] * scale, v[8 * i + 7] * scale);
            q[i] = o;
        }
    } else {
        static_assert(F % 4 == 0, "fp32 slices are stored 16 bytes at a time");
        float4* q = reinterpret_cast<float4*>(p);
#pragma unroll
        for (int i = 0; i < F / 4; ++i)
            q[i] = make_float4(v[4 * i] * scale, v[4 * i + 1] * scale, v[4 * i + 2] * scale, v[4 * i + 3] * scale);
    }
}

// Sum over the L lanes that share one (node, head).  Groups of 2 or 4 lanes sit
// inside one DPP quad, so the exchanges are quad permutes (xor 1, xor 2) that
// stay off the LDS; every lane of a group is active whenever one is.
template <int L>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (L >= 2) x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
    if constexpr (L >= 4) x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));
#pragma unroll
    for (int o = 4; o < L; o <<= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

}  // namespace gt

// Dispatch a templated launcher over (dtype, d, H).  FN<T, D, H>(args...) must
// return gt_status.
#define GT_DISPATCH_ATTN(dtype, d, H, FN, ...)                                               \
    [&]() -> gt_status {                                                                     \
        if ((dtype) == GT_BF16) {                                                            \
            if ((d) == 32) {                                                                 \
                switch (H) {                                                                 \
                    case 1: return FN<uint16_t, 32, 1>(__VA_ARGS__);                         \
                    case 2: return FN<uint16_t, 32, 2>(__VA_ARGS__);                         \
                    case 4: return FN<uint16_t, 32, 4>(__VA_ARGS__);                         \
                    case 8: return FN<uint16_t, 32, 8>(__VA_ARGS__);                         \
                    case 16: return FN<uint16_t, 32, 16>(__VA_ARGS__);                       \
                }                                                                            \
            } else if ((d) == 64) {                                                          \
                switch (H) {                                                                 \
                    case 1: return FN<uint16_t, 64, 1>(__VA_ARGS__);                         \
                    case 2: return FN<uint16_t, 64, 2>(__VA_ARGS__);                         \
                    case 4: return FN<uint16_t, 64, 4>(__VA_ARGS__);                         \
                    case 8: return FN<uint16_t, 64, 8>(__VA_ARGS__);                         \
                    case 16: return FN<uint16_t, 64, 16>(__VA_ARGS__);                       \
                }                                                                            \
            }                                                                                \
        } else if ((dtype) == GT_F32) {                                                      \
            if ((d) == 32) {                                                                 \
                switch (H) {                                                                 \
                    case 1: return FN<float, 32, 1>(__VA_ARGS__);                            \
                    case 2: return FN<float, 32, 2>(__VA_ARGS__);                            \
                    case 4: return FN<float, 32, 4>(__VA_ARGS__);                            \
                    case 8: return FN<float, 32, 8>(__VA_ARGS__);                            \
                    case 16: return FN<float, 32, 16>(__VA_ARGS__);                          \
                }                                                                            \
            } else if ((d) == 64) {                                                          \
                switch (H) {                                                                 \
                    case 1: return FN<float, 64, 1>(__VA_ARGS__);                            \
                    case 2: return FN<float, 64, 2>(__VA_ARGS__);                            \
                    case 4: return FN<float, 64, 4>(__VA_ARGS__);                            \
                    case 8: return FN<float, 64, 8>(__VA_ARGS__);                            \
                    case 16: return FN<float, 64, 16>(__VA_ARGS__);                          \
                }                                                                            \
            }                                                                                \
        }                                                                                    \
        return gt::fail(GT_ERR_UNSUPPORTED, "attention: unsupported (dtype, d, H)");         \
    }()
