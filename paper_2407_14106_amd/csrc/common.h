// Shared host/device helpers of libgt (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "gt.h"

namespace gt {

// ---------------------------------------------------------------- host side

void set_error(const std::string& msg);
gt_status fail(gt_status code, const std::string& msg);
gt_status hip_fail(hipError_t e, const char* what);

#define GT_HIP(call)                                      \
    do {                                                  \
        hipError_t e_ = (call);                           \
        if (e_ != hipSuccess) return gt::hip_fail(e_, #call); \
    } while (0)

// After a kernel launch: report a launch failure as GT_ERR_HIP.
#define GT_LAUNCH_CHECK(name)                               \
    do {                                                    \
        hipError_t e_ = hipGetLastError();                  \
        if (e_ != hipSuccess) return gt::hip_fail(e_, name); \
    } while (0)

// Bump allocator over the caller workspace.  With base == nullptr it only
// measures, so the *_workspace_size() functions and the calls share one layout.
struct Ws {
    char* base;
    size_t off = 0;
    explicit Ws(void* b) : base(static_cast<char*>(b)) {}
    template <typename T>
    T* take(size_t count) {
        off = (off + 255) & ~size_t(255);
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
    size_t size() const { return (off + 255) & ~size_t(255); }
};

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// MI355X has 8 XCDs (each with its own L2) and hands consecutive workgroup ids
// to them round-robin.  Kernels whose neighbouring workgroups share data
// remap their id so that each XCD walks one contiguous range: launch a grid
// padded to a multiple of kXcds (xcd_grid) and call xcd_block(blockIdx.x).
constexpr int kXcds = 8;
inline unsigned xcd_grid(int64_t blocks) { return static_cast<unsigned>(cdiv(blocks > 0 ? blocks : 1, kXcds) * kXcds); }
__device__ __forceinline__ int64_t xcd_block(int64_t b, int64_t grid) {
    return (b % kXcds) * (grid / kXcds) + b / kXcds;
}

inline unsigned grid_for(int64_t work, int per_block, int64_t cap = 1 << 20) {
    int64_t g = cdiv(work, per_block);
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return static_cast<unsigned>(g);
}

// ------------------------------------------------------------- device side

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    // SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014).
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest, ties to even (finite values; NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return uint32_t(f32_to_bf16(lo)) | (uint32_t(f32_to_bf16(hi)) << 16);
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        T w = __shfl_xor(v, o, kWave);
        v = v > w ? v : w;
    }
    return v;
}
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint64_t lanemask_lt() {
    int l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

template <typename T>
__device__ __forceinline__ T uniform(T v) {
    return static_cast<T>(__builtin_amdgcn_readfirstlane(static_cast<int>(v)));
}
__device__ __forceinline__ int64_t uniform64(int64_t v) {
    uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32));
    return static_cast<int64_t>((uint64_t(hi) << 32) | lo);
}

}  // namespace gt
