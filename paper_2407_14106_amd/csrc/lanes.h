// Lane exchanges at a fixed power-of-two distance inside a wavefront, for
// the integer stages' row groups: quad permutes (DPP) and lane swizzles,
// which need no LDS address and no lane index, instead of a general lane
// permute.  Every lane of the wavefront must be active where they run.
#pragma once

#include "common.h"

namespace gt {

// x of lane (lane ^ O), 0 < O < 64: a quad permute (DPP) for O < 4, a
// bit-mode lane swizzle (lane' = lane ^ O inside each 32-lane half) up to
// 31, a lane permute across the halves for 32.
template <int O>
__device__ __forceinline__ int xor_lane(int x) {
    static_assert(O > 0 && (O < 32 || O == 32), "one lane bit");
    if constexpr (O == 1) return __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);  // quad [1,0,3,2]
    else if constexpr (O == 2) return __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);  // [2,3,0,1]
    else if constexpr (O == 3) return __builtin_amdgcn_update_dpp(0, x, 0x1B, 0xF, 0xF, false);  // [3,2,1,0]
    else if constexpr (O < 32) return __builtin_amdgcn_ds_swizzle(x, 0x1F | (O << 10));  // and 0x1F, xor O
    else return __shfl_xor(x, 32, kWave);
}
template <int O>
__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t x) {
    const uint32_t lo = uint32_t(xor_lane<O>(int(uint32_t(x))));
    const uint32_t hi = uint32_t(xor_lane<O>(int(uint32_t(x >> 32))));
    return (uint64_t(hi) << 32) | lo;
}

// xor_lane<o> for o known where the call is unrolled (1, 2, 4, ..., 32).
__device__ __forceinline__ int xor_lane_pow2(int x, int o) {
    switch (o) {
        case 1: return xor_lane<1>(x);
        case 2: return xor_lane<2>(x);
        case 4: return xor_lane<4>(x);
        case 8: return xor_lane<8>(x);
        case 16: return xor_lane<16>(x);
        default: return xor_lane<32>(x);
    }
}

}  // namespace gt
