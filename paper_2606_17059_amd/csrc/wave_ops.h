// wave_ops.h -- small wavefront (64-lane) helpers shared by the kernels.
#ifndef PR_WAVE_OPS_H
#define PR_WAVE_OPS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pr {

// Value of v in the wave's first active lane, as a wave-uniform scalar.
__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// 64-bit value of v in lane src (src must be wave-uniform).
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int src) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, src);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
}

}  // namespace pr

#endif
