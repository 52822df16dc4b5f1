// narrow_kernels.h -- gfx950 kernel that keeps the narrow copy of the label
// pool (the low 16 bits of every token, and a plane of bit 16) in step with
// the int32 pool after merges append labels.  Routes read labels from that
// copy while every label token fits 17 bits.
#ifndef PR_NARROW_KERNELS_H
#define PR_NARROW_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"

namespace pr {

// The narrow copy of the label pool for tokens [from, to): p16[i] = the low
// 16 bits of pool[i], and bit i % 32 of hib[i / 32] = bit 16 of pool[i].  One
// wave per 64-token chunk (grid-stride), a lane per token: the chunk's two bit
// words come from one ballot.  Chunks start at a multiple of 64, so the first
// one may rewrite entries below `from` with the values they already hold.
// *hi becomes nonzero if a token of the range lies in [65536, 131071] (the
// bit plane is needed), *wide if one lies outside [0, 131071] (the copy is
// unusable); each workgroup reduces its finds and writes each flag at most
// once, so the waves do not queue on one address.
constexpr int kNarrowWave = 64;
constexpr int kNarrowThreads = 256;
// to_dev (if not nullptr): the range ends at min(*to_dev, to) instead, for a
// pool whose used size only the device knows.
__global__ __launch_bounds__(kNarrowThreads) void pool_narrow_kernel(const int32_t *__restrict__ pool,
                                                                     uint16_t *__restrict__ p16,
                                                                     uint32_t *__restrict__ hib, int64_t from,
                                                                     int64_t to, unsigned long long *__restrict__ hi,
                                                                     unsigned long long *__restrict__ wide,
                                                                     const unsigned long long *to_dev) {
    __shared__ int found[2];
    if (to_dev) to = min(to, (int64_t)*to_dev);
    const int lane = (int)(threadIdx.x & (kNarrowWave - 1));
    if (threadIdx.x < 2) found[threadIdx.x] = 0;
    __syncthreads();
    const int64_t waves = (int64_t)gridDim.x * (kNarrowThreads / kNarrowWave);
    bool h = false, o = false;
    for (int64_t k = from / kNarrowWave + (int64_t)blockIdx.x * (kNarrowThreads / kNarrowWave) + threadIdx.x / kNarrowWave;
         k * kNarrowWave < to; k += waves) {
        const int64_t i = k * kNarrowWave + lane;
        const bool in = i < to;
        const uint32_t t = in ? (uint32_t)pool[i] : 0u;
        if (in) p16[i] = (uint16_t)t;
        const uint64_t bits = __ballot((t >> 16) & 1u);
        if (lane == 0) hib[2 * k] = (uint32_t)bits;
        if (lane == 32) hib[2 * k + 1] = (uint32_t)(bits >> 32);
        h |= in && i >= from && t > 0xFFFFu && t <= 0x1FFFFu;
        o |= in && i >= from && t > 0x1FFFFu;
    }
    if (__ballot(h) && lane == 0) found[0] = 1;
    if (__ballot(o) && lane == 0) found[1] = 1;
    __syncthreads();
    if (threadIdx.x == 0 && found[0] && __hip_atomic_load(hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0)
        atomicOr(hi, 1ull);
    if (threadIdx.x == 1 && found[1] && __hip_atomic_load(wide, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0)
        atomicOr(wide, 1ull);
}

}  // namespace pr

#endif
