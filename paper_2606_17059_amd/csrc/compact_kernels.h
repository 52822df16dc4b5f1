// compact_kernels.h -- rebuild the device forest without the records and
// labels that no peer's tree uses any more.
//
// Merges leave the old child blocks of rebuilt parents behind, and cleared or
// evicted peers leave nodes that no peer holds.  A node some peer holds has
// an ancestor chain of nodes that peer holds (masks never grow away from the
// root), so the live forest is the root plus every node with a non-empty mask
// that is reachable through such nodes.  The rebuild copies it level by level
// into fresh arrays:
//   1. per level, one wave per frontier node x (old id, new id known) keeps
//      x's children with a non-empty mask, in their (token-sorted) order, as
//      one new contiguous block; the block start is x's offset in an
//      exclusive scan of the kept counts over the frontier;
//   2. the kept children's records, first tokens, mask words and access times
//      are copied to their new ids, and they form the next frontier;
//   3. once all levels are done, a scan of label lengths gives every node a
//      span of the new pool, labels are copied, and wide blocks get their
//      separators.
// The root stays node 0.  Match results, exports and access times are those of
// the old forest.
#ifndef PR_COMPACT_KERNELS_H
#define PR_COMPACT_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"
#include "merge_kernels.h"

namespace pr {

constexpr int kCompactWavesPerBlock = 4;

__device__ __forceinline__ bool node_has_peers(const DevForest &F, int64_t x) {
    if (F.nodes[x].mask0) return true;
    for (int w = 1; w < F.W; w++)
        if (F.mext[x * (F.W - 1) + (w - 1)]) return true;
    return false;
}

// Root into the new image; frontier = {root}.
__global__ void compact_init_kernel(DevForest O, DevForest N, int32_t *front_old, int32_t *front_new) {
    Node r = O.nodes[0];
    r.aux = 0;
    N.nodes[0] = r;
    N.ntok[0] = O.ntok[0];
    for (int w = 1; w < O.W; w++) N.mext[w - 1] = O.mext[w - 1];
    if (O.ltime && N.ltime) N.ltime[0] = O.ltime[0];
    front_old[0] = 0;
    front_new[0] = 0;
}

// kept[i] = children of frontier node i that some peer holds.
__global__ __launch_bounds__(64 * kCompactWavesPerBlock) void compact_count_kernel(
    DevForest O, const int32_t *__restrict__ front_old, int32_t n_front, int64_t *__restrict__ kept) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * kCompactWavesPerBlock + (threadIdx.x >> 6);
    if (i >= n_front) return;
    const Node x = O.nodes[front_old[i]];
    int32_t k = 0;
    for (int32_t base = 0; base < x.ct_cnt; base += 64) {
        const int32_t j = base + lane;
        const bool keep = j < x.ct_cnt && node_has_peers(O, x.ct_beg + j);
        k += __popcll(__ballot(keep));
    }
    if (lane == 0) kept[i] = k;
}

// Copy the kept children of frontier node i to new ids first_new + start[i] ..,
// point x's new record at them, and list them as the next frontier.
__global__ __launch_bounds__(64 * kCompactWavesPerBlock) void compact_copy_kernel(
    DevForest O, DevForest N, const int32_t *__restrict__ front_old, const int32_t *__restrict__ front_new,
    int32_t n_front, const int64_t *__restrict__ start, int64_t first_new, int32_t *__restrict__ next_old,
    int32_t *__restrict__ next_new, int64_t next_base) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * kCompactWavesPerBlock + (threadIdx.x >> 6);
    if (i >= n_front) return;
    const Node x = O.nodes[front_old[i]];
    const int64_t beg = first_new + start[i];
    int64_t pos = 0;
    for (int32_t base = 0; base < x.ct_cnt; base += 64) {
        const int32_t j = base + lane;
        const bool keep = j < x.ct_cnt && node_has_peers(O, x.ct_beg + j);
        const uint64_t b = __ballot(keep);
        if (keep) {
            const int64_t rank = pos + __popcll(b & ((1ull << lane) - 1ull));
            const int32_t src = x.ct_beg + j;
            const int64_t dst = beg + rank;
            Node c = O.nodes[src];
            c.aux = 0;
            N.nodes[dst] = c;  // ct_beg / ct_cnt / lab_off fixed later
            N.ntok[dst] = O.ntok[src];
            for (int w = 1; w < O.W; w++) N.mext[dst * (O.W - 1) + (w - 1)] = O.mext[(int64_t)src * (O.W - 1) + (w - 1)];
            if (O.ltime && N.ltime) N.ltime[dst] = O.ltime[src];
            next_old[next_base + start[i] + rank] = src;
            next_new[next_base + start[i] + rank] = (int32_t)dst;
        }
        pos += __popcll(b);
    }
    if (lane == 0) {
        const int32_t xn = front_new[i];
        N.nodes[xn].ct_beg = (int32_t)beg;
        N.nodes[xn].ct_cnt = (int32_t)pos;
    }
}

// len1[i + 1] = label length of new node i, len1[0] = 0.
__global__ void compact_lab_len_kernel(DevForest N, int64_t n, int64_t *__restrict__ len1) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) len1[0] = 0;
    if (i < n) len1[i + 1] = N.nodes[i].lab_len;
}

// One wave per new node: copy its label to its span of the new pool.
__global__ __launch_bounds__(64 * kCompactWavesPerBlock) void compact_labels_kernel(
    const int32_t *__restrict__ old_pool, DevForest N, int64_t n, const int64_t *__restrict__ off) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * kCompactWavesPerBlock + (threadIdx.x >> 6);
    if (i >= n) return;
    const Node r = N.nodes[i];
    for (int32_t k = lane; k < r.lab_len; k += 64) N.pool[off[i] + k] = old_pool[r.lab_off + k];
    if (lane == 0) N.nodes[i].lab_off = (uint32_t)off[i];
}

// Separators of every wide block of the new image.
__global__ __launch_bounds__(64 * kCompactWavesPerBlock) void compact_sep_kernel(DevForest N, int64_t n) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * kCompactWavesPerBlock + (threadIdx.x >> 6);
    if (i >= n) return;
    const Node r = N.nodes[i];
    if (r.ct_cnt > kSepCount) N.nsep[r.ct_beg + lane] = N.ntok[r.ct_beg + PR_SEP_INDEX(lane, r.ct_cnt)];
    if (r.ct_cnt >= kSep2Min) sep2_write(N.nsep + r.ct_beg, N.ntok + r.ct_beg, r.ct_cnt, lane);
}

}  // namespace pr

#endif
