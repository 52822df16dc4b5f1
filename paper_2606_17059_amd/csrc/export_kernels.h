// export_kernels.h -- snapshot export (sendTrie) from the device forest.
//
// A peer's tree is fixed by its root paths, so the export is the set of paths
// that end at a node holding the peer none of whose children holds it: the
// members of the peer's set that are no proper prefix of another (System
// Design, sendTrie; Section "Trie-broadcast loss": a broadcast is a complete
// snapshot).
//
//   1. export_level_kernel walks the forest level by level from the root,
//      only through nodes whose mask holds p (merges leave unreachable blocks
//      behind, which a walk from the root never visits).  Every visited node
//      gets its depth (tokens from the root through its label) and its
//      parent; a visited node none of whose children holds p is a leaf.
//      The LRU eviction uses the same walk and also lists every visited node.
//   2. The host sorts the leaves by node id (a deterministic order) and scans
//      their depths into CSR offsets.
//   3. export_write_kernel: one wave per leaf climbs the parent chain and
//      writes every label on the path at its depth, lanes over tokens.
#ifndef PR_EXPORT_KERNELS_H
#define PR_EXPORT_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"
#include "merge_kernels.h"

namespace pr {

constexpr int kExportWavesPerBlock = 4;

__device__ __forceinline__ bool node_holds(const DevForest &F, int64_t x, int32_t p) {
    const int32_t w = p >> 6;
    const uint64_t word = w == 0 ? F.nodes[x].mask0 : F.mext[x * (F.W - 1) + (w - 1)];
    return (word >> (p & 63)) & 1ull;
}

__global__ void export_init_kernel(int32_t *front, int64_t *depth, int32_t *counts) {
    front[0] = 0;
    depth[0] = 0;
    counts[0] = 0;  // next frontier size
    counts[1] = 0;  // leaves so far
    counts[2] = 0;  // visited nodes so far (root excluded)
}

__global__ void export_reset_kernel(int32_t *counts) { counts[0] = 0; }

// One wave per frontier node x: children holding p join the next frontier
// with their depth and parent; x becomes a leaf if none holds p.
// The frontier, the leaf list, depth and parent hold n_nodes entries; a walk
// of a well-formed forest never exceeds them, and the host reports counts
// above n_nodes as a broken forest (the writes past the end are dropped).
__global__ __launch_bounds__(64 * kExportWavesPerBlock) void export_level_kernel(
    DevForest F, int64_t n_nodes, int32_t p, const int32_t *__restrict__ front, int32_t n_front,
    int32_t *__restrict__ next, int32_t *__restrict__ leaves, int64_t *__restrict__ depth,
    int32_t *__restrict__ parent, int32_t *__restrict__ counts, int32_t *__restrict__ all) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * kExportWavesPerBlock + (threadIdx.x >> 6);
    if (i >= n_front) return;
    const int32_t x = front[i];
    const int32_t beg = F.nodes[x].ct_beg, cnt = F.nodes[x].ct_cnt;
    const int64_t dx = depth[x];
    bool found = false;
    // slots are taken with one atomic per wave and 64 children: atomics on
    // one counter serialise
    const uint64_t below = (1ull << lane) - 1ull;
    for (int32_t base = 0; base < cnt; base += 64) {
        const int32_t c = beg + base + lane;
        const bool h = base + lane < cnt && c >= 0 && c < n_nodes && node_holds(F, c, p);
        const uint64_t b = __ballot(h);
        if (!b) continue;
        found = true;
        const int32_t n = (int32_t)__popcll(b);
        int32_t s0 = 0, k0 = 0;
        if (lane == 0) {
            s0 = atomicAdd(&counts[0], n);
            if (all) k0 = atomicAdd(&counts[2], n);
        }
        s0 = __shfl(s0, 0);
        k0 = __shfl(k0, 0);
        if (h) {
            const int32_t r = (int32_t)__popcll(b & below);
            depth[c] = dx + F.nodes[c].lab_len;
            parent[c] = x;
            if (s0 + r < n_nodes) next[s0 + r] = c;
            if (all && k0 + r < n_nodes) all[k0 + r] = c;
        }
    }
    if (!found && x != 0 && lane == 0) {
        const int32_t slot = atomicAdd(&counts[1], 1);
        if (slot < n_nodes) leaves[slot] = x;
    }
}

// Sequence lengths of the sorted leaves, written one slot to the right so
// that an inclusive scan over [1, n] gives the CSR offsets.
__global__ void export_lengths_kernel(const int32_t *__restrict__ leaves, int32_t n, const int64_t *__restrict__ depth,
                                      int64_t *__restrict__ len1) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) len1[0] = 0;
    if (i < n) len1[i + 1] = depth[leaves[i]];
}

// One wave per leaf: climb to the root, writing each label at its depth.
__global__ __launch_bounds__(64 * kExportWavesPerBlock) void export_write_kernel(
    DevForest F, const int32_t *__restrict__ leaves, int32_t n, const int64_t *__restrict__ depth,
    const int32_t *__restrict__ parent, const int64_t *__restrict__ offsets, int32_t *__restrict__ out) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * kExportWavesPerBlock + (threadIdx.x >> 6);
    if (i >= n) return;
    const int64_t base = offsets[i];
    int32_t c = leaves[i];
    // depth falls by at least one token per step, so the climb ends at the root
    while (c != 0) {
        const Node r = F.nodes[c];
        const int64_t d = depth[c];
        if (r.lab_len <= 0 || d < r.lab_len) break;  // not a well-formed path: stop
        const int64_t start = base + d - r.lab_len;
        const int32_t *lab = F.pool + r.lab_off;
        for (int32_t k = lane; k < r.lab_len; k += 64) out[start + k] = lab[k];
        c = parent[c];
    }
}

// Tokens a peer's tree holds: the label lengths of the nodes the walk visited
// (a wave sum, then one atomic per wave).
__global__ void tree_tokens_kernel(DevForest F, const int32_t *__restrict__ all, int32_t V,
                                   unsigned long long *__restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    unsigned long long v = i < V ? (unsigned long long)F.nodes[all[i]].lab_len : 0ull;
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & 63) == 0 && v) atomicAdd(out, v);
}

}  // namespace pr

#endif
