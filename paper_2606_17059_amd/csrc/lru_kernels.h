// lru_kernels.h -- access times and LRU eviction of the local peer's tree.
//
// Algorithm 1: a node that runs a request itself and lacks GPU memory evicts
// least-recently-used leaf tokens of its local tree (EvictLRUTrie) and frees
// their KV cache until the request fits.  Every path of the local tree has an
// access time: loads and merges into the local peer stamp the inserted paths,
// a touch (serving a query) stamps the query's matched prefix.  One eviction
// removes the leaf with the smallest time; ties go to the deepest leaf, then
// to the lexicographically smallest path.  Times never grow along a path, so
// n evictions remove exactly the first n paths of the local tree in the order
// (time ascending, depth descending, path ascending) -- the batched form
// computed here:
//   1. the local peer's nodes (a walk from the root) are sorted by time; a
//      node's time covers all of its label's tokens (node boundaries are made
//      wherever a touch or a partial eviction ends inside a label);
//   2. whole time classes are evicted while the budget lasts; in the class
//      where it runs out, tokens deeper than a depth D go entirely and at depth
//      D the lexicographically smallest paths go, as many as remain;
//   3. nodes evicted entirely lose the local peer's bit; a node cut inside its
//      label is first split there (by inserting the kept path through the
//      merge kernels, without stamping times) and the lower part loses the bit.
#ifndef PR_LRU_KERNELS_H
#define PR_LRU_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"
#include "merge_kernels.h"

namespace pr {

__device__ __forceinline__ bool lru_holds(const DevForest &F, int64_t x, int32_t p) {
    const int32_t w = p >> 6;
    const uint64_t word = w == 0 ? F.nodes[x].mask0 : F.mext[x * (F.W - 1) + (w - 1)];
    return (word >> (p & 63)) & 1ull;
}

__device__ __forceinline__ void lru_clear(const DevForest &F, int64_t x, int32_t p) {
    const int32_t w = p >> 6;
    const unsigned long long keep = ~(1ull << (p & 63));
    if (w == 0)
        F.nodes[x].mask0 &= keep;
    else
        F.mext[x * (F.W - 1) + (w - 1)] &= keep;
}

// Nodes the local peer holds get time t, all others 0.
__global__ void lru_init_kernel(DevForest F, int64_t n_nodes, unsigned long long t) {
    const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= n_nodes) return;
    F.ltime[x] = lru_holds(F, x, F.local) ? t : 0ull;
}

// Touch: the matched prefix of query i in the local tree has match_len[i][L]
// tokens (-1 for a query with invalid offsets: nothing).  len1[i + 1] gets
// that length, len1[0] = 0, so an inclusive scan gives CSR offsets.
__global__ void touch_lengths_kernel(const int32_t *__restrict__ match_len, int32_t P, int32_t L, int64_t n,
                                     int64_t *__restrict__ len1) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) len1[0] = 0;
    if (i < n) len1[i + 1] = max(0, match_len[i * (int64_t)P + L]);
}

// One wave per query: copy its matched prefix to out[toff[i] .. toff[i + 1]).
__global__ __launch_bounds__(256) void touch_gather_kernel(const int32_t *__restrict__ qtok,
                                                           const int64_t *__restrict__ qoff,
                                                           const int64_t *__restrict__ toff, int64_t n,
                                                           int32_t *__restrict__ out) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= n) return;
    const int64_t len = toff[i + 1] - toff[i];
    const int32_t *src = qtok + qoff[i];
    for (int64_t k = lane; k < len; k += 64) out[toff[i] + k] = src[k];
}

// ---- eviction ---------------------------------------------------------------

struct EvictPlan {
    int64_t a, b;   // sorted nodes [0, a) go entirely; [a, b) is the class where the budget runs out
    int64_t r;      // tokens to evict inside that class (0: none, [0, b) go entirely)
    int64_t total;  // tokens the local tree holds
    int64_t depth;  // cut depth D inside the class
    int64_t r_at;   // tokens to evict at depth D (lexicographically smallest paths)
    int32_t maxd;   // deepest token of the class
    int32_t bad;    // a split did not leave the expected structure
};

// Time and id of every node the walk visited (sorted by time next).
__global__ void lru_keys_kernel(DevForest F, const int32_t *__restrict__ all, int64_t V,
                                unsigned long long *__restrict__ keys, int32_t *__restrict__ vals) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= V) return;
    keys[i] = F.ltime[all[i]];
    vals[i] = all[i];
}

// cnt1[i + 1] = label tokens of the i-th node in time order, cnt1[0] = 0.
__global__ void lru_counts_kernel(DevForest F, const int32_t *__restrict__ vals, int64_t V, int64_t *__restrict__ cnt1) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) cnt1[0] = 0;
    if (i < V) cnt1[i + 1] = F.nodes[vals[i]].lab_len;
}

// One thread: the time class in which n evictions end.  cum[i] = tokens of
// the first i nodes in time order (cum[0] = 0, cum[V] = all).
__global__ void lru_plan_kernel(const unsigned long long *__restrict__ keys, const int64_t *__restrict__ cum,
                                int64_t V, int64_t n, EvictPlan *plan) {
    EvictPlan p{};
    p.total = cum[V];
    if (n >= p.total) {
        p.a = p.b = V;
        p.r = 0;
    } else {
        int64_t lo = 0, hi = V;  // first node i whose tokens reach the n-th: cum[i + 1] >= n
        while (lo < hi) {
            const int64_t mid = (lo + hi) / 2;
            if (cum[mid + 1] >= n) hi = mid; else lo = mid + 1;
        }
        const unsigned long long t = keys[lo];
        int64_t l = 0, h = V;  // first key == t
        while (l < h) {
            const int64_t mid = (l + h) / 2;
            if (keys[mid] < t) l = mid + 1; else h = mid;
        }
        const int64_t a = l;
        l = 0;
        h = V;  // first key > t
        while (l < h) {
            const int64_t mid = (l + h) / 2;
            if (keys[mid] <= t) l = mid + 1; else h = mid;
        }
        const int64_t b = l;
        p.a = a;
        p.b = b;
        p.r = n - cum[a];
        if (p.r == cum[b] - cum[a]) {  // the class goes entirely
            p.a = b;
            p.r = 0;
        }
    }
    *plan = p;
}

// Slot in a list shared by every wave: one atomic per wave (atomics on one
// counter serialise), ranks by ballot.  Called by every active lane; returns
// -1 for lanes that take no slot.
__device__ __forceinline__ int32_t lru_wave_slot(int32_t *ctr, bool want) {
    const uint64_t b = __ballot(want);
    if (!b) return -1;
    const int lane = (int)(threadIdx.x & 63);
    const int leader = __ffsll((unsigned long long)b) - 1;
    int32_t base = 0;
    if (lane == leader) base = atomicAdd(ctr, (int32_t)__popcll(b));
    base = __shfl(base, leader);
    return want ? base + (int32_t)__popcll(b & ((1ull << lane) - 1ull)) : -1;
}

// The local peer leaves the first a nodes in time order.
__global__ void lru_clear_sorted_kernel(DevForest F, const int32_t *__restrict__ vals, int64_t a) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < a) lru_clear(F, vals[i], F.local);
}

// Deepest token of the class.
__global__ void lru_maxdepth_kernel(const int32_t *__restrict__ vals, int64_t a, int64_t b,
                                    const int64_t *__restrict__ depth, EvictPlan *plan) {
    const int64_t i = a + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int32_t m = i < b ? (int32_t)depth[vals[i]] : 0;
    for (int off = 32; off >= 1; off >>= 1) m = max(m, __shfl_xor(m, off));
    if ((threadIdx.x & 63) == 0 && m > 0) atomicMax(&plan->maxd, m);
}

// Difference array of the class's token depths: a node covers depths
// [depth - lab_len + 1, depth].
__global__ void lru_hist_kernel(DevForest F, const int32_t *__restrict__ vals, int64_t a, int64_t b,
                                const int64_t *__restrict__ depth, long long *__restrict__ hist) {
    const int64_t i = a + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= b) return;
    const int32_t v = vals[i];
    const int64_t e = depth[v], s = e - F.nodes[v].lab_len + 1;
    atomicAdd((unsigned long long *)&hist[s], 1ull);
    atomicAdd((unsigned long long *)&hist[e + 1], (unsigned long long)-1ll);
}

// rev[k] = class tokens at depth maxd - k, k in [0, maxd).
__global__ void lru_reverse_kernel(const long long *__restrict__ cnt, int32_t maxd, long long *__restrict__ rev) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k < maxd) rev[k] = cnt[maxd - k];
}

// One thread: with S[k] = class tokens at depth >= maxd - k, the cut depth D
// is the shallowest depth whose deeper tokens do not yet cover r.
__global__ void lru_depth_plan_kernel(const long long *__restrict__ S, EvictPlan *plan) {
    EvictPlan p = *plan;
    int64_t lo = 0, hi = p.maxd;  // first k with S[k] >= r
    while (lo < hi) {
        const int64_t mid = (lo + hi) / 2;
        if (S[mid] >= p.r) hi = mid; else lo = mid + 1;
    }
    p.depth = p.maxd - lo;
    p.r_at = p.r - (lo > 0 ? S[lo - 1] : 0);
    *plan = p;
}

// Class nodes that cover the cut depth.
__global__ void lru_level_nodes_kernel(DevForest F, const int32_t *__restrict__ vals, int64_t a, int64_t b,
                                       const int64_t *__restrict__ depth, const EvictPlan *plan,
                                       int32_t *__restrict__ level, int32_t *__restrict__ n_level) {
    const int64_t i = a + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= b) return;
    const int32_t v = vals[i];
    const int64_t e = depth[v], s = e - F.nodes[v].lab_len + 1;
    const int32_t k = lru_wave_slot(n_level, s <= plan->depth && plan->depth <= e);
    if (k >= 0) level[k] = v;
}

// Is the path through u lexicographically before the path through v?  u and
// v both cover the cut depth, so neither is an ancestor of the other: climb
// to the two children of their lowest common ancestor and compare their first
// tokens (siblings' first tokens differ).
__device__ __forceinline__ bool lru_path_before(const int32_t *__restrict__ ntok, const int32_t *__restrict__ parent,
                                                const int64_t *__restrict__ depth, int32_t u, int32_t v) {
    while (parent[u] != parent[v]) {
        const int32_t pu = parent[u], pv = parent[v];
        const int64_t du = pu == 0 ? 0 : depth[pu], dv = pv == 0 ? 0 : depth[pv];
        if (du >= dv) u = pu;
        if (dv >= du) v = pv;
    }
    return ntok[u] < ntok[v];
}

// rank_of[v] = number of level nodes whose path comes before v's.
__global__ void lru_rank_kernel(DevForest F, const int32_t *__restrict__ level, int32_t n_level,
                                const int32_t *__restrict__ parent, const int64_t *__restrict__ depth,
                                int32_t *__restrict__ rank_of) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_level) return;
    const int32_t v = level[i];
    int32_t r = 0;
    for (int32_t j = 0; j < n_level; j++)
        if (j != i && lru_path_before(F.ntok, parent, depth, level[j], v)) r++;
    rank_of[v] = r;
}

// Class nodes: keep the tokens up to keep_end.  Nodes evicted entirely lose
// the local peer's bit; a node cut inside its label is listed with its kept
// path length for the split.
__global__ void lru_apply_kernel(DevForest F, const int32_t *__restrict__ vals, int64_t a, int64_t b,
                                 const int64_t *__restrict__ depth, const int32_t *__restrict__ rank_of,
                                 const EvictPlan *plan, int32_t *__restrict__ cut_node,
                                 int64_t *__restrict__ cut_len1, int32_t *__restrict__ n_cut) {
    const int64_t i = a + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= b) return;
    const int32_t v = vals[i];
    const int64_t e = depth[v], s = e - F.nodes[v].lab_len + 1, D = plan->depth;
    int64_t keep;
    if (s <= D && D <= e)
        keep = rank_of[v] < plan->r_at ? D - 1 : D;
    else
        keep = s > D ? s - 1 : e;
    if (keep < s) lru_clear(F, v, F.local);
    const int32_t k = lru_wave_slot(n_cut, keep >= s && keep < e);
    if (k >= 0) {
        cut_node[k] = v;
        cut_len1[k + 1] = keep;
    }
}

// One wave per cut node: write the root path up to its kept length.
__global__ __launch_bounds__(256) void lru_cut_paths_kernel(DevForest F, const int32_t *__restrict__ cut_node,
                                                            int32_t n_cut, const int64_t *__restrict__ offs,
                                                            const int32_t *__restrict__ parent,
                                                            const int64_t *__restrict__ depth,
                                                            int32_t *__restrict__ out) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= n_cut) return;
    const int64_t base = offs[i], keep = offs[i + 1] - offs[i];
    int32_t c = cut_node[i];
    {
        const Node r = F.nodes[c];
        const int64_t s = depth[c] - r.lab_len;  // tokens above the node
        for (int64_t k = lane; k < keep - s; k += 64) out[base + s + k] = F.pool[r.lab_off + k];
        c = parent[c];
    }
    while (c != 0) {
        const Node r = F.nodes[c];
        const int64_t d = depth[c];
        if (r.lab_len <= 0 || d < r.lab_len) break;
        for (int32_t k = lane; k < r.lab_len; k += 64) out[base + d - r.lab_len + k] = F.pool[r.lab_off + k];
        c = parent[c];
    }
}

// After the split, each cut node holds the kept part and has the rest as its
// only child: the local peer leaves that child.
__global__ void lru_clear_lower_kernel(DevForest F, const int32_t *__restrict__ cut_node, int32_t n_cut,
                                       const int64_t *__restrict__ offs, const int64_t *__restrict__ depth,
                                       const int64_t *__restrict__ old_len, EvictPlan *plan) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_cut) return;
    const int32_t v = cut_node[i];
    const Node r = F.nodes[v];
    const int64_t kept = (offs[i + 1] - offs[i]) - (depth[v] - old_len[i]);
    if (r.ct_cnt != 1 || r.lab_len != kept) {
        atomicAdd(&plan->bad, 1);
        return;
    }
    lru_clear(F, r.ct_beg, F.local);
}

__global__ void lru_old_len_kernel(DevForest F, const int32_t *__restrict__ cut_node, int32_t n_cut,
                                   int64_t *__restrict__ old_len) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_cut) old_len[i] = F.nodes[cut_node[i]].lab_len;
}

}  // namespace pr

#endif
