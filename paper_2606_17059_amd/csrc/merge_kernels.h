// merge_kernels.h -- gfx950 kernels that insert a batch of sequences into the
// union forest (updateTrie / updateTrieEstimate applied to a batch).
//
// The batch is applied in rounds.  Every round each unfinished insert walks the
// current forest (one wave per insert) and ends in one of three states:
//   DONE   the sequence ends exactly at a node: nothing structural is missing;
//   ADD    at node x no child starts with the next token: a leaf must be hung
//          below x;
//   SPLIT  the sequence leaves (or ends inside) the label of child c of x
//          after l tokens: c's edge must be cut there.
// A round applies both kinds the walk found.  The add phase comes first: ADD
// inserts are sorted by (x, next token); per slot the lowest batch index wins,
// and every parent x gets a new, sorted child block holding its old children
// and one leaf per winning slot.  The phase is data-parallel however the
// inserts crowd on one parent: scans over the sorted entries give every winner
// its slot, one wave per 64 old children moves them, and one wave per winner
// writes its leaf.  A round of at most kPlanMax ADD entries sorts, scans and
// allocates in one workgroup (add_plan_kernel); larger rounds take a rocPRIM
// radix sort, four scans and per-parent allocation.  Records that move are
// stamped with their new position, so that a parent rebuilt in the same round,
// and a child whose edge the split phase then cuts, are found wherever their
// records live.  The split phase: per child c the insert with the lowest batch
// index wins (an atomic max claim), rewrites c's record in place as the upper
// part of the edge and gives it a new child block holding the lower part (c's
// old record, label advanced) and, if the winner's sequence goes on, a leaf
// with the winner's remaining tokens.  Winners of both phases are done.
// Allocations come from device counters; one that does not fit the capacity
// is refused whole and counted, and the host grows the forest and repeats the
// round.
// Losers walk again in the next round and find the structure the winners
// built.  Peer masks follow the walks: a walk sets its insert's peer bit in
// every node it passes through whole (the root included), a new leaf holds
// its winner's bit, and a cut edge's upper part adds it; records carry their
// masks when they move or split, so every node on an insert's final path holds
// its bit.  The match function afterwards is that of the old sets plus the
// batch; it does not depend on the batch order.
#ifndef PR_MERGE_KERNELS_H
#define PR_MERGE_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"
#include "wave_ops.h"

namespace pr {

enum InsKind : int32_t { kInsSkip = 0, kInsActive = 1, kInsDone = 2, kInsAdd = 3, kInsSplit = 4 };

struct InsState {
    int32_t kind;
    int32_t x;  // node the walk stopped at (ADD, SPLIT) or ended at (DONE)
    int32_t c;  // SPLIT: the child whose label is cut
    int32_t l;  // SPLIT: tokens of c's label shared with the insert
    int32_t d;  // depth of x
    int32_t t;  // next token below x (ADD, SPLIT)
};

// Device-side counters of one merge call; the host reads them between rounds.
struct MergeCounters {
    unsigned long long n_nodes;   // node records in use
    unsigned long long n_pool;    // pool tokens in use
    unsigned long long n_add;     // inserts in state ADD after the last walk
    unsigned long long n_split;   // inserts in state SPLIT after the last walk
    unsigned long long pool_need; // upper bound of pool tokens the next round adds
    unsigned long long node_need; // add round: exact node records the next round adds
    unsigned long long overflow;  // allocations refused for lack of capacity
    unsigned long long skipped;   // inserts with invalid peer or offsets
    unsigned long long bad_path;  // an invariant of the round broke (the merge fails)
    unsigned long long move_chunks;  // add round: 64-child chunks of the old blocks that move
    unsigned long long wide_tokens;  // nonzero: an appended label token lies outside [0, 131071] (no narrow copy)
    unsigned long long hi_tokens;    // nonzero: an appended label token lies in [65536, 131071] (17-bit labels)
    unsigned long long add_pool_base;  // add round planned in one workgroup: first pool token of its labels
    unsigned long long plan_n;         // ADD entries the one-workgroup plan took this round (0: none)
    unsigned long long plan_fallback;  // nonzero: this round's ADD entries do not fit the one-workgroup plan
};

// Entry count of an add step: the host's, or (n_add < 0, rounds the host does
// not read back) the one-workgroup plan's.
__device__ __forceinline__ int64_t add_count(int64_t n_add, const MergeCounters *ctr) {
    return n_add >= 0 ? n_add : (int64_t)ctr->plan_n;
}

struct DevForest {
    Node *nodes;
    int32_t *ntok;
    int32_t *nsep;
    uint64_t *mext;
    int32_t *pool;
    long long *moved;  // (stamp << 32) | new position, per node id
    int64_t cap_nodes, cap_pool;
    int32_t W;
    // access times of the local peer's nodes (nullptr: no local peer); a node's
    // time covers every token of its label, so records carry it when they
    // move or split
    unsigned long long *ltime;
    int32_t local;
    unsigned long long now;
};

struct Batch {
    const int32_t *peer_of;
    const int32_t *tokens;
    const int64_t *offsets;
    int64_t num_tokens;
    int64_t n;
    int32_t P;
    int32_t stamp;  // 1: inserts into the local peer stamp their path with F.now
};

constexpr int kMergeWavesPerBlock = 4;
constexpr int kMoveBlocks = 1024;  // workgroups of the grid-stride move kernel

__device__ __forceinline__ int64_t m_wave_index() {
    return (int64_t)blockIdx.x * kMergeWavesPerBlock + uniform((int32_t)(threadIdx.x / 64));
}

// Atomic add by lane 0, result broadcast to the wave.
__device__ __forceinline__ unsigned long long wave_atomic_add(unsigned long long *p, unsigned long long v, int lane) {
    unsigned long long r = 0;
    if (lane == 0) r = atomicAdd(p, v);
    return (unsigned long long)readlane64((uint64_t)r, 0);
}

// First i < n with a[i] != b[i], or n (wave-cooperative).  Steps of 1024
// tokens: a step's loads are all issued before its first wait, so a 1024-token
// label costs one round trip.
constexpr int kMergeLcpVectors = 16;
__device__ __forceinline__ int64_t m_lcp(const int32_t *a, const int32_t *b, int64_t n, int lane) {
    for (int64_t base = 0; base < n; base += 64 * kMergeLcpVectors) {
        uint64_t bal[kMergeLcpVectors];
#pragma unroll
        for (int j = 0; j < kMergeLcpVectors; j++) {
            const int64_t i = base + j * 64 + lane;
            bool mis = false;
            if (i < n) mis = a[i] != b[i];
            bal[j] = __ballot(mis);
        }
#pragma unroll
        for (int j = 0; j < kMergeLcpVectors; j++)
            if (bal[j]) return base + j * 64 + (__ffsll((unsigned long long)bal[j]) - 1);
    }
    return n;
}

// The insert's peer bit in node x's mask, set only where it is missing (the
// nodes near the root lie on almost every path, and atomics on one address
// serialise); inserts into the local peer also stamp x with the current time.
// mask0: x's first mask word as the caller read it.  Lane 0 only.
__device__ __forceinline__ void m_mark(const DevForest &F, int32_t x, uint64_t mask0, int32_t w,
                                       unsigned long long bit, bool stamp) {
    unsigned long long *mw = w == 0 ? (unsigned long long *)&F.nodes[x].mask0
                                    : (unsigned long long *)&F.mext[(int64_t)x * (F.W - 1) + (w - 1)];
    const unsigned long long cur =
        w == 0 ? (unsigned long long)mask0 : __hip_atomic_load(mw, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!(cur & bit)) atomicOr(mw, bit);
    if (stamp && __hip_atomic_load(&F.ltime[x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < F.now)
        atomicMax(&F.ltime[x], F.now);
}

// Second-level separators of a block of cnt >= kSep2Min children whose first
// tokens are tok[0, cnt): every sub-range's 64, sixteen sub-ranges' loads
// issued before their stores (the two arrays share an allocation, so the
// compiler would otherwise wait for each store before the next load).
__device__ __forceinline__ void sep2_write(int32_t *sep, const int32_t *tok, int32_t cnt, int lane) {
    for (int q0 = 0; q0 < kSepCount; q0 += 16) {
        int32_t v[16];
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const int32_t lo = PR_SEP_INDEX(q0 + u, cnt), span = PR_SEP_HI(q0 + u, cnt) - lo;
            v[u] = tok[lo + PR_SEP_INDEX(lane, span)];
        }
#pragma unroll
        for (int u = 0; u < 16; u++) sep[kSepCount + kSepCount * (q0 + u) + lane] = v[u];
    }
}

// Child of node x whose first token is t, or -1 (wave-cooperative).  Blocks
// of up to 64 children take one ballot over their first tokens; wider blocks
// first pick their sub-range through the block's 64 separators (and, from
// kSep2Min children on, through the sub-range's own 64).
__device__ __forceinline__ int32_t m_find_child(const DevForest &F, const Node &x, int32_t t, int lane) {
    const int32_t beg = x.ct_beg, cnt = x.ct_cnt;
    if (cnt <= kSepCount) {
        const uint64_t b = __ballot(lane < cnt && F.ntok[beg + lane] == t);
        return b ? beg + (int32_t)(__ffsll((unsigned long long)b) - 1) : -1;
    }
    // separators ascend, so the lanes with sep <= t form a prefix
    const uint64_t b = __ballot(F.nsep[beg + lane] <= t);
    if (!b) return -1;  // t is below every first token
    const int32_t k = (int32_t)__popcll(b) - 1;
    int32_t lo = PR_SEP_INDEX(k, cnt);
    int32_t hi = PR_SEP_HI(k, cnt);
    if (cnt >= kSep2Min) {
        // the sub-range's own 64 separators (lane 0's is the first level's k-th, <= t)
        const int32_t span = hi - lo;
        const uint64_t b2 = __ballot(F.nsep[beg + kSepCount + kSepCount * k + lane] <= t);
        const int32_t j = (int32_t)__popcll(b2) - 1;
        hi = PR_SEP_HI(j, span) + lo;
        lo += PR_SEP_INDEX(j, span);
    }
    while (hi - lo > 64) {  // sub-ranges of more than 64 children: 64-ary search
        const int32_t stride = (hi - lo + 63) / 64;
        const int32_t j = lo + lane * stride;
        const uint64_t bl = __ballot(j < hi && F.ntok[beg + j] <= t);
        if (!bl) return -1;
        lo = lo + (__popcll(bl) - 1) * stride;
        hi = min(lo + stride, hi);
    }
    const int32_t j = lo + lane;
    const uint64_t be = __ballot(j < hi && F.ntok[beg + j] == t);
    return be ? beg + lo + (int32_t)(__ffsll((unsigned long long)be) - 1) : -1;
}

__global__ void merge_validate_kernel(Batch B, InsState *st, MergeCounters *ctr) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B.n) return;
    const int64_t b = B.offsets[i], e = B.offsets[i + 1];
    const int32_t p = B.peer_of[i];
    const bool ok = p >= 0 && p < B.P && b >= 0 && e >= b && e <= B.num_tokens && e - b <= (int64_t)INT32_MAX;
    st[i].kind = ok ? kInsActive : kInsSkip;
    if (!ok) atomicAdd(&ctr->skipped, 1ull);
}

// Walk every active insert; classify it as DONE, ADD or SPLIT.
__global__ __launch_bounds__(64 *kMergeWavesPerBlock) void merge_walk_kernel(DevForest F, Batch B, InsState *st,
                                                                            MergeCounters *ctr) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t i = m_wave_index();
    if (i >= B.n) return;
    const int32_t kind = st[i].kind;
    if (kind == kInsSkip || kind == kInsDone) return;
    const int32_t *s = B.tokens + B.offsets[i];
    const int64_t len = B.offsets[i + 1] - B.offsets[i];
    const int32_t p = B.peer_of[i];
    const int32_t w = p >> 6;
    const unsigned long long bit = 1ull << (p & 63);
    const bool stamp = F.ltime && B.stamp && p == F.local;
    int32_t x = 0;
    int64_t d = 0;
    InsState r;
    r.c = -1;
    r.l = 0;
    r.t = 0;
    if (lane == 0) m_mark(F, 0, F.nodes[0].mask0, w, bit, stamp);
    while (true) {
        if (d == len) {
            r.kind = kInsDone;
            break;
        }
        const Node nx = F.nodes[x];
        const int32_t t = s[d];
        const int32_t c = m_find_child(F, nx, t, lane);
        if (c < 0) {
            r.kind = kInsAdd;
            r.t = t;
            break;
        }
        const Node nc = F.nodes[c];
        const int64_t n = min((int64_t)nc.lab_len, len - d);
        const int64_t l = m_lcp(F.pool + nc.lab_off, s + d, n, lane);
        if (l == nc.lab_len && nc.lab_len > 0) {
            x = c;
            d += l;
            if (lane == 0) m_mark(F, c, nc.mask0, w, bit, stamp);
            continue;
        }
        r.kind = kInsSplit;
        r.c = c;
        r.l = (int32_t)l;
        r.t = t;
        break;
    }
    r.x = x;
    r.d = (int32_t)d;
    if (lane == 0) st[i] = r;  // merge_tally_kernel counts the kinds
}

// Counts of the walk's ADD and SPLIT inserts and the pool tokens they may
// need, reduced per block before one atomic each: per-insert atomics on the
// same counters would serialise.
constexpr int kTallyThreads = 256;
// arest[i] (if not nullptr): the label tokens ADD insert i needs, else -1 (the
// one-workgroup add plan reads it).
__global__ __launch_bounds__(kTallyThreads) void merge_tally_kernel(Batch B, const InsState *st,
                                                                    MergeCounters *ctr, int32_t *arest) {
    __shared__ unsigned long long part[3][kTallyThreads / 64];
    unsigned long long n_add = 0, n_split = 0, pool = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < B.n; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t kind = st[i].kind;
        int32_t ar = -1;
        if (kind == kInsAdd || kind == kInsSplit) {
            n_add += kind == kInsAdd;
            n_split += kind == kInsSplit;
            const int64_t rest = B.offsets[i + 1] - B.offsets[i] - st[i].d;
            pool += (unsigned long long)rest;
            if (kind == kInsAdd) ar = (int32_t)rest;
        }
        if (arest) arest[i] = ar;
    }
    for (int off = 32; off >= 1; off >>= 1) {
        n_add += __shfl_xor(n_add, off);
        n_split += __shfl_xor(n_split, off);
        pool += __shfl_xor(pool, off);
    }
    const int wv = (int)(threadIdx.x / 64);
    if ((threadIdx.x & 63) == 0) {
        part[0][wv] = n_add;
        part[1][wv] = n_split;
        part[2][wv] = pool;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long a = 0, b = 0, c = 0;
        for (int k = 0; k < kTallyThreads / 64; k++) {
            a += part[0][k];
            b += part[1][k];
            c += part[2][k];
        }
        if (a) atomicAdd(&ctr->n_add, a);
        if (b) atomicAdd(&ctr->n_split, b);
        if (c) atomicAdd(&ctr->pool_need, c);
    }
}

// Where node c's record lives now: an add phase earlier in the same round
// (stamp > 0) may have moved it into its parent's rebuilt block.
__device__ __forceinline__ int32_t current_pos(const DevForest &F, int32_t c, long long stamp) {
    if (stamp <= 0) return c;
    const long long mv = F.moved[c];
    return (mv >> 32) == stamp ? (int32_t)(uint32_t)mv : c;
}

// SPLIT phase, step 1: per child c, the lowest batch index wins the claim.
// stamp: that of the add phase that ran earlier in this round, or 0.
__global__ void split_claim_kernel(DevForest F, Batch B, const InsState *st, long long stamp) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B.n || st[i].kind != kInsSplit) return;
    atomicMax(&F.nodes[current_pos(F, st[i].c, stamp)].aux, (int32_t)(INT32_MAX - i));
}

// Mask words past the first of a cut edge: the lower part (dst) keeps the
// edge's peers, the upper part (src, in place) adds peer p.  Each word is read
// and written by one lane.
__device__ __forceinline__ void cut_mext(const DevForest &F, int64_t dst, int64_t src, int32_t p, int lane) {
    for (int w = lane; w < F.W - 1; w += 64) {
        const uint64_t v = F.mext[src * (F.W - 1) + w];
        F.mext[dst * (F.W - 1) + w] = v;
        if ((p >> 6) == w + 1) F.mext[src * (F.W - 1) + w] = v | (1ull << (p & 63));
    }
}

// Mask words past the first of a new leaf: the bit of peer p only.
__device__ __forceinline__ void leaf_mext(const DevForest &F, int64_t dst, int32_t p, int lane) {
    for (int w = lane; w < F.W - 1; w += 64)
        F.mext[dst * (F.W - 1) + w] = (p >> 6) == w + 1 ? 1ull << (p & 63) : 0ull;
}

// Copy n tokens into freshly allocated pool space (wave-cooperative).
__device__ __forceinline__ void copy_tokens(int32_t *dst, const int32_t *src, int64_t n, int lane) {
    for (int64_t k = lane; k < n; k += 64) dst[k] = src[k];
}

// Cut child c's edge after l tokens; the winning insert's rest becomes a leaf,
// and the winner is done.  An add phase earlier in the round may have moved
// c's record (stamp, as for the claim); it also may have given c a new child
// block, which the lower part of the edge takes along.  reset_round: also
// clear the round's counters for the next walk (every kernel that reads them
// has finished; this one only allocates), which saves a launch per round.
// Waves per workgroup of split_apply_kernel: a workgroup takes one allocation
// of records and one of pool tokens for all its winners (two atomics on the
// merge's counters instead of two per winner, which serialise on their two
// addresses when a batch cuts thousands of edges).
constexpr int kSplitWaves = 16;

__global__ __launch_bounds__(64 *kSplitWaves) void split_apply_kernel(DevForest F, Batch B, InsState *st,
                                                                     MergeCounters *ctr, long long stamp,
                                                                     int reset_round) {
    __shared__ unsigned long long s_need[2][kSplitWaves];  // records, pool tokens per wave
    __shared__ unsigned long long s_base[2];
    const int lane = (int)(threadIdx.x & 63);
    const int wv = uniform((int32_t)(threadIdx.x / 64));
    const int64_t i = (int64_t)blockIdx.x * kSplitWaves + wv;
    if (reset_round && blockIdx.x == 0 && threadIdx.x == 0) {
        ctr->n_add = 0;
        ctr->n_split = 0;
        ctr->pool_need = 0;
        ctr->node_need = 0;
        ctr->move_chunks = 0;
        ctr->plan_n = 0;
        ctr->plan_fallback = 0;
    }
    // every wave reaches the workgroup's allocation below; only the winner of
    // its edge's claim takes a share
    bool win = false;
    InsState r{};
    const int32_t *s = nullptr;
    int64_t rest = 0;  // tokens after the cut (0: the insert ends at the cut)
    int32_t k = 0;
    if (i < B.n && st[i].kind == kInsSplit) {
        r = st[i];
        r.c = current_pos(F, r.c, stamp);
        if (F.nodes[r.c].aux == (int32_t)(INT32_MAX - i)) {  // else another insert cuts c this round
            s = B.tokens + B.offsets[i];
            rest = B.offsets[i + 1] - B.offsets[i] - (int64_t)r.d - r.l;
            k = rest > 0 ? 2 : 1;
            if (r.l > 0)
                win = true;
            else if (lane == 0)  // a first-token match guarantees l >= 1; refuse anything else
                atomicAdd(&ctr->overflow, 1ull);
        }
    }
    if (lane == 0) {
        s_need[0][wv] = win ? (unsigned long long)k : 0ull;
        s_need[1][wv] = win && rest > 0 ? (unsigned long long)rest : 0ull;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long tn = 0, tp = 0;
        for (int w = 0; w < kSplitWaves; w++) {
            tn += s_need[0][w];
            tp += s_need[1][w];
        }
        s_base[0] = tn ? atomicAdd(&ctr->n_nodes, tn) : 0ull;
        s_base[1] = tp ? atomicAdd(&ctr->n_pool, tp) : 0ull;
    }
    __syncthreads();
    if (!win) return;
    int64_t nb = (int64_t)s_base[0], pb = (int64_t)s_base[1];
    for (int w = 0; w < wv; w++) {
        nb += (int64_t)s_need[0][w];
        pb += (int64_t)s_need[1][w];
    }
    if (rest <= 0) pb = 0;  // no pool span
    if (nb + k > F.cap_nodes || pb + rest > F.cap_pool) {
        // refused: nothing is written, the claim is withdrawn, and the insert
        // walks again once the host has grown the forest
        if (lane == 0) {
            atomicAdd(&ctr->overflow, 1ull);
            F.nodes[r.c].aux = 0;
        }
        return;
    }
    const Node old = F.nodes[r.c];
    Node lower = old;
    lower.tok = F.pool[old.lab_off + r.l];
    lower.lab_off = old.lab_off + (uint32_t)r.l;
    lower.lab_len = old.lab_len - r.l;
    lower.aux = 0;
    int64_t pos_lower = nb, pos_leaf = nb + 1;
    if (rest > 0 && s[r.d + r.l] < lower.tok) {
        pos_leaf = nb;
        pos_lower = nb + 1;
    }
    if (rest > 0) copy_tokens(F.pool + pb, s + r.d + r.l, rest, lane);
    // the winner's peer holds the upper part and its leaf; the lower part
    // keeps the edge's peers
    const int32_t p = B.peer_of[i];
    const unsigned long long bit0 = (p >> 6) == 0 ? 1ull << (p & 63) : 0ull;
    const bool local = F.ltime && B.stamp && p == F.local;
    cut_mext(F, pos_lower, r.c, p, lane);
    if (rest > 0) leaf_mext(F, pos_leaf, p, lane);
    if (lane == 0) {
        F.nodes[pos_lower] = lower;
        F.ntok[pos_lower] = lower.tok;
        if (F.ltime) {
            const unsigned long long tc = F.ltime[r.c];
            F.ltime[pos_lower] = tc;  // both parts of the edge keep its time
            if (local && tc < F.now) F.ltime[r.c] = F.now;
            if (rest > 0) F.ltime[pos_leaf] = local ? F.now : 0ull;
        }
        if (rest > 0) {
            Node leaf;
            leaf.tok = s[r.d + r.l];
            leaf.lab_off = (uint32_t)pb;
            leaf.lab_len = (int32_t)rest;
            leaf.ct_beg = 0;
            leaf.ct_cnt = 0;
            leaf.aux = 0;
            leaf.mask0 = bit0;
            F.nodes[pos_leaf] = leaf;
            F.ntok[pos_leaf] = leaf.tok;
        }
        Node upper = old;  // keeps tok, label start, peers and c's slot in its parent
        upper.mask0 |= bit0;
        upper.lab_len = r.l;
        upper.ct_beg = (int32_t)nb;
        upper.ct_cnt = k;
        upper.aux = 0;
        F.nodes[r.c] = upper;
        st[i].kind = kInsDone;  // the sequence ends at the leaf, or at upper (rest 0)
    }
}

// Sort keys of ADD inserts: (parent, next token) in (unsigned, signed) order;
// other inserts sort last.  A stable sort keeps batch order inside a slot.
__global__ void add_keys_kernel(Batch B, const InsState *st, unsigned long long *keys, int32_t *vals) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B.n) return;
    const InsState r = st[i];
    keys[i] = r.kind == kInsAdd ? (((unsigned long long)(uint32_t)r.x << 32) | (uint32_t)(r.t ^ (int32_t)0x80000000))
                                : ~0ull;
    vals[i] = (int32_t)i;
}

__device__ __forceinline__ int32_t key_parent(unsigned long long k) { return (int32_t)(k >> 32); }

// Number of entries of the sorted int32 array a[0..n) that are < v.
__device__ __forceinline__ int32_t lower_count(const int32_t *a, int32_t n, int32_t v) {
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (a[mid] < v)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

__device__ __forceinline__ bool add_is_head(const unsigned long long *keys, int64_t e) {
    return e == 0 || key_parent(keys[e - 1]) != key_parent(keys[e]);
}

// ADD round, step 1 (one thread per sorted ADD entry e, plus one): the slot
// winner flag (first entry of each (parent, token) key) and the winner's label
// tokens; the entry index if e heads its parent's group (else -1, for a max
// scan); per group head the 64-child chunks of the parent's old block.
__global__ void add_mark_kernel(DevForest F, Batch B, const unsigned long long *keys, const int32_t *vals,
                                int64_t n_add, const InsState *st, int32_t *win, int64_t *rest, int32_t *headv,
                                int32_t *nch) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e == n_add) nch[n_add] = 0;  // the chunk scan's total lands at n_add
    if (e >= n_add) return;
    const bool head = add_is_head(keys, e);
    const bool w = e == 0 || keys[e] != keys[e - 1];
    const int32_t i = vals[e];
    win[e] = w ? 1 : 0;
    rest[e] = w ? B.offsets[i + 1] - B.offsets[i] - st[i].d : 0;
    headv[e] = head ? (int32_t)e : -1;
    nch[e] = head ? (F.nodes[key_parent(keys[e])].ct_cnt + 63) / 64 : 0;
}

// Step 2 (one thread per entry; widx, poff: exclusive scans of win, rest; hd:
// the entry's group head; cstart: exclusive scan of nch).  Winners go to
// win_tok / win_ins [k + w] of their group (head k, ordinal w, token order),
// and the last entry of each group records the group's winner count and label
// tokens and counts the records it needs.
__global__ void add_group_kernel(DevForest F, const unsigned long long *keys, const int32_t *vals, int64_t n_add,
                                 const InsState *st, const int32_t *win, const int64_t *rest, const int32_t *widx,
                                 const int64_t *poff, const int32_t *hd, const int32_t *cstart, int32_t *grp_nw,
                                 int64_t *grp_pool, int32_t *win_tok, int32_t *win_ins, MergeCounters *ctr) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_add) return;
    const int32_t k = hd[e];
    if (win[e]) {
        const int32_t w = widx[e] - widx[k];
        win_tok[k + w] = st[vals[e]].t;
        win_ins[k + w] = vals[e];
    }
    if (e + 1 < n_add && !add_is_head(keys, e + 1)) return;  // not the group's last entry
    const int32_t nw = widx[e] + win[e] - widx[k];
    const int64_t pool = poff[e] + rest[e] - poff[k];
    grp_nw[k] = nw;
    grp_pool[k] = pool;
    atomicAdd(&ctr->node_need, (unsigned long long)(F.nodes[key_parent(keys[e])].ct_cnt + nw));
    atomicAdd(&ctr->pool_need, (unsigned long long)pool);
    if (e == n_add - 1) ctr->move_chunks = (unsigned long long)cstart[n_add];
}

// ---- the add plan in one workgroup -------------------------------------------
// For a round whose ADD entries fit one workgroup's LDS, one launch replaces
// steps 0-3 (sort keys, radix sort, marks, the four scans, groups and their
// allocation):
//  1. the batch is read in coalesced chunks; ADD entries are gathered in batch
//     order, and each gets its label span in one pool allocation for the whole
//     round, in batch order (`pofs`, indexed by insert; a slot loser's span
//     stays unused, zero-filled);
//  2. parents are numbered through a hash table in LDS, so that the sort key
//     (parent slot, token) needs about 11 + 17 bits instead of 31 + 32; with
//     more distinct parents than the table takes, the key keeps the node id;
//  3. a stable least-significant-digit radix sort in LDS, 4-bit digits, a pass
//     only for digits that differ between keys; digit counts are LDS atomics on
//     each thread's own counters, which also give the entry's rank among the
//     thread's entries of that digit;
//  4. marks and scans in registers; one node allocation for every rebuilt
//     block of the round, refused as a whole when the capacity runs out.
// The outputs keep the multi-launch path's layout (keys hold the parent's node
// id), so the move, leaf, separator and fix steps serve both paths.
constexpr int kPlanThreads = 1024;
constexpr int kPlanItems = 10;                              // sorted entries per thread
constexpr int kPlanMax = kPlanThreads * kPlanItems;         // ADD entries per round
constexpr int kPlanBatchItems = 16;                         // batch chunks of kPlanThreads
constexpr int64_t kPlanMaxBatch = (int64_t)kPlanThreads * kPlanBatchItems;  // insert ids fit 16 bits
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kPlanSlots = 2048;                            // parent hash table
constexpr int kPlanMaxParents = kPlanSlots / 2;
constexpr int kPlanSmall = 256;                             // rounds ranked by counting instead

// Inclusive scan over the wave.
template <typename T, typename Op>
__device__ __forceinline__ T plan_wave_incl(T v, Op op) {
    const int lane = (int)(threadIdx.x & 63);
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const T u = __shfl_up(v, off);
        if (lane >= off) v = op(v, u);
    }
    return v;
}

// Inclusive sum over the wave through DPP lane moves: a Hillis-Steele scan
// within each row of 16 lanes (row shifts by 1, 2, 4, 8; a lane with no
// source adds 0), then each row adds the totals of the rows before it (row
// broadcasts of lanes 15 and 31).
__device__ __forceinline__ uint32_t wave_incl_add_u32(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15 -> rows 1, 3
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31 -> rows 2, 3
    return v;
}

// Inclusive sum over the wave of values below 2^25 each (so no sum
// overflows 32 bits), else of any values.
__device__ __forceinline__ long long wave_incl_add_i64(long long v) {
    if (__ballot(v >= (1ll << 25)) == 0) return (long long)wave_incl_add_u32((uint32_t)v);
    return plan_wave_incl(v, [](long long a, long long b) { return a + b; });
}

// Exclusive scan over the workgroup in thread order (id: the identity of op);
// *total receives the reduction of every thread's v.  Every thread calls it.
template <typename T, typename Op>
__device__ T plan_block_excl(T v, T id, Op op, T *tmp, T *total) {
    const int lane = (int)(threadIdx.x & 63), w = (int)(threadIdx.x >> 6);
    const T inc = plan_wave_incl(v, op);
    if (lane == 63) tmp[w] = inc;
    __syncthreads();
    T pre = id, tot = id;
#pragma unroll
    for (int k = 0; k < kPlanWaves; k++) {
        const T x = tmp[k];
        if (k < w) pre = op(pre, x);
        tot = op(tot, x);
    }
    __syncthreads();  // tmp is free for the next scan
    T ex = __shfl_up(inc, 1);
    if (lane == 0) ex = id;
    *total = tot;
    return op(pre, ex);
}

__device__ __forceinline__ uint32_t plan_hash(int32_t x) {
    return ((uint32_t)x * 2654435761u) >> 21;  // 11 bits: kPlanSlots
}

// Slot of parent x in the table (x >= 0), inserting it; -1 when the table is full.
__device__ __forceinline__ int plan_slot_insert(int32_t *tab, int *n_new, int32_t x) {
    uint32_t h = plan_hash(x);
    for (int p = 0; p < kPlanSlots; p++, h = (h + 1) & (kPlanSlots - 1)) {
        const int32_t cur = tab[h];
        if (cur == x) return (int)h;
        if (cur == -1) {
            const int32_t old = atomicCAS(&tab[h], -1, x);
            if (old == -1) {
                atomicAdd(n_new, 1);
                return (int)h;
            }
            if (old == x) return (int)h;
        }
    }
    return -1;
}

__device__ __forceinline__ int plan_slot_find(const int32_t *tab, int32_t x) {
    uint32_t h = plan_hash(x);
    for (int p = 0; p < kPlanSlots; p++, h = (h + 1) & (kPlanSlots - 1))
        if (tab[h] == x) return (int)h;
    return -1;  // not reached for a parent that was inserted
}

// LDS index of sorted entry p: one pad entry per 32, so that the threads'
// blocked runs of entries (a stride of kPlanItems) spread over the banks.
__device__ __forceinline__ int plan_pad(int p) { return p + (p >> 5); }
constexpr int kPlanPadded = kPlanMax + kPlanMax / 32;

// One workgroup of kPlanThreads, for batches of at most kPlanMaxBatch inserts
// whose round has at most kPlanMax ADD entries.  n_add is the walk's tally of
// ADD inserts (< 0: take the tally from ctr, for rounds the host does not read
// back; a round that does not fit then raises plan_fallback and plans
// nothing), and arest the tally's per-insert label tokens (-1: not ADD); a
// count that differs from the host's raises bad_path and plans nothing (the
// merge then fails).  pofs[i]: the label span of ADD insert i from the round's
// pool base (ctr->add_pool_base); ctr->plan_n: the entries planned.
__global__ __launch_bounds__(kPlanThreads) void add_plan_kernel(DevForest F, Batch B, const InsState *st,
                                                                const int32_t *arest, int64_t n_add,
                                                                unsigned long long *keys, int32_t *vals,
                                                                int32_t *win, int32_t *widx, int32_t *hd,
                                                                int32_t *cstart, int32_t *grp_nw, int32_t *grp_nb,
                                                                int32_t *win_tok, int64_t *pofs,
                                                                MergeCounters *ctr) {
    __shared__ unsigned long long s_key[kPlanPadded];        // sort keys; later staged outputs
    __shared__ uint16_t s_val[kPlanPadded];                  // insert ids; later each entry's widx
    __shared__ uint32_t s_cnt[8 * kPlanThreads];             // digits d, d + 8 of thread t: word d * T + t
    __shared__ int32_t s_tab[kPlanSlots];                    // parent node id per slot, or -1
    __shared__ int s_cw[kPlanBatchItems * kPlanWaves];       // ADD entries per (chunk, wave), then their scan
    __shared__ long long s_rw[kPlanBatchItems * kPlanWaves]; // their label tokens, then the scan
    __shared__ uint32_t s_wt[kPlanWaves * 8];                // per wave: packed digit totals, then prefixes
    __shared__ uint32_t s_dt[8];                             // packed digit totals of the workgroup
    __shared__ long long s_tmp[kPlanWaves];
    __shared__ int s_tmp32[kPlanWaves];
    __shared__ int s_misc[4];                                // distinct parents, table full, ADD entries
    constexpr int T = kPlanThreads;
    const int t = (int)threadIdx.x;
    const int lane = t & 63, wv = t >> 6;
    const uint64_t lt_mask = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    const auto plus = [](int a, int b) { return a + b; };
    const auto plus64 = [](long long a, long long b) { return a + b; };

    if (n_add < 0) {
        const unsigned long long na = ctr->n_add;  // the tally's, complete before this launch
        if (na == 0 || na > (unsigned long long)kPlanMax || B.n > kPlanMaxBatch) {
            if (t == 0) {
                ctr->plan_n = 0;
                ctr->move_chunks = 0;
                if (na) ctr->plan_fallback = 1;
            }
            return;
        }
        n_add = (int64_t)na;
    }
    for (int q = t; q < kPlanSlots; q += T) s_tab[q] = -1;
    if (t < 4) s_misc[t] = 0;

    // 1. chunk j holds inserts [j*T, (j+1)*T): count the ADD entries and their
    // label tokens per (chunk, wave), in batch order
    const int n = (int)min<int64_t>(B.n, kPlanMaxBatch);
    const int R = (n + T - 1) / T;
    int32_t ar[kPlanBatchItems];
#pragma unroll
    for (int j = 0; j < kPlanBatchItems; j++) ar[j] = (j < R && j * T + t < n) ? arest[j * T + t] : -1;
    uint32_t addbits = 0;
#pragma unroll
    for (int j = 0; j < kPlanBatchItems; j++) {
        if (j < R) {
            const bool a = ar[j] >= 0;
            addbits |= (uint32_t)a << j;
            const uint64_t bal = __ballot(a);
            const long long rs = wave_incl_add_i64((long long)(a ? ar[j] : 0));
            if (lane == 63) {
                s_cw[j * kPlanWaves + wv] = (int)__popcll(bal);
                s_rw[j * kPlanWaves + wv] = rs;
            }
        }
    }
    __syncthreads();
    if (wv == 0) {
        // exclusive scans of the (chunk, wave) tables in their order, 4 entries a lane
        int c[4];
        long long r[4];
        int cs = 0;
        long long rsum = 0;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const int idx = lane * 4 + q;
            c[q] = idx < R * kPlanWaves ? s_cw[idx] : 0;
            r[q] = idx < R * kPlanWaves ? s_rw[idx] : 0;
            cs += c[q];
            rsum += r[q];
        }
        const int ci = plan_wave_incl(cs, plus);
        const long long ri = plan_wave_incl(rsum, plus64);
        int cp = ci - cs;
        long long rp = ri - rsum;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const int idx = lane * 4 + q;
            if (idx < R * kPlanWaves) {
                s_cw[idx] = cp;
                s_rw[idx] = rp;
            }
            cp += c[q];
            rp += r[q];
        }
        if (lane == 63) {
            s_misc[3] = ci;  // ADD entries
            s_tmp[0] = ri;   // their label tokens
        }
    }
    __syncthreads();
    const int m = s_misc[3];
    const long long pool_total = s_tmp[0];
    if ((int64_t)m != n_add || m > kPlanMax || B.n > kPlanMaxBatch) {
        if (t == 0) {
            atomicAdd(&ctr->bad_path, 1ull);
            ctr->plan_n = 0;
            ctr->move_chunks = 0;
        }
        return;  // the same in every thread
    }
    __syncthreads();  // s_tmp is reused by the scans below
    // second sweep: place each ADD entry, record its span, hash its parent
    // (parents are looked up until the table holds kPlanMaxParents of them;
    // small rounds are ranked by counting and keep node ids)
    const bool small = m <= kPlanSmall;
    if (small && t == 0) s_misc[1] = 1;
    __syncthreads();
    {
        int32_t xs[kPlanBatchItems], ts[kPlanBatchItems];
#pragma unroll
        for (int j = 0; j < kPlanBatchItems; j++) {
            xs[j] = 0;
            ts[j] = 0;
            if ((addbits >> j) & 1u) {
                xs[j] = st[j * T + t].x;
                ts[j] = st[j * T + t].t;
            }
        }
#pragma unroll
        for (int j = 0; j < kPlanBatchItems; j++) {
            if (j < R) {
                const int i = j * T + t;
                const bool a = (addbits >> j) & 1u;
                const long long rest = a ? ar[j] : 0;
                const uint64_t bal = __ballot(a);
                const long long rs = wave_incl_add_i64(rest) - rest;
                if (a) {
                    const int pos = s_cw[j * kPlanWaves + wv] + (int)__popcll(bal & lt_mask);
                    pofs[i] = s_rw[j * kPlanWaves + wv] + rs;
                    if (s_misc[1] == 0) {
                        if (s_misc[0] > kPlanMaxParents || plan_slot_insert(s_tab, &s_misc[0], xs[j]) < 0)
                            s_misc[1] = 1;
                    }
                    s_key[plan_pad(pos)] =
                        ((unsigned long long)(uint32_t)xs[j] << 32) | (uint32_t)(ts[j] ^ (int32_t)0x80000000);
                    s_val[plan_pad(pos)] = (uint16_t)i;
                }
            }
        }
    }
    __syncthreads();
    const bool slotted = !small && s_misc[1] == 0 && s_misc[0] <= kPlanMaxParents;
    if (slotted) {
        for (int p = t; p < m; p += T) {
            const unsigned long long kk = s_key[plan_pad(p)];
            const int sl = plan_slot_find(s_tab, (int32_t)(kk >> 32));
            s_key[plan_pad(p)] = ((unsigned long long)(uint32_t)sl << 32) | (kk & 0xFFFFFFFFull);
        }
    }
    __syncthreads();

    if (small) {
        // rank of entry t: the entries with a smaller key, or an equal key
        // earlier in the batch (every lane of a wave reads the same key: an
        // LDS broadcast)
        unsigned long long mk = 0;
        int mv = 0, rank = 0;
        if (t < m) {
            mk = s_key[plan_pad(t)];
            mv = s_val[plan_pad(t)];
#pragma unroll 8
            for (int j = 0; j < m; j++) {
                const unsigned long long kj = s_key[plan_pad(j)];
                rank += (int)((kj < mk) | ((kj == mk) & (j < t)));
            }
        }
        __syncthreads();
        if (t < m) {
            s_key[plan_pad(rank)] = mk;
            s_val[plan_pad(rank)] = (uint16_t)mv;
        }
        __syncthreads();
    }

    // 2. stable LSD radix sort; thread t holds the entries [t*C, t*C + nv)
    const int C = (m + T - 1) / T;
    const int e0 = t * C;
    const int nv = max(0, min(C, m - e0));
    unsigned long long k[kPlanItems];
    int32_t v[kPlanItems];
    unsigned long long kor = 0, kand = ~0ull;
#pragma unroll
    for (int j = 0; j < kPlanItems; j++) {
        k[j] = j < nv ? s_key[plan_pad(e0 + j)] : 0ull;
        v[j] = j < nv ? (int32_t)s_val[plan_pad(e0 + j)] : 0;
        if (j < nv) {
            kor |= k[j];
            kand &= k[j];
        }
    }
    if (small) {
        kor = 0;  // ranked above: no radix pass
    } else {
        long long o, a;
        (void)plan_block_excl<long long>((long long)kor, 0, [](long long x, long long y) { return x | y; }, s_tmp,
                                         &o);
        (void)plan_block_excl<long long>((long long)kand, -1, [](long long x, long long y) { return x & y; }, s_tmp,
                                         &a);
        kor = (unsigned long long)o ^ (unsigned long long)a;  // bits that differ between keys
    }
#pragma unroll 1
    for (int b = 0; b < 64; b += 4) {
        if (((kor >> b) & 15ull) == 0) continue;  // the same digit in every key
        // counts of the thread's own entries per digit, in its own column
        // (digit d in the low half of word (d & 7) * T + t for d < 8, else the
        // high half); the atomics' old values rank each entry among the
        // thread's earlier entries of its digit
#pragma unroll
        for (int q = 0; q < 8; q++) s_cnt[q * T + t] = 0u;
        uint32_t lr[kPlanItems];
#pragma unroll
        for (int j = 0; j < kPlanItems; j++) {
            lr[j] = 0;
            if (j < nv) {
                const int d = (int)((k[j] >> b) & 15ull);
                const uint32_t old = atomicAdd(&s_cnt[(d & 7) * T + t], (d >> 3) ? 0x10000u : 1u);
                lr[j] = (old >> ((d >> 3) << 4)) & 0xFFFFu;
            }
        }
        // rank base of (digit, thread) in digit-major order: the digit's
        // offset, plus the same digit's counts of the threads before.  Both
        // halves of a word scan together (no half exceeds kPlanMax < 2^16).
        uint32_t ex[8];
#pragma unroll
        for (int q = 0; q < 8; q++) {
            const uint32_t cw = s_cnt[q * T + t];
            const uint32_t inc = wave_incl_add_u32(cw);
            ex[q] = inc - cw;
            if (lane == 63) s_wt[wv * 8 + q] = inc;
        }
        __syncthreads();
        if (t < 8) {
            // exclusive prefix over the waves of each packed word, and the total
            uint32_t x[kPlanWaves];
#pragma unroll
            for (int w = 0; w < kPlanWaves; w++) x[w] = s_wt[w * 8 + t];
            uint32_t run = 0;
#pragma unroll
            for (int w = 0; w < kPlanWaves; w++) {
                s_wt[w * 8 + t] = run;
                run += x[w];
            }
            s_dt[t] = run;
        }
        __syncthreads();
        {
            // digit offsets, packed like the counts: digits 0-7 in the low
            // halves, 8-15 in the high (no half reaches 2^16, so packed sums
            // do not carry)
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int q = 0; q < 8; q++) hi += s_dt[q] & 0xFFFFu;  // digits 8-15 start after all of 0-7
#pragma unroll
            for (int q = 0; q < 8; q++) {
                const uint32_t dt = s_dt[q];
                s_cnt[q * T + t] = ex[q] + s_wt[wv * 8 + q] + ((hi << 16) | lo);
                lo += dt & 0xFFFFu;
                hi += dt >> 16;
            }
        }
#pragma unroll
        for (int j = 0; j < kPlanItems; j++) {
            if (j < nv) {
                const int d = (int)((k[j] >> b) & 15ull);
                const uint32_t base = (s_cnt[(d & 7) * T + t] >> ((d >> 3) << 4)) & 0xFFFFu;
                const int rank = (int)(base + lr[j]);
                s_key[plan_pad(rank)] = k[j];
                s_val[plan_pad(rank)] = (uint16_t)v[j];
            }
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kPlanItems; j++) {
            if (j < nv) {
                k[j] = s_key[plan_pad(e0 + j)];
                v[j] = (int32_t)s_val[plan_pad(e0 + j)];
            }
        }
        // no barrier here: the next pass writes only its own wave's s_wt
        // entries and its own column before its first barrier, and s_dt and
        // the entries after it
    }

    // 3. marks: slot winners, group heads and ends; per-thread totals
    const unsigned long long before = (nv > 0 && e0 > 0) ? s_key[plan_pad(e0 - 1)] : 0ull;
    const unsigned long long after = (nv > 0 && e0 + nv < m) ? s_key[plan_pad(e0 + nv)] : 0ull;
    for (int p = t; p < m; p += T) {
        const unsigned long long kk = s_key[plan_pad(p)];
        const uint32_t x = slotted ? (uint32_t)s_tab[(int)(kk >> 32)] : (uint32_t)(kk >> 32);
        keys[p] = ((unsigned long long)x << 32) | (kk & 0xFFFFFFFFull);
        vals[p] = (int32_t)s_val[plan_pad(p)];
    }
    uint32_t wbits = 0, hbits = 0, lbits = 0;
    int sw = 0, sc = 0, lh = -1;
#pragma unroll
    for (int j = 0; j < kPlanItems; j++) {
        if (j < nv) {
            const int e = e0 + j;
            const unsigned long long kp = j == 0 ? before : k[j - 1];
            const unsigned long long kn = j + 1 < nv ? k[j + 1] : after;
            const bool w = e == 0 || k[j] != kp;
            const bool h = e == 0 || (k[j] >> 32) != (kp >> 32);
            const bool l = e + 1 == m || (k[j] >> 32) != (kn >> 32);
            wbits |= (uint32_t)w << j;
            hbits |= (uint32_t)h << j;
            lbits |= (uint32_t)l << j;
            sw += w;
            if (h) {
                const int32_t x = slotted ? s_tab[(int)(k[j] >> 32)] : (int32_t)(k[j] >> 32);
                sc += (F.nodes[x].ct_cnt + 63) / 64;
                lh = e;
            }
        }
    }
    int tw, tc, th;
    int pw = plan_block_excl<int>(sw, 0, plus, s_tmp32, &tw);
    int pc = plan_block_excl<int>(sc, 0, plus, s_tmp32, &tc);
    int ph = plan_block_excl<int>(lh, -1, [](int x, int y) { return x > y ? x : y; }, s_tmp32, &th);
    // 4. per entry: widx, hd and cstart, staged in LDS (s_key's entries and
    // s_val's ids were read before the scans' barriers) and written out
    // coalesced; widx stays in s_val for the group ends
    const int ph0 = ph;
#pragma unroll
    for (int j = 0; j < kPlanItems; j++) {
        if (j < nv) {
            const int e = e0 + j;
            const bool h = (hbits >> j) & 1u;
            if (h) ph = e;
            s_val[plan_pad(e)] = (uint16_t)pw;
            s_key[plan_pad(e)] = ((unsigned long long)(uint32_t)pc << 32) | (uint32_t)ph;
            pw += (wbits >> j) & 1u;
            if (h) {
                const int32_t x = slotted ? s_tab[(int)(k[j] >> 32)] : (int32_t)(k[j] >> 32);
                pc += (F.nodes[x].ct_cnt + 63) / 64;
            }
        }
    }
    __syncthreads();
    for (int p = t; p < m; p += T) {
        const unsigned long long sk = s_key[plan_pad(p)];
        const int wi = (int)s_val[plan_pad(p)];
        const int wn = p + 1 < m ? (int)s_val[plan_pad(p + 1)] : tw;
        win[p] = wn - wi;
        widx[p] = wi;
        hd[p] = (int32_t)(uint32_t)sk;
        cstart[p] = (int32_t)(sk >> 32);
    }
    // 5. records per rebuilt block (old children + winners), scanned over the
    // groups in order; one allocation for all of them and one for the pool
    int hcur = ph0;
    int need = 0;
#pragma unroll
    for (int j = 0; j < kPlanItems; j++) {
        if (j < nv) {
            const int e = e0 + j;
            if ((hbits >> j) & 1u) hcur = e;
            if ((lbits >> j) & 1u) {
                const int32_t x = slotted ? s_tab[(int)(k[j] >> 32)] : (int32_t)(k[j] >> 32);
                const int nw = (int)s_val[plan_pad(e)] + (int)((wbits >> j) & 1u) - (int)s_val[plan_pad(hcur)];
                need += F.nodes[x].ct_cnt + nw;
            }
        }
    }
    int need_all;
    int noff = plan_block_excl<int>(need, 0, plus, s_tmp32, &need_all);
    if (t == 0) {
        const long long nb = (long long)atomicAdd(&ctr->n_nodes, (unsigned long long)need_all);
        const long long pb = (long long)atomicAdd(&ctr->n_pool, (unsigned long long)pool_total);
        const bool ok = nb + need_all <= F.cap_nodes && pb + pool_total <= F.cap_pool;
        if (!ok) atomicAdd(&ctr->overflow, 1ull);
        ctr->add_pool_base = (unsigned long long)pb;
        ctr->move_chunks = (unsigned long long)tc;
        ctr->plan_n = (unsigned long long)m;
        cstart[m] = tc;
        s_tmp[0] = ok ? nb : -1;
    }
    __syncthreads();
    // winners' tokens go to LDS at their place in win_tok (head + ordinal) and
    // out coalesced; entries past a group's winners hold no token
    const long long nb0 = s_tmp[0];
    uint32_t *s_tok = reinterpret_cast<uint32_t *>(s_key);  // the staged outputs were read above
    hcur = ph0;
#pragma unroll
    for (int j = 0; j < kPlanItems; j++) {
        if (j < nv) {
            const int e = e0 + j;
            const bool w = (wbits >> j) & 1u;
            if ((hbits >> j) & 1u) hcur = e;
            const int wk = (int)s_val[plan_pad(hcur)];
            if (w) s_tok[plan_pad(hcur + ((int)s_val[plan_pad(e)] - wk))] = (uint32_t)k[j] ^ 0x80000000u;
            if ((lbits >> j) & 1u) {
                const int32_t x = slotted ? s_tab[(int)(k[j] >> 32)] : (int32_t)(k[j] >> 32);
                const int nw = (int)s_val[plan_pad(e)] + (int)w - wk;
                grp_nw[hcur] = nw;
                grp_nb[hcur] = nb0 < 0 ? -1 : (int32_t)(nb0 + noff);
                noff += F.nodes[x].ct_cnt + nw;
            }
        }
    }
    __syncthreads();
    for (int p = t; p < m; p += T) win_tok[p] = (int32_t)s_tok[plan_pad(p)];
}

// Step 3 (one thread per group head): records and label tokens of the new
// block, or grp_nb = -1 (nothing is written; the parent keeps its old,
// consistent block) when the capacity runs out.
__global__ void add_alloc_kernel(DevForest F, const unsigned long long *keys, int64_t n_add, const int32_t *grp_nw,
                                 const int64_t *grp_pool, int32_t *grp_nb, int64_t *grp_pb, MergeCounters *ctr) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n_add || !add_is_head(keys, k)) return;
    const int32_t cnt = F.nodes[key_parent(keys[k])].ct_cnt + grp_nw[k];
    const int64_t nb = (int64_t)atomicAdd(&ctr->n_nodes, (unsigned long long)cnt);
    const int64_t pb = (int64_t)atomicAdd(&ctr->n_pool, (unsigned long long)grp_pool[k]);
    if (nb + cnt > F.cap_nodes || pb + grp_pool[k] > F.cap_pool) {
        atomicAdd(&ctr->overflow, 1ull);
        grp_nb[k] = -1;
        return;
    }
    grp_nb[k] = (int32_t)nb;
    grp_pb[k] = pb;
}

// Step 4 (64-child chunks of every rebuilt parent's old block, a wave per
// chunk, grid-stride over the chunk count step 2 recorded): old children keep
// their order, each moving up by the winners below it, and are stamped with
// their new position.  The grid is small and fixed, so its size does not
// follow the forest's record count.
__global__ __launch_bounds__(64 *kMergeWavesPerBlock) void add_move_kernel(
    DevForest F, const unsigned long long *keys, int64_t n_add, const int32_t *cstart,
    const MergeCounters *__restrict__ ctr, const int32_t *grp_nw, const int32_t *grp_nb, const int32_t *win_tok,
    long long stamp) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t nchunks = (int64_t)ctr->move_chunks;
    const int64_t waves = (int64_t)gridDim.x * kMergeWavesPerBlock;
    n_add = add_count(n_add, ctr);
    for (int64_t c = m_wave_index(); c < nchunks; c += waves) {
        // the group whose chunks hold c: cstart[k] <= c < cstart[k + 1]
        int64_t lo = 0, hi = n_add;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (cstart[mid] <= c)
                lo = mid + 1;
            else
                hi = mid;
        }
        const int64_t k = lo - 1;
        const int32_t nb = grp_nb[k];
        if (nb < 0) continue;
        const Node nx = F.nodes[key_parent(keys[k])];
        const int32_t j = (int32_t)(c - cstart[k]) * 64 + lane;
        if (j >= nx.ct_cnt) continue;
        const int32_t src = nx.ct_beg + j;
        const int64_t dst = nb + j + lower_count(win_tok + k, grp_nw[k], F.ntok[src]);
        F.nodes[dst] = F.nodes[src];
        F.ntok[dst] = F.ntok[src];
        if (F.ltime) F.ltime[dst] = F.ltime[src];
        for (int w = 0; w < F.W - 1; w++) F.mext[dst * (F.W - 1) + w] = F.mext[(int64_t)src * (F.W - 1) + w];
        F.moved[src] = (stamp << 32) | (long long)(uint32_t)dst;
    }
}

// Step 5 (one wave per winning entry): the leaf holding the rest of the
// winner's sequence, in its token's slot among the parent's children.
// pofs: nullptr after the multi-launch steps (spans from poff and grp_pb),
// else the one-workgroup plan's spans per insert from ctr->add_pool_base.
// Steps 5-7 stride over their entries, so a grid sized without the count
// (rounds the host does not read back) serves as well.
__global__ __launch_bounds__(64 *kMergeWavesPerBlock) void add_leaf_kernel(
    DevForest F, Batch B, const unsigned long long *keys, const int32_t *vals, int64_t n_add, InsState *st,
    const int32_t *win, const int32_t *widx, const int64_t *poff, const int32_t *hd, const int32_t *grp_nb,
    const int64_t *grp_pb, const int64_t *pofs, const MergeCounters *ctr) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t cnt = add_count(n_add, ctr);
    const int64_t waves = (int64_t)gridDim.x * kMergeWavesPerBlock;
    for (int64_t e = m_wave_index(); e < cnt; e += waves) {
        if (!win[e]) continue;
        const int32_t k = hd[e];
        const int32_t nb = grp_nb[k];
        if (nb < 0) continue;
        const int32_t i = vals[e];
        const Node nx = F.nodes[key_parent(keys[e])];
        const int32_t *s = B.tokens + B.offsets[i];
        const int64_t len = B.offsets[i + 1] - B.offsets[i];
        const int32_t d = st[i].d;
        const int64_t rest = len - d;  // >= 1: an ADD insert has a next token
        const int64_t dst = nb + (widx[e] - widx[k]) + lower_count(F.ntok + nx.ct_beg, nx.ct_cnt, s[d]);
        const int64_t pb = pofs ? (int64_t)ctr->add_pool_base + pofs[i] : grp_pb[k] + (poff[e] - poff[k]);
        const int32_t p = B.peer_of[i];
        copy_tokens(F.pool + pb, s + d, rest, lane);
        leaf_mext(F, dst, p, lane);
        if (lane == 0) {
            Node leaf;
            leaf.tok = s[d];
            leaf.lab_off = (uint32_t)pb;
            leaf.lab_len = (int32_t)rest;
            leaf.ct_beg = 0;
            leaf.ct_cnt = 0;
            leaf.aux = 0;
            leaf.mask0 = (p >> 6) == 0 ? 1ull << (p & 63) : 0ull;  // the winner's peer holds its leaf
            F.nodes[dst] = leaf;
            F.ntok[dst] = leaf.tok;
            if (F.ltime) F.ltime[dst] = (B.stamp && p == F.local) ? F.now : 0ull;
            st[i].kind = kInsDone;  // the winner's sequence ends at its new leaf
        }
    }
}

// Separators of every rebuilt wide block (runs after the build, before the
// parents are pointed at their new blocks; the old record of x still holds the
// old child count).
__global__ __launch_bounds__(64 *kMergeWavesPerBlock) void add_sep_kernel(DevForest F,
                                                                         const unsigned long long *keys,
                                                                         int64_t n_add, const int32_t *grp_nw,
                                                                         const int32_t *grp_nb,
                                                                         const MergeCounters *ctr) {
    const int lane = (int)(threadIdx.x & 63);
    const int64_t cnt = add_count(n_add, ctr);
    const int64_t waves = (int64_t)gridDim.x * kMergeWavesPerBlock;
    for (int64_t k = m_wave_index(); k < cnt; k += waves) {
        if (k > 0 && key_parent(keys[k - 1]) == key_parent(keys[k])) continue;
        const int32_t nb = grp_nb[k];
        if (nb < 0) continue;
        const int32_t c = F.nodes[key_parent(keys[k])].ct_cnt + grp_nw[k];
        if (c <= kSepCount) continue;
        F.nsep[nb + lane] = F.ntok[nb + PR_SEP_INDEX(lane, c)];
        if (c < kSep2Min) continue;
        sep2_write(F.nsep + nb, F.ntok + nb, c, lane);
    }
}

// Point every rebuilt parent at its new block, wherever its record lives now.
__global__ void add_fix_kernel(DevForest F, const unsigned long long *keys, int64_t n_add, const int32_t *grp_nw,
                               const int32_t *grp_nb, long long stamp, const MergeCounters *ctr) {
    const int64_t cnt = add_count(n_add, ctr);
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < cnt; k += (int64_t)gridDim.x * blockDim.x) {
        if (k > 0 && key_parent(keys[k - 1]) == key_parent(keys[k])) continue;
        if (grp_nb[k] < 0) continue;  // the build of this group was refused
        const int32_t x = key_parent(keys[k]);
        const long long mv = F.moved[x];
        const int64_t pos = (mv >> 32) == stamp ? (int64_t)(uint32_t)mv : (int64_t)x;
        F.nodes[pos].ct_cnt = F.nodes[pos].ct_cnt + grp_nw[k];
        F.nodes[pos].ct_beg = grp_nb[k];
    }
}

// A replaced snapshot: remove peer p from every mask (its old paths stay as
// structure that no peer holds until something is inserted there again).
__global__ void clear_peer_kernel(DevForest F, int64_t n_nodes, int32_t p) {
    const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= n_nodes) return;
    const int32_t w = p >> 6;
    const unsigned long long keep = ~(1ull << (p & 63));
    if (w == 0)
        F.nodes[x].mask0 &= keep;
    else
        F.mext[x * (F.W - 1) + (w - 1)] &= keep;
}

// Fill a peer id array (snapshot loads insert every sequence into one peer).
__global__ void fill_peer_kernel(int32_t *peer_of, int64_t n, int32_t p) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) peer_of[i] = p;
}

}  // namespace pr

#endif
