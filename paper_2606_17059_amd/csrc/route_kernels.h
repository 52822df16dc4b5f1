// route_kernels.h -- gfx950 kernels of the batched router (device code).
//
// One wavefront (64 lanes) serves one query and walks the union forest from
// the root.  Per tree level the wave
//   1. locates the child whose first label token is the next query token:
//      the node's child block was already loaded into the lanes (one child
//      record per lane for blocks of <= 64 children, 8 first tokens per lane
//      for blocks of <= 512, a 64-ary separator search beyond that), so a
//      ballot finds the child and the lanes already hold its record;
//   2. issues, in one batch, the loads of the child's label, of the matching
//      query tokens (64 x kLcpVectors per step), of the query token after the
//      label and of the child's own child block (speculatively, for the next
//      level), so one memory round trip serves the whole level;
//   3. narrows the wave-uniform set of peers still matching by the child's peer
//      mask; every peer that drops out records the depth reached so far (lane
//      i owns peers i, i+64, ...), and takes the common-prefix length of label
//      and query from a ballot of mismatches.
// Peers still in the set at the end matched the whole walked depth.  A wave
// reduction then takes the largest match and the lowest peer id holding it
// (the argmax of Algorithm 1, ties to the lowest id).
#ifndef PR_ROUTE_KERNELS_H
#define PR_ROUTE_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"
#include "wave_ops.h"

namespace pr {

#ifndef PR_ROUTE_WAVES_PER_BLOCK
#define PR_ROUTE_WAVES_PER_BLOCK 4
#endif
#ifndef PR_LCP_VECTORS
#define PR_LCP_VECTORS 8
#endif
#ifndef PR_WIDE_VECTORS
#define PR_WIDE_VECTORS 8
#endif
#ifndef PR_ROUTE_LDS
#define PR_ROUTE_LDS 1
#endif
#ifndef PR_QUERY_NT
#define PR_QUERY_NT 1
#endif
#ifndef PR_NARROW_RECORDS
#define PR_NARROW_RECORDS 0
#endif

constexpr int kWave = 64;
constexpr int kRouteWavesPerBlock = PR_ROUTE_WAVES_PER_BLOCK;
constexpr int kLcpVectors = PR_LCP_VECTORS;    // 64-token vectors compared per step
constexpr int kWideVectors = PR_WIDE_VECTORS;  // first tokens held per lane for wide blocks


// Query tokens are read once: mark their loads non-temporal so they stream
// through the caches that hold the forest's labels.
__device__ __forceinline__ int32_t load_stream(const int32_t *p) {
#if PR_QUERY_NT
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}

// Length of the common prefix of a[0..n) (a label) and b[0..n) (query
// tokens): the first i < n with a[i] != b[i], or n.  Wave-cooperative; every
// lane returns the same value.
__device__ __forceinline__ int64_t wave_lcp(const int32_t *__restrict__ a, const int32_t *__restrict__ b,
                                            int64_t n, int lane) {
    for (int64_t base = 0; base < n; base += (int64_t)kWave * kLcpVectors) {
        int32_t va[kLcpVectors], vb[kLcpVectors];
#pragma unroll
        for (int j = 0; j < kLcpVectors; j++) {
            const int64_t i = base + j * kWave + lane;
            va[j] = 0;
            vb[j] = 0;
            if (i < n) {
                va[j] = a[i];
                vb[j] = load_stream(b + i);
            }
        }
#pragma unroll
        for (int j = 0; j < kLcpVectors; j++) {
            const int64_t i = base + j * kWave + lane;
            const uint64_t bal = __ballot(i < n && va[j] != vb[j]);
            if (bal) return base + j * kWave + (__ffsll((unsigned long long)bal) - 1);
        }
    }
    return n;
}

// A node's child block as held by the wave.
struct ChildBlock {
    int32_t beg, cnt;  // uniform
    // cnt <= 64: lane j holds the record of child beg + j
    int32_t tok, lab_off, lab_len, ct_beg, ct_cnt;
    uint64_t mask0;
    // 64 < cnt <= 64 * kWideVectors: lane j holds ntok[beg + 64 v + j]
    int32_t wt[kWideVectors];
};

// Uniform view of the located child.
struct Child {
    int32_t id, lab_off, lab_len, ct_beg, ct_cnt;
    uint64_t mask0;
};

__device__ __forceinline__ void load_block(ChildBlock &cb, const Node *__restrict__ nodes,
                                           const int32_t *__restrict__ ntok, int32_t beg, int32_t cnt, int lane) {
    cb.beg = beg;
    cb.cnt = cnt;
    cb.tok = 0;
    cb.lab_off = 0;
    cb.lab_len = 0;
    cb.ct_beg = 0;
    cb.ct_cnt = 0;
    cb.mask0 = 0ull;
    if (PR_NARROW_RECORDS && cnt <= kWave) {
        if (lane < cnt) {
            const Node r = nodes[beg + lane];
            cb.tok = r.tok;
            cb.lab_off = (int32_t)r.lab_off;
            cb.lab_len = r.lab_len;
            cb.ct_beg = r.ct_beg;
            cb.ct_cnt = r.ct_cnt;
            cb.mask0 = r.mask0;
        }
    } else if (cnt <= kWave * kWideVectors) {
#pragma unroll
        for (int v = 0; v < kWideVectors; v++) {
            const int32_t j = v * kWave + lane;
            cb.wt[v] = j < cnt ? ntok[beg + j] : 0;
        }
    }
}

// Find the child whose first token is t.  Returns false if there is none.
__device__ __forceinline__ bool locate(const ChildBlock &cb, int32_t t, const Node *__restrict__ nodes,
                                       const int32_t *__restrict__ ntok, int lane, Child &c) {
    if (PR_NARROW_RECORDS && cb.cnt <= kWave) {
        const uint64_t b = __ballot(lane < cb.cnt && cb.tok == t);
        if (!b) return false;
        const int src = (int)(__ffsll((unsigned long long)b) - 1);
        c.id = cb.beg + src;
        c.lab_off = __builtin_amdgcn_readlane(cb.lab_off, src);
        c.lab_len = __builtin_amdgcn_readlane(cb.lab_len, src);
        c.ct_beg = __builtin_amdgcn_readlane(cb.ct_beg, src);
        c.ct_cnt = __builtin_amdgcn_readlane(cb.ct_cnt, src);
        c.mask0 = readlane64(cb.mask0, src);
        return true;
    }
    int32_t idx = -1;
    if (cb.cnt <= kWave * kWideVectors) {
#pragma unroll
        for (int v = 0; v < kWideVectors; v++) {
            const uint64_t b = __ballot(v * kWave + lane < cb.cnt && cb.wt[v] == t);
            if (b) {
                idx = v * kWave + (int32_t)(__ffsll((unsigned long long)b) - 1);
                break;
            }
        }
    } else {
        // 64-ary search: separators ascend, so the lanes with sep <= t form a prefix
        int32_t lo = 0, hi = cb.cnt;
        while (hi - lo > kWave) {
            const int32_t stride = (hi - lo + kWave - 1) / kWave;
            const int32_t j = lo + lane * stride;
            bool le = false;
            if (j < hi) le = ntok[cb.beg + j] <= t;
            const uint64_t b = __ballot(le);
            if (!b) return false;
            lo = lo + (__popcll(b) - 1) * stride;
            hi = min(lo + stride, hi);
        }
        const int32_t j = lo + lane;
        bool eq = false;
        if (j < hi) eq = ntok[cb.beg + j] == t;
        const uint64_t b = __ballot(eq);
        if (b) idx = lo + (int32_t)(__ffsll((unsigned long long)b) - 1);
    }
    if (idx < 0) return false;
    const Node r = nodes[cb.beg + idx];
    c.id = cb.beg + idx;
    c.lab_off = (int32_t)r.lab_off;
    c.lab_len = r.lab_len;
    c.ct_beg = r.ct_beg;
    c.ct_cnt = r.ct_cnt;
    c.mask0 = r.mask0;
    return true;
}

// The query is staged in a per-wave LDS ring of kRing tokens: position p of
// the query lives at ring[p % kRing].  Direct global->LDS loads (one dword per
// lane, 64 consecutive positions per instruction) fill it without passing
// through VGPRs, so a whole edge's worth of query tokens can be in flight while
// the wave holds only the label tokens it compares.  Only positions the walk
// may read are fetched, and never more than kRing ahead of the current depth.
constexpr int kRing = 1024;

typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(1))) void global_void_t;

// Issue the loads of query positions [from, to) into the ring (to <= query
// length, to - from <= kRing).  Lanes outside the range do not load.
__device__ __forceinline__ void ring_fetch(int32_t *ring, const int32_t *__restrict__ qs, int64_t from, int64_t to,
                                           int lane) {
    for (int64_t v = from & ~(int64_t)(kWave - 1); v < to; v += kWave) {
        const int64_t p = v + lane;
        if (p >= from && p < to)
            __builtin_amdgcn_global_load_lds((global_void_t *)(qs + p), (lds_void_t *)(ring + (v & (kRing - 1))), 4,
                                             0, 0);
    }
}

// Wait until every vector memory operation of the wave, the ring loads
// included, has completed (s_waitcnt vmcnt(0) expcnt(7) lgkmcnt(15)).
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <int W>
__global__ __launch_bounds__(kWave *kRouteWavesPerBlock) void route_kernel(
    const Node *__restrict__ nodes, const int32_t *__restrict__ ntok, const uint64_t *__restrict__ mext,
    const int32_t *__restrict__ pool, const int32_t *__restrict__ qtok, int64_t num_tokens,
    const int64_t *__restrict__ qoff, int64_t nq, int32_t P, int32_t *__restrict__ match_len,
    int32_t *__restrict__ chosen) {
    const int lane = (int)(threadIdx.x & (kWave - 1));
    const int64_t q = (int64_t)blockIdx.x * kRouteWavesPerBlock + uniform((int32_t)(threadIdx.x / kWave));
    if (q >= nq) return;
    int32_t *row = match_len + q * (int64_t)P;
    const int64_t qb = qoff[q], qe = qoff[q + 1];
    if (qb < 0 || qe < qb || qe > num_tokens || qe - qb > (int64_t)INT32_MAX) {
        for (int p = lane; p < P; p += kWave) row[p] = -1;
        if (lane == 0) chosen[q] = -1;
        return;
    }
    const int32_t *qs = qtok + qb;
    const int64_t qlen = qe - qb;

    int32_t m[W];
    uint64_t alive[W];
#pragma unroll
    for (int w = 0; w < W; w++) {
        m[w] = 0;
        const int rem = P - 64 * w;
        alive[w] = rem >= 64 ? ~0ull : (rem > 0 ? ((1ull << rem) - 1ull) : 0ull);
    }

#if PR_ROUTE_LDS
    __shared__ int32_t ring_all[kRouteWavesPerBlock][kRing];
    int32_t *ring = ring_all[threadIdx.x / kWave];
    int64_t d = 0;
    int64_t fetched = 0;  // query positions [0, fetched) have ring loads issued
    ChildBlock cb;
    // the first positions of the query are fetched speculatively, beside the root block
    {
        const int64_t f0 = min(qlen, (int64_t)kLcpVectors * kWave);
        ring_fetch(ring, qs, 0, f0, lane);
        fetched = f0;
        const Node root = nodes[0];
        load_block(cb, nodes, ntok, root.ct_beg, root.ct_cnt, lane);
        wait_vm_all();
    }
    int32_t t = qlen > 0 ? ring[0] : 0;
    while (d < qlen) {
        Child c;
        if (!locate(cb, t, nodes, ntok, lane, c)) break;
        if (c.lab_len <= 0) break;  // only the root has an empty label
        const int64_t eend = d + c.lab_len;          // depth at the child
        const int64_t want = min(qlen, eend + 1);     // positions this level may read
        const int64_t lend = min(eend, qlen);         // compared positions: [d, lend)
        // one batch per level: the query tokens of the whole label (as far as
        // the ring allows), the child's mask words and child block, and the
        // first segment's labels
        {
            const int64_t to = min(want, d + kRing);
            if (to > fetched) {
                ring_fetch(ring, qs, fetched, to, lane);
                fetched = to;
            }
        }
        uint64_t mx[W];
        mx[0] = c.mask0;
#pragma unroll
        for (int wi = 1; wi < W; wi++) mx[wi] = mext[(int64_t)c.id * (W - 1) + (wi - 1)];
        load_block(cb, nodes, ntok, c.ct_beg, c.ct_cnt, lane);
        const int32_t *lab = pool + (uint32_t)c.lab_off;
        int64_t l = lend - d;
        for (int64_t base = d; base < lend; base += (int64_t)kWave * kLcpVectors) {
            if (base > d) {  // later segments: top the ring up to what it can hold
                const int64_t to = min(want, base + kRing);
                if (to > fetched) {
                    ring_fetch(ring, qs, fetched, to, lane);
                    fetched = to;
                }
            }
            int32_t lv[kLcpVectors];
#pragma unroll
            for (int j = 0; j < kLcpVectors; j++) {
                const int64_t p = base + j * kWave + lane;
                lv[j] = 0;
                if (p < lend) lv[j] = lab[p - d];
            }
            wait_vm_all();
            int64_t found = -1;
#pragma unroll
            for (int j = 0; j < kLcpVectors; j++) {
                const int64_t p = base + j * kWave + lane;
                bool mis = false;
                if (p < lend) mis = ring[p & (kRing - 1)] != lv[j];
                const uint64_t b = __ballot(mis);
                if (b && found < 0) found = base + j * kWave + (__ffsll((unsigned long long)b) - 1);
            }
            if (found >= 0) {
                l = found - d;
                break;
            }
        }
        bool any = false;
#pragma unroll
        for (int wi = 0; wi < W; wi++) {
            const uint64_t nm = alive[wi] & mx[wi];
            if (((alive[wi] & ~nm) >> lane) & 1ull) m[wi] = (int32_t)d;
            alive[wi] = nm;
            any |= nm != 0ull;
        }
        if (!any) break;  // no peer holds this edge (left behind by a replaced snapshot)
        d += l;
        if (l < c.lab_len || d >= qlen) break;
        // next token: in the ring (fetched with the label) unless the label ran
        // past the ring's reach
        if (d >= fetched) {
            const int64_t to = min(qlen, d + (int64_t)kLcpVectors * kWave);
            ring_fetch(ring, qs, d, to, lane);
            fetched = to;
        }
        wait_vm_all();
        t = ring[d & (kRing - 1)];
    }
#else
    int64_t d = 0;
    ChildBlock cb;
    {
        const Node root = nodes[0];
        load_block(cb, nodes, ntok, root.ct_beg, root.ct_cnt, lane);
    }
    int32_t t = qlen > 0 ? qs[0] : 0;
    while (d < qlen) {
        Child c;
        if (!locate(cb, t, nodes, ntok, lane, c)) break;
        if (c.lab_len <= 0) break;  // only the root has an empty label
        // one batch of loads per level: next token, ext mask words, the next
        // child block (used if the label matches in full) and the label compare
        const int64_t end = d + c.lab_len;
        const int32_t tnext = end < qlen ? qs[end] : 0;
        uint64_t mx[W];
        mx[0] = c.mask0;
#pragma unroll
        for (int w = 1; w < W; w++) mx[w] = mext[(int64_t)c.id * (W - 1) + (w - 1)];
        load_block(cb, nodes, ntok, c.ct_beg, c.ct_cnt, lane);
        const int64_t n = min((int64_t)c.lab_len, qlen - d);
        const int64_t l = wave_lcp(pool + (uint32_t)c.lab_off, qs + d, n, lane);
        bool any = false;
#pragma unroll
        for (int w = 0; w < W; w++) {
            const uint64_t nm = alive[w] & mx[w];
            if (((alive[w] & ~nm) >> lane) & 1ull) m[w] = (int32_t)d;
            alive[w] = nm;
            any |= nm != 0ull;
        }
        if (!any) break;  // no peer holds this edge (left behind by a replaced snapshot)
        d += l;
        if (l < c.lab_len) break;
        t = tnext;
    }

#endif

    // peers still holding the walked path matched all of it
    int32_t bm = -1, bp = INT32_MAX;
#pragma unroll
    for (int w = 0; w < W; w++) {
        if ((alive[w] >> lane) & 1ull) m[w] = (int32_t)d;
        const int p = lane + 64 * w;
        if (p < P && m[w] > bm) {
            bm = m[w];
            bp = p;
        }
    }
    // argmax over peers: the largest match, then the lowest peer id holding it
    int32_t M = bm;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = max(M, __shfl_xor(M, off));
    int32_t cand = (bm == M) ? bp : INT32_MAX;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) cand = min(cand, __shfl_xor(cand, off));

#pragma unroll
    for (int w = 0; w < W; w++) {
        const int p = lane + 64 * w;
        if (p < P) row[p] = m[w];
    }
    if (lane == 0) chosen[q] = cand;
}

}  // namespace pr

#endif
