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

constexpr int kWave = 64;
constexpr int kRouteWavesPerBlock = PR_ROUTE_WAVES_PER_BLOCK;
constexpr int kLcpVectors = PR_LCP_VECTORS;    // 64-token vectors compared per step
constexpr int kWideVectors = PR_WIDE_VECTORS;  // first tokens held per lane for wide blocks

// Length of the common prefix of a[0..n) and b[0..n): the first i < n with
// a[i] != b[i], or n.  Wave-cooperative; every lane returns the same value.
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
                vb[j] = b[i];
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
    if (cnt <= kWave) {
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
    if (cb.cnt <= kWave) {
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
