// route_kernels.h -- gfx950 kernels of the batched router (device code).
//
// One wavefront (64 lanes) serves one query.  The wave walks the union forest
// from the root:
//   child locate  : lanes load the node's sorted (first token, child) slots and
//                   a ballot finds the slot equal to the next query token; wide
//                   tables are first narrowed by a 64-ary separator search;
//   mask narrowing: the wave-uniform set of peers still matching is ANDed with
//                   the child's peer mask; every peer that drops out records
//                   the depth reached so far (lane i owns peers i, i+64, ...);
//   label compare : lanes compare label and query tokens 64 x U per step and a
//                   ballot of mismatches gives the common-prefix length.
// Peers still in the set at the end matched the whole walked depth.  A wave
// reduction then takes the largest match and the lowest peer id holding it
// (the argmax of Algorithm 1, ties to the lowest id).
#ifndef PR_ROUTE_KERNELS_H
#define PR_ROUTE_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forest_layout.h"

namespace pr {

constexpr int kWave = 64;
constexpr int kRouteWavesPerBlock = 4;
constexpr int kLcpVectors = 4;   // 64-token vectors compared per step (256 tokens)
constexpr int kScanVectors = 4;  // child slots scanned per step: 64 x 4 = 256

__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

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
            if (bal) {
                const int64_t r = base + j * kWave + (__ffsll((unsigned long long)bal) - 1);
                return r;
            }
        }
    }
    return n;
}

// Child of a node whose first label token is t, or -1.  ct[0..cnt) is sorted
// by token (distinct tokens).
__device__ __forceinline__ int32_t find_child(const ChildSlot *__restrict__ ct, int32_t cnt, int32_t t, int lane) {
    int32_t lo = 0, hi = cnt;
    while (hi - lo > kWave * kScanVectors) {
        const int32_t stride = (hi - lo + kWave - 1) / kWave;
        const int32_t idx = lo + lane * stride;
        bool le = false;
        if (idx < hi) le = ct[idx].tok <= t;
        const uint64_t b = __ballot(le);
        if (!b) return -1;  // t is below every token
        const int32_t k = __popcll(b) - 1;  // separators ascend, so set lanes are a prefix
        lo = lo + k * stride;
        hi = min(lo + stride, hi);
    }
    int32_t tok[kScanVectors], node[kScanVectors];
#pragma unroll
    for (int j = 0; j < kScanVectors; j++) {
        const int32_t idx = lo + j * kWave + lane;
        tok[j] = 0;
        node[j] = -1;
        if (idx < hi) {
            const ChildSlot s = ct[idx];
            tok[j] = s.tok;
            node[j] = s.node;
        }
    }
#pragma unroll
    for (int j = 0; j < kScanVectors; j++) {
        const int32_t idx = lo + j * kWave + lane;
        const uint64_t b = __ballot(idx < hi && tok[j] == t);
        if (b) return __builtin_amdgcn_readlane(node[j], (int)(__ffsll((unsigned long long)b) - 1));
    }
    return -1;
}

template <int W>
__global__ __launch_bounds__(kWave *kRouteWavesPerBlock) void route_kernel(
    const Node *__restrict__ nodes, const uint64_t *__restrict__ masks, const ChildSlot *__restrict__ ctab,
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
    Node nx = nodes[0];
    while (d < qlen && nx.ct_cnt > 0) {
        const int32_t t = qs[d];
        const int32_t c = find_child(ctab + nx.ct_beg, nx.ct_cnt, t, lane);
        if (c < 0) break;
        const Node nc = nodes[c];
        if (nc.lab_len <= 0) break;  // only the root has an empty label
        bool any = false;
#pragma unroll
        for (int w = 0; w < W; w++) {
            const uint64_t nm = alive[w] & masks[(int64_t)c * W + w];
            if (((alive[w] & ~nm) >> lane) & 1ull) m[w] = (int32_t)d;
            alive[w] = nm;
            any |= nm != 0ull;
        }
        if (!any) break;  // no peer holds this edge (left behind by a replaced snapshot)
        const int64_t n = min((int64_t)nc.lab_len, qlen - d);
        const int64_t l = wave_lcp(pool + nc.lab_off, qs + d, n, lane);
        d += l;
        if (l < nc.lab_len) break;
        nx = nc;
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
