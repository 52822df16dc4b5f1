// route_kernels.h -- gfx950 kernel of the batched router (device code).
//
// One wavefront (64 lanes) serves one query and walks the union forest from
// the root.  Per tree level the wave
//   1. locates the child whose first label token is the next query token: the
//      node's child block was already loaded into the lanes (its first tokens
//      for up to 64 children, else its 64 separators, two cache lines either
//      way), a ballot finds the slot (for a wide block, the sub-range whose
//      first tokens one more load brings), and one scalar load fetches the
//      child's 32-byte record;
//   2. issues, in one batch, the loads of the query token after the label, of
//      the child's mask words, of the child's own first-token array
//      (speculatively, for the next level), and of the label and query tokens
//      it compares: raw buffer loads ranged to the step, 64 tokens per
//      instruction, all of a step in flight at once; query tokens are read
//      once, so their loads are non-temporal (except the first level's, which
//      come with the query's first token, before the walk starts);
//   3. narrows the wave-uniform set of peers still matching by the child's peer
//      mask; every peer that drops out records the depth reached so far (lane
//      i owns peers i, i+64, ...), and takes the common-prefix length of label
//      and query from a ballot of mismatches.
// Peers still in the set at the end matched the whole walked depth.  A wave
// reduction then takes the largest match and the lowest peer id holding it
// (the argmax of Algorithm 1, ties to the lowest id).  Rows of whole cache
// lines are stored non-temporally, so that they do not evict labels.
// When the root has a single child (a prompt prefix every stored sequence
// shares), its record is loaded before the walk and the first level's batch
// goes out without waiting for the query's first token.  The first level
// compares its label against a window of the query's first 128 tokens, or 256
// when the host chose the wide window for a long shared prefix.  Batches of long
// queries can be served in an order computed on the device (longest first,
// route_order_count_kernel and route_order_scatter_kernel below).
// Labels are read from the int32 pool, or, while every label token lies in
// [0, 65535], from a 16-bit copy of it (half the label bytes and requests; a
// query token outside that range equals no label token either way), or,
// while every label token lies in [0, 131071], from that copy of the low 16
// bits plus a plane of bit 16 (one 32-bit word per 32 tokens, loaded once per
// compare step and handed to the lanes by cross-lane permutes).
#ifndef PR_ROUTE_KERNELS_H
#define PR_ROUTE_KERNELS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "forest_layout.h"
#include "wave_ops.h"

#ifndef PR_ROUTE_WAVES_PER_BLOCK
#define PR_ROUTE_WAVES_PER_BLOCK 1
#endif
#ifndef PR_LCP_VECTORS
#define PR_LCP_VECTORS 16
#endif
#ifndef PR_LCP_FIRST_VECTORS
#define PR_LCP_FIRST_VECTORS 9
#endif
#ifndef PR_QUERY_NT
#define PR_QUERY_NT 1
#endif
#ifndef PR_ALIGN_STEPS
#define PR_ALIGN_STEPS 1
#endif
#ifndef PR_FIRST_WINDOW
#define PR_FIRST_WINDOW 1
#endif
#ifndef PR_WIN_VECTORS
#define PR_WIN_VECTORS 2
#endif
#ifndef PR_ROUTE_WAVES_PER_EU
#define PR_ROUTE_WAVES_PER_EU 8
#endif
#ifndef PR_OUT_NT
#define PR_OUT_NT 1
#endif
#ifndef PR_WIN_POLICY
#define PR_WIN_POLICY 0
#endif

namespace pr {

constexpr int kWave = 64;
constexpr int kRouteWavesPerBlock = PR_ROUTE_WAVES_PER_BLOCK;
constexpr int kLcpVectors = PR_LCP_VECTORS;               // 64-token vectors per compare step
constexpr int kLcpFirstVectors = PR_LCP_FIRST_VECTORS;    // ... in a label's first step

// Raw buffer resource over bytes [p, p + bytes): loads past the end return 0
// without touching memory (the hardware range check of stride-0 buffers).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t token_rsrc(const int32_t *p, int32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(p), (short)0, bytes, 0x00020000);
}

// Cache policy of the query loads: non-temporal (read once).
#ifdef PR_QUERY_POLICY
constexpr int kQueryPolicy = PR_QUERY_POLICY;
#else
constexpr int kQueryPolicy = PR_QUERY_NT ? 2 : 0;
#endif

// Output stores of the match rows.  They are written once and never read by
// the kernel; when a row fills whole 128-byte lines (P a multiple of 32),
// non-temporal stores keep them from pushing the labels, which every query
// reads, out of the L2.  Shorter rows share lines with their neighbours, which
// plain stores let the L2 merge (as for the 4-byte chosen peer).  The
// non-temporal path is a raw buffer store over the row (a different operation
// from the plain store, so the compiler cannot fold the two paths into one
// store and lose the policy); lanes past the row are dropped by its range.
template <int W>
__device__ __forceinline__ void store_row(int32_t *row, const int32_t (&m)[W], int32_t P, int lane) {
#if PR_OUT_NT
    if ((P & 31) == 0) {
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(row, (short)0, P * 4, 0x00020000);
#pragma unroll
        for (int w = 0; w < W; w++) __builtin_amdgcn_raw_buffer_store_b32(m[w], r, (lane + 64 * w) * 4, 0, 2);
        return;
    }
#endif
#pragma unroll
    for (int w = 0; w < W; w++) {
        const int p = lane + 64 * w;
        if (p < P) row[p] = m[w];
    }
}

// Label tokens: int32, or uint16 (the 16-bit copy of the pool).  Raw buffer
// resources over the label bytes and loads of one token per lane.
template <typename LT>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t label_rsrc(const LT *p, int32_t cnt) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<LT *>(p), (short)0, cnt * (int32_t)sizeof(LT), 0x00020000);
}

template <typename LT>
__device__ __forceinline__ int32_t load_label(__amdgpu_buffer_rsrc_t r, int32_t off) {
    if constexpr (sizeof(LT) == 2)
        return (int32_t)(uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
    else
        return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}

// Where a compare step reads its labels.  p: the label's first token in the
// pool (int32), or in its 16-bit copy.  HB (17-bit labels, with the 16-bit
// copy): bit 16 of pool token i is bit i % 32 of hib[i / 32], and abs is the
// label's offset in the pool, so that a step knows which bit words to load.
template <typename LT, bool HB>
struct LabelSrc {
    const LT *p;
    const uint32_t *hib;
    uint32_t abs;
};

// The bit words of a step over pool tokens [A, A + cnt), A = abs + base: lane w
// holds word A / 32 + w (w <= 32 for cnt <= 1024), with the bits of tokens at
// or past A + cnt cleared, so that lanes past the step compare equal as with
// plain labels.  Lane l of every 64-token vector j then takes bit
// (A % 32 + l) % 32 of lane 2 j + (A % 32 + l) / 32's word (hb_take).
struct HiBits {
    uint32_t word;   // this lane's bit word
    int32_t addr;    // ds_bpermute byte address of vector 0's source lane
    uint32_t shift;  // bit position inside it
};

// The load is issued by hb_load; hb_trim, called once every load of the step
// has been issued, clears the bits past the step (so that the first use of
// the word does not make the compiler wait on it before the other loads).
__device__ __forceinline__ HiBits hb_load(const uint32_t *hib, uint32_t A, int32_t cnt, int lane) {
    const uint32_t a0 = A & 31u;
    const int32_t nwords = (int32_t)((a0 + (uint32_t)cnt + 31u) >> 5);
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t *>(hib + (A >> 5)), (short)0, nwords * 4, 0x00020000);
    HiBits h;
    h.word = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, lane * 4, 0, 0);
    h.addr = (int32_t)(((a0 + (uint32_t)lane) >> 5) << 2);
    h.shift = (a0 + (uint32_t)lane) & 31u;
    return h;
}

__device__ __forceinline__ void hb_trim(HiBits &h, uint32_t A, int32_t cnt, int lane) {
    const int32_t lim = cnt + (int32_t)(A & 31u) - 32 * lane;  // bits of this lane's word inside the step
    h.word = lim >= 32 ? h.word : (lim <= 0 ? 0u : h.word & ((1u << lim) - 1u));
}

// Bit 16 of the label token lane `lane` holds in vector j.
__device__ __forceinline__ int32_t hb_take(const HiBits &h, int j) {
    const uint32_t w = (uint32_t)__builtin_amdgcn_ds_bpermute(h.addr + 8 * j, (int32_t)h.word);
    return (int32_t)(((w >> h.shift) & 1u) << 16);
}

// One compare step over cnt <= 64 * NV tokens: ra holds the label tokens
// (LT wide), rb the query tokens, both ranged to cnt tokens so that lanes past
// the end read 0 on both sides and compare equal.  Returns the first
// mismatch, or -1.
template <int NV, typename LT, bool HB = false>
__device__ __forceinline__ int32_t lcp_step(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb, int lane,
                                            const uint32_t *hib = nullptr, uint32_t A = 0, int32_t cnt = 0) {
    int32_t va[NV], vb[NV];
    // opaque lane offset: with its range unknown the per-vector constant stays
    // an add, which folds into the loads' immediate offsets; and as each step
    // size gets its own opaque value, the compiler cannot merge the first loads
    // of the short and the long step into one block that waits before the long
    // step issues the rest
    int32_t off = lane * 4;
    asm volatile("" : "+v"(off));
    // 16-bit labels take their own (opaque) lane offset
    int32_t offa = off;
    if constexpr (sizeof(LT) != 4) {
        offa = lane * (int32_t)sizeof(LT);
        asm volatile("" : "+v"(offa));
    }
#pragma unroll
    for (int j = 0; j < NV; j++) {
        va[j] = load_label<LT>(ra, offa + j * kWave * (int32_t)sizeof(LT));
        vb[j] = __builtin_amdgcn_raw_buffer_load_b32(rb, off + j * kWave * 4, 0, kQueryPolicy);
    }
    if constexpr (HB) {
        HiBits hb = hb_load(hib, A, cnt, lane);
        hb_trim(hb, A, cnt, lane);
#pragma unroll
        for (int j = 0; j < NV; j++) va[j] |= hb_take(hb, j);
    }
    // fold every vector's mismatches into a lane mask before branching, so
    // that no load of the step can be deferred behind an early exit
    uint32_t mm = 0;
#pragma unroll
    for (int j = 0; j < NV; j++) mm |= (uint32_t)(va[j] != vb[j]) << j;
    if (!__ballot(mm != 0)) return -1;
#pragma unroll
    for (int j = 0; j < NV; j++) {
        const uint64_t bal = __ballot((mm >> j) & 1u);
        if (bal) return j * kWave + (int32_t)(__ffsll((unsigned long long)bal) - 1);
    }
    return -1;
}

// Length of the common prefix of a[0..n) (a label) and b[0..n) (query
// tokens), from position base on: the first i in [base, n) with a[i] != b[i],
// or n.  Wave-cooperative; every lane returns the same value.  The first step
// compares up to `first` tokens (a label's first step: 64 * kLcpFirstVectors,
// which bounds what a mismatch early in a long label reads in vain), later
// steps up to 64 * kLcpVectors, which halves the round trips over long labels
// that match in full.  Every step but a label's last ends at a query line, 0 to
// 31 tokens short of its nominal size; the nine-vector first step leaves the
// rest of a 1024-token label to an eight-vector step.  Steps of at most 128
// and 512 tokens take two- and eight-vector forms.
template <typename LT, bool HB>
__device__ __forceinline__ int64_t wave_lcp(const LabelSrc<LT, HB> &lab, const int32_t *__restrict__ b,
                                            int64_t n, int64_t base, int64_t first, int lane) {
    const LT *__restrict__ a = lab.p;
    for (int64_t step = first; base < n; step = (int64_t)kWave * kLcpVectors) {
        int32_t cnt = (int32_t)min(n - base, step);
#if PR_ALIGN_STEPS
        // a step that is not the label's last ends at a 128-byte line of the
        // query, so no line is split between two steps: its non-temporal read
        // would not keep the line in the L2 for the next step
        if (n - base > step) cnt -= (int32_t)(((uint32_t)((uintptr_t)(b + base) >> 2) + (uint32_t)step) & 31u);
#endif
        const __amdgpu_buffer_rsrc_t ra = label_rsrc(a + base, cnt);
        const __amdgpu_buffer_rsrc_t rb = token_rsrc(b + base, cnt * 4);
        const uint32_t A = lab.abs + (uint32_t)base;
        int32_t r;
        if (cnt <= 2 * kWave)
            r = lcp_step<2, LT, HB>(ra, rb, lane, lab.hib, A, cnt);
        else if (cnt <= 8 * kWave)
            r = lcp_step<8, LT, HB>(ra, rb, lane, lab.hib, A, cnt);
        else if (kLcpFirstVectors > 8 && kLcpVectors > kLcpFirstVectors && cnt <= kWave * kLcpFirstVectors)
            r = lcp_step<kLcpFirstVectors, LT, HB>(ra, rb, lane, lab.hib, A, cnt);
        else
            r = lcp_step<kLcpVectors, LT, HB>(ra, rb, lane, lab.hib, A, cnt);
        if (r >= 0 && r < cnt) return base + r;
        base += cnt;
    }
    return n;
}

constexpr int kWinVectors = PR_WIN_VECTORS;
constexpr int kWideWinVectors = 4;
static_assert(kWinVectors >= 2 && kWinVectors <= 16, "window of 2 to 16 vectors");

#if PR_FIRST_WINDOW
// First-level window: the query's first 64 * WV tokens are loaded into
// registers together with its first token, whose HBM round trip the walk
// waits for anyway, so that the first level's compare waits only on its label,
// which the L2 holds.  Lane l of vector j holds token 64 j + l (0 past the
// query).  The loads use the default cache policy: they also bring the lines
// that the first level's next-token load reads.  A window wider than the first
// level's label reads tokens that the second level reads again, so the wide
// window (kWideWinVectors) is for forests whose root has one child with a
// label of at least that many tokens (a long shared system prompt).

template <int WV>
__device__ __forceinline__ void load_window(int32_t (&win)[WV], const int32_t *p, int32_t cnt, int lane) {
    const __amdgpu_buffer_rsrc_t r = token_rsrc(p, cnt * 4);
    int32_t off = lane * 4;  // opaque, as in lcp_step
    asm volatile("" : "+v"(off));
#pragma unroll
    for (int j = 0; j < WV; j++)
        win[j] = __builtin_amdgcn_raw_buffer_load_b32(r, off + j * kWave * 4, 0, PR_WIN_POLICY);
}

// Label tokens [0, cnt) (ra, LT wide, cnt <= 64 * NL) against the window,
// which may hold query tokens past cnt: only lanes below cnt count.  Returns
// the first mismatch, or -1.
template <int NL, typename LT, bool HB, int WV>
__device__ __forceinline__ int32_t lcp_step_win(__amdgpu_buffer_rsrc_t ra, const int32_t (&win)[WV],
                                                int32_t cnt, int lane, const uint32_t *hib, uint32_t A) {
    int32_t va[NL];
    int32_t off = lane * (int32_t)sizeof(LT);  // opaque, as in lcp_step
    asm volatile("" : "+v"(off));
#pragma unroll
    for (int j = 0; j < NL; j++) va[j] = load_label<LT>(ra, off + j * kWave * (int32_t)sizeof(LT));
    if constexpr (HB) {
        HiBits hb = hb_load(hib, A, cnt, lane);
        hb_trim(hb, A, cnt, lane);
#pragma unroll
        for (int j = 0; j < NL; j++) va[j] |= hb_take(hb, j);
    }
    // both sides of the & are evaluated, so no label load becomes conditional
    uint32_t mm = 0;
#pragma unroll
    for (int j = 0; j < NL; j++) mm |= (uint32_t)((j * kWave + lane < cnt) & (va[j] != win[j])) << j;
    if (!__ballot(mm != 0)) return -1;
#pragma unroll
    for (int j = 0; j < NL; j++) {
        const uint64_t bal = __ballot((mm >> j) & 1u);
        if (bal) return j * kWave + (int32_t)(__ffsll((unsigned long long)bal) - 1);
    }
    return -1;
}

// wave_lcp for the first level, whose first query tokens are in win.
template <typename LT, bool HB, int WV>
__device__ __forceinline__ int64_t wave_lcp_first(const LabelSrc<LT, HB> &lab, const int32_t *__restrict__ b,
                                                  int64_t n, const int32_t (&win)[WV], int lane) {
    constexpr int32_t kTokens = kWave * WV;
    const int32_t cnt = (int32_t)min(n, (int64_t)kTokens);
    const __amdgpu_buffer_rsrc_t ra = label_rsrc(lab.p, cnt);
    const int32_t r = cnt <= 2 * kWave ? lcp_step_win<2, LT, HB, WV>(ra, win, cnt, lane, lab.hib, lab.abs)
                                       : lcp_step_win<WV, LT, HB, WV>(ra, win, cnt, lane, lab.hib, lab.abs);
    if (r >= 0 && r < cnt) return r;
    return wave_lcp<LT, HB>(lab, b, n, kTokens, (int64_t)kWave * kLcpVectors, lane);
}
#endif

// A node's child block as held by the wave: lane j holds the first token of
// child beg + j (cnt <= 64) or the block's separator j (cnt > 64).
struct ChildBlock {
    int32_t beg, cnt;  // uniform
    int32_t tok;
};

// Uniform view of the located child.
struct Child {
    int32_t id, lab_off, lab_len, ct_beg, ct_cnt;
    uint64_t mask0;
};

__device__ __forceinline__ void load_block(ChildBlock &cb, const int32_t *__restrict__ ntok,
                                           const int32_t *__restrict__ nsep, int32_t beg, int32_t cnt, int lane) {
    cb.beg = beg;
    cb.cnt = cnt;
    cb.tok = 0;
    if (cnt > kSepCount)
        cb.tok = nsep[beg + lane];
    else if (lane < cnt)
        cb.tok = ntok[beg + lane];
}

// Find the child whose first token is t.  Returns false if there is none.
__device__ __forceinline__ bool locate(const ChildBlock &cb, int32_t t, const Node *__restrict__ nodes,
                                       const int32_t *__restrict__ ntok, const int32_t *__restrict__ nsep, int lane,
                                       Child &c) {
    int32_t idx = -1;
    if (cb.cnt <= kSepCount) {
        const uint64_t b = __ballot(lane < cb.cnt && cb.tok == t);
        if (b) idx = (int32_t)(__ffsll((unsigned long long)b) - 1);
    } else {
        // separators ascend, so the lanes with sep <= t form a prefix
        const uint64_t b = __ballot(cb.tok <= t);
        if (!b) return false;  // t is below every first token
        const int32_t k = (int32_t)__popcll(b) - 1;
        int32_t lo = PR_SEP_INDEX(k, cb.cnt);
        int32_t hi = PR_SEP_HI(k, cb.cnt);
        if (cb.cnt >= kSep2Min) {
            // blocks of 4,160 children or more: the sub-range's own 64
            // separators, two contiguous lines (lane 0's is the first level's
            // k-th, <= t); the rest is at most ceil(span / 64) first tokens
            const int32_t span = hi - lo;
            const uint64_t b2 = __ballot(nsep[cb.beg + kSepCount + kSepCount * k + lane] <= t);
            const int32_t j = (int32_t)__popcll(b2) - 1;
            hi = lo + PR_SEP_HI(j, span);
            lo += PR_SEP_INDEX(j, span);
        }
        while (hi - lo > kWave) {  // sub-ranges of more than 64 children (blocks over 262,144): 64-ary search
            const int32_t stride = (hi - lo + kWave - 1) / kWave;
            const int32_t j = lo + lane * stride;
            bool le = false;
            if (j < hi) le = ntok[cb.beg + j] <= t;
            const uint64_t bl = __ballot(le);
            if (!bl) return false;
            lo = lo + (__popcll(bl) - 1) * stride;
            hi = min(lo + stride, hi);
        }
        const int32_t j = lo + lane;
        bool eq = false;
        if (j < hi) eq = ntok[cb.beg + j] == t;
        const uint64_t be = __ballot(eq);
        if (be) idx = lo + (int32_t)(__ffsll((unsigned long long)be) - 1);
    }
    if (idx < 0) return false;
    const Node r = nodes[cb.beg + idx];  // wave-uniform address: a scalar load
    c.id = cb.beg + idx;
    c.lab_off = (int32_t)r.lab_off;
    c.lab_len = r.lab_len;
    c.ct_beg = r.ct_beg;
    c.ct_cnt = r.ct_cnt;
    c.mask0 = r.mask0;
    return true;
}

// Peer selection (the argmax of Algorithm 1, with the push-back and failover
// rules of Sections "Hot specialist push-back" and "In-flight forwarded
// request failure").  Candidates are ordered by larger match, then, when
// prefer_local is set, the local peer, then the lower id; best is the first
// eligible candidate and second the next (-1 when there is none).  The local
// peer is always eligible.  Plain routing is the case "every peer eligible,
// no local peer, no second".
struct Select {
    const uint64_t *eligible;  // ceil(P / 64) words, bit p % 64 of word p / 64; nullptr: every peer
    int32_t local;             // -1: none
    int32_t prefer_local;
    int32_t *second;           // nullptr: not wanted
};

// Order key of a candidate: larger is earlier; 0 for peers that are not
// candidates (every real key is above 2^32 - 1026).
__device__ __forceinline__ uint64_t select_key(int32_t m, int32_t p, const Select &sel) {
    const uint32_t tie = (sel.prefer_local && p == sel.local) ? 0u : (uint32_t)p + 1u;
    return ((uint64_t)(uint32_t)m << 32) | (uint64_t)(0xFFFFFFFFu - tie);
}

__device__ __forceinline__ int32_t select_decode(uint64_t key, const Select &sel) {
    if (key == 0) return -1;
    const uint32_t tie = 0xFFFFFFFFu - (uint32_t)key;
    return tie == 0 ? sel.local : (int32_t)(tie - 1u);
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint64_t o = __shfl_xor(v, off);
        v = o > v ? o : v;
    }
    return v;
}

// elig: the eligibility words, loaded by the caller (all ones for every peer).
template <int W>
__device__ __forceinline__ int32_t select_peers(const int32_t (&m)[W], int32_t P, int lane, const Select &sel,
                                                const uint64_t (&elig)[W], bool want_second, int32_t &second) {
    uint64_t key[W];
#pragma unroll
    for (int w = 0; w < W; w++) {
        const int p = lane + 64 * w;
        const bool ok = p < P && (((elig[w] >> lane) & 1ull) || p == sel.local);
        key[w] = ok ? select_key(m[w], p, sel) : 0ull;
    }
    uint64_t k1 = 0;
#pragma unroll
    for (int w = 0; w < W; w++) k1 = key[w] > k1 ? key[w] : k1;
    k1 = wave_max_u64(k1);
    second = -1;
    if (want_second) {
        uint64_t k2 = 0;
#pragma unroll
        for (int w = 0; w < W; w++) k2 = (key[w] != k1 && key[w] > k2) ? key[w] : k2;
        second = select_decode(wave_max_u64(k2), sel);
    }
    return select_decode(k1, sel);
}

// SEL = false: plain routing (every peer eligible, ties to the lowest id, no
// second pick); the selection options are compiled out.  LT: the label
// pool's token type (int32_t, or uint16_t for the 16-bit copy); HB (with
// uint16_t): bit 16 of every label token comes from the bit plane hib
// (17-bit labels).  WV: vectors of the first-level window.
template <int W, bool SEL, typename LT, bool HB = false, int WV = kWinVectors>
__global__ __launch_bounds__(kWave *kRouteWavesPerBlock)
__attribute__((amdgpu_waves_per_eu(PR_ROUTE_WAVES_PER_EU))) void route_kernel(
    const Node *__restrict__ nodes, const int32_t *__restrict__ ntok, const int32_t *__restrict__ nsep,
    const uint64_t *__restrict__ mext, const LT *__restrict__ pool, const uint32_t *__restrict__ hib,
    const int32_t *__restrict__ qtok, int64_t num_tokens,
    const int64_t *__restrict__ qoff, int64_t nq, int32_t P, const Select sel_in, int32_t *__restrict__ match_len,
    int32_t *__restrict__ chosen, const int32_t *__restrict__ order) {
    const Select sel = SEL ? sel_in : Select{nullptr, -1, 0, nullptr};
    const int lane = (int)(threadIdx.x & (kWave - 1));
    const int64_t slot = (int64_t)blockIdx.x * kRouteWavesPerBlock + uniform((int32_t)(threadIdx.x / kWave));
    if (slot >= nq) return;
    // order (optional) is a permutation of the queries: the dispatcher starts
    // slots in index order, so slot i serves query order[i]
    const int64_t q = order ? (int64_t)order[slot] : slot;
    int32_t *row = match_len + q * (int64_t)P;
    // The offsets and the root's record are loaded together, and a query with
    // bad offsets runs as an empty one (its row is written as -1 at the end),
    // so that no branch on the offsets sits between those loads and the
    // walk's first loads.
    int64_t qb0 = qoff[q], qe0 = qoff[q + 1];
    const Node root = nodes[0];
    int32_t root_beg = root.ct_beg, root_cnt = root.ct_cnt;
    // both loads are issued before anything waits on either (the compiler
    // would otherwise sink the offsets' load below the root's branches)
    asm volatile("" : "+s"(qb0), "+s"(qe0), "+s"(root_beg), "+s"(root_cnt));
    const bool bad = qb0 < 0 || qe0 < qb0 || qe0 > num_tokens || qe0 - qb0 > (int64_t)INT32_MAX;
    const int64_t qb = bad ? 0 : qb0;
    const int64_t qlen = bad ? 0 : qe0 - qb0;
    const int32_t *qs = qtok + qb;
    // the eligibility words are read now and used after the walk, so their
    // load is not one more round trip at the end
    uint64_t elig[W];
#pragma unroll
    for (int w = 0; w < W; w++) elig[w] = (SEL && sel.eligible) ? sel.eligible[w] : ~0ull;

    int32_t m[W];
    uint64_t alive[W];
#pragma unroll
    for (int w = 0; w < W; w++) {
        m[w] = 0;
        const int rem = P - 64 * w;
        alive[w] = rem >= 64 ? ~0ull : (rem > 0 ? ((1ull << rem) - 1ull) : 0ull);
    }

    int64_t d = 0;
    // The root's child block and, when the root has a single child (every
    // stored sequence starts with the same token, as behind a shared system
    // prompt), that child's record: the first level then issues its batch of
    // loads without waiting for the query's first token or a record load.
    ChildBlock cb;
    load_block(cb, ntok, nsep, root_beg, root_cnt, lane);
    const bool single = root_cnt == 1;
    const int32_t c0_id = single ? root_beg : 0;  // node 0 always exists
    const Node r0 = nodes[c0_id];
    const Child c0{c0_id, (int32_t)r0.lab_off, r0.lab_len, r0.ct_beg, r0.ct_cnt, r0.mask0};
    const int32_t c0_tok = r0.tok;
#if PR_FIRST_WINDOW
    // the query's first token comes with the window (lane 0 of its first
    // vector), read where the first level needs it
    int32_t t = 0;
#else
    int32_t t = qlen > 0 ? qs[0] : 0;
#endif
    // One tree level; returns whether the walk goes on.  The first level is a
    // separate instance (FIRST), so that the window's registers die after it.
    // With `known` the level's child is the root's single child c0, taken on
    // the assumption that the query starts with its first token; the check
    // waits until the level's loads are issued.
    auto level = [&](auto first_tag, const auto &win, auto known_tag) __attribute__((always_inline)) -> bool {
        constexpr bool FIRST = decltype(first_tag)::value;
        constexpr bool KNOWN = FIRST && decltype(known_tag)::value;
        Child c;
        if constexpr (KNOWN) {
            c = c0;
        } else {
            if constexpr (FIRST && PR_FIRST_WINDOW) t = uniform(win[0]);
            if (!locate(cb, t, nodes, ntok, nsep, lane, c)) return false;
        }
        if (c.lab_len <= 0) return false;  // only the root has an empty label
        // one batch of loads per level: next token, ext mask words, the next
        // child block (used if the label matches in full) and the label compare
        const int64_t end = d + c.lab_len;
        const int32_t tnext = end < qlen ? qs[end] : 0;
        uint64_t mx[W];
        mx[0] = c.mask0;
#pragma unroll
        for (int w = 1; w < W; w++) mx[w] = mext[(int64_t)c.id * (W - 1) + (w - 1)];
        load_block(cb, ntok, nsep, c.ct_beg, c.ct_cnt, lane);
        const int64_t n = min((int64_t)c.lab_len, qlen - d);
        const LabelSrc<LT, HB> lab{pool + (uint32_t)c.lab_off, hib, (uint32_t)c.lab_off};
        int64_t l;
        if constexpr (FIRST)
            l = wave_lcp_first<LT, HB, WV>(lab, qs, n, win, lane);
        else
            l = wave_lcp<LT, HB>(lab, qs + d, n, 0, (int64_t)kWave * kLcpFirstVectors, lane);
        if constexpr (KNOWN) {
            if constexpr (PR_FIRST_WINDOW) t = uniform(win[0]);
            if (t != c0_tok) return false;  // no child starts with the query's first token
        }
        bool any = false;
#pragma unroll
        for (int w = 0; w < W; w++) {
            const uint64_t nm = alive[w] & mx[w];
            if (((alive[w] & ~nm) >> lane) & 1ull) m[w] = (int32_t)d;
            alive[w] = nm;
            any |= nm != 0ull;
        }
        if (!any) return false;  // no peer holds this edge (left behind by a replaced snapshot)
        d += l;
        if (l < c.lab_len) return false;
        t = tnext;
        return d < qlen;
    };
    struct NoWindow {};
#if PR_FIRST_WINDOW
    int32_t win[WV];
    load_window<WV>(win, qs, (int32_t)min(qlen, (int64_t)kWave * WV), lane);
    bool more = false;
    if (qlen > 0) more = single ? level(std::true_type{}, win, std::true_type{})
                                : level(std::true_type{}, win, std::false_type{});
#else
    bool more = qlen > 0 && level(std::false_type{}, NoWindow{}, std::false_type{});
#endif
    while (more) more = level(std::false_type{}, NoWindow{}, std::false_type{});

    if (bad) {
        if (match_len)
            for (int p = lane; p < P; p += kWave) row[p] = -1;
        if (lane == 0) {
            chosen[q] = -1;
            if (sel.second) sel.second[q] = -1;
        }
        return;
    }
    // peers still holding the walked path matched all of it
#pragma unroll
    for (int w = 0; w < W; w++)
        if ((alive[w] >> lane) & 1ull) m[w] = (int32_t)d;

    if (match_len) store_row<W>(row, m, P, lane);
    int32_t second;
    const int32_t best = select_peers<W>(m, P, lane, sel, elig, sel.second != nullptr, second);
    if (lane == 0) {
        chosen[q] = best;  // 4 bytes a query: plain stores, which the L2 merges into whole lines
        if (sel.second) sel.second[q] = second;
    }
}

// Longest-first order of a batch, a counting sort in two launches of a few
// workgroups: every query gets a length bucket (unit tokens wide, the last
// one open-ended), and order lists the queries by bucket, longest bucket
// first.  Within a bucket the order is fixed by the layout below, so it is
// deterministic.  Offsets are not checked here (a bad pair lands in some
// bucket); the route kernel checks every query's offsets itself.
constexpr int kOrderThreads = 1024;
constexpr int kOrderWaves = kOrderThreads / kWave;
constexpr int kOrderPerThread = 4;
constexpr int kOrderChunk = kOrderThreads * kOrderPerThread;  // queries per workgroup
constexpr int kOrderBuckets = 16;
constexpr int kOrderMaxBlocks = 16;
constexpr int32_t kOrderMaxQueries = kOrderChunk * kOrderMaxBlocks;  // 65,536

// Query i of thread t in workgroup b: base + i * kOrderThreads + t.
__device__ __forceinline__ int32_t order_query(int b, int i, int t) {
    return b * kOrderChunk + i * kOrderThreads + t;
}

// Launch 1: each query's bucket, and each workgroup's bucket counts.
__global__ __launch_bounds__(kOrderThreads) void route_order_count_kernel(const int64_t *__restrict__ qoff,
                                                                          int32_t nq, uint32_t unit,
                                                                          uint8_t *__restrict__ bkt,
                                                                          int32_t *__restrict__ blockcnt) {
    __shared__ int32_t cnt[kOrderWaves][kOrderBuckets];
    const int t = (int)threadIdx.x, lane = t & (kWave - 1), wv = t / kWave, b = (int)blockIdx.x;
    int64_t lo[kOrderPerThread], hi[kOrderPerThread];
#pragma unroll
    for (int i = 0; i < kOrderPerThread; i++) {
        const int32_t q = min(order_query(b, i, t), nq - 1);
        lo[i] = qoff[q];
        hi[i] = qoff[q + 1];
    }
    int32_t c[kOrderBuckets];
#pragma unroll
    for (int k = 0; k < kOrderBuckets; k++) c[k] = 0;
#pragma unroll
    for (int i = 0; i < kOrderPerThread; i++) {
        const int32_t q = order_query(b, i, t);
        int bk = -1;
        if (q < nq) {
            const int64_t len = hi[i] - lo[i];
            const uint32_t l32 = len <= 0 ? 0u : (len > (int64_t)INT32_MAX ? (uint32_t)INT32_MAX : (uint32_t)len);
            const uint32_t x = l32 / unit;
            bk = (int)(x < kOrderBuckets - 1 ? x : kOrderBuckets - 1);
            bkt[q] = (uint8_t)bk;
        }
#pragma unroll
        for (int k = 0; k < kOrderBuckets; k++) c[k] += __popcll(__ballot(bk == k));
    }
    if (lane == 0)
#pragma unroll
        for (int k = 0; k < kOrderBuckets; k++) cnt[wv][k] = c[k];
    __syncthreads();
    if (t < kOrderBuckets) {
        int32_t sum = 0;
        for (int w = 0; w < kOrderWaves; w++) sum += cnt[w][t];
        blockcnt[b * kOrderBuckets + t] = sum;
    }
}

// Launch 2: position of every query.  Bucket k of workgroup b starts after
// every longer bucket and after bucket k of the earlier workgroups; inside
// the workgroup, wave by wave, each wave in query order i then lane.
__global__ __launch_bounds__(kOrderThreads) void route_order_scatter_kernel(const uint8_t *__restrict__ bkt,
                                                                            int32_t nq,
                                                                            const int32_t *__restrict__ blockcnt,
                                                                            int32_t *__restrict__ order) {
    __shared__ int32_t cnt[kOrderWaves][kOrderBuckets];
    __shared__ int32_t bc[kOrderMaxBlocks * kOrderBuckets];
    const int t = (int)threadIdx.x, lane = t & (kWave - 1), wv = t / kWave, b = (int)blockIdx.x;
    const int nb = (int)gridDim.x;
    if (t < nb * kOrderBuckets) bc[t] = blockcnt[t];  // every workgroup's counts, one load per thread
    int bk[kOrderPerThread];
#pragma unroll
    for (int i = 0; i < kOrderPerThread; i++) {
        const int32_t q = order_query(b, i, t);
        bk[i] = q < nq ? (int)bkt[q] : -1;
    }
    int32_t c[kOrderBuckets];
#pragma unroll
    for (int k = 0; k < kOrderBuckets; k++) c[k] = 0;
#pragma unroll
    for (int i = 0; i < kOrderPerThread; i++)
#pragma unroll
        for (int k = 0; k < kOrderBuckets; k++) c[k] += __popcll(__ballot(bk[i] == k));
    if (lane == 0)
#pragma unroll
        for (int k = 0; k < kOrderBuckets; k++) cnt[wv][k] = c[k];
    __syncthreads();
    // bucket totals over all workgroups, and bucket t's count in earlier ones
    __shared__ int32_t tot[kOrderBuckets], pre[kOrderBuckets];
    if (t < kOrderBuckets) {
        int32_t all = 0, earlier = 0;
        for (int j = 0; j < nb; j++) {
            const int32_t v = bc[j * kOrderBuckets + t];
            all += v;
            earlier += j < b ? v : 0;
        }
        tot[t] = all;
        pre[t] = earlier;
    }
    __syncthreads();
    if (t < kOrderBuckets) {
        // this workgroup's start in bucket t, then the waves' starts inside it
        int32_t before = pre[t];
        for (int k = t + 1; k < kOrderBuckets; k++) before += tot[k];  // longer buckets come first
        int32_t run = before;
        for (int w = 0; w < kOrderWaves; w++) {
            const int32_t v = cnt[w][t];
            cnt[w][t] = run;
            run += v;
        }
    }
    __syncthreads();
    int32_t start[kOrderBuckets];
#pragma unroll
    for (int k = 0; k < kOrderBuckets; k++) start[k] = cnt[wv][k];
    const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
    for (int i = 0; i < kOrderPerThread; i++) {
        const int32_t q = order_query(b, i, t);
#pragma unroll
        for (int k = 0; k < kOrderBuckets; k++) {
            const uint64_t m = __ballot(bk[i] == k);
            if (bk[i] == k) order[start[k] + __popcll(m & below)] = q;
            start[k] += __popcll(m);
        }
    }
}

}  // namespace pr

#endif
