// forest_layout.h -- the device layout of the union radix forest.
//
// All peers' trees are stored as ONE compressed trie over the union of their
// sequences, and every node carries a bitmask of the peers whose tree holds
// the node's whole path.  A node exists at every branch point of the union and
// wherever some peer's sequence ends, so a peer either holds all of an edge or
// none of it; masks shrink monotonically from the root outwards.  A query is
// walked once instead of once per peer: peer p's match length is the depth at
// which p leaves the masks of the walked path (or the final depth if it never
// leaves).  The paper keeps one radix tree per node (System Design); the union
// with masks answers the same PrefixMatch for all of them in one walk.
//
// Arrays (device resident):
//   nodes[n]  32-byte Node records.  The children of a node are one contiguous
//             block nodes[ct_beg .. ct_beg + ct_cnt), sorted by first label
//             token (signed int32 order), so the position of a child in the
//             first-token array is its id.  Node 0 is the root (empty label).
//   ntok[n]   first label token of node n (= nodes[n].tok), dense, for
//             scanning child blocks with coalesced 4-byte loads.
//   nsep[n]   separators of wide child blocks: for a block [b, b + cnt) with
//             cnt > 64, nsep[b + k] = ntok[b + PR_SEP_INDEX(k, cnt)] for
//             k < 64 (ascending).  A wave loads the 64 separators (two cache
//             lines), a ballot picks the sub-range that can hold a token, and
//             one more load of at most ceil(cnt / 64) first tokens settles it.
//             Blocks of at least kSep2Min (4,160) children also keep a second
//             level: sub-range k (first tokens [lo_k, hi_k), lo_k =
//             PR_SEP_INDEX(k, cnt), hi_k = PR_SEP_HI(k, cnt)) has its own 64
//             separators, contiguous, at nsep[b + 64 + 64 k + j] =
//             ntok[b + lo_k + PR_SEP_INDEX(j, hi_k - lo_k)]; they sit in slots
//             of the block that the first level leaves unused, and the search
//             of a sub-range reads two cache lines instead of gathering one
//             token from each of 64 lines.  Other entries are unused.
//   mext[n*(W-1) + w-1]  peer-mask words 1..W-1 of node n (W > 1 only);
//             word 0 lives in the record.
//   pool[t]   int32 label tokens; node n's label is pool[lab_off .. +lab_len).
//   pool16[t] the low 16 bits of pool[t], kept while every label token lies in
//             [0, 131071]; routes read labels from it (half the bytes).
//   hib[t/32] bit t % 32 is bit 16 of pool[t] (kept with pool16); routes read
//             it once some label token is 65536 or more (17-bit labels: one
//             32-bit word covers the high bits of 32 label tokens).
#ifndef PR_FOREST_LAYOUT_H
#define PR_FOREST_LAYOUT_H

#include <stdint.h>

namespace pr {

struct alignas(32) Node {
    int32_t tok;       // first token of the edge label (0 for the root)
    uint32_t lab_off;  // first token of the edge label in pool
    int32_t lab_len;   // label length; >= 1 except for the root
    int32_t ct_beg;    // first child node id
    int32_t ct_cnt;    // number of children
    int32_t aux;       // scratch for tree updates (0 at rest)
    uint64_t mask0;    // peers 0..63 holding this node's path
};

static_assert(sizeof(Node) == 32, "Node is one 32-byte record");

// Child blocks with more than this many children carry separators.
constexpr int kSepCount = 64;

// Position in a wide block of cnt children of its k-th separator (k < 64).
#define PR_SEP_INDEX(k, cnt) ((int32_t)(((int64_t)(k) * (int64_t)(cnt)) / 64))
// End of sub-range k (the next separator's position, or cnt after the last).
#define PR_SEP_HI(k, cnt) ((k) == kSepCount - 1 ? (int32_t)(cnt) : PR_SEP_INDEX((k) + 1, cnt))

// Child blocks of at least this many children carry second-level separators
// (the first level's 64 slots plus 64 per sub-range fit in the block).
constexpr int32_t kSep2Min = kSepCount + kSepCount * kSepCount;

// Mask words per node for a peer count (template instances exist for these).
inline int mask_words_for(int num_peers) {
    int w = (num_peers + 63) / 64;
    int r = 1;
    while (r < w) r <<= 1;
    return r;  // 1, 2, 4, 8 or 16
}

}  // namespace pr

#endif
