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
//             token (signed int32 order), so a wave that loads the block finds
//             the child for a token with one ballot and already holds the
//             child's record.  Node 0 is the root (empty label).
//   ntok[n]   first label token of node n (= nodes[n].tok), dense, for
//             scanning wide child blocks with coalesced 4-byte loads.
//   mext[n*(W-1) + w-1]  peer-mask words 1..W-1 of node n (W > 1 only);
//             word 0 lives in the record.
//   pool[t]   int32 label tokens; node n's label is pool[lab_off .. +lab_len).
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

// Mask words per node for a peer count (template instances exist for these).
inline int mask_words_for(int num_peers) {
    int w = (num_peers + 63) / 64;
    int r = 1;
    while (r < w) r <<= 1;
    return r;  // 1, 2, 4, 8 or 16
}

}  // namespace pr

#endif
