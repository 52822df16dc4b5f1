// forest_layout.h -- the device layout of the union radix forest.
//
// All peers' trees are stored as ONE compressed trie over the union of their
// sequences, and every node carries a bitmask of the peers whose tree holds
// the node's whole path.  A node exists at every branch point of the union and
// wherever some peer's sequence ends, so a peer either holds all of an edge or
// none of it; masks shrink monotonically from the root outwards.  A query is
// walked once per batch item instead of once per peer: peer p's match length
// is the depth at which p leaves the mask of the walked path (or the final
// depth if it never leaves).  The paper keeps one radix tree per node (System
// Design); the union with masks answers the same PrefixMatch for all of them.
//
// Arrays (structure of arrays, device resident):
//   nodes[n]       Node: edge label span in the pool + child-table span.
//   masks[n*W + w] 64-bit peer-mask word w of node n (W = mask words).
//   ctab[k]        ChildSlot: (first label token, child node id); the slots of
//                  one node are contiguous and sorted by first token (signed).
//   pool[t]        int32 label tokens.
// Node 0 is the root (empty label).
#ifndef PR_FOREST_LAYOUT_H
#define PR_FOREST_LAYOUT_H

#include <stdint.h>

namespace pr {

struct Node {
    uint32_t lab_off;  // first token of the edge label in pool
    int32_t lab_len;   // label length; >= 1 except for the root
    int32_t ct_beg;    // first child slot
    int32_t ct_cnt;    // number of child slots
};

struct ChildSlot {
    int32_t tok;   // first token of the child's label
    int32_t node;  // child node id
};

static_assert(sizeof(Node) == 16, "Node is one 16-byte record");
static_assert(sizeof(ChildSlot) == 8, "ChildSlot is 8 bytes");

// Mask words per node for a peer count (template instances exist for these).
inline int mask_words_for(int num_peers) {
    int w = (num_peers + 63) / 64;
    int r = 1;
    while (r < w) r <<= 1;
    return r;  // 1, 2, 4, 8 or 16
}

}  // namespace pr

#endif
