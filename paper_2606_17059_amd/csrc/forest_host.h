// forest_host.h -- host-side construction of the union radix forest image.
#ifndef PR_FOREST_HOST_H
#define PR_FOREST_HOST_H

#include <stdint.h>

#include <string>
#include <vector>

#include "forest_layout.h"

namespace pr {

// One peer's sequence set in CSR form (offsets.size() == count + 1).
struct PeerSeqs {
    std::vector<int32_t> tokens;
    std::vector<int64_t> offsets{0};
    int64_t count() const { return (int64_t)offsets.size() - 1; }
};

// The flattened layout, host side (see forest_layout.h).
struct HostImage {
    int W = 1;
    std::vector<Node> nodes;
    std::vector<int32_t> ntok;
    std::vector<int32_t> nsep;   // separators of wide child blocks
    std::vector<uint64_t> mext;  // words 1..W-1 per node
    std::vector<int32_t> pool;
};

// Build the union image of every peer's set.  W is the mask-word count
// (>= ceil(P/64)).  Returns false with *err set on overflow or allocation
// failure.
bool build_union_image(const std::vector<PeerSeqs> &sets, int W, HostImage *out, std::string *err);

}  // namespace pr

#endif
