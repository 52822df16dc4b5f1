// forest_host.cpp -- build the union radix forest of all peers on the host and
// flatten it into the device layout of forest_layout.h.
//
// Construction inserts every (peer, sequence) pair into one compressed trie:
// walk the sequence from the root; on reaching a node without a child for the
// next token, hang the rest of the sequence below it as a new leaf edge; on a
// mismatch or sequence end inside an edge, split the edge there.  Every node on
// the walked path gets the peer's bit.  A node then exists at every branch
// point and every sequence end, so a peer's bit is uniform along each edge.
//
// Afterwards chains are compressed: a node with a single child whose peer mask
// equals its own absorbs that child, since no match length can end between
// them.  The flattened image gives the children of every node one contiguous
// block of ids, sorted by first token.
#include "forest_host.h"

#include <algorithm>
#include <cstddef>
#include <cstring>
#include <limits>
#include <new>

namespace pr {

namespace {

struct BNode {
    const int32_t *lab = nullptr;  // label tokens (points into a stored sequence)
    int64_t len = 0;
    std::vector<int32_t> kids;     // child BNode ids, sorted by first label token
};

class Builder {
   public:
    explicit Builder(int W) : W_(W) {
        nodes_.emplace_back();  // root
        masks_.assign((size_t)W_, 0ull);
    }

    void insert(int peer, const int32_t *s, int64_t n) {
        int32_t x = 0;
        int64_t i = 0;
        set_bit(0, peer);
        while (i < n) {
            const int32_t t = s[i];
            std::vector<int32_t> &K = nodes_[x].kids;
            auto it = std::lower_bound(K.begin(), K.end(), t, [&](int32_t k, int32_t v) {
                return nodes_[k].lab[0] < v;
            });
            const size_t pos = (size_t)(it - K.begin());
            if (it == K.end() || nodes_[*it].lab[0] != t) {
                const int32_t c = new_node(s + i, n - i);
                nodes_[c].kids.clear();
                set_bit(c, peer);
                std::vector<int32_t> &K2 = nodes_[x].kids;  // new_node may reallocate
                K2.insert(K2.begin() + (std::ptrdiff_t)pos, c);
                return;
            }
            int32_t c = *it;
            const int64_t l = lcp(nodes_[c].lab, nodes_[c].len, s + i, n - i);
            if (l < nodes_[c].len) {  // split c's edge after l tokens
                const int32_t mid = new_node(nodes_[c].lab, l);
                for (int w = 0; w < W_; w++) masks_[(size_t)mid * W_ + w] = masks_[(size_t)c * W_ + w];
                nodes_[mid].kids.assign(1, c);
                nodes_[c].lab += l;
                nodes_[c].len -= l;
                nodes_[x].kids[pos] = mid;
                c = mid;
            }
            set_bit(c, peer);
            x = c;
            i += l;
        }
    }

    void compress() {
        std::vector<int32_t> stack{0};
        while (!stack.empty()) {
            const int32_t x = stack.back();
            stack.pop_back();
            if (x != 0) {
                while (nodes_[x].kids.size() == 1) {
                    const int32_t c = nodes_[x].kids[0];
                    if (!same_mask(x, c)) break;
                    // c's label is preceded by x's label in the sequence it was cut from
                    nodes_[x].lab = nodes_[c].lab - nodes_[x].len;
                    nodes_[x].len += nodes_[c].len;
                    nodes_[x].kids.swap(nodes_[c].kids);
                    nodes_[c].kids.clear();
                }
            }
            for (int32_t k : nodes_[x].kids) stack.push_back(k);
        }
    }

    bool flatten(HostImage *out, std::string *err) {
        // Ids: the root is 0; when a node is visited, its children receive one
        // contiguous block of ids in first-token order; children are then
        // visited depth first.  Labels are laid out in id order.
        const size_t n = nodes_.size();
        if (n > (size_t)std::numeric_limits<int32_t>::max()) {
            *err = "too many nodes";
            return false;
        }
        // nodes absorbed by compression are unreachable and get no id
        std::vector<int32_t> order;  // order[id] = builder node
        order.reserve(n);
        order.push_back(0);
        std::vector<int32_t> stack{0};
        std::vector<int32_t> first_child_id(n, -1);
        while (!stack.empty()) {
            const int32_t x = stack.back();
            stack.pop_back();
            const auto &K = nodes_[x].kids;
            first_child_id[x] = (int32_t)order.size();
            for (int32_t k : K) order.push_back(k);
            for (size_t j = K.size(); j-- > 0;) stack.push_back(K[j]);
        }
        uint64_t pool_len = 0;
        for (int32_t x : order) pool_len += (uint64_t)nodes_[x].len;
        if (pool_len > (uint64_t)std::numeric_limits<uint32_t>::max()) {
            *err = "label pool exceeds 2^32 tokens";
            return false;
        }
        const size_t m = order.size();
        out->W = W_;
        out->nodes.assign(m, Node{});
        out->ntok.assign(m, 0);
        out->nsep.assign(m, 0);
        out->mext.assign(m * (size_t)(W_ - 1), 0ull);
        out->pool.resize((size_t)pool_len);
        uint64_t po = 0;
        for (size_t id = 0; id < m; id++) {
            const int32_t x = order[id];
            const BNode &b = nodes_[x];
            Node &nd = out->nodes[id];
            nd.tok = b.len ? b.lab[0] : 0;
            nd.lab_off = (uint32_t)po;
            nd.lab_len = (int32_t)b.len;
            if (b.len) std::memcpy(out->pool.data() + po, b.lab, (size_t)b.len * sizeof(int32_t));
            po += (uint64_t)b.len;
            nd.ct_beg = b.kids.empty() ? 0 : first_child_id[x];
            nd.ct_cnt = (int32_t)b.kids.size();
            nd.aux = 0;
            nd.mask0 = masks_[(size_t)x * W_];
            out->ntok[id] = nd.tok;
            for (int w = 1; w < W_; w++)
                out->mext[id * (size_t)(W_ - 1) + (w - 1)] = masks_[(size_t)x * W_ + w];
        }
        for (size_t id = 0; id < m; id++) {  // separators of wide child blocks
            const Node &nd = out->nodes[id];
            if (nd.ct_cnt <= kSepCount) continue;
            for (int k = 0; k < kSepCount; k++)
                out->nsep[(size_t)nd.ct_beg + k] = out->ntok[(size_t)nd.ct_beg + PR_SEP_INDEX(k, nd.ct_cnt)];
            if (nd.ct_cnt < kSep2Min) continue;
            for (int k = 0; k < kSepCount; k++) {  // second level, per sub-range
                const int32_t lo = PR_SEP_INDEX(k, nd.ct_cnt), span = PR_SEP_HI(k, nd.ct_cnt) - lo;
                for (int j = 0; j < kSepCount; j++)
                    out->nsep[(size_t)nd.ct_beg + kSepCount + (size_t)kSepCount * k + j] =
                        out->ntok[(size_t)nd.ct_beg + lo + PR_SEP_INDEX(j, span)];
            }
        }
        return true;
    }

   private:
    static int64_t lcp(const int32_t *a, int64_t na, const int32_t *b, int64_t nb) {
        const int64_t n = na < nb ? na : nb;
        int64_t i = 0;
        while (i < n && a[i] == b[i]) i++;
        return i;
    }

    int32_t new_node(const int32_t *lab, int64_t len) {
        nodes_.emplace_back();
        nodes_.back().lab = lab;
        nodes_.back().len = len;
        masks_.resize(masks_.size() + (size_t)W_, 0ull);
        return (int32_t)(nodes_.size() - 1);
    }

    void set_bit(int32_t x, int peer) { masks_[(size_t)x * W_ + (peer >> 6)] |= 1ull << (peer & 63); }

    bool same_mask(int32_t a, int32_t b) const {
        for (int w = 0; w < W_; w++)
            if (masks_[(size_t)a * W_ + w] != masks_[(size_t)b * W_ + w]) return false;
        return true;
    }

    int W_;
    std::vector<BNode> nodes_;
    std::vector<uint64_t> masks_;
};

}  // namespace

bool build_union_image(const std::vector<PeerSeqs> &sets, int W, HostImage *out, std::string *err) {
    try {
        Builder b(W);
        for (size_t p = 0; p < sets.size(); p++) {
            const PeerSeqs &S = sets[p];
            for (int64_t i = 0; i < S.count(); i++) {
                const int64_t o = S.offsets[(size_t)i];
                b.insert((int)p, S.tokens.data() + o, S.offsets[(size_t)i + 1] - o);
            }
        }
        b.compress();
        return b.flatten(out, err);
    } catch (const std::bad_alloc &) {
        *err = "host allocation failed while building the forest";
        return false;
    }
}

}  // namespace pr
