/*
 * prefix_router.h -- C ABI of the MI355X (gfx950) prefix-cache-aware router.
 *
 * The library keeps, on one GPU, a node's view of every peer's prefix cache:
 * its own exact radix tree plus one read-only estimate per other peer
 * (paper, System Design).  It answers getBestNode for a whole batch of
 * requests at once (Algorithm 1, the argmax of PrefixMatch over all N trees),
 * and applies the tree updates the paper names: full-snapshot replacement
 * (sendTrie received; Section "Trie-broadcast loss") and per-request inserts
 * (updateTrie / updateTrieEstimate).
 *
 * Conventions shared by every call
 *   - Status: every call returns pr_status; 0 is success, negative is an error.
 *     Nothing is thrown across the ABI.  pr_last_error() gives a message for
 *     the calling thread's last failure.
 *   - Peers are 0 .. num_peers-1; peer p's tree is "slot p".  Which slot is
 *     the local node's own tree is the caller's business: routing treats all
 *     slots alike (the argmax runs over every tree, the node's own included).
 *   - Tokens are int32; every int32 value is a legal token.  Sequence batches
 *     are CSR: sequence i is tokens[offsets[i] .. offsets[i+1]), offsets are
 *     int64, offsets[0] == 0 and non-decreasing.
 *   - Match semantics: match_len[q][p] is the length of the longest prefix of
 *     query q that is also a prefix of some sequence inserted into peer p's
 *     tree (0 for an empty tree or query).  chosen[q] is the lowest peer id
 *     whose match length is the largest (so an all-zero row chooses peer 0).
 *   - Single writer: calls on one forest must be serialised by the caller
 *     (each tree has one writer, paper Section 1).  pr_route only reads the
 *     forest; calls that update it (merge, loads, touch, eviction, compaction)
 *     change the device image in place, so a route still queued on another
 *     stream must be ordered before them (the same stream, or an event).  When
 *     they move the image (growth, rebuild) they wait for the whole device
 *     before freeing the old arrays.
 *   - Device calls (pr_merge, pr_route) take device pointers and a HIP stream
 *     (NULL = the legacy default stream) and are ordered on that stream after
 *     the work already queued there.  pr_route returns without waiting for the
 *     GPU: its inputs must stay valid, and its outputs untouched, until the
 *     stream has passed the call.  pr_merge returns when the merge is complete
 *     (it reads small counters back between its insert rounds).
 *   - A forest lives on the HIP device that is current when it first touches
 *     the GPU; later calls switch to that device for their duration.
 */
#ifndef PREFIX_ROUTER_H
#define PREFIX_ROUTER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t pr_status;

#define PR_OK 0
#define PR_EINVAL (-1)  /* bad argument; the forest is unchanged, no output is written */
#define PR_ENOMEM (-2)  /* host or device allocation failed; the forest is unchanged unless
                           the call's description says otherwise */
#define PR_EDEVICE (-3) /* a HIP call failed; destroy the forest */
#define PR_ESTATE (-4)  /* call not valid in the forest's current state */

#define PR_MAX_PEERS 1024

typedef struct pr_forest pr_forest;

/* ABI version of this header (incremented on incompatible changes). */
#define PR_ABI_VERSION 7

/* PR_ABI_VERSION of the header the library was built with; a client built
 * against another version must not call the library. */
int32_t pr_abi_version(void);

/* Message describing the calling thread's last failed call ("" if none). */
const char *pr_last_error(void);

/*
 * Create an empty forest of num_peers trees (1 <= num_peers <= PR_MAX_PEERS):
 * one node's view of the network (paper, System Design: every node keeps a
 * radix tree of its own cache and one estimate of each other node's).
 * Every tree starts empty.  No GPU work happens here.
 * Which tree is the node's own needs no argument here: routing treats every
 * tree alike (Algorithm 1 takes the argmax over all N trees), and the tree
 * whose LRU state is kept (Algorithm 1's EvictLRUTrie) is chosen later with
 * pr_set_local_peer.  Nor does the layout take a split granularity: edges
 * split at fixed token blocks would change no match length (the match is
 * token-exact), so every tree is a plain path-compressed radix tree.
 * Errors: PR_EINVAL (num_peers out of range, out == NULL), PR_ENOMEM.
 * Ownership: the caller owns *out and releases it with pr_forest_destroy.
 */
pr_status pr_forest_create(int32_t num_peers, pr_forest **out);

/* Release a forest and all its host and device memory (the node leaving the
 * network, or its router restarting: paper, System Design).  NULL is a no-op.
 * Waits for the forest's device to finish outstanding work first. */
void pr_forest_destroy(pr_forest *f);

/*
 * sendTrie, receive side (paper: sendTrie broadcasts the local trie; Section
 * "Trie-broadcast loss": every broadcast is a complete snapshot, so receiving
 * it replaces the estimate, and a duplicated broadcast changes nothing).
 * REPLACES peer's tree by the set of num_seqs sequences given as a HOST CSR
 * batch.  Any merges into that peer since its last snapshot are dropped with
 * the old tree; other peers are untouched.  An empty snapshot (num_seqs == 0)
 * empties the tree, e.g. a peer that crashed and lost its cache.
 * The data is copied before the call returns.  Until the first pr_merge on
 * this forest, the device copy of the forest is rebuilt from the host copies
 * of all snapshots before the next pr_merge or pr_route runs (that call then
 * blocks the host for the rebuild and upload).  Once merges have run, the
 * replacement happens on the device within this call: the peer is removed
 * from every node, then the snapshot is inserted as by pr_merge.
 * Errors: PR_EINVAL (peer out of range, num_seqs < 0, NULL offsets, NULL tokens
 * with a non-empty batch, offsets[0] != 0 or decreasing offsets), PR_ENOMEM,
 * PR_ESTATE (an earlier device update failed), PR_EDEVICE.
 */
pr_status pr_load_snapshot(pr_forest *f, int32_t peer, const int32_t *tokens,
                           const int64_t *offsets, int64_t num_seqs);

/*
 * updateTrie / updateTrieEstimate (paper, System Design; Algorithm 1 inserts a
 * request into the local tree after serving it, or into the estimate of the
 * peer it was forwarded to once that peer acknowledges).
 * Inserts DEVICE sequence i (tokens[offsets[i] .. offsets[i+1]), offsets within
 * [0, num_tokens]) into peer peer_of[i]'s tree, for every i < num_seqs, on the
 * given stream, and returns when the forest holds them.  The result depends
 * only on the set of inserts (order and duplicates do not matter).  Entries
 * with a peer out of range or offsets outside [0, num_tokens] or decreasing
 * are skipped and counted; see pr_forest_check.
 * Errors: PR_EINVAL (NULL pointers with num_seqs > 0, negative counts; nothing
 * is enqueued), PR_ESTATE (an earlier device update failed), PR_ENOMEM (the
 * forest's device capacity could not grow) and PR_EDEVICE (a HIP call failed
 * or an internal invariant check tripped); after PR_ENOMEM or PR_EDEVICE the
 * forest refuses every call but destroy.
 */
pr_status pr_merge(pr_forest *f, const int32_t *peer_of, const int32_t *tokens,
                   int64_t num_tokens, const int64_t *offsets, int64_t num_seqs,
                   void *hip_stream);

/*
 * getBestNode for a batch (paper, System Design; Algorithm 1: the node picks
 * k = argmax over all N trees of PrefixMatch(r, tree_j)).
 * DEVICE inputs: query q is q_tokens[q_offsets[q] .. q_offsets[q+1]), offsets
 * within [0, num_tokens].  DEVICE outputs, caller-allocated:
 *   match_len  int32 [num_queries][num_peers], row-major;
 *   chosen     int32 [num_queries].
 * A query whose offsets are outside [0, num_tokens], decreasing, or span more
 * than INT32_MAX tokens gets match_len -1 in every column and chosen -1.
 * num_queries == 0 is a no-op.  Reads the forest only.
 * Batches of more than 8,192 and at most 65,536 queries averaging at least
 * 4,096 tokens are walked longest first (a length bucketing on the stream
 * before the walk; results are unchanged).  The order lives in a buffer the
 * forest keeps: the first such call, or a larger batch, allocates it (after
 * waiting for the previous user), and such calls on one forest are ordered on
 * the device through an event even when issued on different streams.
 * HIP graph capture: on a capturing stream the call enqueues the route kernel
 * only (no allocation, copy, wait or event), walking the batch in index order
 * (same results); a replay routes what the captured buffers hold at replay
 * time.  Under capture, a forest whose snapshots changed since its last
 * upload (pr_load_snapshot without a route, merge or device call after it)
 * returns PR_ESTATE: route once outside capture first.  The graph holds the
 * addresses of the forest's device arrays: replay it only while the forest
 * lives and pr_forest_info's layout_epoch still has its value at capture
 * (after the arrays move, a replay would read freed memory; capture again).
 * Errors (host side, nothing enqueued): PR_EINVAL (NULL pointers with
 * num_queries > 0, negative counts), PR_ESTATE (see capture above),
 * PR_ENOMEM / PR_EDEVICE (rebuild after a snapshot load failed, or the order
 * buffer could not be allocated).
 */
pr_status pr_route(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens,
                   const int64_t *q_offsets, int64_t num_queries, int32_t *match_len,
                   int32_t *chosen, void *hip_stream);

/*
 * pr_route for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, results and stream behaviour as pr_route, except:
 *   - at most PR_NOALLOC_MAX_QUERIES queries per call (PR_EINVAL beyond);
 *   - the forest must already be on the device: after pr_load_snapshot, run
 *     pr_route (or any other device call) once first, else PR_ESTATE;
 *   - the longest-first order of a batch (see pr_route) is kept in a static
 *     device array of the library, not in a buffer of the forest: about
 *     321 KiB on each GPU the library runs on, held until the process ends.
 *     Every call on one GPU, for any forest, uses that GPU's array, which
 *     keeps the previous call's contents (each call writes every entry it
 *     reads first).  Calls that overlap on one GPU (different streams or host
 *     threads) race on it: order them, e.g. on one stream.
 * The call allocates no host or device memory and enqueues kernel launches
 * only (no copy, wait or event).
 * Errors (host side, nothing enqueued): PR_EINVAL (as pr_route, or more than
 * PR_NOALLOC_MAX_QUERIES queries), PR_ESTATE, PR_EDEVICE.
 */
#define PR_NOALLOC_MAX_QUERIES 65536

pr_status pr_route_noalloc(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens,
                           const int64_t *q_offsets, int64_t num_queries, int32_t *match_len,
                           int32_t *chosen, void *hip_stream);

/*
 * sendTrie, receive side, for a snapshot already in DEVICE memory (for
 * example received by a GPU-direct transfer).  Same semantics as
 * pr_load_snapshot: REPLACES peer's tree by the set of num_seqs sequences
 * tokens[offsets[i] .. offsets[i+1]), offsets within [0, num_tokens].  The
 * replacement runs on the device: the peer is removed from every node, then
 * the sequences are inserted as by pr_merge (a sequence with invalid offsets
 * is skipped and counted for pr_forest_check).  Host-synchronous like
 * pr_merge; the inputs may be reused when the call returns.  Afterwards the
 * forest has no host copy of this peer's snapshot.
 * Errors: PR_EINVAL (peer out of range, negative counts, NULL offsets with
 * num_seqs > 0, NULL tokens with num_tokens > 0), PR_ENOMEM, PR_ESTATE,
 * PR_EDEVICE; after PR_ENOMEM or PR_EDEVICE the forest refuses every call but
 * destroy.
 */
pr_status pr_load_snapshot_device(pr_forest *f, int32_t peer, const int32_t *tokens,
                                  int64_t num_tokens, const int64_t *offsets, int64_t num_seqs,
                                  void *hip_stream);

/*
 * sendTrie, send side (paper, System Design: each node periodically
 * broadcasts its own tree; Section "Trie-broadcast loss": as a complete
 * snapshot).  Writes peer's tree as the set of sequences that rebuilds it:
 * the root paths that end at a node holding the peer none of whose children
 * holds it, i.e. the members of the peer's set that are no proper prefix of
 * another member, each once (empty sequences add nothing and are left out).
 * Loading the result with pr_load_snapshot(_device) gives the same tree.
 * Order: by node id in the device layout (deterministic for a given forest).
 * Outputs:
 *   *num_seqs, *num_tokens   HOST: the export's size, always written;
 *   offsets  DEVICE int64 [num_seqs + 1] (CSR, offsets[0] = 0), capacity
 *            seqs_cap entries;
 *   tokens   DEVICE int32 [num_tokens], capacity tokens_cap.
 * With tokens and offsets both NULL the call only reports the size; with
 * buffers that are too small it returns PR_EINVAL (sizes still written) and
 * writes nothing.  Host-synchronous; reads the forest only.  The size query
 * and the fill each walk the tree.
 * Errors: PR_EINVAL (peer out of range, NULL size outputs, negative or too
 * small capacities), PR_ENOMEM, PR_ESTATE, PR_EDEVICE.
 */
pr_status pr_export_snapshot(pr_forest *f, int32_t peer, int32_t *tokens, int64_t tokens_cap,
                             int64_t *offsets, int64_t seqs_cap, int64_t *num_seqs,
                             int64_t *num_tokens, void *hip_stream);

/*
 * Tokens peer's tree holds: the number of distinct non-empty prefixes of its
 * set (one KV-cache entry each for the local peer).  *tokens is HOST.  Walks
 * the tree on the device; host-synchronous.
 * Errors: PR_EINVAL (peer out of range, tokens NULL), PR_ESTATE, PR_ENOMEM,
 * PR_EDEVICE.
 */
pr_status pr_tree_tokens(pr_forest *f, int32_t peer, int64_t *tokens, void *hip_stream);

/*
 * Rebuild the device forest from the nodes some peer still holds.  Device
 * merges (Sec. 3.3's delta updates) rebuild a parent's child block elsewhere
 * and leave the old one behind, and cleared snapshots or evictions leave
 * nodes no peer holds; routing never reaches either, but they take HBM.  The
 * rebuild copies the live nodes level by level into fresh arrays with
 * contiguous child blocks and a fresh label pool.  Routing, exports, token
 * counts and local access times are unchanged; node ids are not kept.
 * Outputs: *nodes_before, *nodes_after HOST, may be NULL (node records in
 * use).  Host-synchronous; waits for the whole device before it frees the old
 * image, so no launch on any stream may still read it.  Holds the old and new
 * image at once while it runs.
 * Errors: PR_EINVAL (f NULL), PR_ESTATE, PR_ENOMEM, PR_EDEVICE.  After an
 * error before the install the old image stays in use; a failed install
 * leaves the forest broken (PR_ESTATE from then on).
 */
pr_status pr_forest_compact(pr_forest *f, int64_t *nodes_before, int64_t *nodes_after, void *hip_stream);

/*
 * The local tree's LRU state (paper, Algorithm 1: a node that runs a request
 * itself and lacks GPU memory calls EvictLRUTrie -- which removes one
 * least-recently-used leaf token of its local tree -- and frees that token's
 * KV cache, until the request fits).  One peer of the forest, the local one,
 * keeps an access time on every path (prefix) of its tree:
 *   - a snapshot load, device load or merge into the local peer stamps the
 *     inserted sequences' prefixes with the current time;
 *   - pr_touch stamps each query's matched prefix (serving a query reuses the
 *     cached prefix it matches);
 *   - pr_evict_lru removes least-recently-used leaf tokens: one eviction
 *     removes the leaf with the smallest time, ties to the deepest leaf, then
 *     to the lexicographically smallest path (signed tokens).
 * Times come from the caller and never decrease (pr_set_time).
 */

/* Make peer the local one (-1: none).  Its current tree gets the current
 * time.  Errors: PR_EINVAL (peer outside [-1, num_peers)), PR_ESTATE,
 * PR_ENOMEM, PR_EDEVICE. */
pr_status pr_set_local_peer(pr_forest *f, int32_t peer);

/* Set the current time (>= the previous one; 0 at creation).  Host only.
 * Errors: PR_EINVAL (NULL forest, time going backwards). */
pr_status pr_set_time(pr_forest *f, int64_t t);

/*
 * Serve num_queries queries at the current time: the prefix of each query
 * that the local tree matches is stamped (DEVICE CSR input as in pr_route; a
 * query with invalid offsets is ignored).  Where a matched prefix ends inside
 * an edge label the edge is split, so the stamp covers exactly the matched
 * tokens.  Match lengths are unchanged.  Host-synchronous.
 * Errors: PR_EINVAL (NULL pointers with num_queries > 0, negative counts),
 * PR_ESTATE (no local peer), PR_ENOMEM, PR_EDEVICE.
 */
pr_status pr_touch(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens,
                   const int64_t *q_offsets, int64_t num_queries, void *hip_stream);

/*
 * EvictLRUTrie, max_tokens times (or until the local tree is empty): removes
 * the first max_tokens paths of the local tree in the order (time ascending,
 * depth descending, path ascending), which is what max_tokens successive
 * single evictions remove since times never grow along a path.  *evicted
 * (HOST) gets the number removed.  Other peers' trees are unchanged.
 * Host-synchronous.
 * Errors: PR_EINVAL (evicted NULL, max_tokens < 0), PR_ESTATE (no local
 * peer), PR_ENOMEM, PR_EDEVICE.  A PR_ENOMEM before the first device change
 * leaves the forest unchanged; one after it (the eviction's later scratch),
 * like every PR_EDEVICE, leaves the forest refusing every call but destroy.
 */
pr_status pr_evict_lru(pr_forest *f, int64_t max_tokens, int64_t *evicted, void *hip_stream);

/*
 * Peer selection under push-back and failover (paper, Section "Hot specialist
 * push-back": originating nodes stop routing to a node that advertised
 * back-pressure, and such a request runs locally or on a slightly inferior
 * peer; Section "In-flight forwarded request failure": on a forward timeout
 * the originating node falls back to the next-best target, which may be
 * itself).  Same walk as pr_route; then the candidates are ordered by larger
 * match length, then (flag PR_SELECT_PREFER_LOCAL) the local peer, then the
 * lower peer id, and
 *   best[q]    = the first eligible candidate, -1 if none;
 *   second[q]  = the next eligible candidate, -1 if none.
 * Arguments:
 *   eligible    DEVICE uint64 [ceil(num_peers / 64)]: bit p % 64 of word
 *               p / 64 set if peer p may receive requests (clear: pushed back
 *               or suspected failed); NULL means every peer.
 *   local_peer  the calling node's own peer id, or -1.  It is always eligible:
 *               the originating node can always run a request itself.
 *   flags       0 or PR_SELECT_PREFER_LOCAL (on equal match the local peer
 *               comes first; with 0, ties go to the lowest id as in pr_route).
 *   match_len   DEVICE int32 [num_queries][num_peers] as in pr_route, or NULL
 *               to skip writing it (the selection still uses every peer's match).
 *   best        DEVICE int32 [num_queries], required.
 *   second      DEVICE int32 [num_queries], or NULL.
 * With eligible NULL, local_peer -1 and flags 0, best equals pr_route's chosen.
 * A query with invalid offsets gets match_len -1, best -1 and second -1.
 * Longest-first order and graph capture as in pr_route.
 * Errors (host side, nothing enqueued): PR_EINVAL (local_peer outside
 * [-1, num_peers), unknown flags, NULL q_offsets or best with num_queries > 0,
 * negative counts), PR_ESTATE / PR_ENOMEM / PR_EDEVICE as in pr_route.
 */
#define PR_SELECT_PREFER_LOCAL 1u

pr_status pr_route_select(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens,
                          const int64_t *q_offsets, int64_t num_queries,
                          const uint64_t *eligible, int32_t local_peer, uint32_t flags,
                          int32_t *match_len, int32_t *best, int32_t *second,
                          void *hip_stream);

/*
 * Wait for the forest's device work and report inputs that device calls
 * skipped since the last check: returns PR_OK if none, else PR_EINVAL with the
 * count in the message (and resets the count).
 */
pr_status pr_forest_check(pr_forest *f);

/* Sizes of the forest's current device layout (for reports and tests). */
typedef struct {
    int32_t num_peers;
    int32_t mask_words;      /* 64-bit peer-mask words per node */
    int64_t num_nodes;       /* union-tree node records in use, root included */
    int64_t pool_tokens;     /* edge-label tokens in use */
    int64_t device_bytes;    /* device memory held by the forest */
    int64_t host_seq_tokens; /* tokens of the host-side snapshot copies */
    int64_t layout_epoch;    /* advances whenever the device arrays that routes
                                read move: an upload after host snapshot loads,
                                growth inside a merge, device load, touch or
                                eviction, compaction, and every change of
                                label_bits (16 to 17 or 32, 17 to 32) */
    int64_t label_token_bytes; /* 2 while routes read a 16-bit copy of the label
                                  pool (every label token in [0, 131071]), else 4 */
    int64_t label_bits;        /* bits routes read per label token: 16 (every label
                                  token in [0, 65535]), 17 (in [0, 131071]: the
                                  16-bit copy plus a plane of bit 16), else 32 */
    int64_t merge_refusals;    /* device update rounds that ran out of capacity and
                                  ran again after the forest grew (their refused
                                  allocations wrote nothing) */
    int64_t first_window_tokens; /* query tokens a route loads before its walk
                                    starts: 256 while, at the last upload of host
                                    snapshots, the root had a single child with a
                                    label of 256 tokens or more, else 128.  Speed
                                    only: results do not depend on it */
} pr_forest_info;

pr_status pr_forest_info_get(pr_forest *f, pr_forest_info *out);

/*
 * Host-side image of the union layout built from the forest's host snapshot
 * copies, for inspection without a GPU (layout tests).  No GPU work.  The
 * pointers stay valid until the next call on f.  PR_ESTATE once merges have
 * run (the host copies no longer describe the forest).  Layout:
 *   nodes  int32 [num_nodes][8]: first label token, label offset in pool
 *          (uint32 bits), label length, first child id, child count, 0,
 *          peer-mask word 0 (low 32 bits, high 32 bits).  Node 0 is the root;
 *          the children of a node are the contiguous ids [first child id,
 *          first child id + child count), sorted by first label token.
 *          Bit p of the mask is set if peer p's tree holds the path from the
 *          root through the node's whole label;
 *   ntok   int32 [num_nodes]: first label token of every node;
 *   nsep   int32 [num_nodes]: for a child block [b, b + cnt) with cnt > 64,
 *          nsep[b + k] = ntok[b + (k * cnt) / 64] for k < 64; with cnt >= 4160
 *          also, for sub-range k = [lo, hi) (lo = (k * cnt) / 64, hi the next
 *          sub-range's lo, or cnt for k = 63) and j < 64,
 *          nsep[b + 64 + 64 k + j] = ntok[b + lo + (j * (hi - lo)) / 64]
 *          (other entries 0);
 *   mext   uint64 [num_nodes][mask_words - 1]: peer-mask words 1.. ;
 *   pool   int32 [pool_tokens]: label tokens.
 */
typedef struct {
    int32_t mask_words;
    int64_t num_nodes, pool_tokens;
    const int32_t *nodes;
    const int32_t *ntok;
    const int32_t *nsep;
    const uint64_t *mext;
    const int32_t *pool;
} pr_image_view;

pr_status pr_forest_host_image(pr_forest *f, pr_image_view *out);

#ifdef __cplusplus
}
#endif

#endif /* PREFIX_ROUTER_H */
