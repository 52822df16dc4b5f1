// router.hip -- C ABI of the gfx950 prefix-cache-aware router (see
// include/prefix_router.h for the contract of every entry point).
//
// Host side: per-peer snapshot copies, the union-forest build, device memory
// with spare capacity for merges, argument checks, the merge round loop and
// launches.  Device side: route_kernels.h, merge_kernels.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_scan.hpp>
#include <string>
#include <vector>

#include "forest_host.h"
#include "forest_layout.h"
#include "compact_kernels.h"
#include "export_kernels.h"
#include "lru_kernels.h"
#include "merge_kernels.h"
#include "narrow_kernels.h"
#include "prefix_router.h"
#include "route_kernels.h"

using pr::Node;

namespace {

thread_local std::string g_err;

pr_status fail(pr_status s, const std::string &msg) {
    g_err = msg;
    return s;
}

pr_status ok() {
    g_err.clear();
    return PR_OK;
}

// Device arrays of the forest.  Node ids and pool offsets never move: growing
// a capacity copies the arrays into larger ones.
struct DevImage {
    // nodes, ntok, nsep, mext and moved share one allocation (node_block)
    void *node_block = nullptr;
    size_t node_block_bytes = 0;
    Node *nodes = nullptr;
    int32_t *ntok = nullptr;
    int32_t *nsep = nullptr;
    uint64_t *mext = nullptr;
    int32_t *pool = nullptr;
    long long *moved = nullptr;
    unsigned long long *ltime = nullptr;  // local peer's access times (allocated while a local peer is set)
    uint16_t *pool16 = nullptr;  // low 16 bits of pool, which routes read while every label token fits 17 bits
    int64_t cap_pool16 = 0;
    uint32_t *hib = nullptr;     // bit 16 of pool token i: bit i % 32 of hib[i / 32] (hib_words(cap_pool16) words)
    int64_t cap_nodes = 0, cap_pool = 0;
    int64_t n_nodes = 0, n_pool = 0;  // host mirror of the device counters
};

// Scratch of one merge call, kept between calls and grown on demand.
struct MergeScratch {
    pr::InsState *st = nullptr;
    unsigned long long *keys_in = nullptr, *keys_out = nullptr;
    int32_t *vals_in = nullptr, *vals_out = nullptr;
    int32_t *grp_nw = nullptr, *grp_nb = nullptr, *win_tok = nullptr, *win_ins = nullptr;
    // add rounds: per sorted entry (cap + 1 entries)
    int32_t *win = nullptr, *widx = nullptr, *headv = nullptr, *hd = nullptr, *nch = nullptr, *cstart = nullptr;
    int32_t *arest = nullptr;  // per insert: label tokens of an ADD insert, else -1
    int64_t *rest = nullptr, *poff = nullptr, *grp_pool = nullptr, *grp_pb = nullptr;
    int64_t cap = 0;
    void *sort_tmp = nullptr;
    size_t sort_tmp_bytes = 0;
    // snapshot loads on the device path stage their host batch here
    int32_t *load_tok = nullptr, *load_peer = nullptr;
    int64_t *load_off = nullptr;
    int64_t load_tok_cap = 0, load_seq_cap = 0;
};

// Scratch of snapshot exports, kept between calls and grown on demand.
struct ExportScratch {
    int64_t *depth = nullptr, *len1 = nullptr, *offs = nullptr;
    int32_t *parent = nullptr, *front = nullptr, *next = nullptr, *leaves = nullptr, *sorted = nullptr;
    int32_t *all = nullptr;  // every visited node (LRU eviction)
    int32_t *counts = nullptr;
    void *tmp = nullptr;
    size_t tmp_bytes = 0;
    int64_t cap = 0;  // node capacity of the per-node arrays
};

// Longest-first order of one route call: each query's length bucket, the
// per-workgroup bucket counts and the order itself.  One set per forest,
// grown on demand; `done` is recorded on the stream of the last route that
// used it, and a route on any stream waits for it before reusing the set.
struct RouteScratch {
    int32_t *order = nullptr;
    uint8_t *bkt = nullptr;
    int32_t *blockcnt = nullptr;
    int64_t cap = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
};

}  // namespace

struct pr_forest {
    int32_t P = 0;
    int32_t W = 1;
    int device = -1;
    std::vector<pr::PeerSeqs> sets;
    bool dirty = true;            // host sets changed since the device image was built
    bool merged = false;          // the device image holds merges the host sets lack
    pr::HostImage host_img;
    bool host_img_valid = false;
    DevImage dev;
    bool has_dev = false;
    pr::MergeCounters *d_ctr = nullptr;
    void *h_stage = nullptr;      // pinned host staging for the small readbacks between device rounds
    uint32_t *d_stage = nullptr;  // h_stage as the device addresses it (nullptr: readbacks by DMA)
    unsigned long long *d_skipped = nullptr;  // inputs skipped by device calls
    MergeScratch ms;
    ExportScratch xs;
    RouteScratch rs;
    long long stamp = 0;          // add-round counter (stamps of moved records)
    int64_t round_nodes = 0;      // records the last merge added (spare capacity kept for the next)
    int64_t round_pool = 0;       // pool tokens the last merge added (0: no merge yet)
    int64_t refusals = 0;         // merge rounds repeated after running out of capacity
    int32_t local = -1;           // peer whose tree keeps access times (-1: none)
    int64_t now = 0;              // current time, set by the caller, never decreasing
    int64_t local_load_time = 0;  // time of the local peer's last host snapshot
    int64_t device_bytes = 0;
    int64_t layout_epoch = 0;     // advances whenever the device arrays the route reads move
    bool narrow = false;          // dev.pool16 and dev.hib mirror dev.pool[0, n_pool) (every label token in
                                  // [0, 131071])
    bool hi17 = false;            // some label token is in [65536, 131071]: routes need the bit plane
    bool wide_window = false;     // routes load the wide first-level window: at the last upload the root
                                  // had one child, with a label at least that long (a choice of speed
                                  // only: both windows give the same results)
    bool broken = false;          // a device update failed; only destroy is valid
};

namespace {

#ifndef PR_ROUTE_LONGEST_FIRST
#define PR_ROUTE_LONGEST_FIRST 1
#endif
// Narrow (16- or 17-bit) label copies for routes; 0 keeps every forest on int32 labels.
// Rounds of at most pr::kPlanMax ADD inserts plan their add phase in one
// workgroup (0: always the multi-launch path, for comparisons).
#ifndef PR_MERGE_PLAN
#define PR_MERGE_PLAN 1
#endif

#ifndef PR_NARROW_LABELS
#define PR_NARROW_LABELS 1
#endif

// Wide first-level window for forests whose root has one long-labelled child
// (0: always the narrow window, for comparisons).
#ifndef PR_WIDE_WINDOW
#define PR_WIDE_WINDOW 1
#endif

// Makes the forest's device current for the duration of a call.
class DeviceScope {
   public:
    explicit DeviceScope(pr_forest *f) {
        if (hipGetDevice(&prev_) != hipSuccess) {
            ok_ = false;
            return;
        }
        if (f->device < 0) f->device = prev_;
        if (f->device != prev_) ok_ = hipSetDevice(f->device) == hipSuccess;
        switched_ = f->device != prev_;
    }
    ~DeviceScope() {
        if (switched_) (void)hipSetDevice(prev_);
    }
    bool ok() const { return ok_; }

   private:
    int prev_ = -1;
    bool ok_ = true;
    bool switched_ = false;
};

constexpr size_t kStageBytes = 256;  // pinned readback staging per forest
constexpr int kDeviceRounds = 2;     // merge rounds queued before the first readback

unsigned grid_threads(int64_t n, int bs) { return (unsigned)((n + bs - 1) / bs); }
unsigned grid_waves(int64_t n) { return (unsigned)((n + pr::kMergeWavesPerBlock - 1) / pr::kMergeWavesPerBlock); }
unsigned grid_split(int64_t n) { return (unsigned)((n + pr::kSplitWaves - 1) / pr::kSplitWaves); }

template <typename T>
bool dalloc(pr_forest *f, T **p, int64_t count) {
    const size_t n = (size_t)std::max<int64_t>(count, 1) * sizeof(T);
    if (hipMalloc((void **)p, n) != hipSuccess) {
        (void)hipGetLastError();
        *p = nullptr;
        return false;
    }
    f->device_bytes += (int64_t)n;
    return true;
}

template <typename T>
void dfree(pr_forest *f, T **p, int64_t count) {
    if (*p) {
        (void)hipFree(*p);
        f->device_bytes -= (int64_t)((size_t)std::max<int64_t>(count, 1) * sizeof(T));
    }
    *p = nullptr;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Words of the bit plane for a pool capacity of cap tokens: two per 64-token
// chunk (the narrow copy kernel writes a chunk's two words together).
int64_t hib_words(int64_t cap) { return 2 * ((cap + 63) / 64) + 2; }

// The per-node arrays of one capacity (records, first tokens, separators,
// extra mask words, move stamps) in one device allocation, each 256-byte
// aligned: growing the forest costs one hipMalloc and one hipFree instead of
// one per array.  Sets d's array pointers and d.cap_nodes.
bool alloc_node_arrays(pr_forest *f, DevImage &d, int64_t cap) {
    const size_t c = (size_t)std::max<int64_t>(cap, 1);
    const size_t o_ntok = align256(c * sizeof(Node));
    const size_t o_nsep = o_ntok + align256(c * sizeof(int32_t));
    const size_t o_mext = o_nsep + align256(c * sizeof(int32_t));
    const size_t o_moved = o_mext + align256(std::max<size_t>(c * (size_t)(f->W - 1), 1) * sizeof(uint64_t));
    const size_t bytes = o_moved + c * sizeof(long long);
    void *b = nullptr;
    if (hipMalloc(&b, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    f->device_bytes += (int64_t)bytes;
    char *p = static_cast<char *>(b);
    d.node_block = b;
    d.node_block_bytes = bytes;
    d.nodes = reinterpret_cast<Node *>(p);
    d.ntok = reinterpret_cast<int32_t *>(p + o_ntok);
    d.nsep = reinterpret_cast<int32_t *>(p + o_nsep);
    d.mext = reinterpret_cast<uint64_t *>(p + o_mext);
    d.moved = reinterpret_cast<long long *>(p + o_moved);
    d.cap_nodes = (int64_t)c;
    return true;
}

void free_node_arrays(pr_forest *f, DevImage &d) {
    if (d.node_block) {
        (void)hipFree(d.node_block);
        f->device_bytes -= (int64_t)d.node_block_bytes;
    }
    d.node_block = nullptr;
    d.node_block_bytes = 0;
    d.nodes = nullptr;
    d.ntok = d.nsep = nullptr;
    d.mext = nullptr;
    d.moved = nullptr;
}

void free_image(pr_forest *f) {
    DevImage &d = f->dev;
    free_node_arrays(f, d);
    dfree(f, &d.pool, d.cap_pool);
    dfree(f, &d.ltime, d.cap_nodes);
    dfree(f, &d.pool16, d.cap_pool16);
    dfree(f, &d.hib, hib_words(d.cap_pool16));
    d = DevImage();
    f->has_dev = false;
    f->narrow = false;
    f->hi17 = false;
}

void free_export_scratch(pr_forest *f) {
    ExportScratch &X = f->xs;
    dfree(f, &X.depth, X.cap);
    dfree(f, &X.len1, X.cap + 1);
    dfree(f, &X.offs, X.cap + 1);
    dfree(f, &X.parent, X.cap);
    dfree(f, &X.front, X.cap);
    dfree(f, &X.next, X.cap);
    dfree(f, &X.leaves, X.cap);
    dfree(f, &X.sorted, X.cap);
    dfree(f, &X.all, X.cap);
    dfree(f, &X.counts, 3);
    if (X.tmp) (void)hipFree(X.tmp);
    f->device_bytes -= (int64_t)X.tmp_bytes;
    X = ExportScratch();
}

void free_add_scratch(pr_forest *f) {
    MergeScratch &m = f->ms;
    const int64_t c = m.cap + 1;
    dfree(f, &m.win, c);
    dfree(f, &m.widx, c);
    dfree(f, &m.headv, c);
    dfree(f, &m.hd, c);
    dfree(f, &m.nch, c);
    dfree(f, &m.cstart, c);
    dfree(f, &m.rest, c);
    dfree(f, &m.poff, c);
    dfree(f, &m.grp_pool, c);
    dfree(f, &m.grp_pb, c);
    dfree(f, &m.arest, c);
}

void free_scratch(pr_forest *f) {
    MergeScratch &m = f->ms;
    dfree(f, &m.st, m.cap);
    dfree(f, &m.keys_in, m.cap);
    dfree(f, &m.keys_out, m.cap);
    dfree(f, &m.vals_in, m.cap);
    dfree(f, &m.vals_out, m.cap);
    dfree(f, &m.grp_nw, m.cap);
    dfree(f, &m.grp_nb, m.cap);
    dfree(f, &m.win_tok, m.cap);
    dfree(f, &m.win_ins, m.cap);
    free_add_scratch(f);
    if (m.sort_tmp) (void)hipFree(m.sort_tmp);
    f->device_bytes -= (int64_t)m.sort_tmp_bytes;
    dfree(f, &m.load_tok, m.load_tok_cap);
    dfree(f, &m.load_peer, m.load_seq_cap);
    dfree(f, &m.load_off, m.load_seq_cap + 1);
    m = MergeScratch();
    free_export_scratch(f);
}

// Buffers only (the event stays); callers make sure no route still uses them.
void free_route_buffers(pr_forest *f) {
    RouteScratch &R = f->rs;
    dfree(f, &R.order, R.cap);
    dfree(f, &R.bkt, R.cap);
    dfree(f, &R.blockcnt, (int64_t)pr::kOrderMaxBlocks * pr::kOrderBuckets);
    R.cap = 0;
}

pr_status ensure_host_image(pr_forest *f) {
    if (f->host_img_valid) return PR_OK;
    std::string err;
    pr::HostImage img;
    if (!pr::build_union_image(f->sets, f->W, &img, &err)) return fail(PR_ENOMEM, err);
    f->host_img = std::move(img);
    f->host_img_valid = true;
    return PR_OK;
}

void drop_pool16(pr_forest *f);

// Grow the node and pool capacities to hold at least the given totals.
pr_status ensure_capacity(pr_forest *f, int64_t need_nodes, int64_t need_pool, hipStream_t s) {
    DevImage &d = f->dev;
    if (need_pool > (int64_t)UINT32_MAX) return fail(PR_ENOMEM, "label pool would exceed 2^32 tokens");
    if (need_nodes > (int64_t)INT32_MAX) return fail(PR_ENOMEM, "node count would exceed 2^31");
    if (need_nodes > d.cap_nodes) {
        // rebuilt child blocks append records with every add round, so node
        // arrays grow fourfold: each growth (allocate, copy, wait for the
        // device, free) costs milliseconds of host time
        const int64_t cap = std::min<int64_t>(std::max<int64_t>(need_nodes, 4 * d.cap_nodes), (int64_t)INT32_MAX);
        DevImage nd;
        if (!alloc_node_arrays(f, nd, cap)) return fail(PR_ENOMEM, "hipMalloc failed while growing the forest");
        const int64_t n = d.n_nodes;
        if (hipMemcpyAsync(nd.nodes, d.nodes, n * sizeof(Node), hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemcpyAsync(nd.ntok, d.ntok, n * sizeof(int32_t), hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemcpyAsync(nd.nsep, d.nsep, n * sizeof(int32_t), hipMemcpyDeviceToDevice, s) != hipSuccess ||
            (f->W > 1 && hipMemcpyAsync(nd.mext, d.mext, n * (f->W - 1) * sizeof(uint64_t), hipMemcpyDeviceToDevice,
                                        s) != hipSuccess) ||
            hipMemcpyAsync(nd.moved, d.moved, d.cap_nodes * sizeof(long long), hipMemcpyDeviceToDevice, s) !=
                hipSuccess ||
            hipMemsetAsync(nd.moved + d.cap_nodes, 0, (nd.cap_nodes - d.cap_nodes) * sizeof(long long), s) !=
                hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) {
            free_node_arrays(f, nd);
            return fail(PR_EDEVICE, "device copy failed while growing the forest");
        }
        unsigned long long *lt = nullptr;
        if (d.ltime && (!dalloc(f, &lt, nd.cap_nodes) ||
                        hipMemcpyAsync(lt, d.ltime, n * sizeof(unsigned long long), hipMemcpyDeviceToDevice, s) !=
                            hipSuccess ||
                        hipStreamSynchronize(s) != hipSuccess)) {
            dfree(f, &lt, nd.cap_nodes);
            free_node_arrays(f, nd);
            return fail(PR_ENOMEM, "growing the access times failed");
        }
        // a route launched earlier on another stream may still read the old arrays
        if (hipDeviceSynchronize() != hipSuccess) {
            dfree(f, &lt, nd.cap_nodes);
            free_node_arrays(f, nd);
            return fail(PR_EDEVICE, "hipDeviceSynchronize failed while growing the forest");
        }
        if (lt) {
            dfree(f, &d.ltime, d.cap_nodes);
            d.ltime = lt;
        }
        free_node_arrays(f, d);
        d.node_block = nd.node_block;
        d.node_block_bytes = nd.node_block_bytes;
        d.nodes = nd.nodes;
        d.ntok = nd.ntok;
        d.nsep = nd.nsep;
        d.mext = nd.mext;
        d.moved = nd.moved;
        d.cap_nodes = nd.cap_nodes;
        f->layout_epoch++;
    }
    if (need_pool > d.cap_pool) {
        const int64_t cap = std::min<int64_t>(std::max<int64_t>(need_pool, d.cap_pool + d.cap_pool / 2),
                                              (int64_t)UINT32_MAX);
        int32_t *np = nullptr;
        if (!dalloc(f, &np, cap)) return fail(PR_ENOMEM, "hipMalloc failed while growing the label pool");
        // the narrow copy grows with the pool, under the same wait (without
        // the memory, routes fall back to the int32 pool)
        uint16_t *n16 = nullptr;
        uint32_t *nhb = nullptr;
        const bool narrow = f->narrow && d.pool16 && d.hib;
        const bool keep16 = narrow && dalloc(f, &n16, cap) && dalloc(f, &nhb, hib_words(cap));
        // the tail is zeroed: a merge round refused for lack of capacity can
        // leave unwritten tokens below the used size, which the narrow copy
        // then converts
        if (hipMemcpyAsync(np, d.pool, d.n_pool * sizeof(int32_t), hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemsetAsync(np + d.n_pool, 0, (cap - d.n_pool) * sizeof(int32_t), s) != hipSuccess ||
            (keep16 &&
             (hipMemcpyAsync(n16, d.pool16, d.n_pool * sizeof(uint16_t), hipMemcpyDeviceToDevice, s) != hipSuccess ||
              hipMemcpyAsync(nhb, d.hib, hib_words(d.n_pool) * sizeof(uint32_t), hipMemcpyDeviceToDevice, s) !=
                  hipSuccess)) ||
            hipStreamSynchronize(s) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
            dfree(f, &np, cap);
            dfree(f, &n16, cap);
            dfree(f, &nhb, hib_words(cap));
            return fail(PR_EDEVICE, "device copy failed while growing the label pool");
        }
        dfree(f, &d.pool, d.cap_pool);
        d.pool = np;
        d.cap_pool = cap;
        if (keep16) {
            dfree(f, &d.pool16, d.cap_pool16);
            dfree(f, &d.hib, hib_words(d.cap_pool16));
            d.pool16 = n16;
            d.hib = nhb;
            d.cap_pool16 = cap;
        } else if (narrow) {
            dfree(f, &n16, cap);
            drop_pool16(f);
        }
        f->layout_epoch++;
    }
    return PR_OK;
}

pr::DevForest dev_view(const pr_forest *f);

// The narrow label copy.  While every label token lies in [0, 131071], routes
// read labels from pool16 (the low 16 bits: half the label bytes) and, once
// some token is 65536 or more, from hib (bit 16, one bit per token) as well;
// otherwise from the int32 pool.  Labels are only ever appended to the pool
// (a split reuses a span of its label), so the copy follows merges by
// converting the appended range.
void drop_pool16(pr_forest *f) {
    DevImage &d = f->dev;
    if (d.pool16 || d.hib) {
        // a route launched earlier on another stream may still read them
        (void)hipDeviceSynchronize();
        dfree(f, &d.pool16, d.cap_pool16);
        dfree(f, &d.hib, hib_words(d.cap_pool16));
        f->layout_epoch++;
    }
    d.cap_pool16 = 0;
    f->narrow = false;
    f->hi17 = false;
}

// Enqueue the copy of pool[from, n_pool) on s, first growing the copy to the
// pool's capacity (then it is rebuilt from 0).  Tokens in [65536, 131071] are
// counted in the merge counters' hi_tokens, tokens outside [0, 131071] in
// wide_tokens; the caller reads them with its next counter readback, turns
// the bit plane on for the former and drops the copy for the latter.  Without
// memory for a larger copy, routes fall back to the int32 pool.
// device_end: the range ends at the device counters' n_pool (a merge whose
// rounds the host has not read back), on a grid sized without it.
pr_status pool16_extend(pr_forest *f, int64_t from, hipStream_t s, bool device_end = false) {
    DevImage &d = f->dev;
    if (!f->narrow) return PR_OK;
    if (d.cap_pool16 < d.cap_pool) {
        uint16_t *np = nullptr;
        uint32_t *nh = nullptr;
        if (!dalloc(f, &np, d.cap_pool) || !dalloc(f, &nh, hib_words(d.cap_pool))) {
            dfree(f, &np, d.cap_pool);
            drop_pool16(f);
            return PR_OK;
        }
        if (d.pool16) {
            if (hipDeviceSynchronize() != hipSuccess) {
                dfree(f, &np, d.cap_pool);
                dfree(f, &nh, hib_words(d.cap_pool));
                return fail(PR_EDEVICE, "hipDeviceSynchronize failed while growing the narrow labels");
            }
            dfree(f, &d.pool16, d.cap_pool16);
            dfree(f, &d.hib, hib_words(d.cap_pool16));
        }
        d.pool16 = np;
        d.hib = nh;
        d.cap_pool16 = d.cap_pool;
        from = 0;
        f->layout_epoch++;
    }
    const int64_t to = device_end ? d.cap_pool : d.n_pool;
    if (to > from) {
        const int64_t chunks = (to + pr::kWave - 1) / pr::kWave - from / pr::kWave;
        // a wave per chunk: each wave's load waits on memory, so waves, not
        // iterations, carry the chunks
        const int64_t blocks = device_end && from > 0 ? 2048 : std::min<int64_t>((chunks + 3) / 4, 16384);
        hipLaunchKernelGGL(pr::pool_narrow_kernel, dim3((unsigned)blocks), dim3(pr::kNarrowThreads), 0, s, d.pool,
                           d.pool16, d.hib, from, to, &f->d_ctr->hi_tokens, &f->d_ctr->wide_tokens,
                           device_end ? (const unsigned long long *)&f->d_ctr->n_pool : nullptr);
        if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "narrow label copy failed to launch");
    }
    return PR_OK;
}

// Access times of the local peer: every node it holds gets time t, others 0.
pr_status init_local_times(pr_forest *f, int64_t t) {
    DevImage &d = f->dev;
    if (!d.ltime && !dalloc(f, &d.ltime, d.cap_nodes)) return fail(PR_ENOMEM, "hipMalloc failed for access times");
    hipLaunchKernelGGL(pr::lru_init_kernel, dim3(grid_threads(std::max<int64_t>(d.n_nodes, 1), 256)), dim3(256), 0,
                       nullptr, dev_view(f), d.n_nodes, (unsigned long long)t);
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(nullptr) != hipSuccess)
        return fail(PR_EDEVICE, "access-time initialisation failed");
    return PR_OK;
}

// Rebuild and upload the device image if snapshots changed since the last one.
pr_status commit(pr_forest *f) {
    if (!f->dirty && f->has_dev) return PR_OK;
    pr_status s = ensure_host_image(f);
    if (s) return s;
    if (!f->d_skipped) {
        if (!dalloc(f, &f->d_skipped, 1) || !dalloc(f, &f->d_ctr, 1)) return fail(PR_ENOMEM, "hipMalloc failed");
        if (!f->h_stage && hipHostMalloc(&f->h_stage, kStageBytes, hipHostMallocDefault) != hipSuccess) {
            f->h_stage = nullptr;
            return fail(PR_ENOMEM, "hipHostMalloc failed for the readback staging");
        }
        void *dp = nullptr;
        if (hipHostGetDevicePointer(&dp, f->h_stage, 0) == hipSuccess)
            f->d_stage = static_cast<uint32_t *>(dp);
        else
            (void)hipGetLastError();  // readbacks fall back to DMA copies
        if (hipMemset(f->d_skipped, 0, sizeof(unsigned long long)) != hipSuccess)
            return fail(PR_EDEVICE, "hipMemset failed");
    }
    // earlier launches may still read the old image
    if (f->has_dev && hipDeviceSynchronize() != hipSuccess) return fail(PR_EDEVICE, "hipDeviceSynchronize failed");
    if (f->has_dev) free_image(f);
    const pr::HostImage &h = f->host_img;
    DevImage &d = f->dev;
    const int64_t n = (int64_t)h.nodes.size(), np = (int64_t)h.pool.size();
    // merges append records (rebuilt blocks move), so node capacity starts at
    // four times the image (a few merge batches before the first growth);
    // labels grow only by new leaves
    d.cap_pool = std::max<int64_t>(np + np / 4, 4096);
    if (!alloc_node_arrays(f, d, std::max<int64_t>(4 * n, 1024)) || !dalloc(f, &d.pool, d.cap_pool)) {
        free_image(f);
        return fail(PR_ENOMEM, "hipMalloc failed for the forest image");
    }
    if (hipMemcpy(d.nodes, h.nodes.data(), n * sizeof(Node), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(d.ntok, h.ntok.data(), n * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(d.nsep, h.nsep.data(), n * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess ||
        (f->W > 1 && hipMemcpy(d.mext, h.mext.data(), h.mext.size() * sizeof(uint64_t), hipMemcpyHostToDevice) !=
                         hipSuccess) ||
        (np > 0 && hipMemcpy(d.pool, h.pool.data(), np * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess) ||
        hipMemset(d.pool + np, 0, (d.cap_pool - np) * sizeof(int32_t)) != hipSuccess ||
        hipMemset(d.moved, 0, d.cap_nodes * sizeof(long long)) != hipSuccess) {
        free_image(f);
        return fail(PR_EDEVICE, "upload of the forest image failed");
    }
    d.n_nodes = n;
    d.n_pool = np;
    f->wide_window = PR_WIDE_WINDOW && n > 1 && h.nodes[0].ct_cnt == 1 &&
                     h.nodes[(size_t)h.nodes[0].ct_beg].lab_len >= pr::kWave * pr::kWideWinVectors;
    pr::MergeCounters c;
    std::memset(&c, 0, sizeof(c));
    c.n_nodes = (unsigned long long)n;
    c.n_pool = (unsigned long long)np;
    if (hipMemcpy(f->d_ctr, &c, sizeof(c), hipMemcpyHostToDevice) != hipSuccess)
        return fail(PR_EDEVICE, "counter upload failed");
    // narrow labels when every token fits 17 bits (else, or without the memory,
    // int32): the low 16 bits, and bit 16 as a plane once some token needs it
    f->narrow = PR_NARROW_LABELS &&
                std::all_of(h.pool.begin(), h.pool.end(), [](int32_t t) { return (uint32_t)t <= 0x1FFFFu; });
    f->hi17 = f->narrow && std::any_of(h.pool.begin(), h.pool.end(), [](int32_t t) { return (uint32_t)t > 0xFFFFu; });
    if (f->narrow) {
        std::vector<uint16_t> p16;
        std::vector<uint32_t> hb;
        try {
            p16.assign(h.pool.begin(), h.pool.end());  // the low 16 bits
            hb.assign((size_t)hib_words(np), 0u);
            for (int64_t i = 0; i < np; i++) hb[(size_t)(i >> 5)] |= (((uint32_t)h.pool[(size_t)i] >> 16) & 1u) << (i & 31);
        } catch (const std::bad_alloc &) {
            f->narrow = false;
        }
        if (f->narrow && dalloc(f, &d.pool16, d.cap_pool) && dalloc(f, &d.hib, hib_words(d.cap_pool))) {
            d.cap_pool16 = d.cap_pool;
            if ((np > 0 && hipMemcpy(d.pool16, p16.data(), np * sizeof(uint16_t), hipMemcpyHostToDevice) != hipSuccess) ||
                hipMemcpy(d.hib, hb.data(), hb.size() * sizeof(uint32_t), hipMemcpyHostToDevice) != hipSuccess) {
                d.cap_pool16 = d.cap_pool;
                free_image(f);
                return fail(PR_EDEVICE, "upload of the narrow labels failed");
            }
        } else {
            dfree(f, &d.pool16, d.cap_pool);
            dfree(f, &d.hib, hib_words(d.cap_pool));
            f->narrow = false;
        }
    }
    if (!f->narrow) f->hi17 = false;
    f->has_dev = true;
    f->dirty = false;
    f->merged = false;
    f->layout_epoch++;
    if (f->local >= 0) {
        pr_status r = init_local_times(f, f->local_load_time);
        if (r) return r;
    }
    // the device image is the state of record now; drop the host copy of it
    f->host_img = pr::HostImage();
    f->host_img_valid = false;
    return PR_OK;
}

// Longest-first order: the dispatcher starts one wave per query in index
// order and refills a slot when its query ends, so with only a few long
// queries per slot the last long ones to start leave most slots idle at the
// end of the launch.  Taking the batch longest first removes that tail.  It
// pays where a wave slot of the chip (256 CUs x 32 waves) gets between one
// and eight queries of at least 4,096 tokens on average; elsewhere the order
// kernel (a few microseconds) costs more than the tail.
bool use_longest_first(int64_t nq, int64_t ntok) {
    const int64_t slots = 256 * 32;
    return PR_ROUTE_LONGEST_FIRST && nq > slots && nq <= 8 * slots && nq <= pr::kOrderMaxQueries &&
           ntok >= 4096 * nq;
}

// The two order launches (at most 16 workgroups each) on stream s: bkt gets
// every query's length bucket (a quarter of the mean query wide), blockcnt
// the per-workgroup bucket counts, order the queries longest first.  Every
// entry read is written earlier in the same two launches, so the buffers need
// no clearing.  nq <= pr::kOrderMaxQueries.
pr_status launch_order(const int64_t *q_offsets, int64_t nq, int64_t ntok, hipStream_t s, uint8_t *bkt,
                       int32_t *blockcnt, int32_t *order) {
    const uint32_t unit = (uint32_t)std::min<int64_t>(std::max<int64_t>(1, ntok / nq / 4), INT32_MAX);
    const unsigned blocks = (unsigned)((nq + pr::kOrderChunk - 1) / pr::kOrderChunk);
    hipLaunchKernelGGL(pr::route_order_count_kernel, dim3(blocks), dim3(pr::kOrderThreads), 0, s, q_offsets,
                       (int32_t)nq, unit, bkt, blockcnt);
    hipLaunchKernelGGL(pr::route_order_scatter_kernel, dim3(blocks), dim3(pr::kOrderThreads), 0, s, bkt,
                       (int32_t)nq, blockcnt, order);
    if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "route order launch failed");
    return PR_OK;
}

// Fill f->rs.order with the queries longest first (two launches of at most 16
// workgroups) on stream s; length buckets are a quarter of the mean query wide.
pr_status route_order(pr_forest *f, const int64_t *q_offsets, int64_t nq, int64_t ntok, hipStream_t s,
                      const int32_t **order) {
    RouteScratch &R = f->rs;
    if (!R.done && hipEventCreateWithFlags(&R.done, hipEventDisableTiming) != hipSuccess) {
        R.done = nullptr;
        return fail(PR_EDEVICE, "hipEventCreate failed");
    }
    if (nq > R.cap) {
        // an earlier route, on any stream, may still read the old buffer
        if (R.pending && hipEventSynchronize(R.done) != hipSuccess)
            return fail(PR_EDEVICE, "waiting for an earlier route failed");
        R.pending = false;
        free_route_buffers(f);
        const int64_t cap = std::max<int64_t>(nq, std::min<int64_t>(2 * R.cap, pr::kOrderMaxQueries));
        R.cap = cap;  // sizes for free_route_buffers, also after a partial allocation
        if (!dalloc(f, &R.order, cap) || !dalloc(f, &R.bkt, cap) ||
            !dalloc(f, &R.blockcnt, (int64_t)pr::kOrderMaxBlocks * pr::kOrderBuckets)) {
            free_route_buffers(f);
            return fail(PR_ENOMEM, "hipMalloc failed for the route order");
        }
    }
    if (R.pending && hipStreamWaitEvent(s, R.done, 0) != hipSuccess)
        return fail(PR_EDEVICE, "hipStreamWaitEvent failed");
    pr_status r = launch_order(q_offsets, nq, ntok, s, R.bkt, R.blockcnt, R.order);
    if (r) return r;
    *order = R.order;
    return PR_OK;
}

template <int W, bool SEL, typename LT, bool HB>
void launch_route_t(const pr_forest *f, const LT *pool, const int32_t *qt, int64_t ntok, const int64_t *qo,
                    int64_t nq, const pr::Select &sel, int32_t *ml, int32_t *ch, const int32_t *order,
                    hipStream_t s) {
    const int64_t blocks = (nq + pr::kRouteWavesPerBlock - 1) / pr::kRouteWavesPerBlock;
    const uint32_t *hib = HB ? f->dev.hib : nullptr;
    if (f->wide_window)
        hipLaunchKernelGGL((pr::route_kernel<W, SEL, LT, HB, pr::kWideWinVectors>), dim3((unsigned)blocks),
                           dim3(pr::kWave * pr::kRouteWavesPerBlock), 0, s, f->dev.nodes, f->dev.ntok, f->dev.nsep,
                           f->dev.mext, pool, hib, qt, ntok, qo, nq, f->P, sel, ml, ch, order);
    else
        hipLaunchKernelGGL((pr::route_kernel<W, SEL, LT, HB>), dim3((unsigned)blocks),
                           dim3(pr::kWave * pr::kRouteWavesPerBlock), 0, s, f->dev.nodes, f->dev.ntok, f->dev.nsep,
                           f->dev.mext, pool, hib, qt, ntok, qo, nq, f->P, sel, ml, ch, order);
}

template <int W, bool SEL>
void launch_route_l(const pr_forest *f, const int32_t *qt, int64_t ntok, const int64_t *qo, int64_t nq,
                    const pr::Select &sel, int32_t *ml, int32_t *ch, const int32_t *order, hipStream_t s) {
    const bool narrow = f->narrow && f->dev.pool16 && f->dev.hib;
    if (narrow && f->hi17)
        launch_route_t<W, SEL, uint16_t, true>(f, f->dev.pool16, qt, ntok, qo, nq, sel, ml, ch, order, s);
    else if (narrow)
        launch_route_t<W, SEL, uint16_t, false>(f, f->dev.pool16, qt, ntok, qo, nq, sel, ml, ch, order, s);
    else
        launch_route_t<W, SEL, int32_t, false>(f, f->dev.pool, qt, ntok, qo, nq, sel, ml, ch, order, s);
}

// Plain routing or selection, over the narrow labels when they are current.
template <int W>
hipError_t launch_route(const pr_forest *f, const int32_t *qt, int64_t ntok, const int64_t *qo, int64_t nq,
                        const pr::Select &sel, int32_t *ml, int32_t *ch, const int32_t *order, hipStream_t s) {
    const bool plain = !sel.eligible && !sel.prefer_local && !sel.second;
    if (plain)
        launch_route_l<W, false>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
    else
        launch_route_l<W, true>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
    return hipGetLastError();
}

// The route kernel for the forest's mask-word count.
hipError_t launch_route_w(const pr_forest *f, const int32_t *qt, int64_t ntok, const int64_t *qo, int64_t nq,
                          const pr::Select &sel, int32_t *ml, int32_t *ch, const int32_t *order, hipStream_t s) {
    switch (f->W) {
        case 1: return launch_route<1>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
        case 2: return launch_route<2>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
        case 4: return launch_route<4>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
        case 8: return launch_route<8>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
        default: return launch_route<16>(f, qt, ntok, qo, nq, sel, ml, ch, order, s);
    }
}

// ---- routes without allocation ----------------------------------------------
// The longest-first order of one pr_route_noalloc call lives in one
// file-scope device array per GPU (`scratch`, held until the process ends):
// order (int32 per query), the per-workgroup bucket counts, then each query's
// length bucket (uint8).  On the host the array's name stands for no device
// address; its address on each device comes from hipGetSymbolAddress, taken
// once per device with that device current, and only that address is passed
// to kernels.
constexpr int64_t kNoAllocOrder = 0;
constexpr int64_t kNoAllocBlockcnt = kNoAllocOrder + 4 * (int64_t)pr::kOrderMaxQueries;
constexpr int64_t kNoAllocBkt = kNoAllocBlockcnt + 4 * (int64_t)pr::kOrderMaxBlocks * pr::kOrderBuckets;
constexpr int64_t kNoAllocBytes = kNoAllocBkt + (int64_t)pr::kOrderMaxQueries;
static_assert(PR_NOALLOC_MAX_QUERIES == pr::kOrderMaxQueries, "the header's limit is the order's capacity");
static_assert(kNoAllocBlockcnt % 256 == 0 && kNoAllocBkt % 256 == 0, "aligned sub-arrays");
constexpr int kNoAllocMaxDevices = 64;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace {

std::mutex g_scratch_mu;
unsigned char *g_scratch_dev[kNoAllocMaxDevices] = {};

// The current device's address of `scratch` (dev must be current).
pr_status noalloc_scratch(int dev, unsigned char **out) {
    if (dev < 0 || dev >= kNoAllocMaxDevices) return fail(PR_EDEVICE, "device id beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(PR_EDEVICE, std::string("hipGetSymbolAddress of the route scratch failed: ") +
                                        hipGetErrorString(e));
        }
        g_scratch_dev[dev] = static_cast<unsigned char *>(p);
    }
    *out = g_scratch_dev[dev];
    return PR_OK;
}

// ---- merge ------------------------------------------------------------------

pr_status ensure_merge_scratch(pr_forest *f, int64_t n, hipStream_t s) {
    MergeScratch &m = f->ms;
    if (n > m.cap) {
        const int64_t cap = std::max<int64_t>(n, m.cap * 2);
        dfree(f, &m.st, m.cap);
        dfree(f, &m.keys_in, m.cap);
        dfree(f, &m.keys_out, m.cap);
        dfree(f, &m.vals_in, m.cap);
        dfree(f, &m.vals_out, m.cap);
        dfree(f, &m.grp_nw, m.cap);
        dfree(f, &m.grp_nb, m.cap);
        dfree(f, &m.win_tok, m.cap);
        dfree(f, &m.win_ins, m.cap);
        free_add_scratch(f);
        m.cap = 0;
        const int64_t c1 = cap + 1;
        if (!dalloc(f, &m.st, cap) || !dalloc(f, &m.keys_in, cap) || !dalloc(f, &m.keys_out, cap) ||
            !dalloc(f, &m.vals_in, cap) || !dalloc(f, &m.vals_out, cap) || !dalloc(f, &m.grp_nw, cap) ||
            !dalloc(f, &m.grp_nb, cap) || !dalloc(f, &m.win_tok, cap) || !dalloc(f, &m.win_ins, cap) ||
            !dalloc(f, &m.win, c1) || !dalloc(f, &m.widx, c1) || !dalloc(f, &m.headv, c1) ||
            !dalloc(f, &m.hd, c1) || !dalloc(f, &m.nch, c1) || !dalloc(f, &m.cstart, c1) ||
            !dalloc(f, &m.rest, c1) || !dalloc(f, &m.poff, c1) || !dalloc(f, &m.grp_pool, c1) ||
            !dalloc(f, &m.grp_pb, c1) || !dalloc(f, &m.arest, c1)) {
            m.cap = cap;  // so that free_scratch releases the add arrays by their size
            free_scratch(f);
            return fail(PR_ENOMEM, "hipMalloc failed for merge scratch");
        }
        m.cap = cap;
    }
    // one temporary buffer serves the sort and the add round's scans
    size_t need = 0, q = 0;
    if (rocprim::radix_sort_pairs(nullptr, need, m.keys_in, m.keys_out, m.vals_in, m.vals_out, n, 0, 64, s) !=
        hipSuccess)
        return fail(PR_EDEVICE, "radix sort size query failed");
    if (rocprim::exclusive_scan(nullptr, q, m.win, m.widx, 0, (size_t)n, rocprim::plus<int32_t>(), s) != hipSuccess)
        return fail(PR_EDEVICE, "scan size query failed");
    need = std::max(need, q);
    if (rocprim::exclusive_scan(nullptr, q, m.rest, m.poff, (int64_t)0, (size_t)n, rocprim::plus<int64_t>(), s) !=
        hipSuccess)
        return fail(PR_EDEVICE, "scan size query failed");
    need = std::max(need, q);
    if (rocprim::inclusive_scan(nullptr, q, m.headv, m.hd, (size_t)n, rocprim::maximum<int32_t>(), s) != hipSuccess)
        return fail(PR_EDEVICE, "scan size query failed");
    need = std::max(need, q);
    if (rocprim::exclusive_scan(nullptr, q, m.nch, m.cstart, 0, (size_t)n + 1, rocprim::plus<int32_t>(), s) !=
        hipSuccess)
        return fail(PR_EDEVICE, "scan size query failed");
    need = std::max(need, q);
    if (need > m.sort_tmp_bytes) {
        if (m.sort_tmp) (void)hipFree(m.sort_tmp);
        f->device_bytes -= (int64_t)m.sort_tmp_bytes;
        m.sort_tmp_bytes = 0;
        m.sort_tmp = nullptr;
        if (hipMalloc(&m.sort_tmp, need) != hipSuccess) {
            (void)hipGetLastError();
            return fail(PR_ENOMEM, "hipMalloc failed for sort scratch");
        }
        m.sort_tmp_bytes = need;
        f->device_bytes += (int64_t)need;
    }
    return PR_OK;
}

__global__ void reset_round_kernel(pr::MergeCounters *c) {
    c->n_add = 0;
    c->n_split = 0;
    c->pool_need = 0;
    c->node_need = 0;
    c->move_chunks = 0;
    c->plan_n = 0;
    c->plan_fallback = 0;
}

__global__ void reset_call_kernel(pr::MergeCounters *c) {
    c->wide_tokens = 0;
    c->hi_tokens = 0;
    c->n_add = 0;
    c->n_split = 0;
    c->pool_need = 0;
    c->node_need = 0;
    c->overflow = 0;
    c->skipped = 0;
    c->bad_path = 0;
    c->move_chunks = 0;
    c->plan_n = 0;
    c->plan_fallback = 0;
}

__global__ void add_skipped_kernel(unsigned long long *acc, const pr::MergeCounters *c) { *acc += c->skipped; }

// Counters after refused allocations: the used sizes the host clipped to the
// capacities, and no refusal pending.
__global__ void set_used_kernel(pr::MergeCounters *c, unsigned long long n_nodes, unsigned long long n_pool) {
    c->n_nodes = n_nodes;
    c->n_pool = n_pool;
    c->overflow = 0;
}

// One wave stores the words of a small readback straight into the pinned
// staging buffer, at system scope (past the GPU's caches).
__global__ void stage_copy_kernel(const uint32_t *src, uint32_t *dst, int words) {
    for (int i = (int)threadIdx.x; i < words; i += (int)blockDim.x)
        __hip_atomic_store(&dst[i], src[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Copy `bytes` (<= kStageBytes) of device memory to the host through the
// forest's pinned staging buffer and wait.  Whole aligned words go through a
// one-wave kernel that writes the buffer directly (a DMA copy of a few bytes
// costs a blit launch several times as long); anything else by DMA.
bool read_small(pr_forest *f, void *out, const void *dsrc, size_t bytes, hipStream_t s) {
    if (bytes > kStageBytes || !f->h_stage) return false;
    if (f->d_stage && bytes % 4 == 0 && reinterpret_cast<uintptr_t>(dsrc) % 4 == 0) {
        hipLaunchKernelGGL(stage_copy_kernel, dim3(1), dim3(64), 0, s, static_cast<const uint32_t *>(dsrc),
                           f->d_stage, (int)(bytes / 4));
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return false;
    } else if (hipMemcpyAsync(f->h_stage, dsrc, bytes, hipMemcpyDeviceToHost, s) != hipSuccess ||
               hipStreamSynchronize(s) != hipSuccess) {
        return false;
    }
    std::memcpy(out, f->h_stage, bytes);
    return true;
}

static_assert(sizeof(pr::MergeCounters) <= kStageBytes && sizeof(pr::EvictPlan) <= kStageBytes,
              "readbacks fit the staging buffer");

// Read the device counters and refresh the host mirror of the used sizes
// (growing the arrays copies exactly the used part).
pr_status read_counters(pr_forest *f, pr::MergeCounters *c, hipStream_t s) {
    if (!read_small(f, c, f->d_ctr, sizeof(*c), s)) return fail(PR_EDEVICE, "reading merge counters failed");
    f->dev.n_nodes = (int64_t)c->n_nodes;
    f->dev.n_pool = (int64_t)c->n_pool;
    return PR_OK;
}

// The counters only (the caller decides what the used sizes are).
pr_status read_counters_raw(pr_forest *f, pr::MergeCounters *c, hipStream_t s) {
    if (!read_small(f, c, f->d_ctr, sizeof(*c), s)) return fail(PR_EDEVICE, "reading merge counters failed");
    return PR_OK;
}

pr::DevForest dev_view(const pr_forest *f) {
    pr::DevForest F;
    F.nodes = f->dev.nodes;
    F.ntok = f->dev.ntok;
    F.nsep = f->dev.nsep;
    F.mext = f->dev.mext;
    F.pool = f->dev.pool;
    F.moved = f->dev.moved;
    F.ltime = f->local >= 0 ? f->dev.ltime : nullptr;
    F.local = f->local;
    F.now = (unsigned long long)f->now;
    F.cap_nodes = f->dev.cap_nodes;
    F.cap_pool = f->dev.cap_pool;
    F.W = f->W;
    return F;
}


// Insert a device batch into the device forest (see merge_kernels.h).
pr_status run_merge(pr_forest *f, const int32_t *peer_of, const int32_t *tokens, int64_t num_tokens,
                    const int64_t *offsets, int64_t n, hipStream_t s, int32_t stamp = 1) {
    pr_status r = ensure_merge_scratch(f, n, s);
    if (r) return r;
    const int64_t pool0 = f->dev.n_pool;  // labels appended from here on
    const int64_t nodes0 = f->dev.n_nodes;
    MergeScratch &m = f->ms;
    pr::Batch B{peer_of, tokens, offsets, num_tokens, n, f->P, stamp};
    const int bs = 256, wb = 64 * pr::kMergeWavesPerBlock;
    hipLaunchKernelGGL(reset_call_kernel, dim3(1), dim3(1), 0, s, f->d_ctr);
    hipLaunchKernelGGL(pr::merge_validate_kernel, dim3(grid_threads(n, bs)), dim3(bs), 0, s, B, m.st, f->d_ctr);
    pr::MergeCounters c;
    const int max_rounds = 100000;
    int round = 0;
    int refusals = 0;
    bool done = false;
    // Rounds the device drives: kDeviceRounds full rounds, each sized on the
    // device (the add phase planned in one workgroup, the later add steps
    // striding over what it planned), then a checking walk, the narrow copy
    // and one readback.  Most batches end there: the first round places every
    // insert but the losers of a slot or an edge, the second places those.
    // Anything else (work left, a round too large for the one-workgroup plan,
    // a refused allocation) continues in the host-driven rounds below, which
    // read the counters back after every walk.  A forest's first merge takes
    // the host-driven rounds, which size its spare capacity.
    if (PR_MERGE_PLAN && n <= pr::kPlanMaxBatch && f->round_pool > 0) {
        if ((r = ensure_capacity(f, f->dev.n_nodes + 2 * std::max<int64_t>(f->round_nodes, n),
                                 f->dev.n_pool + 2 * f->round_pool, s)))
            return r;
        const pr::DevForest F = dev_view(f);
        // the round counters start cleared (reset_call_kernel above), and each
        // round's split kernel clears them for the next walk
        for (int k = 0; k < kDeviceRounds; k++) {
            hipLaunchKernelGGL(pr::merge_walk_kernel, dim3(grid_waves(n)), dim3(wb), 0, s, F, B, m.st, f->d_ctr);
            hipLaunchKernelGGL(pr::merge_tally_kernel,
                               dim3((unsigned)std::min<int64_t>(256, (n + pr::kTallyThreads - 1) / pr::kTallyThreads)),
                               dim3(pr::kTallyThreads), 0, s, B, m.st, f->d_ctr, m.arest);
            hipLaunchKernelGGL(pr::add_plan_kernel, dim3(1), dim3(pr::kPlanThreads), 0, s, F, B, m.st, m.arest,
                               (int64_t)-1, m.keys_out, m.vals_out, m.win, m.widx, m.hd, m.cstart, m.grp_nw, m.grp_nb,
                               m.win_tok, m.rest, f->d_ctr);
            const long long stamp = ++f->stamp;
            hipLaunchKernelGGL(pr::add_move_kernel, dim3(pr::kMoveBlocks), dim3(wb), 0, s, F, m.keys_out, (int64_t)-1,
                               m.cstart, f->d_ctr, m.grp_nw, m.grp_nb, m.win_tok, stamp);
            hipLaunchKernelGGL(pr::add_leaf_kernel, dim3(grid_waves(std::min<int64_t>(n, pr::kPlanMax))), dim3(wb), 0,
                               s, F, B, m.keys_out, m.vals_out, (int64_t)-1, m.st, m.win, m.widx, m.poff, m.hd,
                               m.grp_nb, m.grp_pb, m.rest, f->d_ctr);
            hipLaunchKernelGGL(pr::add_sep_kernel, dim3(grid_waves(std::min<int64_t>(n, pr::kPlanMax))), dim3(wb), 0,
                               s, F, m.keys_out, (int64_t)-1, m.grp_nw, m.grp_nb, f->d_ctr);
            hipLaunchKernelGGL(pr::add_fix_kernel, dim3(grid_threads(std::min<int64_t>(n, pr::kPlanMax), bs)),
                               dim3(bs), 0, s, F, m.keys_out, (int64_t)-1, m.grp_nw, m.grp_nb, stamp, f->d_ctr);
            hipLaunchKernelGGL(pr::split_claim_kernel, dim3(grid_threads(n, bs)), dim3(bs), 0, s, F, B, m.st, stamp);
            hipLaunchKernelGGL(pr::split_apply_kernel, dim3(grid_split(n)), dim3(64 * pr::kSplitWaves), 0, s, F, B,
                               m.st, f->d_ctr, stamp, 1);
        }
        hipLaunchKernelGGL(pr::merge_walk_kernel, dim3(grid_waves(n)), dim3(wb), 0, s, F, B, m.st, f->d_ctr);
        hipLaunchKernelGGL(pr::merge_tally_kernel,
                           dim3((unsigned)std::min<int64_t>(256, (n + pr::kTallyThreads - 1) / pr::kTallyThreads)),
                           dim3(pr::kTallyThreads), 0, s, B, m.st, f->d_ctr, m.arest);
        if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "merge launch failed");
        if ((r = pool16_extend(f, pool0, s, true))) return r;
        if ((r = read_counters_raw(f, &c, s))) return r;
        done = !c.overflow && !c.plan_fallback && !c.bad_path && c.n_add == 0 && c.n_split == 0;
        if (!c.overflow) {
            f->dev.n_nodes = (int64_t)c.n_nodes;
            f->dev.n_pool = (int64_t)c.n_pool;
        }  // else the first host-driven readback sees the refusal and clips the counters
    }
    for (; !done && round < max_rounds; round++) {
        hipLaunchKernelGGL(reset_round_kernel, dim3(1), dim3(1), 0, s, f->d_ctr);
        hipLaunchKernelGGL(pr::merge_walk_kernel, dim3(grid_waves(n)), dim3(wb), 0, s, dev_view(f), B, m.st,
                           f->d_ctr);
        hipLaunchKernelGGL(pr::merge_tally_kernel,
                           dim3((unsigned)std::min<int64_t>(256, (n + pr::kTallyThreads - 1) / pr::kTallyThreads)),
                           dim3(pr::kTallyThreads), 0, s, B, m.st, f->d_ctr, m.arest);
        if ((r = read_counters_raw(f, &c, s))) return r;
        if (c.overflow) {
            // The last round ran out of capacity.  Every refused allocation
            // wrote nothing and left its inserts to walk again (above), but
            // the refused requests still advanced the counters: records and
            // tokens past the last allocation that fit were never written, so
            // the counters are clipped to the capacities, and the forest grows
            // to what the round asked for before the round is repeated.
            if (++refusals > 4) break;  // reported below
            f->refusals++;
            const int64_t want_nodes = (int64_t)c.n_nodes, want_pool = (int64_t)c.n_pool;
            f->dev.n_nodes = std::min<int64_t>(want_nodes, f->dev.cap_nodes);
            f->dev.n_pool = std::min<int64_t>(want_pool, f->dev.cap_pool);
            hipLaunchKernelGGL(set_used_kernel, dim3(1), dim3(1), 0, s, f->d_ctr,
                               (unsigned long long)f->dev.n_nodes, (unsigned long long)f->dev.n_pool);
            if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "merge launch failed");
            if ((r = ensure_capacity(f, std::max<int64_t>(want_nodes, f->dev.n_nodes + 1),
                                     std::max<int64_t>(want_pool, f->dev.n_pool + (int64_t)c.pool_need), s)))
                return r;
            continue;
        }
        f->dev.n_nodes = (int64_t)c.n_nodes;
        f->dev.n_pool = (int64_t)c.n_pool;
        if (c.n_add == 0 && c.n_split == 0) break;
        // One round applies both kinds from the same walk: the add phase first
        // (rebuilt child blocks move records; the split phase finds them through
        // their move stamps), then the split phase.  The winners of either are
        // done; the losers (the same slot or the same edge as a winner) walk
        // again.  Allocations come from the device counters; one that does not
        // fit the capacity is refused (see above), so no readback sits between
        // the phases.  A forest whose spare capacity is short of what the last
        // merges added grows first (the walk's tally bounds the pool tokens).
        const int64_t n_split = (int64_t)c.n_split;
        if ((r = ensure_capacity(f, f->dev.n_nodes + 2 * std::max<int64_t>(f->round_nodes, n),
                                 f->dev.n_pool + (int64_t)c.pool_need, s)))
            return r;
        long long add_stamp = 0;
        if (c.n_add > 0) {
            const int64_t n_add = (int64_t)c.n_add;
            const bool plan = PR_MERGE_PLAN && n_add <= pr::kPlanMax && n <= pr::kPlanMaxBatch;
            if (plan) {
                // sort, marks, scans and groups in one workgroup
                hipLaunchKernelGGL(pr::add_plan_kernel, dim3(1), dim3(pr::kPlanThreads), 0, s, dev_view(f), B, m.st,
                                   m.arest, n_add, m.keys_out, m.vals_out, m.win, m.widx, m.hd, m.cstart, m.grp_nw,
                                   m.grp_nb, m.win_tok, m.rest, f->d_ctr);
            } else {
                hipLaunchKernelGGL(pr::add_keys_kernel, dim3(grid_threads(n, bs)), dim3(bs), 0, s, B, m.st, m.keys_in,
                                   m.vals_in);
                size_t tmp = m.sort_tmp_bytes;
                if (rocprim::radix_sort_pairs(m.sort_tmp, tmp, m.keys_in, m.keys_out, m.vals_in, m.vals_out, n, 0, 64,
                                              s) != hipSuccess)
                    return fail(PR_EDEVICE, "radix sort failed");
                // winners, group heads and chunks; their scans; per-group totals
                hipLaunchKernelGGL(pr::add_mark_kernel, dim3(grid_threads(n_add + 1, bs)), dim3(bs), 0, s, dev_view(f),
                                   B, m.keys_out, m.vals_out, n_add, m.st, m.win, m.rest, m.headv, m.nch);
                size_t t1 = m.sort_tmp_bytes;
                if (rocprim::exclusive_scan(m.sort_tmp, t1, m.win, m.widx, 0, (size_t)n_add, rocprim::plus<int32_t>(),
                                            s) != hipSuccess)
                    return fail(PR_EDEVICE, "add scan failed");
                t1 = m.sort_tmp_bytes;
                if (rocprim::exclusive_scan(m.sort_tmp, t1, m.rest, m.poff, (int64_t)0, (size_t)n_add,
                                            rocprim::plus<int64_t>(), s) != hipSuccess)
                    return fail(PR_EDEVICE, "add scan failed");
                t1 = m.sort_tmp_bytes;
                if (rocprim::inclusive_scan(m.sort_tmp, t1, m.headv, m.hd, (size_t)n_add, rocprim::maximum<int32_t>(),
                                            s) != hipSuccess)
                    return fail(PR_EDEVICE, "add scan failed");
                t1 = m.sort_tmp_bytes;
                if (rocprim::exclusive_scan(m.sort_tmp, t1, m.nch, m.cstart, 0, (size_t)n_add + 1,
                                            rocprim::plus<int32_t>(), s) != hipSuccess)
                    return fail(PR_EDEVICE, "add scan failed");
                hipLaunchKernelGGL(reset_round_kernel, dim3(1), dim3(1), 0, s, f->d_ctr);
                hipLaunchKernelGGL(pr::add_group_kernel, dim3(grid_threads(n_add, bs)), dim3(bs), 0, s, dev_view(f),
                                   m.keys_out, m.vals_out, n_add, m.st, m.win, m.rest, m.widx, m.poff, m.hd, m.cstart,
                                   m.grp_nw, m.grp_pool, m.win_tok, m.win_ins, f->d_ctr);
            }
            const long long stamp = ++f->stamp;
            add_stamp = stamp;
            const pr::DevForest F = dev_view(f);
            if (!plan)
                hipLaunchKernelGGL(pr::add_alloc_kernel, dim3(grid_threads(n_add, bs)), dim3(bs), 0, s, F, m.keys_out,
                                   n_add, m.grp_nw, m.grp_pool, m.grp_nb, m.grp_pb, f->d_ctr);
            hipLaunchKernelGGL(pr::add_move_kernel, dim3(pr::kMoveBlocks), dim3(wb), 0, s, F, m.keys_out, n_add,
                               m.cstart, f->d_ctr, m.grp_nw, m.grp_nb, m.win_tok, stamp);
            hipLaunchKernelGGL(pr::add_leaf_kernel, dim3(grid_waves(n_add)), dim3(wb), 0, s, F, B, m.keys_out,
                               m.vals_out, n_add, m.st, m.win, m.widx, m.poff, m.hd, m.grp_nb, m.grp_pb,
                               plan ? m.rest : nullptr, f->d_ctr);
            hipLaunchKernelGGL(pr::add_sep_kernel, dim3(grid_waves(n_add)), dim3(wb), 0, s, F, m.keys_out, n_add,
                               m.grp_nw, m.grp_nb, f->d_ctr);
            hipLaunchKernelGGL(pr::add_fix_kernel, dim3(grid_threads(n_add, bs)), dim3(bs), 0, s, F, m.keys_out,
                               n_add, m.grp_nw, m.grp_nb, stamp, f->d_ctr);
        }
        if (n_split > 0) {
            const pr::DevForest F = dev_view(f);
            hipLaunchKernelGGL(pr::split_claim_kernel, dim3(grid_threads(n, bs)), dim3(bs), 0, s, F, B, m.st,
                               add_stamp);
            hipLaunchKernelGGL(pr::split_apply_kernel, dim3(grid_split(n)), dim3(64 * pr::kSplitWaves), 0, s, F, B,
                               m.st, f->d_ctr, add_stamp, 0);
        }
        if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "merge launch failed");
    }
    if (round == max_rounds) return fail(PR_EDEVICE, "merge did not converge");
    // records and pool tokens this merge added: the spare capacity the next
    // one keeps free
    f->round_nodes = std::max<int64_t>(f->dev.n_nodes - nodes0, 0);
    f->round_pool = std::max<int64_t>(f->dev.n_pool - pool0, 1);
    hipLaunchKernelGGL(add_skipped_kernel, dim3(1), dim3(1), 0, s, f->d_skipped, f->d_ctr);
    if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "merge launch failed");
    if (!done) {  // the device-driven rounds read everything back with the narrow copy done
        if ((r = pool16_extend(f, pool0, s))) return r;
        if ((r = read_counters(f, &c, s))) return r;
    }
    if (c.overflow || c.bad_path)
        return fail(PR_EDEVICE, "merge invariant broken (overflow " + std::to_string(c.overflow) + ", bad paths " +
                                    std::to_string(c.bad_path) + "); destroy the forest");
    if (c.wide_tokens)
        drop_pool16(f);  // a label token outside [0, 131071] arrived
    else if (c.hi_tokens && f->narrow && !f->hi17) {
        f->hi17 = true;  // routes now read the bit plane too (a new kernel: the arrays stay)
        f->layout_epoch++;
    }
    f->merged = true;
    return PR_OK;
}

// Snapshot load once merges have run: the host copies no longer describe the
// device forest, so the replacement happens on the device: clear the peer from
// every mask, then insert the snapshot for it.
pr_status device_load(pr_forest *f, int32_t peer, const pr::PeerSeqs &S) {
    MergeScratch &m = f->ms;
    const int64_t ns = S.count(), nt = (int64_t)S.tokens.size();
    hipStream_t s = nullptr;
    hipLaunchKernelGGL(pr::clear_peer_kernel, dim3(grid_threads(f->dev.n_nodes, 256)), dim3(256), 0, s,
                       dev_view(f), f->dev.n_nodes, peer);
    if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "snapshot kernels failed to launch");
    if (ns == 0) return hipStreamSynchronize(s) == hipSuccess ? PR_OK : fail(PR_EDEVICE, "sync failed");
    if (nt > m.load_tok_cap) {
        dfree(f, &m.load_tok, m.load_tok_cap);
        m.load_tok_cap = 0;
        if (!dalloc(f, &m.load_tok, nt)) return fail(PR_ENOMEM, "hipMalloc failed for the snapshot");
        m.load_tok_cap = nt;
    }
    if (ns > m.load_seq_cap) {
        dfree(f, &m.load_peer, m.load_seq_cap);
        dfree(f, &m.load_off, m.load_seq_cap + 1);
        m.load_seq_cap = 0;
        if (!dalloc(f, &m.load_peer, ns) || !dalloc(f, &m.load_off, ns + 1))
            return fail(PR_ENOMEM, "hipMalloc failed for the snapshot");
        m.load_seq_cap = ns;
    }
    if ((nt > 0 && hipMemcpy(m.load_tok, S.tokens.data(), nt * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess) ||
        hipMemcpy(m.load_off, S.offsets.data(), (ns + 1) * sizeof(int64_t), hipMemcpyHostToDevice) != hipSuccess)
        return fail(PR_EDEVICE, "snapshot upload failed");
    hipLaunchKernelGGL(pr::fill_peer_kernel, dim3(grid_threads(ns, 256)), dim3(256), 0, s, m.load_peer, ns, peer);
    if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "snapshot kernels failed to launch");
    return run_merge(f, m.load_peer, m.load_tok, nt, m.load_off, ns, s);
}

pr_status ensure_export_scratch(pr_forest *f, int64_t nn) {
    ExportScratch &X = f->xs;
    if (nn <= X.cap && X.counts) return PR_OK;
    const int64_t cap = std::max<int64_t>(nn, X.cap + X.cap / 2);
    free_export_scratch(f);
    if (!dalloc(f, &X.depth, cap) || !dalloc(f, &X.len1, cap + 1) || !dalloc(f, &X.offs, cap + 1) ||
        !dalloc(f, &X.parent, cap) || !dalloc(f, &X.front, cap) || !dalloc(f, &X.next, cap) ||
        !dalloc(f, &X.leaves, cap) || !dalloc(f, &X.sorted, cap) || !dalloc(f, &X.all, cap) ||
        !dalloc(f, &X.counts, 3)) {
        free_export_scratch(f);
        return fail(PR_ENOMEM, "hipMalloc failed for the export");
    }
    X.cap = cap;
    return PR_OK;
}

// Walk peer's nodes level by level from the root (export_kernels.h) into the
// forest's export scratch: depth and parent of every visited node, the leaves
// (counts[1]) and, if want_all, every visited node (counts[2]).
pr_status walk_peer(pr_forest *f, int32_t peer, bool want_all, hipStream_t s, int32_t counts[3]) {
    const int64_t nn = f->dev.n_nodes;
    pr_status r = ensure_export_scratch(f, nn);
    if (r) return r;
    ExportScratch &X = f->xs;
    const pr::DevForest F = dev_view(f);
    const int wb = 64 * pr::kExportWavesPerBlock;
    hipLaunchKernelGGL(pr::export_init_kernel, dim3(1), dim3(1), 0, s, X.front, X.depth, X.counts);
    int32_t n_front = 1;
    counts[0] = counts[1] = counts[2] = 0;
    while (n_front > 0) {
        hipLaunchKernelGGL(pr::export_reset_kernel, dim3(1), dim3(1), 0, s, X.counts);
        hipLaunchKernelGGL(pr::export_level_kernel,
                           dim3((unsigned)((n_front + pr::kExportWavesPerBlock - 1) / pr::kExportWavesPerBlock)),
                           dim3(wb), 0, s, F, nn, peer, X.front, n_front, X.next, X.leaves, X.depth, X.parent,
                           X.counts, want_all ? X.all : nullptr);
        if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "tree walk launch failed");
        if (!read_small(f, counts, X.counts, 3 * sizeof(int32_t), s))
            return fail(PR_EDEVICE, "tree walk readback failed");
        if (counts[0] > nn || counts[1] > nn || counts[2] > nn)
            return fail(PR_EDEVICE, "tree walk visited more nodes than exist");
        n_front = counts[0];
        std::swap(X.front, X.next);
    }
    return PR_OK;
}

// sendTrie for one peer (see export_kernels.h).  Host-synchronous.  Writes the
// sizes always; the data only if both buffers are given and large enough.
pr_status export_impl(pr_forest *f, int32_t peer, int32_t *tokens, int64_t tokens_cap, int64_t *offsets,
                      int64_t seqs_cap, int64_t *num_seqs, int64_t *num_tokens, hipStream_t s) {
    const int64_t nn = f->dev.n_nodes;
    pr_status r = ensure_export_scratch(f, nn);
    if (r) return r;
    ExportScratch &X = f->xs;
    const pr::DevForest F = dev_view(f);
    const int wb = 64 * pr::kExportWavesPerBlock;
    int32_t counts[3] = {0, 0, 0};
    r = walk_peer(f, peer, false, s, counts);
    if (r) return r;
    const int32_t n_leaves = counts[1];
    int64_t total = 0;
    if (n_leaves > 0) {
        size_t need = 0, need2 = 0;
        if (rocprim::radix_sort_keys(nullptr, need, X.leaves, X.sorted, (size_t)n_leaves, 0, 32, s) != hipSuccess ||
            rocprim::inclusive_scan(nullptr, need2, X.len1 + 1, X.offs + 1, (size_t)n_leaves,
                                    rocprim::plus<int64_t>(), s) != hipSuccess)
            return fail(PR_EDEVICE, "export sort / scan sizing failed");
        need = std::max(need, need2);
        if (need > X.tmp_bytes) {
            if (X.tmp) (void)hipFree(X.tmp);
            f->device_bytes -= (int64_t)X.tmp_bytes;
            X.tmp = nullptr;
            X.tmp_bytes = 0;
            if (hipMalloc(&X.tmp, need) != hipSuccess) {
                (void)hipGetLastError();
                return fail(PR_ENOMEM, "hipMalloc failed for the export");
            }
            X.tmp_bytes = need;
            f->device_bytes += (int64_t)need;
        }
        size_t t1 = need;
        if (rocprim::radix_sort_keys(X.tmp, t1, X.leaves, X.sorted, (size_t)n_leaves, 0, 32, s) != hipSuccess)
            return fail(PR_EDEVICE, "export sort failed");
        hipLaunchKernelGGL(pr::export_lengths_kernel, dim3(grid_threads(n_leaves, 256)), dim3(256), 0, s, X.sorted,
                           n_leaves, X.depth, X.len1);
        size_t t2 = need;
        if (rocprim::inclusive_scan(X.tmp, t2, X.len1 + 1, X.offs + 1, (size_t)n_leaves, rocprim::plus<int64_t>(),
                                    s) != hipSuccess)
            return fail(PR_EDEVICE, "export scan failed");
        if (!read_small(f, &total, X.offs + n_leaves, sizeof(total), s))
            return fail(PR_EDEVICE, "export readback failed");
    }
    *num_seqs = n_leaves;
    *num_tokens = total;
    if (!tokens && !offsets) return ok();
    if (!offsets || (total > 0 && !tokens) || tokens_cap < total || seqs_cap < (int64_t)n_leaves + 1)
        return fail(PR_EINVAL, "export buffers too small: need " + std::to_string(n_leaves + 1) + " offsets and " +
                                   std::to_string(total) + " tokens");
    const int64_t zero = 0;
    if (hipMemcpyAsync(offsets, &zero, sizeof(zero), hipMemcpyHostToDevice, s) != hipSuccess)
        return fail(PR_EDEVICE, "export copy failed");
    if (n_leaves > 0) {
        if (hipMemcpyAsync(offsets + 1, X.offs + 1, (size_t)n_leaves * sizeof(int64_t), hipMemcpyDeviceToDevice,
                           s) != hipSuccess)
            return fail(PR_EDEVICE, "export copy failed");
        hipLaunchKernelGGL(pr::export_write_kernel,
                           dim3((unsigned)((n_leaves + pr::kExportWavesPerBlock - 1) / pr::kExportWavesPerBlock)),
                           dim3(wb), 0, s, F, X.sorted, n_leaves, X.depth, X.parent, offsets, tokens);
        if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "export launch failed");
    }
    if (hipStreamSynchronize(s) != hipSuccess) return fail(PR_EDEVICE, "export failed");
    return ok();
}

// Device buffers of one touch or eviction call, released on every return path.
struct CallScratch {
    std::vector<void *> bufs;
    template <typename T>
    bool get(T **p, int64_t count) {
        *p = nullptr;
        if (hipMalloc((void **)p, (size_t)std::max<int64_t>(count, 1) * sizeof(T)) != hipSuccess) {
            (void)hipGetLastError();
            *p = nullptr;
            return false;
        }
        bufs.push_back((void *)*p);
        return true;
    }
    ~CallScratch() {
        for (void *b : bufs) (void)hipFree(b);
    }
};

}  // namespace

extern "C" {

int32_t pr_abi_version(void) { return PR_ABI_VERSION; }

const char *pr_last_error(void) { return g_err.c_str(); }

pr_status pr_forest_create(int32_t num_peers, pr_forest **out) {
    if (!out) return fail(PR_EINVAL, "out is NULL");
    *out = nullptr;
    if (num_peers < 1 || num_peers > PR_MAX_PEERS)
        return fail(PR_EINVAL, "num_peers must be in [1, " + std::to_string(PR_MAX_PEERS) + "]");
    pr_forest *f = new (std::nothrow) pr_forest();
    if (!f) return fail(PR_ENOMEM, "host allocation failed");
    f->P = num_peers;
    f->W = pr::mask_words_for(num_peers);
    try {
        f->sets.resize((size_t)num_peers);
    } catch (const std::bad_alloc &) {
        delete f;
        return fail(PR_ENOMEM, "host allocation failed");
    }
    *out = f;
    return ok();
}

void pr_forest_destroy(pr_forest *f) {
    if (!f) return;
    if (f->device >= 0) {
        DeviceScope ds(f);
        (void)hipDeviceSynchronize();
        free_image(f);
        free_scratch(f);
        dfree(f, &f->d_skipped, 1);
        dfree(f, &f->d_ctr, 1);
        if (f->h_stage) (void)hipHostFree(f->h_stage);
        free_route_buffers(f);
        if (f->rs.done) (void)hipEventDestroy(f->rs.done);
    }
    delete f;
}

pr_status pr_load_snapshot(pr_forest *f, int32_t peer, const int32_t *tokens, const int64_t *offsets,
                           int64_t num_seqs) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (peer < 0 || peer >= f->P) return fail(PR_EINVAL, "peer out of range");
    if (num_seqs < 0) return fail(PR_EINVAL, "num_seqs < 0");
    if (!offsets) return fail(PR_EINVAL, "offsets is NULL");
    if (offsets[0] != 0) return fail(PR_EINVAL, "offsets[0] != 0");
    for (int64_t i = 0; i < num_seqs; i++)
        if (offsets[i + 1] < offsets[i]) return fail(PR_EINVAL, "offsets decrease at sequence " + std::to_string(i));
    if (offsets[num_seqs] > 0 && !tokens) return fail(PR_EINVAL, "tokens is NULL");
    if (num_seqs > (int64_t)INT32_MAX) return fail(PR_EINVAL, "too many sequences");
    const int64_t ntok = offsets[num_seqs];
    pr::PeerSeqs S;
    try {
        S.tokens.assign(tokens, tokens + ntok);
        S.offsets.assign(offsets, offsets + num_seqs + 1);
    } catch (const std::bad_alloc &) {
        return fail(PR_ENOMEM, "host allocation failed");
    }
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    if (f->has_dev && f->merged) {
        DeviceScope ds(f);
        if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
        pr_status r = device_load(f, peer, S);
        if (r) {
            f->broken = true;
            return r;
        }
        f->sets[(size_t)peer] = std::move(S);
        return ok();
    }
    f->sets[(size_t)peer] = std::move(S);
    f->dirty = true;
    f->host_img_valid = false;
    if (peer == f->local) f->local_load_time = f->now;
    return ok();
}

pr_status pr_merge(pr_forest *f, const int32_t *peer_of, const int32_t *tokens, int64_t num_tokens,
                   const int64_t *offsets, int64_t num_seqs, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_seqs < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (num_seqs == 0) return ok();
    if (!peer_of || !offsets) return fail(PR_EINVAL, "NULL device pointer");
    if (num_tokens > 0 && !tokens) return fail(PR_EINVAL, "tokens is NULL");
    if (num_seqs > (int64_t)INT32_MAX) return fail(PR_EINVAL, "too many sequences");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status s = commit(f);
    if (s) return s;
    s = run_merge(f, peer_of, tokens, num_tokens, offsets, num_seqs, (hipStream_t)hip_stream);
    if (s) {
        f->broken = true;
        return s;
    }
    return ok();
}

pr_status pr_load_snapshot_device(pr_forest *f, int32_t peer, const int32_t *tokens, int64_t num_tokens,
                                  const int64_t *offsets, int64_t num_seqs, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (peer < 0 || peer >= f->P) return fail(PR_EINVAL, "peer out of range");
    if (num_seqs < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (num_seqs > 0 && !offsets) return fail(PR_EINVAL, "offsets is NULL");
    if (num_tokens > 0 && !tokens) return fail(PR_EINVAL, "tokens is NULL");
    if (num_seqs > (int64_t)INT32_MAX) return fail(PR_EINVAL, "too many sequences");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status r = commit(f);
    if (r) return r;
    hipStream_t s = (hipStream_t)hip_stream;
    MergeScratch &m = f->ms;
    hipLaunchKernelGGL(pr::clear_peer_kernel, dim3(grid_threads(f->dev.n_nodes, 256)), dim3(256), 0, s,
                       dev_view(f), f->dev.n_nodes, peer);
    if (hipGetLastError() != hipSuccess) {
        f->broken = true;
        return fail(PR_EDEVICE, "snapshot kernels failed to launch");
    }
    if (num_seqs > 0) {
        if (num_seqs > m.load_seq_cap) {
            dfree(f, &m.load_peer, m.load_seq_cap);
            dfree(f, &m.load_off, m.load_seq_cap + 1);
            m.load_seq_cap = 0;
            if (!dalloc(f, &m.load_peer, num_seqs) || !dalloc(f, &m.load_off, num_seqs + 1)) {
                f->broken = true;
                return fail(PR_ENOMEM, "hipMalloc failed for the snapshot");
            }
            m.load_seq_cap = num_seqs;
        }
        hipLaunchKernelGGL(pr::fill_peer_kernel, dim3(grid_threads(num_seqs, 256)), dim3(256), 0, s, m.load_peer,
                           num_seqs, peer);
        r = run_merge(f, m.load_peer, tokens, num_tokens, offsets, num_seqs, s);
    } else {
        r = hipStreamSynchronize(s) == hipSuccess ? PR_OK : fail(PR_EDEVICE, "sync failed");
        f->merged = true;
    }
    if (r) {
        f->broken = true;
        return r;
    }
    f->sets[(size_t)peer] = pr::PeerSeqs();  // the host copy no longer describes the peer
    return ok();
}

pr_status pr_export_snapshot(pr_forest *f, int32_t peer, int32_t *tokens, int64_t tokens_cap, int64_t *offsets,
                             int64_t seqs_cap, int64_t *num_seqs, int64_t *num_tokens, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (peer < 0 || peer >= f->P) return fail(PR_EINVAL, "peer out of range");
    if (!num_seqs || !num_tokens) return fail(PR_EINVAL, "size outputs are NULL");
    if (tokens_cap < 0 || seqs_cap < 0) return fail(PR_EINVAL, "negative capacity");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status r = commit(f);
    if (r) return r;
    return export_impl(f, peer, tokens, tokens_cap, offsets, seqs_cap, num_seqs, num_tokens,
                       (hipStream_t)hip_stream);
}

pr_status pr_forest_compact(pr_forest *f, int64_t *nodes_before, int64_t *nodes_after, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status r = commit(f);
    if (r) return r;
    hipStream_t s = (hipStream_t)hip_stream;
    DevImage &d = f->dev;
    const int64_t n_old = d.n_nodes;
    const bool narrow_before = f->narrow;
    if (nodes_before) *nodes_before = n_old;
    // the new image (capacity: the old node count plus spare; labels sized below)
    DevImage nw;
    nw.cap_nodes = std::max<int64_t>(n_old + n_old / 8, 1024);
    auto free_new = [&]() {
        dfree(f, &nw.ltime, nw.cap_nodes);
        dfree(f, &nw.pool, nw.cap_pool);
        free_node_arrays(f, nw);
    };
    if (!alloc_node_arrays(f, nw, nw.cap_nodes) || (d.ltime && !dalloc(f, &nw.ltime, nw.cap_nodes))) {
        free_new();
        return fail(PR_ENOMEM, "hipMalloc failed for the compacted forest");
    }
    CallScratch X;
    int32_t *fo = nullptr, *fn = nullptr, *go = nullptr, *gn = nullptr;
    int64_t *kept1 = nullptr, *start1 = nullptr;
    if (!X.get(&fo, n_old) || !X.get(&fn, n_old) || !X.get(&go, n_old) || !X.get(&gn, n_old) ||
        !X.get(&kept1, n_old + 1) || !X.get(&start1, n_old + 1)) {
        free_new();
        return fail(PR_ENOMEM, "hipMalloc failed for the compaction");
    }
    const pr::DevForest O = dev_view(f);
    pr::DevForest N = O;
    N.nodes = nw.nodes;
    N.ntok = nw.ntok;
    N.nsep = nw.nsep;
    N.mext = nw.mext;
    N.moved = nw.moved;
    N.ltime = nw.ltime;
    N.pool = nullptr;
    N.cap_nodes = nw.cap_nodes;
    auto fail_dev = [&](const char *m) {
        free_new();
        return fail(PR_EDEVICE, m);
    };
    hipLaunchKernelGGL(pr::compact_init_kernel, dim3(1), dim3(1), 0, s, O, N, fo, fn);
    size_t need = 0;
    if (rocprim::inclusive_scan(nullptr, need, kept1, start1, (size_t)n_old + 1, rocprim::plus<int64_t>(), s) !=
        hipSuccess)
        return fail_dev("compaction scan sizing failed");
    char *tmp = nullptr;
    if (!X.get(&tmp, (int64_t)need)) {
        free_new();
        return fail(PR_ENOMEM, "hipMalloc failed for the compaction");
    }
    const int wb = 64 * pr::kCompactWavesPerBlock;
    int64_t n_front = 1, first_new = 1;
    while (n_front > 0) {
        const unsigned g = (unsigned)((n_front + pr::kCompactWavesPerBlock - 1) / pr::kCompactWavesPerBlock);
        if (hipMemsetAsync(kept1, 0, sizeof(int64_t), s) != hipSuccess) return fail_dev("compaction memset failed");
        hipLaunchKernelGGL(pr::compact_count_kernel, dim3(g), dim3(wb), 0, s, O, fo, (int32_t)n_front, kept1 + 1);
        size_t t = need;
        if (rocprim::inclusive_scan(tmp, t, kept1, start1, (size_t)n_front + 1, rocprim::plus<int64_t>(), s) !=
            hipSuccess)
            return fail_dev("compaction scan failed");
        int64_t total = 0;
        if (!read_small(f, &total, start1 + n_front, sizeof(total), s))
            return fail_dev("compaction readback failed");
        // live nodes are distinct old records: more than n_old means a malformed forest
        if (total < 0 || first_new + total > n_old) return fail_dev("compaction found more live nodes than exist");
        hipLaunchKernelGGL(pr::compact_copy_kernel, dim3(g), dim3(wb), 0, s, O, N, fo, fn, (int32_t)n_front, start1,
                           first_new, go, gn, (int64_t)0);
        if (hipGetLastError() != hipSuccess) return fail_dev("compaction launch failed");
        first_new += total;
        n_front = total;
        std::swap(fo, go);
        std::swap(fn, gn);
    }
    const int64_t n_new = first_new;
    // labels into a fresh pool, then separators
    int64_t *len1 = nullptr, *off = nullptr;
    if (!X.get(&len1, n_new + 1) || !X.get(&off, n_new + 1)) {
        free_new();
        return fail(PR_ENOMEM, "hipMalloc failed for the compaction");
    }
    hipLaunchKernelGGL(pr::compact_lab_len_kernel, dim3(grid_threads(n_new, 256)), dim3(256), 0, s, N, n_new, len1);
    size_t need2 = 0;
    if (rocprim::inclusive_scan(nullptr, need2, len1, off, (size_t)n_new + 1, rocprim::plus<int64_t>(), s) !=
        hipSuccess)
        return fail_dev("compaction scan sizing failed");
    char *tmp2 = nullptr;
    if (!X.get(&tmp2, (int64_t)need2)) {
        free_new();
        return fail(PR_ENOMEM, "hipMalloc failed for the compaction");
    }
    if (rocprim::inclusive_scan(tmp2, need2, len1, off, (size_t)n_new + 1, rocprim::plus<int64_t>(), s) != hipSuccess)
        return fail_dev("compaction scan failed");
    int64_t n_pool = 0;
    if (!read_small(f, &n_pool, off + n_new, sizeof(n_pool), s))
        return fail_dev("compaction readback failed");
    if (n_pool > (int64_t)UINT32_MAX) return fail_dev("compacted label pool exceeds 2^32 tokens");
    nw.cap_pool = std::min<int64_t>(std::max<int64_t>(n_pool + n_pool / 8, 4096), (int64_t)UINT32_MAX);
    if (!dalloc(f, &nw.pool, nw.cap_pool)) {
        free_new();
        return fail(PR_ENOMEM, "hipMalloc failed for the compacted label pool");
    }
    N.pool = nw.pool;
    N.cap_pool = nw.cap_pool;
    const unsigned gn_all = (unsigned)((n_new + pr::kCompactWavesPerBlock - 1) / pr::kCompactWavesPerBlock);
    if (hipMemsetAsync(nw.pool + n_pool, 0, (nw.cap_pool - n_pool) * sizeof(int32_t), s) != hipSuccess)
        return fail_dev("compaction memset failed");
    hipLaunchKernelGGL(pr::compact_labels_kernel, dim3(gn_all), dim3(wb), 0, s, d.pool, N, n_new, off);
    hipLaunchKernelGGL(pr::compact_sep_kernel, dim3(gn_all), dim3(wb), 0, s, N, n_new);
    if (hipGetLastError() != hipSuccess ||
        hipMemsetAsync(nw.moved, 0, nw.cap_nodes * sizeof(long long), s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return fail_dev("compaction failed");
    // install the new image once no launch on another stream still reads the old one
    if (hipDeviceSynchronize() != hipSuccess) return fail_dev("hipDeviceSynchronize failed");
    free_image(f);
    nw.n_nodes = n_new;
    nw.n_pool = n_pool;
    f->dev = nw;
    f->has_dev = true;
    f->layout_epoch++;
    pr::MergeCounters c;
    std::memset(&c, 0, sizeof(c));
    c.n_nodes = (unsigned long long)n_new;
    c.n_pool = (unsigned long long)n_pool;
    if (hipMemcpy(f->d_ctr, &c, sizeof(c), hipMemcpyHostToDevice) != hipSuccess) {
        f->broken = true;
        return fail(PR_EDEVICE, "counter upload failed");
    }
    // the 16-bit copy of the new pool (its labels are a subset of the old ones)
    f->narrow = narrow_before;
    if ((r = pool16_extend(f, 0, s))) {
        f->broken = true;
        return r;
    }
    pr::MergeCounters cc;
    if (f->narrow && !read_small(f, &cc, f->d_ctr, sizeof(cc), s)) {
        f->broken = true;
        return fail(PR_EDEVICE, "reading the narrow label check failed");
    }
    if (f->narrow) {
        if (cc.wide_tokens)
            drop_pool16(f);
        else
            f->hi17 = cc.hi_tokens > 0;  // the rebuilt pool holds only live labels
    }
    f->host_img_valid = false;  // the host image no longer mirrors the device layout
    if (nodes_after) *nodes_after = n_new;
    return ok();
}

pr_status pr_tree_tokens(pr_forest *f, int32_t peer, int64_t *tokens, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (peer < 0 || peer >= f->P) return fail(PR_EINVAL, "peer out of range");
    if (!tokens) return fail(PR_EINVAL, "tokens is NULL");
    *tokens = 0;
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status r = commit(f);
    if (r) return r;
    hipStream_t s = (hipStream_t)hip_stream;
    int32_t counts[3];
    if ((r = walk_peer(f, peer, true, s, counts))) return r;
    if (counts[2] == 0) return ok();
    CallScratch X;
    unsigned long long *d = nullptr;
    if (!X.get(&d, 1)) return fail(PR_ENOMEM, "hipMalloc failed");
    unsigned long long h = 0;
    if (hipMemsetAsync(d, 0, sizeof(h), s) != hipSuccess) return fail(PR_EDEVICE, "hipMemsetAsync failed");
    hipLaunchKernelGGL(pr::tree_tokens_kernel, dim3(grid_threads(counts[2], 256)), dim3(256), 0, s, dev_view(f),
                       f->xs.all, counts[2], d);
    if (hipGetLastError() != hipSuccess || !read_small(f, &h, d, sizeof(h), s))
        return fail(PR_EDEVICE, "tree size failed");
    *tokens = (int64_t)h;
    return ok();
}

pr_status pr_set_local_peer(pr_forest *f, int32_t peer) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (peer < -1 || peer >= f->P) return fail(PR_EINVAL, "peer out of range");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    f->local = peer;
    f->local_load_time = f->now;
    if (!f->has_dev) return ok();
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    if (hipDeviceSynchronize() != hipSuccess) return fail(PR_EDEVICE, "hipDeviceSynchronize failed");
    if (peer < 0) {
        dfree(f, &f->dev.ltime, f->dev.cap_nodes);
        return ok();
    }
    if (f->dirty) return ok();  // the next rebuild initialises the times
    pr_status r = init_local_times(f, f->now);
    if (r) {
        f->broken = true;
        return r;
    }
    return ok();
}

pr_status pr_set_time(pr_forest *f, int64_t t) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (t < f->now) return fail(PR_EINVAL, "time must not decrease");
    f->now = t;
    return ok();
}

static pr_status route_impl(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                            int64_t num_queries, const pr::Select &sel, int32_t *match_len, int32_t *chosen,
                            void *hip_stream);

pr_status pr_touch(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                   int64_t num_queries, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_queries < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (f->local < 0) return fail(PR_ESTATE, "no local peer is set");
    if (num_queries == 0) return ok();
    if (!q_offsets) return fail(PR_EINVAL, "NULL device pointer");
    if (num_tokens > 0 && !q_tokens) return fail(PR_EINVAL, "q_tokens is NULL");
    if (num_queries > (int64_t)INT32_MAX) return fail(PR_EINVAL, "too many queries");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    hipStream_t s = (hipStream_t)hip_stream;
    CallScratch X;
    int32_t *ml = nullptr, *ch = nullptr, *peer_of = nullptr, *ttok = nullptr;
    int64_t *len1 = nullptr, *toff = nullptr;
    if (!X.get(&ml, num_queries * (int64_t)f->P) || !X.get(&ch, num_queries) || !X.get(&len1, num_queries + 1) ||
        !X.get(&toff, num_queries + 1) || !X.get(&peer_of, num_queries))
        return fail(PR_ENOMEM, "hipMalloc failed for the touch");
    // 1. the matched prefix of every query in the local tree
    const pr::Select sel{nullptr, -1, 0, nullptr};
    pr_status r = route_impl(f, q_tokens, num_tokens, q_offsets, num_queries, sel, ml, ch, hip_stream);
    if (r) return r;
    // 2. gather the prefixes into one batch
    hipLaunchKernelGGL(pr::touch_lengths_kernel, dim3(grid_threads(num_queries, 256)), dim3(256), 0, s, ml, f->P,
                       f->local, num_queries, len1);
    size_t need = 0;
    if (rocprim::inclusive_scan(nullptr, need, len1, toff, (size_t)num_queries + 1, rocprim::plus<int64_t>(), s) !=
        hipSuccess)
        return fail(PR_EDEVICE, "touch scan sizing failed");
    void *tmp = nullptr;
    if (!X.get((char **)&tmp, (int64_t)need)) return fail(PR_ENOMEM, "hipMalloc failed for the touch");
    if (rocprim::inclusive_scan(tmp, need, len1, toff, (size_t)num_queries + 1, rocprim::plus<int64_t>(), s) !=
        hipSuccess)
        return fail(PR_EDEVICE, "touch scan failed");
    int64_t total = 0;
    if (!read_small(f, &total, toff + num_queries, sizeof(total), s))
        return fail(PR_EDEVICE, "touch readback failed");
    if (!X.get(&ttok, total)) return fail(PR_ENOMEM, "hipMalloc failed for the touch");
    hipLaunchKernelGGL(pr::touch_gather_kernel, dim3((unsigned)((num_queries + 3) / 4)), dim3(256), 0, s, q_tokens,
                       q_offsets, toff, num_queries, ttok);
    hipLaunchKernelGGL(pr::fill_peer_kernel, dim3(grid_threads(num_queries, 256)), dim3(256), 0, s, peer_of,
                       num_queries, f->local);
    if (hipGetLastError() != hipSuccess) return fail(PR_EDEVICE, "touch launch failed");
    // 3. inserting the prefixes into the local peer adds nothing but node
    //    boundaries where a prefix ends inside a label, and stamps the paths
    r = run_merge(f, peer_of, ttok, total, toff, num_queries, s, 1);
    if (r) {
        f->broken = true;
        return r;
    }
    return ok();
}

pr_status pr_evict_lru(pr_forest *f, int64_t max_tokens, int64_t *evicted, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (!evicted) return fail(PR_EINVAL, "evicted is NULL");
    *evicted = 0;
    if (max_tokens < 0) return fail(PR_EINVAL, "max_tokens < 0");
    if (f->local < 0) return fail(PR_ESTATE, "no local peer is set");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    if (max_tokens == 0) return ok();
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status r = commit(f);
    if (r) return r;
    if (!f->dev.ltime && (r = init_local_times(f, f->local_load_time))) return r;
    hipStream_t s = (hipStream_t)hip_stream;
    int32_t counts[3];
    if ((r = walk_peer(f, f->local, true, s, counts))) return r;
    const int64_t V = counts[2];
    if (V == 0) return ok();
    ExportScratch &W = f->xs;
    CallScratch X;
    unsigned long long *keys = nullptr, *keys_s = nullptr;
    int32_t *vals = nullptr, *vals_s = nullptr;
    int64_t *cnt1 = nullptr, *cum = nullptr;
    pr::EvictPlan *d_plan = nullptr;
    if (!X.get(&keys, V) || !X.get(&keys_s, V) || !X.get(&vals, V) || !X.get(&vals_s, V) || !X.get(&cnt1, V + 1) ||
        !X.get(&cum, V + 1) || !X.get(&d_plan, 1))
        return fail(PR_ENOMEM, "hipMalloc failed for the eviction");  // nothing changed yet
    auto fail_dev = [&](const char *m) {
        f->broken = true;
        return fail(PR_EDEVICE, m);
    };
    // once a launch has changed the forest, a failed allocation leaves it
    // partly evicted: the forest is then broken, as after a device failure
    bool mutated = false;
    auto fail_nomem = [&](const char *m) {
        if (mutated) f->broken = true;
        return fail(PR_ENOMEM, m);
    };
    const pr::DevForest F = dev_view(f);
    hipLaunchKernelGGL(pr::lru_keys_kernel, dim3(grid_threads(V, 256)), dim3(256), 0, s, F, W.all, V, keys, vals);
    size_t need = 0, need2 = 0;
    if (rocprim::radix_sort_pairs(nullptr, need, keys, keys_s, vals, vals_s, (size_t)V, 0, 64, s) != hipSuccess ||
        rocprim::inclusive_scan(nullptr, need2, cnt1, cum, (size_t)V + 1, rocprim::plus<int64_t>(), s) != hipSuccess)
        return fail_dev("eviction sort sizing failed");
    char *tmp = nullptr;
    const size_t tmp_bytes = std::max(need, need2);
    if (!X.get(&tmp, (int64_t)tmp_bytes)) return fail_nomem("hipMalloc failed for the eviction");
    size_t t1 = tmp_bytes;
    if (rocprim::radix_sort_pairs(tmp, t1, keys, keys_s, vals, vals_s, (size_t)V, 0, 64, s) != hipSuccess)
        return fail_dev("eviction sort failed");
    hipLaunchKernelGGL(pr::lru_counts_kernel, dim3(grid_threads(V, 256)), dim3(256), 0, s, F, vals_s, V, cnt1);
    size_t t2 = tmp_bytes;
    if (rocprim::inclusive_scan(tmp, t2, cnt1, cum, (size_t)V + 1, rocprim::plus<int64_t>(), s) != hipSuccess)
        return fail_dev("eviction scan failed");
    hipLaunchKernelGGL(pr::lru_plan_kernel, dim3(1), dim3(1), 0, s, keys_s, cum, V, max_tokens, d_plan);
    pr::EvictPlan plan;
    if (!read_small(f, &plan, d_plan, sizeof(plan), s))
        return fail_dev("eviction readback failed");
    const int64_t n_evict = std::min<int64_t>(max_tokens, plan.total);
    if (plan.a > 0) {
        hipLaunchKernelGGL(pr::lru_clear_sorted_kernel, dim3(grid_threads(plan.a, 256)), dim3(256), 0, s, F, vals_s,
                           plan.a);
        mutated = true;
    }
    if (plan.r > 0) {
        const int64_t a = plan.a, b = plan.b, nc = b - a;
        hipLaunchKernelGGL(pr::lru_maxdepth_kernel, dim3(grid_threads(nc, 256)), dim3(256), 0, s, vals_s, a, b,
                           W.depth, d_plan);
        if (!read_small(f, &plan, d_plan, sizeof(plan), s))
            return fail_dev("eviction readback failed");
        const int32_t maxd = plan.maxd;
        long long *hist = nullptr, *cnt = nullptr, *rev = nullptr, *S = nullptr;
        int32_t *level = nullptr, *n_level = nullptr, *rank_of = nullptr, *cut_node = nullptr, *n_cut = nullptr;
        int64_t *cut_len1 = nullptr;
        if (!X.get(&hist, maxd + 2) || !X.get(&cnt, maxd + 2) || !X.get(&rev, maxd) || !X.get(&S, maxd) ||
            !X.get(&level, nc) || !X.get(&n_level, 1) || !X.get(&rank_of, f->dev.n_nodes) ||
            !X.get(&cut_node, nc) || !X.get(&n_cut, 1) || !X.get(&cut_len1, nc + 1))
            return fail_nomem("hipMalloc failed for the eviction");
        if (hipMemsetAsync(hist, 0, (maxd + 2) * sizeof(long long), s) != hipSuccess ||
            hipMemsetAsync(n_level, 0, sizeof(int32_t), s) != hipSuccess ||
            hipMemsetAsync(n_cut, 0, sizeof(int32_t), s) != hipSuccess ||
            hipMemsetAsync(cut_len1, 0, (nc + 1) * sizeof(int64_t), s) != hipSuccess)
            return fail_dev("eviction memset failed");
        hipLaunchKernelGGL(pr::lru_hist_kernel, dim3(grid_threads(nc, 256)), dim3(256), 0, s, F, vals_s, a, b,
                           W.depth, hist);
        size_t n3 = 0, n4 = 0;
        if (rocprim::inclusive_scan(nullptr, n3, hist, cnt, (size_t)maxd + 2, rocprim::plus<long long>(), s) !=
                hipSuccess ||
            rocprim::inclusive_scan(nullptr, n4, rev, S, (size_t)maxd, rocprim::plus<long long>(), s) != hipSuccess)
            return fail_dev("eviction scan sizing failed");
        char *tmp2 = nullptr;
        const size_t tb2 = std::max(n3, n4);
        if (!X.get(&tmp2, (int64_t)tb2)) return fail_nomem("hipMalloc failed for the eviction");
        size_t u3 = tb2, u4 = tb2;
        if (rocprim::inclusive_scan(tmp2, u3, hist, cnt, (size_t)maxd + 2, rocprim::plus<long long>(), s) !=
            hipSuccess)
            return fail_dev("eviction scan failed");
        hipLaunchKernelGGL(pr::lru_reverse_kernel, dim3(grid_threads(maxd, 256)), dim3(256), 0, s, cnt, maxd, rev);
        if (rocprim::inclusive_scan(tmp2, u4, rev, S, (size_t)maxd, rocprim::plus<long long>(), s) != hipSuccess)
            return fail_dev("eviction scan failed");
        hipLaunchKernelGGL(pr::lru_depth_plan_kernel, dim3(1), dim3(1), 0, s, S, d_plan);
        hipLaunchKernelGGL(pr::lru_level_nodes_kernel, dim3(grid_threads(nc, 256)), dim3(256), 0, s, F, vals_s, a, b,
                           W.depth, d_plan, level, n_level);
        int32_t h_level = 0;
        if (!read_small(f, &h_level, n_level, sizeof(h_level), s))
            return fail_dev("eviction readback failed");
        if (h_level > nc) return fail_dev("eviction level list overflow");
        hipLaunchKernelGGL(pr::lru_rank_kernel, dim3(grid_threads(h_level, 256)), dim3(256), 0, s, F, level, h_level,
                           W.parent, W.depth, rank_of);
        hipLaunchKernelGGL(pr::lru_apply_kernel, dim3(grid_threads(nc, 256)), dim3(256), 0, s, F, vals_s, a, b,
                           W.depth, rank_of, d_plan, cut_node, cut_len1, n_cut);
        int32_t h_cut = 0;
        if (hipGetLastError() != hipSuccess ||
            !read_small(f, &h_cut, n_cut, sizeof(h_cut), s))
            return fail_dev("eviction failed");
        if (h_cut > 0) {
            int64_t *offs = nullptr, *old_len = nullptr;
            int32_t *peer_of = nullptr, *ctok = nullptr;
            if (!X.get(&offs, h_cut + 1) || !X.get(&old_len, h_cut) || !X.get(&peer_of, h_cut))
                return fail_nomem("hipMalloc failed for the eviction");
            size_t n5 = 0;
            if (rocprim::inclusive_scan(nullptr, n5, cut_len1, offs, (size_t)h_cut + 1, rocprim::plus<int64_t>(),
                                        s) != hipSuccess)
                return fail_dev("eviction scan sizing failed");
            char *tmp3 = nullptr;
            if (!X.get(&tmp3, (int64_t)n5)) return fail_nomem("hipMalloc failed for the eviction");
            if (rocprim::inclusive_scan(tmp3, n5, cut_len1, offs, (size_t)h_cut + 1, rocprim::plus<int64_t>(), s) !=
                hipSuccess)
                return fail_dev("eviction scan failed");
            int64_t total_cut = 0;
            if (!read_small(f, &total_cut, offs + h_cut, sizeof(total_cut), s))
                return fail_dev("eviction readback failed");
            if (!X.get(&ctok, total_cut)) return fail_nomem("hipMalloc failed for the eviction");
            hipLaunchKernelGGL(pr::lru_cut_paths_kernel, dim3((unsigned)((h_cut + 3) / 4)), dim3(256), 0, s, F,
                               cut_node, h_cut, offs, W.parent, W.depth, ctok);
            hipLaunchKernelGGL(pr::lru_old_len_kernel, dim3(grid_threads(h_cut, 256)), dim3(256), 0, s, F, cut_node,
                               h_cut, old_len);
            hipLaunchKernelGGL(pr::fill_peer_kernel, dim3(grid_threads(h_cut, 256)), dim3(256), 0, s, peer_of,
                               (int64_t)h_cut, f->local);
            if (hipGetLastError() != hipSuccess) return fail_dev("eviction launch failed");
            // the kept paths are held already: inserting them only splits the cut nodes
            if ((r = run_merge(f, peer_of, ctok, total_cut, offs, h_cut, s, 0))) {
                f->broken = true;
                return r;
            }
            hipLaunchKernelGGL(pr::lru_clear_lower_kernel, dim3(grid_threads(h_cut, 256)), dim3(256), 0, s,
                               dev_view(f), cut_node, h_cut, offs, W.depth, old_len, d_plan);
            if (!read_small(f, &plan, d_plan, sizeof(plan), s))
                return fail_dev("eviction readback failed");
            if (plan.bad) return fail_dev("eviction split left an unexpected structure; destroy the forest");
        }
    }
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return fail_dev("eviction failed");
    f->merged = true;
    f->sets[(size_t)f->local] = pr::PeerSeqs();  // the host copy no longer describes the local peer
    *evicted = n_evict;
    return ok();
}

static pr_status route_impl(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                            int64_t num_queries, const pr::Select &sel, int32_t *match_len, int32_t *chosen,
                            void *hip_stream) {
    if (num_queries > (int64_t)0x7fffffff * pr::kRouteWavesPerBlock) return fail(PR_EINVAL, "too many queries");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    hipStream_t st = (hipStream_t)hip_stream;
    // Under graph capture only the launch may be enqueued: no upload of a
    // changed forest (allocations, copies, waits) and no longest-first order
    // (its buffer, events and cross-stream wait); the batch goes in index
    // order, with the same results.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cap) != hipSuccess) return fail(PR_EDEVICE, "hipStreamIsCapturing failed");
    const bool capturing = cap != hipStreamCaptureStatusNone;
    if (capturing && (f->dirty || !f->has_dev))
        return fail(PR_ESTATE, "snapshots changed since the forest's last upload; route once outside graph capture");
    pr_status s = commit(f);
    if (s) return s;
    const int32_t *order = nullptr;
    if (!capturing && use_longest_first(num_queries, num_tokens) &&
        (s = route_order(f, q_offsets, num_queries, num_tokens, st, &order)))
        return s;
    const hipError_t e = launch_route_w(f, q_tokens, num_tokens, q_offsets, num_queries, sel, match_len, chosen,
                                        order, st);
    if (e != hipSuccess) return fail(PR_EDEVICE, std::string("route launch failed: ") + hipGetErrorString(e));
    if (order) {
        // the order buffers are in use until the stream passes this launch
        if (hipEventRecord(f->rs.done, st) != hipSuccess) return fail(PR_EDEVICE, "hipEventRecord failed");
        f->rs.pending = true;
    }
    return ok();
}

pr_status pr_route(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                   int64_t num_queries, int32_t *match_len, int32_t *chosen, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_queries < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (num_queries == 0) return ok();
    if (!q_offsets || !match_len || !chosen) return fail(PR_EINVAL, "NULL device pointer");
    if (num_tokens > 0 && !q_tokens) return fail(PR_EINVAL, "q_tokens is NULL");
    const pr::Select sel{nullptr, -1, 0, nullptr};
    return route_impl(f, q_tokens, num_tokens, q_offsets, num_queries, sel, match_len, chosen, hip_stream);
}

pr_status pr_route_noalloc(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                           int64_t num_queries, int32_t *match_len, int32_t *chosen, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_queries < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (num_queries > PR_NOALLOC_MAX_QUERIES)
        return fail(PR_EINVAL, "pr_route_noalloc takes at most " + std::to_string(PR_NOALLOC_MAX_QUERIES) +
                                   " queries per call");
    if (num_queries == 0) return ok();
    if (!q_offsets || !match_len || !chosen) return fail(PR_EINVAL, "NULL device pointer");
    if (num_tokens > 0 && !q_tokens) return fail(PR_EINVAL, "q_tokens is NULL");
    if (f->broken) return fail(PR_ESTATE, "an earlier device update failed; destroy the forest");
    if (f->dirty || !f->has_dev)
        return fail(PR_ESTATE, "snapshots changed since the forest's last upload; call pr_route once first");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    hipStream_t st = (hipStream_t)hip_stream;
    unsigned char *sp = nullptr;
    pr_status r = noalloc_scratch(f->device, &sp);
    if (r) return r;
    const int32_t *order = nullptr;
    if (use_longest_first(num_queries, num_tokens)) {
        int32_t *ord = reinterpret_cast<int32_t *>(sp + kNoAllocOrder);
        if ((r = launch_order(q_offsets, num_queries, num_tokens, st, sp + kNoAllocBkt,
                              reinterpret_cast<int32_t *>(sp + kNoAllocBlockcnt), ord)))
            return r;
        order = ord;
    }
    const pr::Select sel{nullptr, -1, 0, nullptr};
    const hipError_t e = launch_route_w(f, q_tokens, num_tokens, q_offsets, num_queries, sel, match_len, chosen,
                                        order, st);
    if (e != hipSuccess) return fail(PR_EDEVICE, std::string("route launch failed: ") + hipGetErrorString(e));
    return ok();
}

pr_status pr_route_select(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                          int64_t num_queries, const uint64_t *eligible, int32_t local_peer, uint32_t flags,
                          int32_t *match_len, int32_t *best, int32_t *second, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_queries < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (local_peer < -1 || local_peer >= f->P) return fail(PR_EINVAL, "local_peer out of range");
    if (flags & ~(uint32_t)PR_SELECT_PREFER_LOCAL) return fail(PR_EINVAL, "unknown flags");
    if (num_queries == 0) return ok();
    if (!q_offsets || !best) return fail(PR_EINVAL, "NULL device pointer");
    if (num_tokens > 0 && !q_tokens) return fail(PR_EINVAL, "q_tokens is NULL");
    const pr::Select sel{eligible, local_peer, (flags & PR_SELECT_PREFER_LOCAL) ? 1 : 0, second};
    return route_impl(f, q_tokens, num_tokens, q_offsets, num_queries, sel, match_len, best, hip_stream);
}

pr_status pr_forest_check(pr_forest *f) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (f->device < 0 || !f->d_skipped) return ok();
    DeviceScope ds(f);
    unsigned long long n = 0;
    if (hipDeviceSynchronize() != hipSuccess) return fail(PR_EDEVICE, "hipDeviceSynchronize failed");
    if (hipMemcpy(&n, f->d_skipped, sizeof(n), hipMemcpyDeviceToHost) != hipSuccess)
        return fail(PR_EDEVICE, "hipMemcpy failed");
    if (!n) return ok();
    if (hipMemset(f->d_skipped, 0, sizeof(n)) != hipSuccess) return fail(PR_EDEVICE, "hipMemset failed");
    return fail(PR_EINVAL, std::to_string(n) + " device inputs were skipped");
}

pr_status pr_forest_info_get(pr_forest *f, pr_forest_info *out) {
    if (!f || !out) return fail(PR_EINVAL, "NULL argument");
    std::memset(out, 0, sizeof(*out));
    out->num_peers = f->P;
    out->mask_words = f->W;
    if (f->has_dev && !f->dirty) {
        out->num_nodes = f->dev.n_nodes;
        out->pool_tokens = f->dev.n_pool;
    } else if (f->host_img_valid) {
        out->num_nodes = (int64_t)f->host_img.nodes.size();
        out->pool_tokens = (int64_t)f->host_img.pool.size();
    }
    out->device_bytes = f->device_bytes;
    out->layout_epoch = f->layout_epoch;
    out->label_token_bytes = f->narrow ? 2 : 4;
    out->label_bits = f->narrow ? (f->hi17 ? 17 : 16) : 32;
    out->merge_refusals = f->refusals;
    out->first_window_tokens = (int64_t)pr::kWave * (f->wide_window ? pr::kWideWinVectors : pr::kWinVectors);
    int64_t t = 0;
    for (const auto &S : f->sets) t += (int64_t)S.tokens.size();
    out->host_seq_tokens = t;
    return ok();
}

pr_status pr_forest_host_image(pr_forest *f, pr_image_view *out) {
    if (!f || !out) return fail(PR_EINVAL, "NULL argument");
    if (f->merged) return fail(PR_ESTATE, "the device forest holds merges; the host copies do not describe it");
    pr_status s = ensure_host_image(f);
    if (s) return s;
    const pr::HostImage &h = f->host_img;
    out->mask_words = h.W;
    out->num_nodes = (int64_t)h.nodes.size();
    out->pool_tokens = (int64_t)h.pool.size();
    out->nodes = reinterpret_cast<const int32_t *>(h.nodes.data());
    out->ntok = h.ntok.data();
    out->nsep = h.nsep.data();
    out->mext = h.mext.data();
    out->pool = h.pool.data();
    return ok();
}

}  // extern "C"
