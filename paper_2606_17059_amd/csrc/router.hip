// router.hip -- C ABI of the gfx950 prefix-cache-aware router (see
// include/prefix_router.h for the contract of every entry point).
//
// Host side: per-peer snapshot copies, the union-forest build, device memory,
// argument checks and launches.  Device side: route_kernels.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "forest_host.h"
#include "forest_layout.h"
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

struct DevImage {
    Node *nodes = nullptr;
    int32_t *ntok = nullptr;
    uint64_t *mext = nullptr;
    int32_t *pool = nullptr;
    int64_t n_nodes = 0, n_pool = 0;
    int64_t bytes = 0;
};

}  // namespace

struct pr_forest {
    int32_t P = 0;
    int32_t W = 1;
    int device = -1;
    std::vector<pr::PeerSeqs> sets;
    bool dirty = true;  // host sets changed since the device image was built
    pr::HostImage host_img;
    bool host_img_valid = false;
    DevImage dev;
    bool has_dev = false;
    unsigned long long *d_skipped = nullptr;  // inputs skipped by device calls
};

namespace {

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

void free_image(DevImage *d) {
    (void)hipFree(d->nodes);
    (void)hipFree(d->ntok);
    (void)hipFree(d->mext);
    (void)hipFree(d->pool);
    *d = DevImage();
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

template <typename T>
pr_status upload(T **dst, const std::vector<T> &src, int64_t *bytes) {
    const size_t n = std::max<size_t>(src.size(), 1) * sizeof(T);
    if (hipMalloc((void **)dst, n) != hipSuccess) {
        (void)hipGetLastError();
        return fail(PR_ENOMEM, "hipMalloc failed for the forest image");
    }
    *bytes += (int64_t)n;
    if (!src.empty() && hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice) != hipSuccess)
        return fail(PR_EDEVICE, "hipMemcpy of the forest image failed");
    return PR_OK;
}

// Rebuild and upload the device image if snapshots changed since the last one.
pr_status commit(pr_forest *f) {
    if (!f->dirty && f->has_dev) return PR_OK;
    pr_status s = ensure_host_image(f);
    if (s) return s;
    if (!f->d_skipped) {
        if (hipMalloc((void **)&f->d_skipped, sizeof(unsigned long long)) != hipSuccess)
            return fail(PR_ENOMEM, "hipMalloc failed");
        if (hipMemset(f->d_skipped, 0, sizeof(unsigned long long)) != hipSuccess)
            return fail(PR_EDEVICE, "hipMemset failed");
    }
    // earlier launches may still read the old image
    if (f->has_dev && hipDeviceSynchronize() != hipSuccess) return fail(PR_EDEVICE, "hipDeviceSynchronize failed");
    DevImage d;
    const pr::HostImage &h = f->host_img;
    if ((s = upload(&d.nodes, h.nodes, &d.bytes)) || (s = upload(&d.ntok, h.ntok, &d.bytes)) ||
        (s = upload(&d.mext, h.mext, &d.bytes)) || (s = upload(&d.pool, h.pool, &d.bytes))) {
        free_image(&d);
        return s;
    }
    d.n_nodes = (int64_t)h.nodes.size();
    d.n_pool = (int64_t)h.pool.size();
    if (f->has_dev) free_image(&f->dev);
    f->dev = d;
    f->has_dev = true;
    f->dirty = false;
    // the device image is the state of record now; drop the host copy of it
    f->host_img = pr::HostImage();
    f->host_img_valid = false;
    return PR_OK;
}

template <int W>
hipError_t launch_route(const pr_forest *f, const int32_t *qt, int64_t ntok, const int64_t *qo, int64_t nq,
                        int32_t *ml, int32_t *ch, hipStream_t s) {
    const int64_t blocks = (nq + pr::kRouteWavesPerBlock - 1) / pr::kRouteWavesPerBlock;
    hipLaunchKernelGGL(pr::route_kernel<W>, dim3((unsigned)blocks), dim3(pr::kWave * pr::kRouteWavesPerBlock), 0, s,
                       f->dev.nodes, f->dev.ntok, f->dev.mext, f->dev.pool, qt, ntok, qo, nq, f->P, ml, ch);
    return hipGetLastError();
}

}  // namespace

extern "C" {

int32_t pr_abi_version(void) { return 1; }

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
        if (f->has_dev) free_image(&f->dev);
        (void)hipFree(f->d_skipped);
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
    const int64_t ntok = offsets[num_seqs];
    if (ntok > 0 && !tokens) return fail(PR_EINVAL, "tokens is NULL");
    pr::PeerSeqs S;
    try {
        S.tokens.assign(tokens, tokens + ntok);
        S.offsets.assign(offsets, offsets + num_seqs + 1);
    } catch (const std::bad_alloc &) {
        return fail(PR_ENOMEM, "host allocation failed");
    }
    f->sets[(size_t)peer] = std::move(S);
    f->dirty = true;
    f->host_img_valid = false;
    return ok();
}

pr_status pr_merge(pr_forest *f, const int32_t *peer_of, const int32_t *tokens, int64_t num_tokens,
                   const int64_t *offsets, int64_t num_seqs, void *hip_stream) {
    (void)peer_of;
    (void)tokens;
    (void)num_tokens;
    (void)offsets;
    (void)hip_stream;
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_seqs < 0) return fail(PR_EINVAL, "num_seqs < 0");
    return fail(PR_ESTATE, "pr_merge is not available in this build");
}

pr_status pr_route(pr_forest *f, const int32_t *q_tokens, int64_t num_tokens, const int64_t *q_offsets,
                   int64_t num_queries, int32_t *match_len, int32_t *chosen, void *hip_stream) {
    if (!f) return fail(PR_EINVAL, "forest is NULL");
    if (num_queries < 0 || num_tokens < 0) return fail(PR_EINVAL, "negative count");
    if (num_queries == 0) return ok();
    if (!q_offsets || !match_len || !chosen) return fail(PR_EINVAL, "NULL device pointer");
    if (num_tokens > 0 && !q_tokens) return fail(PR_EINVAL, "q_tokens is NULL");
    if (num_queries > (int64_t)0x7fffffff * pr::kRouteWavesPerBlock) return fail(PR_EINVAL, "too many queries");
    DeviceScope ds(f);
    if (!ds.ok()) return fail(PR_EDEVICE, "cannot select the forest's device");
    pr_status s = commit(f);
    if (s) return s;
    hipStream_t st = (hipStream_t)hip_stream;
    hipError_t e;
    switch (f->W) {
        case 1: e = launch_route<1>(f, q_tokens, num_tokens, q_offsets, num_queries, match_len, chosen, st); break;
        case 2: e = launch_route<2>(f, q_tokens, num_tokens, q_offsets, num_queries, match_len, chosen, st); break;
        case 4: e = launch_route<4>(f, q_tokens, num_tokens, q_offsets, num_queries, match_len, chosen, st); break;
        case 8: e = launch_route<8>(f, q_tokens, num_tokens, q_offsets, num_queries, match_len, chosen, st); break;
        default: e = launch_route<16>(f, q_tokens, num_tokens, q_offsets, num_queries, match_len, chosen, st); break;
    }
    if (e != hipSuccess) return fail(PR_EDEVICE, std::string("route launch failed: ") + hipGetErrorString(e));
    return ok();
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
    out->device_bytes = f->has_dev ? f->dev.bytes : 0;
    int64_t t = 0;
    for (const auto &S : f->sets) t += (int64_t)S.tokens.size();
    out->host_seq_tokens = t;
    return ok();
}

pr_status pr_forest_host_image(pr_forest *f, pr_image_view *out) {
    if (!f || !out) return fail(PR_EINVAL, "NULL argument");
    pr_status s = ensure_host_image(f);
    if (s) return s;
    const pr::HostImage &h = f->host_img;
    out->mask_words = h.W;
    out->num_nodes = (int64_t)h.nodes.size();
    out->pool_tokens = (int64_t)h.pool.size();
    out->nodes = reinterpret_cast<const int32_t *>(h.nodes.data());
    out->ntok = h.ntok.data();
    out->mext = h.mext.data();
    out->pool = h.pool.data();
    return ok();
}

}  // extern "C"
