/*
 * A plain C11 client of the router's C ABI (include/prefix_router.h), with no
 * Python or torch in between: it shows that the boundary is usable from C.
 *
 *   abi_check host    argument and state checks that run before any GPU work
 *   abi_check device  a small forest on the GPU: load, route, merge, route,
 *                     select, export, each compared with values worked out
 *                     by hand from the match definition (the longest prefix
 *                     of the query that is a prefix of some stored sequence)
 *
 * Exit status 0 on success; every failed check prints its line and the
 * library's last error.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "prefix_router.h"

static int failures = 0;

#define CHECK(cond)                                                                   \
    do {                                                                              \
        if (!(cond)) {                                                                \
            fprintf(stderr, "check failed at line %d: %s (last error: %s)\n", __LINE__, \
                    #cond, pr_last_error());                                          \
            failures++;                                                               \
        }                                                                             \
    } while (0)

static int host_checks(void) {
    pr_forest *f = NULL;
    CHECK(pr_abi_version() == PR_ABI_VERSION);
    CHECK(pr_forest_create(0, &f) == PR_EINVAL);
    CHECK(pr_forest_create(PR_MAX_PEERS + 1, &f) == PR_EINVAL);
    CHECK(pr_forest_create(3, NULL) == PR_EINVAL);
    CHECK(pr_forest_create(3, &f) == PR_OK && f != NULL);
    if (!f) return 1;
    const int32_t toks[4] = {1, 2, 3, 4};
    const int64_t good[2] = {0, 4};
    const int64_t bad_start[2] = {1, 4};
    const int64_t decreasing[3] = {0, 3, 2};
    CHECK(pr_load_snapshot(f, 3, toks, good, 1) == PR_EINVAL);      /* peer out of range */
    CHECK(pr_load_snapshot(f, -1, toks, good, 1) == PR_EINVAL);
    CHECK(pr_load_snapshot(f, 0, toks, bad_start, 1) == PR_EINVAL); /* offsets[0] != 0 */
    CHECK(pr_load_snapshot(f, 0, toks, decreasing, 2) == PR_EINVAL);
    CHECK(pr_load_snapshot(f, 0, toks, good, -1) == PR_EINVAL);
    CHECK(pr_load_snapshot(f, 0, toks, good, 1) == PR_OK);          /* host copy only, no GPU yet */
    CHECK(pr_route(NULL, NULL, 0, NULL, 1, NULL, NULL, NULL) == PR_EINVAL);
    CHECK(pr_route(f, NULL, -1, NULL, 1, NULL, NULL, NULL) == PR_EINVAL);
    CHECK(pr_route(f, NULL, 0, NULL, 0, NULL, NULL, NULL) == PR_OK); /* zero queries: no-op */
    CHECK(pr_merge(f, NULL, NULL, 0, NULL, -1, NULL) == PR_EINVAL);
    CHECK(pr_set_time(f, 5) == PR_OK);
    CHECK(pr_set_time(f, 4) == PR_EINVAL);
    CHECK(pr_set_local_peer(f, 3) == PR_EINVAL);
    CHECK(strlen(pr_last_error()) > 0);
    pr_forest_destroy(f);
    pr_forest_destroy(NULL);
    return failures;
}

/* device buffer of `bytes`, filled from src unless src is NULL */
static void *upload(const void *src, size_t bytes) {
    void *d = NULL;
    if (hipMalloc(&d, bytes ? bytes : 4) != hipSuccess) return NULL;
    if (src && bytes && hipMemcpy(d, src, bytes, hipMemcpyHostToDevice) != hipSuccess) return NULL;
    return d;
}

static int device_checks(void) {
    pr_forest *f = NULL;
    CHECK(pr_forest_create(3, &f) == PR_OK);
    if (!f) return 1;
    /* peer 0 holds [1 2 3 4 5]; peer 2 holds [1 2 9] and [7]; peer 1 is empty */
    const int32_t t0[5] = {1, 2, 3, 4, 5};
    const int64_t o0[2] = {0, 5};
    const int32_t t2[4] = {1, 2, 9, 7};
    const int64_t o2[3] = {0, 3, 4};
    CHECK(pr_load_snapshot(f, 0, t0, o0, 1) == PR_OK);
    CHECK(pr_load_snapshot(f, 2, t2, o2, 2) == PR_OK);
    /* queries: [1 2 3 4], [3 4 1 2 9], [1 2 9 7], [7 7], [] */
    const int32_t qt[15] = {1, 2, 3, 4, 3, 4, 1, 2, 9, 1, 2, 9, 7, 7, 7};
    const int64_t qo[6] = {0, 4, 9, 13, 15, 15};
    const int64_t nq = 5;
    int32_t *d_qt = upload(qt, sizeof(qt));
    int64_t *d_qo = upload(qo, sizeof(qo));
    int32_t *d_m = upload(NULL, nq * 3 * sizeof(int32_t));
    int32_t *d_c = upload(NULL, nq * sizeof(int32_t));
    int32_t *d_s = upload(NULL, nq * sizeof(int32_t));
    CHECK(d_qt && d_qo && d_m && d_c && d_s);
    if (!(d_qt && d_qo && d_m && d_c && d_s)) return 1;
    int32_t m[15], c[5], s2[5];
    CHECK(pr_route(f, d_qt, 15, d_qo, nq, d_m, d_c, NULL) == PR_OK);
    CHECK(hipDeviceSynchronize() == hipSuccess);
    CHECK(hipMemcpy(m, d_m, sizeof(m), hipMemcpyDeviceToHost) == hipSuccess && hipMemcpy(c, d_c, sizeof(c), hipMemcpyDeviceToHost) == hipSuccess);
    const int32_t m_exp[15] = {4, 0, 2, 0, 0, 0, 2, 0, 3, 0, 0, 1, 0, 0, 0};
    const int32_t c_exp[5] = {0, 0, 2, 2, 0};
    CHECK(memcmp(m, m_exp, sizeof(m)) == 0);
    CHECK(memcmp(c, c_exp, sizeof(c)) == 0);
    /* the info struct as this header lays it out: small tokens, 16-bit labels */
    pr_forest_info info;
    memset(&info, 0xAB, sizeof(info));
    CHECK(pr_forest_info_get(f, &info) == PR_OK);
    CHECK(info.num_peers == 3 && info.mask_words == 1 && info.num_nodes > 1 && info.pool_tokens > 0);
    CHECK(info.layout_epoch >= 1 && info.label_token_bytes == 2);
    CHECK(info.first_window_tokens == 128); /* the root has two children (1 and 7) */
    /* merge [3 4 1] into peer 1 and [1 2 3 4 5 6] into peer 2 */
    const int32_t mt[9] = {3, 4, 1, 1, 2, 3, 4, 5, 6};
    const int64_t mo[3] = {0, 3, 9};
    const int32_t mp[2] = {1, 2};
    int32_t *d_mt = upload(mt, sizeof(mt));
    int64_t *d_mo = upload(mo, sizeof(mo));
    int32_t *d_mp = upload(mp, sizeof(mp));
    CHECK(d_mt && d_mo && d_mp);
    if (!(d_mt && d_mo && d_mp)) return 1;
    CHECK(pr_merge(f, d_mp, d_mt, 9, d_mo, 2, NULL) == PR_OK);
    CHECK(pr_route(f, d_qt, 15, d_qo, nq, d_m, d_c, NULL) == PR_OK);
    CHECK(hipDeviceSynchronize() == hipSuccess);
    CHECK(hipMemcpy(m, d_m, sizeof(m), hipMemcpyDeviceToHost) == hipSuccess && hipMemcpy(c, d_c, sizeof(c), hipMemcpyDeviceToHost) == hipSuccess);
    const int32_t m_exp2[15] = {4, 0, 4, 0, 3, 0, 2, 0, 3, 0, 0, 1, 0, 0, 0};
    const int32_t c_exp2[5] = {0, 1, 2, 2, 0};
    CHECK(memcmp(m, m_exp2, sizeof(m)) == 0);
    CHECK(memcmp(c, c_exp2, sizeof(c)) == 0);
    /* selection: peer 2 pushed back (not eligible), peer 0 local and preferred */
    const uint64_t elig = 0x3;
    uint64_t *d_e = upload(&elig, sizeof(elig));
    CHECK(d_e != NULL);
    if (!d_e) return 1;
    CHECK(pr_route_select(f, d_qt, 15, d_qo, nq, d_e, 0, PR_SELECT_PREFER_LOCAL, NULL, d_c, d_s, NULL) == PR_OK);
    CHECK(hipDeviceSynchronize() == hipSuccess);
    CHECK(hipMemcpy(c, d_c, sizeof(c), hipMemcpyDeviceToHost) == hipSuccess && hipMemcpy(s2, d_s, sizeof(s2), hipMemcpyDeviceToHost) == hipSuccess);
    /* rows after the merge: q0 (4,0,4) -> 0 then 1; q1 (0,3,0) -> 1 then 0;
       q2 (2,0,3) -> 0 then 1; q3 (0,0,1) -> 0 then 1; q4 (0,0,0) -> 0 then 1 */
    const int32_t b_exp[5] = {0, 1, 0, 0, 0};
    const int32_t s_exp[5] = {1, 0, 1, 1, 1};
    CHECK(memcmp(c, b_exp, sizeof(c)) == 0);
    CHECK(memcmp(s2, s_exp, sizeof(s2)) == 0);
    /* export peer 2: its maximal sequences [1 2 9], [7] and [1 2 3 4 5 6] */
    int64_t n_seq = -1, n_tok = -1;
    CHECK(pr_export_snapshot(f, 2, NULL, 0, NULL, 0, &n_seq, &n_tok, NULL) == PR_OK);
    CHECK(n_seq == 3 && n_tok == 10);
    CHECK(pr_forest_check(f) == PR_OK);
    pr_forest_destroy(f);
    void *bufs[9] = {d_qt, d_qo, d_m, d_c, d_s, d_mt, d_mo, d_mp, d_e};
    for (int i = 0; i < 9; i++) (void)hipFree(bufs[i]);
    return failures;
}

int main(int argc, char **argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s host|device\n", argv[0]);
        return 2;
    }
    int r;
    if (strcmp(argv[1], "host") == 0)
        r = host_checks();
    else if (strcmp(argv[1], "device") == 0)
        r = device_checks();
    else
        return 2;
    if (r == 0) printf("abi_check %s: ok\n", argv[1]);
    return r == 0 ? 0 : 1;
}
