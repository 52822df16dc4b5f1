/*
 * prefix_oracle.c -- CPU oracle for the prefix-cache-aware router.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, calls or
 * includes this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header or table with the device
 * path.
 *
 * What it computes is the plain definition behind the paper's routing rule
 * (System Design: every node keeps one prefix tree per node and sends a request
 * to the node whose tree has the largest prefix match; Algorithm 1, the argmax
 * of PrefixMatch over all N trees including the node's own):
 *
 *   S_p        the multiset of token sequences inserted into peer p's tree:
 *              the last full snapshot loaded for p (a snapshot replaces the
 *              estimate, Section "Trie-broadcast loss") plus every sequence
 *              merged into p since (updateTrie / updateTrieEstimate).
 *   LCP(a, b)  length of the longest common prefix of two token sequences.
 *   m[q][p]    = max over s in S_p of LCP(q, s)        (0 when S_p is empty).
 *              A radix tree over S_p holds exactly the prefixes of its members
 *              as root paths, so this is the tree's longest prefix match.
 *   chosen[q]  = the smallest p with m[q][p] = max_j m[q][j]  (ties go to the
 *              lowest peer id; the paper leaves the tie rule open).
 *
 * It is deliberately a linear scan over every stored sequence: slow, and
 * checkable by eye.  Threads only split the query list into contiguous ranges.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int64_t n, cap;
    int32_t **seq;
    int64_t *len;
} or_set;

/* The local peer's tree with access times (see "local LRU tree" below). */
typedef struct {
    int32_t tok, parent, depth, alive;
    int64_t tau;
    int32_t nch, cap;
    int32_t *ch; /* children, sorted by token */
} lru_node;

typedef struct {
    lru_node *v;
    int64_t n, cap;
} lru_trie;

typedef struct {
    int32_t num_peers;
    or_set *sets;
    int32_t local; /* -1: no peer keeps access times */
    int64_t now;   /* current time, set by the caller, never decreasing */
    lru_trie lt;   /* the local peer's tree when local >= 0 */
} or_forest;

/* ---- the definition ---------------------------------------------------- */

/* Length of the longest common prefix of a[0..na) and b[0..nb). */
int64_t or_lcp(const int32_t *a, int64_t na, const int32_t *b, int64_t nb) {
    int64_t n = na < nb ? na : nb;
    int64_t i = 0;
#ifdef PLANT_LCP_OFF_BY_ONE
    while (i < n && a[i] == b[i]) i++;
    return i > 0 ? i - 1 : 0;
#else
    while (i < n && a[i] == b[i]) i++;
    return i;
#endif
}

static int64_t lru_match(const lru_trie *t, const int32_t *q, int64_t qlen);

/* PrefixMatch(q, T_p): the longest prefix of q shared with any s in S_p. */
int64_t or_prefix_match(const or_forest *f, int32_t peer, const int32_t *q, int64_t qlen) {
    if (peer == f->local) return lru_match(&f->lt, q, qlen);
    const or_set *s = &f->sets[peer];
    int64_t best = 0;
    for (int64_t i = 0; i < s->n; i++) {
        int64_t l = or_lcp(q, qlen, s->seq[i], s->len[i]);
#ifdef PLANT_MIN_NOT_MAX
        if (i == 0 || l < best) best = l;
#else
        if (l > best) best = l;
#endif
    }
    return best;
}

/* getBestNode: argmax over peers, lowest id among equal maxima. */
static int32_t argmax_lowest(const int32_t *m, int32_t P) {
    int32_t best = 0;
    for (int32_t p = 1; p < P; p++) {
#ifdef PLANT_TIE_HIGHEST
        if (m[p] >= m[best]) best = p;
#else
        if (m[p] > m[best]) best = p;
#endif
    }
    return best;
}

/* ---- sets --------------------------------------------------------------- */

or_forest *or_create(int32_t num_peers) {
    if (num_peers <= 0) return NULL;
    or_forest *f = (or_forest *)calloc(1, sizeof(or_forest));
    if (!f) return NULL;
    f->num_peers = num_peers;
    f->local = -1;
    f->sets = (or_set *)calloc((size_t)num_peers, sizeof(or_set));
    if (!f->sets) { free(f); return NULL; }
    return f;
}

static void set_clear(or_set *s) {
    for (int64_t i = 0; i < s->n; i++) free(s->seq[i]);
    free(s->seq);
    free(s->len);
    memset(s, 0, sizeof(*s));
}

static void lru_free(lru_trie *t);

void or_destroy(or_forest *f) {
    if (!f) return;
    lru_free(&f->lt);
    for (int32_t p = 0; p < f->num_peers; p++) set_clear(&f->sets[p]);
    free(f->sets);
    free(f);
}

static int set_add(or_set *s, const int32_t *tok, int64_t len) {
    if (s->n == s->cap) {
        int64_t nc = s->cap ? 2 * s->cap : 16;
        int32_t **ns = (int32_t **)realloc(s->seq, (size_t)nc * sizeof(int32_t *));
        if (!ns) return -2;
        s->seq = ns;
        int64_t *nl = (int64_t *)realloc(s->len, (size_t)nc * sizeof(int64_t));
        if (!nl) return -2;
        s->len = nl;
        s->cap = nc;
    }
    int32_t *c = (int32_t *)malloc((size_t)(len > 0 ? len : 1) * sizeof(int32_t));
    if (!c) return -2;
    if (len > 0) memcpy(c, tok, (size_t)len * sizeof(int32_t));
    s->seq[s->n] = c;
    s->len[s->n] = len;
    s->n++;
    return 0;
}

static int check_csr(const int64_t *offsets, int64_t n) {
    if (n < 0 || !offsets || offsets[0] != 0) return -1;
    for (int64_t i = 0; i < n; i++)
        if (offsets[i + 1] < offsets[i]) return -1;
    return 0;
}

/* sendTrie receive: the snapshot REPLACES peer's set. */
static int lru_reset(lru_trie *t);
static int lru_insert(lru_trie *t, const int32_t *s, int64_t len, int64_t now);

int or_load(or_forest *f, int32_t peer, const int32_t *tokens, const int64_t *offsets, int64_t n) {
    if (!f || peer < 0 || peer >= f->num_peers || check_csr(offsets, n)) return -1;
    if (peer == f->local) {
        if (lru_reset(&f->lt)) return -2;
        for (int64_t i = 0; i < n; i++)
            if (lru_insert(&f->lt, tokens + offsets[i], offsets[i + 1] - offsets[i], f->now)) return -2;
    }
#ifndef PLANT_LOAD_APPENDS
    set_clear(&f->sets[peer]);
#endif
    for (int64_t i = 0; i < n; i++) {
        int r = set_add(&f->sets[peer], tokens + offsets[i], offsets[i + 1] - offsets[i]);
        if (r) return r;
    }
    return 0;
}

/* updateTrie / updateTrieEstimate: insert sequence i into peer_of[i]'s set. */
int or_merge(or_forest *f, const int32_t *peer_of, const int32_t *tokens, const int64_t *offsets, int64_t n) {
    if (!f || check_csr(offsets, n)) return -1;
    for (int64_t i = 0; i < n; i++)
        if (peer_of[i] < 0 || peer_of[i] >= f->num_peers) return -1;
    for (int64_t i = 0; i < n; i++) {
        int32_t p = peer_of[i];
#ifdef PLANT_MERGE_WRONG_PEER
        p = (p + 1) % f->num_peers;
#endif
        int r = set_add(&f->sets[p], tokens + offsets[i], offsets[i + 1] - offsets[i]);
        if (r) return r;
        if (p == f->local && lru_insert(&f->lt, tokens + offsets[i], offsets[i + 1] - offsets[i], f->now)) return -2;
    }
    return 0;
}

int64_t or_set_size(const or_forest *f, int32_t peer) {
    if (!f || peer < 0 || peer >= f->num_peers) return -1;
    return f->sets[peer].n;
}

/* ---- batched route ------------------------------------------------------ */

typedef struct {
    const or_forest *f;
    const int32_t *qt;
    const int64_t *qo;
    int64_t lo, hi;
    int32_t *match_len, *chosen;
} route_job;

static void *route_range(void *arg) {
    route_job *j = (route_job *)arg;
    int32_t P = j->f->num_peers;
    for (int64_t q = j->lo; q < j->hi; q++) {
        const int32_t *qs = j->qt + j->qo[q];
        int64_t ql = j->qo[q + 1] - j->qo[q];
        int32_t *row = j->match_len + q * (int64_t)P;
        for (int32_t p = 0; p < P; p++) row[p] = (int32_t)or_prefix_match(j->f, p, qs, ql);
        j->chosen[q] = argmax_lowest(row, P);
    }
    return NULL;
}

/* Route queries [0, nq): match_len is [nq][P] row-major, chosen is [nq]. */
int or_route(const or_forest *f, const int32_t *q_tokens, const int64_t *q_offsets, int64_t nq,
             int32_t *match_len, int32_t *chosen, int32_t nthreads) {
    if (!f || check_csr(q_offsets, nq)) return -1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > nq) nthreads = nq > 0 ? (int32_t)nq : 1;
    route_job *jobs = (route_job *)calloc((size_t)nthreads, sizeof(route_job));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !th) { free(jobs); free(th); return -2; }
    for (int32_t t = 0; t < nthreads; t++) {
        jobs[t].f = f;
        jobs[t].qt = q_tokens;
        jobs[t].qo = q_offsets;
        jobs[t].lo = nq * t / nthreads;
        jobs[t].hi = nq * (t + 1) / nthreads;
        jobs[t].match_len = match_len;
        jobs[t].chosen = chosen;
    }
    for (int32_t t = 1; t < nthreads; t++) pthread_create(&th[t], NULL, route_range, &jobs[t]);
    route_range(&jobs[0]);
    for (int32_t t = 1; t < nthreads; t++) pthread_join(th[t], NULL);
    free(jobs);
    free(th);
    return 0;
}

/* ---- selection with push-back and failover ------------------------------
 *
 * Section "Hot specialist push-back": a node whose queue is too deep
 * advertises back-pressure, and originating nodes stop routing to it for a
 * while; the request then runs locally or on a slightly inferior peer.
 * Section "In-flight forwarded request failure": when a forward times out the
 * originating node falls back to the next-best target, which may be itself.
 *
 *   eligible[p]   nonzero if p may receive requests (zero: pushed back or
 *                 suspected failed).  NULL means every peer.  The local peer
 *                 (local >= 0) is always eligible: the originating node can
 *                 always run the request itself.
 *   order         larger m first; among equal m the local peer first when
 *                 prefer_local is set, then the lower peer id.
 *   best[q]       the first eligible peer in that order, -1 if none;
 *   second[q]     the first eligible peer after best[q], -1 if none.
 *
 * m[q][p] is the same matrix as in or_route, over every peer.
 */
static int is_eligible(const uint8_t *eligible, int32_t p, int32_t local) {
#ifdef PLANT_IGNORE_ELIGIBLE
    (void)eligible; (void)p; (void)local;
    return 1;
#else
    return p == local || !eligible || eligible[p] != 0;
#endif
}

/* Does peer a come before peer b in the selection order? */
static int comes_before(int32_t a, int32_t b, const int32_t *m, int32_t local, int32_t prefer_local) {
#ifdef PLANT_LOCAL_ALWAYS_FIRST
    if (prefer_local && a == local) return 1;
    if (prefer_local && b == local) return 0;
#endif
    if (m[a] != m[b]) return m[a] > m[b];
    if (prefer_local && a == local) return 1;
    if (prefer_local && b == local) return 0;
    return a < b;
}

typedef struct {
    const or_forest *f;
    const int32_t *qt;
    const int64_t *qo;
    int64_t lo, hi;
    const uint8_t *eligible;
    int32_t local, prefer_local;
    int32_t *match_len, *best, *second;
} select_job;

static void *select_range(void *arg) {
    select_job *j = (select_job *)arg;
    int32_t P = j->f->num_peers;
    for (int64_t q = j->lo; q < j->hi; q++) {
        const int32_t *qs = j->qt + j->qo[q];
        int64_t ql = j->qo[q + 1] - j->qo[q];
        int32_t *row = j->match_len + q * (int64_t)P;
        for (int32_t p = 0; p < P; p++) row[p] = (int32_t)or_prefix_match(j->f, p, qs, ql);
        int32_t b1 = -1, b2 = -1;
        for (int32_t p = 0; p < P; p++) {
            if (!is_eligible(j->eligible, p, j->local)) continue;
            if (b1 < 0 || comes_before(p, b1, row, j->local, j->prefer_local)) {
                b2 = b1;
                b1 = p;
            } else if (b2 < 0 || comes_before(p, b2, row, j->local, j->prefer_local)) {
                b2 = p;
            }
        }
        j->best[q] = b1;
        j->second[q] = b2;
    }
    return NULL;
}

/* Route queries [0, nq) with the selection above.  local in [-1, P). */
int or_route_select(const or_forest *f, const int32_t *q_tokens, const int64_t *q_offsets, int64_t nq,
                    const uint8_t *eligible, int32_t local, int32_t prefer_local, int32_t *match_len,
                    int32_t *best, int32_t *second, int32_t nthreads) {
    if (!f || check_csr(q_offsets, nq) || local < -1 || local >= f->num_peers) return -1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > nq) nthreads = nq > 0 ? (int32_t)nq : 1;
    select_job *jobs = (select_job *)calloc((size_t)nthreads, sizeof(select_job));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !th) { free(jobs); free(th); return -2; }
    for (int32_t t = 0; t < nthreads; t++) {
        jobs[t].f = f;
        jobs[t].qt = q_tokens;
        jobs[t].qo = q_offsets;
        jobs[t].lo = nq * t / nthreads;
        jobs[t].hi = nq * (t + 1) / nthreads;
        jobs[t].eligible = eligible;
        jobs[t].local = local;
        jobs[t].prefer_local = prefer_local;
        jobs[t].match_len = match_len;
        jobs[t].best = best;
        jobs[t].second = second;
    }
    for (int32_t t = 1; t < nthreads; t++) pthread_create(&th[t], NULL, select_range, &jobs[t]);
    select_range(&jobs[0]);
    for (int32_t t = 1; t < nthreads; t++) pthread_join(th[t], NULL);
    free(jobs);
    free(th);
    return 0;
}

/* ---- snapshot export (sendTrie) ------------------------------------------
 *
 * System Design: each node periodically broadcasts its own tree to every peer
 * (sendTrie), and a receiver replaces its estimate with it (Section
 * "Trie-broadcast loss": a broadcast is a complete snapshot).  A tree over S_p
 * is fixed by its root paths, the prefixes of S_p's members; the members that
 * are no proper prefix of another member (each once) have exactly the same
 * prefixes, so they are the smallest set of sequences that rebuilds the tree.
 * Empty sequences add no root path and are left out.
 *
 * In lexicographic order every member that has s as a proper prefix comes
 * after s, and so does every member between s and it (they all start with s),
 * so s is kept exactly when the member right after it does not start with s.
 * Output: the kept sequences in that order, as CSR.
 */
static const or_set *cmp_set;

static int cmp_seq(const void *pa, const void *pb) {
    const int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
    const int32_t *sa = cmp_set->seq[a], *sb = cmp_set->seq[b];
    const int64_t la = cmp_set->len[a], lb = cmp_set->len[b];
    const int64_t n = la < lb ? la : lb;
    for (int64_t i = 0; i < n; i++)
        if (sa[i] != sb[i]) return sa[i] < sb[i] ? -1 : 1;
    return la < lb ? -1 : (la > lb ? 1 : 0);
}

static int starts_with(const or_set *s, int64_t t, int64_t pre) {
    if (s->len[t] < s->len[pre]) return 0;
    return or_lcp(s->seq[t], s->len[t], s->seq[pre], s->len[pre]) == s->len[pre];
}

/* Returns 0, or -3 if the buffers are too small (the sizes are set either way;
   tokens / offsets may be NULL to ask for the sizes). */
static int lru_export(const lru_trie *t, int32_t *tokens, int64_t tok_cap, int64_t *offsets, int64_t seq_cap,
                      int64_t *num_seqs, int64_t *num_tokens);

int or_export(const or_forest *f, int32_t peer, int32_t *tokens, int64_t tok_cap, int64_t *offsets,
              int64_t seq_cap, int64_t *num_seqs, int64_t *num_tokens) {
    if (!f || peer < 0 || peer >= f->num_peers || !num_seqs || !num_tokens) return -1;
    if (peer == f->local) return lru_export(&f->lt, tokens, tok_cap, offsets, seq_cap, num_seqs, num_tokens);
    const or_set *s = &f->sets[peer];
    int64_t *ord = (int64_t *)malloc((size_t)(s->n > 0 ? s->n : 1) * sizeof(int64_t));
    if (!ord) return -2;
    int64_t k = 0;
    for (int64_t i = 0; i < s->n; i++)
        if (s->len[i] > 0) ord[k++] = i;
    cmp_set = s;  /* the oracle is not reentrant across threads here */
    qsort(ord, (size_t)k, sizeof(int64_t), cmp_seq);
    int64_t ns = 0, nt = 0;
    for (int64_t i = 0; i < k; i++) {
#ifndef PLANT_EXPORT_KEEPS_PREFIXES
        if (i + 1 < k && starts_with(s, ord[i + 1], ord[i])) continue;
#endif
        ns++;
        nt += s->len[ord[i]];
    }
    *num_seqs = ns;
    *num_tokens = nt;
    if (!tokens || !offsets || tok_cap < nt || seq_cap < ns + 1) {
        free(ord);
        return (tokens || offsets) ? -3 : 0;
    }
    int64_t j = 0, pos = 0;
    offsets[0] = 0;
    for (int64_t i = 0; i < k; i++) {
#ifndef PLANT_EXPORT_KEEPS_PREFIXES
        if (i + 1 < k && starts_with(s, ord[i + 1], ord[i])) continue;
#endif
        memcpy(tokens + pos, s->seq[ord[i]], (size_t)s->len[ord[i]] * sizeof(int32_t));
        pos += s->len[ord[i]];
        offsets[++j] = pos;
    }
    free(ord);
    return 0;
}

/* ---- local LRU tree --------------------------------------------------------
 *
 * Algorithm 1: when a node runs a request itself and its GPU memory is short,
 * it calls EvictLRUTrie() -- which removes one least-recently-used leaf token
 * from the local tree and returns it -- and frees that token's KV cache, until
 * the request fits.  The local peer's tree is kept here as a plain token trie
 * (one node per token; the root is the empty path) whose every path pi has an
 * access time tau(pi):
 *   - a load or merge of s into the local peer at time t sets tau = max(tau, t)
 *     on every non-empty prefix of s (a load first empties the tree);
 *   - or_touch(q) at time t does the same on the prefixes of q up to its match
 *     in the tree (the cached prefix that serving q reuses);
 *   - EvictLRUTrie removes the leaf with the smallest tau; among equal tau the
 *     deepest; among equal depth the lexicographically smallest path (the
 *     paper leaves ties open).
 * Times come from the caller (or_set_time), never decreasing, so tau never
 * grows along a path.  or_evict(n) calls EvictLRUTrie up to n times.
 */
static void lru_free(lru_trie *t) {
    for (int64_t i = 0; i < t->n; i++) free(t->v[i].ch);
    free(t->v);
    memset(t, 0, sizeof(*t));
}

static int64_t lru_new(lru_trie *t, int32_t tok, int32_t parent, int32_t depth, int64_t tau) {
    if (t->n == t->cap) {
        int64_t nc = t->cap ? 2 * t->cap : 64;
        lru_node *nv = (lru_node *)realloc(t->v, (size_t)nc * sizeof(lru_node));
        if (!nv) return -1;
        t->v = nv;
        t->cap = nc;
    }
    lru_node *x = &t->v[t->n];
    memset(x, 0, sizeof(*x));
    x->tok = tok;
    x->parent = parent;
    x->depth = depth;
    x->alive = 1;
    x->tau = tau;
    return t->n++;
}

static int lru_reset(lru_trie *t) {
    lru_free(t);
    return lru_new(t, 0, -1, 0, 0) < 0 ? -1 : 0;
}

/* child of x with token tok, or -1 */
static int32_t lru_child(const lru_trie *t, int32_t x, int32_t tok) {
    const lru_node *n = &t->v[x];
    for (int32_t i = 0; i < n->nch; i++)
        if (t->v[n->ch[i]].tok == tok) return n->ch[i];
    return -1;
}

static int lru_insert(lru_trie *t, const int32_t *s, int64_t len, int64_t now) {
    if (t->n == 0 && lru_reset(t)) return -1;
    int32_t x = 0;
    for (int64_t i = 0; i < len; i++) {
        int32_t c = lru_child(t, x, s[i]);
        if (c < 0) {
            int64_t id = lru_new(t, s[i], x, t->v[x].depth + 1, now);
            if (id < 0) return -1;
            lru_node *p = &t->v[x];
            if (p->nch == p->cap) {
                int32_t nc = p->cap ? 2 * p->cap : 4;
                int32_t *nch = (int32_t *)realloc(p->ch, (size_t)nc * sizeof(int32_t));
                if (!nch) return -1;
                p->ch = nch;
                p->cap = nc;
            }
            int32_t k = p->nch++;
            while (k > 0 && t->v[p->ch[k - 1]].tok > s[i]) {  /* keep children sorted */
                p->ch[k] = p->ch[k - 1];
                k--;
            }
            p->ch[k] = (int32_t)id;
            c = (int32_t)id;
        }
        if (t->v[c].tau < now) t->v[c].tau = now;
        x = c;
    }
    return 0;
}

static int64_t lru_match(const lru_trie *t, const int32_t *q, int64_t qlen) {
    if (t->n == 0) return 0;
    int32_t x = 0;
    int64_t m = 0;
    while (m < qlen) {
        int32_t c = lru_child(t, x, q[m]);
        if (c < 0) break;
        x = c;
        m++;
    }
    return m;
}

/* fills path[0 .. depth) with the tokens from the root to x */
static void lru_path(const lru_trie *t, int32_t x, int32_t *path) {
    for (int32_t d = t->v[x].depth; d > 0; d--) {
        path[d - 1] = t->v[x].tok;
        x = t->v[x].parent;
    }
}

/* does leaf a come before leaf b in the eviction order? */
static int lru_before(const lru_trie *t, int32_t a, int32_t b, int32_t *pa, int32_t *pb) {
    const lru_node *x = &t->v[a], *y = &t->v[b];
#ifdef PLANT_EVICT_MRU
    if (x->tau != y->tau) return x->tau > y->tau;
#else
    if (x->tau != y->tau) return x->tau < y->tau;
#endif
    if (x->depth != y->depth) return x->depth > y->depth;
    lru_path(t, a, pa);
    lru_path(t, b, pb);
    for (int32_t i = 0; i < x->depth; i++)
        if (pa[i] != pb[i]) return pa[i] < pb[i];
    return a < b;
}

static int32_t lru_max_depth(const lru_trie *t) {
    int32_t d = 0;
    for (int64_t i = 0; i < t->n; i++)
        if (t->v[i].alive && t->v[i].depth > d) d = t->v[i].depth;
    return d;
}

/* EvictLRUTrie, n times (or until the tree is empty). */
static int64_t lru_evict(lru_trie *t, int64_t n) {
    if (t->n == 0) return 0;
    int32_t D = lru_max_depth(t);
    int32_t *pa = (int32_t *)malloc((size_t)(D > 0 ? D : 1) * sizeof(int32_t));
    int32_t *pb = (int32_t *)malloc((size_t)(D > 0 ? D : 1) * sizeof(int32_t));
    if (!pa || !pb) { free(pa); free(pb); return -1; }
    int64_t done = 0;
    for (; done < n; done++) {
        int32_t best = -1;
        for (int64_t i = 1; i < t->n; i++) {
            const lru_node *x = &t->v[i];
            if (!x->alive || x->nch > 0) continue;  /* leaves only */
            if (best < 0 || lru_before(t, (int32_t)i, best, pa, pb)) best = (int32_t)i;
        }
        if (best < 0) break;
        lru_node *x = &t->v[best], *p = &t->v[x->parent];
        x->alive = 0;
        int32_t k = 0;
        while (p->ch[k] != best) k++;
        for (; k + 1 < p->nch; k++) p->ch[k] = p->ch[k + 1];
        p->nch--;
    }
    free(pa);
    free(pb);
    return done;
}

/* leaves in lexicographic order (depth-first over sorted children) */
static void lru_collect(const lru_trie *t, int32_t x, int32_t *path, int32_t *tokens, int64_t *offsets,
                        int64_t *ns, int64_t *nt, int fill) {
    const lru_node *n = &t->v[x];
    if (x != 0) path[n->depth - 1] = n->tok;
    if (n->nch == 0) {
        if (x == 0) return;
        if (fill) {
            memcpy(tokens + *nt, path, (size_t)n->depth * sizeof(int32_t));
            offsets[*ns + 1] = *nt + n->depth;
        }
        (*ns)++;
        *nt += n->depth;
        return;
    }
    for (int32_t i = 0; i < n->nch; i++) lru_collect(t, n->ch[i], path, tokens, offsets, ns, nt, fill);
}

static int lru_export(const lru_trie *t, int32_t *tokens, int64_t tok_cap, int64_t *offsets, int64_t seq_cap,
                      int64_t *num_seqs, int64_t *num_tokens) {
    *num_seqs = 0;
    *num_tokens = 0;
    if (t->n == 0) {
        if (offsets && seq_cap >= 1) offsets[0] = 0;
        return 0;
    }
    int32_t D = lru_max_depth(t);
    int32_t *path = (int32_t *)malloc((size_t)(D > 0 ? D : 1) * sizeof(int32_t));
    if (!path) return -2;
    int64_t ns = 0, nt = 0;
    lru_collect(t, 0, path, NULL, NULL, &ns, &nt, 0);
    *num_seqs = ns;
    *num_tokens = nt;
    if (!tokens || !offsets || tok_cap < nt || seq_cap < ns + 1) {
        free(path);
        return (tokens || offsets) ? -3 : 0;
    }
    offsets[0] = 0;
    ns = 0;
    nt = 0;
    lru_collect(t, 0, path, tokens, offsets, &ns, &nt, 1);
    free(path);
    return 0;
}

/* Make peer the local one (its tree keeps access times; -1: none).  Its
   current sequences get the current time. */
int or_set_local(or_forest *f, int32_t peer) {
    if (!f || peer < -1 || peer >= f->num_peers) return -1;
    lru_free(&f->lt);
    f->local = peer;
    if (peer < 0) return 0;
    if (lru_reset(&f->lt)) return -2;
    const or_set *s = &f->sets[peer];
    for (int64_t i = 0; i < s->n; i++)
        if (lru_insert(&f->lt, s->seq[i], s->len[i], f->now)) return -2;
    return 0;
}

int or_set_time(or_forest *f, int64_t t) {
    if (!f || t < f->now) return -1;
    f->now = t;
    return 0;
}

/* Serving the queries at the current time: their matched prefixes in the
   local tree become the most recently used. */
int or_touch(or_forest *f, const int32_t *q_tokens, const int64_t *q_offsets, int64_t nq) {
    if (!f || f->local < 0 || check_csr(q_offsets, nq)) return -1;
    lru_trie *t = &f->lt;
    if (t->n == 0) return 0;
    for (int64_t q = 0; q < nq; q++) {
        const int32_t *s = q_tokens + q_offsets[q];
        const int64_t len = q_offsets[q + 1] - q_offsets[q];
        int32_t x = 0;
        for (int64_t i = 0; i < len; i++) {
            int32_t c = lru_child(t, x, s[i]);
            if (c < 0) break;
#ifndef PLANT_TOUCH_NOTHING
            if (t->v[c].tau < f->now) t->v[c].tau = f->now;
#endif
            x = c;
        }
    }
    return 0;
}

/* Evict up to n tokens from the local tree; returns the number evicted. */
int64_t or_evict(or_forest *f, int64_t n) {
    if (!f || f->local < 0 || n < 0) return -1;
    return lru_evict(&f->lt, n);
}

/* ---- tree size -------------------------------------------------------------
 * Tokens a peer's tree holds: the number of distinct non-empty prefixes of
 * its set (one KV-cache entry each).  For the local peer, the live nodes of
 * its token trie; otherwise, in lexicographic order every member adds the
 * tokens it does not share with the member before it.
 */
int64_t or_tree_tokens(const or_forest *f, int32_t peer) {
    if (!f || peer < 0 || peer >= f->num_peers) return -1;
    if (peer == f->local) {
        int64_t n = 0;
        for (int64_t i = 1; i < f->lt.n; i++) n += f->lt.v[i].alive;
        return n;
    }
    const or_set *s = &f->sets[peer];
    int64_t *ord = (int64_t *)malloc((size_t)(s->n > 0 ? s->n : 1) * sizeof(int64_t));
    if (!ord) return -2;
    for (int64_t i = 0; i < s->n; i++) ord[i] = i;
    cmp_set = s;
    qsort(ord, (size_t)s->n, sizeof(int64_t), cmp_seq);
    int64_t total = 0;
    for (int64_t i = 0; i < s->n; i++) {
        int64_t shared = i == 0 ? 0 : or_lcp(s->seq[ord[i]], s->len[ord[i]], s->seq[ord[i - 1]], s->len[ord[i - 1]]);
        total += s->len[ord[i]] - shared;
    }
    free(ord);
    return total;
}
