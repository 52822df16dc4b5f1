/*
 * radix_oracle.c -- second CPU oracle: one radix tree per peer, as the paper
 * keeps them.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, calls or
 * includes this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header or table with the device
 * path, and none with prefix_oracle.c either: the two oracles are independent
 * formulations and the tests compare them.
 *
 * The paper (System Design) gives every node one radix tree per peer: its own
 * exact tree and one estimate per other node, each holding the prefixes of
 * the requests inserted into it (updateTrie / updateTrieEstimate) or of the
 * last full snapshot received (sendTrie; Section "Trie-broadcast loss": a
 * snapshot replaces the estimate).  getBestNode walks each tree with the
 * request (PrefixMatch, the largest prefix match) and Algorithm 1 picks the
 * argmax over all N trees.  This file does exactly that, step by step:
 *
 *   node      (label, children keyed by their first label token, end count);
 *             the root has the empty label.  A label is a span of the tree's
 *             token arena.
 *   INSERT(T, s)   x <- root, i <- 0; while i < |s|: the child c of x whose
 *             label starts with s[i]; none: hang a new leaf with label s[i:]
 *             and stop; l <- LCP(label(c), s[i:]); l = |label(c)|: descend
 *             (x <- c, i += l); otherwise split c: a new node with label
 *             label(c)[:l] takes c's place under x and gets c, whose label
 *             becomes label(c)[l:], as its only child; descend into the new
 *             node.  At i = |s| the node's end count grows.
 *   MATCH(T, q)    x <- root, m <- 0; while m < |q|: the child c of x whose
 *             label starts with q[m], else stop; l <- LCP(label(c), q[m:]);
 *             m += l; l < |label(c)| stops; else x <- c.  Returns m.
 *   ROUTE(q)  m[p] = MATCH(T_p, q) for every peer; chosen = the lowest p with
 *             the largest m[p] (ties go to the lowest peer id; the paper
 *             leaves the tie rule open).
 *   LOAD(p, S)     T_p <- empty tree, then INSERT every member of S.
 *   MERGE(list)    INSERT each (p, s) into T_p, in the given order.
 *
 * split_block B > 0 (the long-context workload's "edges split at 16-token
 * blocks") additionally keeps a node at every depth that is a multiple of B on
 * every stored path: a new leaf is hung as a chain of nodes cut at those
 * depths.  Splits only ever add node boundaries, so no edge label then
 * straddles a multiple of B.  Match lengths do not depend on B.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t tok; /* first label token of the child */
    int32_t id;  /* node id of the child */
} rx_edge;

typedef struct {
    int64_t lab;   /* label: tok[lab .. lab + len) of the tree's arena */
    int32_t len;   /* 0 only for the root */
    int32_t depth; /* tokens from the root through this node's label */
    int64_t ends;  /* inserted sequences that end exactly here */
    int32_t nch, cap;
    rx_edge *ch;   /* children, sorted by first label token */
} rx_node;

typedef struct {
    rx_node *v;
    int64_t n, cap;
    int32_t *tok; /* label arena: labels of leaves, appended as they are hung */
    int64_t ntok, tcap;
} rx_tree;

typedef struct {
    int32_t num_peers;
    int32_t split_block;
    rx_tree *t;
} rx_forest;

/* ---- one tree ----------------------------------------------------------- */

static void tree_free(rx_tree *t) {
    for (int64_t i = 0; i < t->n; i++) free(t->v[i].ch);
    free(t->v);
    free(t->tok);
    memset(t, 0, sizeof(*t));
}

static int64_t new_node(rx_tree *t, int64_t lab, int32_t len, int32_t depth) {
    if (t->n == t->cap) {
        int64_t nc = t->cap ? 2 * t->cap : 64;
        rx_node *nv = (rx_node *)realloc(t->v, (size_t)nc * sizeof(rx_node));
        if (!nv) return -1;
        t->v = nv;
        t->cap = nc;
    }
    rx_node *x = &t->v[t->n];
    memset(x, 0, sizeof(*x));
    x->lab = lab;
    x->len = len;
    x->depth = depth;
    return t->n++;
}

static int tree_reset(rx_tree *t) {
    tree_free(t);
    return new_node(t, 0, 0, 0) < 0 ? -2 : 0; /* the root */
}

/* Append n tokens to the arena; returns their offset, or -1. */
static int64_t arena_put(rx_tree *t, const int32_t *s, int64_t n) {
    if (t->ntok + n > t->tcap) {
        int64_t nc = t->tcap ? t->tcap : 1024;
        while (nc < t->ntok + n) nc *= 2;
        int32_t *nt = (int32_t *)realloc(t->tok, (size_t)nc * sizeof(int32_t));
        if (!nt) return -1;
        t->tok = nt;
        t->tcap = nc;
    }
    int64_t at = t->ntok;
    if (n > 0) memcpy(t->tok + at, s, (size_t)n * sizeof(int32_t));
    t->ntok += n;
    return at;
}

/* Position of the child of x whose first label token is tok (binary search
 * over the sorted keys); *found tells whether it exists, and the position is
 * where it would be inserted otherwise. */
static int32_t child_pos(const rx_node *x, int32_t tok, int *found) {
    int32_t lo = 0, hi = x->nch;
    while (lo < hi) {
        int32_t mid = lo + (hi - lo) / 2;
        if (x->ch[mid].tok < tok)
            lo = mid + 1;
        else
            hi = mid;
    }
#ifdef PLANT_RX_CHILD_LOWER_BOUND
    *found = lo < x->nch; /* takes the next larger key as a match */
#else
    *found = lo < x->nch && x->ch[lo].tok == tok;
#endif
    return lo;
}

static int add_child(rx_tree *t, int64_t x, int32_t pos, int32_t tok, int32_t id) {
    rx_node *p = &t->v[x];
    if (p->nch == p->cap) {
        int32_t nc = p->cap ? 2 * p->cap : 2;
        rx_edge *ne = (rx_edge *)realloc(p->ch, (size_t)nc * sizeof(rx_edge));
        if (!ne) return -2;
        p->ch = ne;
        p->cap = nc;
    }
    memmove(p->ch + pos + 1, p->ch + pos, (size_t)(p->nch - pos) * sizeof(rx_edge));
    p->ch[pos].tok = tok;
    p->ch[pos].id = id;
    p->nch++;
    return 0;
}

static int64_t lcp(const int32_t *a, const int32_t *b, int64_t n) {
    int64_t i = 0;
    while (i < n && a[i] == b[i]) i++;
    return i;
}

/* Hang s[0..n) (which starts at depth d) under x as a new leaf, or, with
 * split_block B, as a chain of nodes cut at the multiples of B.  Returns the
 * last node of the chain, or -1. */
static int64_t hang_leaf(rx_tree *t, int64_t x, int32_t pos, const int32_t *s, int64_t n, int32_t d, int32_t B) {
#ifdef PLANT_RX_LEAF_DROPS_LAST
    if (n > 1) n--; /* the new leaf loses the sequence's last token */
#endif
    const int64_t at0 = arena_put(t, s, n);
    if (at0 < 0) return -1;
    int64_t done = 0;
    while (done < n) {
        int64_t piece = n - done;
        if (B > 0) {
            const int64_t to_cut = B - (int64_t)(d % B); /* tokens up to the next multiple of B */
            if (piece > to_cut) piece = to_cut;
        }
        const int64_t c = new_node(t, at0 + done, (int32_t)piece, (int32_t)(d + piece));
        if (c < 0) return -1;
        if (add_child(t, x, pos, s[done], (int32_t)c)) return -1;
        x = c;
        pos = 0;
        done += piece;
        d += (int32_t)piece;
    }
    return x;
}

/* INSERT(T, s) as described at the top of the file. */
static int tree_insert(rx_tree *t, const int32_t *s, int64_t len, int32_t B) {
    int64_t x = 0, i = 0;
    for (;;) {
        if (i == len) {
            t->v[x].ends++;
            return 0;
        }
        int found;
        const int32_t pos = child_pos(&t->v[x], s[i], &found);
        if (!found) {
            int64_t leaf = hang_leaf(t, x, pos, s + i, len - i, t->v[x].depth, B);
            if (leaf < 0) return -2;
            t->v[leaf].ends++;
            return 0;
        }
        const int64_t c = t->v[x].ch[pos].id;
        const rx_node cn = t->v[c];
        int64_t n = len - i < cn.len ? len - i : cn.len;
        const int64_t l = lcp(t->tok + cn.lab, s + i, n);
        if (l == 0) return -3; /* a child keyed by s[i] must start with s[i]: the tree is corrupt */
        if (l == cn.len) {
            x = c;
            i += l;
            continue;
        }
        /* split: mid takes c's place under x, with c below it */
        const int64_t mid = new_node(t, cn.lab, (int32_t)l, cn.depth - cn.len + (int32_t)l);
        if (mid < 0) return -2;
        rx_node *cp = &t->v[c];
#ifndef PLANT_RX_SPLIT_NO_ADVANCE
        cp->lab += l;
#endif
        cp->len -= (int32_t)l;
        t->v[x].ch[pos].id = (int32_t)mid; /* same first token: the order holds */
        if (add_child(t, mid, 0, t->tok[t->v[c].lab], (int32_t)c)) return -2;
        x = mid;
        i += l;
    }
}

/* MATCH(T, q) as described at the top of the file. */
static int64_t tree_match(const rx_tree *t, const int32_t *q, int64_t qlen) {
    int64_t x = 0, m = 0;
    while (m < qlen) {
        int found;
        const int32_t pos = child_pos(&t->v[x], q[m], &found);
        if (!found) break;
        const rx_node *c = &t->v[t->v[x].ch[pos].id];
        const int64_t n = qlen - m < c->len ? qlen - m : c->len;
        const int64_t l = lcp(t->tok + c->lab, q + m, n);
        m += l;
#ifndef PLANT_RX_MATCH_PAST_PARTIAL /* the plant walks on below a partly matched label */
        if (l < c->len) break;
#endif
        x = t->v[x].ch[pos].id;
    }
    return m;
}

/* ---- the forest --------------------------------------------------------- */

static int check_csr(const int64_t *offsets, int64_t n) {
    if (n < 0 || !offsets || offsets[0] != 0) return -1;
    for (int64_t i = 0; i < n; i++)
        if (offsets[i + 1] < offsets[i]) return -1;
    return 0;
}

rx_forest *rx_create(int32_t num_peers, int32_t split_block) {
    if (num_peers <= 0 || split_block < 0) return NULL;
    rx_forest *f = (rx_forest *)calloc(1, sizeof(rx_forest));
    if (!f) return NULL;
    f->num_peers = num_peers;
    f->split_block = split_block;
    f->t = (rx_tree *)calloc((size_t)num_peers, sizeof(rx_tree));
    if (!f->t) {
        free(f);
        return NULL;
    }
    for (int32_t p = 0; p < num_peers; p++)
        if (tree_reset(&f->t[p])) {
            for (int32_t k = 0; k <= p; k++) tree_free(&f->t[k]);
            free(f->t);
            free(f);
            return NULL;
        }
    return f;
}

void rx_destroy(rx_forest *f) {
    if (!f) return;
    for (int32_t p = 0; p < f->num_peers; p++) tree_free(&f->t[p]);
    free(f->t);
    free(f);
}

/* LOAD: sendTrie received, the snapshot replaces peer's tree. */
int rx_load(rx_forest *f, int32_t peer, const int32_t *tokens, const int64_t *offsets, int64_t n) {
    if (!f || peer < 0 || peer >= f->num_peers || check_csr(offsets, n)) return -1;
#ifndef PLANT_RX_LOAD_APPENDS
    if (tree_reset(&f->t[peer])) return -2;
#endif
    for (int64_t i = 0; i < n; i++)
        if (tree_insert(&f->t[peer], tokens + offsets[i], offsets[i + 1] - offsets[i], f->split_block)) return -2;
    return 0;
}

/* MERGE: updateTrie / updateTrieEstimate, sequence i into peer_of[i]'s tree. */
int rx_merge(rx_forest *f, const int32_t *peer_of, const int32_t *tokens, const int64_t *offsets, int64_t n) {
    if (!f || check_csr(offsets, n)) return -1;
    for (int64_t i = 0; i < n; i++)
        if (peer_of[i] < 0 || peer_of[i] >= f->num_peers) return -1;
    for (int64_t i = 0; i < n; i++)
        if (tree_insert(&f->t[peer_of[i]], tokens + offsets[i], offsets[i + 1] - offsets[i], f->split_block))
            return -2;
    return 0;
}

int64_t rx_match(const rx_forest *f, int32_t peer, const int32_t *q, int64_t qlen) {
    if (!f || peer < 0 || peer >= f->num_peers || qlen < 0) return -1;
    return tree_match(&f->t[peer], q, qlen);
}

typedef struct {
    const rx_forest *f;
    const int32_t *qt;
    const int64_t *qo;
    int64_t lo, hi;
    int32_t *match_len, *chosen;
} rx_job;

static void *route_range(void *arg) {
    rx_job *j = (rx_job *)arg;
    const int32_t P = j->f->num_peers;
    for (int64_t q = j->lo; q < j->hi; q++) {
        const int32_t *qs = j->qt + j->qo[q];
        const int64_t ql = j->qo[q + 1] - j->qo[q];
        int32_t *row = j->match_len + q * (int64_t)P;
        int32_t best = 0;
        for (int32_t p = 0; p < P; p++) {
            row[p] = (int32_t)tree_match(&j->f->t[p], qs, ql);
            if (row[p] > row[best]) best = p;
        }
        j->chosen[q] = best;
    }
    return NULL;
}

/* ROUTE for queries [0, nq): match_len is [nq][P] row-major, chosen is [nq].
 * Threads split the queries into contiguous ranges. */
int rx_route(const rx_forest *f, const int32_t *q_tokens, const int64_t *q_offsets, int64_t nq, int32_t *match_len,
             int32_t *chosen, int32_t nthreads) {
    if (!f || check_csr(q_offsets, nq)) return -1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > nq) nthreads = nq > 0 ? (int32_t)nq : 1;
    rx_job *jobs = (rx_job *)calloc((size_t)nthreads, sizeof(rx_job));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !th) {
        free(jobs);
        free(th);
        return -2;
    }
    for (int32_t t = 0; t < nthreads; t++) {
        jobs[t].f = f;
        jobs[t].qt = q_tokens;
        jobs[t].qo = q_offsets;
        jobs[t].lo = nq * t / nthreads;
        jobs[t].hi = nq * (t + 1) / nthreads;
        jobs[t].match_len = match_len;
        jobs[t].chosen = chosen;
    }
    int32_t started = 1;
    for (int32_t t = 1; t < nthreads; t++, started++)
        if (pthread_create(&th[t], NULL, route_range, &jobs[t])) break;
    for (int32_t t = started; t < nthreads; t++) route_range(&jobs[t]); /* threads that did not start */
    route_range(&jobs[0]);
    for (int32_t t = 1; t < started; t++) pthread_join(th[t], NULL);
    free(jobs);
    free(th);
    return 0;
}

/* ---- inspection (for the pins) ------------------------------------------ */

/* Nodes of peer's tree, the root not counted. */
int64_t rx_node_count(const rx_forest *f, int32_t peer) {
    if (!f || peer < 0 || peer >= f->num_peers) return -1;
    return f->t[peer].n - 1;
}

/* Tokens peer's tree holds: the sum of its label lengths, i.e. its distinct
 * non-empty prefixes. */
int64_t rx_tree_tokens(const rx_forest *f, int32_t peer) {
    if (!f || peer < 0 || peer >= f->num_peers) return -1;
    const rx_tree *t = &f->t[peer];
    int64_t s = 0;
    for (int64_t i = 1; i < t->n; i++) s += t->v[i].len;
    return s;
}

/* Structure of peer's tree: 0 if every node is as INSERT leaves it, else the
 * number of the first rule broken:
 *   1  a child key differs from its child's first label token, or the keys
 *      of a node are not strictly ascending;
 *   2  a non-root label is empty, or a depth is not the parent's depth plus
 *      the label length;
 *   3  a non-root node that ends no sequence has a single child, other than
 *      at a multiple of split_block (the tree is not path-compressed);
 *   4  a leaf ends no sequence;
 *   5  with split_block B, an edge straddles a multiple of B. */
int rx_check(const rx_forest *f, int32_t peer) {
    if (!f || peer < 0 || peer >= f->num_peers) return -1;
    const rx_tree *t = &f->t[peer];
    const int32_t B = f->split_block;
    for (int64_t x = 0; x < t->n; x++) {
        const rx_node *p = &t->v[x];
        for (int32_t k = 0; k < p->nch; k++) {
            const rx_node *c = &t->v[p->ch[k].id];
            if (c->len <= 0 || c->depth != p->depth + c->len) return 2;
            if (t->tok[c->lab] != p->ch[k].tok) return 1;
            if (k > 0 && p->ch[k - 1].tok >= p->ch[k].tok) return 1;
            if (B > 0 && (c->depth - 1) / B > p->depth / B) return 5; /* some k B in (parent, child) */
        }
        if (x == 0) continue;
        if (p->nch == 1 && p->ends == 0 && !(B > 0 && p->depth % B == 0)) return 3;
        if (p->nch == 0 && p->ends == 0) return 4;
    }
    return 0;
}
