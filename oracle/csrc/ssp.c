/*
 * Oracle (test infrastructure only): exact solve of the balanced assignment
 * problem of Eq. 2 (Sec. 3.2.1),
 *     maximise  sum_t S[t][a_t]   subject to  |{t : a_t = e}| = T/E  for all e,
 * as a transportation problem solved by successive shortest paths on the E
 * expert nodes. It shares nothing with the GPU path.
 *
 * Tokens are inserted one at a time (t = 0, 1, ...). Inserting token t looks
 * for the cheapest chain "t goes to e0, a token of e0 moves to e1, ..., a token
 * of e_{k-1} moves to e_k" that ends at an expert e_k with a free slot. Moving
 * token t' from expert u to expert v costs S[t'][u] - S[t'][v]; the cheapest
 * such move between u and v is an arc of weight
 *     w(u, v) = min over tokens t' held by u of (S[t'][u] - S[t'][v]).
 * Each w(u, v) is the top of a min-heap of (S[t'][u] - S[t'][v], t') over the
 * tokens of u, with stale entries (tokens that have since left u) dropped when
 * they reach the top. Expert potentials phi keep the reduced arc weights
 * w(u,v) + phi[u] - phi[v] non-negative, so a dense O(E^2) Dijkstra finds the
 * cheapest chain. After the search, phi[e] += min(dist[e], dist[target]).
 * Every insertion keeps the partial assignment optimal for the tokens seen so
 * far (the incremental form of the Hungarian method), so the final assignment
 * is optimal, and p = -phi are dual prices with
 *     S[t][a_t] - p[a_t] >= S[t][e] - p[e]   for every t and e,
 * i.e. sum_t max_e (S[t][e] - p[e]) + (T/E) sum_e p[e] equals the optimum.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

typedef struct { double key; int32_t tok; } entry_t;
typedef struct { entry_t *a; int64_t n, cap; } heap_t;

static int entry_less(entry_t x, entry_t y)
{
    return x.key < y.key || (x.key == y.key && x.tok < y.tok);
}

static int heap_push(heap_t *h, double key, int32_t tok)
{
    if (h->n == h->cap) {
        int64_t cap = h->cap ? 2 * h->cap : 16;
        entry_t *a = realloc(h->a, (size_t)cap * sizeof(entry_t));
        if (!a) return -1;
        h->a = a; h->cap = cap;
    }
    int64_t i = h->n++;
    entry_t x = { key, tok };
    while (i > 0) {
        int64_t p = (i - 1) / 2;
        if (!entry_less(x, h->a[p])) break;
        h->a[i] = h->a[p];
        i = p;
    }
    h->a[i] = x;
    return 0;
}

static void sift_down(heap_t *h, int64_t i)
{
    entry_t x = h->a[i];
    for (;;) {
        int64_t c = 2 * i + 1;
        if (c >= h->n) break;
        if (c + 1 < h->n && entry_less(h->a[c + 1], h->a[c])) ++c;
        if (!entry_less(h->a[c], x)) break;
        h->a[i] = h->a[c];
        i = c;
    }
    h->a[i] = x;
}

static void heap_pop(heap_t *h)
{
    h->a[0] = h->a[--h->n];
    if (h->n > 0) sift_down(h, 0);
}

typedef struct {
    int64_t T, E;
    const double *S;
    int32_t *owner;      /* expert holding each token, -1 if not inserted yet */
    heap_t *heaps;       /* E*E heaps, index u*E + v */
    int32_t *mark;       /* scratch for compaction */
    int32_t mark_id;
} state_t;

/* Drop stale tops; return the valid top entry of heap (u, v) or NULL. */
static const entry_t *valid_top(state_t *st, int64_t u, int64_t v)
{
    heap_t *h = &st->heaps[u * st->E + v];
    while (h->n > 0 && st->owner[h->a[0].tok] != (int32_t)u) heap_pop(h);
    return h->n > 0 ? &h->a[0] : NULL;
}

/* Rebuild heap (u, v) from its live, distinct entries once stale ones pile up. */
static void compact(state_t *st, int64_t u, int64_t v)
{
    heap_t *h = &st->heaps[u * st->E + v];
    ++st->mark_id;
    int64_t k = 0;
    for (int64_t i = 0; i < h->n; ++i) {
        int32_t tok = h->a[i].tok;
        if (st->owner[tok] != (int32_t)u || st->mark[tok] == st->mark_id) continue;
        st->mark[tok] = st->mark_id;
        h->a[k++] = h->a[i];
    }
    h->n = k;
    for (int64_t i = k / 2 - 1; i >= 0; --i) sift_down(h, i);
}

/* Token tok now belongs to expert u: add it to every heap (u, v). */
static int enter(state_t *st, int32_t tok, int64_t u, int64_t C)
{
    const double *row = st->S + (int64_t)tok * st->E;
    st->owner[tok] = (int32_t)u;
    for (int64_t v = 0; v < st->E; ++v) {
        if (v == u) continue;
        heap_t *h = &st->heaps[u * st->E + v];
        if (heap_push(h, row[u] - row[v], tok)) return -1;
        if (h->n > 4 * C + 64) compact(st, u, v);
    }
    return 0;
}

/* S: T*E row-major scores (fp64). assign[T] out: expert per token.
 * prices[E] out (may be NULL): dual prices certifying optimality.
 * Returns 0 on success, -1 on bad sizes (T % E != 0 or non-positive), -2 on
 * allocation failure. */
int oracle_ssp_solve(int64_t T, int64_t E, const double *S, int32_t *assign, double *prices)
{
    if (T <= 0 || E <= 0 || T % E != 0 || T > INT32_MAX) return -1;
    const int64_t C = T / E;
    int rc = 0;
    state_t st = { T, E, S, NULL, NULL, NULL, 0 };
    st.owner = malloc((size_t)T * sizeof(int32_t));
    st.mark = calloc((size_t)T, sizeof(int32_t));
    st.heaps = calloc((size_t)(E * E), sizeof(heap_t));
    double *phi = calloc((size_t)E, sizeof(double));
    double *dist = malloc((size_t)E * sizeof(double));
    int64_t *cnt = calloc((size_t)E, sizeof(int64_t));
    int64_t *prev = malloc((size_t)E * sizeof(int64_t));
    int32_t *via = malloc((size_t)E * sizeof(int32_t));
    char *done = malloc((size_t)E);
    if (!st.owner || !st.mark || !st.heaps || !phi || !dist || !cnt || !prev || !via || !done) {
        rc = -2;
        goto out;
    }
    for (int64_t t = 0; t < T; ++t) st.owner[t] = -1;

    for (int64_t t = 0; t < T; ++t) {
        const double *row = S + t * E;
        /* Labels start from the direct moves "token t goes to expert e". */
        for (int64_t e = 0; e < E; ++e) {
            dist[e] = -row[e] - phi[e];
            prev[e] = -1;
            done[e] = 0;
        }
        int64_t target = -1;
        for (;;) {
            int64_t u = -1;
            for (int64_t e = 0; e < E; ++e)
                if (!done[e] && (u < 0 || dist[e] < dist[u])) u = e;
            done[u] = 1;
            if (cnt[u] < C) { target = u; break; }
            for (int64_t v = 0; v < E; ++v) {
                if (done[v]) continue;
                const entry_t *top = valid_top(&st, u, v);
                if (!top) continue;
                const double nd = dist[u] + top->key + phi[u] - phi[v];
                if (nd < dist[v]) { dist[v] = nd; prev[v] = u; via[v] = top->tok; }
            }
        }
        const double reach = dist[target];
        for (int64_t e = 0; e < E; ++e) phi[e] += (dist[e] < reach ? dist[e] : reach);
        /* Apply the chain: every arc u -> v moves token via[v] from u to v. */
        int64_t v = target;
        while (prev[v] >= 0) {
            if (enter(&st, via[v], v, C)) { rc = -2; goto out; }
            v = prev[v];
        }
        if (enter(&st, (int32_t)t, v, C)) { rc = -2; goto out; }
        cnt[target] += 1;
    }
    for (int64_t t = 0; t < T; ++t) assign[t] = st.owner[t];
    if (prices) for (int64_t e = 0; e < E; ++e) prices[e] = -phi[e];
out:
    if (st.heaps) for (int64_t i = 0; i < E * E; ++i) free(st.heaps[i].a);
    free(st.heaps); free(st.owner); free(st.mark);
    free(phi); free(dist); free(cnt); free(prev); free(via); free(done);
    return rc;
}
