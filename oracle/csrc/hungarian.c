/*
 * Oracle (test infrastructure only): exact minimum-cost perfect matching of a
 * square cost matrix, the textbook shortest-augmenting-path Hungarian method
 * with row and column potentials, O(n^3).
 *
 * Used to solve the balanced assignment of Eq. 2 (Sec. 3.2.1) on the matrix
 * whose columns replicate every expert T/E times: cost[t][e*C + j] = -S[t][e].
 * It shares nothing with the GPU path.
 *
 * Method: rows are inserted one at a time. For the new row, a Dijkstra-style
 * search over columns, on reduced costs cost[i][j] - u[i] - v[j] (kept >= 0 by
 * the potentials), grows a tree of alternating paths until it reaches a free
 * column; the potentials of the tree are then shifted by the search distances
 * and the matching is flipped along the path back to the new row.
 */
#include <stdint.h>
#include <stdlib.h>
#include <math.h>

/* cost: n*n row-major. row_to_col[n] out. u[n], v[n] out (may be NULL): dual
 * potentials with cost[i][j] >= u[i] + v[j] and equality on matched pairs.
 * Returns 0 on success, -1 on allocation failure or bad n. */
int oracle_hungarian(int64_t n, const double *cost, int64_t *row_to_col,
                     double *u_out, double *v_out)
{
    if (n <= 0) return -1;
    /* Index 0 is a virtual column used as the root of each search. */
    double *u = calloc((size_t)n + 1, sizeof(double));       /* row potentials */
    double *v = calloc((size_t)n + 1, sizeof(double));       /* column potentials */
    double *dist = malloc(((size_t)n + 1) * sizeof(double)); /* search labels per column */
    int64_t *col_row = calloc((size_t)n + 1, sizeof(int64_t)); /* row matched to column j (1-based, 0 = free) */
    int64_t *parent = calloc((size_t)n + 1, sizeof(int64_t)); /* previous column on the path */
    char *in_tree = malloc((size_t)n + 1);
    if (!u || !v || !dist || !col_row || !parent || !in_tree) {
        free(u); free(v); free(dist); free(col_row); free(parent); free(in_tree);
        return -1;
    }
    for (int64_t row = 1; row <= n; ++row) {
        col_row[0] = row;
        int64_t cur = 0;                   /* column whose matched row is expanded next */
        for (int64_t j = 0; j <= n; ++j) { dist[j] = INFINITY; in_tree[j] = 0; }
        for (;;) {
            in_tree[cur] = 1;
            const int64_t i = col_row[cur];
            const double *ci = cost + (i - 1) * n;
            double best = INFINITY;
            int64_t best_col = -1;
            for (int64_t j = 1; j <= n; ++j) {
                if (in_tree[j]) continue;
                const double red = ci[j - 1] - u[i] - v[j];
                if (red < dist[j]) { dist[j] = red; parent[j] = cur; }
                if (dist[j] < best) { best = dist[j]; best_col = j; }
            }
            /* Shift potentials so the tree's edges stay tight and the
             * closest outside column becomes tight too. */
            for (int64_t j = 0; j <= n; ++j) {
                if (in_tree[j]) { u[col_row[j]] += best; v[j] -= best; }
                else dist[j] -= best;
            }
            cur = best_col;
            if (col_row[cur] == 0) break;   /* reached a free column */
        }
        /* Flip the matching along the alternating path back to the root. */
        while (cur != 0) {
            const int64_t prev = parent[cur];
            col_row[cur] = col_row[prev];
            cur = prev;
        }
    }
    for (int64_t j = 1; j <= n; ++j) row_to_col[col_row[j] - 1] = j - 1;
    if (u_out) for (int64_t i = 0; i < n; ++i) u_out[i] = u[i + 1];
    if (v_out) for (int64_t j = 0; j < n; ++j) v_out[j] = v[j + 1];
    free(u); free(v); free(dist); free(col_row); free(parent); free(in_tree);
    return 0;
}
