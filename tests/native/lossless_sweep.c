/*
 * Brute-force driver for the lossless-property pin of the oracle's tree sampler
 * (test code; links the oracle library).
 *
 * Star tree: a root and K children, child k drafted from q[k] independently.  For
 * every assignment of the children's tokens, weighted by prod_k q_k(x_k), and every
 * cell of a midpoint grid of G values for each u_acc[k] and for u_res[0], the
 * sampler runs once; the cell's weight goes to the first emitted token (the token of
 * the accepted child, or the draw at the root).  By the lossless property of
 * speculative sampling the result is pi_CD of the root up to the grid resolution.
 */
#include <stdint.h>
#include <stdlib.h>

void dco_sample_tree(int N, int V, const int32_t *parents, const int32_t *tokens,
                     const double *lp_cd, const float *q, const float *u_acc, const float *u_res,
                     int32_t *accept_len, int32_t *path, int32_t *next_token, double *ratio_out,
                     double *walk_ratio, double *res_gap);

int sweep_star(int K, int V, const double *lp_cd, const float *q, int G, double *out)
{
    if (K < 1 || K > 3 || V < 1 || G < 1) return -1;
    const int N = K + 1;
    int32_t parents[4], tokens[4], path[4], L, nxt;
    float ua[4], ur[4];
    for (int i = 0; i < N; ++i) {
        parents[i] = i == 0 ? -1 : 0;
        tokens[i] = 0;
        ua[i] = 0.5f;
        ur[i] = 0.5f;
    }
    for (int v = 0; v < V; ++v) out[v] = 0.0;
    long n_assign = 1, n_cells = G;
    for (int k = 0; k < K; ++k) {
        n_assign *= V;
        n_cells *= G;
    }
    const double cell = 1.0 / (double)n_cells;
    for (long a = 0; a < n_assign; ++a) {
        double wx = 1.0;
        long r = a;
        for (int k = 1; k <= K; ++k) {
            tokens[k] = (int32_t)(r % V);
            r /= V;
            wx *= (double)q[(size_t)k * V + tokens[k]];
        }
        if (wx == 0.0) continue;
        for (long c = 0; c < n_cells; ++c) {
            long t = c;
            for (int k = 1; k <= K; ++k) {
                ua[k] = (float)(((double)(t % G) + 0.5) / G);
                t /= G;
            }
            ur[0] = (float)(((double)t + 0.5) / G);
            dco_sample_tree(N, V, parents, tokens, lp_cd, q, ua, ur, &L, path, &nxt, NULL, NULL,
                            NULL);
            out[L > 0 ? tokens[path[1]] : nxt] += wx * cell;
        }
    }
    return 0;
}
