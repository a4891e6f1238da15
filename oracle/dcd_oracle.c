/*
 * dcd_oracle.c -- plain fp64 CPU oracle for contrastive-decoding (CD) tree
 * verification, written from "Decoupled Contrastive Decoding via
 * Expert-Aligned Drafting" (arXiv 2608.12913).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this file.  It shares no code,
 * header, table or helper with the GPU library; the GPU library never calls it.
 *
 * Everything is computed in double precision from the exact input values (the
 * float inputs hold bf16 or fp32 values, both exactly representable in double).
 * Each dot product is one serial sum in ascending k; threads only split
 * independent dot products, so results do not depend on the thread count.
 *
 * What each function follows:
 *   row_logits          Alg. 1 "parallel model evaluation": each model's LM head
 *                       maps a node's hidden state to next-token logits.
 *   max_and_lse         log pi = z - logsumexp(z): the log of the softmax.
 *   cd_row              Sec. 2.1, Eq. (1) contrastive target
 *                         log pi_CD = (1+s) log pi_p - s log pi_q - log Z_CD,
 *                       with the plausibility mask of Sec. 2.1
 *                         P(h) = { x : pi_p(x) >= theta * max pi_p }
 *                       applied before renormalising (Appendix remark
 *                       "Plausibility-constrained CD").  s is the contrastive
 *                       strength, theta the plausibility cutoff.
 *   row_diag            diagnostics of Sec. 3.1 and of the KL-decomposition lemma
 *                       (App. B.1): the expert's own
 *                       top-1 token, D_KL(pi_p || pi_q) and D_KL(pi_p || pi_CD),
 *                       each summed from its definition.
 *   dco_propose         the decomposed dual-drafter of Sec. 3.1: the CD target of
 *                       two drafter heads, pi_hat ~ pi_e^(1+s) pi_f^(-s) (with
 *                       the same mask), as a proposal distribution per row and a
 *                       token drawn from it.
 *   dco_rmsnorm         the models' final RMS normalisation, the step that produces
 *                       the hidden states the LM heads read (Alg. 1's model
 *                       evaluation ends with it in the Llama-family models the
 *                       paper uses).
 *   dco_greedy_walk     greedy (T = 0) verification of a draft tree: a draft
 *                       token is accepted iff it equals the target's argmax
 *                       (Alg. 1 with a one-hot target), walked from the root.
 *   dco_sample_tree     Alg. 1 speculative accept / residual / bonus steps, on a
 *                       tree: the children of a node are tried in turn, each
 *                       against the residual left by the siblings rejected before
 *                       it (multi-draft speculative sampling as in SpecInfer, Miao
 *                       et al. 2024; the paper runs sampled verification on chains
 *                       only, where this is exactly Alg. 1).
 *
 * Readings where the paper is silent (all documented with the design notes):
 *   - mask test in log space: z_p - max z_p >= ln(theta); theta = 0 means no mask;
 *   - argmax ties go to the lowest token id; duplicate-token siblings: lowest
 *     node index wins;
 *   - accept iff pi_CD(tok) > 0 and u <= pi_CD(tok) / pi_e(tok); pi_e(tok) = 0
 *     gives ratio = +inf;
 *   - "sample" = inverse CDF in token-id order with one uniform; a residual
 *     that sums to zero (rounding only) leaves the distribution as it was;
 *   - siblings are tried in increasing node index;
 *   - temperature divides both models' logits before everything (sampled mode);
 *     greedy mode uses the models' own distributions (T = 1);
 *   - final RMS normalisation: y = g * round(x / sqrt(mean(x^2) + eps)) with both the
 *     normalised value and the product rounded to the input's type (bf16 inputs;
 *     no rounding for fp32), as Llama-family implementations compute it.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* per-sequence status codes (values are part of the checked contract) */
#define SEQ_OK 0
#define SEQ_BAD_TREE 1
#define SEQ_BAD_TOKEN 2
#define SEQ_NONFINITE 3
#define SEQ_NOT_CHAIN 4

/* row statistics slots */
enum { RS_MAXP = 0, RS_LSEP, RS_LSEQ, RS_LOGZ, RS_TOP1, RS_MARGIN, RS_COUNT, RS_SIGNAL, RS_N };
/* row diagnostics slots */
enum { RD_ARGMAX_P = 0, RD_KL_PQ, RD_KL_PCD, RD_MARGIN_P, RD_N };
/* node statistics slots */
enum { NS_LPP = 0, NS_LPQ, NS_CD, NS_LPCD, NS_INMASK, NS_RATIO, NS_N };

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* z[v] = (sum_{k ascending} h[k] * W[v][k] + b[v]) / T, W row-major [V][d]. */
static void row_logits(const float *h, const float *W, const float *b, int V, int d,
                       double T, double *z)
{
    long v;
#pragma omp parallel for schedule(static)
    for (v = 0; v < V; ++v) {
        const float *w = W + (size_t)v * (size_t)d;
        double acc = 0.0;
        for (int k = 0; k < d; ++k) acc += (double)h[k] * (double)w[k];
        if (b) acc += (double)b[v];
        z[v] = acc / T;
    }
}

/* M = max_v z[v];  lse = M + ln sum_v exp(z[v] - M). */
static void max_and_lse(const double *z, int V, double *M, double *lse)
{
    double m = -INFINITY;
    for (int v = 0; v < V; ++v)
        if (z[v] > m) m = z[v];
    double sum = 0.0;
    for (int v = 0; v < V; ++v) sum += exp(z[v] - m);
    *M = m;
    *lse = m + log(sum);
}

typedef struct {
    double stats[RS_N];
    int argmax;
    double gap; /* min over v below the max of |z_p[v] - M_p - ln theta|; +inf when
                   theta = 0 or every token is at the max */
} row_result;

/*
 * One row of the masked contrastive target, from the two models' logits.
 * Optionally returns lp_cd[v] = log pi_CD(v) (-inf off the mask).
 */
static void cd_row(const double *zp, const double *zq, int V, double theta, double s,
                   row_result *r, double *lp_cd)
{
    double Mp, lsep, Mq, lseq;
    max_and_lse(zp, V, &Mp, &lsep);
    max_and_lse(zq, V, &Mq, &lseq);
    const double log_theta = theta > 0.0 ? log(theta) : -INFINITY;

    /* pass 1: mask membership, cd score, argmax (lowest id on ties), runner-up.
       gap: how close a token's membership test comes to flipping.  A token at the
       expert max is a member for every theta (its test is 0 >= ln theta), so only
       the tokens below the max count. */
    int best = -1, count = 0;
    double top1 = -INFINITY, top2 = -INFINITY, gap = INFINITY;
    for (int v = 0; v < V; ++v) {
        if (theta > 0.0 && zp[v] != Mp) {
            double dist = fabs(zp[v] - Mp - log_theta);
            if (dist < gap) gap = dist;
        }
        int in_mask = (zp[v] - Mp) >= log_theta;
        if (!in_mask) continue;
        ++count;
        double cd = (1.0 + s) * (zp[v] - lsep) - s * (zq[v] - lseq);
        if (best < 0 || cd > top1) {
            if (best >= 0) top2 = top1;
            top1 = cd;
            best = v;
        } else if (cd > top2) {
            top2 = cd;
        }
    }
    /* pass 2: log Z over the mask, max-shifted */
    double sum = 0.0;
    for (int v = 0; v < V; ++v) {
        if (!((zp[v] - Mp) >= log_theta)) continue;
        double cd = (1.0 + s) * (zp[v] - lsep) - s * (zq[v] - lseq);
        sum += exp(cd - top1);
    }
    double logZ = top1 + log(sum);
    if (lp_cd) {
        for (int v = 0; v < V; ++v) {
            if ((zp[v] - Mp) >= log_theta)
                lp_cd[v] = (1.0 + s) * (zp[v] - lsep) - s * (zq[v] - lseq) - logZ;
            else
                lp_cd[v] = -INFINITY;
        }
    }
    r->argmax = best;
    r->gap = gap;
    r->stats[RS_MAXP] = Mp;
    r->stats[RS_LSEP] = lsep;
    r->stats[RS_LSEQ] = lseq;
    r->stats[RS_LOGZ] = logZ;
    r->stats[RS_TOP1] = top1;
    r->stats[RS_MARGIN] = count > 1 ? top1 - top2 : INFINITY;
    r->stats[RS_COUNT] = (double)count;
    r->stats[RS_SIGNAL] = best >= 0 ? (zp[best] - lsep) - (zq[best] - lseq) : NAN;
}

/*
 * Diagnostics of one row, after cd_row:
 *   RD_ARGMAX_P  argmax_x pi_p(x), the expert's own greedy token (lowest id on ties);
 *   RD_KL_PQ     D_KL(pi_p || pi_q)  = sum_x pi_p(x) (log pi_p(x) - log pi_q(x));
 *   RD_KL_PCD    D_KL(pi_p || pi_CD) = sum_x pi_p(x) (log pi_p(x) - log pi_CD(x)), with
 *                pi_CD the target of cd_row.  Off the mask pi_CD = 0 while pi_p > 0, so
 *                a mask that leaves out a token with pi_p > 0 gives +inf;
 *   RD_MARGIN_P  largest minus second-largest expert logit (0 on a tie), the margin
 *                that decides RD_ARGMAX_P.
 * Terms with pi_p(x) = 0 contribute 0 (x log x -> 0).
 */
static void row_diag(const double *zp, const double *zq, int V, double theta, double s,
                     const row_result *r, double *diag)
{
    const double Mp = r->stats[RS_MAXP], lsep = r->stats[RS_LSEP], lseq = r->stats[RS_LSEQ];
    const double logZ = r->stats[RS_LOGZ];
    const double log_theta = theta > 0.0 ? log(theta) : -INFINITY;
    int amax = -1;
    double second = -INFINITY;
    for (int v = 0; v < V; ++v) {
        if (amax < 0 && zp[v] == Mp)
            amax = v;
        else if (zp[v] > second)
            second = zp[v];
    }
    double kl_pq = 0.0, kl_pcd = 0.0;
    for (int v = 0; v < V; ++v) {
        const double lpp = zp[v] - lsep, lpq = zq[v] - lseq, pp = exp(lpp);
        if (pp == 0.0) continue;
        kl_pq += pp * (lpp - lpq);
        if ((zp[v] - Mp) >= log_theta) {
            const double lpcd = (1.0 + s) * lpp - s * lpq - logZ;
            kl_pcd += pp * (lpp - lpcd);
        } else {
            kl_pcd = INFINITY;
        }
    }
    diag[RD_ARGMAX_P] = (double)amax;
    diag[RD_KL_PQ] = kl_pq;
    diag[RD_KL_PCD] = kl_pcd;
    diag[RD_MARGIN_P] = Mp - second;
}

/*
 * Evaluate n_rows rows (row_ids[i], or i when row_ids is NULL) of an R-row problem.
 * Outputs per evaluated row: argmax, stats[8], boundary gap, and optionally the
 * diagnostics [RD_N], the logits of both models and log pi_CD over the vocabulary.
 */
int dco_eval_rows(int V, int dp, int dq,
                  const float *hp, const float *hq, const float *wp, const float *wq,
                  const float *bp, const float *bq, double temperature, double theta, double s,
                  const int32_t *row_ids, int n_rows,
                  int32_t *argmax_out, double *stats_out, double *gap_out, double *diag_out,
                  double *zp_out, double *zq_out, double *lpcd_out, int nthreads)
{
    if (V <= 0 || dp <= 0 || dq <= 0 || n_rows < 0 || !(temperature > 0.0)) return -2;
    set_threads(nthreads);
    double *zp = (double *)malloc(sizeof(double) * (size_t)V);
    double *zq = (double *)malloc(sizeof(double) * (size_t)V);
    if (!zp || !zq) { free(zp); free(zq); return -1; }
    for (int i = 0; i < n_rows; ++i) {
        long r = row_ids ? row_ids[i] : i;
        row_logits(hp + (size_t)r * dp, wp, bp, V, dp, temperature, zp);
        row_logits(hq + (size_t)r * dq, wq, bq, V, dq, temperature, zq);
        row_result res;
        cd_row(zp, zq, V, theta, s, &res, lpcd_out ? lpcd_out + (size_t)i * V : NULL);
        if (argmax_out) argmax_out[i] = res.argmax;
        if (stats_out) memcpy(stats_out + (size_t)i * RS_N, res.stats, sizeof(res.stats));
        if (gap_out) gap_out[i] = res.gap;
        if (diag_out) row_diag(zp, zq, V, theta, s, &res, diag_out + (size_t)i * RD_N);
        if (zp_out) memcpy(zp_out + (size_t)i * V, zp, sizeof(double) * (size_t)V);
        if (zq_out) memcpy(zq_out + (size_t)i * V, zq, sizeof(double) * (size_t)V);
    }
    free(zp);
    free(zq);
    return 0;
}

/* round-to-nearest-even of a double to bf16 (8 significant bits), returned as double */
static double round_bf16(double x)
{
    if (!isfinite(x) || x == 0.0) return x;
    int e;
    const double m = frexp(x, &e);           /* x = m * 2^e, 0.5 <= |m| < 1 */
    const double scaled = ldexp(m, 8);       /* 8 significant bits before the point */
    double r = nearbyint(scaled);            /* ties to even in the default rounding mode */
    return ldexp(r, e - 8);
}

/*
 * Final RMS normalisation of R rows of width d (the step before the LM heads):
 *   r = 1 / sqrt(mean_k x_k^2 + eps);  y_k = g_k * [x_k * r]
 * For bf16 data ([.] and the product rounded to bf16, round-to-nearest-even; the
 * rows, g and y hold bf16 values as floats) and without rounding for fp32.
 */
void dco_rmsnorm(int R, int d, const float *x, const float *g, double eps, int bf16, float *y)
{
    for (long r = 0; r < R; ++r) {
        const float *xr = x + (size_t)r * d;
        double ss = 0.0;
        for (int k = 0; k < d; ++k) ss += (double)xr[k] * (double)xr[k];
        const double inv = 1.0 / sqrt(ss / d + eps);
        for (int k = 0; k < d; ++k) {
            double v = (double)xr[k] * inv;
            if (bf16) v = round_bf16(v);
            v *= (double)g[k];
            if (bf16) v = round_bf16(v);
            y[(size_t)r * d + k] = (float)v;
        }
    }
}

/*
 * Greedy walk over one sequence's draft tree.  Node 0 is the root (last
 * committed token); node c scores its children with row c.  Starting at the
 * root, accept the lowest-index child whose token equals the argmax of the
 * current row; stop when no child matches.  next_token is the argmax at the
 * last accepted node (the token the target emits after the accepted prefix).
 */
void dco_greedy_walk(int N, const int32_t *parents, const int32_t *tokens,
                     const int32_t *row_argmax, int32_t *accept_len, int32_t *path,
                     int32_t *next_token)
{
    for (int i = 0; i < N; ++i) path[i] = -1;
    path[0] = 0;
    int cur = 0, len = 0;
    for (;;) {
        int target = row_argmax[cur], chosen = -1;
        for (int c = cur + 1; c < N; ++c) {
            if (parents[c] == cur && tokens[c] == target) { chosen = c; break; }
        }
        if (chosen < 0) break;
        path[++len] = chosen;
        cur = chosen;
    }
    *accept_len = len;
    *next_token = row_argmax[cur];
}

/* smallest index v with cumulative weight > u * total, in index order */
static int inverse_cdf(const double *w, int V, double u)
{
    double total = 0.0;
    int last = -1;
    for (int v = 0; v < V; ++v) {
        total += w[v];
        if (w[v] > 0.0) last = v;
    }
    double target = u * total, cum = 0.0;
    for (int v = 0; v < V; ++v) {
        cum += w[v];
        if (w[v] > 0.0 && cum > target) return v;
    }
    return last;
}

/* distance of u*total to the nearest cumulative breakpoint, relative to total */
static double cdf_gap(const double *w, int V, double u)
{
    double total = 0.0;
    for (int v = 0; v < V; ++v) total += w[v];
    double target = u * total, cum = 0.0, gap = INFINITY;
    for (int v = 0; v < V; ++v) {
        cum += w[v];
        if (w[v] > 0.0) {
            double d = fabs(cum - target);
            if (d < gap) gap = d;
        }
    }
    return total > 0.0 ? gap / total : 0.0;
}

/*
 * Alg. 1 speculative accept / fallback over one draft tree of N nodes (parents[i] < i).
 *   lp_cd    [N][V]  log pi_CD of each row (-inf off the mask)
 *   q        [N][V]  node-indexed proposal probabilities: row i is pi_e^(i),
 *                    the distribution draft token i was drawn from (row 0 unused)
 *   u_acc[i] decides node i; u_res[j] draws the token emitted after row j.
 * The walk starts at the root with p = pi_CD of the current row.  The children
 * c_1 < c_2 < ... of the current node are tried in index order: c_m (token x,
 * proposal q_m) is accepted iff p(x) > 0 and u_acc[c_m] <= p(x) / q_m(x), and the walk
 * moves to it with p = pi_CD of its row; a rejection replaces p by the residual
 * Normalize(max(0, p - q_m)) (p stays as it was if that sums to zero).  When every
 * child of the current node is rejected, or it has none, the emitted token is drawn
 * from p with u_res of the current node.  On a chain (one child per node) this is
 * Alg. 1: the first rejected node k is replaced by a draw from
 * Normalize(max(0, pi_CD^(k-1) - pi_e^(k))), and a fully accepted chain gets the
 * bonus token from pi_CD^(N-1).
 * ratio_out[i] receives pi_CD(tok_i) / pi_e^(i)(tok_i) under the parent row (all
 * i >= 1); walk_ratio[i] the ratio node i was actually tested with (its parent's
 * residual), NaN for nodes the walk never tested.  res_gap receives the relative
 * distance of the final draw to its CDF breakpoints (the parity gate for the
 * emitted token).
 */
void dco_sample_tree(int N, int V, const int32_t *parents, const int32_t *tokens,
                     const double *lp_cd, const float *q, const float *u_acc, const float *u_res,
                     int32_t *accept_len, int32_t *path, int32_t *next_token, double *ratio_out,
                     double *walk_ratio, double *res_gap)
{
    double *p = (double *)malloc(sizeof(double) * (size_t)V);
    double *w = (double *)malloc(sizeof(double) * (size_t)V);
    for (int i = 0; i < N; ++i) {
        path[i] = -1;
        if (walk_ratio) walk_ratio[i] = NAN;
        if (ratio_out) ratio_out[i] = NAN;
    }
    if (ratio_out)
        for (int i = 1; i < N; ++i) {
            double p_cd = exp(lp_cd[(size_t)parents[i] * V + tokens[i]]);
            double p_e = (double)q[(size_t)i * V + tokens[i]];
            ratio_out[i] = p_e > 0.0 ? p_cd / p_e : INFINITY;
        }
    path[0] = 0;
    int cur = 0, len = 0;
    for (;;) {
        const double *lrow = lp_cd + (size_t)cur * V;
        for (int v = 0; v < V; ++v) p[v] = exp(lrow[v]);
        int next = -1;
        for (int c = cur + 1; c < N && next < 0; ++c) {
            if (parents[c] != cur) continue;
            const float *qc = q + (size_t)c * V;
            const int x = tokens[c];
            double ratio = qc[x] > 0.0f ? p[x] / (double)qc[x] : INFINITY;
            if (walk_ratio) walk_ratio[c] = ratio;
            if (p[x] > 0.0 && (double)u_acc[c] <= ratio) {
                next = c;
                break;
            }
            double total = 0.0;
            for (int v = 0; v < V; ++v) {
                double r = p[v] - (double)qc[v];
                w[v] = r > 0.0 ? r : 0.0;
                total += w[v];
            }
            if (total > 0.0)
                for (int v = 0; v < V; ++v) p[v] = w[v] / total;
        }
        if (next < 0) break;
        path[++len] = next;
        cur = next;
    }
    *accept_len = len;
    *next_token = inverse_cdf(p, V, (double)u_res[cur]);
    if (res_gap) *res_gap = cdf_gap(p, V, (double)u_res[cur]);
    free(p);
    free(w);
}

/*
 * Proposals from the contrastive recombination of two heads (Sec. 3.1, decomposed
 * dual-drafter; App. A.1): for each of R rows, pi_hat = the CD target of the two
 * heads given as expert and amateur (Eq. (1) with the mask of cd_row, logits
 * divided by the temperature), written densely to probs_out [R][V]; and a token
 * drawn from it by inverse CDF with u[r] (tokens_out [R]), with the draw's relative
 * distance to its CDF breakpoints in gap_out [R] (the parity gate).
 */
int dco_propose(int R, int V, int de, int df, const float *he, const float *hf, const float *we,
                const float *wf, const float *be, const float *bf, double temperature, double theta,
                double s, const float *u, int32_t *tokens_out, double *probs_out, double *gap_out,
                int32_t *argmax_out, int nthreads)
{
    if (R <= 0 || V <= 0 || !(temperature > 0.0)) return -2;
    double *lp = (double *)malloc(sizeof(double) * (size_t)R * V);
    double *p = (double *)malloc(sizeof(double) * (size_t)V);
    if (!lp || !p) { free(lp); free(p); return -1; }
    int rc = dco_eval_rows(V, de, df, he, hf, we, wf, be, bf, temperature, theta, s, NULL, R,
                           argmax_out, NULL, NULL, NULL, NULL, NULL, lp, nthreads);
    if (rc) { free(lp); free(p); return rc; }
    for (int r = 0; r < R; ++r) {
        for (int v = 0; v < V; ++v) p[v] = exp(lp[(size_t)r * V + v]);
        if (probs_out) memcpy(probs_out + (size_t)r * V, p, sizeof(double) * (size_t)V);
        if (tokens_out) tokens_out[r] = inverse_cdf(p, V, (double)u[r]);
        if (gap_out) gap_out[r] = cdf_gap(p, V, (double)u[r]);
    }
    free(lp);
    free(p);
    return 0;
}

/* status of one sequence from its tree and tokens (before any numerics) */
static int check_sequence(int N, int V, const int32_t *parents, const int32_t *tokens)
{
    if (parents[0] != -1) return SEQ_BAD_TREE;
    for (int i = 1; i < N; ++i)
        if (parents[i] < 0 || parents[i] >= i) return SEQ_BAD_TREE;
    for (int i = 1; i < N; ++i)
        if (tokens[i] < 0 || tokens[i] >= V) return SEQ_BAD_TOKEN;
    return SEQ_OK;
}

static void reset_sequence(int N, int32_t *accept_len, int32_t *path, int32_t *next_token,
                           double *node_stats)
{
    *accept_len = 0;
    for (int i = 0; i < N; ++i) path[i] = -1;
    *next_token = -1;
    if (node_stats)
        for (int i = 0; i < N * NS_N; ++i) node_stats[i] = NAN;
}

/*
 * Full verification of B sequences of N nodes each (rows are b*N + i).
 * mode 0 = greedy (temperature ignored), mode 1 = sampled (dco_sample_tree).
 * Optional outputs may be NULL: row_argmax [R], row_stats [R][8], node_stats [R][6],
 * row_diag [R][RD_N], row_gap [R], res_gap [B], walk_ratio [R] (sampled: the ratio
 * each node was tested with, NaN if untested).
 */
int dco_verify(int mode, int B, int N, int V, int dp, int dq,
               const float *hp, const float *hq, const float *wp, const float *wq,
               const float *bp, const float *bq, const int32_t *parents, const int32_t *tokens,
               double theta, double s, double temperature,
               const float *draft_probs, const float *u_acc, const float *u_res,
               int32_t *accept_len, int32_t *accept_path, int32_t *next_token, int32_t *status,
               int32_t *row_argmax, double *row_stats, double *node_stats, double *row_diag,
               double *row_gap, double *res_gap, double *walk_ratio, int nthreads)
{
    if (B <= 0 || N <= 0 || V <= 0) return -2;
    if (mode == 1 && (!draft_probs || !u_acc || !u_res || !(temperature > 0.0))) return -3;
    const double T = mode == 1 ? temperature : 1.0;
    const long R = (long)B * N;
    int32_t *amax = (int32_t *)malloc(sizeof(int32_t) * (size_t)R);
    double *stats = (double *)malloc(sizeof(double) * (size_t)R * RS_N);
    double *gap = (double *)malloc(sizeof(double) * (size_t)R);
    double *lp_cd = (double *)malloc(sizeof(double) * (size_t)N * V);   /* one sequence */
    double *zp = (double *)malloc(sizeof(double) * (size_t)N * V);
    double *zq = (double *)malloc(sizeof(double) * (size_t)N * V);
    if (!amax || !stats || !gap || !lp_cd || !zp || !zq) {
        free(amax); free(stats); free(gap); free(lp_cd); free(zp); free(zq);
        return -1;
    }
    for (int b = 0; b < B; ++b) {
        const long r0 = (long)b * N;
        /* every row of the sequence: logits, stats, log pi_CD */
        int rc = dco_eval_rows(V, dp, dq, hp + (size_t)r0 * dp, hq + (size_t)r0 * dq, wp, wq, bp,
                               bq, T, theta, s, NULL, N, amax + r0, stats + (size_t)r0 * RS_N,
                               gap + r0, row_diag ? row_diag + (size_t)r0 * RD_N : NULL, zp, zq,
                               lp_cd, nthreads);
        if (rc) { free(amax); free(stats); free(gap); free(lp_cd); free(zp); free(zq); return rc; }

        const int32_t *par = parents + r0, *tok = tokens + r0;
        int32_t *path = accept_path + r0;
        double *ns = node_stats ? node_stats + (size_t)r0 * NS_N : NULL;
        int st = check_sequence(N, V, par, tok);
        if (st == SEQ_OK) {
            for (int i = 0; i < N; ++i) {
                const double *rs = stats + (size_t)(r0 + i) * RS_N;
                if (!isfinite(rs[RS_MAXP]) || !isfinite(rs[RS_LSEP]) || !isfinite(rs[RS_LSEQ]) ||
                    !isfinite(rs[RS_LOGZ]))
                    st = SEQ_NONFINITE;
            }
        }
        status[b] = st;
        if (st != SEQ_OK) {
            reset_sequence(N, accept_len + b, path, next_token + b, ns);
            if (walk_ratio)
                for (int i = 0; i < N; ++i) walk_ratio[r0 + i] = NAN;
            if (res_gap) res_gap[b] = INFINITY;
            continue;
        }
        /* node statistics: node i is scored by its parent's row */
        if (ns) {
            for (int c = 0; c < NS_N; ++c) ns[c] = NAN;
            for (int i = 1; i < N; ++i) {
                int j = par[i], x = tok[i];
                const double *rs = stats + (size_t)(r0 + j) * RS_N;
                double lpp = zp[(size_t)j * V + x] - rs[RS_LSEP];
                double lpq = zq[(size_t)j * V + x] - rs[RS_LSEQ];
                double lpc = lp_cd[(size_t)j * V + x];
                ns[i * NS_N + NS_LPP] = lpp;
                ns[i * NS_N + NS_LPQ] = lpq;
                ns[i * NS_N + NS_CD] = (1.0 + s) * lpp - s * lpq;
                ns[i * NS_N + NS_LPCD] = lpc;
                ns[i * NS_N + NS_INMASK] = isinf(lpc) ? 0.0 : 1.0;
                ns[i * NS_N + NS_RATIO] = NAN;
            }
        }
        if (mode == 0) {
            dco_greedy_walk(N, par, tok, amax + r0, accept_len + b, path, next_token + b);
            if (res_gap) res_gap[b] = INFINITY;
            if (walk_ratio)
                for (int i = 0; i < N; ++i) walk_ratio[r0 + i] = NAN;
        } else {
            double *ratio = (double *)malloc(sizeof(double) * (size_t)N);
            double g = INFINITY;
            dco_sample_tree(N, V, par, tok, lp_cd, draft_probs + (size_t)r0 * V, u_acc + r0,
                            u_res + r0, accept_len + b, path, next_token + b, ratio,
                            walk_ratio ? walk_ratio + r0 : NULL, &g);
            if (ns)
                for (int i = 1; i < N; ++i) ns[i * NS_N + NS_RATIO] = ratio[i];
            if (res_gap) res_gap[b] = g;
            free(ratio);
        }
    }
    if (row_argmax) memcpy(row_argmax, amax, sizeof(int32_t) * (size_t)R);
    if (row_stats) memcpy(row_stats, stats, sizeof(double) * (size_t)R * RS_N);
    if (row_gap) memcpy(row_gap, gap, sizeof(double) * (size_t)R);
    free(amax); free(stats); free(gap); free(lp_cd); free(zp); free(zq);
    return 0;
}
