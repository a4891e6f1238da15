/*
 * dcd.h -- C ABI of libdcd: contrastive-decoding (CD) verification of a drafted
 * token tree on one AMD Instinct MI355X (gfx950).
 *
 * Method: "Decoupled Contrastive Decoding via Expert-Aligned Drafting"
 * (arXiv 2608.12913).  For every node of a draft tree the library
 *   1. projects the expert's and the amateur's final hidden states through their
 *      LM heads (Alg. 1, "parallel model evaluation"): z_m = H_m W_m^T + b_m;
 *   2. forms the contrastive target of Sec. 2.1, Eq. (1),
 *        log pi_CD(x) = (1+s) log pi_p(x) - s log pi_q(x) - log Z_CD,
 *      restricted to the plausibility mask {x : pi_p(x) >= theta * max pi_p}
 *      and renormalised (Sec. 2.1 and the appendix remark on
 *      plausibility-constrained CD);
 *   3. verifies the draft tokens against pi_CD: greedily (T = 0) by walking the
 *      tree from the root, or by speculative rejection sampling (chains and trees)
 *      (Alg. 1: accept test, residual resampling, bonus token).
 *
 * Notation: s = cd_strength (the paper's contrastive strength), theta =
 * plaus_thresh (the paper's plausibility cutoff).  theta = 0 means no mask (the
 * untruncated target the paper's experiments use): every token is in the
 * support and the target's statistics come from both models' full logits, which
 * the LM-head step then keeps in the workspace instead of candidate lists.
 *
 * Conventions shared by every entry point
 *  - Rows: a problem holds B sequences of N nodes each; row r = b*N + i is node i
 *    of sequence b.  Node 0 is the root (the last committed token).  Row i's
 *    hidden states produce the distribution that scores node i's CHILDREN.  A chain
 *    of N nodes therefore verifies N-1 drafted tokens.
 *  - Pointers named "device" are HIP device pointers (or host-coherent memory the
 *    GPU can read); the caller owns every buffer.  Matrices are row-major and
 *    densely packed.  The library allocates no memory and keeps no state between
 *    calls (dcd_verify_greedy_noalloc's static per-GPU array aside); calls on
 *    distinct streams with distinct workspaces may run concurrently.
 *  - Asynchrony: work is enqueued on `hip_stream` (a hipStream_t passed as void*,
 *    NULL = the default stream); calls return without synchronising.  Outputs are
 *    valid once the stream has reached the call.
 *  - Errors: problems detectable on the host (NULL pointers, shapes, parameters,
 *    alignment, workspace size) return a negative DCD_ERR_* code synchronously and
 *    enqueue nothing.  Data-dependent problems are reported per sequence in
 *    `status[b]` (DCD_SEQ_*); such a sequence gets accept_len 0, an accept_path of
 *    -1s and next_token -1 (its row outputs are still written).
 *  - Alignment: h_* and w_* must be 16-byte aligned and their hidden sizes a
 *    multiple of 8 (bf16) or 4 (fp32) so rows can be streamed with 128-bit loads;
 *    every other pointer must be 4-byte aligned.
 *  - Determinism: two calls with identical inputs produce bit-identical outputs.
 */
#ifndef DCD_H
#define DCD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes */
enum {
    DCD_OK = 0,
    DCD_ERR_NULL = -1,        /* a required pointer is NULL */
    DCD_ERR_SHAPE = -2,       /* a size is out of range or inconsistent */
    DCD_ERR_PARAM = -3,       /* plaus_thresh, cd_strength, temperature or dtype invalid */
    DCD_ERR_ALIGN = -4,       /* pointer or hidden-size alignment violated */
    DCD_ERR_WORKSPACE = -5,   /* workspace NULL, not 256-byte aligned, or smaller than dcd_workspace_bytes() */
    DCD_ERR_UNSUPPORTED = -6, /* valid request the library does not implement */
    DCD_ERR_HIP = -7,         /* the HIP runtime rejected a launch */
    DCD_ERR_TOO_LARGE = -8    /* dcd_verify_greedy_noalloc: the problem needs more than
                                 dcd_noalloc_max_bytes() of device memory */
};

/* per-sequence status written to outputs.status[b] */
enum {
    DCD_SEQ_OK = 0,
    DCD_SEQ_BAD_TREE = 1,   /* parents[b,0] != -1 or parents[b,i] outside [0, i) */
    DCD_SEQ_BAD_TOKEN = 2,  /* a draft token (i >= 1) outside [0, vocab) */
    DCD_SEQ_NONFINITE = 3,  /* a row of the sequence has a non-finite max, log-normaliser or log Z */
    DCD_SEQ_NOT_CHAIN = 4,  /* not produced since ABI 3 (sampled verification takes trees) */
    DCD_SEQ_WALK_TIMEOUT = 5 /* sampled, plaus_thresh = 0: the workgroups sharing the sequence's
                                walk did not meet in time (a device fault; outputs undefined) */
};

/* element type of hidden states and LM-head weights (bias is always fp32) */
enum { DCD_F32 = 0, DCD_BF16 = 1 };

/* row_stats slots (8 floats per row) */
enum {
    DCD_ROW_MAX_P = 0,   /* max_x z_p(x)                                             */
    DCD_ROW_LSE_P = 1,   /* log sum_x exp z_p(x): log pi_p = z_p - this               */
    DCD_ROW_LSE_Q = 2,   /* same for the amateur                                      */
    DCD_ROW_LOGZ = 3,    /* log sum over the mask of exp(cd(x)), cd below             */
    DCD_ROW_TOP1 = 4,    /* cd score of the argmax                                     */
    DCD_ROW_MARGIN = 5,  /* top-1 minus top-2 cd score over the mask (+inf: one member) */
    DCD_ROW_COUNT = 6,   /* number of tokens in the mask                               */
    DCD_ROW_SIGNAL = 7   /* log pi_p(x*) - log pi_q(x*) at the argmax x*               */
};
/* node_stats slots (6 floats per row; row 0 of every sequence is NaN) */
enum {
    DCD_NODE_LOGP_P = 0, /* log pi_p(tok_i) under the parent row                      */
    DCD_NODE_LOGP_Q = 1, /* log pi_q(tok_i)                                           */
    DCD_NODE_CD = 2,     /* cd score (1+s) log pi_p - s log pi_q                      */
    DCD_NODE_LOGP_CD = 3,/* log pi_CD(tok_i), -inf outside the mask                    */
    DCD_NODE_IN_MASK = 4,/* 1 if tok_i is in the parent row's mask, else 0            */
    DCD_NODE_RATIO = 5   /* sampled: pi_CD(tok_i) / pi_e(tok_i) (+inf if pi_e = 0); greedy: NaN */
};
/*
 * row_kl slots (2 floats per row): the divergences of the KL-decomposition lemma
 * (App. B.1), per row and over the whole vocabulary.
 *   DCD_KL_P_Q   D_KL(pi_p || pi_q)
 *   DCD_KL_P_CD  D_KL(pi_p || pi_CD) = log Z_CD - s * D_KL(pi_p || pi_q) (the lemma)
 * Both need both models' logits at every token, which only the untruncated target
 * (plaus_thresh = 0) keeps; with a mask DCD_KL_P_Q is NaN and DCD_KL_P_CD is +inf
 * (pi_p > 0 where pi_CD = 0) when the mask leaves out any token, NaN otherwise.
 */
enum { DCD_KL_P_Q = 0, DCD_KL_P_CD = 1 };

typedef struct {
    int32_t batch;       /* B >= 1 sequences                                            */
    int32_t nodes;       /* 1 <= N <= 4096 nodes per sequence, root included            */
    int32_t vocab;       /* V >= 1                                                      */
    int32_t d_expert;    /* expert hidden size d_p                                      */
    int32_t d_amateur;   /* amateur hidden size d_q                                     */
    int32_t dtype;       /* DCD_BF16 or DCD_F32 for h_* and w_*                         */
    float plaus_thresh;  /* theta in [0, 1]; 0 = untruncated target                     */
    float cd_strength;   /* s >= 0 (finite)                                             */
    float temperature;   /* sampled mode: T > 0 divides both models' logits before
                            anything else, mask included; ignored by greedy mode         */
    int32_t final_norm;  /* 1: h_* are the models' hidden states BEFORE their final RMS
                            normalisation, which the call applies first (norm_* and
                            norm_eps below); 0: h_* are already normalised            */
    float norm_eps;      /* final_norm = 1: eps >= 0 of that normalisation            */
} dcd_problem;

typedef struct {                 /* device pointers, read only                          */
    const void *h_expert;        /* [B*N, d_p] final expert hidden state of every node   */
    const void *h_amateur;       /* [B*N, d_q]                                           */
    const void *w_expert;        /* [V, d_p]  expert LM head (nn.Linear [out, in] layout) */
    const void *w_amateur;       /* [V, d_q]                                             */
    const float *bias_expert;    /* [V] fp32 logit bias, or NULL for none                */
    const float *bias_amateur;   /* [V] fp32, or NULL; may alias bias_expert             */
    const int32_t *parents;      /* [B, N] parent node of each node; parents[b,0] = -1   */
    const int32_t *tokens;       /* [B, N] draft token of each node (entry 0 ignored)    */
    /* final_norm = 1: the scales g of the models' final RMS normalisation, [d_p] and
       [d_q] in the dtype of h_*.  Each row x becomes y = g * [x / sqrt(mean(x^2) + eps)]
       with, for bf16, the normalised value [.] and the product rounded to bf16
       (round to nearest even; fp32: no rounding), as Llama-family models compute
       it; the LM heads then read y.  Unused (may be NULL) when final_norm = 0.   */
    const void *norm_expert;
    const void *norm_amateur;
} dcd_inputs;

typedef struct {                 /* device pointers, written by the call                 */
    int32_t *accept_len;         /* [B] number of accepted draft nodes                    */
    int32_t *accept_path;        /* [B, N] node ids: 0, then accepted nodes, then -1      */
    int32_t *next_token;         /* [B] greedy: argmax of pi_CD at the last accepted node;
                                    sampled: the residual or bonus token                  */
    int32_t *status;             /* [B] DCD_SEQ_*                                         */
    int32_t *row_argmax;         /* [B*N] optional (NULL skips): argmax of pi_CD per row;
                                    ties go to the lowest token id                        */
    float *row_stats;            /* [B*N, 8] optional: DCD_ROW_* slots                    */
    float *node_stats;           /* [B*N, 6] optional: DCD_NODE_* slots                   */
    /* diagnostics of Sec. 3.1 (signal and top-1 agreement at x* = argmax pi_CD; the
       signal itself is DCD_ROW_SIGNAL) and of the KL lemma of App. B.1        */
    int32_t *row_argmax_expert;  /* [B*N] optional: argmax of pi_p, the expert's own greedy
                                    token (lowest id on ties); top-1 agreement with the
                                    target is row_argmax_expert == row_argmax          */
    float *row_kl;               /* [B*N, 2] optional: DCD_KL_* slots                     */
} dcd_outputs;

/*
 * Bytes of device workspace a call with problem `p` needs (0 if `p` is invalid);
 * with final_norm = 1 it includes the normalised copies of h_* (B*N*(d_p + d_q)
 * elements).
 * The workspace holds per-tile softmax partials, the candidate logits that may
 * fall inside the plausibility mask (theta > 0) or, with theta = 0 (every token in
 * the support), a dense row of y = (1+s) z_p - s z_q per row (the expert logits as
 * well from 65 to 511 rows) and two rows of V doubles per sequence for the
 * residuals of sampled verification, and per-row results; it is O(B*N*V) bytes
 * (at most about 8.1 bytes per row and vocabulary entry).  The size depends on the
 * problem, so a workspace sized for one problem may be too small for another.
 */
size_t dcd_workspace_bytes(const dcd_problem *p);

/*
 * Greedy (T = 0) verification of B draft trees.
 * For every row: logits of both LM heads, max and log-normaliser of each, the
 * plausibility mask, the cd score, its log normaliser over the mask and its
 * argmax.  Then, per sequence, starting at the root: accept the lowest-index
 * child whose draft token equals the current row's argmax, repeat from it, stop
 * when no child matches; next_token is the argmax of the last accepted node.
 * A draft token outside the mask is never accepted.
 * Workspace: device memory of at least dcd_workspace_bytes(p) bytes, 256-byte
 * aligned, not used by any concurrently running call.  Its first 8 bytes hold a
 * count of the calls made on it, which the library keeps from call to call (for
 * every problem the workspace is large enough for); zero-fill a new workspace
 * once.  The rest is scratch.
 */
int dcd_verify_greedy(const dcd_problem *p, const dcd_inputs *in, const dcd_outputs *out,
                      void *workspace, size_t workspace_bytes, void *hip_stream);

/*
 * Sampled verification (Alg. 1) of B draft trees (chains included).
 *   draft_probs [B*N, V] fp32 device: row b*N+i is pi_e^(i), the proposal draft
 *               token i was drawn from (row b*N+0 unused)
 *   u_accept    [B*N] fp32 device, in (0,1): u_accept[b*N+i] decides node i
 *   u_resample  [B*N] fp32 device, in (0,1): u_resample[b*N+j] draws the token
 *               emitted after row j
 * The walk starts at the root with p = pi_CD of the root's row.  The children of
 * the current node are tried in increasing node index: child c with token x is
 * accepted iff p(x) > 0 and u_accept[c] <= p(x) / pi_e^(c)(x), and the walk moves
 * to it with p = pi_CD of its row; a rejected child replaces p by the residual
 * Normalize(max(0, p - pi_e^(c))) (p is kept if that sums to zero).  When every
 * child of the current node is rejected, or it has none, the emitted token
 * (next_token) is drawn from p with u_resample of the current node.  On a chain
 * this is Alg. 1: stop at the first rejected node k and draw from
 * Normalize(max(0, pi_CD^(k-1) - pi_e^(k))), or draw the bonus token from
 * pi_CD^(N-1).  The paper runs sampled verification on chains only; for trees
 * this is multi-draft speculative sampling (SpecInfer's rule), lossless when
 * siblings are drafted independently from their pi_e.  A draw is the inverse CDF
 * in token-id order: the smallest token whose cumulative weight exceeds
 * u_resample times the total.  node_stats[DCD_NODE_RATIO] is pi_CD / pi_e of the
 * node's token under its parent row (the ratio of a first sibling).
 * With plaus_thresh = 0 and at most 64 sequences, each sequence's walk is spread
 * over several workgroups (at most one per CU, all of them resident together on a
 * device running nothing else), which meet at barriers with bounded waits; a
 * sequence whose workgroups failed to meet (other work holding the CUs for seconds)
 * gets status DCD_SEQ_WALK_TIMEOUT.
 */
int dcd_verify_sample(const dcd_problem *p, const dcd_inputs *in, const float *draft_probs,
                      const float *u_accept, const float *u_resample, const dcd_outputs *out,
                      void *workspace, size_t workspace_bytes, void *hip_stream);

/*
 * Proposals from the contrastive recombination of two heads: the decomposed
 * dual-drafter of Sec. 3.1 (App. A.1), pi_hat(x) ~ pi_e(x)^(1+s) pi_f(x)^(-s), is the
 * CD target computed by the verify calls with the drafter's expert-aligned head in
 * the expert slots of `in` and its amateur-aligned head in the amateur slots (any
 * two heads work; with the models' own heads it is pi_CD itself).  Per row
 * r < batch*nodes: the logits of both heads divided by the problem's temperature,
 * the plausibility mask, then
 *   probs  [B*N, V] fp32 device, optional: pi_hat of every token (0 off the mask);
 *   tokens [B*N] int32 device, optional: a token drawn from pi_hat with u[r] by
 *          inverse CDF in token-id order (needs u [B*N] fp32 device in (0,1));
 *   argmax [B*N] int32 device, optional: argmax of pi_hat, lowest id on ties.
 * At least one output must be given.  Only h_*, w_* and bias_* of `in` are read;
 * the rows need no tree.  A row with non-finite logits gets token -1.  Workspace
 * and errors as for the verify calls.  A proposer that keeps `probs` can pass
 * them as the draft_probs of a later dcd_verify_sample.
 */
int dcd_propose(const dcd_problem *p, const dcd_inputs *in, const float *u, int32_t *tokens,
                float *probs, int32_t *argmax, void *workspace, size_t workspace_bytes,
                void *hip_stream);

/*
 * First stage of dcd_verify_greedy / dcd_verify_sample on its own: both LM-head
 * projections of every row with their per-tile softmax partials and plausibility
 * candidates, written to `workspace` (one kernel launch, everything else of the
 * verification left undone).  `sampled` != 0 applies the problem's temperature as
 * dcd_verify_sample does.  Only h_*, w_* and bias_* of `in` are read.  For callers
 * that time or schedule the projection separately; the workspace contents are
 * internal.  Errors as for the verify calls.
 */
int dcd_lmhead_partials(const dcd_problem *p, const dcd_inputs *in, int sampled, void *workspace,
                        size_t workspace_bytes, void *hip_stream);

/*
 * dcd_verify_greedy without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Same arguments, outputs and errors as dcd_verify_greedy,
 * same kernels; the workspace is a static device array inside the library instead
 * of the caller's memory.
 *  - The call allocates nothing (no hipMalloc, hipFree or allocating library call).
 *  - One array per GPU, of dcd_noalloc_max_bytes() bytes (80 MiB: 64 rows of a
 *    128,256-token vocabulary in every mode), created when the library's code is
 *    loaded on that GPU and held until the process ends.  A problem whose
 *    dcd_workspace_bytes() exceeds it returns DCD_ERR_TOO_LARGE before anything
 *    touches a device.
 *  - The GPU is the one of hip_stream (of the current device for NULL); the first
 *    call on a GPU looks up the array's device address (DCD_ERR_HIP if that fails).
 *  - Every call on a GPU uses that GPU's one array and leaves its contents behind:
 *    calls that overlap on one GPU (on different streams, or from several threads)
 *    race and must be serialised by the caller.  Calls in stream order are safe.
 */
int dcd_verify_greedy_noalloc(const dcd_problem *p, const dcd_inputs *in, const dcd_outputs *out,
                              void *hip_stream);

/* bytes of device memory the allocation-free entry point holds per GPU */
size_t dcd_noalloc_max_bytes(void);

/* static description of a return code (never NULL) */
const char *dcd_error_string(int code);

/* ABI version of this header: 7 (2: dcd_outputs gained row_argmax_expert and row_kl;
   3: dcd_verify_sample takes trees; 4: dcd_propose; 5: the final RMS normalisation;
   6: dcd_verify_greedy_noalloc; 7: sequence status DCD_SEQ_WALK_TIMEOUT) */
int dcd_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DCD_H */
