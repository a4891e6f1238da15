// Internal declarations of libdcd (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dcd {

// LM-head tile geometry (gfx950: 64-lane waves, 16x16 MFMA blocks).  Every LM-head
// kernel reduces its logits per vocabulary tile of kTileTokens tokens; the
// streaming kernel has two row shapes, 64 and 128 rows per workgroup.
constexpr int kWaveSize = 64;
constexpr int kTileTokens = 256;                     // tokens per vocabulary tile
constexpr int kStreamRowsSmall = 64;                 // rows per workgroup up to 64 rows
constexpr int kStreamRowsLarge = 128;                // rows per workgroup from 65 to 511 rows
constexpr int kWordsPerTile = kTileTokens / 32;      // candidate bit words per row and tile
constexpr int kRowInfo = 16;                         // floats of per-row results
constexpr int kMaxNodes = 4096;                      // nodes per sequence (staged in LDS)
constexpr int kWideRows = 256;                       // rows per workgroup of the many-row LM-head kernel
constexpr int kWideMinRows = 512;                    // rows from which that kernel is used
constexpr int kWalkMaxGroup = 64;                    // workgroups per sequence of the spread walk

// rowinfo slots (floats; the argmax is stored as an int bit pattern)
enum {
    RI_MAXP = 0, RI_LSEP, RI_LSEQ, RI_LOGZ, RI_TOP1, RI_MARGIN, RI_COUNT, RI_SIGNAL,
    RI_THRESH = 8, RI_ARGMAX = 9, RI_ARGMAX_P = 10, RI_KL_PQ = 11, RI_KL_PCD = 12
};

enum ElemType { kF32 = 0, kBF16 = 1 };

// Everything a launch needs, resolved on the host.
struct Plan {
    int B, N, R, V, dp, dq, dtype;
    int ntiles;        // ceil(V / kTileTokens)
    int rows_blk;      // rows per workgroup of the streaming LM-head kernel (64 or 128)
    int nrb;           // ceil(R / rows_blk)
    int wstride;       // candidate bit words per row (ntiles * kWordsPerTile)
    float log_theta;   // ln(plaus_thresh); -inf when the mask is off
    float s;           // cd_strength
    float inv_T;       // 1 / temperature (1 for greedy)
    int full;          // plaus_thresh = 0: the untruncated target (every token in the support);
                       // no candidates, dense logits instead
    int zstride;       // ntiles * kTileTokens: row stride of the dense logit arrays
    int store_y;       // full, and sampled or proposing: the dense y rows are written (y_full)
    int final_norm;    // the rows of h_* are normalised first (into hn_p, hn_q)
    float norm_eps;
    // workspace carve-up
    float4 *partials;  // [R][ntiles]   (max_p, sumexp_p, max_q, sumexp_q) per vocabulary tile
    // masked target (full = 0)
    float2 *cand;      // [R][V]        (z_p, z_q) of candidate tokens (sparse)
    uint32_t *bits;    // [R][wstride]  candidate bitmap
    // untruncated target (full = 1)
    float *zp_full;    // [R][zstride]  expert logits (divided by T), where the 128-row shape keeps
                       //   them between its two passes
    float *y_full;     // [R][zstride]  sampled and proposal calls: y = (1+s) z_p - s z_q (logits
                       //   divided by T), so pi_CD(t) = exp(y(t) - target_shift(row))
    double *resbuf;    // [B][2][zstride] sampled verification: the residual after the
                       //   last applied rejection of the walk's current node (two rows)
    float4 *ypart;     // [R][ntiles][2] per tile, over y = (1+s) z_p - s z_q:
                       //   (max y, sum exp(y - max y), second-best y, sum exp(z_p - max_p)(z_p - z_q))
                       //   (argmax bits, z_p and z_q at the argmax, bits of the lowest
                       //    token whose z_p is the tile's expert max)
    uint32_t *ctl;     // [2] at the workspace's start: the call counter and the ready word (below)
    float *rowinfo;    // [R][kRowInfo]
    int *tcount;       // [R][ntiles]   candidates per (row, tile); bitmap words valid where > 0
    uint32_t *bound;   // [kBoundCopies][R] running lower bound on max z_p (bound_key; 0: none)
    float4 *nodez;     // [R]           node r's token under its parent row: (z_p, z_q) as a candidate
                       //   (NaN: not one), (z_p, z_q) by dot product (NaN: not computed)
    int *seqdone;      // [B]           rows of each sequence finished by the combine step
    int *seqfail;      // [B]           (after seqdone, cleared with it) sampled, masked: a row of
                       //   the sequence could not settle its children's walk decisions
    double *wratio;    // [R]           sampled, masked: node r's accept ratio under its parent
                       //   (every earlier sibling rejected; -1: rejected whatever u is)
    int *wterm;        // [R]           sampled, masked: the token emitted if the walk ends at
                       //   node r (-1: an empty support)
    // untruncated sampled verification with the walk spread over a group of
    // workgroups per sequence (walk_kernel; walk_group = 0: the finish kernel walks)
    int walk_group;    // workgroups per sequence
    int *walkbar;      // [B][2] barrier arrivals of each group, and a failed-wait flag
    double *walkpart;  // [B][2][kWalkMaxGroup] the group's slice sums of a pass (two passes kept)
    void *hn_p, *hn_q; // [R][d_p], [R][d_q] final_norm: the normalised hidden states
};

struct Inputs {
    const void *hp, *hq, *wp, *wq;
    const float *bp, *bq;
    const int32_t *parents, *tokens;
    const void *gp, *gq;  // scales of the final RMS normalisation (final_norm)
};

struct Outputs {
    int32_t *accept_len, *accept_path, *next_token, *status, *row_argmax;
    float *row_stats, *node_stats;
    int32_t *row_argmax_p;  // argmax of pi_p per row
    float *row_kl;          // [R][2] D_KL(pi_p||pi_q), D_KL(pi_p||pi_CD)
};

struct SampleInputs {
    const float *draft_probs, *u_acc, *u_res;
};

// float -> unsigned keys whose order is the float order, every key above 0 (so an
// all-zero word is an empty bound, below every float; for atomicMax)
__device__ __forceinline__ uint32_t bound_key(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // -inf -> 0x007fffff > 0
}
__device__ __forceinline__ float bound_value(uint32_t k) {
    if (k == 0u) return -INFINITY;
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// The streaming LM-head kernel keeps the running row bounds in one copy per XCD (a
// workgroup raises the copy of its XCD, blockIdx.x % 8): every tile's expert
// epilogue raises the bounds of its rows at about the same time, and 8 copies
// divide the contention on each word by 8.  A reader takes the max over the
// copies, a lower bound on the row's max either way.  The many-row kernel, whose
// epilogues are spread out, uses copy 0 alone.
constexpr int kBoundCopies = 8;

__device__ __forceinline__ void raise_bound(uint32_t *bound, int R, int row, float v) {
    atomicMax(&bound[(int)(blockIdx.x % kBoundCopies) * R + row], bound_key(v));
}

__device__ __forceinline__ float read_bound(const uint32_t *bound, int R, int row) {
    uint32_t k = __atomic_load_n(&bound[row], __ATOMIC_RELAXED);
#pragma unroll
    for (int c = 1; c < kBoundCopies; ++c) k = max(k, __atomic_load_n(&bound[c * R + row], __ATOMIC_RELAXED));
    return bound_value(k);
}

// Per-call clearing of the bounds and the per-sequence row counters, inside the
// LM-head launch.  The workspace starts with two words: ctl[0] counts the calls
// made on it and ctl[1] is the ready word.  Workgroup 0 of the LM-head kernel
// clears the bounds and counters, then stores ready = count + 1 (release); every
// other workgroup waits for that value (acquire) before it touches a bound, which
// it first does at its expert epilogue, long after.  The last kernel of the call
// advances the count (advance_call), so the next call waits for a new value.
// The wait is bounded: a workgroup that gives up prunes nothing and raises no
// bound (its candidates are then a larger superset of the mask, still exact).
__device__ __forceinline__ void clear_call_state(const uint32_t *ctl, uint32_t *bound, int nbound,
                                                 int *seqdone, int B) {
    const uint32_t count = ctl[0];
    for (int i = threadIdx.x; i < nbound; i += blockDim.x) bound[i] = 0u;
    for (int i = threadIdx.x; i < B; i += blockDim.x) seqdone[i] = 0;
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_store(const_cast<uint32_t *>(ctl) + 1, count + 1, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Called by every thread of a workgroup (contains a barrier); true once the bounds
// of this call are cleared, false if the wait gave up.
// The same in two halves, so that the first reads travel while the caller works:
// thread 0 reads the call count and the ready word (start_call_state), and later
// checks them, polls on if the word is not there yet, and shares the outcome with
// the workgroup (finish_call_state, which every thread calls).
struct CallState {
    uint32_t want, seen;
};
__device__ __forceinline__ CallState start_call_state(const uint32_t *ctl) {
    CallState c{0u, 0u};
    if (threadIdx.x == 0) {
        c.want = ctl[0] + 1;
        c.seen = __hip_atomic_load(ctl + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return c;
}
__device__ __forceinline__ bool finish_call_state(const uint32_t *ctl, CallState c) {
    __shared__ int ok;
    if (threadIdx.x == 0) {
        int tries = 0;
        while (c.seen != c.want && ++tries < (1 << 16)) {
            __builtin_amdgcn_s_sleep(8);
            c.seen = __hip_atomic_load(ctl + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        ok = tries < (1 << 16);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    return ok != 0;
}

__device__ __forceinline__ bool await_call_state(const uint32_t *ctl) {
    __shared__ int ok;
    if (threadIdx.x == 0) {
        const uint32_t want = ctl[0] + 1;
        int tries = 0;
        while (__hip_atomic_load(ctl + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want &&
               ++tries < (1 << 16))
            __builtin_amdgcn_s_sleep(8);
        ok = tries < (1 << 16);
        // after the poll, once for the workgroup (it invalidates the CU's and the
        // XCD's caches, which all of its waves share)
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    return ok != 0;
}

// The call's last kernel advances the call count (one thread of one workgroup).
__device__ __forceinline__ void advance_call(uint32_t *ctl) { ctl[0] = ctl[0] + 1; }

// Untruncated target: log pi_CD(t) = y(t) - shift, with y = (1+s) z_p - s z_q and
// shift = (1+s) lse_p - s lse_q + log Z of the row (cd = y - (1+s) lse_p + s lse_q).
__device__ __forceinline__ float target_shift(const float *rowinfo_row, float s) {
    return (1.f + s) * rowinfo_row[RI_LSEP] - s * rowinfo_row[RI_LSEQ] + rowinfo_row[RI_LOGZ];
}

// Untruncated target: statistics of y = (1+s) z_p - s z_q over a set of tokens.
// cd = y - (1+s) lse_p + s lse_q, so the argmax, margin and log-normaliser of the
// cd score follow from these and the two models' normalisers.
struct YStat {
    float y1;   // best y (-inf when empty)
    int i1;     // its token (lowest id on ties; -1 when empty)
    float y2;   // second-best y
    float ys;   // sum of exp(y - y1)
    float zp1, zq1;  // z_p, z_q at i1
    float a;    // sum of exp(z_p - tile max_p) * (z_p - z_q)
    int ip;     // lowest token whose z_p equals the tile's expert max (-1: none seen)
};

__device__ __forceinline__ YStat ystat_merge(const YStat &u, const YStat &v) {
    const bool u_wins = v.i1 < 0 || (u.i1 >= 0 && (u.y1 > v.y1 || (u.y1 == v.y1 && u.i1 < v.i1)));
    const YStat &w = u_wins ? u : v, &l = u_wins ? v : u;
    YStat r = w;
    if (l.i1 >= 0) {
        r.y2 = fmaxf(w.y2, l.y1);
        r.ys = w.ys + l.ys * __builtin_amdgcn_exp2f((l.y1 - w.y1) * 1.4426950408889634f);
    }
    r.a = u.a + v.a;
    r.ip = (int)min((unsigned)u.ip, (unsigned)v.ip);  // -1 (none) is the largest unsigned
    return r;
}

size_t workspace_layout(Plan &p, char *base);  // fills the pointers when base != nullptr

// final RMS normalisation of both models' rows into hn_p / hn_q (final_norm)
hipError_t launch_rmsnorm(const Plan &p, const Inputs &in, hipStream_t st);
// LM heads with softmax partials and candidates (clears bound and seqdone itself)
hipError_t launch_lmhead(const Plan &p, const Inputs &in, hipStream_t st);
// advances the workspace's call count (after an LM-head launch no other kernel follows)
hipError_t launch_advance_call(const Plan &p, hipStream_t st);
// the many-row variant (bf16, R >= kWideMinRows): same outputs
bool use_wide_lmhead(const Plan &p);
hipError_t launch_lmhead_wide(const Plan &p, const Inputs &in, hipStream_t st);
// the streaming LM-head kernel in its two row shapes (p.rows_blk selects)
hipError_t launch_lmhead_rows64(const Plan &p, const Inputs &in, hipStream_t st);
hipError_t launch_lmhead_rows128(const Plan &p, const Inputs &in, hipStream_t st);
// proposals from the recombined heads (rows only, after launch_lmhead)
struct ProposeOutputs {
    const float *u;
    int32_t *tokens;
    float *probs;
    int32_t *argmax;
};
hipError_t launch_propose(const Plan &p, const Inputs &in, const ProposeOutputs &out, hipStream_t st);
// per-row combination and per-sequence verification (greedy when smp is null)
hipError_t launch_finish(const Plan &p, const Inputs &in, const Outputs &out,
                         const SampleInputs *smp, hipStream_t st);
// untruncated sampled verification: workgroups per sequence for the spread walk
// (0 when there are too many sequences for one workgroup per CU), and that launch
int walk_group_size(const Plan &p, hipStream_t st);
hipError_t launch_walk(const Plan &p, const Inputs &in, const Outputs &out, const SampleInputs &smp,
                       hipStream_t st);

}  // namespace dcd
