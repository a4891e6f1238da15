// Per-row combination of the LM-head partials and per-sequence verification, in
// one launch.
//
// Row phase (one workgroup per row):
//   max_p and the log-normalisers of both models from the per-tile
//   (max, sum exp) pairs; the plausibility mask z_p >= max_p + ln theta
//   (Sec. 2.1) over the candidate tokens; the cd score
//   (1+s)(z_p - lse_p) - s(z_q - lse_q) of Eq. (1); its log normaliser over the
//   mask, argmax (lowest id on ties) and top-2 margin; and the row's own draft
//   token's logits under its parent row.
// Sequence phase (the workgroup that completes a sequence's last row):
//   tree / token checks, draft-token statistics under the parent row, then either
//   the greedy walk from the root or Alg. 1's accept test with the residual /
//   bonus draw along a chain.
// Repeated calls are bit-identical.  All reductions run in a fixed order, and
// nothing read depends on timing: which vocabulary tiles keep their candidates
// depends on when each read the running bound of the LM-head step, so the row
// phase takes only the tiles whose own expert max reaches the row's threshold
// (those are never dropped, and hold every mask member), and a draft token's
// logits come from the candidates only when the token is a mask member.
#include <atomic>

#include "dcd.h"
#include "dcd_internal.h"

namespace dcd {
namespace {

constexpr int NT = 256;                  // threads of the finish kernel (4 waves)
constexpr int kTileU4 = kWordsPerTile / 4;  // 16-byte bitmap words per vocabulary tile
constexpr int kTilesPerLane = kTileTokens <= 256 ? 8 : 4;  // tiles a lane takes per pass
static_assert(kWordsPerTile % 4 == 0, "a tile's bitmap is whole 16-byte words");
constexpr int kPass = kWaveSize * kTilesPerLane;
constexpr int kList = 1024;              // candidate ids gathered per round
// masked target, sampled verification: the walk's decisions settled per row (settle_children)
constexpr int kMembers = kList;          // mask members of a row kept in LDS
constexpr int kMaxKids = 64;             // children of a node
constexpr int kKidQ = 4096;              // proposal values gathered: children x members
constexpr size_t kSettleLds = (size_t)kMaxKids * 3 * 4 + (size_t)kMembers * 8 + (size_t)kKidQ * 4;

struct Lse {  // running log-sum-exp: value = m + log(s)
    float m, s;
};

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    if (a.m == -INFINITY) return b;
    if (b.m == -INFINITY) return a;
    const float m = fmaxf(a.m, b.m);
    return Lse{m, a.s * __expf(a.m - m) + b.s * __expf(b.m - m)};
}

// log-sum-exp with a weighted sum alongside: value = m + log(s), and
// sum_x exp(z_x - m) w_x = a (rescaled with s)
struct LseW {
    float m, s, a;
};

__device__ __forceinline__ LseW lsew_merge(LseW x, LseW y) {
    if (x.m == -INFINITY) return y;
    if (y.m == -INFINITY) return x;
    const float m = fmaxf(x.m, y.m), fx = __expf(x.m - m), fy = __expf(y.m - m);
    return LseW{m, x.s * fx + y.s * fy, x.a * fx + y.a * fy};
}

// largest value with the lowest id on ties (-1 = none, ordered last)
struct Best {
    float v;
    int id;
};

__device__ __forceinline__ Best best_merge(Best x, Best y) {
    return (x.v > y.v || (x.v == y.v && (unsigned)x.id < (unsigned)y.id)) ? x : y;
}

struct Top2 {  // best value and id, runner-up value; both models' logits at the best
    float v;
    int id;
    float v2;
    float zp, zq;
};

__device__ __forceinline__ Top2 top2_merge(Top2 a, Top2 b) {
    const bool a_wins = b.id < 0 || (a.id >= 0 && (a.v > b.v || (a.v == b.v && a.id < b.id)));
    const Top2 w = a_wins ? a : b, l = a_wins ? b : a;
    return Top2{w.v, w.id, fmaxf(w.v2, l.id >= 0 ? l.v : -INFINITY), w.zp, w.zq};
}

// ---------------------------------------------------------------------------
// Wave-level reductions (64 lanes).  Each is a fixed tree towards lane 0, so the
// result does not depend on timing; only lane 0's value is meaningful.
__device__ __forceinline__ Lse wave_lse(Lse x) {
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1)
        x = lse_merge(x, Lse{__shfl_down(x.m, d, kWaveSize), __shfl_down(x.s, d, kWaveSize)});
    return x;
}

__device__ __forceinline__ LseW wave_lsew(LseW x) {
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1)
        x = lsew_merge(x, LseW{__shfl_down(x.m, d, kWaveSize), __shfl_down(x.s, d, kWaveSize),
                               __shfl_down(x.a, d, kWaveSize)});
    return x;
}

__device__ __forceinline__ Best wave_best(Best x) {
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1)
        x = best_merge(x, Best{__shfl_down(x.v, d, kWaveSize), __shfl_down(x.id, d, kWaveSize)});
    return x;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1) x += __shfl_down(x, d, kWaveSize);
    return x;
}

// Orders one wave's LDS writes before its later LDS reads of other lanes' data
// (a wave's LDS operations complete in issue order; this stops the compiler
// from moving memory operations across the point).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// exclusive prefix sum over the wave; *total receives the sum of all lanes
__device__ __forceinline__ int wave_exclusive_scan(int x, int lane, int *total) {
    int incl = x;
#pragma unroll
    for (int d = 1; d < kWaveSize; d <<= 1) {
        const int y = __shfl_up(incl, d, kWaveSize);
        if (lane >= d) incl += y;
    }
    *total = __shfl(incl, kWaveSize - 1, kWaveSize);
    return incl - x;
}

// Dot product h . w over d elements by one wave (fp32, fixed order); lane 0 holds it.
template <int DT>
__device__ float wave_dot(const void *h, const void *w, int d, int lane) {
    float acc = 0.f;
    if constexpr (DT == kBF16) {
        const uint16_t *hr = (const uint16_t *)h, *wr = (const uint16_t *)w;
        // unrolled 8 times: a 4096-element row is one round of loads
#pragma unroll 8
        for (int k = lane * 8; k < d; k += kWaveSize * 8) {
            const uint4 hv = *(const uint4 *)(hr + k), wv = *(const uint4 *)(wr + k);
            const uint32_t hs[4] = {hv.x, hv.y, hv.z, hv.w}, ws[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc += __uint_as_float(hs[e] << 16) * __uint_as_float(ws[e] << 16);
                acc += __uint_as_float(hs[e] & 0xffff0000u) * __uint_as_float(ws[e] & 0xffff0000u);
            }
        }
    } else {
        const float *hr = (const float *)h, *wr = (const float *)w;
#pragma unroll 8
        for (int k = lane * 4; k < d; k += kWaveSize * 4) {
            const float4 hv = *(const float4 *)(hr + k), wv = *(const float4 *)(wr + k);
            acc += hv.x * wv.x + hv.y * wv.y + hv.z * wv.z + hv.w * wv.w;
        }
    }
    return wave_sum(acc);
}

__device__ __forceinline__ uint4 mask4(uint4 v, uint32_t m) {
    return uint4{v.x & m, v.y & m, v.z & m, v.w & m};
}

__device__ __forceinline__ int popc_tile(const uint4 (&w)[kTileU4]) {
    int c = 0;
#pragma unroll
    for (int q = 0; q < kTileU4; ++q) c += __popc(w[q].x) + __popc(w[q].y) + __popc(w[q].z) + __popc(w[q].w);
    return c;
}

// Writes the ids of the set bits of one tile's bitmap words whose running index
// (*idx, advanced over every set bit) falls in [lo, lo + kList) to list[].
__device__ __forceinline__ void emit_ids(const uint4 (&w)[kTileU4], int tile, int lo, int *idx,
                                         int *list) {
#pragma unroll
    for (int e = 0; e < kWordsPerTile; ++e) {
        const uint4 q = w[e / 4];
        uint32_t b = e % 4 == 0 ? q.x : e % 4 == 1 ? q.y : e % 4 == 2 ? q.z : q.w;
        while (b) {
            if (*idx >= lo && *idx < lo + kList)
                list[*idx - lo] = (tile * kWordsPerTile + e) * 32 + __ffs(b) - 1;
            ++*idx;
            b &= b - 1;
        }
    }
}

// Shared memory of the finish kernel (the dynamic part holds the sequence's
// parents, tokens and row argmax: 12 bytes per node).
struct Smem {
    int list[kList];    // candidate ids (row phase: wave 0; draw: whole group)
    double wts[kList];  // draw weights; in a sampled call's row phase, the row's mask
                        //   members in token order (token, cd score) packed (kMembers)
    int mcount;         // sampled, masked: the row's mask members (more than kMembers: not kept)
    float mlogz;        //   and its log Z
    int nkids;          //   and its node's children (the first kMaxKids listed in LDS)
    float4 nodez;       // the row's draft token under its parent row (waves 1-3)
    int node_ok;        // nodez is to be written
    int wave_tot[NT / kWaveSize];
    int flag[4];
    int ints[4];
    double dbl, dbl2;
};

// Writes a row's results: rowinfo (for the sequence phase) and the optional outputs.
__device__ __forceinline__ void write_row(const Plan &P, int row, const float (&ri)[kRowInfo],
                                          const Outputs &out) {
    float4 *dst = reinterpret_cast<float4 *>(P.rowinfo + (size_t)row * kRowInfo);
#pragma unroll
    for (int k = 0; k < kRowInfo / 4; ++k) dst[k] = float4{ri[4 * k], ri[4 * k + 1], ri[4 * k + 2], ri[4 * k + 3]};
    if (out.row_argmax) out.row_argmax[row] = __float_as_int(ri[RI_ARGMAX]);
    if (out.row_stats) {
#pragma unroll
        for (int k = 0; k < 8; ++k) out.row_stats[(size_t)row * 8 + k] = ri[k];
    }
    if (out.row_argmax_p) out.row_argmax_p[row] = __float_as_int(ri[RI_ARGMAX_P]);
    if (out.row_kl) {
        out.row_kl[(size_t)row * 2] = ri[RI_KL_PQ];
        out.row_kl[(size_t)row * 2 + 1] = ri[RI_KL_PCD];
    }
}

// Row statistics of the untruncated target (wave 0): the two models' normalisers
// from the per-tile (max, sum exp) pairs and the statistics of
// y = (1+s) z_p - s z_q from the per-tile y statistics, both fetched in one round;
// cd = y - (1+s) lse_p + s lse_q over the whole vocabulary.  Alongside: the
// expert's top-1 (the first tile holding max z_p, and that tile's lowest token at
// its max) and D_KL(pi_p || pi_q) = sum_x pi_p (z_p - z_q) - lse_p + lse_q, whose sum
// is merged like the expert's sum of exp (per tile: sum exp(z_p - tile max)(z_p - z_q));
// D_KL(pi_p || pi_CD) = log Z - s D_KL(pi_p || pi_q) by the KL-decomposition lemma.
__device__ __forceinline__ void row_stats_full(const Plan &P, int row, int lane, const Outputs &out) {
    const float4 *pr = P.partials + (size_t)row * P.ntiles;
    const float4 *yp = P.ypart + (size_t)row * P.ntiles * 2;
    LseW lp{-INFINITY, 0.f, 0.f};
    Lse lq{-INFINITY, 0.f};
    Best top_p{-INFINITY, -1};
    YStat st{-INFINITY, -1, -INFINITY, 0.f, 0.f, 0.f, 0.f, -1};
    for (int base = 0; base < P.ntiles; base += kPass) {
        float4 v[kTilesPerLane], u[kTilesPerLane], w2[kTilesPerLane];
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            const int t = min(base + lane + k * kWaveSize, P.ntiles - 1);
            v[k] = pr[t];
            u[k] = yp[2 * t];
            w2[k] = yp[2 * t + 1];
        }
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            if (base + lane + k * kWaveSize >= P.ntiles) continue;
            lp = lsew_merge(lp, LseW{v[k].x, v[k].y, u[k].w});
            lq = lse_merge(lq, Lse{v[k].z, v[k].w});
            top_p = best_merge(top_p, Best{v[k].x, __float_as_int(w2[k].w)});
            st = ystat_merge(st, YStat{u[k].x, __float_as_int(w2[k].x), u[k].z, u[k].y, w2[k].y, w2[k].z,
                                       0.f, -1});
        }
    }
    lp = wave_lsew(lp);
    lq = wave_lse(lq);
    top_p = wave_best(top_p);
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1)
        st = ystat_merge(st, YStat{__shfl_down(st.y1, d, kWaveSize), __shfl_down(st.i1, d, kWaveSize),
                                   __shfl_down(st.y2, d, kWaveSize), __shfl_down(st.ys, d, kWaveSize),
                                   __shfl_down(st.zp1, d, kWaveSize), __shfl_down(st.zq1, d, kWaveSize),
                                   0.f, -1});
    if (lane != 0) return;
    const float max_p = lp.m, lse_p = lp.m + __logf(lp.s), lse_q = lq.m + __logf(lq.s);
    const float shift = -(1.f + P.s) * lse_p + P.s * lse_q;  // cd - y
    float ri[kRowInfo] = {};
    ri[RI_MAXP] = max_p;
    ri[RI_LSEP] = lse_p;
    ri[RI_LSEQ] = lse_q;
    ri[RI_LOGZ] = st.y1 + __logf(st.ys) + shift;
    ri[RI_TOP1] = st.y1 + shift;
    ri[RI_MARGIN] = st.y1 - st.y2;  // +inf with a single token
    ri[RI_COUNT] = (float)P.V;
    ri[RI_SIGNAL] = st.i1 >= 0 ? (st.zp1 - lse_p) - (st.zq1 - lse_q) : NAN;
    ri[RI_THRESH] = max_p + P.log_theta;  // -inf: no mask
    ri[RI_ARGMAX] = __int_as_float(st.i1);
    ri[RI_ARGMAX_P] = __int_as_float(top_p.id);
    const float kl_pq = lp.a / lp.s - lse_p + lse_q;
    ri[RI_KL_PQ] = kl_pq;
    ri[RI_KL_PCD] = ri[RI_LOGZ] - P.s * kl_pq;
    write_row(P, row, ri, out);
}

// ---------------------------------------------------------------------------
// Row phase.  wave 0: the row's statistics; waves 1-3: the row as a draft node,
// its token's logits under the parent row, left in sm.nodez (node_ok set) for the
// thread that counts the row.
template <int DT>
__device__ __forceinline__ void combine_row(const Plan &P, const Inputs &in, const Outputs &out, int row, int lane,
                            int wave, Smem &sm, bool members = false) {
    const bool want_node_logits = out.node_stats != nullptr;
    if (wave >= 1) {
        if (!in.parents) return;  // rows without a tree (proposals)
        const int i = row % P.N;
        if (i == 0) return;
        const int j = in.parents[row], x = in.tokens[row];
        if (j < 0 || j >= i || x < 0 || x >= P.V) return;  // the sequence is rejected later
        const size_t rowj = (size_t)(row - i + j);
        const size_t esz = DT == kBF16 ? 2 : 4;
        // the three parts go to the three waves, so their loads are in flight together
        if (P.full) {  // every token is in the support
            // the logits are not stored densely (only y, for sampled calls): the node's,
            // needed for the sampled walk and for its statistics, are dot products
            const bool need = want_node_logits || P.store_y;
            if (wave == 1 && lane == 0) {
                if (!need) sm.nodez = float4{0.f, 0.f, 0.f, 0.f};
                sm.node_ok = 1;
            } else if (wave == 2 && need) {
                float zp = wave_dot<DT>((const char *)in.hp + rowj * P.dp * esz,
                                        (const char *)in.wp + (size_t)x * P.dp * esz, P.dp, lane);
                if (lane == 0) sm.nodez.x = sm.nodez.z = (zp + (in.bp ? in.bp[x] : 0.f)) * P.inv_T;
            } else if (wave == 3 && need) {
                float zq = wave_dot<DT>((const char *)in.hq + rowj * P.dq * esz,
                                        (const char *)in.wq + (size_t)x * P.dq * esz, P.dq, lane);
                if (lane == 0) sm.nodez.y = sm.nodez.w = (zq + (in.bq ? in.bq[x] : 0.f)) * P.inv_T;
            }
            return;
        }
        // The parent row's threshold is not known yet, so both forms are kept: the
        // candidate's logits (NaN when the token is not a candidate of a kept tile)
        // and, when node statistics are wanted, a dot product.  The sequence phase
        // takes the candidate's only for a mask member, whose tile is never dropped,
        // so the choice does not depend on which tiles the running bound pruned.
        if (wave == 1) {
            if (lane == 0) {  // count, bitmap word and candidate slot fetched together
                const int tcnt = P.tcount[rowj * P.ntiles + x / kTileTokens];
                const uint32_t word = P.bits[rowj * P.wstride + (x >> 5)];
                const float2 c = P.cand[rowj * P.V + x];
                const bool cand = tcnt > 0 && (word >> (x & 31) & 1u);
                sm.nodez.x = cand ? c.x : NAN;
                sm.nodez.y = cand ? c.y : NAN;
                if (!want_node_logits) sm.nodez.z = sm.nodez.w = NAN;
                sm.node_ok = 1;
            }
        } else if (want_node_logits && wave == 2) {
            float zp = wave_dot<DT>((const char *)in.hp + rowj * P.dp * esz,
                                    (const char *)in.wp + (size_t)x * P.dp * esz, P.dp, lane);
            if (lane == 0) sm.nodez.z = (zp + (in.bp ? in.bp[x] : 0.f)) * P.inv_T;
        } else if (want_node_logits && wave == 3) {
            float zq = wave_dot<DT>((const char *)in.hq + rowj * P.dq * esz,
                                    (const char *)in.wq + (size_t)x * P.dq * esz, P.dq, lane);
            if (lane == 0) sm.nodez.w = (zq + (in.bq ? in.bq[x] : 0.f)) * P.inv_T;
        }
        return;
    }
    int *list = sm.list;
    if (P.full) {
        row_stats_full(P, row, lane, out);
        return;
    }

    const float4 *pr = P.partials + (size_t)row * P.ntiles;
    const int *tc = P.tcount + (size_t)row * P.ntiles;
    const uint4 *bw = reinterpret_cast<const uint4 *>(P.bits + (size_t)row * P.wstride);
    const float2 *cz = P.cand + (size_t)row * P.V;

    // the first pass's partials, counts and bitmap words are fetched together
    float4 v[kTilesPerLane];
    uint4 w[kTilesPerLane][kTileU4];
    // Loads are issued unconditionally from clamped indices and masked
    // afterwards (with selects), so that all of them are in flight together.
    int c[kTilesPerLane];
    float tm[kTilesPerLane];  // the tile's expert max (its partial)
    auto issue_partials = [&](int base) {
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) v[k] = pr[min(base + lane + k * kWaveSize, P.ntiles - 1)];
    };
    auto issue_cands = [&](int base) {
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            const int t = min(base + lane + k * kWaveSize, P.ntiles - 1);
            c[k] = tc[t];
            tm[k] = pr[t].x;
#pragma unroll
            for (int q = 0; q < kTileU4; ++q) w[k][q] = bw[kTileU4 * t + q];
        }
    };
    auto mask_partials = [&](int base) {
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            const bool ok = base + lane + k * kWaveSize < P.ntiles;
            v[k] = ok ? v[k] : float4{-INFINITY, 0.f, -INFINITY, 0.f};
        }
    };
    // (called once thr is known) the words of a tile count only if the tile kept
    // candidates (otherwise they are stale) and its expert max reaches thr: only
    // such a tile can hold mask members, and the LM-head step never drops it,
    // whatever the timing; the others are dropped here too
    float thr = 0.f;
    auto mask_cands = [&](int base) {
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            const uint32_t keep =
                (base + lane + k * kWaveSize < P.ntiles && c[k] > 0 && tm[k] >= thr) ? ~0u : 0u;
#pragma unroll
            for (int q = 0; q < kTileU4; ++q) w[k][q] = mask4(w[k][q], keep);
        }
    };
    issue_partials(0);
    issue_cands(0);
    __builtin_amdgcn_sched_barrier(0);
    mask_partials(0);

    // 1. per-tile (max, sum exp) pairs of both models -> max_p, lse_p, lse_q
    Lse lp{-INFINITY, 0.f}, lq{-INFINITY, 0.f};
    for (int base = 0;;) {
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            lp = lse_merge(lp, Lse{v[k].x, v[k].y});
            lq = lse_merge(lq, Lse{v[k].z, v[k].w});
        }
        base += kPass;
        if (base >= P.ntiles) break;
        issue_partials(base);
        mask_partials(base);
    }
    // both trees one level at a time (the same merges as two separate trees)
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1) {
        const Lse op{__shfl_down(lp.m, d, kWaveSize), __shfl_down(lp.s, d, kWaveSize)};
        const Lse oq{__shfl_down(lq.m, d, kWaveSize), __shfl_down(lq.s, d, kWaveSize)};
        lp = lse_merge(lp, op);
        lq = lse_merge(lq, oq);
    }
    const float max_p = __shfl(lp.m, 0, kWaveSize);
    const float lse_p = __shfl(lp.m + __logf(lp.s), 0, kWaveSize);
    const float lse_q = __shfl(lq.m + __logf(lq.s), 0, kWaveSize);
    thr = max_p + P.log_theta;
    const float s = P.s;

    // 2. candidates of the tiles that kept any, compacted into LDS so that their
    //    logits are fetched in one round
    Lse lc{-INFINITY, 0.f};
    Top2 best{-INFINITY, -1, -INFINITY, 0.f, 0.f};
    int count = 0;
    int top_p = -1;  // the expert's top-1: the lowest candidate whose z_p is max_p
    // members: the mask members (token, cd) in token order, for the children's walk
    // decisions settled in the same workgroup (kept: how many seen so far)
    unsigned long long *const mlist = reinterpret_cast<unsigned long long *>(sm.wts);
    int kept = 0;
    for (int base = 0; base < P.ntiles; base += kPass) {
        if (base > 0) issue_cands(base);
        mask_cands(base);
        // list positions in token order: tile base + lane + k * 64 is the (k * 64 +
        // lane)-th tile of the pass, so the tiles are counted k-major
        int nset[kTilesPerLane], first[kTilesPerLane];
        int total = 0;
#pragma unroll
        for (int k = 0; k < kTilesPerLane; ++k) {
            nset[k] = popc_tile(w[k]);
            int tk;
            first[k] = total + wave_exclusive_scan(nset[k], lane, &tk);
            total += tk;
        }
        for (int lo = 0; lo < total; lo += kList) {
#pragma unroll
            for (int k = 0; k < kTilesPerLane; ++k)
                if (nset[k] > 0 && first[k] < lo + kList && first[k] + nset[k] > lo) {
                    int idx = first[k];
                    emit_ids(w[k], base + lane + k * kWaveSize, lo, &idx, list);
                }
            wave_lds_sync();
            const int n = min(kList, total - lo);
            for (int mb = 0; mb < n; mb += kWaveSize) {
                const int m = mb + lane;
                const int t = list[min(m, n - 1)];
                const float2 c = cz[t];
                const bool member = m < n && c.x >= thr;
                const float cd = (1.f + s) * (c.x - lse_p) - s * (c.y - lse_q);
                if (members) {  // kept in token order: list order, then lane order
                    const unsigned long long mask = __ballot(member);
                    const int pos = kept + __popcll(mask & ((1ull << lane) - 1ull));
                    if (member && pos < kMembers)
                        mlist[pos] = (unsigned long long)(uint32_t)t << 32 | __float_as_uint(cd);
                    kept += __popcll(mask);
                }
                if (!member) continue;
                ++count;
                top_p = c.x == max_p ? (int)min((unsigned)top_p, (unsigned)t) : top_p;
                best = top2_merge(best, Top2{cd, t, -INFINITY, c.x, c.y});
                lc = lse_merge(lc, Lse{cd, 1.f});
            }
            wave_lds_sync();
        }
    }
    // the four trees one level at a time (the same merges as separate trees)
#pragma unroll
    for (int d = kWaveSize / 2; d > 0; d >>= 1) {
        const Lse oc{__shfl_down(lc.m, d, kWaveSize), __shfl_down(lc.s, d, kWaveSize)};
        const Top2 ob{__shfl_down(best.v, d, kWaveSize), __shfl_down(best.id, d, kWaveSize),
                      __shfl_down(best.v2, d, kWaveSize), __shfl_down(best.zp, d, kWaveSize),
                      __shfl_down(best.zq, d, kWaveSize)};
        const int on = __shfl_down(count, d, kWaveSize), ot = __shfl_down(top_p, d, kWaveSize);
        lc = lse_merge(lc, oc);
        best = top2_merge(best, ob);
        count += on;
        top_p = (int)min((unsigned)top_p, (unsigned)ot);
    }

    if (lane == 0) {
        const float logZ = lc.m + __logf(lc.s);
        if (members) {
            sm.mcount = kept;
            sm.mlogz = logZ;
        }
        // the best candidate's logits came along with it (no second fetch)
        const float signal = best.id >= 0 ? (best.zp - lse_p) - (best.zq - lse_q) : NAN;
        float ri[kRowInfo] = {};
        ri[RI_MAXP] = max_p;
        ri[RI_LSEP] = lse_p;
        ri[RI_LSEQ] = lse_q;
        ri[RI_LOGZ] = logZ;
        ri[RI_TOP1] = best.v;
        ri[RI_MARGIN] = count > 1 ? best.v - best.v2 : INFINITY;
        ri[RI_COUNT] = (float)count;
        ri[RI_SIGNAL] = signal;
        ri[RI_THRESH] = thr;
        ri[RI_ARGMAX] = __int_as_float(best.id);
        ri[RI_ARGMAX_P] = __int_as_float(top_p);
        // the divergences need every token's logits of both models, which only the
        // untruncated target keeps; with tokens outside the mask pi_p has mass
        // where pi_CD = 0
        ri[RI_KL_PQ] = NAN;
        ri[RI_KL_PCD] = count < P.V ? INFINITY : NAN;
        write_row(P, row, ri, out);
    }
}

// ---------------------------------------------------------------------------
// Sequence phase.

// (max_p, lse_p, lse_q, log Z) and (threshold, argmax bits, -, -) of one row
struct RowInfo {
    float4 a, b;
};

__device__ __forceinline__ RowInfo load_rowinfo(const float *ri, size_t r) {
    const float4 *p = reinterpret_cast<const float4 *>(ri + r * kRowInfo);
    return RowInfo{p[0], p[2]};
}

// Statistics of a draft node under its parent row from the raw logits gathered
// in the row phase: log pi_p, log pi_q, cd score, log pi_CD (-inf outside the mask).
struct NodeStat {
    float lpp, lpq, cd, lpcd;
    bool in_mask;
};

// nz = (z_p, z_q) of the token as a candidate (NaN: not one) and by dot product
// (NaN when node statistics are not wanted).  A token is a mask member iff it is a
// candidate at or above the row's threshold; then the candidate's values are the
// ones the row phase used, otherwise the dot product's.
__device__ __forceinline__ NodeStat node_stat(float4 nz, RowInfo rj, float s) {
    NodeStat n;
    n.in_mask = nz.x >= rj.b.x;
    const float zp = n.in_mask ? nz.x : nz.z, zq = n.in_mask ? nz.y : nz.w;
    n.lpp = zp - rj.a.y;
    n.lpq = zq - rj.a.z;
    n.cd = (1.f + s) * n.lpp - s * n.lpq;
    n.lpcd = n.in_mask ? n.cd - rj.a.w : -INFINITY;
    return n;
}

__device__ __forceinline__ void write_node_stats(float *ns, const NodeStat &n, float ratio) {
    ns[0] = n.lpp;
    ns[1] = n.lpq;
    ns[2] = n.cd;
    ns[3] = n.lpcd;
    ns[4] = n.in_mask ? 1.f : 0.f;
    ns[5] = ratio;
}

// exclusive prefix sum over the whole group (fixed order); *total = the sum
__device__ int group_exclusive_scan(int x, int tid, int *total, Smem &sm) {
    const int lane = tid % kWaveSize, wave = tid / kWaveSize;
    int wt;
    const int in_wave = wave_exclusive_scan(x, lane, &wt);
    if (lane == 0) sm.wave_tot[wave] = wt;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int q = 0; q < NT / kWaveSize; ++q) {
        before += q < wave ? sm.wave_tot[q] : 0;
        all += sm.wave_tot[q];
    }
    __syncthreads();
    *total = all;
    return before + in_wave;
}

// The target at a node after the rejection of some of its drafted children, as a
// weight per token t (Alg. 1's residual, applied once per rejected sibling, in
// order): starting from p0 = pi_CD(t) of the node's row, each rejected sibling j
// (proposal q_j, normaliser 1/Z_j; 0 when that residual summed to zero and was not
// applied) maps w -> max(0, w - q_j(t)) / Z_j.  With `qnext`, the unnormalised
// residual of one more rejection, max(0, w - qnext(t)), whose sum is the next Z.
//
// The untruncated target's scans (full_scan) take the chain from a stored row
// instead: `x` holds max(0, w - q_j(t)) of the last applied rejection, so that
// w = x[t] * xs with xs its 1/Z (x = null: w = p0), and with `xout` a rejection
// pass stores its own max(0, w - qnext(t)) there.  Both give the same doubles as
// the chain; the stored row makes a pass read two rows instead of one per
// rejection.
struct Residual {
    const float *dprobs;  // draft_probs rows of the sequence (row i = pi_e^(i))
    const int *rej;       // rejected siblings in order (LDS)
    const double *invz;   // their 1/Z (LDS)
    int nrej;
    const float *qnext;
    int V;
    const double *x = nullptr;  // full_scan: the stored residual row, or null
    double xs = 0.0;
    double *xout = nullptr;     // full_scan with qnext: where the new residual goes
    __device__ double operator()(float p0, int t) const {
        double w = (double)p0;
        for (int m = 0; m < nrej; ++m)
            if (invz[m] > 0.0) w = fmax(0.0, w - (double)dprobs[(size_t)rej[m] * V + t]) * invz[m];
        if (qnext) w = fmax(0.0, w - (double)qnext[t]);
        return w;
    }
};

// Over the mask members of row jrow (the support of pi_CD), in token-id order: the
// sum of the residual's weights, and with `draw` the inverse-CDF draw at u times
// that sum (the smallest token whose cumulative weight exceeds it; the last token
// of positive weight if rounding leaves none).  Called by the whole group; returns
// the drawn token (-1 without `draw` or with an empty support), *total the sum.
__device__ __forceinline__ int masked_scan(const Plan &P, size_t jrow, const Residual &res, bool draw, float u,
                           double *total_out, int tid, Smem &sm) {
    const float *rj = P.rowinfo + jrow * kRowInfo;
    const float thr = rj[RI_THRESH], lse_p = rj[RI_LSEP], lse_q = rj[RI_LSEQ], logZ = rj[RI_LOGZ];
    const int *tc = P.tcount + jrow * P.ntiles;
    const uint4 *bw = reinterpret_cast<const uint4 *>(P.bits + jrow * P.wstride);
    const float2 *cz = P.cand + jrow * P.V;
    // each thread takes a contiguous range of tiles, so the gathered ids are in
    // token order
    const int t0 = (int)((long long)tid * P.ntiles / NT);
    const int t1 = (int)((long long)(tid + 1) * P.ntiles / NT);
    const float4 *pr = P.partials + jrow * P.ntiles;
    auto tile_words = [&](int t, uint4 (&w)[kTileU4]) {
        const int c = tc[t];
        const float tmax = pr[t].x;
#pragma unroll
        for (int q = 0; q < kTileU4; ++q) w[q] = bw[kTileU4 * t + q];
        // words are stale without candidates; a tile below thr holds no mask member
        // (the row phase's rule, so the gathered list never depends on timing)
        const uint32_t keep = c > 0 && tmax >= thr ? ~0u : 0u;
#pragma unroll
        for (int q = 0; q < kTileU4; ++q) w[q] = mask4(w[q], keep);
    };
    int mine = 0;
    for (int t = t0; t < t1; ++t) {
        uint4 w[kTileU4];
        tile_words(t, w);
        mine += popc_tile(w);
    }
    int L;
    const int first = group_exclusive_scan(mine, tid, &L, sm);
    auto weight = [&](int t) -> double {
        const float2 c = cz[t];
        if (!(c.x >= thr)) return 0.0;
        return res(__expf((1.f + P.s) * (c.x - lse_p) - P.s * (c.y - lse_q) - logZ), t);
    };
    // ids of list positions [lo, lo + kList) into sm.list
    auto fill = [&](int lo) {
        if (mine > 0 && first < lo + kList && first + mine > lo) {
            int idx = first;
            for (int t = t0; t < t1; ++t) {
                uint4 w[kTileU4];
                tile_words(t, w);
                emit_ids(w, t, lo, &idx, sm.list);
            }
        }
        __syncthreads();
    };
    auto weigh = [&](int lo) {
        const int n = min(kList, L - lo);
        for (int m = tid; m < n; m += NT) sm.wts[m] = weight(sm.list[m]);
        __syncthreads();
        return n;
    };
    const bool one_round = L <= kList;
    // pass 1: the total, summed sequentially in token order by thread 0
    double run = 0.0;
    for (int lo = 0; lo < L; lo += kList) {
        fill(lo);
        const int n = weigh(lo);
        if (tid == 0)
            for (int m = 0; m < n; ++m) run += sm.wts[m];
        __syncthreads();
    }
    if (tid == 0) sm.dbl = run;
    __syncthreads();
    const double total = sm.dbl;
    *total_out = total;
    __syncthreads();
    if (!draw) return -1;
    // pass 2: with one round the ids and weights of pass 1 are still in place
    const double target = (double)u * total;
    run = 0.0;
    int last = -1;
    if (tid == 0) sm.ints[1] = -1;
    __syncthreads();
    for (int lo = 0; lo < L; lo += kList) {
        int n = min(kList, L - lo);
        if (!one_round) {
            fill(lo);
            n = weigh(lo);
        }
        if (tid == 0) {
            int found = -1;
            for (int m = 0; m < n; ++m) {
                const double wt = sm.wts[m];
                run += wt;
                if (wt > 0.0) {
                    last = sm.list[m];
                    if (run > target) {
                        found = last;
                        break;
                    }
                }
            }
            sm.ints[1] = found >= 0 ? found : (lo + kList >= L ? last : -1);
        }
        __syncthreads();
        const int got = sm.ints[1];
        __syncthreads();
        if (got >= 0) return got;
    }
    return -1;  // empty support (a row without mask members)
}

// Untruncated target: the same over the whole vocabulary of row jrow, from the
// dense logits or the stored residual row (res.x; res.nrej must be 0).  The
// vocabulary is cut into at most kList blocks of bt consecutive tokens (lane l
// holding the k = bt/64 tokens l*k .. l*k+k-1 of a block, k a multiple of 4 so that
// every load is 16 bytes); wave w takes blocks w, w+4, ..., kUnroll at a time, and
// issues the loads of all of them before it weighs any, so that a lane has
// several blocks' loads in flight.  Block sums (a fixed shuffle tree) go to LDS;
// wave 0 adds them in token order; for a draw it finds the block holding u times
// the total, and wave 0 scans that block's lanes in order to find the token.  With
// `reuse` the block sums and the total of the previous call (the same row and
// weights) are still in LDS and only the draw is done.  A rejection pass with
// res.xout stores its weights there.
__device__ __forceinline__ int full_scan(const Plan &P, size_t jrow, const Residual &res, bool draw, float u,
                         double *total_out, int tid, Smem &sm, bool reuse = false) {
    constexpr int kUnroll = 8;
    const float shift = target_shift(P.rowinfo + jrow * kRowInfo, P.s);
    const float *yrow = P.y_full + jrow * P.zstride;
    const int lane = tid % kWaveSize, wave = tid / kWaveSize;
    constexpr int NW = NT / kWaveSize;
    const int k = 4 * max(1, (P.V + 4 * kList * kWaveSize - 1) / (4 * kList * kWaveSize));
    const int bt = k * kWaveSize;
    const int nblk = (P.V + bt - 1) / bt;
    // 16-byte loads of the proposal row only where it is 16-byte aligned (the ABI
    // asks 4 bytes of draft_probs)
    const bool q4 = P.V % 4 == 0 && (reinterpret_cast<uintptr_t>(res.qnext) & 15) == 0;
    // the raw inputs of tokens t .. t+3: loads clamped into the rows (the dense and
    // stored rows have zstride entries, the proposal rows V), values past the
    // vocabulary discarded by weigh4
    // (lo: y of the 4 tokens; or lo, hi: their 4 stored doubles)
    struct Raw4 {
        uint4 lo, hi;
        float4 qn;
    };
    auto load4 = [&](int t, Raw4 &r) {
        const int tl = min(t, P.zstride - 4);
        if (res.x) {
            r.lo = *reinterpret_cast<const uint4 *>(res.x + tl);
            r.hi = *reinterpret_cast<const uint4 *>(res.x + tl + 2);
        } else {
            r.lo = *reinterpret_cast<const uint4 *>(yrow + tl);
            r.hi = uint4{0u, 0u, 0u, 0u};
        }
        if (res.qnext) {
            if (q4) {
                r.qn = *reinterpret_cast<const float4 *>(res.qnext + min(t, P.V - 4));
            } else {
                r.qn.x = t < P.V ? res.qnext[t] : 0.f;
                r.qn.y = t + 1 < P.V ? res.qnext[t + 1] : 0.f;
                r.qn.z = t + 2 < P.V ? res.qnext[t + 2] : 0.f;
                r.qn.w = t + 3 < P.V ? res.qnext[t + 3] : 0.f;
            }
        }
    };
    auto weigh4 = [&](int t, const Raw4 &r, double (&w)[4]) {
        const float yv[4] = {__uint_as_float(r.lo.x), __uint_as_float(r.lo.y), __uint_as_float(r.lo.z),
                             __uint_as_float(r.lo.w)};
        const float qn[4] = {r.qn.x, r.qn.y, r.qn.z, r.qn.w};
        auto dbl = [](uint32_t l, uint32_t h) { return __hiloint2double((int)h, (int)l); };
        const double xv[4] = {dbl(r.lo.x, r.lo.y), dbl(r.lo.z, r.lo.w), dbl(r.hi.x, r.hi.y), dbl(r.hi.z, r.hi.w)};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            double v = res.x ? xv[i] * res.xs : (double)__expf(yv[i] - shift);
            if (res.qnext) v = fmax(0.0, v - (double)qn[i]);
            w[i] = t + i < P.V ? v : 0.0;
        }
    };
    auto weight4 = [&](int t, double (&w)[4]) {
        Raw4 r;
        load4(t, r);
        weigh4(t, r, w);
    };
    auto lane_sum = [&](int b) {  // this lane's tokens of block b, in order
        const int t0 = b * bt + lane * k;
        double s = 0.0;
        for (int j = 0; j < k; j += 4) {
            double w[4];
            weight4(t0 + j, w);
            s += w[0];
            s += w[1];
            s += w[2];
            s += w[3];
        }
        return s;
    };
    if (!reuse) {
        // pass 1: block sums (and the stored residual of a rejection pass); the
        // loads of all kUnroll blocks first (blocks past the end re-read the last)
        for (int b0 = wave; b0 < nblk; b0 += kUnroll * NW) {
            double ls[kUnroll];
#pragma unroll
            for (int i = 0; i < kUnroll; ++i) ls[i] = 0.0;
            for (int j = 0; j < k; j += 4) {
                Raw4 r[kUnroll];
#pragma unroll
                for (int i = 0; i < kUnroll; ++i) load4(min(b0 + i * NW, nblk - 1) * bt + lane * k + j, r[i]);
#pragma unroll
                for (int i = 0; i < kUnroll; ++i) {
                    const int t = (b0 + i * NW) * bt + lane * k + j;
                    if (b0 + i * NW >= nblk) continue;
                    double w[4];
                    weigh4(t, r[i], w);
                    ls[i] += w[0];
                    ls[i] += w[1];
                    ls[i] += w[2];
                    ls[i] += w[3];
                    if (res.xout && t < P.V) {  // the stored row has zstride >= t + 4 entries
                        *reinterpret_cast<double2 *>(res.xout + t) = double2{w[0], w[1]};
                        *reinterpret_cast<double2 *>(res.xout + t + 2) = double2{w[2], w[3]};
                    }
                }
            }
            // the blocks' sums by a shuffle tree (xor 32, 16, ..., 1), one level for
            // all blocks at a time, so that their independent shuffles are in
            // flight together
#pragma unroll
            for (int o = kWaveSize / 2; o > 0; o >>= 1)
#pragma unroll
                for (int i = 0; i < kUnroll; ++i) ls[i] += __shfl_xor(ls[i], o);
#pragma unroll
            for (int i = 0; i < kUnroll; ++i)
                if (lane == 0 && b0 + i * NW < nblk) sm.wts[b0 + i * NW] = ls[i];
        }
        __syncthreads();
    }
    // wave 0 takes the block sums in token order: lane l adds its cb consecutive
    // blocks, an inclusive scan over the lanes gives the running sums; the total is
    // the last lane's (the same order every time, so the draw that reuses a pass
    // sees the same total)
    const int cb = (nblk + kWaveSize - 1) / kWaveSize;
    if (wave == 0) {
        const int b0 = lane * cb;
        double part = 0.0;
        for (int b = b0; b < min(b0 + cb, nblk); ++b) part += sm.wts[b];
        double incl = part;
#pragma unroll
        for (int o = 1; o < kWaveSize; o <<= 1) {
            const double v = __shfl_up(incl, o);
            if (lane >= o) incl += v;
        }
        const double tot = __shfl(incl, kWaveSize - 1);
        if (lane == 0) sm.dbl = tot;
        if (draw) {
            // the block holding u * total: the first lane whose blocks cross it walks
            // them (the last block of positive weight if rounding leaves none)
            const double target = (double)u * tot, start = incl - part;
            const unsigned long long cross = __ballot(part > 0.0 && start + part > target);
            const unsigned long long pos = __ballot(part > 0.0);
            const int pick = cross ? __builtin_ctzll(cross) : (pos ? 63 - __builtin_clzll(pos) : -1);
            if (lane == pick) {
                double before = start, last_before = start;
                int hit = -1, last = -1;
                for (int b = b0; b < min(b0 + cb, nblk); ++b) {
                    const double w = sm.wts[b];
                    if (w > 0.0) {
                        last = b;
                        last_before = before;
                        if (before + w > target) {
                            hit = b;
                            break;
                        }
                    }
                    before += w;
                }
                sm.ints[1] = hit >= 0 ? hit : last;
                sm.dbl2 = hit >= 0 ? before : last_before;  // running sum before that block
            }
            if (pick < 0 && lane == 0) sm.ints[1] = -1;
        }
    }
    __syncthreads();
    const double total = sm.dbl;
    *total_out = total;
    if (!draw) {
        __syncthreads();
        return -1;
    }
    const int blk = sm.ints[1];
    const double before_blk = sm.dbl2;
    __syncthreads();
    if (blk < 0) return -1;  // empty support
    if (wave == 0) {
        const double target = (double)u * total;
        const double ls = lane_sum(blk);
        double incl = ls;
#pragma unroll
        for (int o = 1; o < kWaveSize; o <<= 1) {
            const double v = __shfl_up(incl, o);
            if (lane >= o) incl += v;
        }
        const double start = before_blk + incl - ls;  // running sum before this lane's tokens
        const unsigned long long cross = __ballot(ls > 0.0 && start + ls > target);
        const unsigned long long pos = __ballot(ls > 0.0);
        // the first lane whose tokens cross the target, else the last lane of positive weight
        const int pick = cross ? __builtin_ctzll(cross) : (pos ? 63 - __builtin_clzll(pos) : -1);
        if (lane == pick) {
            double run = start;
            int found = -1, lastpos = -1;
            const int t0 = blk * bt + lane * k;
            for (int j = 0; j < k && found < 0; j += 4) {
                double w[4];
                weight4(t0 + j, w);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    run += w[i];
                    if (w[i] > 0.0 && found < 0) {
                        lastpos = t0 + j + i;
                        if (run > target) found = t0 + j + i;
                    }
                }
            }
            sm.ints[2] = found >= 0 ? found : lastpos;
        }
        if (pick < 0 && lane == 0) sm.ints[2] = -1;
    }
    __syncthreads();
    const int got = sm.ints[2];
    __syncthreads();
    return got;
}

template <int DT, bool SAMPLE>
__device__ __forceinline__ void verify_sequence(const Plan &P, const Inputs &in, const Outputs &out,
                                const SampleInputs &smp, int b, int tid, Smem &sm, int *dyn) {
    const int N = P.N, V = P.V;
    const size_t r0 = (size_t)b * N;
    int *s_par = dyn, *s_tok = dyn + N, *s_amax = dyn + 2 * N;
    // sampled: the walk's state (see seq_lds_bytes)
    float *s_p0 = reinterpret_cast<float *>(dyn + 3 * N), *s_qx = s_p0 + N;
    int *s_rej = reinterpret_cast<int *>(s_qx + N);
    double *s_invz = reinterpret_cast<double *>(dyn + 6 * N);  // 24 N bytes in: 8-byte aligned

    if (tid < 4) sm.flag[tid] = 0;
    __syncthreads();
    for (int i = tid; i < N; i += NT) {
        const int p = in.parents[r0 + i], x = in.tokens[r0 + i];
        const RowInfo r = load_rowinfo(P.rowinfo, r0 + i);
        s_par[i] = p;
        s_tok[i] = x;
        s_amax[i] = __float_as_int(r.b.y);
        if (i == 0 ? p != -1 : (p < 0 || p >= i)) atomicOr(&sm.flag[0], 1);
        if (i > 0 && (x < 0 || x >= V)) atomicOr(&sm.flag[1], 1);
        if (!isfinite(r.a.x) || !isfinite(r.a.y) || !isfinite(r.a.z) || !isfinite(r.a.w))
            atomicOr(&sm.flag[3], 1);
    }
    __syncthreads();
    const int status = sm.flag[0] ? 1 : sm.flag[1] ? 2 : sm.flag[3] ? 3 : 0;
    if (status != 0) {
        for (int i = tid; i < N; i += NT) {
            out.accept_path[r0 + i] = -1;
            if (out.node_stats)
                for (int k = 0; k < 6; ++k) out.node_stats[(r0 + i) * 6 + k] = NAN;
        }
        if (tid == 0) {
            out.status[b] = status;
            out.accept_len[b] = 0;
            out.next_token[b] = -1;
        }
        return;
    }

    if (!SAMPLE) {
        if (tid >= kWaveSize) {
            // node statistics (waves 1..)
            if (!out.node_stats) return;
            const int t1 = tid - kWaveSize;
            if (t1 < 6) out.node_stats[r0 * 6 + t1] = NAN;
            for (int i = 1 + t1; i < N; i += NT - kWaveSize)
                write_node_stats(out.node_stats + (r0 + i) * 6,
                                 node_stat(P.nodez[r0 + i], load_rowinfo(P.rowinfo, r0 + s_par[i]), P.s),
                                 NAN);
            return;
        }
        // greedy walk (wave 0): the lowest-index child carrying the current row's
        // argmax; children have larger indices than their parent
        const int lane = tid;
        int cur = 0, len = 0;
        for (;;) {
            const int target = s_amax[cur];
            int chosen = N;
            for (int c0 = cur + 1; c0 < N; c0 += kWaveSize) {
                const int c = c0 + lane;
                const unsigned long long hit =
                    __ballot(c < N && s_par[c] == cur && s_tok[c] == target);
                if (hit) {
                    chosen = c0 + __builtin_ctzll(hit);
                    break;
                }
            }
            if (chosen >= N) break;
            ++len;
            cur = chosen;
            if (lane == 0) out.accept_path[r0 + len] = cur;
        }
        // every path entry is written once
        for (int i = len + 1 + lane; i < N; i += kWaveSize) out.accept_path[r0 + i] = -1;
        if (lane == 0) {
            out.accept_path[r0] = 0;
            out.status[b] = 0;
            out.accept_len[b] = len;
            out.next_token[b] = s_amax[cur];
        }
        return;
    }

    // sampled: node statistics, and per node the target probability of its token
    // under the parent row and its proposal probability, staged for the walk.  With
    // a mask, the rows settled the walk's decisions (settle_children) unless one of
    // them could not: then each child's accept ratio, its uniform and each node's
    // terminal token are staged instead, in the same round.
    const bool settled = !P.full && P.seqfail[b] == 0;
    float *s_u = reinterpret_cast<float *>(s_amax);  // the sampled walk has no use for the argmax
    if (out.node_stats && tid < 6) out.node_stats[r0 * 6 + tid] = NAN;
    for (int i = 1 + tid; i < N; i += NT) {
        const int x = s_tok[i];
        const NodeStat n = node_stat(P.nodez[r0 + i], load_rowinfo(P.rowinfo, r0 + s_par[i]), P.s);
        const float pe = smp.draft_probs[(r0 + i) * V + x];
        const float p0 = n.in_mask ? __expf(n.lpcd) : 0.f;
        s_p0[i] = p0;
        s_qx[i] = pe;
        if (settled) {
            s_invz[i] = P.wratio[r0 + i];
            s_u[i] = smp.u_acc[r0 + i];
        }
        if (out.node_stats) write_node_stats(out.node_stats + (r0 + i) * 6, n, pe > 0.f ? p0 / pe : INFINITY);
    }
    if (settled)
        for (int i = tid; i < N; i += NT) s_rej[i] = P.wterm[r0 + i];
    __syncthreads();
    if (settled) {
        // the walk from the settled decisions: child c of the current node (every
        // earlier child of it rejected) is accepted iff its uniform is at most its
        // ratio; where the walk ends, the node's terminal token is emitted
        if (tid == 0) {
            int cur = 0, len = 0;
            for (int c = 1; c < N; ++c) {
                if (s_par[c] != cur) continue;
                if ((double)s_u[c] <= s_invz[c]) {
                    ++len;
                    out.accept_path[r0 + len] = c;
                    cur = c;  // its children have larger indices
                }
            }
            sm.ints[0] = len;
            sm.ints[1] = s_rej[cur];
        }
        __syncthreads();
        const int len = sm.ints[0];
        for (int i = len + 1 + tid; i < N; i += NT) out.accept_path[r0 + i] = -1;
        if (tid == 0) {
            out.accept_path[r0] = 0;
            out.status[b] = 0;
            out.accept_len[b] = len;
            out.next_token[b] = sm.ints[1];
        }
        return;
    }
    // The walk (Alg. 1 over a tree): the children of the current node are tried in
    // index order, each against the target left by the siblings rejected before it;
    // an accepted child becomes the current node; when every child is rejected (or
    // there is none) the emitted token is drawn from what is left.  Every thread
    // follows the walk; thread 0 takes the accept decisions.
    Residual res{smp.draft_probs + r0 * V, s_rej, s_invz, 0, nullptr, V};
    // untruncated target: the residual after the last applied rejection at the
    // current node is kept as a stored row (null: none yet) and its 1/Z; the next
    // rejection pass writes the other of the sequence's two rows
    double *const xrow0 = P.full ? P.resbuf + (size_t)b * 2 * P.zstride : nullptr;
    double *const xrow1 = P.full ? xrow0 + P.zstride : nullptr;
    const double *xcur = nullptr;
    double xs = 0.0;
    double total;
    int cur = 0, len = 0;
    for (int c = 1; c < N; ++c) {
        if (s_par[c] != cur) continue;
        if (tid == 0) {
            const double w = res(s_p0[c], s_tok[c]);
            const double ratio = s_qx[c] > 0.f ? w / (double)s_qx[c] : INFINITY;
            sm.ints[3] = w > 0.0 && (double)smp.u_acc[r0 + c] <= ratio;
        }
        __syncthreads();
        const bool accepted = sm.ints[3] != 0;
        __syncthreads();
        if (accepted) {
            ++len;
            if (tid == 0) out.accept_path[r0 + len] = c;
            cur = c;  // its children have larger indices
            res.nrej = 0;
            xcur = nullptr;
            continue;
        }
        // rejected: the normaliser of the residual it leaves
        res.qnext = smp.draft_probs + (r0 + c) * V;
        if (P.full) {
            Residual fr{res.dprobs, s_rej, s_invz, 0, res.qnext, V, xcur, xs, xcur == xrow0 ? xrow1 : xrow0};
            full_scan(P, r0 + cur, fr, false, 0.f, &total, tid, sm);
            if (total > 0.0) {  // applied: the stored row becomes the current residual
                xcur = fr.xout;
                xs = 1.0 / total;
            }
        } else {
            masked_scan(P, r0 + cur, res, false, 0.f, &total, tid, sm);
        }
        res.qnext = nullptr;
        if (tid == 0) {
            s_rej[res.nrej] = c;
            s_invz[res.nrej] = total > 0.0 ? 1.0 / total : 0.0;  // zero sum: not applied
        }
        __syncthreads();
        ++res.nrej;
    }
    const float u = smp.u_res[r0 + cur];
    int next;
    if (P.full && res.nrej > 0 && s_invz[res.nrej - 1] > 0.0) {
        // the residual left by the last rejection is proportional to the weights of
        // its normaliser pass, stored in xcur, whose block sums are still in LDS:
        // draw from those (a rejection whose residual summed to zero left nothing
        // to reuse)
        const Residual last{res.dprobs, s_rej, s_invz, 0, nullptr, V, xcur, 1.0};
        next = full_scan(P, r0 + cur, last, true, u, &total, tid, sm, true);
    } else if (P.full) {
        const Residual fin{res.dprobs, s_rej, s_invz, 0, nullptr, V, xcur, xs};
        next = full_scan(P, r0 + cur, fin, true, u, &total, tid, sm);
    } else {
        next = masked_scan(P, r0 + cur, res, true, u, &total, tid, sm);
    }
    for (int i = len + 1 + tid; i < N; i += NT) out.accept_path[r0 + i] = -1;
    if (tid == 0) {
        out.accept_path[r0] = 0;
        out.status[b] = 0;
        out.accept_len[b] = len;
        out.next_token[b] = next;
    }
}


// ---------------------------------------------------------------------------
// Untruncated target, sampled verification: each sequence's walk spread over a
// group of G workgroups (one launch of at most one workgroup per CU).
//
// With plaus_thresh = 0 every token is in the support, so a rejection needs the
// normaliser Z of the residual max(0, p - pi_e) over the whole vocabulary, and the
// final draw an inverse CDF over it: passes over V tokens that one workgroup can
// only stream at latency-bound rates.  Here every workgroup of the group takes a
// contiguous slice of the vocabulary (each thread a contiguous run of it), and all
// of them follow the same walk: the decisions are taken from the same values by
// thread 0 of each workgroup, and a pass's slice sums are exchanged through the
// workspace with a group barrier in between (each workgroup adds them in slice
// order, so all agree on the total).  The residual of the last applied rejection
// is kept as a stored row (two rows of V doubles per sequence, as in the
// single-workgroup walk), written slice by slice.  The draw finds the slice that
// holds u times the total from the slice sums; that slice's workgroup finds the
// token.  Each slice sum is the last entry of a fixed-order scan of its threads'
// run sums, the same scan the draw walks, so the two agree.

// The walk's current target over the vocabulary of its current row: the stored
// residual row x (scaled by xs), or, with x null, pi_CD = exp(y - shift) from the
// row's dense y.
struct WalkTarget {
    const double *x;
    double xs;
    const float *y;
    float shift;

    __device__ __forceinline__ double at(int t) const {
        if (x) return x[t] * xs;
        return (double)__expf(y[t] - shift);
    }
    // the weights of the 8 * NC tokens from t (t a multiple of 4) and, with q, the
    // residuals max(0, w - q) instead: every load of the NC chunks is issued before
    // any weight is formed, so that they are in flight together (q4: q is 16-byte
    // aligned)
    template <int NC>
    __device__ __forceinline__ void chunk(int t, const float *q, bool q4, double (&w)[8 * NC]) const {
        double xv[8 * NC];
        float yz[8 * NC], pr[8 * NC];
        if (x) {
#pragma unroll
            for (int i = 0; i < 4 * NC; ++i) {
                const double2 a = *reinterpret_cast<const double2 *>(x + t + 2 * i);
                xv[2 * i] = a.x;
                xv[2 * i + 1] = a.y;
            }
        } else {
#pragma unroll
            for (int i = 0; i < 2 * NC; ++i) {
                const float4 a = *reinterpret_cast<const float4 *>(y + t + 4 * i);
                yz[4 * i] = a.x, yz[4 * i + 1] = a.y, yz[4 * i + 2] = a.z, yz[4 * i + 3] = a.w;
            }
        }
        if (q4) {
#pragma unroll
            for (int i = 0; i < 2 * NC; ++i) {
                const float4 a = *reinterpret_cast<const float4 *>(q + t + 4 * i);
                pr[4 * i] = a.x, pr[4 * i + 1] = a.y, pr[4 * i + 2] = a.z, pr[4 * i + 3] = a.w;
            }
        } else if (q) {
#pragma unroll
            for (int i = 0; i < 8 * NC; ++i) pr[i] = q[t + i];
        }
#pragma unroll
        for (int i = 0; i < 8 * NC; ++i) {
            const double cur = x ? xv[i] * xs : (double)__expf(yz[i] - shift);
            w[i] = q ? fmax(0.0, cur - (double)pr[i]) : cur;
        }
    }
};

struct WalkShared {
    double wave_tot[NT / kWaveSize];
    double dval, dval2;
    int ival[4];
};

// inclusive scan of one double per thread over the workgroup, in thread order;
// *total = the last thread's value (every thread gets it)
__device__ __forceinline__ double block_inclusive_scan(double x, int tid, double *total, WalkShared &ws) {
    const int lane = tid % kWaveSize, wave = tid / kWaveSize;
    double incl = x;
#pragma unroll
    for (int d = 1; d < kWaveSize; d <<= 1) {
        const double y = __shfl_up(incl, d, kWaveSize);
        if (lane >= d) incl += y;
    }
    if (lane == kWaveSize - 1) ws.wave_tot[wave] = incl;
    __syncthreads();
    double before = 0.0, all = 0.0;
#pragma unroll
    for (int w = 0; w < NT / kWaveSize; ++w) {
        before += w < wave ? ws.wave_tot[w] : 0.0;
        all += ws.wave_tot[w];
    }
    __syncthreads();
    *total = all;
    return before + incl;
}

// Arrival at the group's barrier number k (1, 2, ...): the workgroup's writes are
// released at agent scope, then it waits (acquire) until all G workgroups arrived.
// The wait is bounded; a workgroup that gives up sets the group's failure flag and
// goes on, and a workgroup that sees the flag stops waiting at once, so every
// workgroup ends, after at most one bounded wait, even if the group never met.
// Every wave first waits for its own stores to complete (vmcnt(0)); thread 0 then
// releases the workgroup's writes at agent scope with its arrival and, once all
// have arrived, acquires at agent scope for the workgroup (the caches it
// invalidates are the CU's and its XCD's, shared by all waves of the workgroup).
// One agent-scope fence pair per workgroup and barrier: each is a cache writeback
// or invalidate, far too costly to issue from every wave.
__device__ __forceinline__ void group_barrier(int *bar, int G, int k, WalkShared &ws) {
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores have landed
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(bar, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        // relaxed polling (an acquire per poll would invalidate the caches every
        // time), one acquire fence once the count is reached
        // (the count and the failure flag are read together, as one 8-byte word)
        const unsigned long long *word = reinterpret_cast<const unsigned long long *>(bar);
        int tries = 0;
        for (;;) {
            const unsigned long long v = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((int)(uint32_t)v >= G * k || (v >> 32) != 0) break;
            if (++tries >= (1 << 22)) {
                __hip_atomic_store(bar + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
}

template <int DT>
__global__ __launch_bounds__(NT) void walk_kernel(Plan P, Inputs in, Outputs out, SampleInputs smp) {
    __shared__ WalkShared ws;
    extern __shared__ __align__(16) int dyn[];
    const int G = P.walk_group;
    const int b = blockIdx.x / G, m = blockIdx.x % G, tid = threadIdx.x;
    const int N = P.N, V = P.V;
    const size_t r0 = (size_t)b * N;
    int *s_par = dyn, *s_tok = dyn + N;
    float *s_p0 = reinterpret_cast<float *>(dyn + 2 * N), *s_qx = s_p0 + N;
    int *bar = P.walkbar + 2 * b;
    double *part = P.walkpart + (size_t)b * 2 * kWalkMaxGroup;
    const bool lead = m == 0;  // writes the sequence's outputs

    // the sequence's tree, tokens and row checks (every workgroup the same)
    if (tid < 4) ws.ival[tid] = 0;
    __syncthreads();
    for (int i = tid; i < N; i += NT) {
        const int p = in.parents[r0 + i], x = in.tokens[r0 + i];
        const RowInfo r = load_rowinfo(P.rowinfo, r0 + i);
        s_par[i] = p;
        s_tok[i] = x;
        if (i == 0 ? p != -1 : (p < 0 || p >= i)) atomicOr(&ws.ival[0], 1);
        if (i > 0 && (x < 0 || x >= V)) atomicOr(&ws.ival[1], 1);
        if (!isfinite(r.a.x) || !isfinite(r.a.y) || !isfinite(r.a.z) || !isfinite(r.a.w))
            atomicOr(&ws.ival[2], 1);
    }
    __syncthreads();
    const int status = ws.ival[0] ? DCD_SEQ_BAD_TREE : ws.ival[1] ? DCD_SEQ_BAD_TOKEN
                                                       : ws.ival[2] ? DCD_SEQ_NONFINITE : 0;
    if (status != 0) {
        if (!lead) return;
        for (int i = tid; i < N; i += NT) {
            out.accept_path[r0 + i] = -1;
            if (out.node_stats)
                for (int k = 0; k < 6; ++k) out.node_stats[(r0 + i) * 6 + k] = NAN;
        }
        if (tid == 0) {
            out.status[b] = status;
            out.accept_len[b] = 0;
            out.next_token[b] = -1;
        }
        return;
    }
    // per node: the target probability of its token under the parent row and its
    // proposal probability; the lead writes the node statistics
    if (lead && out.node_stats && tid < 6) out.node_stats[r0 * 6 + tid] = NAN;
    for (int i = 1 + tid; i < N; i += NT) {
        const int x = s_tok[i];
        const NodeStat n = node_stat(P.nodez[r0 + i], load_rowinfo(P.rowinfo, r0 + s_par[i]), P.s);
        const float pe = smp.draft_probs[(r0 + i) * V + x];
        const float p0 = n.in_mask ? __expf(n.lpcd) : 0.f;
        s_p0[i] = p0;
        s_qx[i] = pe;
        if (lead && out.node_stats)
            write_node_stats(out.node_stats + (r0 + i) * 6, n, pe > 0.f ? p0 / pe : INFINITY);
    }
    __syncthreads();

    // this workgroup's slice of the vocabulary and this thread's run of it
    const int S = ((V + G - 1) / G + 3) / 4 * 4;
    const int v0 = min(V, m * S), v1 = min(V, v0 + S);
    const int k = ((S + NT - 1) / NT + 3) / 4 * 4;
    const int t0 = v0 + tid * k, t1 = min(v1, t0 + k);
    double *const xrow0 = P.resbuf + (size_t)b * 2 * P.zstride, *const xrow1 = xrow0 + P.zstride;
    const double *xcur = nullptr;  // the stored residual row (null: pi_CD of the row)
    double xs = 0.0;               // its normaliser 1/Z
    int cur = 0, len = 0, nbar = 0;
    bool last_pass_applied = false;  // the slice sums of the last pass are the current weights
    double last_rs = 0.0;            // this thread's run sum in the last pass
    float shift = 0.f;
    const float *yrow = nullptr;
    auto set_row = [&](int j) {
        shift = target_shift(P.rowinfo + (r0 + j) * kRowInfo, P.s);
        yrow = P.y_full + (r0 + j) * P.zstride;
    };
    set_row(0);
    auto current_target = [&]() {
        return WalkTarget{xcur, xs, yrow, shift};
    };
    // one pass over this thread's run: with q, the residual max(0, w - q) is stored
    // to xout; returns the run's sum, added in token order.  Groups of four chunks
    // of 8 tokens (the run starts at a multiple of 4), then single chunks, then the
    // partial last chunk.
    auto run_sum = [&](const float *q, double *xout) -> double {
        const WalkTarget wt = current_target();
        double sum = 0.0;
        const bool q4 = q && (reinterpret_cast<uintptr_t>(q) & 15) == 0;
        int t = t0;
        for (; t + 32 <= t1; t += 32) {
            double w[32];
            wt.chunk<4>(t, q, q4, w);
#pragma unroll
            for (int i = 0; i < 32; i += 2)
                if (q) *reinterpret_cast<double2 *>(xout + t + i) = double2{w[i], w[i + 1]};
#pragma unroll
            for (int i = 0; i < 32; ++i) sum += w[i];
        }
        for (; t + 8 <= t1; t += 8) {
            double w[8];
            wt.chunk<1>(t, q, q4, w);
#pragma unroll
            for (int i = 0; i < 8; i += 2)
                if (q) *reinterpret_cast<double2 *>(xout + t + i) = double2{w[i], w[i + 1]};
#pragma unroll
            for (int i = 0; i < 8; ++i) sum += w[i];
        }
        for (; t < t1; ++t) {  // the run's last, partial chunk
            double w = wt.at(t);
            if (q) {
                w = fmax(0.0, w - (double)q[t]);
                xout[t] = w;
            }
            sum += w;
        }
        return sum;
    };
    // The group's slice sums as wave 0 sees them: lane g loads slice g's sum (all
    // in one round) and a fixed-order inclusive scan over the lanes gives each the
    // running sum up to its slice, so every workgroup computes the same numbers.
    auto slice_scan = [&](const double *src, double *mine, double *incl) {
        const int lane = tid % kWaveSize;
        const double v = lane < G ? src[lane] : 0.0;
        double x = v;
#pragma unroll
        for (int d = 1; d < kWaveSize; d <<= 1) {
            const double y = __shfl_up(x, d, kWaveSize);
            if (lane >= d) x += y;
        }
        *mine = v;
        *incl = x;
    };
    // slice sums of a pass exchanged through `part` (pass parity nbar % 2); returns
    // the group total
    auto exchange = [&](double slice_sum) -> double {
        double *dst = part + (nbar % 2) * kWalkMaxGroup;
        if (tid == 0) dst[m] = slice_sum;
        group_barrier(bar, G, ++nbar, ws);
        if (tid < kWaveSize) {
            double mine, incl;
            slice_scan(dst, &mine, &incl);
            if (tid == kWaveSize - 1) ws.dval = incl;
        }
        __syncthreads();
        const double tot = ws.dval;
        __syncthreads();
        return tot;
    };

    for (int c = 1; c < N; ++c) {
        if (s_par[c] != cur) continue;
        // Alg. 1's accept test, taken alike by every workgroup
        if (tid == 0) {
            const double w = xcur ? xcur[s_tok[c]] * xs : (double)s_p0[c];
            const double ratio = s_qx[c] > 0.f ? w / (double)s_qx[c] : INFINITY;
            ws.ival[3] = w > 0.0 && (double)smp.u_acc[r0 + c] <= ratio;
        }
        __syncthreads();
        const bool accepted = ws.ival[3] != 0;
        __syncthreads();
        if (accepted) {
            ++len;
            if (lead && tid == 0) out.accept_path[r0 + len] = c;
            cur = c;
            xcur = nullptr;
            last_pass_applied = false;
            set_row(cur);
            continue;
        }
        // rejected: the residual max(0, p - pi_e^(c)), stored and summed slice by slice
        double *xout = xcur == xrow0 ? xrow1 : xrow0;
        double tot_all;
        last_rs = run_sum(smp.draft_probs + (r0 + c) * V, xout);
        block_inclusive_scan(last_rs, tid, &tot_all, ws);
        const double total = exchange(tot_all);
        if (total > 0.0) {  // applied; a zero residual (rounding only) leaves p as it was
            xcur = xout;
            xs = 1.0 / total;
        }
        last_pass_applied = total > 0.0;
    }

    // the emitted token: inverse CDF of the current weights in token order
    const float u = smp.u_res[r0 + cur];
    double total;
    if (last_pass_applied) {
        // the last pass stored exactly these weights, unnormalised: its slice sums
        // serve (the draw uses xcur without the 1/Z scale)
        xs = 1.0;
    } else {
        double tot_all;
        last_rs = run_sum(nullptr, nullptr);
        block_inclusive_scan(last_rs, tid, &tot_all, ws);
        exchange(tot_all);
    }
    const double *sums = part + ((nbar - 1) % 2) * kWalkMaxGroup;
    // the slice holding u * total (the last slice of positive weight if rounding
    // leaves none), found alike by every workgroup: wave 0's lanes hold the slices
    if (tid < kWaveSize) {
        double mine, incl;
        slice_scan(sums, &mine, &incl);
        const double tot = __shfl(incl, kWaveSize - 1, kWaveSize);
        const double target = (double)u * tot, before = incl - mine;
        const unsigned long long cross = __ballot(tid < G && mine > 0.0 && before + mine > target);
        const unsigned long long pos = __ballot(tid < G && mine > 0.0);
        const int pick = cross ? __builtin_ctzll(cross) : (pos ? 63 - __builtin_clzll(pos) : -1);
        if (tid == (pick < 0 ? 0 : pick)) {
            ws.ival[0] = pick;
            ws.dval = before;
        }
        if (tid == 0) ws.dval2 = tot;
    }
    __syncthreads();
    total = ws.dval2;
    const int slice = ws.ival[0];
    const double slice_before = ws.dval;
    __syncthreads();
    if (m == slice) {
        // this workgroup's slice: the thread whose run crosses the target scans it.
        // The run sums are those of the last pass, which summed the current weights
        // (as stored, when that pass was an applied rejection, which is why xs is 1)
        const double target = (double)u * total;
        const double rs = last_rs;
        double tot_all;
        const double incl = block_inclusive_scan(rs, tid, &tot_all, ws);
        const double start = slice_before + incl - rs;
        if (tid == 0) ws.ival[1] = NT;
        __syncthreads();
        if (rs > 0.0 && start + rs > target) atomicMin(&ws.ival[1], tid);
        __syncthreads();
        int who = ws.ival[1];
        if (who == NT) {  // rounding left no crossing: the last thread of positive weight
            if (tid == 0) ws.ival[1] = -1;
            __syncthreads();
            if (rs > 0.0) atomicMax(&ws.ival[1], tid);
            __syncthreads();
            who = ws.ival[1];
        }
        if (tid == who) {
            // the run's weights in groups (loads in flight together), added in order
            const WalkTarget wt = current_target();
            double run = start;
            int found = -1, lastpos = -1, t = t0;
            auto scan = [&](const double *w, int n, int at) {
                for (int i = 0; i < n && found < 0; ++i) {
                    run += w[i];
                    if (w[i] > 0.0) {
                        lastpos = at + i;
                        if (run > target) found = at + i;
                    }
                }
            };
            for (; t + 32 <= t1 && found < 0; t += 32) {
                double w[32];
                wt.chunk<4>(t, nullptr, false, w);
                scan(w, 32, t);
            }
            for (; t + 8 <= t1 && found < 0; t += 8) {
                double w[8];
                wt.chunk<1>(t, nullptr, false, w);
                scan(w, 8, t);
            }
            for (; t < t1 && found < 0; ++t) {
                const double w = wt.at(t);
                scan(&w, 1, t);
            }
            out.next_token[b] = found >= 0 ? found : lastpos;
        }
    }
    if (lead) {
        for (int i = len + 1 + tid; i < N; i += NT) out.accept_path[r0 + i] = -1;
        if (tid == 0) {
            out.accept_path[r0] = 0;
            out.accept_len[b] = len;
            if (slice < 0) out.next_token[b] = -1;  // empty support
            // a barrier wait that gave up: the walk's workgroups may not have agreed
            out.status[b] = __hip_atomic_load(bar + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                ? DCD_SEQ_WALK_TIMEOUT : 0;
        }
    }
}

// ---------------------------------------------------------------------------
// Masked target, sampled verification: the walk's decisions at a node, settled by
// the node's own row workgroup before the sequence phase.

// The children of node i (later nodes whose parent is i) in index order, with their
// tokens (clamped into the vocabulary: a token outside it fails the sequence later)
// and their proposal probability of their own token: kids, ktok and kq in LDS (the
// first kMaxKids of them), their number in sm.nkids.  One wave, which runs it while
// wave 0 takes the row phase (it needs only the inputs); lane l scans a contiguous
// range of the later nodes, a wave scan orders them.
__device__ __forceinline__ void gather_children(const Plan &P, const Inputs &in, const SampleInputs &smp,
                                                int row, int lane, Smem &sm, int *dyn) {
    const int N = P.N, V = P.V, i = row % N;
    const size_t r0 = (size_t)row - i;
    int *kids = dyn, *ktok = dyn + kMaxKids;
    float *kq = reinterpret_cast<float *>(dyn + 2 * kMaxKids);
    const int per = (N - 1 - i + kWaveSize - 1) / kWaveSize;
    const int c0 = i + 1 + lane * per, c1 = min(N, c0 + per);
    int mine = 0;
    for (int c = c0; c < c1; ++c) mine += in.parents[r0 + c] == i;
    int m;
    int k = wave_exclusive_scan(mine, lane, &m);
    if (mine > 0)
        for (int c = c0; c < c1; ++c)
            if (in.parents[r0 + c] == i) {
                if (k < kMaxKids) {
                    const int x = min(max(in.tokens[r0 + c], 0), V - 1);
                    kids[k] = c;
                    ktok[k] = x;
                    kq[k] = smp.draft_probs[(r0 + c) * V + x];
                }
                ++k;
            }
    if (lane == 0) sm.nkids = m;
}
//
// At node i the walk (Alg. 1 over a tree) tries i's children in index order; when
// it reaches child c every earlier child of i has been rejected, so what it does at
// c depends only on row i's target, those children's proposals and c's uniform:
// the ratio of the residual left by the earlier children, at c's token, to c's
// proposal of that token.  If the walk ends at i, every child of i was rejected, so
// the token it emits is the draw, with u_resample of node i, from the residual left
// by all of them.  Row i's workgroup holds the row's mask members (the support) in
// LDS after the row phase, so it computes these: per child the accept ratio (-1:
// rejected whatever its uniform) and the residual's normaliser, and the row's
// terminal token.  The sequence phase then only compares uniforms with ratios.  The
// residual arithmetic is the walk's own (Residual): w <- max(0, w - q) * (1/Z) per
// applied rejection, Z the residual's sum over the support (a rejection whose
// residual sums to zero leaves w as it was).  A row with more mask members than
// kMembers, a node with more than kMaxKids children, or more than kKidQ proposal
// values to gather marks its sequence, which the sequence phase then walks itself.
template <int DT>
__device__ __forceinline__ void settle_children(const Plan &P, const Inputs &in, const SampleInputs &smp, int row, int tid,
                                Smem &sm, int *dyn) {
    const int N = P.N, V = P.V, i = row % N, b = row / N;
    const size_t r0 = (size_t)row - i;
    int *kids = dyn, *ktok = dyn + kMaxKids;
    float *kq = reinterpret_cast<float *>(dyn + 2 * kMaxKids);
    double *w = reinterpret_cast<double *>(dyn + 3 * kMaxKids);  // [kMembers]
    float *q = reinterpret_cast<float *>(w + kMembers);          // [kKidQ]: child k, member t at k*L + t
    const unsigned long long *mlist = reinterpret_cast<const unsigned long long *>(sm.wts);
    const int L = sm.mcount;
    const float logZ = sm.mlogz;
    // the children of node i in index order, listed by gather_children
    const int m = sm.nkids;
    const bool ok = L <= kMembers && m <= kMaxKids && (size_t)m * (size_t)L <= (size_t)kKidQ;
    // the target over the support (the row phase's cd scores, in token order)
    if (ok)
        for (int t = tid; t < L; t += NT) w[t] = (double)__expf(__uint_as_float((uint32_t)mlist[t]) - logZ);
    __syncthreads();
    if (ok)  // every child's proposal over the support, gathered in one round
        for (int e = tid; e < m * L; e += NT)
            q[e] = smp.draft_probs[(r0 + kids[e / L]) * V + (int)(mlist[e % L] >> 32)];
    __syncthreads();
    if (!ok) {
        if (tid == 0) atomicOr(&P.seqfail[b], 1);
        return;
    }
    if (tid >= kWaveSize) return;
    const int lane = tid;
    // sums over the support in a fixed order: lane-strided partials, then a tree
    auto wave_sum_d = [&](double x) {
#pragma unroll
        for (int d = kWaveSize / 2; d > 0; d >>= 1) x += __shfl_down(x, d, kWaveSize);
        return __shfl(x, 0, kWaveSize);
    };
    for (int k = 0; k < m; ++k) {
        // the residual left by the earlier children, at this child's token (0 off
        // the support; a token appears at most once there)
        int at = -1;
        for (int t = lane; t < L; t += kWaveSize) at = (int)(mlist[t] >> 32) == ktok[k] ? t : at;
#pragma unroll
        for (int d = kWaveSize / 2; d > 0; d >>= 1) at = max(at, __shfl_xor(at, d, kWaveSize));
        const double wx = at >= 0 ? w[at] : 0.0;
        if (lane == 0) {
            const double ratio = kq[k] > 0.f ? wx / (double)kq[k] : INFINITY;
            P.wratio[r0 + kids[k]] = wx > 0.0 ? ratio : -1.0;
        }
        const float *qk = q + (size_t)k * L;
        double part = 0.0;
        for (int t = lane; t < L; t += kWaveSize) part += fmax(0.0, w[t] - (double)qk[t]);
        const double total = wave_sum_d(part);
        if (total > 0.0) {
            const double invz = 1.0 / total;
            for (int t = lane; t < L; t += kWaveSize) w[t] = fmax(0.0, w[t] - (double)qk[t]) * invz;
        }
        wave_lds_sync();
    }
    // the terminal draw: inverse CDF of what is left, in token order (lane l a
    // contiguous run of the support, an inclusive scan over the lanes), at u * total;
    // the last token of positive weight if rounding leaves none above it
    const int per2 = (L + kWaveSize - 1) / kWaveSize;
    const int ta = min(L, lane * per2), te = min(L, ta + per2);
    double run = 0.0;
    for (int t = ta; t < te; ++t) run += w[t];
    double incl = run;
#pragma unroll
    for (int d = 1; d < kWaveSize; d <<= 1) {
        const double y = __shfl_up(incl, d, kWaveSize);
        if (lane >= d) incl += y;
    }
    const double tot = __shfl(incl, kWaveSize - 1, kWaveSize);
    const double target = (double)smp.u_res[row] * tot, before = incl - run;
    const unsigned long long cross = __ballot(run > 0.0 && before + run > target);
    const unsigned long long pos = __ballot(run > 0.0);
    const int who = cross ? __builtin_ctzll(cross) : (pos ? 63 - __builtin_clzll(pos) : -1);
    if (who < 0) {
        if (lane == 0) P.wterm[row] = -1;  // an empty support
    } else if (lane == who) {
        double acc = before;
        int found = -1, last = -1;
        for (int t = ta; t < te && found < 0; ++t) {
            acc += w[t];
            if (w[t] > 0.0) {
                last = t;
                if (acc > target) found = t;
            }
        }
        P.wterm[row] = (int)(mlist[found >= 0 ? found : last] >> 32);
    }
}

// One workgroup per row; the workgroup that finishes a sequence's last row
// (counted in seqdone, cleared by the LM-head launch) runs the sequence phase.
template <int DT, bool SAMPLE>
__global__ __launch_bounds__(NT) void finish_kernel(Plan P, Inputs in, Outputs out,
                                                    SampleInputs smp) {
    __shared__ Smem sm;
    __shared__ int last;
    extern __shared__ __align__(16) int dyn[];
    const int row = blockIdx.x, tid = threadIdx.x;
    if (row == 0 && tid == 0) advance_call(P.ctl);  // the call's last use of the call count
    if (tid == 0) sm.node_ok = 0;
    // the spread walk that follows starts its group's barrier count from zero
    if (SAMPLE && P.walk_group && row % P.N == 0 && tid < 2) P.walkbar[(row / P.N) * 2 + tid] = 0;
    __syncthreads();
    combine_row<DT>(P, in, out, row, tid % kWaveSize, tid / kWaveSize, sm, SAMPLE && !P.full);
    // sampled, masked: wave 1 lists the node's children while wave 0 takes the row phase
    if (SAMPLE && !P.full && tid / kWaveSize == 1) gather_children(P, in, smp, row, tid % kWaveSize, sm, dyn);
    // count the row once all of its waves are done; thread 0 stores the node's
    // logits, and the release half of the counting atomic publishes them together
    // with wave 0's results and the settled walk decisions (the workgroup barrier
    // orders those before it)
    __syncthreads();
    if (SAMPLE && !P.full) {
        settle_children<DT>(P, in, smp, row, tid, sm, dyn);
        __syncthreads();
    }
    const int b = row / P.N;
    if (tid == 0) {
        if (sm.node_ok) P.nodez[row] = sm.nodez;
        last = __hip_atomic_fetch_add(&P.seqdone[b], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT) ==
               P.N - 1;
    }
    __syncthreads();
    if (!last || (SAMPLE && P.walk_group)) return;  // walk_kernel walks the sequence
    // acquire: the other rows of the sequence are visible from here on
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    verify_sequence<DT, SAMPLE>(P, in, out, smp, b, tid, sm, dyn);
}

// Proposals from the recombined heads: one workgroup per row.  The row phase
// (wave 0) gives the row's normalisers and argmax; then the whole group draws a
// token from the row's target.  The dense target rows are written afterwards by
// propose_probs_kernel, which spreads them over many workgroups.
template <int DT>
__global__ __launch_bounds__(NT) void propose_kernel(Plan P, Inputs in, ProposeOutputs po) {
    __shared__ Smem sm;
    const int row = blockIdx.x, tid = threadIdx.x;
    if (row == 0 && tid == 0) advance_call(P.ctl);  // the last kernel using the call state
    Outputs out{};
    out.row_argmax = po.argmax;
    combine_row<DT>(P, in, out, row, tid % kWaveSize, tid / kWaveSize, sm);
    __syncthreads();  // the row's statistics are visible to the whole group
    const Residual target{nullptr, nullptr, nullptr, 0, nullptr, P.V};
    if (po.tokens) {
        double total;
        const int t = P.full ? full_scan(P, row, target, true, po.u[row], &total, tid, sm)
                             : masked_scan(P, row, target, true, po.u[row], &total, tid, sm);
        if (tid == 0) po.tokens[row] = t;
    }
}

constexpr int kProbTokens = NT * 4;  // tokens of a row per workgroup of propose_probs_kernel

// The proposal rows written densely: pi_hat(t) of row blockIdx.x for the
// kProbTokens tokens of slice blockIdx.y, 0 off the mask.  A thread takes 4
// consecutive tokens (one 16-byte store when the rows are 16-byte aligned); the
// values are computed exactly as in the row phase's target.
template <bool FULL>
__global__ __launch_bounds__(NT) void propose_probs_kernel(Plan P, float *probs, bool aligned) {
    const int row = blockIdx.x;
    const int t0 = blockIdx.y * kProbTokens + threadIdx.x * 4;
    if (t0 >= P.V) return;
    const float *rj = P.rowinfo + (size_t)row * kRowInfo;
    const float thr = rj[RI_THRESH], lse_p = rj[RI_LSEP], lse_q = rj[RI_LSEQ], logZ = rj[RI_LOGZ];
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (FULL) {
        // the dense y rows are padded to whole tiles, so the load stays inside the row
        const float4 yv = *reinterpret_cast<const float4 *>(P.y_full + (size_t)row * P.zstride + t0);
        const float shift = target_shift(rj, P.s), y[4] = {yv.x, yv.y, yv.z, yv.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = __expf(y[i] - shift);
    } else {
        // bitmap words are valid only in tiles that kept candidates; the 4 tokens
        // share a tile and a word (t0 is a multiple of 4)
        const uint32_t word = P.tcount[(size_t)row * P.ntiles + t0 / kTileTokens] > 0
                                  ? P.bits[(size_t)row * P.wstride + (t0 >> 5)] >> (t0 & 31)
                                  : 0u;
        const float2 *cz = P.cand + (size_t)row * P.V;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if ((word >> i & 1u) && t0 + i < P.V) {
                const float2 c = cz[t0 + i];
                if (c.x >= thr) v[i] = __expf((1.f + P.s) * (c.x - lse_p) - P.s * (c.y - lse_q) - logZ);
            }
        }
    }
    float *dst = probs + (size_t)row * P.V + t0;
    if (aligned && t0 + 3 < P.V) {
        *reinterpret_cast<float4 *>(dst) = float4{v[0], v[1], v[2], v[3]};
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (t0 + i < P.V) dst[i] = v[i];
    }
}

}  // namespace

hipError_t launch_propose(const Plan &p, const Inputs &in, const ProposeOutputs &out, hipStream_t st) {
    if (p.dtype == kBF16)
        hipLaunchKernelGGL((propose_kernel<kBF16>), dim3(p.R), dim3(NT), 0, st, p, in, out);
    else
        hipLaunchKernelGGL((propose_kernel<kF32>), dim3(p.R), dim3(NT), 0, st, p, in, out);
    if (out.probs) {
        const dim3 grid(p.R, (p.V + kProbTokens - 1) / kProbTokens);
        const bool aligned = p.V % 4 == 0 && reinterpret_cast<uintptr_t>(out.probs) % 16 == 0;
        if (p.full)
            hipLaunchKernelGGL(propose_probs_kernel<true>, grid, dim3(NT), 0, st, p, out.probs, aligned);
        else
            hipLaunchKernelGGL(propose_probs_kernel<false>, grid, dim3(NT), 0, st, p, out.probs, aligned);
    }
    return hipGetLastError();
}

// dynamic LDS of the sequence phase: parents, tokens and row argmax (12 bytes per
// node); sampled also the walk's state: target and proposal probability of each
// node's token, the rejected siblings and their normalisers (20 more bytes per
// node; the doubles follow 6 N 4-byte slots, so they are 8-byte aligned for any N)
// dynamic LDS of the spread walk: parents, tokens, target and proposal probability
// of each node's token (16 bytes per node)
size_t walk_lds_bytes(int N) { return (size_t)4 * N * sizeof(int); }

// The spread walk pays where the single-workgroup walk leaves the chip idle (B
// sequences walked by B CUs).  Each sequence gets CUs / B workgroups, one per CU, at
// most kWalkMaxGroup; with fewer than 4 per sequence (B > 64 on 256 CUs) the finish
// kernel walks each sequence in its own workgroup.  One workgroup per CU in all: with
// 16 sequences of 64 workgroups each (4 per CU) the walk took 133 us, against about
// 110 us for the finish kernel's walk; with 16 each, the step dropped by 48 us.
int walk_group_size(const Plan &p, hipStream_t st) {
    // per device, looked up once: its CU count and whether a workgroup of the walk
    // (at the largest LDS it asks for) fits on a CU, per element type
    constexpr int kDevices = 64;
    static std::atomic<int> cus_of[kDevices], fits_of[kDevices][2];  // 0: not looked up yet
    int dev = -1;
    if ((st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev)) != hipSuccess || dev < 0 || dev >= kDevices)
        return 0;
    int cus = cus_of[dev].load(std::memory_order_relaxed);
    if (cus == 0) {
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            return 0;
        cus_of[dev].store(cus, std::memory_order_relaxed);
    }
    const int G = cus / p.B < kWalkMaxGroup ? cus / p.B : kWalkMaxGroup;
    if (G < 4) return 0;
    const int t = p.dtype == kBF16 ? 1 : 0;
    int fits = fits_of[dev][t].load(std::memory_order_relaxed);
    if (fits == 0) {
        // the group barrier needs every workgroup of a group resident; the launch
        // has at most one per CU, so a single workgroup with the most LDS the walk
        // uses must fit on a CU
        int per_cu = 0, cur = -1;
        const void *fn = t ? (const void *)walk_kernel<kBF16> : (const void *)walk_kernel<kF32>;
        if (hipGetDevice(&cur) != hipSuccess) return 0;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return 0;
        const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, NT,
                                                                          walk_lds_bytes(kMaxNodes));
        if (cur != dev) (void)hipSetDevice(cur);
        if (e != hipSuccess) return 0;
        fits = per_cu >= 1 ? 1 : 2;
        fits_of[dev][t].store(fits, std::memory_order_relaxed);
    }
    return fits == 1 ? G : 0;
}

hipError_t launch_walk(const Plan &p, const Inputs &in, const Outputs &out, const SampleInputs &smp,
                       hipStream_t st) {
    // B * G <= CUs workgroups, each of which fits on a CU (walk_group_size): on a
    // device with nothing else running they are all resident together
    const unsigned lds = (unsigned)walk_lds_bytes(p.N);
    if (p.dtype == kBF16)
        hipLaunchKernelGGL(walk_kernel<kBF16>, dim3(p.B * p.walk_group), dim3(NT), lds, st, p, in, out, smp);
    else
        hipLaunchKernelGGL(walk_kernel<kF32>, dim3(p.B * p.walk_group), dim3(NT), lds, st, p, in, out, smp);
    return hipGetLastError();
}

size_t seq_lds_bytes(int N, bool sampled, bool masked) {
    if (!sampled) return (size_t)3 * N * sizeof(int);
    const size_t walk = (size_t)6 * N * sizeof(int) + (size_t)N * sizeof(double);
    // with a mask, the settled walk decisions use it first
    return masked && kSettleLds > walk ? kSettleLds : walk;
}

hipError_t launch_finish(const Plan &p, const Inputs &in, const Outputs &out,
                         const SampleInputs *smp, hipStream_t st) {
    const SampleInputs s = smp ? *smp : SampleInputs{nullptr, nullptr, nullptr};
    const size_t lds = seq_lds_bytes(p.N, smp != nullptr, !p.full);
    // the sampled walk's LDS can exceed the default 64 KB limit of dynamic LDS
    static const hipError_t attr = [] {
        const int most = (int)seq_lds_bytes(kMaxNodes, true, true);
        hipError_t e = hipFuncSetAttribute((const void *)finish_kernel<kBF16, true>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, most);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)finish_kernel<kF32, true>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, most);
        return e;
    }();
    if (attr != hipSuccess) return attr;
    if (p.dtype == kBF16) {
        if (smp)
            hipLaunchKernelGGL((finish_kernel<kBF16, true>), dim3(p.R), dim3(NT), lds, st, p, in, out, s);
        else
            hipLaunchKernelGGL((finish_kernel<kBF16, false>), dim3(p.R), dim3(NT), lds, st, p, in, out, s);
    } else {
        if (smp)
            hipLaunchKernelGGL((finish_kernel<kF32, true>), dim3(p.R), dim3(NT), lds, st, p, in, out, s);
        else
            hipLaunchKernelGGL((finish_kernel<kF32, false>), dim3(p.R), dim3(NT), lds, st, p, in, out, s);
    }
    return hipGetLastError();
}

}  // namespace dcd
