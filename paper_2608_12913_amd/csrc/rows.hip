// Per-row combination of the LM-head partials and per-sequence verification.
//
// combine_kernel (one workgroup per row):
//   max_p, log-normalisers of both models from the per-tile (max, sum exp) pairs;
//   the plausibility mask z_p >= max_p + ln theta (Sec. 2.1) over the candidate
//   tokens; the cd score (1+s)(z_p - lse_p) - s(z_q - lse_q) of Eq. (1); its log
//   normaliser over the mask, argmax (lowest id on ties) and top-2 margin.
// sequence_kernel (one workgroup per sequence):
//   tree / token checks, draft-token statistics under the parent row, then either
//   the greedy walk from the root or Alg. 1's accept test with residual / bonus
//   resampling along a chain.
// All reductions run in a fixed order, so repeated calls are bit-identical.
#include "dcd_internal.h"

namespace dcd {
namespace {

constexpr int NT = 256;
constexpr int NWAVES = NT / kWaveSize;

struct Lse {  // running log-sum-exp: value = m + log(s)
    float m, s;
};

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    if (a.m == -INFINITY) return b;
    if (b.m == -INFINITY) return a;
    const float m = fmaxf(a.m, b.m);
    return Lse{m, a.s * __expf(a.m - m) + b.s * __expf(b.m - m)};
}

struct Top2 {  // best value and id, runner-up value
    float v;
    int id;
    float v2;
};

__device__ __forceinline__ Top2 top2_merge(Top2 a, Top2 b) {
    const bool a_wins = b.id < 0 || (a.id >= 0 && (a.v > b.v || (a.v == b.v && a.id < b.id)));
    const Top2 w = a_wins ? a : b, l = a_wins ? b : a;
    return Top2{w.v, w.id, fmaxf(w.v2, l.id >= 0 ? l.v : -INFINITY)};
}

// Fixed-order block reductions through shared memory (tree over thread ids).
template <typename T, typename F>
__device__ T block_reduce(T x, T *sh, F merge) {
    const int tid = threadIdx.x;
    sh[tid] = x;
    __syncthreads();
    for (int w = NT / 2; w > 0; w >>= 1) {
        if (tid < w) sh[tid] = merge(sh[tid], sh[tid + w]);
        __syncthreads();
    }
    T r = sh[0];
    __syncthreads();
    return r;
}

// Dot product h . w over d elements by the whole workgroup (fp32, fixed order).
template <int DT>
__device__ float block_dot(const void *h, const void *w, int d, float *sh) {
    const int tid = threadIdx.x;
    float acc = 0.f;
    if constexpr (DT == kBF16) {
        const uint16_t *hr = (const uint16_t *)h, *wr = (const uint16_t *)w;
        for (int k = tid * 8; k < d; k += NT * 8) {
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
        for (int k = tid * 4; k < d; k += NT * 4) {
            const float4 hv = *(const float4 *)(hr + k), wv = *(const float4 *)(wr + k);
            acc += hv.x * wv.x + hv.y * wv.y + hv.z * wv.z + hv.w * wv.w;
        }
    }
    return block_reduce(acc, sh, [](float a, float b) { return a + b; });
}

template <int DT>
__global__ __launch_bounds__(NT) void combine_kernel(Plan P, Inputs in, int32_t *row_argmax,
                                                     float *row_stats, int want_node_logits) {
    __shared__ Lse sh_lse[NT];
    __shared__ Top2 sh_top[NT];
    __shared__ int sh_cnt[NT];
    __shared__ float sh_f[NT];
    const int row = blockIdx.x, tid = threadIdx.x;
    const size_t esz = DT == kBF16 ? 2 : 4;

    // 1. merge the per-tile (max, sum exp) pairs of both models
    Lse lp{-INFINITY, 0.f}, lq{-INFINITY, 0.f};
    const float4 *pr = P.partials + (size_t)row * P.ntiles;
    for (int t = tid; t < P.ntiles; t += NT) {
        const float4 v = pr[t];
        lp = lse_merge(lp, Lse{v.x, v.y});
        lq = lse_merge(lq, Lse{v.z, v.w});
    }
    lp = block_reduce(lp, sh_lse, lse_merge);
    lq = block_reduce(lq, sh_lse, lse_merge);
    const float max_p = lp.m;
    const float lse_p = lp.m + __logf(lp.s);
    const float lse_q = lq.m + __logf(lq.s);
    const float thr = max_p + P.log_theta;
    const float s = P.s;

    // 2. mask, cd score, argmax, log Z over the candidates; a thread takes whole
    //    tiles (ascending), skipping tiles without candidates
    Lse lc{-INFINITY, 0.f};
    Top2 best{-INFINITY, -1, -INFINITY};
    int count = 0;
    const int *tc = P.tcount + (size_t)row * P.ntiles;
    const uint32_t *bw = P.bits + (size_t)row * P.wstride;
    const float2 *cz = P.cand + (size_t)row * P.V;
    for (int tile = tid; tile < P.ntiles; tile += NT) {
        if (tc[tile] == 0) continue;
        for (int w = 0; w < kWordsPerTile; ++w) {
            uint32_t b = bw[tile * kWordsPerTile + w];
            while (b) {
                const int t = (tile * kWordsPerTile + w) * 32 + __ffs(b) - 1;
                b &= b - 1;
                const float2 c = cz[t];
                if (!(c.x >= thr)) continue;
                ++count;
                const float cd = (1.f + s) * (c.x - lse_p) - s * (c.y - lse_q);
                best = top2_merge(best, Top2{cd, t, -INFINITY});
                lc = lse_merge(lc, Lse{cd, 1.f});
            }
        }
    }
    lc = block_reduce(lc, sh_lse, lse_merge);
    best = block_reduce(best, sh_top, top2_merge);
    count = block_reduce(count, sh_cnt, [](int a, int b) { return a + b; });

    if (tid == 0) {
        const float logZ = lc.m + __logf(lc.s);
        float signal = NAN;
        if (best.id >= 0) {
            const float2 c = cz[best.id];
            signal = (c.x - lse_p) - (c.y - lse_q);
        }
        float *ri = P.rowinfo + (size_t)row * kRowInfo;
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
        if (row_argmax) row_argmax[row] = best.id;
        if (row_stats) {
#pragma unroll
            for (int k = 0; k < 8; ++k) row_stats[(size_t)row * 8 + k] = ri[k];
        }
    }

    // 3. this row as a draft node: its token's logits under its parent row.  A
    //    candidate reuses the tile's values (the same numbers the mask saw);
    //    otherwise the token is outside the mask and, when node statistics are
    //    wanted, its logits are recomputed here.
    const int i = row % P.N;
    if (i == 0) return;
    const int j = in.parents[row], x = in.tokens[row];
    if (j < 0 || j >= i || x < 0 || x >= P.V) return;  // the sequence is rejected later
    const size_t rowj = (size_t)(row - i + j);
    const int xt = x / kTileTokens;
    const bool cand = P.tcount[rowj * P.ntiles + xt] > 0 &&
                      (P.bits[rowj * P.wstride + (x >> 5)] >> (x & 31) & 1u);
    float4 nz{0.f, 0.f, 0.f, 0.f};
    if (cand) {
        const float2 c = P.cand[rowj * P.V + x];
        nz = float4{c.x, c.y, 1.f, 0.f};
    } else if (want_node_logits) {
        float zp = block_dot<DT>((const char *)in.hp + rowj * P.dp * esz,
                                 (const char *)in.wp + (size_t)x * P.dp * esz, P.dp, sh_f);
        float zq = block_dot<DT>((const char *)in.hq + rowj * P.dq * esz,
                                 (const char *)in.wq + (size_t)x * P.dq * esz, P.dq, sh_f);
        zp = (zp + (in.bp ? in.bp[x] : 0.f)) * P.inv_T;
        zq = (zq + (in.bq ? in.bq[x] : 0.f)) * P.inv_T;
        nz = float4{zp, zq, 0.f, 0.f};
    }
    if (tid == 0) P.nodez[row] = nz;
}

template <int DT, bool SAMPLE>
__global__ __launch_bounds__(NT) void sequence_kernel(Plan P, Inputs in, Outputs out,
                                                      SampleInputs smp) {
    __shared__ int sh_flag[4];
    __shared__ int sh_int[2];
    __shared__ double sh_sum[NT];
    __shared__ double sh_prefix[NT + 1];
    const int b = blockIdx.x, tid = threadIdx.x, N = P.N, V = P.V;
    const size_t r0 = (size_t)b * N;
    const int32_t *par = in.parents + r0, *tok = in.tokens + r0;
    const float *ri = P.rowinfo + r0 * kRowInfo;

    if (tid < 4) sh_flag[tid] = 0;
    if (tid == 0) sh_int[0] = N;  // first rejected node (sampled)
    __syncthreads();
    for (int i = tid; i < N; i += NT) {
        const int p = par[i];
        if (i == 0 ? p != -1 : (p < 0 || p >= i)) atomicOr(&sh_flag[0], 1);
        if (i > 0 && (tok[i] < 0 || tok[i] >= V)) atomicOr(&sh_flag[1], 1);
        if (SAMPLE && i > 0 && p != i - 1) atomicOr(&sh_flag[2], 1);
        const float *r = ri + (size_t)i * kRowInfo;
        if (!isfinite(r[RI_MAXP]) || !isfinite(r[RI_LSEP]) || !isfinite(r[RI_LSEQ]) ||
            !isfinite(r[RI_LOGZ]))
            atomicOr(&sh_flag[3], 1);
    }
    __syncthreads();
    const int status = sh_flag[0] ? 1 : sh_flag[1] ? 2 : sh_flag[2] ? 4 : sh_flag[3] ? 3 : 0;
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

    // draft-token statistics under the parent row (logits gathered by the combine)
    if (out.node_stats && tid < 6) out.node_stats[r0 * 6 + tid] = NAN;
    for (int i = 1 + tid; i < N; i += NT) {
        const int j = par[i], x = tok[i];
        const float *rj = ri + (size_t)j * kRowInfo;
        const float4 nz = P.nodez[r0 + i];
        const bool in_mask = nz.z != 0.f && nz.x >= rj[RI_THRESH];
        const float lpp = nz.x - rj[RI_LSEP], lpq = nz.y - rj[RI_LSEQ];
        const float cd = (1.f + P.s) * lpp - P.s * lpq;
        const float lpcd = in_mask ? cd - rj[RI_LOGZ] : -INFINITY;
        float ratio = NAN;
        if (SAMPLE) {
            const float pe = smp.draft_probs[(r0 + i) * V + x];
            ratio = pe > 0.f ? __expf(lpcd) / pe : INFINITY;
            const bool accept = in_mask && smp.u_acc[r0 + i] <= ratio;
            if (!accept) atomicMin(&sh_int[0], i);
        }
        if (out.node_stats) {
            float *ns = out.node_stats + (r0 + i) * 6;
            ns[0] = lpp;
            ns[1] = lpq;
            ns[2] = cd;
            ns[3] = lpcd;
            ns[4] = in_mask ? 1.f : 0.f;
            ns[5] = ratio;
        }
    }
    __syncthreads();

    if (!SAMPLE) {
        // greedy walk: lowest-index child carrying the current row's argmax
        int cur = 0, len = 0;
        if (tid == 0) out.accept_path[r0] = 0;
        for (;;) {
            const int target = __float_as_int(ri[(size_t)cur * kRowInfo + RI_ARGMAX]);
            if (tid == 0) sh_int[1] = N;
            __syncthreads();
            for (int c = cur + 1 + tid; c < N; c += NT)
                if (par[c] == cur && tok[c] == target) atomicMin(&sh_int[1], c);
            __syncthreads();
            const int chosen = sh_int[1];
            __syncthreads();
            if (chosen >= N) break;
            ++len;
            cur = chosen;
            if (tid == 0) out.accept_path[r0 + len] = cur;
        }
        // every path entry is written by exactly one thread
        for (int i = len + 1 + tid; i < N; i += NT) out.accept_path[r0 + i] = -1;
        if (tid == 0) {
            out.status[b] = 0;
            out.accept_len[b] = len;
            out.next_token[b] = __float_as_int(ri[(size_t)cur * kRowInfo + RI_ARGMAX]);
        }
        return;
    }

    // sampled: accept nodes 1..k-1; draw from the residual at k or the bonus row
    const int k = sh_int[0];
    const int jrow = k < N ? k - 1 : N - 1;
    const float *rj = ri + (size_t)jrow * kRowInfo;
    const float thr = rj[RI_THRESH], lse_p = rj[RI_LSEP], lse_q = rj[RI_LSEQ], logZ = rj[RI_LOGZ];
    const float *qrow = k < N ? smp.draft_probs + (r0 + k) * V : nullptr;
    const uint32_t *bw = P.bits + (r0 + jrow) * P.wstride;
    const float2 *cz = P.cand + (r0 + jrow) * V;
    const int nwords = (V + 31) / 32;
    const int w0 = (int)((long long)tid * nwords / NT), w1 = (int)((long long)(tid + 1) * nwords / NT);
    // weight of token t under the chosen distribution (0 outside the mask)
    auto weight = [&](int t, bool residual) -> double {
        const float2 c = cz[t];
        if (!(c.x >= thr)) return 0.0;
        const float p = __expf((1.f + P.s) * (c.x - lse_p) - P.s * (c.y - lse_q) - logZ);
        return residual ? (double)fmaxf(0.f, p - qrow[t]) : (double)p;
    };
    const int *tc = P.tcount + (r0 + jrow) * P.ntiles;
    auto local_sum = [&](bool residual) {
        double acc = 0.0;
        for (int w = w0; w < w1; ++w) {
            if (tc[w / kWordsPerTile] == 0) continue;
            uint32_t bits = bw[w];
            while (bits) {
                const int t = w * 32 + __ffs(bits) - 1;
                bits &= bits - 1;
                acc += weight(t, residual);
            }
        }
        return acc;
    };
    bool residual = qrow != nullptr;
    double local = local_sum(residual);
    sh_sum[tid] = local;
    __syncthreads();
    if (tid == 0) {  // sequential exclusive scan: the partial sums tile [0, total) exactly
        double run = 0.0;
        for (int i = 0; i < NT; ++i) {
            sh_prefix[i] = run;
            run += sh_sum[i];
        }
        sh_prefix[NT] = run;
    }
    __syncthreads();
    if (residual && !(sh_prefix[NT] > 0.0)) {  // degenerate residual: fall back to pi_CD
        __syncthreads();
        residual = false;
        local = local_sum(false);
        sh_sum[tid] = local;
        __syncthreads();
        if (tid == 0) {
            double run = 0.0;
            for (int i = 0; i < NT; ++i) {
                sh_prefix[i] = run;
                run += sh_sum[i];
            }
            sh_prefix[NT] = run;
        }
        __syncthreads();
    }
    const double total = sh_prefix[NT];
    const double target = (double)smp.u_res[r0 + jrow] * total;
    if (tid == 0) sh_int[1] = -1;
    __syncthreads();
    const double prefix = sh_prefix[tid];
    if (local > 0.0 && prefix <= target && target < prefix + local) {
        double run = 0.0;
        int found = -1, last = -1;
        for (int w = w0; w < w1 && found < 0; ++w) {
            if (tc[w / kWordsPerTile] == 0) continue;
            uint32_t bits = bw[w];
            while (bits) {
                const int t = w * 32 + __ffs(bits) - 1;
                bits &= bits - 1;
                const double wt = weight(t, residual);
                run += wt;
                if (wt > 0.0) {
                    last = t;
                    if (prefix + run > target) {
                        found = t;
                        break;
                    }
                }
            }
        }
        sh_int[1] = found >= 0 ? found : last;
    }
    __syncthreads();
    for (int i = tid; i < N; i += NT) out.accept_path[r0 + i] = i < k ? i : -1;
    if (tid == 0) {
        out.status[b] = 0;
        out.accept_len[b] = k - 1;
        out.next_token[b] = sh_int[1];
    }
}

}  // namespace

hipError_t launch_combine(const Plan &p, const Inputs &in, const Outputs &out, hipStream_t st) {
    const int want = out.node_stats != nullptr;
    if (p.dtype == kBF16)
        hipLaunchKernelGGL(combine_kernel<kBF16>, dim3(p.R), dim3(NT), 0, st, p, in, out.row_argmax,
                           out.row_stats, want);
    else
        hipLaunchKernelGGL(combine_kernel<kF32>, dim3(p.R), dim3(NT), 0, st, p, in, out.row_argmax,
                           out.row_stats, want);
    return hipGetLastError();
}

hipError_t launch_sequences(const Plan &p, const Inputs &in, const Outputs &out,
                            const SampleInputs *smp, hipStream_t st) {
    const SampleInputs s = smp ? *smp : SampleInputs{nullptr, nullptr, nullptr};
    if (p.dtype == kBF16) {
        if (smp)
            hipLaunchKernelGGL((sequence_kernel<kBF16, true>), dim3(p.B), dim3(NT), 0, st, p, in, out, s);
        else
            hipLaunchKernelGGL((sequence_kernel<kBF16, false>), dim3(p.B), dim3(NT), 0, st, p, in, out, s);
    } else {
        if (smp)
            hipLaunchKernelGGL((sequence_kernel<kF32, true>), dim3(p.B), dim3(NT), 0, st, p, in, out, s);
        else
            hipLaunchKernelGGL((sequence_kernel<kF32, false>), dim3(p.B), dim3(NT), 0, st, p, in, out, s);
    }
    return hipGetLastError();
}

}  // namespace dcd
