// C ABI of libdcd: argument validation, workspace planning and the launch
// sequence (LM heads + partials -> per-row combine -> per-sequence verification).
#include <math.h>

#include <mutex>

#include "../../include/dcd.h"
#include "dcd_internal.h"

namespace dcd {
namespace {

constexpr size_t kAlign = 256;
constexpr long long kMaxRows = 1 << 24;
constexpr long long kMaxVocab = 1 << 30;
constexpr int kMaxHidden = 1 << 20;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

int make_plan(const dcd_problem *p, bool sample, Plan &P) {
    if (!p) return DCD_ERR_NULL;
    if (p->batch < 1 || p->nodes < 1 || p->vocab < 1 || p->d_expert < 1 || p->d_amateur < 1)
        return DCD_ERR_SHAPE;
    const long long R = (long long)p->batch * p->nodes;
    if (p->nodes > kMaxNodes) return DCD_ERR_SHAPE;
    if (R > kMaxRows || p->vocab > kMaxVocab || p->d_expert > kMaxHidden ||
        p->d_amateur > kMaxHidden)
        return DCD_ERR_SHAPE;
    if (p->dtype != DCD_BF16 && p->dtype != DCD_F32) return DCD_ERR_PARAM;
    const int mult = p->dtype == DCD_BF16 ? 8 : 4;  // 16-byte rows
    if (p->d_expert % mult || p->d_amateur % mult) return DCD_ERR_ALIGN;
    if (!(p->plaus_thresh >= 0.f && p->plaus_thresh <= 1.f)) return DCD_ERR_PARAM;
    if (!(p->cd_strength >= 0.f) || !isfinite(p->cd_strength)) return DCD_ERR_PARAM;
    if (sample && (!(p->temperature > 0.f) || !isfinite(p->temperature))) return DCD_ERR_PARAM;
    if (p->final_norm != 0 && p->final_norm != 1) return DCD_ERR_PARAM;
    if (p->final_norm && (!(p->norm_eps >= 0.f) || !isfinite(p->norm_eps))) return DCD_ERR_PARAM;
    P = Plan{};
    P.final_norm = p->final_norm;
    P.norm_eps = p->norm_eps;
    P.B = p->batch;
    P.N = p->nodes;
    P.R = (int)R;
    P.V = p->vocab;
    P.dp = p->d_expert;
    P.dq = p->d_amateur;
    P.dtype = p->dtype == DCD_BF16 ? kBF16 : kF32;
    P.ntiles = (P.V + kTileTokens - 1) / kTileTokens;
    P.wstride = P.ntiles * kWordsPerTile;
    // ln(theta) in double, rounded once; theta = 0 switches the mask off
    P.log_theta = p->plaus_thresh > 0.f ? (float)log((double)p->plaus_thresh) : -INFINITY;
    P.full = p->plaus_thresh == 0.f;
    P.store_y = P.full && sample;
    P.zstride = P.ntiles * kTileTokens;
    P.s = p->cd_strength;
    P.inv_T = sample ? (float)(1.0 / (double)p->temperature) : 1.f;
    // from 65 to 511 rows the streaming kernel takes 128 rows per workgroup, so a
    // weight byte is streamed once for each 128 rows (10% faster at 128 rows); from
    // 512 rows the many-row kernel takes a bf16 problem, and fp32 ones keep 64-row
    // workgroups, two per CU
    P.rows_blk = P.R > kStreamRowsSmall && P.R < kWideMinRows ? kStreamRowsLarge : kStreamRowsSmall;
    P.nrb = (P.R + P.rows_blk - 1) / P.rows_blk;
    const long long groups = (long long)((P.ntiles + 7) / 8) * 8 * P.nrb;
    if (groups > 0x7fffffffLL) return DCD_ERR_SHAPE;
    return DCD_OK;
}

// the final RMS normalisation's scales: required (16-byte aligned) when asked for
int check_norm(const dcd_problem *p, const dcd_inputs *in) {
    if (!p->final_norm) return DCD_OK;
    if (!in->norm_expert || !in->norm_amateur) return DCD_ERR_NULL;
    if (!aligned(in->norm_expert, 16) || !aligned(in->norm_amateur, 16)) return DCD_ERR_ALIGN;
    return DCD_OK;
}

// With the final normalisation the rows are normalised into the workspace first,
// and every later kernel reads the normalised copies.
hipError_t normalise(const Plan &P, Inputs &I, hipStream_t st) {
    if (!P.final_norm) return hipSuccess;
    const hipError_t e = launch_rmsnorm(P, I, st);
    I.hp = P.hn_p;
    I.hq = P.hn_q;
    return e;
}

int check_io(const dcd_inputs *in, const dcd_outputs *out) {
    if (!in || !out) return DCD_ERR_NULL;
    if (!in->h_expert || !in->h_amateur || !in->w_expert || !in->w_amateur || !in->parents ||
        !in->tokens)
        return DCD_ERR_NULL;
    if (!out->accept_len || !out->accept_path || !out->next_token || !out->status)
        return DCD_ERR_NULL;
    if (!aligned(in->h_expert, 16) || !aligned(in->h_amateur, 16) || !aligned(in->w_expert, 16) ||
        !aligned(in->w_amateur, 16))
        return DCD_ERR_ALIGN;
    const void *four[] = {in->bias_expert, in->bias_amateur, in->parents, in->tokens,
                          out->accept_len, out->accept_path, out->next_token, out->status,
                          out->row_argmax, out->row_stats, out->node_stats,
                          out->row_argmax_expert, out->row_kl};
    for (const void *q : four)
        if (q && !aligned(q, 4)) return DCD_ERR_ALIGN;
    return DCD_OK;
}

int run(const dcd_problem *p, const dcd_inputs *in, const SampleInputs *smp,
        const dcd_outputs *out, void *ws, size_t ws_bytes, void *stream) {
    Plan P;
    int rc = make_plan(p, smp != nullptr, P);
    if (rc) return rc;
    if ((rc = check_io(in, out))) return rc;
    if ((rc = check_norm(p, in))) return rc;
    if (smp) {
        if (!smp->draft_probs || !smp->u_acc || !smp->u_res) return DCD_ERR_NULL;
        if (!aligned(smp->draft_probs, 4) || !aligned(smp->u_acc, 4) || !aligned(smp->u_res, 4))
            return DCD_ERR_ALIGN;
    }
    const size_t need = workspace_layout(P, nullptr);
    if (!ws || ws_bytes < need) return DCD_ERR_WORKSPACE;
    if (!aligned(ws, kAlign)) return DCD_ERR_WORKSPACE;
    workspace_layout(P, (char *)ws);

    Inputs I{in->h_expert, in->h_amateur, in->w_expert, in->w_amateur, in->bias_expert,
             in->bias_amateur, in->parents, in->tokens, in->norm_expert, in->norm_amateur};
    const Outputs O{out->accept_len,        out->accept_path, out->next_token, out->status,
                    out->row_argmax,        out->row_stats,   out->node_stats,
                    out->row_argmax_expert, out->row_kl};
    hipStream_t st = (hipStream_t)stream;
    // untruncated sampled verification: each sequence's walk spread over a group of
    // workgroups, one per CU
    P.walk_group = smp && P.full ? walk_group_size(P, (hipStream_t)stream) : 0;
    if (normalise(P, I, st) != hipSuccess) return DCD_ERR_HIP;
    if (launch_lmhead(P, I, st) != hipSuccess) return DCD_ERR_HIP;
    if (launch_finish(P, I, O, smp, st) != hipSuccess) {
        launch_advance_call(P, st);  // the next call must not see this call's ready word
        return DCD_ERR_HIP;
    }
    if (P.walk_group && launch_walk(P, I, O, *smp, st) != hipSuccess) return DCD_ERR_HIP;
    return DCD_OK;
}

int run_lmhead(const dcd_problem *p, const dcd_inputs *in, int sampled, void *ws, size_t ws_bytes,
               void *stream) {
    Plan P;
    int rc = make_plan(p, sampled != 0, P);
    if (rc) return rc;
    if (!in) return DCD_ERR_NULL;
    if (!in->h_expert || !in->h_amateur || !in->w_expert || !in->w_amateur) return DCD_ERR_NULL;
    if (!aligned(in->h_expert, 16) || !aligned(in->h_amateur, 16) || !aligned(in->w_expert, 16) ||
        !aligned(in->w_amateur, 16) || !aligned(in->bias_expert, 4) || !aligned(in->bias_amateur, 4))
        return DCD_ERR_ALIGN;
    if ((rc = check_norm(p, in))) return rc;
    const size_t need = workspace_layout(P, nullptr);
    if (!ws || ws_bytes < need || !aligned(ws, kAlign)) return DCD_ERR_WORKSPACE;
    workspace_layout(P, (char *)ws);
    Inputs I{in->h_expert, in->h_amateur, in->w_expert, in->w_amateur, in->bias_expert,
             in->bias_amateur, in->parents, in->tokens, in->norm_expert, in->norm_amateur};
    if (normalise(P, I, (hipStream_t)stream) != hipSuccess) return DCD_ERR_HIP;
    if (launch_lmhead(P, I, (hipStream_t)stream) != hipSuccess) return DCD_ERR_HIP;
    return launch_advance_call(P, (hipStream_t)stream) == hipSuccess ? DCD_OK : DCD_ERR_HIP;
}

int run_propose(const dcd_problem *p, const dcd_inputs *in, const ProposeOutputs &o, void *ws,
                size_t ws_bytes, void *stream) {
    Plan P;
    int rc = make_plan(p, true, P);  // the temperature applies, both heads' logits are kept
    if (rc) return rc;
    if (!in) return DCD_ERR_NULL;
    if (!in->h_expert || !in->h_amateur || !in->w_expert || !in->w_amateur) return DCD_ERR_NULL;
    if (!o.tokens && !o.probs && !o.argmax) return DCD_ERR_NULL;
    if (o.tokens && !o.u) return DCD_ERR_NULL;
    if ((rc = check_norm(p, in))) return rc;
    if (!aligned(in->h_expert, 16) || !aligned(in->h_amateur, 16) || !aligned(in->w_expert, 16) ||
        !aligned(in->w_amateur, 16) || !aligned(in->bias_expert, 4) || !aligned(in->bias_amateur, 4) ||
        !aligned(o.u, 4) || !aligned(o.tokens, 4) || !aligned(o.probs, 4) || !aligned(o.argmax, 4))
        return DCD_ERR_ALIGN;
    const size_t need = workspace_layout(P, nullptr);
    if (!ws || ws_bytes < need || !aligned(ws, kAlign)) return DCD_ERR_WORKSPACE;
    workspace_layout(P, (char *)ws);
    Inputs I{in->h_expert, in->h_amateur, in->w_expert, in->w_amateur, in->bias_expert,
             in->bias_amateur, nullptr, nullptr, in->norm_expert, in->norm_amateur};
    hipStream_t st = (hipStream_t)stream;
    if (normalise(P, I, st) != hipSuccess) return DCD_ERR_HIP;
    if (launch_lmhead(P, I, st) != hipSuccess) return DCD_ERR_HIP;
    if (launch_propose(P, I, o, st) != hipSuccess) {
        launch_advance_call(P, st);
        return DCD_ERR_HIP;
    }
    return DCD_OK;
}

}  // namespace

size_t workspace_layout(Plan &p, char *base) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *ptr = base ? base + off : nullptr;
        off += round_up(bytes);
        return ptr;
    };
    const size_t R = (size_t)p.R;
    // first, at the same place for every problem: the call count and ready word
    p.ctl = (uint32_t *)take(2 * sizeof(uint32_t));
    p.partials = (float4 *)take(R * p.ntiles * sizeof(float4));
    if (p.full) {  // dense y (and, for the 128-row shape, expert logits), per-tile statistics of y
        p.zp_full = p.rows_blk == kStreamRowsLarge ? (float *)take(R * (size_t)p.zstride * sizeof(float)) : nullptr;
        p.y_full = (float *)take(R * (size_t)p.zstride * sizeof(float));
        p.ypart = (float4 *)take(R * p.ntiles * 2 * sizeof(float4));
        p.resbuf = (double *)take((size_t)p.B * 2 * p.zstride * sizeof(double));
        p.walkbar = (int *)take((size_t)p.B * 2 * sizeof(int));
        p.walkpart = (double *)take((size_t)p.B * 2 * kWalkMaxGroup * sizeof(double));
    } else {  // candidates of the mask
        p.cand = (float2 *)take(R * (size_t)p.V * sizeof(float2));
        p.bits = (uint32_t *)take(R * (size_t)p.wstride * sizeof(uint32_t));
    }
    p.rowinfo = (float *)take(R * kRowInfo * sizeof(float));
    p.tcount = (int *)take(R * p.ntiles * sizeof(int));
    p.bound = (uint32_t *)take((size_t)kBoundCopies * R * sizeof(uint32_t));
    p.nodez = (float4 *)take(R * sizeof(float4));
    p.seqdone = (int *)take((size_t)2 * p.B * sizeof(int));  // seqdone, then seqfail
    p.seqfail = p.seqdone + p.B;
    p.wratio = (double *)take(R * sizeof(double));
    p.wterm = (int *)take(R * sizeof(int));
    if (p.final_norm) {
        const size_t esz = p.dtype == kBF16 ? 2 : 4;
        p.hn_p = take(R * p.dp * esz);
        p.hn_q = take(R * p.dq * esz);
    }
    return off;
}

// ---------------------------------------------------------------------------
// The allocation-free entry point: the same launches as dcd_verify_greedy, with
// the workspace taken from a static device array instead of the caller.
//
// One array per GPU the library runs on, held until the process ends.  Its size
// covers 64 rows of a 128,256-token vocabulary in every mode (about 69 MB at
// plaus_thresh 0, 67 MB with a mask); larger problems are refused.  Host code never
// passes the array's name to a kernel (on the host it is only a handle of the
// symbol): the device address comes from hipGetSymbolAddress, once per device,
// with that device current.  The calls share each GPU's array, so calls that
// overlap on one GPU race.  Like a caller's workspace, it starts with the call
// count and ready word of the LM-head launch's clearing step (zero at load); every
// other word a call reads it has written or cleared first.
constexpr size_t kScratchBytes = (size_t)80 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch[kMaxDevices];  // device address of `scratch` per device (null: not looked up)

// Device address of this device's scratch array, looked up on the first call that
// runs on it (with that device current).  Returns DCD_OK or DCD_ERR_HIP.
int scratch_for(hipStream_t stream, void **out) {
    int dev = -1;
    hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) return DCD_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch[dev]) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return DCD_ERR_HIP;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return DCD_ERR_HIP;
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev) hipSetDevice(cur);
        if (e != hipSuccess || !ptr) return DCD_ERR_HIP;
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return DCD_OK;
}

int run_greedy_noalloc(const dcd_problem *p, const dcd_inputs *in, const dcd_outputs *out,
                       void *stream) {
    // the size check needs no device: refuse before touching one
    Plan P;
    int rc = make_plan(p, false, P);
    if (rc) return rc;
    if (workspace_layout(P, nullptr) > kScratchBytes) return DCD_ERR_TOO_LARGE;
    void *ws = nullptr;
    if ((rc = scratch_for((hipStream_t)stream, &ws))) return rc;
    return run(p, in, nullptr, out, ws, kScratchBytes, stream);
}

}  // namespace

}  // namespace dcd

extern "C" {

int dcd_verify_greedy_noalloc(const dcd_problem *p, const dcd_inputs *in, const dcd_outputs *out,
                              void *hip_stream) {
    return dcd::run_greedy_noalloc(p, in, out, hip_stream);
}

size_t dcd_noalloc_max_bytes(void) { return dcd::kScratchBytes; }

size_t dcd_workspace_bytes(const dcd_problem *p) {
    dcd::Plan P;
    if (dcd::make_plan(p, false, P) != DCD_OK) return 0;
    return dcd::workspace_layout(P, nullptr);
}

int dcd_verify_greedy(const dcd_problem *p, const dcd_inputs *in, const dcd_outputs *out,
                      void *workspace, size_t workspace_bytes, void *hip_stream) {
    return dcd::run(p, in, nullptr, out, workspace, workspace_bytes, hip_stream);
}

int dcd_verify_sample(const dcd_problem *p, const dcd_inputs *in, const float *draft_probs,
                      const float *u_accept, const float *u_resample, const dcd_outputs *out,
                      void *workspace, size_t workspace_bytes, void *hip_stream) {
    const dcd::SampleInputs s{draft_probs, u_accept, u_resample};
    return dcd::run(p, in, &s, out, workspace, workspace_bytes, hip_stream);
}

int dcd_propose(const dcd_problem *p, const dcd_inputs *in, const float *u, int32_t *tokens,
                float *probs, int32_t *argmax, void *workspace, size_t workspace_bytes,
                void *hip_stream) {
    return dcd::run_propose(p, in, dcd::ProposeOutputs{u, tokens, probs, argmax}, workspace,
                            workspace_bytes, hip_stream);
}

int dcd_lmhead_partials(const dcd_problem *p, const dcd_inputs *in, int sampled, void *workspace,
                        size_t workspace_bytes, void *hip_stream) {
    return dcd::run_lmhead(p, in, sampled, workspace, workspace_bytes, hip_stream);
}

const char *dcd_error_string(int code) {
    switch (code) {
        case DCD_OK: return "success";
        case DCD_ERR_NULL: return "a required pointer is NULL";
        case DCD_ERR_SHAPE: return "a size is out of range or inconsistent";
        case DCD_ERR_PARAM: return "invalid plaus_thresh, cd_strength, temperature or dtype";
        case DCD_ERR_ALIGN: return "pointer or hidden-size alignment violated";
        case DCD_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case DCD_ERR_UNSUPPORTED: return "request not supported by this build";
        case DCD_ERR_HIP: return "the HIP runtime rejected a launch";
        case DCD_ERR_TOO_LARGE:
            return "the problem needs more device memory than the allocation-free entry point holds";
        default: return "unknown error code";
    }
}

int dcd_abi_version(void) { return 7; }

}  // extern "C"
