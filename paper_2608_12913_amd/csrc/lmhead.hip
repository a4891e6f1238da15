// LM-head projection of both models with a fused softmax-partials and
// candidate epilogue (Alg. 1 "parallel model evaluation" followed by the
// per-tile pieces of Eq. (1) and the plausibility mask of Sec. 2.1).
//
// One workgroup = 4 waves = one tile of 256 vocabulary tokens x 64 rows.
// Each wave owns 64 tokens (4 blocks of 16) for all 64 rows (4 blocks of 16)
// and accumulates z^T = W_tile * H^T with v_mfma_f32_16x16x32_bf16 (bf16) or
// v_mfma_f32_16x16x4_f32 (fp32): the weight rows are the MFMA A operand, read
// straight from HBM with 128-bit loads (16 tokens x 64 contiguous bytes per
// instruction), the hidden states are the B operand, staged per K-chunk in LDS
// and shared by the four waves.  The expert head is processed first, then the
// amateur head; only one model's accumulators are live at a time.
//
// Per (row, tile) the epilogue writes the tile's max and sum of exp for both
// models, and marks every token whose expert logit is within ln(theta) of the
// tile max as a candidate: the final mask {z_p >= max_row z_p + ln theta} can only
// contain candidates, because the tile max never exceeds the row max.  Candidate
// logits go to a sparse [row][token] array, their positions to a bitmap.
#include "dcd_internal.h"

namespace dcd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int CB = 128;                 // bytes of each row per K-chunk
constexpr int KSTEPS = CB / 64;         // MFMA k-steps per chunk (64 bytes of a row each)
constexpr int LSTRIDE = CB + 16;        // padded LDS row stride in bytes
constexpr int VB = kTileVBlocks;
constexpr int RB = kTileRBlocks;
constexpr int NT = kTileWaves * kWaveSize;  // threads per workgroup

// One 16-byte A fragment x one 16-byte B fragment, accumulated into c.
template <int DT>
__device__ __forceinline__ f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
    if constexpr (DT == kBF16) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    } else {
        f32x4 af = __builtin_bit_cast(f32x4, a), bf = __builtin_bit_cast(f32x4, b);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[0], bf[0], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[1], bf[1], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[2], bf[2], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[3], bf[3], c, 0, 0, 0);
        return c;
    }
}

__device__ __forceinline__ u32x4 ld16(const char *p) {
    return *reinterpret_cast<const u32x4 *>(p);
}

struct ModelArgs {
    const char *h;      // [R][d] elements
    const char *w;      // [V][d] elements
    const float *bias;  // [V] or null
    int d;              // hidden size
};

// Accumulate one model's logits for this workgroup's tile.
//   acc[vb][rb]: lane l holds z[token 16vb + 4(l/16) + j][row 16rb + l%16], j = 0..3
template <int DT>
__device__ __forceinline__ void accumulate(const ModelArgs &m, int R, int V, int row0, int tok0,
                                           char *lds, f32x4 (&acc)[VB][RB]) {
    constexpr int ESZ = DT == kBF16 ? 2 : 4;
    const int lane = threadIdx.x % kWaveSize;
    const int tid = threadIdx.x;
    const int n = lane % 16, g = lane / 16;
    const size_t rowbytes = (size_t)m.d * ESZ;
    const int nch = (int)((rowbytes + CB - 1) / CB);

    // Addresses: a wave-uniform base (kept in SGPRs) plus 32-bit per-lane offsets,
    // so every load uses the scalar-base addressing form.  Tokens past the
    // vocabulary read the last row (their results are discarded later).
    const int tbase = min(tok0, V - 1);
    const char *wbase = m.w + (size_t)tbase * rowbytes;
    uint32_t woff[VB];
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) {
        const int t = min(tok0 + vb * 16 + n, V - 1);
        woff[vb] = (uint32_t)((t - tbase) * rowbytes);
    }
    // hidden-state staging: thread -> (row, 16-byte column) of the chunk
    constexpr int TPR = CB / 16;          // threads per row
    constexpr int RPP = NT / TPR;         // rows per pass
    constexpr int PASSES = kTileRows / RPP;
    const int hcol = (tid % TPR) * 16;
    const int hrow = tid / TPR;
    const char *hbase = m.h + (size_t)row0 * rowbytes;
    uint32_t hoff[PASSES];
    bool hok[PASSES];
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
        const int r = row0 + hrow + p * RPP;
        hok[p] = r < R;
        hoff[p] = (uint32_t)((min(r, R - 1) - row0) * rowbytes);
    }

#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Weight loads are unconditional and never masked: in the K tail a lane's
    // column is clamped to the row's last 16 bytes (finite weights) and the
    // matching hidden-state columns are zero in LDS, so the product vanishes.
    // No select touches the loaded registers, so nothing waits on them before
    // their MFMA.
    auto load_w = [&](int c, u32x4 (&wb)[KSTEPS][VB]) {
        const uint32_t cofs = (uint32_t)c * CB;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const uint32_t col = min(cofs + s * 64 + g * 16, (uint32_t)rowbytes - 16);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) wb[s][vb] = ld16(wbase + woff[vb] + col);
        }
    };
    auto load_h = [&](int c, u32x4 (&hb)[PASSES]) {
        const uint32_t col = (uint32_t)c * CB + hcol;
        const bool kok = col < rowbytes;
        const char *base = hbase + (kok ? col : 0);  // past the row end: read its start, store 0
#pragma unroll
        for (int p = 0; p < PASSES; ++p) {
            const u32x4 v = ld16(base + hoff[p]);
            hb[p] = (kok && hok[p]) ? v : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto store_h = [&](int buf, const u32x4 (&hb)[PASSES]) {
        char *base = lds + buf * (kTileRows * LSTRIDE);
#pragma unroll
        for (int p = 0; p < PASSES; ++p)
            *reinterpret_cast<u32x4 *>(base + (hrow + p * RPP) * LSTRIDE + hcol) = hb[p];
    };
    auto compute = [&](int buf, const u32x4 (&wb)[KSTEPS][VB]) {
        const char *base = lds + buf * (kTileRows * LSTRIDE) + n * LSTRIDE + g * 16;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            u32x4 bfr[RB];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
                bfr[rb] = *reinterpret_cast<const u32x4 *>(base + rb * 16 * LSTRIDE + s * 64);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb)
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = mma<DT>(wb[s][vb], bfr[rb], acc[vb][rb]);
        }
    };

    u32x4 w0[KSTEPS][VB], w1[KSTEPS][VB], hb[PASSES];
    load_h(0, hb);
    load_w(0, w0);
    store_h(0, hb);
    __syncthreads();
    // Steady state: two chunks per iteration (static register double buffer);
    // both prefetches of an iteration exist, so no load is conditional.  The
    // last one or two chunks are peeled.
    int c = 0;
    for (; c + 2 < nch; c += 2) {
        load_h(c + 1, hb);  // hidden states first: the LDS store waits only for them
        load_w(c + 1, w1);
        compute(0, w0);
        store_h(1, hb);
        __syncthreads();
        load_h(c + 2, hb);
        load_w(c + 2, w0);
        compute(1, w1);
        store_h(0, hb);
        __syncthreads();
    }
    if (c + 1 < nch) {
        load_h(c + 1, hb);
        load_w(c + 1, w1);
        compute(0, w0);
        store_h(1, hb);
        __syncthreads();
        compute(1, w1);
    } else {
        compute(0, w0);
    }
    __syncthreads();
    // keep the epilogue's loads and address arithmetic out of the K loop
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ float wave_max16_32(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float wave_sum16_32(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}
__device__ __forceinline__ uint32_t wave_or16_32(uint32_t x) {
    x |= (uint32_t)__shfl_xor((int)x, 16);
    return x | (uint32_t)__shfl_xor((int)x, 32);
}

// Logits of this lane's 64 (token, row) values, tile max and sum of exp per row.
//   z[vb][rb][j]    logit (already divided by T); -inf for tokens >= V
//   tmax[rb], tsum[rb]   tile max / sum exp(z - max) of row 16rb + lane%16
__device__ __forceinline__ void tile_softmax(const f32x4 (&acc)[VB][RB], const float *bias, int V,
                                             int tok0, float inv_T, float *red,
                                             float (&z)[VB][RB][4], float (&tmax)[RB],
                                             float (&tsum)[RB]) {
    const int lane = threadIdx.x % kWaveSize, wave = threadIdx.x / kWaveSize;
    const int n = lane % 16, g = lane / 16;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int t = tok0 + vb * 16 + 4 * g + j;
            const bool ok = t < V;
            const float b = (ok && bias) ? bias[t] : 0.f;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) z[vb][rb][j] = ok ? (acc[vb][rb][j] + b) * inv_T : -INFINITY;
        }
    float wmax[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float m = -INFINITY;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) m = fmaxf(m, z[vb][rb][j]);
        wmax[rb] = wave_max16_32(m);
        if (g == 0) red[wave * kTileRows + rb * 16 + n] = wmax[rb];
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float m = red[rb * 16 + n];
#pragma unroll
        for (int w = 1; w < kTileWaves; ++w) m = fmaxf(m, red[w * kTileRows + rb * 16 + n]);
        tmax[rb] = m;
    }
    __syncthreads();  // red is rewritten below
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float s = 0.f;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) s += __expf(z[vb][rb][j] - tmax[rb]);
        s = wave_sum16_32(s);
        if (g == 0) red[wave * kTileRows + rb * 16 + n] = s;
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kTileWaves; ++w) s += red[w * kTileRows + rb * 16 + n];
        tsum[rb] = s;
    }
    __syncthreads();  // red is reused by the next phase
}

template <int DT>
__global__ __launch_bounds__(NT, 2) void lmhead_kernel(Plan P, Inputs in) {
    extern __shared__ __align__(16) char lds[];
    float *red = reinterpret_cast<float *>(lds + 2 * kTileRows * LSTRIDE);

    // workgroup -> (vocabulary tile, row block); the row blocks of one tile are
    // dispatched back to back on the same XCD (workgroup id modulo 8) so the
    // tile's weights are re-read from that XCD's L2
    const int id = blockIdx.x, xcd = id % 8, local = id / 8;
    const int rblk = local % P.nrb;
    const int tile = (local / P.nrb) * 8 + xcd;
    if (tile >= P.ntiles) return;
    const int row0 = rblk * kTileRows;
    const int lane = threadIdx.x % kWaveSize;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);  // wave-uniform
    const int n = lane % 16, g = lane / 16;
    const int tok0 = tile * kTileTokens + wave * (VB * 16);

    f32x4 acc[VB][RB];
    float z[VB][RB][4];
    float pmax[RB], psum[RB], qmax[RB], qsum[RB];
    uint32_t flags[RB];  // bit (vb*4 + j): candidate

    // ---- expert head
    accumulate<DT>(ModelArgs{(const char *)in.hp, (const char *)in.wp, in.bp, P.dp}, P.R, P.V, row0,
                   tok0, lds, acc);
    tile_softmax(acc, in.bp, P.V, tok0, P.inv_T, red, z, pmax, psum);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = row0 + rb * 16 + n;
        const float thr = pmax[rb] + P.log_theta;
        uint32_t f = 0, word0 = 0, word1 = 0;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int t = tok0 + vb * 16 + 4 * g + j;
                const bool c = t < P.V && z[vb][rb][j] >= thr;
                if (c) {
                    f |= 1u << (vb * 4 + j);
                    if (row < P.R) P.cand[(size_t)row * P.V + t].x = z[vb][rb][j];
                }
                const uint32_t bit = (uint32_t)c << ((vb & 1) * 16 + 4 * g + j);
                if (vb < 2) word0 |= bit; else word1 |= bit;
            }
        flags[rb] = f;
        word0 = wave_or16_32(word0);
        word1 = wave_or16_32(word1);
        if (g == 0 && row < P.R) {
            uint32_t *bw = P.bits + (size_t)row * P.wstride + tile * kWordsPerTile + wave * 2;
            bw[0] = word0;
            bw[1] = word1;
        }
    }

    // ---- amateur head
    accumulate<DT>(ModelArgs{(const char *)in.hq, (const char *)in.wq, in.bq, P.dq}, P.R, P.V, row0,
                   tok0, lds, acc);
    tile_softmax(acc, in.bq, P.V, tok0, P.inv_T, red, z, qmax, qsum);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = row0 + rb * 16 + n;
        if (row >= P.R) continue;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (flags[rb] >> (vb * 4 + j) & 1u) {
                    const int t = tok0 + vb * 16 + 4 * g + j;
                    P.cand[(size_t)row * P.V + t].y = z[vb][rb][j];
                }
        if (wave == 0 && g == 0)
            P.partials[(size_t)row * P.ntiles + tile] = float4{pmax[rb], psum[rb], qmax[rb], qsum[rb]};
    }
}

}  // namespace

hipError_t launch_lmhead(const Plan &p, const Inputs &in, hipStream_t st) {
    const int groups = ((p.ntiles + 7) / 8) * 8 * p.nrb;
    const size_t lds = 2 * kTileRows * LSTRIDE + kTileWaves * kTileRows * sizeof(float);
    if (p.dtype == kBF16)
        hipLaunchKernelGGL(lmhead_kernel<kBF16>, dim3(groups), dim3(NT), lds, st, p, in);
    else
        hipLaunchKernelGGL(lmhead_kernel<kF32>, dim3(groups), dim3(NT), lds, st, p, in);
    return hipGetLastError();
}

}  // namespace dcd
