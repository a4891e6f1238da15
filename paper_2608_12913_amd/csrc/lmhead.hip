// LM-head projection of both models with a fused softmax-partials and
// candidate epilogue (Alg. 1 "parallel model evaluation" followed by the
// per-tile pieces of Eq. (1) and the plausibility mask of Sec. 2.1).
//
// Tiling.  One workgroup = kTileWaves waves = one tile of 16*kTileWaves
// vocabulary tokens x 64 rows.  Each wave owns 16 consecutive tokens and
// accumulates z^T[16 tokens][64 rows] = W * H^T with 4 MFMA blocks per k-step
// (v_mfma_f32_16x16x32_bf16, or 4 x v_mfma_f32_16x16x4_f32 for fp32).  K is
// walked in chunks of 256 bytes of every row.
//
// Weight stream (HBM-bound part).  A wave reads its 16 rows with non-temporal
// 128-bit loads, 4 rows x 256 contiguous bytes per instruction, two chunks in
// flight.  HBM3E delivers the most bandwidth for exactly this shape (long runs
// per row, few rows open per wave, streaming cache policy); the MFMA A-fragment
// shape (16 rows x 64 bytes per instruction) reaches noticeably less.  The
// chunk is therefore transposed through a wave-private LDS buffer into
// fragment order.  Hidden states (the B operand, shared by all waves) are
// staged per chunk in a double-buffered LDS tile.  Both LDS tiles use an XOR
// swizzle (16-byte column c of row m stored at slot c ^ (m mod 16)) so the
// fragment reads of 16 lanes hit 16 distinct bank groups.
//
// Epilogue.  Per (row, tile): the tile max and sum of exp of both models, and
// the plausibility candidates: tokens whose expert logit is within ln(theta)
// of a lower bound on the row max (the larger of the tile max and a running
// per-row maximum shared through an atomic).  The final mask
// {z_p >= row max + ln theta} can only contain candidates.  Candidate logits go
// to a sparse [row][token] array, their positions to a bitmap, their number
// per (row, tile) to a count array.
#include "dcd_internal.h"

namespace dcd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int NW = kTileWaves;
constexpr int VB = kTileVBlocks;          // 16-token blocks per wave
constexpr int NT = NW * kWaveSize;        // threads per workgroup
constexpr int TS = kTileTokens;           // tokens per tile
constexpr int RB = kTileRBlocks;          // 16-row blocks
constexpr int ROWS = kTileRows;           // 64
#ifndef DCD_CHUNK_BYTES
#define DCD_CHUNK_BYTES 128
#endif

constexpr int CB = DCD_CHUNK_BYTES;       // bytes of every row per K-chunk
constexpr int LPR = CB / 16;              // lanes per row in a weight load instruction
constexpr int RPI = kWaveSize / LPR;      // rows per weight load instruction
constexpr int WLOADS = 16 * kTileVBlocks / RPI;  // weight load instructions per wave and chunk
constexpr int KS = CB / 64;               // MFMA k-steps per chunk
constexpr int HLOADS = ROWS * CB / (NT * 16);  // 16-byte hidden-state loads per thread and chunk
constexpr int WTILE = VB * 16 * CB;       // bytes of one wave's weight chunk (16*VB rows)
constexpr int HTILE = ROWS * CB;          // bytes of one hidden-state chunk
static_assert(HLOADS >= 1 && ROWS * CB == HLOADS * NT * 16, "hidden-state staging must tile");
static_assert(CB % 64 == 0 && WLOADS * RPI == 16 * kTileVBlocks, "weight chunk must tile");
static_assert(TS == 16 * VB * NW && TS % 32 == 0, "tile = 16*VB tokens per wave, whole bitmap words");

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

__device__ __forceinline__ u32x4 ld16_stream(const char *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
__device__ __forceinline__ u32x4 ld16(const char *p) { return *reinterpret_cast<const u32x4 *>(p); }
__device__ __forceinline__ void st_lds(char *p, u32x4 v) { *reinterpret_cast<u32x4 *>(p) = v; }
__device__ __forceinline__ u32x4 ld_lds(const char *p) { return *reinterpret_cast<const u32x4 *>(p); }

// byte offset of 16-byte column c of row m inside a swizzled [rows][CB] LDS tile:
// consecutive rows rotate their columns, so 16 lanes reading the same column of 16
// rows touch distinct bank groups
__device__ __forceinline__ int swz(int m, int c) { return m * CB + ((c ^ (m % LPR)) << 4); }

struct ModelArgs {
    const char *h;      // [R][d] elements
    const char *w;      // [V][d] elements
    int d;              // hidden size (elements)
};

// The loads of one K-chunk: this wave's 16 weight rows and this thread's share of
// the 64 hidden-state rows.
struct Batch {
    u32x4 w[WLOADS];
    u32x4 h[HLOADS];
    bool hok;  // the hidden-state columns are inside the row (false only in the K tail)
};

// Accumulate one model's logits for this workgroup's tile.
//   acc[vb][rb]: lane l holds z[token tok0 + 16vb + 4(l/16) + j][row row0 + 16rb + l%16]
// RAGGED: some of the wave's 16*VB rows lie past the vocabulary (only in the last
// tile); their loads are clamped to the last row and their results discarded.
template <int DT, bool RAGGED>
__device__ __forceinline__ void accumulate(const ModelArgs &m, int R, int V, int row0, int tok0,
                                           char *hbuf, char *wbuf, f32x4 (&acc)[VB][RB]) {
    constexpr int ESZ = DT == kBF16 ? 2 : 4;
    const int tid = threadIdx.x, lane = tid % kWaveSize;
    const int n = lane % 16, g = lane / 16;
    const uint32_t rowbytes = (uint32_t)m.d * ESZ;
    const int nch = (int)((rowbytes + CB - 1) / CB);

    // Weight loads: lane (r, c) = (lane / LPR, lane % LPR) reads 16 bytes at column c
    // of row RPI*q + r of the wave's 16*VB rows, RPI rows x CB contiguous bytes per
    // instruction.  Address = wave-uniform row base (scalar registers) + a 32-bit
    // lane offset, so the loads use the scalar-base form.
    const int wr = lane / LPR, wc = lane % LPR;
    const int tbase = min(tok0, V - 1);
    const char *wbase = m.w + (size_t)tbase * rowbytes;
    const uint32_t wlane = (uint32_t)wr * rowbytes;
    uint32_t woff[RAGGED ? WLOADS : 1];  // ragged: per-instruction clamped row offsets
    if constexpr (RAGGED) {
#pragma unroll
        for (int q = 0; q < WLOADS; ++q)
            woff[q] = (uint32_t)(min(tok0 + RPI * q + wr, V - 1) - tbase) * rowbytes;
    }
    // Hidden-state loads: thread -> (row, 16-byte column) of the 64 x CB chunk; rows
    // past R re-read row R-1 (results discarded).
    const int hc = tid % LPR, hr0 = tid / LPR;
    const char *hbase = m.h + (size_t)row0 * rowbytes;
    uint32_t hoff[HLOADS];
#pragma unroll
    for (int p = 0; p < HLOADS; ++p)
        hoff[p] = (uint32_t)(min(row0 + hr0 + p * (NT / LPR), R - 1) - row0) * rowbytes;

    // LDS addresses (swizzled, see swz): the lane-dependent parts are formed once.
    // Weight row RPI*q + wr of the wave tile: its swizzle only depends on q % (LPR/RPI).
    constexpr int QX = LPR / RPI;  // distinct weight-row swizzles per lane
    int wst[QX];
#pragma unroll
    for (int k = 0; k < QX; ++k) wst[k] = swz(RPI * k + wr, wc);
    const int hst = swz(hr0, hc);  // rows hr0 + p*NT/LPR share hr0's swizzle (NT/LPR % LPR == 0)
    static_assert((NT / LPR) % LPR == 0, "hidden-state rows of one thread share a swizzle");
    int frag[KS];  // fragment column 4s+g of row n (rows 16vb+n / 16rb+n add constants)
#pragma unroll
    for (int s = 0; s < KS; ++s) frag[s] = swz(n, 4 * s + g);
    static_assert(16 % LPR == 0 || LPR % 16 == 0, "fragment rows 16vb+n share row n's swizzle");

#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // In the K tail (rowbytes not a multiple of CB) a weight lane past the row end
    // re-reads the row's last 16 bytes (finite values) and the hidden-state
    // columns there are zero, so those products vanish.
    auto issue = [&](int c, Batch &b) {
        const uint32_t col = (uint32_t)c * CB + wc * 16;
        const uint32_t wcol = col < rowbytes ? col : rowbytes - 16;
#pragma unroll
        for (int q = 0; q < WLOADS; ++q) {
            if constexpr (RAGGED)
                b.w[q] = ld16_stream(wbase + (woff[q] + wcol));
            else
                b.w[q] = ld16_stream(wbase + (size_t)q * RPI * rowbytes + (wlane + wcol));
        }
        const uint32_t hcol = (uint32_t)c * CB + hc * 16;
        b.hok = hcol < rowbytes;
#pragma unroll
        for (int p = 0; p < HLOADS; ++p) b.h[p] = ld16(hbase + (hoff[p] + (b.hok ? hcol : 0u)));
    };
    // arrived batch -> LDS: hidden states into the shared tile (zero in the K tail),
    // the wave's weights into its private transpose tile.  Nothing inspects loaded
    // registers before this point, so no wait is forced on loads still in flight.
    auto stage = [&](const Batch &b) {
#pragma unroll
        for (int p = 0; p < HLOADS; ++p)
            st_lds(hbuf + hst + p * (NT / LPR) * CB, b.hok ? b.h[p] : u32x4{0u, 0u, 0u, 0u});
#pragma unroll
        for (int q = 0; q < WLOADS; ++q) st_lds(wbuf + wst[q % QX] + (q / QX) * (QX * RPI) * CB, b.w[q]);
    };
    auto compute = [&]() {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            // one k-step at a time: hoisting every fragment read of the chunk would
            // cost KS times the fragment registers
            __builtin_amdgcn_sched_barrier(0);
            u32x4 bfr[RB];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) bfr[rb] = ld_lds(hbuf + frag[s] + 16 * rb * CB);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) {
                const u32x4 a = ld_lds(wbuf + frag[s] + 16 * vb * CB);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = mma<DT>(a, bfr[rb], acc[vb][rb]);
            }
        }
    };

    // Pipeline: one batch in flight.  Chunk c is staged (its registers are then
    // free), chunk c+1 is issued, chunk c is computed.  One hidden-state tile: a
    // barrier before staging (every wave is done reading chunk c-1) and one after
    // (the tile is complete).  The weight tile is wave-private, so the wave's own
    // program order protects it.  The scheduling barrier pins the prefetch before
    // the compute (left free, the scheduler may sink the loads).
    Batch b0;
    issue(0, b0);
    for (int c = 0; c < nch; ++c) {
        if (c) __syncthreads();
        stage(b0);
        if (c + 1 < nch) issue(c + 1, b0);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        compute();
    }
    __syncthreads();  // LDS tiles are reused by the next pass
}

__device__ __forceinline__ float wave_max16_32(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float wave_sum16_32(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}

// Logits of this lane's 16*VB (token, row) values, tile max and sum of exp per row.
//   z[vb][rb][j]    logit (divided by T); -inf for tokens >= V
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
            const int t = tok0 + 16 * vb + 4 * g + j;
            const bool ok = t < V;
            const float b = (ok && bias) ? bias[t] : 0.f;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
                z[vb][rb][j] = ok ? (acc[vb][rb][j] + b) * inv_T : -INFINITY;
        }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float m = -INFINITY;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) m = fmaxf(m, z[vb][rb][j]);
        m = wave_max16_32(m);
        if (g == 0) red[wave * ROWS + rb * 16 + n] = m;
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float m = red[rb * 16 + n];
#pragma unroll
        for (int w = 1; w < NW; ++w) m = fmaxf(m, red[w * ROWS + rb * 16 + n]);
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
        if (tmax[rb] == -INFINITY) s = 0.f;  // nothing finite in this tile row
        s = wave_sum16_32(s);
        if (g == 0) red[wave * ROWS + rb * 16 + n] = s;
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) s += red[w * ROWS + rb * 16 + n];
        tsum[rb] = s;
    }
    __syncthreads();  // red is reused by the next phase
}

// float <-> int keys whose signed-integer order is the float order (for atomicMax)
__device__ __forceinline__ int ordered_key(float f) {
    const int i = __float_as_int(f);
    return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ __forceinline__ float key_value(int k) {
    return __int_as_float(k >= 0 ? k : k ^ 0x7fffffff);
}

constexpr int kHTiles = 1;  // hidden-state tiles in LDS
// epilogue scratch (row reductions, candidate words and counts) reuses the
// hidden-state tiles, which are idle once a pass has accumulated
constexpr size_t kEpilogueBytes = NW * ROWS * sizeof(float) + ROWS * kWordsPerTile * sizeof(uint32_t) +
                                  ROWS * sizeof(int);
static_assert(kEpilogueBytes <= (size_t)kHTiles * HTILE, "epilogue scratch must fit the hidden-state tiles");
constexpr size_t kLdsBytes = kHTiles * HTILE + NW * WTILE;

// minimum waves per SIMD: 2 keeps two 4-wave tiles resident per CU
#ifndef DCD_LMHEAD_MIN_BLOCKS
#define DCD_LMHEAD_MIN_BLOCKS 2
#endif

template <int DT>
__global__ __launch_bounds__(NT, DCD_LMHEAD_MIN_BLOCKS) void lmhead_kernel(Plan P, Inputs in) {
    extern __shared__ __align__(16) char lds[];
    char *hbuf = lds;                                       // [kHTiles][64][CB] hidden states
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);  // wave-uniform
    char *wbuf = lds + kHTiles * HTILE + wave * WTILE;      // this wave's [16*VB][CB] weights
    // epilogue scratch, aliasing the hidden-state tiles (used only between passes)
    float *red = reinterpret_cast<float *>(lds);                            // [NW][64]
    uint32_t *twords = reinterpret_cast<uint32_t *>(red + NW * ROWS);      // [64][words]
    int *tcnt = reinterpret_cast<int *>(twords + ROWS * kWordsPerTile);     // [64]

    // workgroup -> (vocabulary tile, row block); the row blocks of one tile are
    // dispatched back to back on the same XCD (workgroup id modulo 8) so the
    // tile's weights are re-read from that XCD's L2
    const int id = blockIdx.x, xcd = id % 8, local = id / 8;
    const int rblk = local % P.nrb;
    const int tile = (local / P.nrb) * 8 + xcd;
    if (tile >= P.ntiles) return;
    const int row0 = rblk * ROWS;
    const int lane = threadIdx.x % kWaveSize;
    const int n = lane % 16, g = lane / 16;
    const int tok0 = tile * TS + wave * (16 * VB);

    f32x4 acc[VB][RB];
    float z[VB][RB][4];
    float pmax[RB], psum[RB], qmax[RB], qsum[RB];
    uint32_t flags[RB];  // bit (vb*4 + j): tile-local candidate

    // ---- expert head
    const bool ragged = tok0 + 16 * VB > P.V;  // wave-uniform
    if (ragged)
        accumulate<DT, true>(ModelArgs{(const char *)in.hp, (const char *)in.wp, P.dp}, P.R, P.V,
                             row0, tok0, hbuf, wbuf, acc);
    else
        accumulate<DT, false>(ModelArgs{(const char *)in.hp, (const char *)in.wp, P.dp}, P.R, P.V,
                              row0, tok0, hbuf, wbuf, acc);
    tile_softmax(acc, in.bp, P.V, tok0, P.inv_T, red, z, pmax, psum);
    // Tile-local candidates: z_p within ln(theta) of the tile max.  Their expert
    // logits are parked in the sparse candidate array; the final decision waits
    // for the amateur pass, when the running row bound is (nearly) the row max.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = row0 + rb * 16 + n;
        const float thr = pmax[rb] + P.log_theta;
        uint32_t f = 0;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int t = tok0 + 16 * vb + 4 * g + j;
                if (t < P.V && z[vb][rb][j] >= thr && row < P.R) {
                    f |= 1u << (vb * 4 + j);
                    P.cand[(size_t)row * P.V + t].x = z[vb][rb][j];
                }
            }
        flags[rb] = f;
        // running lower bound on the row's expert max: one update per (row, tile)
        if (wave == 0 && g == 0 && row < P.R) atomicMax(&P.bound[row], ordered_key(pmax[rb]));
    }

    // ---- amateur head
    if (ragged)
        accumulate<DT, true>(ModelArgs{(const char *)in.hq, (const char *)in.wq, P.dq}, P.R, P.V,
                             row0, tok0, hbuf, wbuf, acc);
    else
        accumulate<DT, false>(ModelArgs{(const char *)in.hq, (const char *)in.wq, P.dq}, P.R, P.V,
                              row0, tok0, hbuf, wbuf, acc);
    // the hidden-state tiles are idle now: clear the candidate words and counts
    // (ordered before their use by the barriers inside tile_softmax)
    for (int i = threadIdx.x; i < ROWS * kWordsPerTile; i += NT) twords[i] = 0;
    if (threadIdx.x < ROWS) tcnt[threadIdx.x] = 0;
    tile_softmax(acc, in.bq, P.V, tok0, P.inv_T, red, z, qmax, qsum);
    // Final candidates: z_p >= max(tile max, running row bound) + ln(theta).  Both
    // bounds are <= the row max, so the plausibility mask (z_p >= row max +
    // ln theta) never loses a member.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int row = row0 + rb * 16 + n;
        const uint32_t f = flags[rb];
        if (f == 0) continue;
        const float b = fmaxf(pmax[rb], key_value(__atomic_load_n(&P.bound[row], __ATOMIC_RELAXED)));
        const float thr = b + P.log_theta;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) {
            uint32_t bits = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (f >> (vb * 4 + j) & 1u) {
                    const int t = tok0 + 16 * vb + 4 * g + j;
                    float2 *c = P.cand + (size_t)row * P.V + t;
                    if (c->x >= thr) {
                        c->y = z[vb][rb][j];
                        bits |= 1u << (t % 32);
                    }
                }
            if (bits) {
                const int word = (16 * VB * wave + 16 * vb) / 32;
                atomicOr(&twords[(rb * 16 + n) * kWordsPerTile + word], bits);
                atomicAdd(&tcnt[rb * 16 + n], __popc(bits));
            }
        }
    }
    __syncthreads();
    // per (row, tile): the candidate count, the bitmap words where it is nonzero,
    // and the softmax partials of both models
    for (int i = threadIdx.x; i < ROWS * kWordsPerTile; i += NT) {
        const int r = i / kWordsPerTile, row = row0 + r;
        if (row < P.R && tcnt[r] > 0)
            P.bits[(size_t)row * P.wstride + tile * kWordsPerTile + i % kWordsPerTile] = twords[i];
    }
    if (wave == 0 && g == 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int row = row0 + rb * 16 + n;
            if (row >= P.R) continue;
            P.partials[(size_t)row * P.ntiles + tile] = float4{pmax[rb], psum[rb], qmax[rb], qsum[rb]};
            P.tcount[(size_t)row * P.ntiles + tile] = tcnt[rb * 16 + n];
        }
    }
}

// Row bounds start at -inf for every call.
__global__ void init_bound_kernel(int *bound, int R) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r < R) bound[r] = ordered_key(-INFINITY);
}

}  // namespace

hipError_t launch_lmhead(const Plan &p, const Inputs &in, hipStream_t st) {
    // the tile needs more than 64 KB of LDS (gfx950 has 160 KB per CU)
    static const hipError_t attr = [] {
        hipError_t e = hipFuncSetAttribute((const void *)lmhead_kernel<kBF16>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)lmhead_kernel<kF32>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
        return e;
    }();
    if (attr != hipSuccess) return attr;
    const int groups = ((p.ntiles + 7) / 8) * 8 * p.nrb;
    hipLaunchKernelGGL(init_bound_kernel, dim3((p.R + 255) / 256), dim3(256), 0, st, p.bound, p.R);
    if (p.dtype == kBF16)
        hipLaunchKernelGGL(lmhead_kernel<kBF16>, dim3(groups), dim3(NT), kLdsBytes, st, p, in);
    else
        hipLaunchKernelGGL(lmhead_kernel<kF32>, dim3(groups), dim3(NT), kLdsBytes, st, p, in);
    return hipGetLastError();
}

}  // namespace dcd
