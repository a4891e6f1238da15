// LM-head projection of both models with a fused softmax-partials and
// candidate epilogue (Alg. 1 "parallel model evaluation" followed by the
// per-tile pieces of Eq. (1) and the plausibility mask of Sec. 2.1).
//
// Tiling.  One workgroup = NW waves = one tile of kTileTokens vocabulary tokens x
// ROWS rows.  Each wave owns 16*VB consecutive tokens and accumulates
// z^T[tokens][ROWS rows] = W * H^T in 16x16 MFMA blocks
// (v_mfma_f32_16x16x32_bf16, or 4 x v_mfma_f32_16x16x4_f32 for fp32).  K is
// walked in chunks of CB bytes of every row, each tile from its own starting
// chunk (Stream::init); the expert head first, then the amateur head, through
// the same registers and LDS.
//
// Weight stream (the HBM-bound part).  A wave reads its rows with 128-bit loads
// (non-temporal when a tile has one row block, ld16_weights), RPI rows x CB
// contiguous bytes per instruction.  On MI355X this
// shape (long runs per row, every tile resident at once) streams HBM3E far
// faster than the MFMA A-fragment shape (16 rows x 64 bytes per instruction), so
// each chunk is transposed through a wave-private LDS tile into fragment order.
// Hidden states (the B operand, shared by all waves) are staged per chunk into
// one of two LDS tiles.  Both tiles are XOR-swizzled (16-byte column c of row m
// at slot c ^ (m mod LPR)) so fragment reads of 16 lanes hit distinct bank
// groups.  One batch of loads is in flight per wave; the amateur head's first
// batch is issued before the expert epilogue (64 rows), so the stream does not
// stop between the two heads.
//
// Epilogue.  Per (row, tile): the tile max and sum of exp of both models, and
// the plausibility candidates: tokens whose expert logit is within ln(theta)
// of the tile max.  A tile whose expert max is itself below a running lower
// bound on the row max (an atomic maximum over the tiles that have finished
// their expert pass) + ln(theta) cannot contain mask members and drops its
// candidates.  Both bounds are <= the row max, so the final mask
// {z_p >= row max + ln theta} only contains candidates.  Candidate logits go to
// a sparse [row][token] array, their positions to a bitmap, their number per
// (row, tile) to a count array.
#include "dcd_internal.h"

namespace dcd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Row shape of this translation unit (lmhead128.hip includes this file with 128):
//   64 rows:  4 waves of 64 tokens x 64 rows, 128-byte chunks (32 KB of weights in
//             flight per workgroup), two workgroups per CU;
//   128 rows: 4 waves of 64 tokens x 128 rows (128 accumulators per wave), 128-byte
//             chunks, two workgroups per CU, so that one workgroup's epilogues
//             overlap the other's stream.  Its registers are tight: the weight
//             fragments stay put while the hidden-state fragments stream past
//             them, and the expert pass's row statistics wait in LDS during the
//             amateur pass.
// Either way 64 KB of weights is in flight per CU, and each weight byte serves ROWS
// rows.
#ifndef DCD_STREAM_ROWS
#define DCD_STREAM_ROWS 64
#endif
#if DCD_STREAM_ROWS == 64
constexpr int NW = 4, VB = 4, CB = 128, kMinBlocks = 2;
#elif DCD_STREAM_ROWS == 128
constexpr int NW = 4, VB = 4, CB = 128, kMinBlocks = 2;
#else
#error "DCD_STREAM_ROWS must be 64 or 128"
#endif

constexpr int NT = NW * kWaveSize;        // threads per workgroup
constexpr int TS = kTileTokens;           // tokens per tile
constexpr int ROWS = DCD_STREAM_ROWS;     // rows per workgroup
constexpr int RB = ROWS / 16;             // 16-row blocks
constexpr int LPR = CB / 16;              // lanes per row in a weight load instruction
constexpr int RPI = kWaveSize / LPR;      // rows per weight load instruction
constexpr int WLOADS = 16 * VB / RPI;     // weight load instructions per wave and chunk
constexpr int KS = CB / 64;               // MFMA k-steps per chunk
constexpr int HLOADS = ROWS * CB / (NT * 16);  // 16-byte hidden-state loads per thread and chunk
constexpr int WTILE = VB * 16 * CB;       // bytes of one wave's weight chunk
constexpr int HTILE = ROWS * CB;          // bytes of one hidden-state chunk
constexpr int QX = LPR / RPI > 0 ? LPR / RPI : 1;  // distinct weight-row swizzles per lane
constexpr bool kParkStats = ROWS > 64;    // expert row statistics kept in LDS across the amateur pass
static_assert(HLOADS >= 1 && ROWS * CB == HLOADS * NT * 16, "hidden-state staging must tile");
static_assert(CB % 64 == 0 && WLOADS * RPI == 16 * VB && LPR % RPI == 0 || RPI % LPR == 0,
              "weight chunk must tile");
static_assert(TS == 16 * VB * NW && TS % 32 == 0 && TS <= NT, "tile = 16*VB tokens per wave");
static_assert((NT / LPR) % LPR == 0, "hidden-state rows of one thread share a swizzle");
static_assert(4 * VB <= 32, "a lane's candidate flags of a row block fit one word");

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
// Weight loads: non-temporal when a tile has one row block (the weights are read
// once), ordinary cached loads when several row blocks of a tile read the same
// weights (they run back to back on one XCD and share them through its L2).
template <bool STREAM>
__device__ __forceinline__ u32x4 ld16_weights(const char *p) {
    if constexpr (STREAM)
        return ld16_stream(p);
    else
        return *reinterpret_cast<const u32x4 *>(p);
}
__device__ __forceinline__ u32x4 ld16(const char *p) { return *reinterpret_cast<const u32x4 *>(p); }
__device__ __forceinline__ void st_lds(char *p, u32x4 v) { *reinterpret_cast<u32x4 *>(p) = v; }
__device__ __forceinline__ u32x4 ld_lds(const char *p) { return *reinterpret_cast<const u32x4 *>(p); }

// byte offset of 16-byte column c of row m inside a swizzled [rows][CB] LDS tile:
// consecutive rows rotate their columns, so 16 lanes reading the same column of 16
// rows touch distinct bank groups
__device__ __forceinline__ int swz(int m, int c) { return m * CB + ((c ^ (m % LPR)) << 4); }

// The loads of one K-chunk: this wave's weight rows and this thread's share of the
// 64 hidden-state rows.
struct Batch {
    u32x4 w[WLOADS];
    u32x4 h[HLOADS];
    bool hok;  // the hidden-state columns are inside the row (false only in the K tail)
};

// Per-thread load addresses of one model's weight and hidden-state streams.
// RAGGED: the tile reaches past the vocabulary; weight rows are clamped to the
// last row (their results are discarded).
template <bool RAGGED, bool STREAM>
struct Stream {
    const char *wbase, *hbase;
    uint32_t rowbytes, wlane;
    uint32_t woff[RAGGED ? WLOADS : 1];
    uint32_t hoff[HLOADS];
    int nch, rot, wc, hc;

    // Weight loads: lane (r, c) = (lane / LPR, lane % LPR) reads 16 bytes at column
    // c of row RPI*q + r of the wave's rows (RPI rows x CB contiguous bytes per
    // instruction); address = wave-uniform row base (scalar registers) + a 32-bit
    // lane offset.  Hidden-state loads: thread -> (row, 16-byte column) of the
    // 64 x CB chunk; rows past R re-read row R-1 (results discarded).
    //
    // Chunk order.  Tile `tile` walks K starting at chunk (7*tile mod nch) and
    // wraps around.  Started in step, every tile would request the same 128-byte
    // column of its rows at the same time; with the rows 2^k bytes apart those
    // requests fall on few HBM channels and banks, and a microbenchmark of this
    // load pattern streamed 10-20% slower than with rotated starts (which match a
    // contiguous read).  All waves and row blocks of a tile share the order (the
    // hidden-state chunk is shared in LDS, the weights through L2).
    __device__ __forceinline__ void init(const void *h, const void *w, int d, int esz, int R, int V,
                                         int row0, int tok0, int tile) {
        const int tid = threadIdx.x, lane = tid % kWaveSize;
        const int wr = lane / LPR;
        wc = lane % LPR;
        hc = tid % LPR;
        rowbytes = (uint32_t)d * esz;
        nch = (int)((rowbytes + CB - 1) / CB);
        rot = (int)((7u * (uint32_t)tile) % (uint32_t)nch);
        const int tbase = min(tok0, V - 1);
        wbase = (const char *)w + (size_t)tbase * rowbytes;
        wlane = (uint32_t)wr * rowbytes;
        if constexpr (RAGGED) {
#pragma unroll
            for (int q = 0; q < WLOADS; ++q)
                woff[q] = (uint32_t)(min(tok0 + RPI * q + wr, V - 1) - tbase) * rowbytes;
        }
        hbase = (const char *)h + (size_t)row0 * rowbytes;
        const int hr0 = tid / LPR;
#pragma unroll
        for (int p = 0; p < HLOADS; ++p)
            hoff[p] = (uint32_t)(min(row0 + hr0 + p * (NT / LPR), R - 1) - row0) * rowbytes;
    }

    // In the K tail (rowbytes not a multiple of CB) a weight lane past the row end
    // re-reads the row's last 16 bytes (finite values) and the hidden-state
    // columns there are zero, so those products vanish.  c counts chunks in the
    // tile's order; cr is the chunk's position in the row.
    __device__ __forceinline__ void issue(int c, Batch &b) const {
        const int cr = c + rot < nch ? c + rot : c + rot - nch;
        const uint32_t col = (uint32_t)cr * CB + wc * 16;
        const uint32_t wcol = col < rowbytes ? col : rowbytes - 16;
#pragma unroll
        for (int q = 0; q < WLOADS; ++q) {
            if constexpr (RAGGED)
                b.w[q] = ld16_weights<STREAM>(wbase + (woff[q] + wcol));
            else
                b.w[q] = ld16_weights<STREAM>(wbase + (size_t)q * RPI * rowbytes + (wlane + wcol));
        }
        const uint32_t hcol = (uint32_t)cr * CB + hc * 16;
        b.hok = hcol < rowbytes;
#pragma unroll
        for (int p = 0; p < HLOADS; ++p) b.h[p] = ld16(hbase + (hoff[p] + (b.hok ? hcol : 0u)));
    }
};

// Lane-dependent LDS addresses (the rest are immediates).
struct LdsAddr {
    int wst[QX];   // weight row RPI*k + wr, column wc (rows RPI*q + wr repeat every QX)
    int hst;       // hidden-state row hr0, column hc (rows hr0 + p*NT/LPR share it)
    int frag[KS];  // fragment column 4s+g of row n (rows 16vb+n and 16rb+n add constants)

    __device__ __forceinline__ void init() {
        const int tid = threadIdx.x, lane = tid % kWaveSize;
        const int wr = lane / LPR, wc = lane % LPR;
#pragma unroll
        for (int k = 0; k < QX; ++k) wst[k] = swz(RPI * k + wr, wc);
        hst = swz(tid / LPR, tid % LPR);
        const int n = lane % 16, g = lane / 16;
#pragma unroll
        for (int s = 0; s < KS; ++s) frag[s] = swz(n, 4 * s + g);
    }
};

// arrived batch -> LDS: hidden states into the shared tile `hb` (zero in the K
// tail), the wave's weights into its private transpose tile.  Nothing inspects
// loaded registers before this point, so no wait is forced on loads in flight.
__device__ __forceinline__ void stage(const Batch &b, char *hb, char *wbuf, const LdsAddr &a) {
#pragma unroll
    for (int p = 0; p < HLOADS; ++p)
        st_lds(hb + a.hst + p * (NT / LPR) * CB, b.hok ? b.h[p] : u32x4{0u, 0u, 0u, 0u});
#pragma unroll
    for (int q = 0; q < WLOADS; ++q) st_lds(wbuf + a.wst[q % QX] + (q / QX) * (QX * RPI) * CB, b.w[q]);
}

template <int DT>
__device__ __forceinline__ void compute(const char *hb, const char *wbuf, const LdsAddr &a,
                                        f32x4 (&acc)[VB][RB]) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        // one k-step at a time: hoisting every fragment read of the chunk would
        // cost KS times the fragment registers
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (RB > VB) {
            // more row blocks than token blocks: every fragment of the k-step is read
            // first (the MFMAs then wait only for the ones they use), weights first
            u32x4 wfr[VB], hfr[RB];
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) wfr[vb] = ld_lds(wbuf + a.frag[s] + 16 * vb * CB);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) hfr[rb] = ld_lds(hb + a.frag[s] + 16 * rb * CB);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int vb = 0; vb < VB; ++vb) acc[vb][rb] = mma<DT>(wfr[vb], hfr[rb], acc[vb][rb]);
            // keep that order: left free, the scheduler sinks each read next to its
            // first MFMA and the LDS latency is exposed between every few MFMAs
            __builtin_amdgcn_sched_group_barrier(0x100, VB + RB, 0);  // DS reads
            __builtin_amdgcn_sched_group_barrier(0x008, VB * RB * (DT == kBF16 ? 1 : 4), 0);  // MFMAs
        } else {
            u32x4 bfr[RB];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) bfr[rb] = ld_lds(hb + a.frag[s] + 16 * rb * CB);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) {
                const u32x4 x = ld_lds(wbuf + a.frag[s] + 16 * vb * CB);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = mma<DT>(x, bfr[rb], acc[vb][rb]);
            }
        }
    }
}

// One pass over a model's K chunks, one batch in flight.  Chunk c is staged (its
// registers are then free), chunk c+1 is issued, chunk c is computed.  The two
// hidden-state tiles alternate, so one barrier per chunk suffices: the tile
// chunk c+1 goes to was last read by chunk c-1, which every wave finished before
// passing chunk c's barrier; the weight tile is wave-private and protected by the
// wave's own program order.  Batch b holds chunk 0 on entry.  If `next` is given,
// its chunk 0 is issued into b after the last chunk was staged, so that stream
// starts before this pass's epilogue.  The scheduling barriers pin each prefetch
// ahead of the compute (left free, the scheduler may sink the loads, and the
// next stage would then wait for them too).
template <int DT, bool RAGGED, bool STREAM>
__device__ __forceinline__ void run_pass(const Stream<RAGGED, STREAM> &st, const Stream<RAGGED, STREAM> *next,
                                         Batch &b, char *hbuf, char *wbuf, const LdsAddr &a,
                                         f32x4 (&acc)[VB][RB]) {
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[vb][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    int c = 0;
    for (; c + 1 < st.nch; ++c) {
        char *hb = hbuf + (c & 1) * HTILE;
        stage(b, hb, wbuf, a);
        st.issue(c + 1, b);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        compute<DT>(hb, wbuf, a, acc);
    }
    char *hb = hbuf + (c & 1) * HTILE;
    stage(b, hb, wbuf, a);
    if (next) next->issue(0, b);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    compute<DT>(hb, wbuf, a, acc);
    __syncthreads();  // the LDS tiles are reused next
}

__device__ __forceinline__ float wave_max16_32(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float wave_sum16_32(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}

// Logits of this lane's 16*VB (token, row) values and, per row, the tile's max and
// sum of exp relative to it.  One LDS exchange of (wave max, wave sum) pairs,
// merged in wave order by one thread per row.
//   bias_lds        the tile's bias already divided by T (0 without a bias)
//   z[vb][rb][j]    logit (divided by T); -inf for tokens >= V (ragged tile only)
//   tmax[rb], tsum[rb]   of row 16rb + lane%16
//   keep            if given, (tmax, tsum) of row r are also left in keep[r]
template <bool RAGGED>
__device__ __forceinline__ void tile_softmax(const f32x4 (&acc)[VB][RB], const float *bias_lds,
                                             int V, int tok0, int wtok0, float inv_T, float2 *pairs,
                                             float (&z)[VB][RB][4], float (&tmax)[RB],
                                             float (&tsum)[RB], float2 *keep = nullptr) {
    constexpr float kLog2e = 1.4426950408889634f;
    const int lane = threadIdx.x % kWaveSize, wave = threadIdx.x / kWaveSize;
    const int n = lane % 16, g = lane / 16;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int o = 16 * vb + 4 * g + j;  // token offset inside the wave
            const float b = bias_lds[wtok0 + o];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                z[vb][rb][j] = fmaf(acc[vb][rb][j], inv_T, b);
                if (RAGGED && tok0 + o >= V) z[vb][rb][j] = -INFINITY;
            }
        }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float m = -INFINITY;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) m = fmaxf(m, z[vb][rb][j]);
        m = wave_max16_32(m);
        const float ml = m * kLog2e;
        float s = 0.f;
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) s += __builtin_amdgcn_exp2f(fmaf(z[vb][rb][j], kLog2e, -ml));
        if (m == -INFINITY) s = 0.f;  // nothing finite in this wave row
        s = wave_sum16_32(s);
        if (g == 0) pairs[wave * ROWS + rb * 16 + n] = float2{m, s};
    }
    __syncthreads();
    // one thread per row merges the waves' pairs in wave order and leaves the result
    // in wave 0's slot of the row (only that thread touches the row's slots)
    if (threadIdx.x < ROWS) {
        const int r = threadIdx.x;
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w) m = fmaxf(m, pairs[w * ROWS + r].x);
        float s = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const float2 pw = pairs[w * ROWS + r];
                if (pw.x != -INFINITY) s += pw.y * __expf(pw.x - m);
            }
        }
        pairs[r] = float2{m, s};
        if (keep) keep[r] = float2{m, s};
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const float2 t = pairs[rb * 16 + n];
        tmax[rb] = t.x;
        tsum[rb] = t.y;
    }
    __syncthreads();  // the pairs are reused
}

__device__ __forceinline__ YStat ystat_shfl_xor(const YStat &x, int m) {
    return YStat{__shfl_xor(x.y1, m), __shfl_xor(x.i1, m), __shfl_xor(x.y2, m), __shfl_xor(x.ys, m),
                 __shfl_xor(x.zp1, m), __shfl_xor(x.zq1, m), __shfl_xor(x.a, m), __shfl_xor(x.ip, m)};
}

constexpr int kHTiles = 2;  // hidden-state tiles in LDS
// epilogue scratch (row reductions, candidate words and counts) reuses the
// hidden-state tiles, which are idle between passes
constexpr size_t kEpilogueBytes = NW * ROWS * sizeof(float2) + ROWS * kWordsPerTile * sizeof(uint32_t) +
                                  ROWS * sizeof(int);
static_assert(kEpilogueBytes <= (size_t)kHTiles * HTILE, "epilogue scratch must fit the hidden-state tiles");
static_assert(NW * ROWS * sizeof(YStat) <= (size_t)kHTiles * HTILE, "y statistics must fit the hidden-state tiles");
// expert logit of a lane's first tile-local candidate of each row block, parked
// until the amateur epilogue decides whether the tile survives ([rb][lane] per wave)
constexpr int kStash = RB;
constexpr size_t kParkBytes = kParkStats ? ROWS * sizeof(float2) : 0;  // [ROWS] (pmax, psum)
constexpr size_t kLdsBytes = kHTiles * HTILE + NW * WTILE + 2 * TS * sizeof(float) +
                             NW * kStash * kWaveSize * sizeof(float) + kParkBytes;

template <int DT, bool RAGGED, bool FULL, bool STREAM>
__device__ __forceinline__ void tile_body(const Plan &P, const Inputs &in, int tile, int row0,
                                          char *lds) {
    constexpr int ESZ = DT == kBF16 ? 2 : 4;
    const int tid = threadIdx.x, lane = tid % kWaveSize;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWaveSize);  // wave-uniform
    const int n = lane % 16, g = lane / 16;
    const int wtok0 = wave * (16 * VB);  // wave's first token inside the tile
    const int tok0 = tile * TS + wtok0;

    char *hbuf = lds;                                   // [2][64][CB] hidden states
    char *wbuf = lds + kHTiles * HTILE + wave * WTILE;  // this wave's [16*VB][CB] weights
    float *bias_p = reinterpret_cast<float *>(lds + kHTiles * HTILE + NW * WTILE);  // [TS]
    float *bias_q = bias_p + TS;                                                     // [TS]
    float *stash = bias_q + TS + wave * kStash * kWaveSize;                          // [RB][64]
    float2 *park = reinterpret_cast<float2 *>(bias_q + TS + NW * kStash * kWaveSize);  // [ROWS]
    // epilogue scratch, aliasing the hidden-state tiles (used only between passes)
    float2 *pairs = reinterpret_cast<float2 *>(lds);                       // [NW][64]
    uint32_t *twords = reinterpret_cast<uint32_t *>(pairs + NW * ROWS);   // [64][words]
    int *tcnt = reinterpret_cast<int *>(twords + ROWS * kWordsPerTile);    // [64]

    // both models' bias for the tile divided by T (0 past the vocabulary or without a bias);
    // ordered before their use by the pass barriers
    if (tid < TS) {
        const int t = tile * TS + tid;
        bias_p[tid] = (t < P.V && in.bp) ? in.bp[t] * P.inv_T : 0.f;
        bias_q[tid] = (t < P.V && in.bq) ? in.bq[t] * P.inv_T : 0.f;
    }

    Stream<RAGGED, STREAM> sp, sq;
    sp.init(in.hp, in.wp, P.dp, ESZ, P.R, P.V, row0, tok0, tile);
    sq.init(in.hq, in.wq, P.dq, ESZ, P.R, P.V, row0, tok0, tile);
    LdsAddr a;
    a.init();

    f32x4 acc[VB][RB];
    float z[VB][RB][4];
    // untruncated target, 64 rows: the expert logits stay in registers across the
    // amateur pass (the 128-row shape has no room: it stores and reloads them)
    constexpr bool kKeepZp = !kParkStats;
    float zpk[kKeepZp ? VB : 1][RB][4];
    float pmax[RB], psum[RB], qmax[RB], qsum[RB];
    uint32_t flags[RB];  // bit (vb*4 + j): tile-local candidate
    bool pruning = false;  // the row bounds of this call are usable
    Batch b;

    // ---- expert head (the amateur stream starts before its epilogue)
    sp.issue(0, b);
    // (the 128-row shape issues the amateur stream's first batch only after the expert
    // epilogue: held across it, its registers push that epilogue into spills)
    run_pass<DT, RAGGED, STREAM>(sp, kParkStats ? nullptr : &sq, b, hbuf, wbuf, a, acc);
    // (masked) this call's row bounds are cleared by workgroup 0, long done by now:
    // the reads that confirm it travel during the softmax
    CallState cs{};
    if constexpr (!FULL) cs = start_call_state(P.ctl);
    __builtin_amdgcn_sched_barrier(0);
    tile_softmax<RAGGED>(acc, bias_p, P.V, tok0, wtok0, P.inv_T, pairs, z, pmax, psum,
                         kParkStats ? park : nullptr);
    if constexpr (FULL) {
        // untruncated target: 64 rows keep the expert logits in registers; 128 rows
        // store them to the dense array (16 contiguous bytes per lane and block) for
        // their amateur epilogue
        if constexpr (kKeepZp) {
#pragma unroll
            for (int vb = 0; vb < VB; ++vb)
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                    for (int j = 0; j < 4; ++j) zpk[vb][rb][j] = z[vb][rb][j];
        }
        if constexpr (!kKeepZp) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int row = row0 + rb * 16 + n;
                if (row >= P.R) continue;
#pragma unroll
                for (int vb = 0; vb < VB; ++vb)
                    *reinterpret_cast<float4 *>(P.zp_full + (size_t)row * P.zstride + tok0 + 16 * vb + 4 * g) =
                        float4{z[vb][rb][0], z[vb][rb][1], z[vb][rb][2], z[vb][rb][3]};
            }
        }
    } else {
        // tile-local candidates: z_p within ln(theta) of the tile max (bit vb*4+j of
        // flags[rb]), found without branches.  The lane's first candidate of each row
        // block waits in its LDS slot; most tiles are pruned at the end, and global
        // stores issued here would delay the amateur stream's first loads behind
        // them.  Further candidates of a row block (rare) are stored at once.
        pruning = finish_call_state(P.ctl, cs);
        bool over = false;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int row = row0 + rb * 16 + n;
            const float thr = pmax[rb] + P.log_theta;
            uint32_t f = 0;
            float first = 0.f;
#pragma unroll
            for (int vb = 0; vb < VB; ++vb)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int t = tok0 + 16 * vb + 4 * g + j;
                    const bool c = (!RAGGED || t < P.V) && z[vb][rb][j] >= thr;
                    first = (c && f == 0) ? z[vb][rb][j] : first;
                    f |= c ? 1u << (vb * 4 + j) : 0u;
                }
            f = row < P.R ? f : 0u;
            flags[rb] = f;
            stash[rb * kWaveSize + lane] = first;
            over |= (f & (f - 1)) != 0;
            // running lower bound on the row's expert max: one update per (row, tile)
            if (pruning && wave == 0 && g == 0 && row < P.R) raise_bound(P.bound, P.R, row, pmax[rb]);
        }
        if (__builtin_amdgcn_ballot_w64(over)) {  // wave-uniform: some lane has more than one
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int row = row0 + rb * 16 + n;
                uint32_t rest = flags[rb] & (flags[rb] - 1);  // all but the first
                while (rest) {
                    const int bit = __builtin_ctz(rest);
                    rest &= rest - 1;
                    float v = z[0][rb][0];
#pragma unroll
                    for (int i = 1; i < 4 * VB; ++i) v = bit == i ? z[i / 4][rb][i % 4] : v;
                    P.cand[(size_t)row * P.V + tok0 + 16 * (bit / 4) + 4 * g + bit % 4].x = v;
                }
            }
        }
    }

    // ---- amateur head
    if constexpr (kParkStats) sq.issue(0, b);
    run_pass<DT, RAGGED, STREAM>(sq, nullptr, b, hbuf, wbuf, a, acc);
    if constexpr (kParkStats) {  // the expert statistics back from LDS (written before the pass)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const float2 t = park[rb * 16 + n];
            pmax[rb] = t.x;
            psum[rb] = t.y;
        }
    }
    if constexpr (FULL) {
        tile_softmax<RAGGED>(acc, bias_q, P.V, tok0, wtok0, P.inv_T, pairs, z, qmax, qsum);
        // the lane's expert logits of row block rb: kept, or back from the dense array
        auto load_zp = [&](int rb, float (&d)[VB][4]) {
            if constexpr (kKeepZp) {
#pragma unroll
                for (int vb = 0; vb < VB; ++vb)
#pragma unroll
                    for (int j = 0; j < 4; ++j) d[vb][j] = zpk[vb % (kKeepZp ? VB : 1)][rb][j];
                return;
            }
            const int row = min(row0 + rb * 16 + n, P.R - 1);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) {
                const float4 v = *reinterpret_cast<const float4 *>(
                    P.zp_full + (size_t)row * P.zstride + tok0 + 16 * vb + 4 * g);
                d[vb][0] = v.x;
                d[vb][1] = v.y;
                d[vb][2] = v.z;
                d[vb][3] = v.w;
            }
        };
        // per row: statistics of y over the lane's tokens (ascending, so a strict
        // comparison keeps the lowest id on ties), merged over the wave's lanes of
        // that row and then over the waves in order
        constexpr float kLog2e = 1.4426950408889634f;
        const float s1 = 1.f + P.s;
        YStat *ys_lds = reinterpret_cast<YStat *>(lds);  // [NW][64], over the idle hidden-state tiles
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            YStat st{-INFINITY, -1, -INFINITY, 0.f, 0.f, 0.f, 0.f, -1};
            float y[VB][4], zp[VB][4];
            load_zp(rb, zp);
#pragma unroll
            for (int vb = 0; vb < VB; ++vb)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int t = tok0 + 16 * vb + 4 * g + j;
                    const bool ok = !RAGGED || t < P.V;
                    const float p = zp[vb][j], q = z[vb][rb][j];
                    y[vb][j] = ok ? s1 * p - P.s * q : -INFINITY;
                    st.a += ok ? __builtin_amdgcn_exp2f((p - pmax[rb]) * kLog2e) * (p - q) : 0.f;
                    // the expert's own top-1: the lowest token holding the tile max
                    st.ip = (ok && st.ip < 0 && p == pmax[rb]) ? t : st.ip;
                    if (ok && y[vb][j] > st.y1) {
                        st.y2 = st.y1;
                        st.y1 = y[vb][j];
                        st.i1 = t;
                        st.zp1 = p;
                        st.zq1 = q;
                    } else if (ok) {
                        st.y2 = fmaxf(st.y2, y[vb][j]);
                    }
                }
            // sampled calls and proposals read y densely later (the walk's passes, the
            // proposal rows): 16 contiguous bytes per lane and block
            if (P.store_y && row0 + rb * 16 + n < P.R) {
#pragma unroll
                for (int vb = 0; vb < VB; ++vb)
                    *reinterpret_cast<float4 *>(P.y_full + (size_t)(row0 + rb * 16 + n) * P.zstride + tok0 +
                                                16 * vb + 4 * g) = float4{y[vb][0], y[vb][1], y[vb][2], y[vb][3]};
            }
            if (st.i1 >= 0) {
                const float ml = st.y1 * kLog2e;
#pragma unroll
                for (int vb = 0; vb < VB; ++vb)
#pragma unroll
                    for (int j = 0; j < 4; ++j) st.ys += __builtin_amdgcn_exp2f(fmaf(y[vb][j], kLog2e, -ml));
            }
            st = ystat_merge(st, ystat_shfl_xor(st, 16));
            st = ystat_merge(st, ystat_shfl_xor(st, 32));
            if (g == 0) ys_lds[wave * ROWS + rb * 16 + n] = st;
        }
        __syncthreads();
        if (wave == 0 && g == 0) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int row = row0 + rb * 16 + n;
                YStat st = ys_lds[rb * 16 + n];
#pragma unroll
                for (int w = 1; w < NW; ++w) st = ystat_merge(st, ys_lds[w * ROWS + rb * 16 + n]);
                if (row >= P.R) continue;
                float4 *dst = P.ypart + ((size_t)row * P.ntiles + tile) * 2;
                dst[0] = float4{st.y1, st.ys, st.y2, st.a};
                dst[1] = float4{__int_as_float(st.i1), st.zp1, st.zq1, __int_as_float(st.ip)};
            }
        }
    } else {
        // the running bound of the lane's rows (read before the softmax, so the load
        // latency overlaps it); the hidden-state tiles are idle: clear the candidate
        // words and counts (ordered before their use by the barriers in tile_softmax)
        float bnd[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int row = min(row0 + rb * 16 + n, P.R - 1);
            bnd[rb] = flags[rb] && pruning ? read_bound(P.bound, P.R, row) : -INFINITY;
        }
        for (int i = tid; i < ROWS * kWordsPerTile; i += NT) twords[i] = 0;
        if (tid < ROWS) tcnt[tid] = 0;
        tile_softmax<RAGGED>(acc, bias_q, P.V, tok0, wtok0, P.inv_T, pairs, z, qmax, qsum);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int row = row0 + rb * 16 + n;
            // a tile whose expert max is below the row bound + ln(theta) holds no mask member
            const uint32_t f = pmax[rb] >= bnd[rb] + P.log_theta ? flags[rb] : 0u;
            if (!__builtin_amdgcn_ballot_w64(f != 0)) continue;  // wave-uniform skip
            const uint32_t lowest = f & (0u - f);  // the candidate parked in LDS
#pragma unroll
            for (int vb = 0; vb < VB; ++vb) {
                uint32_t bits = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t bit = 1u << (vb * 4 + j);
                    if (f & bit) {
                        const int t = tok0 + 16 * vb + 4 * g + j;
                        float2 *c = &P.cand[(size_t)row * P.V + t];
                        if (bit == lowest)
                            *c = float2{stash[rb * kWaveSize + lane], z[vb][rb][j]};
                        else
                            c->y = z[vb][rb][j];
                        bits |= 1u << (t % 32);
                    }
                }
                if (bits) {
                    const int word = (wtok0 + 16 * vb) / 32;
                    atomicOr(&twords[(rb * 16 + n) * kWordsPerTile + word], bits);
                    atomicAdd(&tcnt[rb * 16 + n], __popc(bits));
                }
            }
        }
        __syncthreads();
        // per (row, tile): the candidate count and the bitmap words where it is nonzero
        for (int i = tid; i < ROWS * kWordsPerTile; i += NT) {
            const int r = i / kWordsPerTile, row = row0 + r;
            if (row < P.R && tcnt[r] > 0)
                P.bits[(size_t)row * P.wstride + tile * kWordsPerTile + i % kWordsPerTile] = twords[i];
        }
        if (wave == 0 && g == 0) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const int row = row0 + rb * 16 + n;
                if (row < P.R) P.tcount[(size_t)row * P.ntiles + tile] = tcnt[rb * 16 + n];
            }
        }
    }
    // per (row, tile): the softmax partials of both models
    if (wave == 0 && g == 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int row = row0 + rb * 16 + n;
            if (row >= P.R) continue;
            P.partials[(size_t)row * P.ntiles + tile] = float4{pmax[rb], psum[rb], qmax[rb], qsum[rb]};
        }
    }
}

template <int DT, bool FULL, bool STREAM>
__global__ __launch_bounds__(NT, kMinBlocks) void lmhead_kernel(Plan P, Inputs in) {
    extern __shared__ __align__(16) char lds[];
    // workgroup 0 clears this call's row bounds and sequence counters first
    if (blockIdx.x == 0) clear_call_state(P.ctl, P.bound, kBoundCopies * P.R, P.seqdone, 2 * P.B);
    // workgroup -> (vocabulary tile, row block); the row blocks of one tile are
    // dispatched back to back on the same XCD (workgroup id modulo 8) so the
    // tile's weights are re-read from that XCD's L2
    const int id = blockIdx.x, xcd = id % 8, local = id / 8;
    const int rblk = local % P.nrb;
    const int tile = (local / P.nrb) * 8 + xcd;
    if (tile >= P.ntiles) return;
    const int row0 = rblk * ROWS;
    if ((tile + 1) * TS > P.V)  // workgroup-uniform: only the last tile is ragged
        tile_body<DT, true, FULL, STREAM>(P, in, tile, row0, lds);
    else
        tile_body<DT, false, FULL, STREAM>(P, in, tile, row0, lds);
}

#if DCD_STREAM_ROWS == 64
// The call count of a workspace advanced after an LM-head launch that no other
// kernel of the library follows (dcd_lmhead_partials).
__global__ void advance_call_kernel(uint32_t *ctl) { advance_call(ctl); }
#endif

template <int DT, bool FULL, bool STREAM>
hipError_t launch_variant(const Plan &p, const Inputs &in, hipStream_t st) {
    // the tile may need more than 64 KB of LDS (gfx950 has 160 KB per CU)
    static const hipError_t attr = hipFuncSetAttribute((const void *)lmhead_kernel<DT, FULL, STREAM>,
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
    if (attr != hipSuccess) return attr;
    const int groups = ((p.ntiles + 7) / 8) * 8 * p.nrb;
    hipLaunchKernelGGL((lmhead_kernel<DT, FULL, STREAM>), dim3(groups), dim3(NT), kLdsBytes, st, p, in);
    return hipGetLastError();
}

template <int DT, bool FULL>
hipError_t launch_dt_full(const Plan &p, const Inputs &in, hipStream_t st) {
    return p.nrb == 1 ? launch_variant<DT, FULL, true>(p, in, st) : launch_variant<DT, FULL, false>(p, in, st);
}

// the untruncated target (plaus_thresh = 0) has its own kernels: dense logits, no candidates
hipError_t launch_skinny(const Plan &p, const Inputs &in, hipStream_t st) {
    if (p.rows_blk != ROWS) return hipErrorInvalidValue;
    if (p.dtype == kBF16)
        return p.full ? launch_dt_full<kBF16, true>(p, in, st) : launch_dt_full<kBF16, false>(p, in, st);
    return p.full ? launch_dt_full<kF32, true>(p, in, st) : launch_dt_full<kF32, false>(p, in, st);
}

}  // namespace

#if DCD_STREAM_ROWS == 64
hipError_t launch_lmhead_rows64(const Plan &p, const Inputs &in, hipStream_t st) { return launch_skinny(p, in, st); }

hipError_t launch_lmhead(const Plan &p, const Inputs &in, hipStream_t st) {
    if (use_wide_lmhead(p)) return launch_lmhead_wide(p, in, st);
    return p.rows_blk == kStreamRowsLarge ? launch_lmhead_rows128(p, in, st) : launch_lmhead_rows64(p, in, st);
}

hipError_t launch_advance_call(const Plan &p, hipStream_t st) {
    hipLaunchKernelGGL(advance_call_kernel, dim3(1), dim3(1), 0, st, p.ctl);
    return hipGetLastError();
}
#else
hipError_t launch_lmhead_rows128(const Plan &p, const Inputs &in, hipStream_t st) { return launch_skinny(p, in, st); }
#endif

}  // namespace dcd
