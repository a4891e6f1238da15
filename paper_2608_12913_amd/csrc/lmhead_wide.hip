// LM-head projection for many rows (the compute-bound regime), with the same
// epilogues as the streaming kernel (Alg. 1 "parallel model evaluation", the
// per-tile pieces of Eq. (1); with the plausibility mask of Sec. 2.1 or, at
// theta = 0, the untruncated target).
//
// With thousands of rows (many sequences verified together) the projection is a
// dense GEMM far above the MFMA ridge, so the tile is shaped for reuse rather
// than for streaming: a workgroup owns 256 tokens x 256 rows and its 4 waves form
// a 2 x 2 grid of 128 x 128 blocks (64 v_mfma_f32_16x16x32_bf16 blocks, 256 fp32
// accumulators per lane).  K is walked in 128-byte chunks of every row; a chunk's
// 256 weight rows and 256 hidden-state rows are loaded straight into one of two
// XOR-swizzled LDS stages (global_load_lds) while the other stage is multiplied,
// so the waves spend no instructions on staging; one barrier per chunk.  The 8
// row tiles of a vocabulary tile are dispatched together on one XCD, so its
// weights come from HBM once and from that XCD's L2 for the others.
//
// Epilogue: as in the streaming kernel -- per (row, tile) the max and sum of exp of
// both models, tile-local candidates (z_p within ln(theta) of the tile max)
// pruned against the running row bound.  It works one 16-row block at a time and
// recomputes logits from the accumulators; the block's logits also go to an LDS
// buffer so that a lane can fetch the one of a given token.  Untruncated target:
// per (row, tile) the statistics of y = (1+s) z_p - s z_q instead of candidates
// (wide_tile_full).
#include "dcd_internal.h"

namespace dcd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;               // threads per workgroup (4 waves)
constexpr int TT = kTileTokens;       // tokens per tile (the partials' tile)
constexpr int TR = kWideRows;         // rows per workgroup
constexpr int CB = 128;               // bytes of every row per K-chunk
constexpr int LPR = CB / 16;          // lanes per row in a load instruction
constexpr int RPI = kWaveSize / LPR;  // rows per load instruction
constexpr int SLAB = TT / 4;          // rows of each operand one wave loads per chunk
constexpr int LOADS = SLAB / RPI;     // load instructions per operand, wave and chunk
constexpr int BV = 8, BR = 8;         // 16-blocks per wave: tokens, rows
constexpr int KS = CB / 64;           // MFMA k-steps per chunk
constexpr int OPB = TT * CB;          // bytes of one operand chunk in LDS
constexpr int WT = 16 * BV;           // tokens per wave (128)
constexpr int WR = 16 * BR;           // rows per wave (128)
constexpr int NV = 4 * BV;            // logits per lane and row block (32)
static_assert(TT == 256 && TR == 256 && NT == 4 * kWaveSize, "2 x 2 waves of 128 x 128");
static_assert(LPR == RPI && LOADS * RPI == SLAB, "a load instruction covers RPI whole rows");
static_assert(NV == 32, "one bit per logit of a row block in a 32-bit mask");

// LDS: two stages of [weights 256 x CB | hidden states 256 x CB] (two separate
// objects, so the compiler can tell the stage being multiplied from the one being
// filled and adds no wait for the loads into the latter); both biases of the tile
// and the parked candidate logits; the epilogue scratch reuses stage 0.
constexpr size_t kStageBytes = 2 * OPB;
constexpr int kStash = BR;  // one parked logit per lane and row block
constexpr int kMiscFloats = 2 * TT + 4 * kStash * kWaveSize;
// epilogue scratch: (max, sum) pairs of the two token halves, candidate words and
// counts, a row block's logits per wave
constexpr size_t kPairsBytes = 2 * TR * sizeof(float2);
constexpr size_t kWordsBytes = TR * kWordsPerTile * sizeof(uint32_t);
constexpr size_t kCountBytes = TR * sizeof(int);
constexpr size_t kZBytes = 4 * NV * kWaveSize * sizeof(float);
static_assert(kPairsBytes + kWordsBytes + kCountBytes + kZBytes <= kStageBytes,
              "epilogue scratch must fit stage 0");

typedef __attribute__((address_space(3))) void *lds_ptr;

// Waits until every load this wave issued has landed except the two most recent
// (the L2 prefetch of the chunk after next; loads complete in issue order).  The
// compiler does not track loads that write LDS directly.
__device__ __forceinline__ void wait_chunk() { __builtin_amdgcn_s_waitcnt(0x0F72); }  // vmcnt(2)

// Workgroup barrier for LDS data: the wave's LDS reads have returned (lgkmcnt)
// before it arrives.  Unlike __syncthreads() it does not wait for direct-to-LDS
// loads still in flight (each wave waits for its own with wait_chunk), so the next
// chunk stays in flight across it.  The empty asm statements keep the compiler
// from moving memory operations across.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// The wave's index, known to the compiler as uniform: the row bases computed from it
// then sit in scalar registers and every load takes the scalar-base form (a 32-bit
// lane offset), instead of a 64-bit address per lane and load instruction.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize); }

__device__ __forceinline__ void st_lds(char *p, u32x4 v) { *reinterpret_cast<u32x4 *>(p) = v; }
__device__ __forceinline__ u32x4 ld_lds(const char *p) { return *reinterpret_cast<const u32x4 *>(p); }

__device__ __forceinline__ float wave_max16_32(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float wave_sum16_32(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}

// Per-thread load addresses of one model: a wave loads its quarter (slab) of the
// tile's weight rows and of the workgroup's hidden-state rows.  Instruction q
// fills the 1 KB of slab rows RPI*q .. RPI*q+RPI-1 in LDS, lane l landing at byte
// 16 l: row RPI*q + l/LPR, slot l%LPR.  The lane reads the column that slot must
// hold in the XOR-swizzled layout, (l%LPR) ^ (row%LPR); address = wave-uniform row
// base + a 32-bit lane offset.  RAGGED (the tile reaches past the vocabulary or
// past row R): rows past the end are clamped to the last one (their results are
// discarded).
template <bool RAGGED>
struct Stream {
    const char *wbase, *hbase;
    uint32_t rowbytes;
    // RAGGED: the slab's first row may lie past the last valid row, so the base is
    // the first valid row of the slab (or the last valid row), `skip` the slab rows
    // before it and `last` the last valid row, both relative to the base (>= 0)
    int wskip, wlast, hskip, hlast;
    int nch, r, col16;

    __device__ __forceinline__ void init(const void *h, const void *w, int d, int R, int V, int row0,
                                         int tile0) {
        const int lane = threadIdx.x % kWaveSize, wave = wave_id();
        r = lane / LPR;
        col16 = (lane % LPR) ^ (r % LPR);  // the slot's column (slab rows start at multiples of LPR)
        rowbytes = (uint32_t)d * 2;
        nch = (int)((rowbytes + CB - 1) / CB);
        const int ws0 = tile0 + SLAB * wave, hs0 = row0 + SLAB * wave;  // slab first rows
        const int wb = min(ws0, V - 1), hb = min(hs0, R - 1);
        wbase = (const char *)w + (size_t)wb * rowbytes;
        hbase = (const char *)h + (size_t)hb * rowbytes;
        wskip = ws0 - wb;
        wlast = V - 1 - wb;
        hskip = hs0 - hb;
        hlast = R - 1 - hb;
    }

    // Requests chunk c into LDS stage `st`.  In the K tail a lane past the row end
    // re-reads the row's last 16 bytes (finite values); the hidden-state slots there
    // are zeroed after arrival (zero_tail).
    __device__ __forceinline__ void dma(int c, char *st) const {
        const int wave = wave_id();
        const uint32_t col = (uint32_t)c * CB + col16 * 16;
        const uint32_t kcol = col < rowbytes ? col : rowbytes - 16;
        char *wdst = st + SLAB * wave * CB, *hdst = st + OPB + SLAB * wave * CB;
#pragma unroll
        for (int q = 0; q < LOADS; ++q) {
            const char *src = RAGGED ? wbase + (uint32_t)(min(wskip + RPI * q + r, wlast) * rowbytes + kcol)
                                     : wbase + (size_t)q * RPI * rowbytes + (uint32_t)(r * rowbytes + kcol);
            __builtin_amdgcn_global_load_lds(src, (lds_ptr)(wdst + q * RPI * CB), 16, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < LOADS; ++q) {
            const char *src = RAGGED ? hbase + (uint32_t)(min(hskip + RPI * q + r, hlast) * rowbytes + kcol)
                                     : hbase + (size_t)q * RPI * rowbytes + (uint32_t)(r * rowbytes + kcol);
            __builtin_amdgcn_global_load_lds(src, (lds_ptr)(hdst + q * RPI * CB), 16, 0, 0);
        }
    }

    // Warms L2 with chunk c: one 4-byte load per row of the wave's slabs (a 128-byte
    // chunk of a row is one cache line), two instructions, written to the wave's
    // 512 bytes of `sink`, which nothing reads.  Past the last chunk it re-reads the
    // last one.
    __device__ __forceinline__ void prefetch(int c, char *sink) const {
        const int lane = threadIdx.x % kWaveSize, wave = wave_id();
        const uint32_t col = min((uint32_t)c * CB, rowbytes - 16);
        const char *ws = RAGGED ? wbase + (uint32_t)(min(wskip + lane, wlast) * rowbytes + col)
                                : wbase + (uint32_t)(lane * rowbytes + col);
        const char *hs = RAGGED ? hbase + (uint32_t)(min(hskip + lane, hlast) * rowbytes + col)
                                : hbase + (uint32_t)(lane * rowbytes + col);
        static_assert(SLAB == kWaveSize, "one slab row per lane");
        __builtin_amdgcn_global_load_lds(ws, (lds_ptr)(sink + wave * 512), 4, 0, 0);
        __builtin_amdgcn_global_load_lds(hs, (lds_ptr)(sink + wave * 512 + 256), 4, 0, 0);
    }

    // After chunk c (the last, when rows end inside it) has landed in `st`: the
    // wave's hidden-state slots past the row end become zero, so the re-read
    // weights there multiply zeros.
    __device__ __forceinline__ void zero_tail(int c, char *st) const {
        if ((uint32_t)(c + 1) * CB <= rowbytes) return;  // workgroup-uniform
        const int lane = threadIdx.x % kWaveSize, wave = wave_id();
        if ((uint32_t)c * CB + col16 * 16 < rowbytes) return;
        char *hdst = st + OPB + SLAB * wave * CB + lane * 16;
#pragma unroll
        for (int q = 0; q < LOADS; ++q) st_lds(hdst + q * RPI * CB, u32x4{0u, 0u, 0u, 0u});
    }
};

// The wave's 128 x 128 block over one staged chunk.  A = weights (tokens as M),
// B = hidden states (rows as N); lane l supplies row l%16 of a block and K columns
// 8*(l/16).. of the k-step.  All 16 fragments of a k-step are read first, into
// registers of their own: the MFMAs of one token block then never wait behind the
// reads of the next (with registers reused, each block's reads could only start
// once the previous block's MFMAs had taken their operands).
__device__ __forceinline__ void compute(const char *st, int wt, int wr, f32x4 (&acc)[BV][BR]) {
    const int lane = threadIdx.x % kWaveSize, n = lane % 16, g = lane / 16;
    const char *wb = st + (wt * WT + n) * CB, *hb = st + OPB + (wr * WR + n) * CB;
    // a runtime loop over the k-steps: unrolled, the allocator splits the 256
    // accumulators across register files and spills
#pragma unroll 1
    for (int s = 0; s < KS; ++s) {
        const int col = ((4 * s + g) ^ (n % LPR)) << 4;
        u32x4 afr[BV], bfr[BR];
#pragma unroll
        for (int rb = 0; rb < BR; ++rb) bfr[rb] = ld_lds(hb + 16 * rb * CB + col);
#pragma unroll
        for (int vb = 0; vb < BV; ++vb) afr[vb] = ld_lds(wb + 16 * vb * CB + col);
        __builtin_amdgcn_sched_barrier(0);  // keep every read ahead of the MFMAs
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
#pragma unroll
            for (int rb = 0; rb < BR; ++rb)
                acc[vb][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, afr[vb]),
                                                                      __builtin_bit_cast(bf16x8, bfr[rb]),
                                                                      acc[vb][rb], 0, 0, 0);
    }
}

// One pass over a model's K chunks: chunk c is multiplied from stage `first` (c
// even) or `second` (c odd) while chunk c+1 loads into the other and chunk c+2 is
// pulled into L2 (so that its own loads, one chunk later, hit L2: with only two
// stages the loads of one chunk must land within one chunk's MFMAs).  One barrier
// per chunk: before it every wave has waited for its own loads of chunk c (so the
// stage is complete) and finished multiplying chunk c-1 (so the other stage is
// free for chunk c+1).  The caller requested chunk 0 into `first` and prefetched
// chunk 1, the two last loads it issued before any other; no load into a stage is
// in flight on return and every wave is done with both stages.
template <bool RAGGED>
__device__ __forceinline__ void run_pass(const Stream<RAGGED> &st, char *first, char *second, char *sink,
                                         int wt, int wr, f32x4 (&acc)[BV][BR]) {
#pragma unroll
    for (int vb = 0; vb < BV; ++vb)
#pragma unroll
        for (int rb = 0; rb < BR; ++rb) acc[vb][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c = 0;;) {
        wait_chunk();
        st.zero_tail(c, first);
        lds_barrier();
        if (c + 1 < st.nch) st.dma(c + 1, second);  // workgroup-uniform
        st.prefetch(c + 2, sink);
        compute(first, wt, wr, acc);
        if (++c >= st.nch) break;
        wait_chunk();
        st.zero_tail(c, second);
        lds_barrier();
        if (c + 1 < st.nch) st.dma(c + 1, first);
        st.prefetch(c + 2, sink);
        compute(second, wt, wr, acc);
        if (++c >= st.nch) break;
    }
    lds_barrier();
}

// Logits of row block rb for this lane (token 16vb + 4g + j of the wave's half,
// row 16rb + n of its half), divided by T; -inf past the vocabulary.
template <bool RAGGED>
__device__ __forceinline__ void block_logits(const f32x4 (&acc)[BV][BR], int rb, const float *bias,
                                             float inv_T, int tok0, int V, float (&z)[BV][4]) {
    const int g = (threadIdx.x % kWaveSize) / 16;
#pragma unroll
    for (int vb = 0; vb < BV; ++vb) {
        const float4 bv = *reinterpret_cast<const float4 *>(bias + 16 * vb + 4 * g);
        const float bj[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            z[vb][j] = fmaf(acc[vb][rb][j], inv_T, bj[j]);
            if (RAGGED && tok0 + 16 * vb + 4 * g + j >= V) z[vb][j] = -INFINITY;
        }
    }
}

// Per row of the workgroup (this lane's 8 rows): the tile's max and sum of exp of
// one model, from the two token halves (one LDS exchange, merged in order).
template <bool RAGGED>
__device__ __forceinline__ void tile_softmax(const f32x4 (&acc)[BV][BR], const float *bias,
                                             float inv_T, int tok0, int V, int wt, int wr, float2 *pairs,
                                             float (&tmax)[BR], float (&tsum)[BR]) {
    constexpr float kLog2e = 1.4426950408889634f;
    const int lane = threadIdx.x % kWaveSize, n = lane % 16, g = lane / 16;
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        float z[BV][4];
        block_logits<RAGGED>(acc, rb, bias, inv_T, tok0, V, z);
        float m = -INFINITY;
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) m = fmaxf(m, z[vb][j]);
        m = wave_max16_32(m);
        const float ml = m * kLog2e;
        float s = 0.f;
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) s += __builtin_amdgcn_exp2f(fmaf(z[vb][j], kLog2e, -ml));
        if (m == -INFINITY) s = 0.f;
        s = wave_sum16_32(s);
        if (g == 0) pairs[wt * TR + wr * WR + rb * 16 + n] = float2{m, s};
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        const float2 a = pairs[wr * WR + rb * 16 + n], b = pairs[TR + wr * WR + rb * 16 + n];
        const float m = fmaxf(a.x, b.x);
        float s = 0.f;
        if (m != -INFINITY) {
            if (a.x != -INFINITY) s += a.y * __expf(a.x - m);
            if (b.x != -INFINITY) s += b.y * __expf(b.x - m);
        }
        tmax[rb] = m;
        tsum[rb] = s;
    }
    __syncthreads();  // the pairs are reused
}

template <bool RAGGED>
__device__ __forceinline__ void wide_tile(const Plan &P, const Inputs &in, int tile, int row0, char *s0,
                                          char *s1, float *misc, char *sink) {
    const int tid = threadIdx.x, lane = tid % kWaveSize;
    const int wave = wave_id();
    const int wt = wave & 1, wr = wave >> 1;
    const int n = lane % 16, g = lane / 16;
    const int tile0 = tile * TT;
    const int tok0 = tile0 + wt * WT;  // first token of the wave's half

    char *lds = s0;                                                   // epilogue scratch
    float *bias_p = misc;                                             // [TT]
    float *bias_q = bias_p + TT;                                      // [TT]
    float *stash = bias_q + TT + wave * kStash * kWaveSize;           // [BR][64]
    float2 *pairs = reinterpret_cast<float2 *>(lds);                  // [2][TR]
    uint32_t *twords = reinterpret_cast<uint32_t *>(lds + kPairsBytes);                 // [TR][words]
    int *tcnt = reinterpret_cast<int *>(lds + kPairsBytes + kWordsBytes);              // [TR]
    float *zbuf = reinterpret_cast<float *>(lds + kPairsBytes + kWordsBytes + kCountBytes) +
                  wave * NV * kWaveSize;  // [NV][64]: the lane's logits of one row block

    if (tid < TT) {
        const int t = tile0 + tid;
        bias_p[tid] = (t < P.V && in.bp) ? in.bp[t] * P.inv_T : 0.f;
        bias_q[tid] = (t < P.V && in.bq) ? in.bq[t] * P.inv_T : 0.f;
    }

    Stream<RAGGED> sp, sq;
    sp.init(in.hp, in.wp, P.dp, P.R, P.V, row0, tile0);
    sq.init(in.hq, in.wq, P.dq, P.R, P.V, row0, tile0);
    f32x4 acc[BV][BR];
    float pmax[BR], psum[BR], qmax[BR], qsum[BR];
    uint32_t flags[BR];  // bit vb*4 + j: tile-local candidate

    // ---- expert head (chunks from stage 0, 1, 0, ...); the amateur head's first
    // chunk then loads into stage 1 while the expert epilogue uses stage 0
    sp.dma(0, s0);
    sp.prefetch(1, sink);
    run_pass<RAGGED>(sp, s0, s1, sink, wt, wr, acc);
    sq.dma(0, s1);
    sq.prefetch(1, sink);
    const float *bias = bias_p + wt * WT;  // this wave's half of the tile (then bias_q's)
    tile_softmax<RAGGED>(acc, bias, P.inv_T, tok0, P.V, wt, wr, pairs, pmax, psum);
    // the row bounds of this call are cleared by workgroup 0 (long done by now)
    const bool pruning = await_call_state(P.ctl);
    // tile-local candidates; the lane's first of each row block waits in its LDS
    // slot, further ones (rare) are stored now from the row block's logit buffer
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        const int row = row0 + wr * WR + rb * 16 + n;
        const float thr = pmax[rb] + P.log_theta;
        float z[BV][4];
        block_logits<RAGGED>(acc, rb, bias, P.inv_T, tok0, P.V, z);
        uint32_t f = 0;
        float first = 0.f;
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool c = (!RAGGED || tok0 + 16 * vb + 4 * g + j < P.V) && z[vb][j] >= thr;
                first = (c && f == 0) ? z[vb][j] : first;
                f |= c ? 1u << (vb * 4 + j) : 0u;
            }
        f = row < P.R ? f : 0u;
        flags[rb] = f;
        stash[rb * kWaveSize + lane] = first;
        uint32_t rest = f & (f - 1);
        if (__builtin_amdgcn_ballot_w64(rest != 0)) {  // wave-uniform
#pragma unroll
            for (int vb = 0; vb < BV; ++vb)
#pragma unroll
                for (int j = 0; j < 4; ++j) zbuf[(vb * 4 + j) * kWaveSize + lane] = z[vb][j];
            while (rest) {
                const int bit = __builtin_ctz(rest);
                rest &= rest - 1;
                P.cand[(size_t)row * P.V + tok0 + 16 * (bit / 4) + 4 * g + bit % 4].x =
                    zbuf[bit * kWaveSize + lane];
            }
        }
        if (pruning && wt == 0 && g == 0 && row < P.R) atomicMax(&P.bound[row], bound_key(pmax[rb]));
    }

    // ---- amateur head (chunks from stage 1, 0, 1, ...: its second chunk loads into
    // stage 0 only after the barrier that follows every wave's expert epilogue)
    run_pass<RAGGED>(sq, s1, s0, sink, wt, wr, acc);
    float bnd[BR];
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        const int row = min(row0 + wr * WR + rb * 16 + n, P.R - 1);
        bnd[rb] = flags[rb] && pruning ? bound_value(__atomic_load_n(&P.bound[row], __ATOMIC_RELAXED))
                                       : -INFINITY;
    }
    bias = bias_q + wt * WT;
    for (int i = tid; i < TR * kWordsPerTile; i += NT) twords[i] = 0;
    for (int i = tid; i < TR; i += NT) tcnt[i] = 0;
    tile_softmax<RAGGED>(acc, bias, P.inv_T, tok0, P.V, wt, wr, pairs, qmax, qsum);
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        const int rloc = wr * WR + rb * 16 + n, row = row0 + rloc;
        // a tile whose expert max is below the row bound + ln(theta) holds no mask member
        const uint32_t f = pmax[rb] >= bnd[rb] + P.log_theta ? flags[rb] : 0u;
        if (!__builtin_amdgcn_ballot_w64(f != 0)) continue;  // wave-uniform skip
        float z[BV][4];
        block_logits<RAGGED>(acc, rb, bias, P.inv_T, tok0, P.V, z);
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) zbuf[(vb * 4 + j) * kWaveSize + lane] = z[vb][j];
        uint32_t rest = f;
        const uint32_t lowest = f & (0u - f);  // the candidate parked in LDS
        while (rest) {
            const int bit = __builtin_ctz(rest);
            rest &= rest - 1;
            const int t = tok0 + 16 * (bit / 4) + 4 * g + bit % 4;
            float2 *c = &P.cand[(size_t)row * P.V + t];
            const float zq = zbuf[bit * kWaveSize + lane];
            if ((1u << bit) == lowest)
                *c = float2{stash[rb * kWaveSize + lane], zq};
            else
                c->y = zq;
            atomicOr(&twords[rloc * kWordsPerTile + (t - tile0) / 32], 1u << (t % 32));
        }
        atomicAdd(&tcnt[rloc], __popc(f));
    }
    __syncthreads();
    // per (row, tile): the candidate count, the bitmap words where it is nonzero,
    // and the softmax partials of both models
    for (int i = tid; i < TR * kWordsPerTile; i += NT) {
        const int r = i / kWordsPerTile, row = row0 + r;
        if (row < P.R && tcnt[r] > 0)
            P.bits[(size_t)row * P.wstride + tile * kWordsPerTile + i % kWordsPerTile] = twords[i];
    }
    if (wt == 0 && g == 0) {
#pragma unroll
        for (int rb = 0; rb < BR; ++rb) {
            const int rloc = wr * WR + rb * 16 + n, row = row0 + rloc;
            if (row >= P.R) continue;
            P.partials[(size_t)row * P.ntiles + tile] = float4{pmax[rb], psum[rb], qmax[rb], qsum[rb]};
            P.tcount[(size_t)row * P.ntiles + tile] = tcnt[rloc];
        }
    }
}

// Untruncated target (no mask): the same two passes.  The expert epilogue leaves the
// lane's expert logits in the dense y rows (16 contiguous bytes per lane and token
// block); the amateur epilogue reads them back, forms y = (1+s) z_p - s z_q, keeps per
// (row, tile) the statistics of y (best and second-best y, its token, the sum of
// exp(y - best), z_p and z_q at the best token), the expert's own top-1 and the weight
// sum(exp(z_p - tile max) (z_p - z_q)) of D_KL(pi_p || pi_q), and overwrites the dense
// rows with y when they are wanted (sampled verification, proposals).  The two token
// halves of a row are merged in token order through LDS.
__device__ __forceinline__ YStat ystat_shfl_xor(const YStat &x, int m) {
    return YStat{__shfl_xor(x.y1, m), __shfl_xor(x.i1, m), __shfl_xor(x.y2, m), __shfl_xor(x.ys, m),
                 __shfl_xor(x.zp1, m), __shfl_xor(x.zq1, m), __shfl_xor(x.a, m), __shfl_xor(x.ip, m)};
}

template <bool RAGGED>
__device__ __forceinline__ void wide_tile_full(const Plan &P, const Inputs &in, int tile, int row0, char *s0,
                                               char *s1, float *misc, char *sink) {
    constexpr float kLog2e = 1.4426950408889634f;
    const int tid = threadIdx.x, lane = tid % kWaveSize;
    const int wave = wave_id();
    const int wt = wave & 1, wr = wave >> 1;
    const int n = lane % 16, g = lane / 16;
    const int tile0 = tile * TT;
    const int tok0 = tile0 + wt * WT;  // first token of the wave's half

    float *bias_p = misc;                                          // [TT]
    float *bias_q = bias_p + TT;                                   // [TT]
    float2 *pairs = reinterpret_cast<float2 *>(s0);                // [2][TR]
    YStat *ys = reinterpret_cast<YStat *>(s0 + kPairsBytes);       // [2][TR]: the two token halves
    static_assert(kPairsBytes + 2 * TR * sizeof(YStat) <= kStageBytes, "y statistics must fit stage 0");

    if (tid < TT) {
        const int t = tile0 + tid;
        bias_p[tid] = (t < P.V && in.bp) ? in.bp[t] * P.inv_T : 0.f;
        bias_q[tid] = (t < P.V && in.bq) ? in.bq[t] * P.inv_T : 0.f;
    }

    Stream<RAGGED> sp, sq;
    sp.init(in.hp, in.wp, P.dp, P.R, P.V, row0, tile0);
    sq.init(in.hq, in.wq, P.dq, P.R, P.V, row0, tile0);
    f32x4 acc[BV][BR];
    float pmax[BR], psum[BR], qmax[BR], qsum[BR];

    // ---- expert head
    sp.dma(0, s0);
    sp.prefetch(1, sink);
    run_pass<RAGGED>(sp, s0, s1, sink, wt, wr, acc);
    sq.dma(0, s1);
    sq.prefetch(1, sink);
    const float *bias = bias_p + wt * WT;
    tile_softmax<RAGGED>(acc, bias, P.inv_T, tok0, P.V, wt, wr, pairs, pmax, psum);
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        const int row = row0 + wr * WR + rb * 16 + n;
        if (row >= P.R) continue;
        float z[BV][4];
        block_logits<RAGGED>(acc, rb, bias, P.inv_T, tok0, P.V, z);
        float *dst = P.y_full + (size_t)row * P.zstride + tok0 + 4 * g;
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
            *reinterpret_cast<float4 *>(dst + 16 * vb) = float4{z[vb][0], z[vb][1], z[vb][2], z[vb][3]};
    }

    // ---- amateur head
    run_pass<RAGGED>(sq, s1, s0, sink, wt, wr, acc);
    bias = bias_q + wt * WT;
    tile_softmax<RAGGED>(acc, bias, P.inv_T, tok0, P.V, wt, wr, pairs, qmax, qsum);
    const float s1f = 1.f + P.s;
#pragma unroll
    for (int rb = 0; rb < BR; ++rb) {
        const int rloc = wr * WR + rb * 16 + n, row = row0 + rloc;
        float *yrow = P.y_full + (size_t)min(row, P.R - 1) * P.zstride + tok0 + 4 * g;
        float zq[BV][4], zp[BV][4];
        block_logits<RAGGED>(acc, rb, bias, P.inv_T, tok0, P.V, zq);
#pragma unroll
        for (int vb = 0; vb < BV; ++vb) {
            const float4 v = *reinterpret_cast<const float4 *>(yrow + 16 * vb);
            zp[vb][0] = v.x;
            zp[vb][1] = v.y;
            zp[vb][2] = v.z;
            zp[vb][3] = v.w;
        }
        // the lane's tokens in ascending order, so a strict comparison keeps the
        // lowest id on ties
        YStat st{-INFINITY, -1, -INFINITY, 0.f, 0.f, 0.f, 0.f, -1};
        float y[BV][4];
#pragma unroll
        for (int vb = 0; vb < BV; ++vb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int t = tok0 + 16 * vb + 4 * g + j;
                const bool ok = !RAGGED || t < P.V;
                const float p = zp[vb][j], q = zq[vb][j];
                y[vb][j] = ok ? s1f * p - P.s * q : -INFINITY;
                st.a += ok ? __builtin_amdgcn_exp2f((p - pmax[rb]) * kLog2e) * (p - q) : 0.f;
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
        if (P.store_y && row < P.R) {
#pragma unroll
            for (int vb = 0; vb < BV; ++vb)
                *reinterpret_cast<float4 *>(yrow + 16 * vb) = float4{y[vb][0], y[vb][1], y[vb][2], y[vb][3]};
        }
        if (st.i1 >= 0) {
            const float ml = st.y1 * kLog2e;
#pragma unroll
            for (int vb = 0; vb < BV; ++vb)
#pragma unroll
                for (int j = 0; j < 4; ++j) st.ys += __builtin_amdgcn_exp2f(fmaf(y[vb][j], kLog2e, -ml));
        }
        st = ystat_merge(st, ystat_shfl_xor(st, 16));
        st = ystat_merge(st, ystat_shfl_xor(st, 32));
        if (g == 0) ys[wt * TR + rloc] = st;
    }
    __syncthreads();
    // per (row, tile): the y statistics of the two halves merged in token order, and
    // the softmax partials of both models
    if (wt == 0 && g == 0) {
#pragma unroll
        for (int rb = 0; rb < BR; ++rb) {
            const int rloc = wr * WR + rb * 16 + n, row = row0 + rloc;
            if (row >= P.R) continue;
            const YStat st = ystat_merge(ys[rloc], ys[TR + rloc]);
            float4 *dst = P.ypart + ((size_t)row * P.ntiles + tile) * 2;
            dst[0] = float4{st.y1, st.ys, st.y2, st.a};
            dst[1] = float4{__int_as_float(st.i1), st.zp1, st.zq1, __int_as_float(st.ip)};
            P.partials[(size_t)row * P.ntiles + tile] = float4{pmax[rb], psum[rb], qmax[rb], qsum[rb]};
        }
    }
}

template <bool FULL>
__global__ __launch_bounds__(NT, 1) void lmhead_wide_kernel(Plan P, Inputs in) {
    __shared__ __align__(16) char stage0[kStageBytes];
    __shared__ __align__(16) char stage1[kStageBytes];
    __shared__ __align__(16) float misc[kMiscFloats];
    __shared__ __align__(16) char sink[4 * 512];  // L2 prefetches land here, unread
    // workgroup 0 clears this call's row bounds and sequence counters first
    if (blockIdx.x == 0) clear_call_state(P.ctl, P.bound, kBoundCopies * P.R, P.seqdone, 2 * P.B);
    // workgroup -> (vocabulary tile, row tile); the row tiles of one vocabulary tile
    // are dispatched back to back on the same XCD (workgroup id modulo 8), so the
    // tile's weights are read from HBM once and from that XCD's L2 otherwise
    const int nrt = (P.R + TR - 1) / TR;
    const int id = blockIdx.x, xcd = id % 8, local = id / 8;
    const int tile = (local / nrt) * 8 + xcd;
    if (tile >= P.ntiles) return;
    const int row0 = (local % nrt) * TR;
    const bool ragged = (tile + 1) * TT > P.V || row0 + TR > P.R;  // workgroup-uniform
    if constexpr (FULL) {
        if (ragged)
            wide_tile_full<true>(P, in, tile, row0, stage0, stage1, misc, sink);
        else
            wide_tile_full<false>(P, in, tile, row0, stage0, stage1, misc, sink);
    } else {
        if (ragged)
            wide_tile<true>(P, in, tile, row0, stage0, stage1, misc, sink);
        else
            wide_tile<false>(P, in, tile, row0, stage0, stage1, misc, sink);
    }
}

}  // namespace

bool use_wide_lmhead(const Plan &p) { return p.dtype == kBF16 && p.R >= kWideMinRows; }

hipError_t launch_lmhead_wide(const Plan &p, const Inputs &in, hipStream_t st) {
    const int nrt = (p.R + TR - 1) / TR;
    const int groups = ((p.ntiles + 7) / 8) * 8 * nrt;
    if (p.full)
        hipLaunchKernelGGL(lmhead_wide_kernel<true>, dim3(groups), dim3(NT), 0, st, p, in);
    else
        hipLaunchKernelGGL(lmhead_wide_kernel<false>, dim3(groups), dim3(NT), 0, st, p, in);
    return hipGetLastError();
}

}  // namespace dcd
