// Internal declarations of libdcd (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dcd {

// LM-head tile geometry (gfx950: 64-lane waves, 16x16 MFMA blocks).
constexpr int kWaveSize = 64;
#ifndef DCD_TILE_WAVES
#define DCD_TILE_WAVES 4
#endif
#ifndef DCD_TILE_VBLOCKS
#define DCD_TILE_VBLOCKS 4
#endif
constexpr int kTileWaves = DCD_TILE_WAVES;           // waves per workgroup
constexpr int kTileVBlocks = DCD_TILE_VBLOCKS;       // 16-token blocks per wave
constexpr int kTileTokens = kTileWaves * kTileVBlocks * 16;   // tokens per workgroup
constexpr int kTileRBlocks = 4;                      // 16-row blocks per workgroup
constexpr int kTileRows = kTileRBlocks * 16;         // 64 rows per workgroup
constexpr int kWordsPerTile = kTileTokens / 32;      // candidate bit words per row and tile
constexpr int kRowInfo = 16;                         // floats of per-row results

// rowinfo slots (floats; the argmax is stored as an int bit pattern)
enum {
    RI_MAXP = 0, RI_LSEP, RI_LSEQ, RI_LOGZ, RI_TOP1, RI_MARGIN, RI_COUNT, RI_SIGNAL,
    RI_THRESH = 8, RI_ARGMAX = 9
};

enum ElemType { kF32 = 0, kBF16 = 1 };

// Everything a launch needs, resolved on the host.
struct Plan {
    int B, N, R, V, dp, dq, dtype;
    int ntiles;        // ceil(V / kTileTokens)
    int nrb;           // ceil(R / kTileRows)
    int wstride;       // candidate bit words per row (ntiles * kWordsPerTile)
    float log_theta;   // ln(plaus_thresh); -inf when the mask is off
    float s;           // cd_strength
    float inv_T;       // 1 / temperature (1 for greedy)
    // workspace carve-up
    float4 *partials;  // [R][ntiles]   (max_p, sumexp_p, max_q, sumexp_q) per vocabulary tile
    float2 *cand;      // [R][V]        (z_p, z_q) of candidate tokens (sparse)
    uint32_t *bits;    // [R][wstride]  candidate bitmap
    float *rowinfo;    // [R][kRowInfo]
    int *tcount;       // [R][ntiles]   candidates per (row, tile); bitmap words valid where > 0
    int *bound;        // [R]           running lower bound on max z_p (order-preserving int key)
    float4 *nodez;     // [R]           (z_p, z_q, candidate?) of node r's token under its parent row
};

struct Inputs {
    const void *hp, *hq, *wp, *wq;
    const float *bp, *bq;
    const int32_t *parents, *tokens;
};

struct Outputs {
    int32_t *accept_len, *accept_path, *next_token, *status, *row_argmax;
    float *row_stats, *node_stats;
};

struct SampleInputs {
    const float *draft_probs, *u_acc, *u_res;
};

size_t workspace_layout(Plan &p, char *base);  // fills the pointers when base != nullptr

hipError_t launch_lmhead(const Plan &p, const Inputs &in, hipStream_t st);
hipError_t launch_combine(const Plan &p, const Inputs &in, const Outputs &out, hipStream_t st);
hipError_t launch_sequences(const Plan &p, const Inputs &in, const Outputs &out,
                            const SampleInputs *smp, hipStream_t st);

}  // namespace dcd
