// The models' final RMS normalisation, applied to both models' rows before the LM
// heads when a call is given un-normalised hidden states (the step that ends each
// model's forward pass in the Llama family the paper uses):
//   y = g * [x / sqrt(mean(x^2) + eps)]
// with, for bf16, the normalised value [.] and the product rounded to bf16 (round
// to nearest even), as those models compute it; fp32 rows are not rounded.  One
// workgroup per (row, model): the sum of squares in fp32 (per-thread partials,
// then a fixed-order reduction), then the row is rewritten into the workspace copy
// the LM-head and finish kernels read.
#include "dcd_internal.h"

namespace dcd {
namespace {

constexpr int NT = 256;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
// float -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN)
__device__ __forceinline__ uint32_t to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float round_bf16(float f) { return __uint_as_float(to_bf16(f) << 16); }

template <int DT>
__global__ __launch_bounds__(NT) void rmsnorm_kernel(Plan P, Inputs in) {
    __shared__ float part[NT / kWaveSize];
    const int model = blockIdx.y, row = blockIdx.x, tid = threadIdx.x;
    const int d = model ? P.dq : P.dp;
    const size_t esz = DT == kBF16 ? 2 : 4;
    const u32x4 *x = reinterpret_cast<const u32x4 *>((const char *)(model ? in.hq : in.hp) + (size_t)row * d * esz);
    const u32x4 *g = reinterpret_cast<const u32x4 *>(model ? in.gq : in.gp);
    u32x4 *y = reinterpret_cast<u32x4 *>((char *)(model ? P.hn_q : P.hn_p) + (size_t)row * d * esz);
    const int nvec = d * (int)esz / 16;
    float ss = 0.f;
    for (int i = tid; i < nvec; i += NT) {
        const u32x4 v = x[i];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if constexpr (DT == kBF16) {
                const float a = bf16_lo(v[k]), b = bf16_hi(v[k]);
                ss = fmaf(a, a, ss);
                ss = fmaf(b, b, ss);
            } else {
                const float a = __uint_as_float(v[k]);
                ss = fmaf(a, a, ss);
            }
        }
    }
#pragma unroll
    for (int o = kWaveSize / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    if (tid % kWaveSize == 0) part[tid / kWaveSize] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < NT / kWaveSize; ++w) tot += part[w];
    const float r = 1.f / sqrtf(tot / (float)d + P.norm_eps);
    for (int i = tid; i < nvec; i += NT) {
        const u32x4 v = x[i], s = g[i];
        u32x4 o;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if constexpr (DT == kBF16) {
                const float lo = round_bf16(bf16_lo(s[k]) * round_bf16(bf16_lo(v[k]) * r));
                const float hi = round_bf16(bf16_hi(s[k]) * round_bf16(bf16_hi(v[k]) * r));
                o[k] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
            } else {
                o[k] = __float_as_uint(__uint_as_float(s[k]) * (__uint_as_float(v[k]) * r));
            }
        }
        y[i] = o;
    }
}

}  // namespace

hipError_t launch_rmsnorm(const Plan &p, const Inputs &in, hipStream_t st) {
    const dim3 grid(p.R, 2);
    if (p.dtype == kBF16)
        hipLaunchKernelGGL((rmsnorm_kernel<kBF16>), grid, dim3(NT), 0, st, p, in);
    else
        hipLaunchKernelGGL((rmsnorm_kernel<kF32>), grid, dim3(NT), 0, st, p, in);
    return hipGetLastError();
}

}  // namespace dcd
