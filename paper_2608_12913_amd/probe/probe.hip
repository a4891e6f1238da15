// Measurement probes (include/dcd_probe.h): a plain streaming read of device
// memory and a register-only bf16 MFMA loop.  They give the benchmark measured
// ceilings for the two bounds of the verification step; nothing else calls them.
#include "dcd.h"
#include "dcd_probe.h"

#include <hip/hip_runtime.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 8;  // 1 KB loads in flight per wave and round

// Workgroup g streams 16-byte words [g*per, min((g+1)*per, n)) in rounds of
// kThreads*kUnroll words: in each round a wave reads kUnroll consecutive 1 KB
// pieces (lane l: 16 bytes at 16*l of each piece); the words after the last whole
// round are read one per thread.
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4 *p, size_t n, size_t per,
                                                                uint32_t *sink) {
    constexpr size_t kRound = (size_t)kThreads * kUnroll;
    const size_t lo = (size_t)blockIdx.x * per, hi = lo + per < n ? lo + per : n;
    const size_t rounds = (hi - lo) / kRound;
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    uint32_t acc = 0;
    for (size_t r = 0; r < rounds; ++r) {
        const u32x4 *q = p + lo + r * kRound + (size_t)wave * 64 * kUnroll + lane;
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(q + 64 * u);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (size_t j = lo + rounds * kRound + threadIdx.x; j < hi; j += kThreads) {
        const u32x4 v = __builtin_nontemporal_load(p + j);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u) sink[0] = acc;
}

constexpr int kChains = 8;  // independent accumulators per wave

// Eight independent accumulation chains per wave on register operands.  The loop
// is written in assembly: compiled from the builtin, the register allocator copies
// accumulators between AGPRs every iteration and halves the measured rate.  Only
// the rate matters here; the accumulated values just keep the work alive.
__global__ __launch_bounds__(kThreads) void mfma_kernel(int iters, float *sink) {
    const int t = threadIdx.x;
    bf16x8 a, b;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        a[k] = (__bf16)(0.001f * (float)((t + k) % 7));
        b[k] = (__bf16)(0.002f * (float)((t * 3 + k) % 5));
    }
    f32x4 c0{}, c1{}, c2{}, c3{}, c4{}, c5{}, c6{}, c7{};
    for (int i = 0; i < iters; ++i) {
        asm volatile(
            "v_mfma_f32_16x16x32_bf16 %0, %8, %9, %0\n\t"
            "v_mfma_f32_16x16x32_bf16 %1, %8, %9, %1\n\t"
            "v_mfma_f32_16x16x32_bf16 %2, %8, %9, %2\n\t"
            "v_mfma_f32_16x16x32_bf16 %3, %8, %9, %3\n\t"
            "v_mfma_f32_16x16x32_bf16 %4, %8, %9, %4\n\t"
            "v_mfma_f32_16x16x32_bf16 %5, %8, %9, %5\n\t"
            "v_mfma_f32_16x16x32_bf16 %6, %8, %9, %6\n\t"
            "v_mfma_f32_16x16x32_bf16 %7, %8, %9, %7"
            : "+a"(c0), "+a"(c1), "+a"(c2), "+a"(c3), "+a"(c4), "+a"(c5), "+a"(c6), "+a"(c7)
            : "v"(a), "v"(b));
    }
    // let the last MFMAs retire before their results are read
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::);
    const f32x4 s = c0 + c1 + c2 + c3 + c4 + c5 + c6 + c7;
    sink[(size_t)blockIdx.x * kThreads + t] = s[0] + s[1] + s[2] + s[3];
}

}  // namespace

extern "C" int dcd_probe_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *hip_stream) {
    if (!buf || !sink) return DCD_ERR_NULL;
    if (bytes == 0 || bytes % 16) return DCD_ERR_SHAPE;
    if ((uintptr_t)buf % 16 || (uintptr_t)sink % 4) return DCD_ERR_ALIGN;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return DCD_ERR_HIP;
    const size_t n = bytes / 16;
    // 4 workgroups per CU, slices rounded up to whole rounds
    const size_t groups = (size_t)(cus > 0 ? cus : 256) * 4;
    constexpr size_t kRound = (size_t)kThreads * kUnroll;
    size_t per = (n + groups - 1) / groups;
    per = (per + kRound - 1) / kRound * kRound;
    const size_t used = (n + per - 1) / per;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)used), dim3(kThreads), 0, (hipStream_t)hip_stream,
                       (const u32x4 *)buf, n, per, sink);
    return hipGetLastError() == hipSuccess ? DCD_OK : DCD_ERR_HIP;
}

extern "C" int dcd_probe_mfma_bf16(int workgroups, int iters, float *sink, double *flops, void *hip_stream) {
    if (!sink || !flops) return DCD_ERR_NULL;
    if (workgroups < 1 || iters < 1) return DCD_ERR_SHAPE;
    if ((uintptr_t)sink % 4) return DCD_ERR_ALIGN;
    *flops = (double)workgroups * 4 * iters * kChains * 16.0 * 16.0 * 32.0 * 2.0;
    hipLaunchKernelGGL(mfma_kernel, dim3(workgroups), dim3(kThreads), 0, (hipStream_t)hip_stream, iters, sink);
    return hipGetLastError() == hipSuccess ? DCD_OK : DCD_ERR_HIP;
}
