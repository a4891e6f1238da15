/*
 * dcd_probe.h -- measurement probes of libdcd (not part of the verification path).
 *
 * The verification step is bound by HBM bandwidth (tens of rows) or by the bf16
 * MFMA rate (thousands of rows).  These probes measure what the device actually
 * delivers for each of the two, so that a benchmark can report a kernel's
 * achieved rate against a measured ceiling as well as the vendor's figure.
 * Same conventions as dcd.h: device pointers, work enqueued on `hip_stream` (a
 * hipStream_t as void*, NULL = default stream), negative DCD_ERR_* codes for
 * invalid requests, nothing launched on error, no allocation.
 */
#ifndef DCD_PROBE_H
#define DCD_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Reads `bytes` of device memory at `buf` once, with 16-byte non-temporal loads:
 * every workgroup streams one contiguous slice, each wave instruction covers 1 KB
 * of consecutive bytes, 8 instructions in flight per wave.  `buf` must be 16-byte
 * aligned and `bytes` a positive multiple of 16 (else DCD_ERR_ALIGN /
 * DCD_ERR_SHAPE); `sink` (device, 4 bytes) is written only if the data XOR to a
 * fixed pattern, which keeps the loads from being removed.  Achieved read
 * bandwidth = bytes / elapsed time of the launch.
 */
int dcd_probe_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *hip_stream);

/*
 * Dense bf16 MFMA rate: `workgroups` workgroups of 4 waves, each wave issuing
 * `iters` rounds of 8 independent v_mfma_f32_16x16x32_bf16 (the instruction of
 * the many-row LM-head kernel) on register operands, with no memory traffic in
 * the loop.
 * Each MFMA is 16*16*32*2 = 16384 flop, so one launch performs
 * workgroups * 4 * iters * 8 * 16384 flop; *flops (host) receives that number.
 * `sink` (device, workgroups * 256 floats) receives the accumulators.
 * workgroups >= 1, iters >= 1, else DCD_ERR_SHAPE.
 */
int dcd_probe_mfma_bf16(int workgroups, int iters, float *sink, double *flops, void *hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* DCD_PROBE_H */
