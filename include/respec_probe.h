/* respec_probe.h -- measurement probes of librespec_verify.so (not part of the
 * verification step).  They measure what this MI355X reaches in practice, so
 * that the step's kernels can be reported against measured ceilings beside the
 * vendor peaks (HBM 8 TB/s, bf16 dense MFMA 2.5 PFLOP/s).
 *
 * Both only enqueue one kernel on `stream` (a hipStream_t as void*, NULL = the
 * null stream) and return 0, or 1 for bad arguments, 2 if the launch failed.
 * Pointers are caller-owned device memory. */
#ifndef RESPEC_PROBE_H
#define RESPEC_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` (a multiple of 4096 * workgroups, buffer 16-byte aligned) once:
 * `workgroups` workgroups of 256 threads (1..65536), each streaming its own
 * contiguous share in 4 KiB steps with `depth` (4, 8 or 16) steps in flight
 * (16-byte loads); workgroup g writes the XOR of what it read to sink[g]. */
int respec_probe_read(const void* buf, size_t bytes, int32_t workgroups, int32_t depth, uint32_t* sink,
                      void* stream);

/* Matrix-core loop: `workgroups` workgroups of 256 threads, each wave running
 * `iters` rounds of 8 independent bf16 MFMAs on register operands: shape 0 is
 * v_mfma_f32_16x16x32_bf16 (16384 flops each), shape 1 v_mfma_f32_32x32x16_bf16
 * (32768 flops each).  Thread t of workgroup g writes a sum of its accumulators
 * to sink[g * 256 + t] (float32). */
int respec_probe_mfma(int32_t workgroups, int32_t iters, int32_t shape, float* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RESPEC_PROBE_H */
