/*
 * moeq_peaks -- measured roofline denominators for the MI355X (gfx950).
 *
 * Benchmark instrumentation, not part of the layer: two kernels whose rates
 * bound what the layer's kernels can reach on the machine they run on.
 *   - a plain streaming read of device memory with 16-byte coalesced loads:
 *     the practical ceiling of an HBM-bound kernel that only reads (the
 *     decode matrix-vector products stream their packed weights this way);
 *   - a loop of dense v_mfma_f32_32x32x16_f16 instructions on register
 *     operands with no memory traffic: the practical ceiling of the binary16
 *     matrix cores for the instruction the prefill grouped GEMMs issue.
 * The rates are computed by the caller from its own event timing of a launch:
 * bytes read per launch = n_bytes; flops per launch = moeq_peaks_mfma_flops().
 *
 * Conventions: return 0 on success, a HIP error code otherwise; launches are
 * asynchronous on `stream` (a hipStream_t as void*, NULL = default stream);
 * pointers are DEVICE memory of the current device.
 */
#ifndef MOEQ_PEAKS_H
#define MOEQ_PEAKS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads n_bytes of src (16-byte aligned, n_bytes a multiple of 16) with
 * non-temporal 16-byte loads, every byte once, and writes one 32-bit XOR of
 * what each workgroup read to sink[workgroup] so that the loads stay live.
 *   sink   DEVICE uint32 [moeq_peaks_read_workgroups(n_bytes)] */
int moeq_peaks_stream_read(const void* src, size_t n_bytes, uint32_t* sink, void* stream);
int moeq_peaks_read_workgroups(size_t n_bytes);

/* Runs `iters` rounds of 4 independent binary16 MFMA chains on every wave of
 * `workgroups` workgroups of 256 threads, then writes one float per thread
 * (sum of its accumulators) to sink so the work is not removed.
 *   sink   DEVICE float [workgroups * 256] */
int moeq_peaks_mfma(int workgroups, int iters, float* sink, void* stream);
/* Dense flops of one moeq_peaks_mfma launch: workgroups * 4 waves * iters *
 * 4 MFMAs * 2 * 32 * 32 * 16. */
double moeq_peaks_mfma_flops(int workgroups, int iters);

#ifdef __cplusplus
}
#endif

#endif /* MOEQ_PEAKS_H */
