/*
 * logra_peaks.h -- measured ceilings of the GPU the LoGra library runs on
 * (a separate library, libpaper_logra_peaks.so; not part of the hot path).
 *
 * The roofline fractions of the library's kernels are quoted against the
 * published MI355X peaks (HBM 8 TB/s, dense bf16 MFMA 2.5 PFLOP/s).  These
 * two kernels measure what the chip sustains under the same kind of load, so
 * that a fraction can also be read against a measured ceiling:
 *
 * logra_peak_mfma_bf16: every wave issues `iters` rounds of four independent
 *   32x32x16 bf16 MFMAs (fp32 accumulation), 4 x 32,768 flops per round, on a
 *   grid of `groups` workgroups of 256 threads; the caller times the launch.
 *   cycles_out (device, 2 x int64, may be NULL) receives, for workgroup 0,
 *   the core-clock cycles and the constant-rate wall-clock ticks between its
 *   first and last MFMA round (hipDeviceAttributeWallClockRate gives the
 *   wall-clock rate in kHz), hence the clock the MFMA loop ran at.
 *   sink (device, `groups` floats) receives a checksum per workgroup.
 * logra_peak_mfma_bf16_data: the same loop (and the same cycles_out and sink)
 *   with operands that change from one MFMA to the next: ops (device,
 *   16-byte aligned, 1 MiB = 65,536 fragments of eight bf16 values, filled by
 *   the caller, e.g. with random normal values) gives each lane 16 fragments,
 *   taken as a register-tiled GEMM takes them: one A fragment for four MFMAs
 *   in a row, a different B fragment for each.  The multiplier switching, and
 *   so the power drawn, is then that of a GEMM on real data rather than of
 *   one constant operand pair.  iters must be a multiple of 8.
 * logra_peak_hbm_read: streams `bytes` (a multiple of 1,024; buf 1,024-byte
 *   aligned) from device memory on `groups` workgroups of 256 threads, in one
 *   of three ways: mode 0, grid-stride 128-bit loads, four in flight per
 *   thread; mode 1, a contiguous range per workgroup, eight non-temporal
 *   128-bit loads in flight per thread; mode 2, a contiguous range per wave
 *   copied into LDS by asynchronous 1 KB global-to-LDS copies, eight in
 *   flight (the way the projection streams).  sink (device, `groups` floats)
 *   receives a checksum.
 *
 * All three are asynchronous on `stream` and return a logra status code
 * (0 = OK, -1 = invalid argument, -3 = HIP error).
 */
#ifndef LOGRA_PEAKS_H
#define LOGRA_PEAKS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int logra_peak_mfma_bf16(int groups, int64_t iters, float *sink, int64_t *cycles_out, void *stream);
int logra_peak_mfma_bf16_data(int groups, int64_t iters, const void *ops, float *sink, int64_t *cycles_out,
                              void *stream);
int logra_peak_hbm_read(const void *buf, size_t bytes, int groups, int mode, float *sink, void *stream);
/* The constant rate of the wall clock read by logra_peak_mfma_bf16, in kHz, of the current device. */
int logra_peak_wall_clock_khz(int *khz);

#ifdef __cplusplus
}
#endif
#endif /* LOGRA_PEAKS_H */
