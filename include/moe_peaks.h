/*
 * moe_peaks.h -- achievable-peak probes for the roofline denominators.
 *
 * The layer's performance is reported as a fraction of MI355X's published
 * peaks (dense bf16 2.5 PFLOP/s, dense fp8 5.0 PFLOP/s, HBM 8 TB/s).  These
 * probes measure what the device actually reaches, so a fraction can also be
 * read against the achievable ceiling:
 *
 *   moe_peak_mfma   every CU runs eight waves of MFMA-only work (four
 *                   independent accumulator chains per wave, register
 *                   operands, no memory traffic in the loop): bf16
 *                   v_mfma_f32_32x32x16_bf16 or fp8 v_mfma_f32_32x32x64_f8f6f4.
 *                   FLOPs per launch: moe_peak_mfma_flops_per_launch().
 *   moe_peak_read   a streaming read (non-temporal loads) of a buffer larger
 *                   than the caches: the ceiling for kernels that mostly read
 *                   (the expert GEMMs stream weights);
 *   moe_peak_copy   a streaming device copy; it moves 2 * bytes through HBM
 *                   (read and write), a lower ceiling than reads alone.
 *
 * and two per-CU probes of the paths the tiled expert GEMMs stage their
 * operands through (one workgroup of 16 waves per CU):
 *
 *   moe_peak_lds_copy  global -> LDS copies (global_load_lds_dwordx4, 1 KB per
 *                   instruction) issued by the first `waves` waves, one step
 *                   of copies kept in flight across the workgroup barrier;
 *                   from a region small enough to stay in L2, or from HBM;
 *   moe_peak_lds_read  ds_read_b128 in the GEMMs' swizzled fragment pattern,
 *                   sixteen reads in flight per wave.
 *
 * Same conventions as moe.h: device pointers owned by the caller, work
 * enqueued on `stream` and never synchronised, arguments checked on the
 * host before anything is enqueued.  They are measurement tools, not part
 * of the layer, and no layer entry point calls them.
 */
#ifndef MOE_PEAKS_H
#define MOE_PEAKS_H

#include "moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* FLOPs one moe_peak_mfma launch performs on this device (host, pure given
 * the current device's CU count): CUs * 8 waves * iters * 4 chains * 2*M*N*K
 * of the instruction (32x32x64 for fp8 = 1, 32x32x16 for bf16 = 0).  0 if
 * iters < 1. */
long long moe_peak_mfma_flops_per_launch(int fp8, int iters);

/* 4-byte elements the `sink` argument of moe_peak_mfma and moe_peak_read
 * must hold on this device (CUs * 8). */
int moe_peak_sink_elems(void);

/* fp8: 1 for e4m3 operands, 0 for bf16.  iters >= 1 rounds of the four chains
 * per wave.  sink: device, moe_peak_sink_elems() floats, written with one
 * sum per wave (values meaningless; they keep the loop alive).
 * Errors: MOE_ERR_NULL (sink), MOE_ERR_SHAPE (iters < 1 or fp8 not 0/1),
 * MOE_ERR_HIP (launch). */
moe_status moe_peak_mfma(int fp8, int iters, float* sink, hipStream_t stream);

/* Reads src[0..bytes) once.  src: device, 16-byte aligned; bytes a multiple
 * of 16 (0 is a no-op).  sink: device, moe_peak_sink_elems() words that the
 * caller zeroes first; each is XORed with a fold of the bytes one workgroup
 * read.  Errors: MOE_ERR_NULL, MOE_ERR_SHAPE (bytes % 16), MOE_ERR_ALIGN,
 * MOE_ERR_HIP. */
moe_status moe_peak_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream);

/* dst[0..bytes) = src[0..bytes).  src, dst: device, 16-byte aligned, not
 * overlapping; bytes a multiple of 16 (0 is a no-op).  Errors: MOE_ERR_NULL,
 * MOE_ERR_SHAPE (bytes % 16), MOE_ERR_ALIGN, MOE_ERR_HIP. */
moe_status moe_peak_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

/* Bytes one moe_peak_lds_copy launch moves on this device: CUs * waves *
 * copies * steps * 1024; 0 for arguments moe_peak_lds_copy rejects. */
long long moe_peak_lds_copy_bytes_per_launch(int waves, int copies, int steps);

/* Workgroup b (one per CU) copies from region b % 8 of src: src must hold
 * 8 * region_bytes readable bytes, 16-byte aligned; region_bytes a power of
 * two in [64 KiB, 256 MiB].  With round-robin dispatch the workgroups of one
 * XCD share a region, so 1 MiB stays in that XCD's L2 and 256 MiB streams
 * from HBM.  waves in [1, 16] issue copies, copies (4, 8 or 16) per wave per
 * step, steps >= 1.  Nothing is written outside the workgroup's LDS.
 * Errors: MOE_ERR_NULL, MOE_ERR_SHAPE, MOE_ERR_ALIGN, MOE_ERR_HIP. */
moe_status moe_peak_lds_copy(const void* src, size_t region_bytes, int waves, int copies, int steps,
                             hipStream_t stream);

/* Bytes one moe_peak_lds_read launch reads from LDS on this device: CUs *
 * waves * 64 lanes * 16 bytes * 16 reads * iters; 0 for rejected arguments. */
long long moe_peak_lds_read_bytes_per_launch(int waves, int iters);

/* waves in [1, 16] per CU, iters >= 1 rounds of sixteen reads per wave.
 * sink: device, at least moe_peak_sink_elems() words; word b is written by
 * workgroup b (a fold of the values read; meaningless).
 * Errors: MOE_ERR_NULL, MOE_ERR_SHAPE, MOE_ERR_HIP. */
moe_status moe_peak_lds_read(int waves, int iters, uint32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_PEAKS_H */
