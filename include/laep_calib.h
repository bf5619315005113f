/*
 * laep_calib.h -- measurement kernels of the LAEP MoE library (gfx950).
 *
 * Not part of the MoE layer: these calls measure what the chip attains on the
 * resources the layer's kernels are bound by, so that achieved rates can be
 * read against attained as well as published peaks.
 * Conventions (device pointers, void* streams, return codes, no allocation,
 * asynchronous enqueue, laep_last_error) are those of laep_moe.h.
 */
#ifndef LAEP_CALIB_H
#define LAEP_CALIB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * laep_calib_copy -- dst[0, bytes) = src[0, bytes), 16 bytes per thread per
 * step, grid-stride over all compute units: the HBM rate a plain streaming
 * copy attains (2 * bytes moved).
 *   src, dst : device, 16-byte aligned, non-overlapping
 *   bytes    : multiple of 16
 * Errors: LAEP_ERR_INVALID_ARG (null or misaligned pointer, bytes % 16 != 0),
 *         LAEP_ERR_HIP.
 */
int laep_calib_copy(const void* src, void* dst, size_t bytes, void* stream);

/*
 * laep_calib_read -- bytes / block_bytes workgroups of 512 threads; each reads
 * its contiguous block of block_bytes (thread t its 16-byte chunks t, t + 512,
 * ..., all in flight at once) and writes the XOR of what it read to
 * out[workgroup * 512 + t].  With block_bytes = 32 rows of a router input,
 * one workgroup per CU streams the router's x exactly as the router's launch
 * does, without its other work: the router's feed bound.
 *   src : device, 16-byte aligned, bytes readable
 *   out : device float[(bytes / block_bytes) * 512]
 * Errors: LAEP_ERR_INVALID_ARG (null or misaligned pointer; block_bytes not a
 *         multiple of 8192 in [8192, 131072], or not dividing bytes),
 *         LAEP_ERR_HIP.
 */
int laep_calib_read(const void* src, size_t bytes, int block_bytes, float* out, void* stream);

/*
 * laep_calib_mfma -- n_workgroups workgroups of 8 waves; every wave issues
 * iters x 8 v_mfma_f32_32x32x16_bf16 on four independent accumulators
 * (32768 flops each), then writes one float per lane to out (so the work is
 * not removed).  Total flops = n_workgroups * 8 * iters * 8 * 32768: the bf16
 * matrix-core rate the chip attains at its sustained clock.
 *   out : device float[n_workgroups * 512]
 * Errors: LAEP_ERR_INVALID_ARG (null out, n_workgroups < 1, iters < 1),
 *         LAEP_ERR_HIP.
 */
int laep_calib_mfma(int n_workgroups, int iters, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LAEP_CALIB_H */
