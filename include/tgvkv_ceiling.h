/*
 * tgvkv_ceiling.h -- measurement kernels of libtgvkv: the HBM and matrix-core
 * rates the chip delivers, measured in the same process as the eviction pass so
 * that each kernel's rate can be read against them as well as against the vendor
 * peaks.  They compute nothing of the method (its kernels are in tgvkv.h).
 *
 * Buffers are device memory owned by the caller; every call validates its
 * arguments on the host, returns 0 on success, -1 for an invalid argument, -2 for
 * a size beyond what one launch covers, -5 if the launch failed, and enqueues
 * its kernel asynchronously on `stream` (time it with events on that stream).
 */
#ifndef TGVKV_CEILING_H
#define TGVKV_CEILING_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` (a positive multiple of 16) from `src` (16-byte aligned) once, with
 * the 16-byte non-temporal loads of the key sweeps, compaction and decode: every
 * workgroup of 256 threads streams one contiguous 128 KiB chunk, 8 loads in flight
 * per lane.  `sink` (one uint32) is written only for one data pattern; it keeps the
 * loads from being optimised away. */
int32_t tgvkv_ceiling_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream);

/* The same stream as tgvkv_ceiling_read, each 16 bytes also stored to `dst` (a
 * non-temporal store): a device copy that reads and writes `bytes` each. */
int32_t tgvkv_ceiling_copy(const void* src, void* dst, int64_t bytes, hipStream_t stream);

/* `workgroups` workgroups of 4 waves, each wave issuing `iters` rounds of 8
 * independent v_mfma_f32_16x16x32_bf16 (dense bf16, fp32 accumulate).
 * out: float [workgroups * 256], one value per lane (keeps the work live). */
int32_t tgvkv_ceiling_mfma(int32_t workgroups, int32_t iters, float* out, hipStream_t stream);

/* Dense bf16 flops of one tgvkv_ceiling_mfma launch (0 for non-positive arguments). */
long long tgvkv_ceiling_mfma_flops(int32_t workgroups, int32_t iters);

#ifdef __cplusplus
}
#endif

#endif /* TGVKV_CEILING_H */
