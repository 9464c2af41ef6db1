/*
 * stencil_probe.h -- HBM and LDS probes used to calibrate the stencil measurements.
 *
 * The stencil kernels are judged against the compulsory-traffic roofline (each input
 * element read once, each output element written once).  This probe measures what a
 * plain streaming copy achieves on the same device, so that the stencil figures can be
 * read against both the nominal HBM peak and an achievable ceiling, and so that hardware
 * byte counters can be scaled by what they read for a copy of known size.
 */
#ifndef MI355X_STENCIL_PROBE_H
#define MI355X_STENCIL_PROBE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * stencil_probe_copy -- copy `bytes` bytes from `src` to `dst` on `stream` with 16-byte
 * non-temporal vector loads and stores, one kernel launch of one vector per thread.
 *   src, dst : device pointers, 16-byte aligned, non-overlapping (caller-owned).
 *   bytes    : a multiple of 16, >= 0.
 * Asynchronous.  Returns 0 on success, 1 for invalid arguments (checked on the host
 * before any HIP call; also when `bytes` needs more than 2^31 - 1 workgroups of 4 KB), 2
 * if the launch failed.
 */
int stencil_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t stream);

/*
 * stencil_probe_triad -- dst[i] = a[i] * b[i] over `bytes` bytes of fp32 per array on
 * `stream`: two streams read and one written, each element once, with the access shape
 * of stencil_probe_copy.  It is the achievable ceiling for the two-read, one-write mix of
 * a stencil with an output-indexed coefficient field (the input and the field read, the
 * output written).
 *   a, b, dst : device pointers, 16-byte aligned, `dst` overlapping neither (caller-owned).
 *   bytes     : bytes of each array, a multiple of 16, >= 0.
 * Asynchronous.  Returns 0 on success, 1 for invalid arguments (checked on the host
 * before any HIP call), 2 if the launch failed.
 */
int stencil_probe_triad(const void *a, const void *b, void *dst, int64_t bytes,
                        hipStream_t stream);

/*
 * stencil_probe_lds -- an LDS access pattern, for the bank-conflict counters: `blocks`
 * workgroups of 256 threads (4 waves) each hold a 64 KiB LDS buffer; every lane reads
 * (write = 0, ds_read_b128) or writes (write = 1, ds_write_b128) 16 bytes at byte offset
 * lane_bytes[lane % 64] of it, 8 x `iters` times.  The eight accesses of an iteration add
 * 0, 4, ..., 28 KiB to the offset (modulo 64 KiB), which keeps each lane on its own banks,
 * so the counters of one launch (rocprofv3 --pmc SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT
 * SQ_LDS_IDX_ACTIVE) describe that one pattern.
 *   lane_bytes : host array of 64 byte offsets, each a multiple of 16 and at most 65520
 *                (copied into the kernel arguments; the caller keeps ownership).
 *   write      : 0 or 1.   iters, blocks : 1 .. 2^20.
 *   sink       : a device pointer to one float, never written in practice (it keeps the
 *                compiler from removing the reads).
 * Asynchronous.  Returns 0 on success, 1 for invalid arguments (checked on the host
 * before any HIP call), 2 if the launch failed.
 */
int stencil_probe_lds(const int32_t *lane_bytes, int32_t write, int32_t iters, int32_t blocks,
                      float *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MI355X_STENCIL_PROBE_H */
