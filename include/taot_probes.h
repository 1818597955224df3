/* Peak probes for MI355X (gfx950): small kernels that measure the rates the
 * planner's kernels are bounded by, so that roofline fractions can be quoted
 * against measured as well as datasheet peaks.  Measurement helpers of the
 * benchmark (libtaot_probes.so), not part of the planner's interface.
 *
 * Every call enqueues one kernel on `stream` (a hipStream_t; 0 = the null
 * stream) and returns 0, 1 if the launch was rejected, 2 for an invalid
 * argument (nothing enqueued).  `out` is a caller-owned device buffer that
 * receives partial results so the measured work is not dead code: at least
 * `blocks` floats for taot_probe_hbm_read, `blocks` x 256 floats otherwise.
 * Timing is the caller's (events around the call on the same stream).
 */
#ifndef TAOT_PROBES_H
#define TAOT_PROBES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int taot_probe_status;

/* P1: reads `bytes` (a multiple of 16; `src` 16-byte aligned, device memory)
 * once with 16-byte non-temporal loads; `blocks` workgroups of 256 threads,
 * each streaming its own contiguous share (8 loads per thread in flight). */
taot_probe_status taot_probe_hbm_read(const void* src, size_t bytes, int32_t blocks, float* out, void* stream);

/* P2: `blocks` x 256 threads, each 64 x `iters` fp32 FMAs in 8 independent
 * chains (unpacked FMAs; packed fp32 is not used by this build). */
taot_probe_status taot_probe_fma(int32_t blocks, int32_t iters, float* out, void* stream);

/* P3: `blocks` x 256 threads, each 64 x `iters` v_exp_f32 in 8 independent
 * chains; with `with_fma` != 0 every exponential is joined by one FMA of an
 * independent chain. */
taot_probe_status taot_probe_exp(int32_t blocks, int32_t iters, int32_t with_fma, float* out, void* stream);

/* P4: `blocks` x 256 threads, each 8 x `iters` 16-byte LDS reads without bank
 * conflicts (one 32 KiB table per workgroup). */
taot_probe_status taot_probe_lds(int32_t blocks, int32_t iters, float* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* TAOT_PROBES_H */
