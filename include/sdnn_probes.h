/*
 * sdnn_probes.h -- measurement probes for MI355X (gfx950) that report the machine's
 * achievable rates next to its datasheet peaks.  They are not part of the sparse
 * method: they exist so that the sparse kernel's rates can be set against what the
 * same chip delivers on the two on-chip resources its inner loop uses (plain FP32
 * FMA issue and LDS reads of 1 KB rows).
 *
 * Both calls enqueue one kernel on `stream` (a hipStream_t as void*, NULL = default),
 * write one float per thread to `out` (device memory, caller-owned, at least
 * sdnn_probe_out_floats() floats) so that the compiler keeps the work, and return 0,
 * or a nonzero hipError_t on a launch error.  Timing is the caller's (events around
 * the call).  Work done per call:
 *   sdnn_probe_fma:      out_floats * iters * 16 FMAs (2 FLOP each), 8 independent
 *                        chains per thread, unpacked v_fma_f32.
 *   sdnn_probe_lds_read: 256 workgroups x 16 waves x iters x 8 ds_read_b128 of 1 KB
 *                        (one 1 KB row of a 128 KB LDS array per instruction, rows
 *                        chosen pseudo-randomly per wave, lane l reading bytes 16l..16l+15).
 */
#ifndef SDNN_PROBES_H_
#define SDNN_PROBES_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Floats `out` must hold for either probe. */
int64_t sdnn_probe_out_floats(void);
int32_t sdnn_probe_fma(int32_t iters, float* out, void* stream);
int32_t sdnn_probe_lds_read(int32_t iters, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SDNN_PROBES_H_ */
