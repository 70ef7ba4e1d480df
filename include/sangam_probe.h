/*
 * sangam_probe.h - measured ceilings of the two resources the attention call
 * is bound by on AMD Instinct MI355X (gfx950): HBM read bandwidth (block
 * decodes, whose K/V stream is read once) and bf16 matrix-core throughput
 * (whole prefills, Sec. 2.1 and Sec. 3.2 of the Sangam paper: a prefill is
 * compute-bound and cannot be chunked). The benchmark reports the attention
 * kernels' rates against these measured ceilings beside the spec-sheet peaks
 * (8 TB/s, 2.5 PFLOP/s dense bf16), which the chip does not reach under load.
 *
 * Both calls only enqueue one kernel on `stream` (a hipStream_t, NULL for
 * the default stream); the caller times it (e.g. with events) and owns every
 * buffer. Errors: a sangam_status from sangam_attn.h (SANGAM_ERR_INVALID_ARG
 * for a NULL or misaligned buffer or a bad size, SANGAM_ERR_HIP when the
 * launch fails); sangam_last_error() gives the message.
 */
#ifndef SANGAM_PROBE_H
#define SANGAM_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include "sangam_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Streaming read: `grid` work-groups of 256 threads read the `bytes` bytes
 * at `src` (device memory, 16-byte aligned, bytes a multiple of 16) once,
 * in 16-byte vector loads at a grid-wide stride, and each work-group writes
 * one uint32 (an xor of what it read) to sink[blockIdx] so that the reads
 * stay. sink holds `grid` entries. Bytes moved = bytes (+ 4 grid written).
 */
sangam_status sangam_probe_hbm_read(const void *src, size_t bytes, uint32_t *sink, int32_t grid,
                                    void *stream);

/*
 * Matrix-core throughput: `grid` work-groups of 256 threads (four waves);
 * each wave runs `iters` rounds of 8 independent v_mfma_f32_32x32x16_bf16
 * on register operands (no memory traffic in the loop) and writes one float
 * per work-group to sink[blockIdx] so that the work stays. Flops =
 * grid * 4 * iters * 8 * 32768.
 */
sangam_status sangam_probe_mfma_bf16(float *sink, int32_t grid, int32_t iters, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SANGAM_PROBE_H */
