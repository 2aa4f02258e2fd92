/*
 * cw_ceiling.h -- measured ceilings of the MI355X (gfx950) for the attention
 * kernels' two rooflines.
 *
 * The attention kernels are priced against published peaks (dense bf16 MFMA
 * 2516.6 TFLOP/s = 256 CU x 2.4 GHz x 4096 FLOP/clk; HBM3E 8 TB/s).  These
 * calls measure what the chip sustains on the same unit of work with nothing
 * else in the way, so that a kernel can also be placed against a measured
 * ceiling:
 *   - a matrix-core loop: every wave issues independent
 *     v_mfma_f32_32x32x16_bf16 chains and touches no memory (the shader clock
 *     under sustained MFMA load sets the result);
 *   - a streaming read and a streaming copy of a device buffer in 16-byte
 *     pieces by every lane, grid-stride, many loads in flight per lane.
 * They are not part of the attention path.
 *
 * Ownership and ordering as in cw.h: the caller owns every buffer; work is
 * enqueued on `stream` and the call returns before it finishes; time it with
 * events on the same stream.  Arguments are checked before anything is
 * enqueued; errors are cw_status_t codes (cw_last_error_message in cw.h).
 */
#ifndef CW_CEILING_H_
#define CW_CEILING_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "cw.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Matrix-core loop.  `workgroups` workgroups of eight wave64s, each wave
 * running `iters` rounds of four independent 32x32x16 bf16 MFMAs (4 x 32768
 * FLOPs per round).  Total FLOPs = workgroups * 8 * iters * 131072.  A grid
 * that the CUs hold at once (one or two workgroups per CU) measures the matrix
 * pipes; a larger one adds a tail.  `sink` (device, fp32 [workgroups * 8])
 * receives one accumulator element per wave so the loop cannot be removed.
 * CW_ERR_NULL for a NULL sink; CW_ERR_UNSUPPORTED unless 1 <= workgroups
 * <= 65536 and 1 <= iters <= 2^24. */
cw_status_t cw_ceiling_mfma_bf16(int32_t workgroups, int32_t iters, float* sink,
                                 hipStream_t stream);

/* Streaming read of `bytes` (a multiple of 16, > 0) from device buffer `src`
 * (16-byte aligned).  `sink` (device, uint32 [16384]) receives one XOR of
 * the data per workgroup (16384 workgroups of 256 lanes).  Bytes moved = `bytes`.
 * CW_ERR_NULL, CW_ERR_ALIGN (pointers or size not 16-byte multiples), or
 * CW_ERR_UNSUPPORTED for bytes == 0. */
cw_status_t cw_ceiling_stream_read(const void* src, size_t bytes, uint32_t* sink,
                                   hipStream_t stream);

/* Streaming copy of `bytes` (a multiple of 16, > 0) from `src` to `dst`
 * (device, 16-byte aligned, not overlapping).  Bytes moved = 2 * `bytes`.
 * Errors as cw_ceiling_stream_read. */
cw_status_t cw_ceiling_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif  // CW_CEILING_H_
