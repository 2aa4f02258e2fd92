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
 *     under sustained MFMA load sets the result, and that clock depends on the
 *     operand bits: the chip is power-limited, and operands whose bits toggle
 *     like real data draw more power per MFMA than a few repeated patterns);
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

/* Operand bits of the matrix-core loop. */
typedef enum {
  /* a = ((lane + e) & 7) / 1024, b = ((3 lane + e) & 7) / 1024 for element e
   * of a lane's eight: eight bit patterns in all, the same for every chain. */
  CW_CEILING_LOW_ENTROPY = 0,
  /* Every element of every chain's A and B is a bf16 with a random sign, a
   * random 7-bit mantissa and a magnitude in [2^-4, 4) (the bit statistics of
   * N(0,1) data), drawn from a 32-bit integer hash of its global lane and
   * index: h(x) = x ^ x>>16, * 0x7feb352d, ^ >>15, * 0x846ca68b, ^ >>16 (all
   * mod 2^32).  For chain c and element e of global lane g = 512 workgroup +
   * thread, A's bits come from ha = h(64 g + 8 c + e), B's from
   * h(ha ^ 0x9e3779b9); bits(u) = (u >> 31) << 15 | (123 + (u >> 8) % 6) << 7
   * | (u & 127). */
  CW_CEILING_RANDOM = 1,
  CW_CEILING_RANGE_MIN_ = -2147483647 - 1, /* int32-sized enum (ABI) */
  CW_CEILING_RANGE_MAX_ = 2147483647
} cw_ceiling_operands_t;

/* Matrix-core loop.  `workgroups` workgroups of eight wave64s, each wave
 * running `iters` rounds of four independent 32x32x16 bf16 MFMAs (4 x 32768
 * FLOPs per round), chain c accumulating A_c B_c every round.  Total FLOPs =
 * workgroups * 8 * iters * 131072.  A grid that the CUs hold at once (one or
 * two workgroups per CU) measures the matrix pipes; a larger one adds a tail.
 * `sink` (device, fp32 [workgroups * 8]) receives, per wave, the sum over
 * chains c = 0..3 of element (row c, column 0) of chain c's accumulator, so the
 * loop cannot be removed.  CW_ERR_NULL for a NULL sink; CW_ERR_UNSUPPORTED
 * unless 1 <= workgroups <= 65536, 1 <= iters <= 2^24 and `operands` is one of
 * the values above. */
cw_status_t cw_ceiling_mfma_bf16(int32_t workgroups, int32_t iters, cw_ceiling_operands_t operands,
                                 float* sink, hipStream_t stream);

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
