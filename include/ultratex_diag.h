/*
 * ultratex_diag.h -- libutdiag.so: a measurement aid kept out of the product
 * library. It measures the matrix-core rate the board sustains under its power
 * limit, the practical ceiling against which the attention kernels' MFMA
 * rates are read (the published bf16 peak assumes 2.4 GHz on every CU).
 */
#ifndef ULTRATEX_DIAG_H
#define ULTRATEX_DIAG_H

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One launch of `grid` workgroups of 4 waves (two workgroups per CU fill the
 * chip at 2 * CU count) that issue only bf16 MFMAs, iters x 64 of them per
 * wave, on operands read once from `in`:
 *   shape 0: v_mfma_f32_32x32x16_bf16,
 *   shape 1: v_mfma_f32_16x16x32_bf16, two per 32x32x16, so equal FLOPs.
 * FLOPs per launch: grid * 4 * iters * 64 * 32768.
 *
 * in      device, bf16, grid * 256 * 128 elements (16 vectors of 8 per lane);
 *         random values give the power-limited rate, constants the unloaded one.
 * out     device, fp32 [grid * 256]: each lane's accumulator sum (keeps the
 *         work observable; with every operand 1.0 it is 64 * iters * 16 * 16
 *         for shape 0 and 128 * iters * 32 * 4 for shape 1).
 * clocks  device, uint64 [2]: s_memtime and s_memrealtime (100 MHz) deltas
 *         of the first wave, so clocks[0] / clocks[1] * 0.1 is its GHz.
 * Asynchronous on `stream`. Returns 0, -1 for a bad argument (nothing is
 * launched) or a HIP error code. */
int ut_diag_mfma_rate(int shape, int iters, int grid, const void* in, float* out,
                      unsigned long long* clocks, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ULTRATEX_DIAG_H */
