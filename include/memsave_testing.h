/*
 * memsave_testing.h -- test hooks of libmemsave (not for production use).
 */
#ifndef MEMSAVE_TESTING_H
#define MEMSAVE_TESTING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Make the next `n` transient-workspace allocations fail with MS_E_NOMEM,
 * so tests can check that a failed backward launches nothing, keeps its
 * record unconsumed and leaves the ledger unchanged. */
void ms_testing_fail_next_workspace(int32_t n);

/* Number of records currently allocated (leak check). */
int64_t ms_testing_live_records(void);

/* The bf16 GEMM planner's decision for one contraction of a convolution (a
 * Linear layer is the 1x1 case with H = W = 1), without launching anything.
 * geom = {N, C, H, W, K, R, S, P, Q, stride_h, stride_w, pad_h, pad_w};
 * pass 0 forward, 1 input gradient, 2 weight gradient.  Fills out[10] =
 * {tile rows, tile columns, waves, LDS stages, k-groups, splits, input
 * gradient reads W in place (1) or through its transposed copy (0), columns
 * of the first launch of a column split (0: none), the second launch's tile
 * rows and columns}.  Returns 0, or -1 when the bf16 fast path does not take
 * the contraction (channel counts not multiples of 8).  The testing knobs
 * MEMSAVE_GEMM_TILE, MEMSAVE_GEMM_SPLITS, MEMSAVE_DGRAD and MEMSAVE_GEMM_TAIL
 * apply as they do to a launch. */
int32_t ms_testing_gemm_plan(int32_t pass, const int32_t geom[13], int32_t out[10]);

#ifdef __cplusplus
}
#endif

#endif /* MEMSAVE_TESTING_H */
