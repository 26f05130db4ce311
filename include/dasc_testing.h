/*
 * dasc_testing.h -- explicit refresh-kernel selection, for tests and A/B comparisons.
 *
 * dasc_refresh (dasc.h) picks its kernel from the shape alone.  This entry point runs
 * the same bounded-suffix replay (Sec. 4.2, DASC-WR; the gated delta rule of Eq. 1) on
 * a kernel the caller names, so that two kernels can be checked against each other on
 * the same inputs.  It is not part of the serving path: every kernel it can select
 * computes the result dasc_refresh documents, up to rounding.
 */
#ifndef DASC_TESTING_H
#define DASC_TESTING_H

#include "dasc.h"

#ifdef __cplusplus
extern "C" {
#endif

#define DASC_REFRESH_KERNEL_AUTO       0  /* the kernel dasc_refresh runs for this shape     */
#define DASC_REFRESH_KERNEL_COLUMN     1  /* per-column fp32 kernel: one thread per value
                                             column, plain per-token recurrence, no gate
                                             floor (dk in {16, 32, 64, 128}, dv <= 256)     */
#define DASC_REFRESH_KERNEL_CHANNEL_WY 2  /* chunked WY kernel with channel-wise gates on
                                             bf16 MFMA, also for GDN heads (their scalar
                                             gate broadcast over channels); dk = dv = 128   */

/* dasc_refresh with the kernel chosen by `kernel` (one of DASC_REFRESH_KERNEL_*).
 * Arguments, layouts, ownership and errors are those of dasc_refresh; the workspace
 * needed is dasc_refresh_workspace_bytes for AUTO and 0 for the other two.
 * Errors: those of dasc_refresh; DASC_E_INVAL for an unknown `kernel`;
 * DASC_E_UNSUPPORTED when the named kernel is not built for the shape. */
int dasc_refresh_select(const dasc_shape *shape, int32_t layer, const int32_t *inv_row,
                        float *states, int64_t n_pool, const int32_t *slot,
                        const uint16_t *k, const uint16_t *v, const float *g, const float *beta,
                        int32_t n_req, int32_t W, int32_t init_mode,
                        void *workspace, size_t workspace_bytes, int32_t kernel,
                        dasc_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DASC_TESTING_H */
