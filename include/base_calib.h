/*
 * base_calib.h -- the log-energy predictor's fit from calibration
 * statistics (Sec. 3.4, eq. log_energy_predictor; App. A "Calibration
 * Details").  In its own library, libbase_calib.so (it links rocSOLVER);
 * the statistics come from base_calib_accumulate (base.h).
 */
#ifndef BASE_MI355X_BASE_CALIB_H
#define BASE_MI355X_BASE_CALIB_H

#include "base.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Fits pred_a and pred_b from the statistics `stats` (the layout described
 * at base_calib_accumulate) of L->E experts of hidden size L->d.  Per
 * expert u with n_u > 0:
 *   z_mean = sum z_bar / n, y_mean = sum y / n,
 *   G_c = G - n z_mean z_mean^T (fp64, symmetrised),
 *   q_c = sum z_bar y - n z_mean y_mean,
 *   one eigendecomposition G_c = V diag(s) V^T (rocSOLVER dsyevd; s taken
 *   as max(s, 0)); for every lam of `lambdas`:
 *     a(lam) = V (V^T q_c / (s + lam)),
 *     RSS(lam) = y_c^T y_c - 2 a^T q_c + a^T G_c a,
 *     evidence(lam) = -(n/2) log(RSS + lam ||a||^2) + 1/2 sum log(lam / (s + lam));
 *   the lam of largest evidence (ties: the earlier in the list), and
 *   b = y_mean - a . z_mean + RSS / (2 n) (the log-normal bias correction).
 * Experts no calibration token routed get a = 0, b = 0.
 *   stats      device, 256-B aligned, base_calib_stats_bytes(L) bytes
 *   lambdas    host, n_lambda (1 .. 64) positive values
 *   pred_a     [E][d] fp32 out (device); pred_b [E] fp32 out (device)
 *   lam_out    [E] fp32 out (device), the chosen lam, or NULL
 * Unlike the calls of base.h this is an offline step: it allocates its
 * scratch (device memory for the eigensolver and a rocBLAS handle) and
 * returns after the stream has finished the fit. */
base_status base_calib_fit(const base_layer *L, const void *stats, int32_t n_lambda,
                           const double *lambdas, float *pred_a, float *pred_b,
                           float *lam_out, void *stream);

#ifdef __cplusplus
}
#endif

#endif
