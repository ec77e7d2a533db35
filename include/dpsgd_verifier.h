/*
 * dpsgd_verifier.h -- C ABI of the trusted-side verifier of DP-SGD
 * submissions (CPU only; no GPU runtime is loaded).
 *
 * In the paper's protocol the untrusted GPU commits the clipped average
 * gradient g_gpu = (1/B) sum_i c_i g_i of each step (Section 2.2), and the
 * trusted side checks it with the algorithm "TEE Verification" (Section
 * "Two-Stage Verification"):
 *
 *   1. structural invariant, every step: abort if ||g_gpu|| > C (1 + slack);
 *   2. hidden coin V ~ Bernoulli(p): unchecked steps are accepted;
 *   3. body path: z32 = ||g_gpu - g32|| / C against a float32 recomputation
 *      g32; if z32 <= tau_abs the step is accepted and z32 is charged to the
 *      ledger Z_sub, aborting once Z_sub > K_sub;
 *   4. ambiguity path (z32 > tau_abs): a float64 recomputation g64 gives
 *      n_t = B / (2C) ||g_gpu - g64||; n_t > tau_num = rho_amb B / 2 aborts
 *      (hard rejection); otherwise S_amb += 1, aborting once S_amb > K_amb.
 *      A family without the float64 layer (rho_amb = 0) instead accepts an
 *      escalated step only if z32 <= rho_ill, counted by the same S_amb.
 *
 * Conventions
 *  - Every tensor pointer here is a HOST pointer owned by the caller: the
 *    dpsgd_layer descriptors (A [B][T][d_in], G [B][T][d_out], float32 or
 *    bfloat16, contiguous) and the float32 / float64 [d_out][d_in] gradient
 *    buffers. Nothing is kept after a call returns.
 *  - The coin is an input: the trusted caller draws it from its own hidden
 *    entropy after the submission is committed.
 *  - `threads` is the number of worker threads for a recomputation (<= 0:
 *    the hardware concurrency). Results do not depend on it: every sum has a
 *    fixed order.
 *  - Every entry point returns a dpsgd_status (dpsgd.h) or the value below;
 *    nothing throws across the ABI.
 */
#ifndef DPSGD_VERIFIER_H_
#define DPSGD_VERIFIER_H_

#include <stdint.h>

#include "dpsgd.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Returned by dpsgd_verify_step once the run has been aborted: an aborted
 * run accepts no further step. */
#define DPSGD_ERR_ABORTED (-5)

/* Frozen parameters of one model family (paper: appendix table of frozen
 * verifier parameters). Thresholds are in clipping-norm units. */
typedef struct dpsgd_verifier_params {
  double p;           /* audit rate of the caller's coin (recorded, not drawn here) */
  double tau_abs;     /* body / escalation routing threshold on z32, >= 0           */
  double rho_amb;     /* float64 acceptance radius on z64 (= 2 tau_num / B); 0 when
                         the family has no float64 layer                           */
  double rho_ill;     /* hard cap on z32 of an escalated step when rho_amb == 0       */
  double K_sub;       /* body ledger limit, >= 0                                     */
  int64_t K_amb;      /* accepted-escalation limit, >= 0                             */
  double C;           /* clipping norm, > 0                                          */
  int64_t B;          /* aggregation denominator of the average, >= 1                */
  double norm_slack;  /* structural invariant slack (1e-4 in the paper), >= 0        */
} dpsgd_verifier_params;

/* Ledgers of one run; zero-initialise with dpsgd_verifier_init. */
typedef struct dpsgd_verifier_state {
  double Z_sub;       /* cumulative body discrepancy                                 */
  int64_t S_amb;      /* accepted escalations                                        */
  int64_t steps;      /* submissions seen                                            */
  int64_t checked;    /* submissions whose coin was 1                                */
  int32_t aborted;    /* 1 once any step aborted                                     */
  int32_t pad;
} dpsgd_verifier_state;

typedef enum dpsgd_verify_decision { DPSGD_VERIFY_ACCEPT = 0, DPSGD_VERIFY_ABORT = 1 } dpsgd_verify_decision;

typedef enum dpsgd_verify_path {
  DPSGD_PATH_STRUCTURAL = 0,  /* norm invariant violated (decision ABORT)            */
  DPSGD_PATH_UNCHECKED = 1,   /* coin 0 (ACCEPT)                                     */
  DPSGD_PATH_BODY = 2,        /* z32 <= tau_abs (ACCEPT, or ABORT on Z_sub > K_sub)  */
  DPSGD_PATH_AMBIGUITY = 3,   /* escalated and within the radius (ACCEPT, or ABORT on
                                 S_amb > K_amb)                                      */
  DPSGD_PATH_HARD = 4         /* escalated and outside the radius (ABORT)            */
} dpsgd_verify_path;

typedef struct dpsgd_verify_result {
  int32_t decision;   /* dpsgd_verify_decision                                       */
  int32_t path;       /* dpsgd_verify_path                                           */
  double norm;        /* ||g_gpu||_2 over all layers                                 */
  double z32;         /* NaN when not computed                                       */
  double n_t;         /* B / (2C) ||g_gpu - g64||; NaN when not computed             */
} dpsgd_verify_result;

/* Validates params and zeroes *state. Errors: DPSGD_ERR_INVALID_ARG for a NULL
 * pointer, C <= 0, B < 1, a negative or NaN threshold or limit, or
 * rho_amb == 0 and rho_ill == 0 together. */
int dpsgd_verifier_init(const dpsgd_verifier_params* params, dpsgd_verifier_state* state);

/* Trusted recomputation of the clipped average of every layer,
 * out_l = (1/B) sum_i c_i G_{i,l}^T A_{i,l}, with n_i^2 = sum_l ||G_i^T A_i||_F^2
 * (norm over all layers) and c_i = min(1, C / n_i) (n_i = 0 gives 1); paper:
 * Section 2.2 and the verifier's FP32 / FP64 recomputations. Every
 * operation is carried out in float (f32) or double (f64): squared norms in
 * the Gram form sum_{t,s} (a_t.a_s)(g_t.g_s) or from the materialised
 * gradient (whichever needs fewer multiply-adds), the weighted sum in fixed
 * example order. All layers must have the same B (examples) and dtype; B
 * here is the denominator, which may differ from the layers' B.
 * out[l] is [d_out][d_in]. Errors: DPSGD_ERR_INVALID_ARG (NULL pointer, size
 * < 1, mismatched example counts, C <= 0 or NaN), DPSGD_ERR_UNSUPPORTED (dtype). */
int dpsgd_reference_mean_f32(const dpsgd_layer* layers, int n_layers, float C, int64_t B,
                             float* const* out, int threads);
int dpsgd_reference_mean_f64(const dpsgd_layer* layers, int n_layers, double C, int64_t B,
                             double* const* out, int threads);

/* One step of the verifier for the submission g_gpu[l] ([d_out][d_in]
 * float32 per layer): updates *state and fills *result. The recomputations
 * run only when needed (float32 when coin != 0, float64 on escalation).
 * Returns DPSGD_OK whatever the decision; DPSGD_ERR_ABORTED if the run was
 * already aborted (state untouched); DPSGD_ERR_INVALID_ARG / _UNSUPPORTED as
 * for the recomputation or for invalid params. */
int dpsgd_verify_step(const dpsgd_verifier_params* params, dpsgd_verifier_state* state,
                      const dpsgd_layer* layers, int n_layers, const float* const* g_gpu, int coin,
                      int threads, dpsgd_verify_result* result);

#ifdef __cplusplus
}
#endif

#endif  /* DPSGD_VERIFIER_H_ */
