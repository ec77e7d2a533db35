/*
 * dpsgd.h -- C ABI of the MI355X (gfx950) DP-SGD gradient-step library.
 *
 * The library computes, on one GPU, the part of a DP-SGD step that the
 * paper's protocol gives to the untrusted GPU (the algorithm "GPU-side
 * Gradient Computation and Local Update" and Section 2.2, "DP-SGD"):
 *
 *   per-example gradient of each linear layer   g_i = G_i^T A_i
 *   per-example L2 norm over all layers        n_i = sqrt(sum_l ||g_{i,l}||_F^2)
 *   clip factor                                 c_i = min(1, C / n_i)
 *   clipped sum over the batch                  S_l = sum_i c_i g_{i,l}
 *   Gaussian noise of scale sigma*C             out = scale * (S_l + sigma*C*z)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - A linear layer y_t = W x_t is described by a dpsgd_layer: the
 *    activations A [B][T][d_in] and output gradients G [B][T][d_out]
 *    (G[i][t] = dloss_i/dy_t), both row-major and contiguous, both of the
 *    same element type (float32 or bfloat16).
 *  - Gradient-shaped buffers are float32 [d_out][d_in], row-major (the layout
 *    of W itself).
 *  - Every pointer to tensor data is a DEVICE pointer owned by the caller.
 *    The library allocates no device memory, keeps no pointer after a call
 *    returns and holds no mutable global state; calls are thread-safe. The
 *    one exception is dpsgd_per_example_norms_multi_noalloc, whose scratch
 *    array lives in each GPU's memory (see there).
 *  - Arrays of descriptors (dpsgd_layer*, float* const*) are HOST memory and
 *    are read before the call returns.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Every call only enqueues kernels on it and returns; results are valid
 *    once the caller synchronises with the stream. Faults inside a kernel
 *    surface at that synchronisation.
 *  - Every entry point returns a dpsgd_status. Nothing aborts or throws across
 *    the ABI. An error found by the argument checks returns before anything
 *    is enqueued. DPSGD_ERR_HIP (a launch the runtime rejected) and
 *    DPSGD_ERR_INVALID_ARG for a grid too large for one launch (beyond 2^31
 *    workgroups, far past any size the checks accept in practice) can come
 *    after earlier kernels of the same call were enqueued; the outputs are
 *    then unspecified.
 *  - Results are deterministic: the same inputs on the same device give
 *    bitwise-identical outputs (no floating-point atomics).
 *  - Arithmetic: products of bf16 inputs are exact in float32 and all sums
 *    accumulate in float32.
 */
#ifndef DPSGD_H_
#define DPSGD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dpsgd_dtype {
  DPSGD_F32 = 0,   /* IEEE binary32                               */
  DPSGD_BF16 = 1   /* bfloat16 (upper 16 bits of a binary32)       */
} dpsgd_dtype;

typedef enum dpsgd_norm_mode {
  DPSGD_NORM_AUTO = 0,         /* pick per layer by arithmetic cost           */
  DPSGD_NORM_GHOST = 1,        /* Gram form: sum_{t,s} (a_t.a_s)(g_t.g_s)     */
  DPSGD_NORM_MATERIALIZE = 2,  /* ||G_i^T A_i||_F^2, tile kept in registers   */
  DPSGD_NORM_CLOSED_FORM = 3   /* T = 1: ||a_i||^2 ||g_i||^2. Only reported by
                                  dpsgd_select_norm_mode; not accepted as a
                                  mode argument (DPSGD_ERR_UNSUPPORTED)       */
} dpsgd_norm_mode;

typedef enum dpsgd_status {
  DPSGD_OK = 0,
  DPSGD_ERR_INVALID_ARG = -1,  /* null or misaligned required pointer, size < 1 or overflow, C <= 0 or NaN,
                                  sigma < 0 or NaN, scale not finite                      */
  DPSGD_ERR_UNSUPPORTED = -2,  /* unknown dtype or mode, mixed dtypes in one call         */
  DPSGD_ERR_WORKSPACE = -3,    /* workspace NULL or smaller than the *_workspace_bytes value */
  DPSGD_ERR_HIP = -4           /* the HIP runtime rejected a launch                       */
} dpsgd_status;

/* One linear layer y = x W^T (W: [d_out][d_in]) as seen by one batch.
 * Paper: Section 2.2, per-example gradient of the trainable parameters. */
typedef struct dpsgd_layer {
  const void* A;       /* [B][T][d_in]  activations, dtype; 16-byte aligned      */
  const void* G;       /* [B][T][d_out] output gradients dloss_i/dy_t, dtype;
                          16-byte aligned                                         */
  int64_t B;           /* examples in the batch, >= 1                            */
  int64_t T;           /* positions per example (sequence length), >= 1          */
  int64_t d_in;        /* >= 1                                                   */
  int64_t d_out;       /* >= 1                                                   */
  int32_t dtype;       /* dpsgd_dtype, shared by A and G                         */
  uint32_t tensor_id;  /* third Philox counter word of this layer's noise; the
                          layers of one noise call must have distinct ids     */
} dpsgd_layer;

/* ---------------------------------------------------------------------------
 * Per-example norms.  Paper: Section 2.2 (per-example clipping uses
 * ||g_t(x_i)||_2 over all trainable parameters); GPU-side algorithm, clip step.
 *
 * norms_sq[i] = (accumulate ? norms_sq[i] : 0) + sum_l ||G_{l,i}^T A_{l,i}||_F^2
 *
 * over the n_layers layers of the call, all with the same B. One call over all
 * layers of a step gives the squared global norm; per-layer calls with
 * accumulate=1 give the same value up to float32 summation order.
 *   mode      dpsgd_norm_mode, applied to every layer (AUTO picks per layer).
 *   norms_sq  float32 [B], device.
 *   workspace device scratch of at least dpsgd_norms_workspace_bytes(...)
 *             bytes, 16-byte aligned (DPSGD_ERR_INVALID_ARG otherwise); its
 *             contents on entry do not matter and are clobbered. It holds
 *             per-example partials and, when a bf16 layer with T > 256 and
 *             widths that are multiples of 64 runs the Gram form, a park
 *             area of at most 128 MB (256 KB per workgroup of that kernel,
 *             or, when few tiles are split along the columns, two 256 KB
 *             partial tiles per part).
 * T = 1 layers always use the closed form ||a||^2 ||g||^2 whatever the mode.
 * ------------------------------------------------------------------------- */
size_t dpsgd_norms_workspace_bytes(const dpsgd_layer* layers, int32_t n_layers, int32_t mode);

/* The form that dpsgd_per_example_norms[_multi] runs for this layer under
 * DPSGD_NORM_AUTO: DPSGD_NORM_CLOSED_FORM for T = 1 (under every mode),
 * otherwise DPSGD_NORM_GHOST or DPSGD_NORM_MATERIALIZE; or a negative
 * dpsgd_status for an invalid descriptor. (In dpsgd_clipped_sum_multi a
 * layer with a narrow side may take the stored form instead; see there.) */
int32_t dpsgd_select_norm_mode(const dpsgd_layer* layer);

int dpsgd_per_example_norms(const dpsgd_layer* layer, int32_t mode, float* norms_sq,
                            int32_t accumulate, void* workspace, size_t workspace_bytes,
                            void* stream);

int dpsgd_per_example_norms_multi(const dpsgd_layer* layers, int32_t n_layers, int32_t mode,
                                  float* norms_sq, int32_t accumulate, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Per-example norms with no workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.
 *
 * The operation, arguments and results of dpsgd_per_example_norms_multi,
 * with the per-example partials kept in a scratch array of
 * DPSGD_NOALLOC_SCRATCH_BYTES bytes that the library holds in the memory of
 * each GPU it runs on, from the first call on that GPU until the process
 * ends. The call allocates nothing. Results equal the workspace call's bit
 * for bit (the same kernels run), except for bf16 Gram-form layers with
 * T > 256: the workspace call runs them on 256-row tiles, whose park area
 * the array does not hold, this call on 128-row tiles, so their norms agree
 * to float32 rounding.
 *  - Runs on the current device (hipSetDevice), whose stream `stream` must be.
 *    The first call on a device resolves the array's address there (no
 *    stream work); make it before capturing a graph that contains the call.
 *  - DPSGD_ERR_WORKSPACE when the layers need more partial storage than the
 *    array holds (about 2M float partials: B times the sum over layers of
 *    the partials per example, a T > 256 Gram-form layer counting its
 *    128-row tile pairs); checked before anything else touches the device. DPSGD_ERR_HIP when the runtime cannot give the
 *    array's address on the current device. Other errors as in
 *    dpsgd_per_example_norms_multi.
 *  - Every call on one GPU uses that GPU's one array, which keeps the last
 *    call's partials: calls that overlap in time on one GPU (different
 *    streams, or host threads without ordering between them) race, and
 *    their results are undefined.
 * ------------------------------------------------------------------------- */
#define DPSGD_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)

int dpsgd_per_example_norms_multi_noalloc(const dpsgd_layer* layers, int32_t n_layers,
                                          int32_t mode, float* norms_sq, int32_t accumulate,
                                          void* stream);

/* ---------------------------------------------------------------------------
 * Clip factors.  Paper: Section 2.2, g_bar_i = g_i * min(1, C/||g_i||_2).
 *
 *   n_i = sqrt(norms_sq[i]);  factors[i] = n_i > C ? C / n_i : 1;
 *   mask[i] = n_i > C          (1 = clipped; a tie n_i == C is not clipped)
 * computed in float32. C must be > 0 (C = +inf disables clipping).
 * factors (float32 [B]) and mask (uint8 [B]) are device pointers; either may be NULL.
 * ------------------------------------------------------------------------- */
int dpsgd_clip_factors(const float* norms_sq, int64_t B, float C, float* factors,
                       uint8_t* mask, void* stream);

/* ---------------------------------------------------------------------------
 * Clipped sum.  Paper: Section 2.2 aggregation sum_i g_bar_i; GPU-side
 * algorithm, average step (the 1/B is left to dpsgd_add_noise's `scale`).
 *
 *   grad = (accumulate ? grad : 0) + sum_i c_i G_i^T A_i      (float32 [d_out][d_in])
 *
 * with c_i from dpsgd_clip_factors(norms_sq, B, C). factors_out / mask_out
 * (device, optional) receive c and the clip mask. The _multi form does the
 * same for n_layers layers (one grad buffer each, all with the same B) in one
 * grouped launch. workspace: at least dpsgd_clip_workspace_bytes(...) bytes,
 * 16-byte aligned (DPSGD_ERR_INVALID_ARG otherwise).
 * grad must be 16-byte aligned and must not alias any input.
 * ------------------------------------------------------------------------- */
size_t dpsgd_clip_workspace_bytes(const dpsgd_layer* layers, int32_t n_layers);

int dpsgd_clip_accumulate(const dpsgd_layer* layer, const float* norms_sq, float C,
                          float* grad, int32_t accumulate, float* factors_out,
                          uint8_t* mask_out, void* workspace, size_t workspace_bytes,
                          void* stream);

int dpsgd_clip_accumulate_multi(const dpsgd_layer* layers, int32_t n_layers,
                                const float* norms_sq, float C, float* const* grads,
                                int32_t accumulate, float* factors_out, uint8_t* mask_out,
                                void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Norms, factors and clipped sum in one call.  Paper: Section 2.2 (the
 * per-example norm over all layers, the clip factor and the sum of the
 * clipped gradients); GPU-side algorithm, clip and average steps.
 *
 *   norms_sq[i] = sum_l ||G_i^T A_i||_F^2            (float32 [B], overwritten)
 *   c_i, mask_i as in dpsgd_clip_factors(norms_sq, B, C)
 *   grads[l]    = (accumulate ? grads[l] : 0) + sum_i c_i G_i^T A_i
 *
 * the same results as dpsgd_per_example_norms_multi(..., accumulate = 0)
 * followed by dpsgd_clip_accumulate_multi, within float32 rounding. A layer
 * whose narrow side min(d_in, d_out) is at most 16 (a low-rank adapter
 * matrix), whose wide side is a multiple of 4 elements (at most 2^30) and
 * whose per-example gradient (4 d_in d_out bytes) is at most a quarter of its
 * per-example input bytes (T (d_in + d_out) element bytes) is read once:
 * every G_i^T A_i is formed in float32 and stored in the workspace, its
 * squared norm is summed from the stored values and the clipped sum is
 * formed from them. Other layers
 * use the kernels of the separate calls. mode applies to the other layers;
 * DPSGD_NORM_GHOST also turns the stored form off. workspace: at least
 * dpsgd_clipped_sum_workspace_bytes(layers, n_layers, mode) bytes (device,
 * 16-byte aligned; DPSGD_ERR_INVALID_ARG otherwise).
 * factors_out / mask_out are optional. Errors as in the two separate calls;
 * norms_sq must not be NULL.
 * ------------------------------------------------------------------------- */
size_t dpsgd_clipped_sum_workspace_bytes(const dpsgd_layer* layers, int32_t n_layers,
                                         int32_t mode);

int dpsgd_clipped_sum_multi(const dpsgd_layer* layers, int32_t n_layers, int32_t mode, float C,
                            float* const* grads, int32_t accumulate, float* norms_sq,
                            float* factors_out, uint8_t* mask_out, void* workspace,
                            size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Noise.  Paper: Section 2.2, z_t ~ N(0, sigma^2 C^2 I) and
 * g_tilde = (1/|B_t|)(sum + z_t); GPU-side algorithm, noise step
 * (g_tilde = g_bar + Noise(s_noise,t; sigma C)/B).
 *
 *   grad[e] = scale * (grad[e] + sigma * C * z_e),   e in [0, d_out*d_in)
 *
 * in place, float32. z_e is a standard normal from Philox4x32-10 (Salmon et
 * al., SC'11) and Box-Muller (1958): key = (seed mod 2^32, seed >> 32);
 * block j = e/4 has counter (j mod 2^32, j >> 32, layer->tensor_id, step);
 * from its words (r0,r1,r2,r3): u = ((r>>8)+1) 2^-24 for r0, r2 and
 * v = (r>>8) 2^-24 for r1, r3; z_{4j+0,1} = sqrt(-2 ln u_a)(cos, sin)(2 pi v_a),
 * z_{4j+2,3} likewise from (u_b, v_b). sigma == 0 gives exactly scale*grad.
 * Reads only d_in, d_out and tensor_id of the layer descriptor.
 * sigma >= 0, C > 0 and finite, scale finite. The layers of one _multi call
 * must have distinct tensor_ids (DPSGD_ERR_INVALID_ARG otherwise): layers
 * with the same id would get the same normals. Independence across calls is
 * the caller's: every (seed, tensor_id, step) must be used for one release
 * only.
 * ------------------------------------------------------------------------- */
int dpsgd_add_noise(const dpsgd_layer* layer, float* grad, float sigma, float C,
                    uint64_t seed, uint32_t step, float scale, void* stream);

int dpsgd_add_noise_multi(const dpsgd_layer* layers, int32_t n_layers, float* const* grads,
                          float sigma, float C, uint64_t seed, uint32_t step, float scale,
                          void* stream);

/* ---------------------------------------------------------------------------
 * Noise + AdamW step.  Paper: GPU-side algorithm, its last two steps (the
 * noisy average g_tilde = g_bar + Noise(s; sigma C)/B, then OptStep on it);
 * the update is the appendix's one-step AdamW map.
 *
 *   g          = scale * (grad[e] + sigma * C * z_e)       (z_e exactly as dpsgd_add_noise)
 *   m[e]      <- beta1 * m[e] + (1 - beta1) * g
 *   v[e]      <- beta2 * v[e] + (1 - beta2) * g * g
 *   param[e]  <- param[e] - lr * ( (m[e] / (1 - beta1^t)) / (sqrt(v[e] / (1 - beta2^t)) + eps)
 *                                  + weight_decay * param[e] )
 *   noisy_out[e] = g                                       (only when noisy_out is not NULL)
 *
 * for e in [0, d_out*d_in), in float32 (the bias corrections are formed in
 * double on the host). grad is read only. param, exp_avg (m), exp_avg_sq (v),
 * grad and noisy_out are float32 [d_out][d_in] device buffers, 16-byte
 * aligned, pairwise non-overlapping. The _multi form takes one pointer per
 * layer in each array; noisy_outs may be NULL (no layer writes g) or hold
 * NULL entries. The layer descriptor is read as in dpsgd_add_noise.
 * Errors (DPSGD_ERR_INVALID_ARG): a NULL or misaligned required pointer, the
 * noise arguments as in dpsgd_add_noise (distinct tensor_ids included), lr < 0
 * or not finite, beta1 or beta2
 * outside [0, 1), eps <= 0 or not finite, weight_decay < 0 or not finite,
 * t == 0.
 * ------------------------------------------------------------------------- */
typedef struct dpsgd_adamw {
  float lr;            /* learning rate eta_t of this step        */
  float beta1;         /* first-moment decay, in [0, 1)           */
  float beta2;         /* second-moment decay, in [0, 1)          */
  float eps;           /* added to sqrt(v_hat), > 0               */
  float weight_decay;  /* decoupled decay lambda, >= 0            */
  uint32_t t;          /* optimizer step, >= 1 (bias corrections) */
} dpsgd_adamw;

int dpsgd_noise_adamw(const dpsgd_layer* layer, const float* grad, float* param, float* exp_avg,
                      float* exp_avg_sq, float* noisy_out, float sigma, float C, uint64_t seed,
                      uint32_t step, float scale, const dpsgd_adamw* opt, void* stream);

int dpsgd_noise_adamw_multi(const dpsgd_layer* layers, int32_t n_layers,
                            const float* const* grads, float* const* params,
                            float* const* exp_avgs, float* const* exp_avg_sqs,
                            float* const* noisy_outs, float sigma, float C, uint64_t seed,
                            uint32_t step, float scale, const dpsgd_adamw* opt, void* stream);

/* ---------------------------------------------------------------------------
 * Inspection hooks for tests (same stream as dpsgd_add_noise).
 *   dpsgd_philox_u32: out[4*b + w] = word w of block (first_block + b), b < n_blocks.
 *   dpsgd_gaussian:   out[e] = z_e of the stream above for e < n.
 * out is a device pointer.
 * ------------------------------------------------------------------------- */
int dpsgd_philox_u32(uint32_t* out, int64_t first_block, int64_t n_blocks, uint64_t seed,
                     uint32_t tensor_id, uint32_t step, void* stream);
int dpsgd_gaussian(float* out, int64_t n, uint64_t seed, uint32_t tensor_id, uint32_t step,
                   void* stream);

/* Static text for a dpsgd_status value. */
const char* dpsgd_status_string(int status);

/* Library version, for the binding's load check. */
int dpsgd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DPSGD_H_ */
