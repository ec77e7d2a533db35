// C ABI of the DP-SGD gradient-step library: argument checks and dispatch.
// The operations and their conventions are specified in include/dpsgd.h.
#include <math.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"

namespace dpsgd {
namespace {

constexpr int64_t kI32Max = 0x7FFFFFFF;

bool valid_dtype(int32_t d) { return d == DPSGD_F32 || d == DPSGD_BF16; }
bool valid_mode(int32_t m) {
  return m == DPSGD_NORM_AUTO || m == DPSGD_NORM_GHOST || m == DPSGD_NORM_MATERIALIZE;
}

// Shape checks shared by every layer-taking entry point. `data` also requires
// the A and G pointers.
int check_layer(const dpsgd_layer* L, bool data) {
  if (!L) return DPSGD_ERR_INVALID_ARG;
  if (!valid_dtype(L->dtype)) return DPSGD_ERR_UNSUPPORTED;
  if (L->B < 1 || L->T < 1 || L->d_in < 1 || L->d_out < 1) return DPSGD_ERR_INVALID_ARG;
  if (L->B > kI32Max || L->T > kI32Max || L->d_in > kI32Max || L->d_out > kI32Max)
    return DPSGD_ERR_INVALID_ARG;
  // Row and element counts must stay far inside int64 (and rows inside int32).
  const int64_t rows = L->B * L->T;
  if (rows > kI32Max) return DPSGD_ERR_INVALID_ARG;
  if (L->d_in > (INT64_C(1) << 40) / rows || L->d_out > (INT64_C(1) << 40) / rows)
    return DPSGD_ERR_INVALID_ARG;
  if (L->d_out > (INT64_C(1) << 40) / L->d_in) return DPSGD_ERR_INVALID_ARG;
  if (data && (!L->A || !L->G)) return DPSGD_ERR_INVALID_ARG;
  if (data && (!aligned16(L->A) || !aligned16(L->G))) return DPSGD_ERR_INVALID_ARG;
  return DPSGD_OK;
}

// Checks a layer array: every layer valid, one B and one dtype.
int check_layers(const dpsgd_layer* layers, int32_t n, bool data) {
  if (!layers || n < 1) return DPSGD_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n; ++l) {
    const int st = check_layer(&layers[l], data);
    if (st != DPSGD_OK) return st;
    if (layers[l].B != layers[0].B) return DPSGD_ERR_INVALID_ARG;
    if (layers[l].dtype != layers[0].dtype) return DPSGD_ERR_UNSUPPORTED;
  }
  return DPSGD_OK;
}

// Norm workspace: partials [B][P], then (when a layer runs the Gram form on
// 256-row tiles) the park area of those tiles.
struct NormPlan {
  std::vector<NormForm> forms;
  std::vector<int64_t> cols;
  int64_t P = 0;
  size_t park_off = 0;
  size_t bytes = 0;
  float* park(void* ws) const {
    return park_off == bytes ? nullptr : reinterpret_cast<float*>(static_cast<char*>(ws) + park_off);
  }
};

// Form of layer l in a plan: the resolved form, with the Gram form moved to
// 256-row tiles where the layer qualifies and a park area is allowed.
NormForm planned_form(const dpsgd_layer& L, NormForm f, bool park_ok) {
  return f == FORM_GHOST && park_ok && ghost256_ok(L) ? FORM_GHOST256 : f;
}

// Fills cols, P, park_off and bytes from forms. The park area is the largest
// that a launch of 256-row tiles needs, grouped as the norm launcher groups
// the layers (up to 256 layers per group, in order).
void finish_norm_plan(const dpsgd_layer* layers, int32_t n, NormPlan* p) {
  p->P = 0;
  for (int32_t l = 0; l < n; ++l) {
    p->cols[l] = p->P;
    p->P += norm_partials_per_example(layers[l], p->forms[l]);
  }
  size_t park = 0;
  std::vector<int> idx;
  for (int32_t base = 0; base < n; base += 256) {
    idx.clear();
    for (int32_t l = base; l < n && l < base + 256; ++l)
      if (p->forms[l] == FORM_GHOST256) idx.push_back(l);
    if (!idx.empty()) park = std::max(park, ghost256_park_bytes(layers, idx.data(), (int)idx.size()));
  }
  p->park_off = round_up((size_t)layers[0].B * (size_t)p->P * sizeof(float), 256);
  p->bytes = p->park_off + park;
}

NormPlan plan_norms(const dpsgd_layer* layers, int32_t n, int32_t mode, bool park_ok) {
  NormPlan p;
  p.forms.resize(n);
  p.cols.resize(n);
  for (int32_t l = 0; l < n; ++l)
    p.forms[l] = planned_form(layers[l], resolve_norm_form(layers[l], mode), park_ok);
  finish_norm_plan(layers, n, &p);
  return p;
}

constexpr size_t kFactorBytesAlign = 256;

size_t clip_ws_bytes(const dpsgd_layer* layers, int32_t n) {
  size_t part = 0;
  for (int32_t base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    ClipPlan plan;
    plan_clip(layers + base, m, &plan);
    if (plan.partial_bytes > part) part = plan.partial_bytes;
  }
  return round_up((size_t)layers[0].B * sizeof(float), kFactorBytesAlign) + part;
}

bool bad_float(float x) { return isnan(x); }

// The noise of a layer is a function of (seed, tensor_id, step, element):
// two layers of one call with the same tensor_id would receive the same
// normals, and their difference would cancel the noise.
bool distinct_tensor_ids(const dpsgd_layer* layers, int32_t n) {
  std::vector<uint32_t> ids((size_t)n);
  for (int32_t l = 0; l < n; ++l) ids[(size_t)l] = layers[l].tensor_id;
  std::sort(ids.begin(), ids.end());
  return std::adjacent_find(ids.begin(), ids.end()) == ids.end();
}

// Plan of dpsgd_clipped_sum_multi. Workspace: norm partials [B][P], then the
// clip workspace of the other layers (factors first), then the stored
// per-example gradients of the FORM_STORED layers.
struct StepPlan {
  NormPlan norms;
  std::vector<int> stored, other;       // layer indices
  std::vector<int64_t> splits;          // per stored layer
  std::vector<size_t> store_off;        // per stored layer, from the store base
  std::vector<dpsgd_layer> other_layers;
  size_t clip_off = 0, store_base = 0, total = 0;
};

StepPlan plan_step(const dpsgd_layer* layers, int32_t n, int32_t mode) {
  StepPlan p;
  p.norms.forms.resize(n);
  p.norms.cols.resize(n);
  for (int32_t l = 0; l < n; ++l) {
    const bool stored = mode != DPSGD_NORM_GHOST && skinny_ok(layers[l]);
    p.norms.forms[l] =
        stored ? FORM_STORED : planned_form(layers[l], resolve_norm_form(layers[l], mode), true);
    (stored ? p.stored : p.other).push_back(l);
  }
  finish_norm_plan(layers, n, &p.norms);
  const int64_t B = layers[0].B;
  for (int l : p.other) p.other_layers.push_back(layers[l]);
  const size_t clip = p.other.empty()
                          ? round_up((size_t)B * sizeof(float), kFactorBytesAlign)
                          : clip_ws_bytes(p.other_layers.data(), (int32_t)p.other.size());
  p.splits.resize(p.stored.size());
  if (!p.stored.empty())
    plan_skinny(layers, p.stored.data(), (int)p.stored.size(), tr_cu_count(), p.splits.data());
  size_t store = 0;
  for (size_t k = 0; k < p.stored.size(); ++k) {
    p.store_off.push_back(store);
    store += skinny_store_bytes(layers[p.stored[k]], p.splits[k]);
  }
  p.clip_off = p.norms.bytes;
  p.store_base = p.clip_off + round_up(clip, 256);
  p.total = p.store_base + store;
  return p;
}

// Scratch of dpsgd_per_example_norms_multi_noalloc: the per-example norm
// partials. Each GPU the library runs on holds its own copy from the first
// use until the process ends. In host code `scratch` only names the symbol;
// its device address on the current GPU comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[DPSGD_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device, resolved once per
// device; NULL (and *status set) when the runtime cannot provide it.
void* scratch_on_current_device(int* status) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *status = DPSGD_ERR_HIP;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();   // leave no sticky error for the caller's next call
      *status = DPSGD_ERR_HIP;
      return nullptr;
    }
    addr[dev] = p;
  }
  *status = DPSGD_OK;
  return addr[dev];
}

}  // namespace
}  // namespace dpsgd

using namespace dpsgd;

extern "C" {

const char* dpsgd_status_string(int status) {
  switch (status) {
    case DPSGD_OK: return "ok";
    case DPSGD_ERR_INVALID_ARG: return "invalid argument";
    case DPSGD_ERR_UNSUPPORTED: return "unsupported dtype or mode";
    case DPSGD_ERR_WORKSPACE: return "workspace missing or too small";
    case DPSGD_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int dpsgd_version(void) { return 1; }

size_t dpsgd_norms_workspace_bytes(const dpsgd_layer* layers, int32_t n_layers, int32_t mode) {
  if (check_layers(layers, n_layers, false) != DPSGD_OK || !valid_mode(mode)) return 0;
  return plan_norms(layers, n_layers, mode, true).bytes;
}

int32_t dpsgd_select_norm_mode(const dpsgd_layer* layer) {
  const int st = check_layer(layer, false);
  if (st != DPSGD_OK) return st;
  switch (resolve_norm_form(*layer, DPSGD_NORM_AUTO)) {
    case FORM_T1: return DPSGD_NORM_CLOSED_FORM;
    case FORM_MAT: return DPSGD_NORM_MATERIALIZE;
    default: return DPSGD_NORM_GHOST;
  }
}

int dpsgd_per_example_norms_multi(const dpsgd_layer* layers, int32_t n_layers, int32_t mode,
                                  float* norms_sq, int32_t accumulate, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  int st = check_layers(layers, n_layers, true);
  if (st != DPSGD_OK) return st;
  if (!valid_mode(mode)) return DPSGD_ERR_UNSUPPORTED;
  if (!norms_sq) return DPSGD_ERR_INVALID_ARG;
  const NormPlan p = plan_norms(layers, n_layers, mode, true);
  if (!workspace || workspace_bytes < p.bytes) return DPSGD_ERR_WORKSPACE;
  if (!aligned16(workspace)) return DPSGD_ERR_INVALID_ARG;
  return launch_norms(layers, p.forms.data(), n_layers, norms_sq, accumulate ? 1 : 0,
                      static_cast<float*>(workspace), p.P, p.cols.data(), p.park(workspace),
                      static_cast<hipStream_t>(stream));
}

int dpsgd_per_example_norms_multi_noalloc(const dpsgd_layer* layers, int32_t n_layers,
                                          int32_t mode, float* norms_sq, int32_t accumulate,
                                          void* stream) {
  int st = check_layers(layers, n_layers, true);
  if (st != DPSGD_OK) return st;
  if (!valid_mode(mode)) return DPSGD_ERR_UNSUPPORTED;
  if (!norms_sq) return DPSGD_ERR_INVALID_ARG;
  // No park area: T > 256 Gram-form layers take the 128-row tiles here.
  const NormPlan p = plan_norms(layers, n_layers, mode, false);
  if (p.bytes > DPSGD_NOALLOC_SCRATCH_BYTES) return DPSGD_ERR_WORKSPACE;
  void* ws = scratch_on_current_device(&st);
  if (!ws) return st;
  // Every partial slot [i][col] of the plan is written by exactly one job
  // before the reduction reads it, so the scratch needs no clearing.
  return launch_norms(layers, p.forms.data(), n_layers, norms_sq, accumulate ? 1 : 0,
                      static_cast<float*>(ws), p.P, p.cols.data(), nullptr,
                      static_cast<hipStream_t>(stream));
}

int dpsgd_per_example_norms(const dpsgd_layer* layer, int32_t mode, float* norms_sq,
                            int32_t accumulate, void* workspace, size_t workspace_bytes,
                            void* stream) {
  return dpsgd_per_example_norms_multi(layer, 1, mode, norms_sq, accumulate, workspace,
                                       workspace_bytes, stream);
}

int dpsgd_clip_factors(const float* norms_sq, int64_t B, float C, float* factors, uint8_t* mask,
                       void* stream) {
  if (!norms_sq || B < 1 || B > kI32Max) return DPSGD_ERR_INVALID_ARG;
  if (bad_float(C) || !(C > 0.0f)) return DPSGD_ERR_INVALID_ARG;
  return launch_clip_factors(norms_sq, B, C, nullptr, factors, mask,
                             static_cast<hipStream_t>(stream));
}

size_t dpsgd_clip_workspace_bytes(const dpsgd_layer* layers, int32_t n_layers) {
  if (check_layers(layers, n_layers, false) != DPSGD_OK) return 0;
  return clip_ws_bytes(layers, n_layers);
}

int dpsgd_clip_accumulate_multi(const dpsgd_layer* layers, int32_t n_layers,
                                const float* norms_sq, float C, float* const* grads,
                                int32_t accumulate, float* factors_out, uint8_t* mask_out,
                                void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_layers(layers, n_layers, true);
  if (st != DPSGD_OK) return st;
  if (!norms_sq || !grads) return DPSGD_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n_layers; ++l)
    if (!grads[l] || !aligned16(grads[l])) return DPSGD_ERR_INVALID_ARG;
  if (bad_float(C) || !(C > 0.0f)) return DPSGD_ERR_INVALID_ARG;
  const size_t need = clip_ws_bytes(layers, n_layers);
  if (!workspace || workspace_bytes < need) return DPSGD_ERR_WORKSPACE;
  if (!aligned16(workspace)) return DPSGD_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t B = layers[0].B;
  float* factors = static_cast<float*>(workspace);
  float* partial_base = reinterpret_cast<float*>(
      static_cast<char*>(workspace) + round_up((size_t)B * sizeof(float), kFactorBytesAlign));
  st = launch_clip_factors(norms_sq, B, C, factors, factors_out, mask_out, s);
  if (st != DPSGD_OK) return st;
  for (int32_t base = 0; base < n_layers; base += kMaxLayersPerLaunch) {
    const int m = n_layers - base < kMaxLayersPerLaunch ? n_layers - base : kMaxLayersPerLaunch;
    ClipPlan plan;
    plan_clip(layers + base, m, &plan);
    st = launch_clip_sum(layers + base, m, factors, grads + base, accumulate ? 1 : 0,
                         partial_base, plan, s);
    if (st != DPSGD_OK) return st;
  }
  return DPSGD_OK;
}

int dpsgd_clip_accumulate(const dpsgd_layer* layer, const float* norms_sq, float C, float* grad,
                          int32_t accumulate, float* factors_out, uint8_t* mask_out,
                          void* workspace, size_t workspace_bytes, void* stream) {
  float* grads[1] = {grad};
  return dpsgd_clip_accumulate_multi(layer, 1, norms_sq, C, grads, accumulate, factors_out,
                                     mask_out, workspace, workspace_bytes, stream);
}

size_t dpsgd_clipped_sum_workspace_bytes(const dpsgd_layer* layers, int32_t n_layers,
                                         int32_t mode) {
  if (check_layers(layers, n_layers, false) != DPSGD_OK || !valid_mode(mode)) return 0;
  return plan_step(layers, n_layers, mode).total;
}

int dpsgd_clipped_sum_multi(const dpsgd_layer* layers, int32_t n_layers, int32_t mode, float C,
                            float* const* grads, int32_t accumulate, float* norms_sq,
                            float* factors_out, uint8_t* mask_out, void* workspace,
                            size_t workspace_bytes, void* stream) {
  int st = check_layers(layers, n_layers, true);
  if (st != DPSGD_OK) return st;
  if (!valid_mode(mode)) return DPSGD_ERR_UNSUPPORTED;
  if (!norms_sq || !grads) return DPSGD_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n_layers; ++l)
    if (!grads[l] || !aligned16(grads[l])) return DPSGD_ERR_INVALID_ARG;
  if (bad_float(C) || !(C > 0.0f)) return DPSGD_ERR_INVALID_ARG;
  const StepPlan p = plan_step(layers, n_layers, mode);
  if (!workspace || workspace_bytes < p.total) return DPSGD_ERR_WORKSPACE;
  if (!aligned16(workspace)) return DPSGD_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t B = layers[0].B;
  char* ws = static_cast<char*>(workspace);
  float* partials = reinterpret_cast<float*>(ws);
  float* factors = reinterpret_cast<float*>(ws + p.clip_off);
  float* clip_partials = reinterpret_cast<float*>(
      ws + p.clip_off + round_up((size_t)B * sizeof(float), kFactorBytesAlign));
  std::vector<float*> stores, stored_grads;
  for (size_t k = 0; k < p.stored.size(); ++k) {
    stores.push_back(reinterpret_cast<float*>(ws + p.store_base + p.store_off[k]));
    stored_grads.push_back(grads[p.stored[k]]);
  }
  const int n_st = (int)p.stored.size();

  // Norms: the other layers' partials, the stored layers' gradients and
  // partials, then the per-example sums.
  if (!p.other.empty()) {
    st = launch_norm_partials(layers, p.norms.forms.data(), n_layers, partials, p.norms.P,
                              p.norms.cols.data(), p.norms.park(workspace), s);
    if (st != DPSGD_OK) return st;
  }
  if (n_st > 0) {
    st = launch_skinny_norms(layers, p.stored.data(), n_st, p.norms.cols.data(), p.splits.data(),
                             stores.data(), partials, p.norms.P, s);
    if (st != DPSGD_OK) return st;
  }
  st = launch_norms_reduce(partials, p.norms.P, B, norms_sq, 0, s);
  if (st != DPSGD_OK) return st;

  // Factors, then the clipped sums.
  st = launch_clip_factors(norms_sq, B, C, factors, factors_out, mask_out, s);
  if (st != DPSGD_OK) return st;
  const int n_ot = (int)p.other.size();
  std::vector<float*> other_grads;
  for (int l : p.other) other_grads.push_back(grads[l]);
  for (int base = 0; base < n_ot; base += kMaxLayersPerLaunch) {
    const int m = n_ot - base < kMaxLayersPerLaunch ? n_ot - base : kMaxLayersPerLaunch;
    ClipPlan plan;
    plan_clip(p.other_layers.data() + base, m, &plan);
    st = launch_clip_sum(p.other_layers.data() + base, m, factors, other_grads.data() + base,
                         accumulate ? 1 : 0, clip_partials, plan, s);
    if (st != DPSGD_OK) return st;
  }
  if (n_st > 0)
    return launch_skinny_clip(layers, p.stored.data(), n_st, stores.data(), factors,
                              stored_grads.data(), accumulate ? 1 : 0, s);
  return DPSGD_OK;
}

int dpsgd_add_noise_multi(const dpsgd_layer* layers, int32_t n_layers, float* const* grads,
                          float sigma, float C, uint64_t seed, uint32_t step, float scale,
                          void* stream) {
  int st = check_layers(layers, n_layers, false);
  if (st != DPSGD_OK) return st;
  if (!grads) return DPSGD_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n_layers; ++l)
    if (!grads[l]) return DPSGD_ERR_INVALID_ARG;
  if (bad_float(sigma) || sigma < 0.0f || isinf(sigma)) return DPSGD_ERR_INVALID_ARG;
  if (bad_float(C) || !(C > 0.0f) || isinf(C)) return DPSGD_ERR_INVALID_ARG;
  if (!isfinite(scale)) return DPSGD_ERR_INVALID_ARG;
  if (!distinct_tensor_ids(layers, n_layers)) return DPSGD_ERR_INVALID_ARG;
  return launch_noise(layers, n_layers, grads, sigma, C, seed, step, scale,
                      static_cast<hipStream_t>(stream));
}

int dpsgd_add_noise(const dpsgd_layer* layer, float* grad, float sigma, float C, uint64_t seed,
                    uint32_t step, float scale, void* stream) {
  float* grads[1] = {grad};
  return dpsgd_add_noise_multi(layer, 1, grads, sigma, C, seed, step, scale, stream);
}

int dpsgd_noise_adamw_multi(const dpsgd_layer* layers, int32_t n_layers,
                            const float* const* grads, float* const* params,
                            float* const* exp_avgs, float* const* exp_avg_sqs,
                            float* const* noisy_outs, float sigma, float C, uint64_t seed,
                            uint32_t step, float scale, const dpsgd_adamw* opt, void* stream) {
  int st = check_layers(layers, n_layers, false);
  if (st != DPSGD_OK) return st;
  if (!grads || !params || !exp_avgs || !exp_avg_sqs || !opt) return DPSGD_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n_layers; ++l) {
    const void* need[4] = {grads[l], params[l], exp_avgs[l], exp_avg_sqs[l]};
    for (const void* p : need)
      if (!p || !aligned16(p)) return DPSGD_ERR_INVALID_ARG;
    if (noisy_outs && noisy_outs[l] && !aligned16(noisy_outs[l])) return DPSGD_ERR_INVALID_ARG;
  }
  if (bad_float(sigma) || sigma < 0.0f || isinf(sigma)) return DPSGD_ERR_INVALID_ARG;
  if (bad_float(C) || !(C > 0.0f) || isinf(C)) return DPSGD_ERR_INVALID_ARG;
  if (!isfinite(scale)) return DPSGD_ERR_INVALID_ARG;
  const dpsgd_adamw& o = *opt;
  if (!isfinite(o.lr) || o.lr < 0.0f) return DPSGD_ERR_INVALID_ARG;
  if (!(o.beta1 >= 0.0f && o.beta1 < 1.0f) || !(o.beta2 >= 0.0f && o.beta2 < 1.0f))
    return DPSGD_ERR_INVALID_ARG;
  if (!isfinite(o.eps) || !(o.eps > 0.0f)) return DPSGD_ERR_INVALID_ARG;
  if (!isfinite(o.weight_decay) || o.weight_decay < 0.0f) return DPSGD_ERR_INVALID_ARG;
  if (o.t == 0) return DPSGD_ERR_INVALID_ARG;
  if (!distinct_tensor_ids(layers, n_layers)) return DPSGD_ERR_INVALID_ARG;
  return launch_noise_adamw(layers, n_layers, grads, params, exp_avgs, exp_avg_sqs, noisy_outs,
                            sigma, C, seed, step, scale, o, static_cast<hipStream_t>(stream));
}

int dpsgd_noise_adamw(const dpsgd_layer* layer, const float* grad, float* param, float* exp_avg,
                      float* exp_avg_sq, float* noisy_out, float sigma, float C, uint64_t seed,
                      uint32_t step, float scale, const dpsgd_adamw* opt, void* stream) {
  const float* grads[1] = {grad};
  float* params[1] = {param};
  float* ms[1] = {exp_avg};
  float* vs[1] = {exp_avg_sq};
  float* outs[1] = {noisy_out};
  return dpsgd_noise_adamw_multi(layer, 1, grads, params, ms, vs, outs, sigma, C, seed, step,
                                 scale, opt, stream);
}

int dpsgd_philox_u32(uint32_t* out, int64_t first_block, int64_t n_blocks, uint64_t seed,
                     uint32_t tensor_id, uint32_t step, void* stream) {
  if (!out || first_block < 0 || n_blocks < 0) return DPSGD_ERR_INVALID_ARG;
  if (n_blocks > (INT64_C(1) << 36)) return DPSGD_ERR_INVALID_ARG;
  if (n_blocks == 0) return DPSGD_OK;
  return launch_philox_u32(out, first_block, n_blocks, seed, tensor_id, step,
                           static_cast<hipStream_t>(stream));
}

int dpsgd_gaussian(float* out, int64_t n, uint64_t seed, uint32_t tensor_id, uint32_t step,
                   void* stream) {
  if (!out || n < 0 || n > (INT64_C(1) << 38)) return DPSGD_ERR_INVALID_ARG;
  if (n == 0) return DPSGD_OK;
  return launch_gaussian(out, n, seed, tensor_id, step, static_cast<hipStream_t>(stream));
}

}  // extern "C"
