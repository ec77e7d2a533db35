// Internal declarations shared by the library's HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dpsgd.h"

namespace dpsgd {

// ----------------------------------------------------------------- constants

constexpr int kThreads = 256;          // every kernel uses 4 wave64s per workgroup
constexpr int kMaxLayersPerLaunch = 48;  // entries of a per-launch layer table (kernarg space)

// Norm form actually run for a layer (T = 1 always uses the closed form).
// FORM_STORED (only in dpsgd_clipped_sum_multi): per-example gradients of a
// layer with a narrow side are formed once, stored and normed (skinny.hip).
// FORM_GHOST256: the Gram form on 256-row tiles (T > 256, ghost.hip), chosen
// by the workspace plans for FORM_GHOST layers that qualify.
enum NormForm : int { FORM_T1 = 0, FORM_GHOST = 1, FORM_MAT = 2, FORM_STORED = 3, FORM_GHOST256 = 4 };
constexpr int64_t kSkinnyMaxRank = 16;   // narrow side of a FORM_STORED layer

// ----------------------------------------------------------- device helpers

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Round two floats to bf16 (nearest-even) and pack them (lo in bits 0..15).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo;
  __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Deterministic sum over a wave64 (fixed butterfly order).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Deterministic sum over a 256-thread workgroup; result valid in every thread.
// `red` is __shared__ float[4]. Contains barriers: call from uniform control flow.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ------------------------------------------------------------ host helpers

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ------------------------------------------------------------ launchers
// Each launcher validates nothing (the C ABI layer does) and returns a
// dpsgd_status. Tables are built on the host and passed as kernel arguments.

// Norm partial slots of one layer: how many float partials per example the
// chosen form writes.
int64_t norm_partials_per_example(const dpsgd_layer& L, NormForm form);
NormForm resolve_norm_form(const dpsgd_layer& L, int32_t mode);

// Writes per-example partials partials[i * P + col_l + j] for the given layers
// (all with the chosen forms), then reduces them into norms_sq. park: the
// FORM_GHOST256 layers' park area (ghost256_park_bytes of their jobs), else
// unused.
int launch_norms(const dpsgd_layer* layers, const NormForm* forms, int n_layers,
                 float* norms_sq, int accumulate, float* partials, int64_t P,
                 const int64_t* cols, float* park, hipStream_t stream);
// The two halves of launch_norms; the partials pass skips FORM_STORED layers.
int launch_norm_partials(const dpsgd_layer* layers, const NormForm* forms, int n_layers,
                         float* partials, int64_t P, const int64_t* cols, float* park,
                         hipStream_t stream);
int launch_norms_reduce(const float* partials, int64_t P, int64_t B, float* norms_sq,
                        int accumulate, hipStream_t stream);

// Stored per-example gradients of layers with a narrow side (skinny.hip).
// skinny_ok: eligible (narrow side <= kSkinnyMaxRank, wide side a multiple of
// 16 bytes, gradient at most 1/4 of the input bytes); skinny_chunks: norm
// partials per example; plan_skinny: row ranges per layer (idx order);
// skinny_store_bytes: the layer's store. stores[k] / outs[k] / splits[k] are
// per position k of idx, cols per layer index.
bool skinny_ok(const dpsgd_layer& L);
int64_t skinny_chunks(const dpsgd_layer& L);
void plan_skinny(const dpsgd_layer* layers, const int* idx, int n, int cus, int64_t* splits);
size_t skinny_store_bytes(const dpsgd_layer& L, int64_t splits);
int launch_skinny_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                        const int64_t* splits, float* const* stores, float* partials, int64_t P,
                        hipStream_t stream);
int launch_skinny_clip(const dpsgd_layer* layers, const int* idx, int n, float* const* stores,
                       const float* factors, float* const* outs, int accumulate,
                       hipStream_t stream);

// 256x256-tile bf16 kernels (gemm_tr.hip): eligibility (bf16, d_in and d_out
// multiples of 256, T a multiple of 32), K slices of a layer, launchers.
// Gram-form norms with direct LDS loads (ghost.hip): bf16, widths % 64 == 0.
bool ghost_dma_ok(const dpsgd_layer& L);
// Gram-form norms for float32 layers with 2 <= T <= 64 and widths % 64 == 0
// (gram32.hip): one 64 x 64 tile per example, one partial per example.
bool gram64_ok(const dpsgd_layer& L);
int launch_gram64(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                  float* partials, int64_t P, hipStream_t stream);
int launch_ghost_dma(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                     float* partials, int64_t P, hipStream_t stream);
// Gram-form norms on 256-row tiles (ghost.hip): ghost_dma_ok layers with
// T > 256, ghost256_cols partials per example (nt^2 for nt row blocks: one
// per diagonal tile, two per off-diagonal tile). At most kGhost256MaxGrid
// workgroups run. A launch keeps whole tiles, runs its off-diagonal tiles as
// two row halves (each workgroup parks a 256 KB float32 tile), or splits
// every tile's columns into parts that park their partial Gram tiles for a
// combine pass; ghost256_park_bytes: the park area of launch_ghost256 over
// the layers idx[0..n) (the largest launch).
constexpr int64_t kGhost256MaxGrid = 512;
bool ghost256_ok(const dpsgd_layer& L);
int64_t ghost256_cols(const dpsgd_layer& L);
size_t ghost256_park_bytes(const dpsgd_layer* layers, const int* idx, int n);
int launch_ghost256(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                    float* partials, int64_t P, float* park, hipStream_t stream);

bool tr_tile_ok(const dpsgd_layer& L);
// k-major float32 kernel (gemm.hip): float32, T a multiple of 32, d_in and d_out
// multiples of 4 and at most 2^24. Tiles are 64 x 256 for d_out <= 64, else
// 128 x 128 (rows along d_out, columns along d_in).
bool k32_ok(const dpsgd_layer& L);
int k32_tile_m(const dpsgd_layer& L);
int k32_tile_n(const dpsgd_layer& L);
int k32_ex_per_job(const dpsgd_layer& L);   // examples per materialised-norm job
// Layers whose g_i has at most 512 entries (gemm.hip) form g_i on the VALU:
// one norm partial per example; the clip runs tiny_jobs(L) jobs of
// consecutive examples, one partial sum each.
bool tiny_ok(const dpsgd_layer& L);
int tiny_jobs(const dpsgd_layer& L);
// Output tiles of the materialised-norm kernel that takes the layer (one norm
// partial per tile and example).
int64_t mat_tile_count(const dpsgd_layer& L);
int64_t tr_q_total(const dpsgd_layer& L);
int tr_cu_count();

// Work split of one clip launch over the 256-tile kernel: whole tiles for the
// full rounds over the CUs, the last round's K slices spread over tail workers.
struct TrClipPlan {
  int64_t n_tiles = 0, n_full = 0, n_tail = 0, Q = 0, tail_w = 1;
  size_t tail_bytes = 0;  // tail partials in the workspace
};
// K ranges that each of the rem leftover tiles (rem < cus) of a whole-tile
// launch is split into; 1 leaves them whole. Unsplit they take one round of
// whole-tile time; split w ways they take ceil(rem w / cus) rounds of 1 / w of
// it, plus the traffic of rem w partial tiles written and read back by the
// fixup. The estimate prices a tile's flops at a sustained per-CU matrix rate
// and the partial bytes at a sustained HBM rate; ties keep the smaller w.
inline int64_t choose_tail_split(int64_t rem, int64_t cus, int64_t Q, double tile_flops,
                                 double tile_bytes) {
  constexpr double kCuFlops = 4.0e12;   // flop/s of one CU in these kernels
  constexpr double kHbm = 5.0e12;       // B/s for the partial writes and reads
  constexpr int64_t kMaxSplit = 16;
  if (rem <= 0 || cus <= 0) return 1;
  const double t_tile = tile_flops / kCuFlops;
  double best = t_tile;
  int64_t w_best = 1;
  for (int64_t w = 2; w <= kMaxSplit && w <= Q; ++w) {
    const int64_t rounds = (rem * w + cus - 1) / cus;
    const double t = (double)rounds / (double)w * t_tile + 2.0 * (double)(rem * w) * tile_bytes / kHbm;
    if (t < best) { best = t; w_best = w; }
  }
  return w_best;
}
void plan_tr_clip(const dpsgd_layer* layers, const int* idx, int n, int cus, TrClipPlan* plan);
int launch_tr_clip(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                   float* const* outs, int accumulate, const TrClipPlan& plan, float* tail_ws,
                   hipStream_t stream);
// 384x256-tile clip kernel (gemm_wide.hip): bf16, d_in % 256 == 0, T % 64 == 0,
// d_out % 384 == 0, or d_out % 32 == 0 with a ragged last row tile padding at
// most 6 % of d_out when the layer has at least one round of tiles (one per
// CU); preferred over the 256-tile kernel.
bool wide_tile_ok(const dpsgd_layer& L);
void plan_wide_clip(const dpsgd_layer* layers, const int* idx, int n, int cus, TrClipPlan* plan);
int launch_wide_clip(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                     float* const* outs, int accumulate, const TrClipPlan& plan, float* tail_ws,
                     hipStream_t stream);
int launch_tr_mat_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                        float* partials, int64_t P, hipStream_t stream);

// Materialised-norm partials (gemm.hip) for the layers idx[0..n).
int launch_mat_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                     float* partials, int64_t P, hipStream_t stream);

int launch_clip_factors(const float* norms_sq, int64_t B, float C, float* factors,
                        float* factors_out, uint8_t* mask_out, hipStream_t stream);

// Split plan of the clip-weighted sum.
struct ClipPlan {
  int splits[kMaxLayersPerLaunch];
  size_t partial_offset[kMaxLayersPerLaunch];  // bytes from the partial base
  size_t partial_bytes;                          // total (split partials + 256-tile tail)
  TrClipPlan tr;                                 // layers on the 256-tile kernel
  size_t tr_offset;                              // their tail partials, from the partial base
  TrClipPlan wide;                               // layers on the 384x256-tile kernel
  size_t wide_offset;
};
void plan_clip(const dpsgd_layer* layers, int n_layers, ClipPlan* plan);

int launch_clip_sum(const dpsgd_layer* layers, int n_layers, const float* factors,
                    float* const* grads, int accumulate, float* partial_base,
                    const ClipPlan& plan, hipStream_t stream);

int launch_noise(const dpsgd_layer* layers, int n_layers, float* const* grads, float sigma,
                 float C, uint64_t seed, uint32_t step, float scale, hipStream_t stream);

int launch_noise_adamw(const dpsgd_layer* layers, int n_layers, const float* const* grads,
                       float* const* params, float* const* ms, float* const* vs,
                       float* const* noisy, float sigma, float C, uint64_t seed, uint32_t step,
                       float scale, const dpsgd_adamw& opt, hipStream_t stream);
int launch_philox_u32(uint32_t* out, int64_t first_block, int64_t n_blocks, uint64_t seed,
                      uint32_t tensor_id, uint32_t step, hipStream_t stream);
int launch_gaussian(float* out, int64_t n, uint64_t seed, uint32_t tensor_id, uint32_t step,
                    hipStream_t stream);

inline int check_launch() {
  return hipGetLastError() == hipSuccess ? DPSGD_OK : DPSGD_ERR_HIP;
}

}  // namespace dpsgd
