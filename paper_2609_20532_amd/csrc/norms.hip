// Per-example gradient norms and clip factors of the DP-SGD step.
//
// Paper: Section 2.2, per-example clipping by ||g_t(x_i)||_2 over all trainable
// parameters; GPU-side algorithm, clip step. For a linear layer the squared
// norm of g_i = G_i^T A_i can be formed without the [d_out, d_in] gradient:
//
//   T = 1:   ||g_i||^2 = ||a_i||^2 ||g_i||^2                       (rank one)
//   ghost:   ||g_i||^2 = sum_{t,s} (a_t . a_s)(g_t . g_s)
//                      = <A_i A_i^T, G_i G_i^T>_F                  (Gram form)
//   materialise: square-sum of G_i^T A_i tiles kept in registers   (gemm.hip)
//
// The ghost kernel evaluates the Gram form on 128x128 (t, s) tiles of the
// upper triangle (off-diagonal tiles count twice): one MFMA K-loop over d_in
// builds the activation Gram tile, a second over d_out builds the
// output-gradient Gram tile in the same register layout, and the two are
// multiplied element-wise and summed. Each tile writes one float partial;
// a final fixed-order reduction adds the partials of every layer of the call
// into norms_sq, so the result does not depend on scheduling.
#include "mma.h"

namespace dpsgd {
namespace {

// ------------------------------------------------------------------ T = 1

struct T1Entry {
  const void* A;
  const void* G;
  int32_t d_in, d_out;
  int32_t partial_col;
  int32_t pad;
};
struct T1Args {
  T1Entry L[kMaxLayersPerLaunch];
  int32_t n;
  int64_t P;
  float* partials;
};

template <typename TIn>
__global__ __launch_bounds__(kThreads) void t1_norm_kernel(T1Args args) {
  __shared__ float red[4];
  const int64_t i = blockIdx.x;
  const T1Entry& E = args.L[blockIdx.y];
  const TIn* a = static_cast<const TIn*>(E.A) + i * E.d_in;
  const TIn* g = static_cast<const TIn*>(E.G) + i * E.d_out;
  float sa = 0.f, sg = 0.f;
  for (int e = threadIdx.x; e < E.d_in; e += kThreads) { const float v = load_elem(a + e); sa = fmaf(v, v, sa); }
  for (int e = threadIdx.x; e < E.d_out; e += kThreads) { const float v = load_elem(g + e); sg = fmaf(v, v, sg); }
  sa = block_sum(sa, red);
  sg = block_sum(sg, red);
  if (threadIdx.x == 0) args.partials[i * args.P + E.partial_col] = sa * sg;
}

// ------------------------------------------------------------------ ghost

struct GhostEntry {
  const void* A;
  const void* G;
  int32_t d_in, d_out, T;
  int32_t nt;          // 128-row tiles along T
  int32_t pairs;       // nt (nt + 1) / 2 upper-triangle tile pairs
  uint32_t wg_begin;   // first workgroup of this layer in the launch
  int32_t partial_col;
  int32_t pad;
};
struct GhostArgs {
  GhostEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int64_t P;
  float* partials;
};

// Raw 16-byte chunk c of a 128-row x BK tile of a row-major [rows][ld] matrix.
template <typename TIn, bool VEC>
__device__ __forceinline__ uint4 load_chunk(const TIn* X, int64_t ld, int row, int rows_valid,
                                            int k, int d) {
  constexpr int E = TileCfg<TIn>::E;
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (row >= rows_valid) return v;
  const TIn* p = X + (int64_t)row * ld + k;
  if (VEC) {
    if (k < d) v = *reinterpret_cast<const uint4*>(p);
  } else {
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (E == 8) {
      const uint16_t* q = reinterpret_cast<const uint16_t*>(p);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (k + e < d) w[e >> 1] |= (uint32_t)q[e] << (16 * (e & 1));
    } else {
      const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (k + e < d) w[e] = q[e];
    }
    v = make_uint4(w[0], w[1], w[2], w[3]);
  }
  return v;
}

template <typename TIn, bool VEC>
__device__ __forceinline__ void load_tile_rows(const TIn* X, int64_t ld, int rows_valid, int k0,
                                               int d, uint4 (&r)[4]) {
  constexpr int E = TileCfg<TIn>::E;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = threadIdx.x + kThreads * u;
    r[u] = load_chunk<TIn, VEC>(X, ld, c >> 3, rows_valid, k0 + (c & 7) * E, d);
  }
}

template <typename TIn>
__device__ __forceinline__ void store_tile_rows(TIn* Xs, const uint4 (&r)[4]) {
  constexpr int E = TileCfg<TIn>::E;
  constexpr int SK = TileCfg<TIn>::SK;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = threadIdx.x + kThreads * u;
    *reinterpret_cast<uint4*>(Xs + (c >> 3) * SK + (c & 7) * E) = r[u];
  }
}

// acc = Xp[rows_p] Xq[rows_q]^T over k in [0, d), double-buffered through LDS.
template <typename TIn, bool VEC>
__device__ __forceinline__ void gram_phase(const TIn* Xp, const TIn* Xq, int d, int rows_p,
                                           int rows_q, bool diag, f32x4_t (&acc)[4][4],
                                           TIn* lds /* [2 stages][2 operands][OPE] */) {
  constexpr int BK = TileCfg<TIn>::BK;
  constexpr int SK = TileCfg<TIn>::SK;
  constexpr int OPE = lds_operand_elems<TIn>();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int nsteps = (d + BK - 1) / BK;
  uint4 rp[4], rq[4];
  zero_acc(acc);
  load_tile_rows<TIn, VEC>(Xp, d, rows_p, 0, d, rp);
  if (!diag) load_tile_rows<TIn, VEC>(Xq, d, rows_q, 0, d, rq);
  store_tile_rows<TIn>(lds, rp);
  if (!diag) store_tile_rows<TIn>(lds + OPE, rq);
  __syncthreads();
  for (int s = 0; s < nsteps; ++s) {
    const int cur = s & 1;
    const bool more = s + 1 < nsteps;
    if (more) {
      load_tile_rows<TIn, VEC>(Xp, d, rows_p, (s + 1) * BK, d, rp);
      if (!diag) load_tile_rows<TIn, VEC>(Xq, d, rows_q, (s + 1) * BK, d, rq);
    }
    const TIn* P = lds + cur * 2 * OPE;
    const TIn* Q = diag ? P : P + OPE;
    mma_step(P + wm * 64 * SK, Q + wn * 64 * SK, acc, lane);
    if (more) {
      TIn* N = lds + (cur ^ 1) * 2 * OPE;
      store_tile_rows<TIn>(N, rp);
      if (!diag) store_tile_rows<TIn>(N + OPE, rq);
    }
    __syncthreads();
  }
}

template <typename TIn, bool VEC>
__global__ __launch_bounds__(kThreads, 2) void ghost_kernel(GhostArgs args) {
  constexpr int OPE = lds_operand_elems<TIn>();
  __shared__ __attribute__((aligned(16))) TIn lds[2 * 2 * OPE];
  __shared__ float red[4];

  int l = 0;
  {
    int lo = 0, hi = args.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
    }
    l = lo;
  }
  const GhostEntry& E = args.L[l];
  const uint32_t w = blockIdx.x - E.wg_begin;
  const int64_t i = w / (uint32_t)E.pairs;
  const int pr = (int)(w % (uint32_t)E.pairs);
  int p = 0, rem = pr;
  while (rem >= E.nt - p) { rem -= E.nt - p; ++p; }
  const int q = p + rem;
  const int rows_p = min(kTile, E.T - p * kTile);
  const int rows_q = min(kTile, E.T - q * kTile);
  const bool diag = p == q;

  const TIn* A = static_cast<const TIn*>(E.A) + i * (int64_t)E.T * E.d_in;
  const TIn* G = static_cast<const TIn*>(E.G) + i * (int64_t)E.T * E.d_out;

  f32x4_t accA[4][4], accG[4][4];
  gram_phase<TIn, VEC>(A + (int64_t)p * kTile * E.d_in, A + (int64_t)q * kTile * E.d_in, E.d_in,
                       rows_p, rows_q, diag, accA, lds);
  gram_phase<TIn, VEC>(G + (int64_t)p * kTile * E.d_out, G + (int64_t)q * kTile * E.d_out, E.d_out,
                       rows_p, rows_q, diag, accG, lds);
  float s = 0.f;
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) s = fmaf(accA[a][b][v], accG[a][b][v], s);
  s = block_sum(s, red);
  if (threadIdx.x == 0) args.partials[i * args.P + E.partial_col + pr] = diag ? s : 2.0f * s;
}

// ---------------------------------------------------------- reduce, factors

__global__ __launch_bounds__(kThreads) void norms_reduce_kernel(const float* __restrict__ partials,
                                                                int64_t P, int64_t B,
                                                                float* __restrict__ norms_sq,
                                                                int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= B) return;  // uniform per wave
  const int lane = threadIdx.x & 63;
  float s = 0.f;
  for (int64_t j = lane; j < P; j += 64) s += partials[i * P + j];
  s = wave_sum(s);
  if (lane == 0) norms_sq[i] = accumulate ? norms_sq[i] + s : s;
}

__global__ __launch_bounds__(kThreads) void clip_factors_kernel(const float* __restrict__ norms_sq,
                                                                int64_t B, float C,
                                                                float* __restrict__ factors,
                                                                float* __restrict__ factors_out,
                                                                uint8_t* __restrict__ mask_out) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= B) return;
  const float n = sqrtf(norms_sq[i]);
  const bool clipped = n > C;
  const float c = clipped ? C / n : (n == n ? 1.0f : n);  // a NaN norm gives a NaN factor
  if (factors) factors[i] = c;
  if (factors_out) factors_out[i] = c;
  if (mask_out) mask_out[i] = clipped ? 1 : 0;
}

template <typename TIn>
int launch_t1_group(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                    float* partials, int64_t P, int64_t B, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    T1Args args{};
    args.n = m;
    args.P = P;
    args.partials = partials;
    for (int k = 0; k < m; ++k) {
      const dpsgd_layer& L = layers[idx[base + k]];
      args.L[k].A = L.A;
      args.L[k].G = L.G;
      args.L[k].d_in = (int32_t)L.d_in;
      args.L[k].d_out = (int32_t)L.d_out;
      args.L[k].partial_col = (int32_t)cols[idx[base + k]];
    }
    hipLaunchKernelGGL(t1_norm_kernel<TIn>, dim3((uint32_t)B, (uint32_t)m), dim3(kThreads), 0,
                       stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

template <typename TIn, bool VEC>
int launch_ghost_group(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                       float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    GhostArgs args{};
    args.n = m;
    args.P = P;
    args.partials = partials;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const dpsgd_layer& L = layers[idx[base + k]];
      GhostEntry& E = args.L[k];
      E.A = L.A;
      E.G = L.G;
      E.d_in = (int32_t)L.d_in;
      E.d_out = (int32_t)L.d_out;
      E.T = (int32_t)L.T;
      E.nt = (int32_t)ceil_div(L.T, kTile);
      E.pairs = E.nt * (E.nt + 1) / 2;
      E.wg_begin = (uint32_t)wgs;
      E.partial_col = (int32_t)cols[idx[base + k]];
      wgs += L.B * (int64_t)E.pairs;
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL((ghost_kernel<TIn, VEC>), dim3((uint32_t)wgs), dim3(kThreads), 0, stream,
                       args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

// Every row starts 16-byte aligned (the ABI requires aligned A and G).
template <typename TIn>
bool ghost_vec_ok(const dpsgd_layer& L) {
  constexpr int E = TileCfg<TIn>::E;
  return L.d_in % E == 0 && L.d_out % E == 0;
}

template <typename TIn>
int launch_norms_typed(const dpsgd_layer* layers, const NormForm* forms, int n_layers,
                       float* partials, int64_t P, const int64_t* cols, float* park,
                       hipStream_t stream) {
  const int64_t B = layers[0].B;
  int idx_t1[256], n_t1 = 0;
  int idx_gv[256], n_gv = 0;
  int idx_gs[256], n_gs = 0;
  int idx_gd[256], n_gd = 0;
  int idx_g4[256], n_g4 = 0;
  int idx_g64[256], n_g64 = 0;
  int idx_mat[256], n_mat = 0;
  for (int base = 0; base < n_layers; base += 256) {
    n_t1 = n_gv = n_gs = n_gd = n_g4 = n_g64 = n_mat = 0;
    const int m = n_layers - base < 256 ? n_layers - base : 256;
    for (int k = 0; k < m; ++k) {
      const int l = base + k;
      switch (forms[l]) {
        case FORM_T1: idx_t1[n_t1++] = l; break;
        case FORM_STORED: break;   // skinny.hip
        case FORM_GHOST256: idx_g4[n_g4++] = l; break;
        case FORM_GHOST:
          if (ghost_dma_ok(layers[l])) idx_gd[n_gd++] = l;
          else if (gram64_ok(layers[l])) idx_g64[n_g64++] = l;
          else if (ghost_vec_ok<TIn>(layers[l])) idx_gv[n_gv++] = l;
          else idx_gs[n_gs++] = l;
          break;
        default: idx_mat[n_mat++] = l; break;
      }
    }
    int st = DPSGD_OK;
    if (n_t1) st = launch_t1_group<TIn>(layers, idx_t1, n_t1, cols, partials, P, B, stream);
    if (st == DPSGD_OK && n_gv)
      st = launch_ghost_group<TIn, true>(layers, idx_gv, n_gv, cols, partials, P, stream);
    if (st == DPSGD_OK && n_gs)
      st = launch_ghost_group<TIn, false>(layers, idx_gs, n_gs, cols, partials, P, stream);
    if (st == DPSGD_OK && n_gd) st = launch_ghost_dma(layers, idx_gd, n_gd, cols, partials, P, stream);
    if (st == DPSGD_OK && n_g4)
      st = launch_ghost256(layers, idx_g4, n_g4, cols, partials, P, park, stream);
    if (st == DPSGD_OK && n_g64) st = launch_gram64(layers, idx_g64, n_g64, cols, partials, P, stream);
    if (st == DPSGD_OK && n_mat)
      st = launch_mat_norms(layers, idx_mat, n_mat, cols, partials, P, stream);
    if (st != DPSGD_OK) return st;
  }
  return DPSGD_OK;
}

}  // namespace

NormForm resolve_norm_form(const dpsgd_layer& L, int32_t mode) {
  if (L.T == 1) return FORM_T1;
  if (mode == DPSGD_NORM_GHOST) return FORM_GHOST;
  if (mode == DPSGD_NORM_MATERIALIZE) return FORM_MAT;
  // AUTO: compare the MFMA work each form issues at tile granularity.
  const int64_t bk = L.dtype == DPSGD_BF16 ? TileCfg<uint16_t>::BK : TileCfg<float>::BK;
  const int64_t nt = ceil_div(L.T, kTile);
  // (The float32 kernel for T <= 64 takes one 64 x 64 tile: a quarter of the
  // 128 x 128 one.)
  const double ghost = gram64_ok(L) ? (double)(L.d_in + L.d_out) / 4.0
                                    : (double)(nt * (nt + 1) / 2) *
                                          (double)(ceil_div(L.d_in, bk) * bk + ceil_div(L.d_out, bk) * bk);
  // (A k-major float32 tile, 64 x 256 or 128 x 128, has the area of a 128 x 128 one.)
  const int64_t mt = k32_ok(L) ? mat_tile_count(L) : ceil_div(L.d_out, kTile) * ceil_div(L.d_in, kTile);
  const double mat = (double)mt * (double)(ceil_div(L.T, bk) * bk);
  return ghost <= mat ? FORM_GHOST : FORM_MAT;
}

int64_t norm_partials_per_example(const dpsgd_layer& L, NormForm form) {
  switch (form) {
    case FORM_T1: return 1;
    case FORM_STORED: return skinny_chunks(L);
    case FORM_GHOST256: return ghost256_cols(L);
    case FORM_GHOST: {
      const int64_t nt = ceil_div(L.T, kTile);
      return nt * (nt + 1) / 2;
    }
    default:   // the k-major float32 kernel writes one partial per wave of a tile
      return tiny_ok(L) ? 1 : k32_ok(L) ? 4 * mat_tile_count(L) : mat_tile_count(L);
  }
}

int launch_norm_partials(const dpsgd_layer* layers, const NormForm* forms, int n_layers,
                         float* partials, int64_t P, const int64_t* cols, float* park,
                         hipStream_t stream) {
  return layers[0].dtype == DPSGD_BF16
             ? launch_norms_typed<uint16_t>(layers, forms, n_layers, partials, P, cols, park, stream)
             : launch_norms_typed<float>(layers, forms, n_layers, partials, P, cols, park, stream);
}

int launch_norms_reduce(const float* partials, int64_t P, int64_t B, float* norms_sq,
                        int accumulate, hipStream_t stream) {
  const int64_t wgs = ceil_div(B, 4);
  hipLaunchKernelGGL(norms_reduce_kernel, dim3((uint32_t)wgs), dim3(kThreads), 0, stream, partials,
                     P, B, norms_sq, accumulate);
  return check_launch();
}

int launch_norms(const dpsgd_layer* layers, const NormForm* forms, int n_layers, float* norms_sq,
                 int accumulate, float* partials, int64_t P, const int64_t* cols, float* park,
                 hipStream_t stream) {
  const int st = launch_norm_partials(layers, forms, n_layers, partials, P, cols, park, stream);
  if (st != DPSGD_OK) return st;
  return launch_norms_reduce(partials, P, layers[0].B, norms_sq, accumulate, stream);
}

int launch_clip_factors(const float* norms_sq, int64_t B, float C, float* factors,
                        float* factors_out, uint8_t* mask_out, hipStream_t stream) {
  const int64_t wgs = ceil_div(B, kThreads);
  hipLaunchKernelGGL(clip_factors_kernel, dim3((uint32_t)wgs), dim3(kThreads), 0, stream,
                     norms_sq, B, C, factors, factors_out, mask_out);
  return check_launch();
}

}  // namespace dpsgd
