// Transposed-operand MFMA GEMM of the DP-SGD step: clip-weighted sum and
// materialised per-example norms.
//
// Paper: Section 2.2 aggregation sum_i g_bar_i with g_bar_i = c_i g_i and
// g_i = G_i^T A_i; GPU-side algorithm, clip and average steps.
//
//   clip-weighted sum:  S[m][n] = sum_k w_k G[k][m] A[k][n]     k = (i, t), w_k = c_i
//   materialised norm:  sum_{m,n} (sum_{t} G_i[t][m] A_i[t][n])^2   per example i
//
// Both operands are stored k-major (G is [B*T][d_out], A is [B*T][d_in], the
// reduction index is the outer one), while the MFMA operand wants k
// contiguous per lane. Each thread therefore loads an 8(k) x 8(col) bf16
// block (8 x 16-byte coalesced loads), transposes it in registers and writes
// eight 16-byte rows of the [col][k] LDS tile (fp32: 8(k) x 4(col) blocks).
// The MFMA core is shared with the Gram kernel (mma.h).
//
// Clip weights. For bf16 the factor c_i cannot be applied to an operand
// without an extra bf16 rounding, so when every K step of a workgroup lies in
// one example (per-example stepping; rows past the example's end are zero)
// the accumulator is kept in units of the current example's factor and
// rescaled by c_prev / c_next at each example boundary, with one final
// multiply by the last factor: the weights are applied in fp32. When T is too
// small for per-example steps, or for fp32 inputs, the weight is applied to
// the G operand in fp32 while it is transposed (for bf16 that costs one
// rounding of c_i * G to bf16).
//
// Split K. Small outputs are split along K to fill the GPU; each split writes
// its own fp32 partial and a second kernel adds them in split order, so the
// result is deterministic.
#include "mma.h"

namespace dpsgd {
namespace {

enum ScaleMode : int { SCALE_NONE = 0, SCALE_OPERAND = 1, SCALE_ACC = 2 };
enum EpiMode : int { EPI_STORE = 0, EPI_SUMSQ = 1 };

struct TGemmEntry {
  const void* Xm;        // G: [B*T][M]
  const void* Xn;        // A: [B*T][N]
  float* out;            // EPI_STORE: grad (splits == 1) or this layer's split partials
  int32_t M, N, T;
  int32_t tiles_n;       // 128-wide tiles along N
  int32_t splits;        // EPI_STORE: K splits
  int32_t q_per_split;   // EPI_STORE: K steps per split
  uint32_t wg_begin;     // first workgroup of this layer in the launch
  int32_t partial_col;   // EPI_SUMSQ: first partial slot of the layer
  int32_t accumulate;    // EPI_STORE, splits == 1: add to grad
  int32_t pad;
};

struct TGemmArgs {
  TGemmEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  const float* factors;  // clip factors [B] (SCALE modes)
  float* partials;       // EPI_SUMSQ
  int64_t P;
};

// Row range of K step q.
struct StepRows {
  int64_t row0;   // first global row (over B*T)
  int nrows;      // valid rows in this step (<= BK)
  int ex;         // example of the step (per-example stepping only)
};

template <int BK, bool PER_EXAMPLE>
__device__ __forceinline__ StepRows step_rows(int64_t q, int T, int B) {
  StepRows s;
  if (PER_EXAMPLE) {
    const int spe = (T + BK - 1) / BK;
    const int ex = (int)(q / spe);
    const int ls = (int)(q - (int64_t)ex * spe);
    s.row0 = (int64_t)ex * T + (int64_t)ls * BK;
    s.nrows = min(BK, T - ls * BK);
    s.ex = ex;
  } else {
    s.row0 = q * BK;
    const int64_t left = (int64_t)B * T - s.row0;
    s.nrows = left < BK ? (int)left : BK;
    s.ex = -1;
  }
  return s;
}

// ------------------------------------------------------ transposing loader
//
// Thread t of half h (h = 0: G side, rows = M; h = 1: A side, rows = N) owns
// block (kb, cb): k rows kb*8 .. +8 of the step and columns col0 + cb*CW .. +CW
// (CW = 8 for bf16, 4 for fp32).

template <typename TIn> struct TBlock;
template <> struct TBlock<uint16_t> { static constexpr int KB = 8, CW = 8; };
template <> struct TBlock<float> { static constexpr int KB = 4, CW = 4; };

template <typename TIn, bool VEC>
__device__ __forceinline__ void tload(const TIn* __restrict__ X, int R, int col0, const StepRows& sr,
                                      int nrows_eff, uint4 (&r)[8]) {
  constexpr int KB = TBlock<TIn>::KB, CW = TBlock<TIn>::CW;
  const int t = threadIdx.x & 127;
  const int kb = t % KB, cb = t / KB;
  const int c0 = col0 + cb * CW;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int k = kb * 8 + j;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (k < nrows_eff && c0 < R) {
      const TIn* p = X + (sr.row0 + k) * (int64_t)R + c0;
      if (VEC) {
        v = *reinterpret_cast<const uint4*>(p);
      } else {
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        if (CW == 8) {
          const uint16_t* q = reinterpret_cast<const uint16_t*>(p);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (c0 + e < R) w[e >> 1] |= (uint32_t)q[e] << (16 * (e & 1));
        } else {
          const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (c0 + e < R) w[e] = q[e];
        }
        v = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
    r[j] = v;
  }
}

__device__ __forceinline__ uint32_t word_of(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

// Transpose the block into LDS ([col][k], k contiguous). With SCALE, row j of
// the block is multiplied by wrow[j] in fp32 first.
template <bool SCALE>
__device__ __forceinline__ void tstore(uint16_t* Xs, const uint4 (&r)[8], const float (&wrow)[8]) {
  constexpr int SK = TileCfg<uint16_t>::SK;
  const int t = threadIdx.x & 127;
  const int kb = t % 8, cb = t / 8;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    uint32_t o[4];
#pragma unroll
    for (int jp = 0; jp < 4; ++jp) {
      const uint32_t a = word_of(r[2 * jp], c >> 1);
      const uint32_t b = word_of(r[2 * jp + 1], c >> 1);
      if (SCALE) {
        const float fa = (c & 1) ? bf16_hi(a) : bf16_lo(a);
        const float fb = (c & 1) ? bf16_hi(b) : bf16_lo(b);
        o[jp] = pack_bf16x2(fa * wrow[2 * jp], fb * wrow[2 * jp + 1]);
      } else {
        o[jp] = (c & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
      }
    }
    *reinterpret_cast<uint4*>(Xs + (cb * 8 + c) * SK + kb * 8) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

template <bool SCALE>
__device__ __forceinline__ void tstore(float* Xs, const uint4 (&r)[8], const float (&wrow)[8]) {
  constexpr int SK = TileCfg<float>::SK;
  const int t = threadIdx.x & 127;
  const int kb = t % 4, cb = t / 4;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      f[j] = __uint_as_float(word_of(r[j], c));
      if (SCALE) f[j] *= wrow[j];
    }
    float* dst = Xs + (cb * 4 + c) * SK + kb * 8;
    *reinterpret_cast<float4*>(dst) = make_float4(f[0], f[1], f[2], f[3]);
    *reinterpret_cast<float4*>(dst + 4) = make_float4(f[4], f[5], f[6], f[7]);
  }
}

template <typename TIn, bool VEC, int SCALE, int EPI>
__global__ __launch_bounds__(kThreads, 2) void tgemm_kernel(TGemmArgs args) {
  constexpr int BK = TileCfg<TIn>::BK;
  constexpr int SK = TileCfg<TIn>::SK;
  constexpr int OPE = lds_operand_elems<TIn>();
  constexpr bool PER_EXAMPLE = (SCALE == SCALE_ACC) || (EPI == EPI_SUMSQ);
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
  const TGemmEntry& E = args.L[l];
  const int T = E.T, B = args.B;
  const int tiles_mn = ((E.M + kTile - 1) / kTile) * E.tiles_n;
  const uint32_t w = blockIdx.x - E.wg_begin;
  const int outer = (int)(w / (uint32_t)tiles_mn);  // split (STORE) or example (SUMSQ)
  const int tile = (int)(w % (uint32_t)tiles_mn);
  const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;

  const int64_t spe = (T + BK - 1) / BK;
  int64_t q0, q1;
  if (EPI == EPI_SUMSQ) {
    q0 = (int64_t)outer * spe;
    q1 = q0 + spe;
  } else {
    const int64_t q_total = PER_EXAMPLE ? (int64_t)B * spe : ((int64_t)B * T + BK - 1) / BK;
    q0 = (int64_t)outer * E.q_per_split;
    q1 = min(q0 + (int64_t)E.q_per_split, q_total);
  }

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const bool g_side = tid < 128;
  const TIn* X = static_cast<const TIn*>(g_side ? E.Xm : E.Xn);
  const int R = g_side ? E.M : E.N;
  const int col0 = (g_side ? tm : tn) * kTile;

  f32x4_t acc[4][4];
  zero_acc(acc);
  float c_cur = 1.0f;    // accumulator unit (SCALE_ACC): acc * c_cur is the weighted sum
  bool started = false;  // a non-zero factor has been seen
  int ex_cur = -1;

  uint4 rbuf[8];
  float wrow[8];

  auto fetch = [&](int64_t q) {
    const StepRows sr = step_rows<BK, PER_EXAMPLE>(q, T, B);
    int nrows_eff = sr.nrows;
    // Rows of an example whose factor is 0 are read as zeros on both sides, so
    // that example contributes exactly nothing, also when its inputs are not
    // finite.
    if (SCALE == SCALE_ACC && args.factors[sr.ex] == 0.0f) nrows_eff = 0;
    tload<TIn, VEC>(X, R, col0, sr, nrows_eff, rbuf);
    if (SCALE == SCALE_OPERAND) {
      const int kb = (tid & 127) % TBlock<TIn>::KB;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int64_t row = sr.row0 + kb * 8 + j;
        const float c = kb * 8 + j < sr.nrows ? args.factors[row / T] : 1.0f;
        wrow[j] = g_side ? c : 1.0f;
        if (c == 0.0f) rbuf[j] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };
  auto commit = [&](int buf) {
    TIn* dst = lds + buf * 2 * OPE + (g_side ? 0 : OPE);
    if (SCALE == SCALE_OPERAND && g_side) tstore<true>(dst, rbuf, wrow);
    else tstore<false>(dst, rbuf, wrow);
  };

  if (q0 < q1) {
    fetch(q0);
    commit(0);
  }
  __syncthreads();
  for (int64_t q = q0; q < q1; ++q) {
    const int cur = (int)((q - q0) & 1);
    const bool more = q + 1 < q1;
    if (SCALE == SCALE_ACC) {
      const int ex = step_rows<BK, true>(q, T, B).ex;
      if (ex != ex_cur) {
        const float c_new = args.factors[ex];
        if (c_new != 0.0f) {
          if (started && c_cur != c_new) scale_acc(acc, c_cur / c_new);
          c_cur = c_new;
          started = true;
        }
        ex_cur = ex;
      }
    }
    if (more) fetch(q + 1);
    const TIn* Ms = lds + cur * 2 * OPE;
    mma_step(Ms + wm * 64 * SK, Ms + OPE + wn * 64 * SK, acc, lane);
    if (more) commit(cur ^ 1);
    __syncthreads();
  }

  if (EPI == EPI_SUMSQ) {
    float s = 0.f;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) s = fmaf(acc[a][b][v], acc[a][b][v], s);
    s = block_sum(s, red);
    if (tid == 0) args.partials[(int64_t)outer * args.P + E.partial_col + tile] = s;
  } else {
    if (SCALE == SCALE_ACC) scale_acc(acc, c_cur);
    float* out = E.out + (E.splits > 1 ? (int64_t)outer * E.M * E.N : 0);
    const bool add = E.splits == 1 && E.accumulate;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int n = tn * kTile + wn * 64 + b * 16 + (lane & 15);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = tm * kTile + wm * 64 + a * 16 + 4 * (lane >> 4) + v;
          if (m < E.M && n < E.N) {
            float* p = out + (int64_t)m * E.N + n;
            *p = add ? *p + acc[a][b][v] : acc[a][b][v];
          }
        }
      }
  }
}

// --------------------------------------------------------- split-K reduce

struct SplitEntry {
  float* grad;
  const float* part;     // [splits][numel]
  int64_t numel;
  int32_t splits;
  int32_t accumulate;
  uint32_t wg_begin;
  int32_t vec;           // grad, part 16-byte aligned and numel % 4 == 0
};
struct SplitArgs {
  SplitEntry L[kMaxLayersPerLaunch];
  int32_t n;
};

constexpr int kSplitElemsPerWG = kThreads * 4 * 4;  // 4 float4 per thread

__global__ __launch_bounds__(kThreads) void split_reduce_kernel(SplitArgs args) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
  }
  const SplitEntry& E = args.L[lo];
  const int64_t base = (int64_t)(blockIdx.x - E.wg_begin) * kSplitElemsPerWG;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int64_t e = base + ((int64_t)u * kThreads + threadIdx.x) * 4;
    if (e >= E.numel) break;
    if (E.vec) {
      float4 v = E.accumulate ? *reinterpret_cast<const float4*>(E.grad + e)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s = 0; s < E.splits; ++s) {
        const float4 p = *reinterpret_cast<const float4*>(E.part + (int64_t)s * E.numel + e);
        v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
      }
      *reinterpret_cast<float4*>(E.grad + e) = v;
    } else {
      for (int k = 0; k < 4 && e + k < E.numel; ++k) {
        float v = E.accumulate ? E.grad[e + k] : 0.f;
        for (int s = 0; s < E.splits; ++s) v += E.part[(int64_t)s * E.numel + e + k];
        E.grad[e + k] = v;
      }
    }
  }
}

// ------------------------------------------------------------ host side

int clip_scale_mode(const dpsgd_layer& L) {
  const int64_t bk = L.dtype == DPSGD_BF16 ? TileCfg<uint16_t>::BK : TileCfg<float>::BK;
  const int64_t pad = ceil_div(L.T, bk) * bk - L.T;  // zero rows per example
  return pad * 8 <= L.T ? SCALE_ACC : SCALE_OPERAND;
}

int64_t clip_q_total(const dpsgd_layer& L, int scale) {
  const int64_t bk = L.dtype == DPSGD_BF16 ? TileCfg<uint16_t>::BK : TileCfg<float>::BK;
  return scale == SCALE_ACC ? L.B * ceil_div(L.T, bk) : ceil_div(L.B * L.T, bk);
}

// Every row starts 16-byte aligned (the ABI requires aligned A and G).
template <typename TIn>
bool tgemm_vec_ok(const dpsgd_layer& L) {
  constexpr int E = TileCfg<TIn>::E;
  return L.d_in % E == 0 && L.d_out % E == 0;
}

template <typename TIn, bool VEC, int SCALE, int EPI>
int launch_tgemm_group(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                       float* const* outs, const int* splits, const int* accumulate,
                       const int64_t* cols, float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    TGemmArgs args{};
    args.n = m;
    args.B = (int32_t)layers[idx[base]].B;
    args.factors = factors;
    args.partials = partials;
    args.P = P;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const int li = idx[base + k];
      const dpsgd_layer& L = layers[li];
      TGemmEntry& E = args.L[k];
      E.Xm = L.G;
      E.Xn = L.A;
      E.M = (int32_t)L.d_out;
      E.N = (int32_t)L.d_in;
      E.T = (int32_t)L.T;
      E.tiles_n = (int32_t)ceil_div(L.d_in, kTile);
      const int64_t tiles = ceil_div(L.d_out, kTile) * E.tiles_n;
      E.wg_begin = (uint32_t)wgs;
      if (EPI == EPI_STORE) {
        E.out = outs[base + k];
        E.splits = splits[base + k];
        E.q_per_split = (int32_t)ceil_div(clip_q_total(L, SCALE), E.splits);
        E.accumulate = accumulate ? accumulate[base + k] : 0;
        wgs += tiles * E.splits;
      } else {
        E.partial_col = (int32_t)cols[li];
        wgs += tiles * L.B;
      }
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL((tgemm_kernel<TIn, VEC, SCALE, EPI>), dim3((uint32_t)wgs), dim3(kThreads), 0,
                       stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

}  // namespace

void plan_clip(const dpsgd_layer* layers, int n_layers, ClipPlan* plan) {
  // Layers on the 256- and 384x256-tile kernels are balanced by their own
  // plans (whole tiles, then a split tail). The 128-tile layers split their K
  // range so that every workgroup of the launch gets about the same number of
  // K steps: the layers of one call can differ by orders of magnitude in
  // B * T (a convolution's positions) and in output tiles, and a layer with
  // few output tiles but a long K range would otherwise run on a handful of
  // CUs.
  // The balance is per launch: layers of different kernel instances (vector
  // or element loads, weight on the accumulator or on the operand) run in
  // separate launches, one after the other, so each launch fills the GPU on
  // its own.
  const int cus = tr_cu_count();
  int tr_idx[kMaxLayersPerLaunch], n_tr = 0, wd_idx[kMaxLayersPerLaunch], n_wd = 0;
  int64_t work[4] = {0, 0, 0, 0};   // output tiles x K steps per 128-tile launch
  auto group = [](const dpsgd_layer& L) {
    const bool vec = L.dtype == DPSGD_BF16 ? tgemm_vec_ok<uint16_t>(L) : tgemm_vec_ok<float>(L);
    return (vec ? 0 : 1) + (clip_scale_mode(L) == SCALE_ACC ? 0 : 2);
  };
  for (int l = 0; l < n_layers; ++l) {
    const dpsgd_layer& L = layers[l];
    if (wide_tile_ok(L)) wd_idx[n_wd++] = l;
    else if (tr_tile_ok(L)) tr_idx[n_tr++] = l;
    else work[group(L)] += ceil_div(L.d_out, kTile) * ceil_div(L.d_in, kTile) *
                           clip_q_total(L, clip_scale_mode(L));
  }
  constexpr int64_t kMinStepsPerSplit = 4;
  constexpr int64_t kMaxSplits = 1024;
  const int64_t target = 4 * (int64_t)cus;   // workgroups per launch
  size_t off = 0;
  for (int l = 0; l < n_layers; ++l) {
    const dpsgd_layer& L = layers[l];
    int64_t s = 1;
    if (!wide_tile_ok(L) && !tr_tile_ok(L)) {
      const int64_t q_total = clip_q_total(L, clip_scale_mode(L));
      int64_t chunk = ceil_div(work[group(L)], target);
      if (chunk < kMinStepsPerSplit) chunk = kMinStepsPerSplit;
      s = ceil_div(q_total, chunk);
      if (s > q_total / kMinStepsPerSplit) s = q_total / kMinStepsPerSplit;
      if (s > kMaxSplits) s = kMaxSplits;
      if (s < 1) s = 1;
    }
    plan->splits[l] = (int)s;
    plan->partial_offset[l] = off;
    if (s > 1) off += round_up((size_t)s * (size_t)L.d_out * (size_t)L.d_in * sizeof(float), 256);
  }
  plan_tr_clip(layers, tr_idx, n_tr, cus, &plan->tr);
  plan_wide_clip(layers, wd_idx, n_wd, cus, &plan->wide);
  plan->tr_offset = off;
  plan->wide_offset = off + round_up(plan->tr.tail_bytes, 256);
  plan->partial_bytes = plan->wide_offset + round_up(plan->wide.tail_bytes, 256);
}

int launch_clip_sum(const dpsgd_layer* layers, int n_layers, const float* factors,
                    float* const* grads, int accumulate, float* partial_base, const ClipPlan& plan,
                    hipStream_t stream) {
  // Group layers by kernel variant; each group is one grouped launch.
  const bool bf16 = layers[0].dtype == DPSGD_BF16;
  int idx[6][kMaxLayersPerLaunch];
  float* outs[6][kMaxLayersPerLaunch];
  int spl[6][kMaxLayersPerLaunch];
  int acc[6][kMaxLayersPerLaunch];
  int cnt[6] = {0, 0, 0, 0, 0, 0};
  for (int l = 0; l < n_layers; ++l) {
    const dpsgd_layer& L = layers[l];
    const bool vec = bf16 ? tgemm_vec_ok<uint16_t>(L) : tgemm_vec_ok<float>(L);
    const int g = wide_tile_ok(L) ? 5
                  : tr_tile_ok(L) ? 4
                                  : (vec ? 0 : 1) + (clip_scale_mode(L) == SCALE_ACC ? 0 : 2);
    const int k = cnt[g]++;
    idx[g][k] = l;
    spl[g][k] = plan.splits[l];
    outs[g][k] = plan.splits[l] > 1
                     ? reinterpret_cast<float*>(reinterpret_cast<char*>(partial_base) +
                                                plan.partial_offset[l])
                     : grads[l];
    acc[g][k] = accumulate;
  }
  int st = DPSGD_OK;
  if (cnt[4])
    st = launch_tr_clip(layers, idx[4], cnt[4], factors, outs[4], accumulate, plan.tr,
                        reinterpret_cast<float*>(reinterpret_cast<char*>(partial_base) +
                                                 plan.tr_offset),
                        stream);
  if (st == DPSGD_OK && cnt[5])
    st = launch_wide_clip(layers, idx[5], cnt[5], factors, outs[5], accumulate, plan.wide,
                          reinterpret_cast<float*>(reinterpret_cast<char*>(partial_base) +
                                                   plan.wide_offset),
                          stream);
#define DPSGD_TG(T_, V_, S_, g_)                                                                \
  if (st == DPSGD_OK && cnt[g_])                                                               \
  st = launch_tgemm_group<T_, V_, S_, EPI_STORE>(layers, idx[g_], cnt[g_], factors, outs[g_], \
                                                 spl[g_], acc[g_], nullptr, nullptr, 0, stream)
  if (bf16) {
    DPSGD_TG(uint16_t, true, SCALE_ACC, 0);
    DPSGD_TG(uint16_t, false, SCALE_ACC, 1);
    DPSGD_TG(uint16_t, true, SCALE_OPERAND, 2);
    DPSGD_TG(uint16_t, false, SCALE_OPERAND, 3);
  } else {
    DPSGD_TG(float, true, SCALE_ACC, 0);
    DPSGD_TG(float, false, SCALE_ACC, 1);
    DPSGD_TG(float, true, SCALE_OPERAND, 2);
    DPSGD_TG(float, false, SCALE_OPERAND, 3);
  }
#undef DPSGD_TG
  if (st != DPSGD_OK) return st;

  // Split-K fix-up for the layers that were split.
  SplitArgs sargs{};
  int64_t wgs = 0;
  for (int l = 0; l < n_layers; ++l) {
    if (plan.splits[l] <= 1) continue;
    SplitEntry& E = sargs.L[sargs.n++];
    E.grad = grads[l];
    E.part = reinterpret_cast<const float*>(reinterpret_cast<const char*>(partial_base) +
                                            plan.partial_offset[l]);
    E.numel = layers[l].d_out * layers[l].d_in;
    E.splits = plan.splits[l];
    E.accumulate = accumulate;
    E.wg_begin = (uint32_t)wgs;
    E.vec = (aligned16(E.grad) && aligned16(E.part) && E.numel % 4 == 0) ? 1 : 0;
    wgs += ceil_div(E.numel, kSplitElemsPerWG);
  }
  if (sargs.n > 0) {
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL(split_reduce_kernel, dim3((uint32_t)wgs), dim3(kThreads), 0, stream, sargs);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

int launch_mat_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                     float* partials, int64_t P, hipStream_t stream) {
  const bool bf16 = layers[idx[0]].dtype == DPSGD_BF16;
  int iv[256], is[256], ib[256], nv = 0, ns = 0, nb = 0;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    const bool vec = bf16 ? tgemm_vec_ok<uint16_t>(L) : tgemm_vec_ok<float>(L);
    if (tr_tile_ok(L)) ib[nb++] = idx[k];
    else if (vec) iv[nv++] = idx[k];
    else is[ns++] = idx[k];
  }
  int st = DPSGD_OK;
  if (nb) st = launch_tr_mat_norms(layers, ib, nb, cols, partials, P, stream);
  if (st != DPSGD_OK) return st;
  if (bf16) {
    if (nv) st = launch_tgemm_group<uint16_t, true, SCALE_NONE, EPI_SUMSQ>(
                layers, iv, nv, nullptr, nullptr, nullptr, nullptr, cols, partials, P, stream);
    if (st == DPSGD_OK && ns) st = launch_tgemm_group<uint16_t, false, SCALE_NONE, EPI_SUMSQ>(
                layers, is, ns, nullptr, nullptr, nullptr, nullptr, cols, partials, P, stream);
  } else {
    if (nv) st = launch_tgemm_group<float, true, SCALE_NONE, EPI_SUMSQ>(
                layers, iv, nv, nullptr, nullptr, nullptr, nullptr, cols, partials, P, stream);
    if (st == DPSGD_OK && ns) st = launch_tgemm_group<float, false, SCALE_NONE, EPI_SUMSQ>(
                layers, is, ns, nullptr, nullptr, nullptr, nullptr, cols, partials, P, stream);
  }
  return st;
}

}  // namespace dpsgd
