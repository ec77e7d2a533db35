// Per-example gradients of layers with a narrow side, formed in one pass over
// the inputs and stored.
//
// A low-rank adapter matrix (LoRA, the paper's fine-tuning experiments) is a
// linear layer whose d_in or d_out is the rank r. Its per-example gradient
// g_i = G_i^T A_i (Section 2.2) has d_in d_out elements, far fewer than the
// T (d_in + d_out) input elements it is formed from (GPT-2 adapters with r = 4
// and T = 128: 32 times fewer). For such layers one pass over A and G forms
// every g_i in float32 and stores it, the squared norm of Section 2.2 is summed
// from the stored values, and the clip-weighted sum sum_i c_i g_i reads the
// stored gradients instead of A and G a second time.
//
// Forming g_i: the wide side W (d_w = the larger of d_in, d_out) and the
// narrow side n (r <= 16 columns) of an example are row-aligned, and
// g_i = sum_t n_t (outer) W_t. One wave owns 64 V wide columns (V = 4 per
// lane: 16 bytes of float32 or 8 of bf16) and one range of rows, with r x V
// float32 sums per lane, and takes 16 rows per iteration (16 wide loads in
// flight per lane). Narrow values arrive 64 at a time, one per lane (lane L
// holds row L / R and column L % R of a group of 64 / R rows, R = r rounded
// up to 4, 8 or 16), and each is broadcast to the wave with v_readlane. When
// the examples and column chunks alone give too few waves, the rows are split
// into ranges whose partial gradients a second kernel adds in range order.
#include "common.h"

namespace dpsgd {
namespace {

constexpr int kSkWaves = kThreads / 64;   // independent waves per workgroup
static_assert(kSkWaves == 4, "the clip kernel adds four wave sums");

struct SkEntry {
  const void* wide;      // [B][T][d_w]
  const void* narrow;    // [B][T][r]
  float* store;          // [splits][B][d_out * d_in]: per-example gradients (range partials)
  int32_t T, d_w, r;
  int32_t narrow_is_a;   // 1: the narrow side is A (d_in = r), 0: it is G (d_out = r)
  int32_t chunks;        // wide-column chunks of 64 V
  int32_t splits;        // row ranges per example
  uint32_t job_begin;    // first job of this layer in the launch
  int32_t partial_col;   // first norm-partial column (one per chunk)
};

struct SkArgs {
  SkEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  int64_t P;
  float* partials;       // [B][P] norm partials
  uint32_t jobs;         // waves (grad kernel) or workgroups (finish kernel)
};

// V = 4 wide elements per lane and row, loaded as one 16-byte (float32) or
// 8-byte (bf16) access.
template <typename TIn, int V>
struct SkVec;
template <>
struct SkVec<float, 4> {
  typedef uint4 raw;
  __device__ static void cvt(const uint4& w, float (&f)[4]) {
    f[0] = __uint_as_float(w.x);
    f[1] = __uint_as_float(w.y);
    f[2] = __uint_as_float(w.z);
    f[3] = __uint_as_float(w.w);
  }
};
template <>
struct SkVec<uint16_t, 4> {
  typedef uint2 raw;
  __device__ static void cvt(const uint2& w, float (&f)[4]) {
    f[0] = bf16_lo(w.x);
    f[1] = bf16_hi(w.x);
    f[2] = bf16_lo(w.y);
    f[3] = bf16_hi(w.y);
  }
};

__device__ __forceinline__ float sk_load(const float* p) { return *p; }
__device__ __forceinline__ float sk_load(const uint16_t* p) { return bf16_to_f32(*p); }

__device__ __forceinline__ int sk_find_layer(const SkArgs& args, uint32_t job) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].job_begin <= job) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Job w of a layer: chunk w % chunks, example (w / chunks) % B, row range
// w / (chunks B).
template <typename TIn, int R, int V>
__global__ __launch_bounds__(kThreads) void skinny_grad_kernel(SkArgs args) {
  typedef typename SkVec<TIn, V>::raw Raw;
  constexpr int G = 64 / R;   // rows per narrow load
  constexpr int U = 16 / G > 1 ? 16 / G : 1;   // narrow loads per iteration
  constexpr int RI = G * U;   // rows per iteration: 16 wide loads in flight per lane
  // The wave index is read as a scalar, so the layer descriptor below is
  // read with scalar loads, and its fields are copied into registers before
  // the row loop (a field read inside the loop's conditional loads would be
  // reloaded there, each reload waiting for every load in flight).
  const uint32_t job = blockIdx.x * kSkWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (job >= args.jobs) return;   // whole waves
  const int lane = threadIdx.x & 63;
  const SkEntry& E = args.L[sk_find_layer(args, job)];
  const int64_t d_w = E.d_w, r = E.r;
  const int T = E.T;
  const uint32_t w = job - E.job_begin;
  const int chunk = (int)(w % (uint32_t)E.chunks);
  const uint32_t rest = w / (uint32_t)E.chunks;
  const int64_t i = rest % (uint32_t)args.B;
  const int s = (int)(rest / (uint32_t)args.B);
  const int t0 = (int)((int64_t)T * s / E.splits);
  const int t1 = (int)((int64_t)T * (s + 1) / E.splits);
  const int col = (chunk * 64 + lane) * V;
  const bool col_ok = col < d_w;
  const TIn* W = static_cast<const TIn*>(E.wide) + i * T * d_w + (col_ok ? col : 0);
  const TIn* Nr = static_cast<const TIn*>(E.narrow) + i * T * r;
  const int nrow = lane / R, ncol = lane % R;

  float acc[R][V];
#pragma unroll
  for (int j = 0; j < R; ++j)
#pragma unroll
    for (int v = 0; v < V; ++v) acc[j][v] = 0.f;

  for (int tg = t0; tg < t1; tg += RI) {
    const int rows = min(RI, t1 - tg);   // wave-uniform
    float nv[U];
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      nv[uu] = 0.f;
      if (ncol < r && uu * G + nrow < rows)
        nv[uu] = sk_load(Nr + (int64_t)(tg + uu * G + nrow) * r + ncol);
    }
    Raw wv[RI];
#pragma unroll
    for (int u = 0; u < RI; ++u) {
      wv[u] = Raw{};
      if (u < rows && col_ok) wv[u] = *reinterpret_cast<const Raw*>(W + (int64_t)(tg + u) * d_w);
    }
#pragma unroll
    for (int u = 0; u < RI; ++u) {
      if (u < rows) {   // wave-uniform
        float f[V];
        SkVec<TIn, V>::cvt(wv[u], f);
#pragma unroll
        for (int j = 0; j < R; ++j) {
          const float a = __int_as_float(
              __builtin_amdgcn_readlane(__float_as_int(nv[u / G]), (u % G) * R + j));
#pragma unroll
          for (int v = 0; v < V; ++v) acc[j][v] = fmaf(a, f[v], acc[j][v]);
        }
      }
    }
  }

  float* dst = E.store + ((int64_t)s * args.B + i) * ((int64_t)E.d_w * E.r);
  float sq = 0.f;
  if (col_ok) {
#pragma unroll
    for (int j = 0; j < R; ++j)
      if (j < E.r)
#pragma unroll
        for (int v = 0; v < V; ++v) sq = fmaf(acc[j][v], acc[j][v], sq);
    if (!E.narrow_is_a) {
      // Row j of the gradient holds this lane's V columns contiguously.
#pragma unroll
      for (int j = 0; j < R; ++j)
        if (j < E.r)
#pragma unroll
          for (int v = 0; v < V; v += 4)
            *reinterpret_cast<float4*>(dst + (int64_t)j * E.d_w + col + v) =
                make_float4(acc[j][v], acc[j][v + 1], acc[j][v + 2], acc[j][v + 3]);
    } else if (E.r == R) {
      // Rows col .. col + V - 1 of r = R values each: V R contiguous floats.
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int j = 0; j < R; j += 4)
          *reinterpret_cast<float4*>(dst + (int64_t)(col + v) * R + j) =
              make_float4(acc[j][v], acc[j + 1][v], acc[j + 2][v], acc[j + 3][v]);
    } else {
#pragma unroll
      for (int v = 0; v < V; ++v)
#pragma unroll
        for (int j = 0; j < R; ++j)
          if (j < E.r) dst[(int64_t)(col + v) * E.r + j] = acc[j][v];
    }
  }
  if (E.splits == 1) {
    sq = wave_sum(sq);
    if (lane == 0) args.partials[i * args.P + E.partial_col + chunk] = sq;
  }
}

// MFMA form for bfloat16 inputs whose wide side is a multiple of 8. The
// per-example gradient is the product N^T W over the rows (N the narrow
// side, W the wide side), which v_mfma_f32_16x16x32_bf16 takes 32 rows at a
// time (bf16 products are exact in float32, sums accumulate in float32, as on
// the VALU path). One wave owns 128 wide columns and one row range of one
// example. For rows t .. t + 31, lane l loads the 8 x 8 block of W at rows
// t + 8 (l / 16) .. +7 and columns 8 (l % 16) .. +7 (eight 16-byte loads)
// and transposes it in registers, so that operand j holds column
// 8 (l % 16) + j at those eight rows; its narrow operand holds column l % 16
// of N at the same rows (zero past r). MFMA j then gives g rows 0 .. 15 for
// the wide columns 8 n + j, n = 0 .. 15. Narrow columns past r and rows past
// the range are zero on input, so their outputs are zero. The next 32 rows'
// loads are issued before the current block is multiplied.
constexpr int kSkmCols = 128;   // wide columns per wave (and per norm chunk)

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t skm_bits(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  return __builtin_bit_cast(bf16x8_t, (u32x4_t{w0, w1, w2, w3}));
}

__global__ __launch_bounds__(kThreads) void skinny_mfma_kernel(SkArgs args) {
  // Scalar wave index and descriptor fields in registers, as in
  // skinny_grad_kernel.
  const uint32_t job = blockIdx.x * kSkWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (job >= args.jobs) return;   // whole waves
  const int lane = threadIdx.x & 63;
  const SkEntry& E = args.L[sk_find_layer(args, job)];
  const int64_t d_w = E.d_w, r = E.r;
  const int T = E.T;
  const uint32_t w = job - E.job_begin;
  const int chunk = (int)(w % (uint32_t)E.chunks);
  const uint32_t rest = w / (uint32_t)E.chunks;
  const int64_t i = rest % (uint32_t)args.B;
  const int s = (int)(rest / (uint32_t)args.B);
  const int t0 = (int)((int64_t)T * s / E.splits);
  const int t1 = (int)((int64_t)T * (s + 1) / E.splits);
  const int g = lane >> 4, cl = lane & 15;
  const int col = chunk * kSkmCols + 8 * cl;
  const bool col_ok = col < d_w;   // d_w % 8 == 0: all eight columns or none
  const uint16_t* W = static_cast<const uint16_t*>(E.wide) + i * T * d_w + (col_ok ? col : 0);
  const uint16_t* Nr = static_cast<const uint16_t*>(E.narrow) + i * T * r;
  const bool n_ok = cl < r;

  f32x4_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  uint4 wv[8];
  uint32_t nv[8];
  auto load = [&](int tg) {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int t = tg + 8 * g + kk;
      wv[kk] = uint4{0u, 0u, 0u, 0u};
      nv[kk] = 0u;
      if (t < t1) {
        if (col_ok) wv[kk] = *reinterpret_cast<const uint4*>(W + (int64_t)t * d_w);
        if (n_ok) nv[kk] = Nr[(int64_t)t * r + cl];
      }
    }
  };
  if (t0 < t1) load(t0);
  for (int tg = t0; tg < t1; tg += 32) {
    // Transpose the 8 x 8 block: word q of operand j packs rows 2q and
    // 2q + 1 of column j (the low halves of word j / 2 for even j, the high
    // halves for odd j).
    uint32_t c[8][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 x = wv[2 * q], y = wv[2 * q + 1];
      c[0][q] = __builtin_amdgcn_perm(y.x, x.x, 0x05040100u);
      c[1][q] = __builtin_amdgcn_perm(y.x, x.x, 0x07060302u);
      c[2][q] = __builtin_amdgcn_perm(y.y, x.y, 0x05040100u);
      c[3][q] = __builtin_amdgcn_perm(y.y, x.y, 0x07060302u);
      c[4][q] = __builtin_amdgcn_perm(y.z, x.z, 0x05040100u);
      c[5][q] = __builtin_amdgcn_perm(y.z, x.z, 0x07060302u);
      c[6][q] = __builtin_amdgcn_perm(y.w, x.w, 0x05040100u);
      c[7][q] = __builtin_amdgcn_perm(y.w, x.w, 0x07060302u);
    }
    const bf16x8_t a = skm_bits(nv[0] | (nv[1] << 16), nv[2] | (nv[3] << 16),
                                nv[4] | (nv[5] << 16), nv[6] | (nv[7] << 16));
    if (tg + 32 < t1) load(tg + 32);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          a, skm_bits(c[j][0], c[j][1], c[j][2], c[j][3]), acc[j], 0, 0, 0);
  }

  // Output v of MFMA j in lane l: g row m = 4 (l / 16) + v, wide column
  // chunk * 128 + 8 (l % 16) + j.
  float sq = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) sq = fmaf(acc[j][v], acc[j][v], sq);
  float* dst = E.store + ((int64_t)s * args.B + i) * ((int64_t)E.d_w * E.r);
  const int m0 = 4 * g;
  if (col_ok && m0 < E.r) {
    if (!E.narrow_is_a) {
      // g is [r][d_w]: row m holds this lane's eight columns contiguously.
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (m0 + v < E.r) {
          float* p = dst + (int64_t)(m0 + v) * E.d_w + col;
          *reinterpret_cast<float4*>(p) = make_float4(acc[0][v], acc[1][v], acc[2][v], acc[3][v]);
          *reinterpret_cast<float4*>(p + 4) = make_float4(acc[4][v], acc[5][v], acc[6][v], acc[7][v]);
        }
    } else if ((E.r & 3) == 0) {
      // g is [d_w][r]: rows m0 .. m0 + 3 of column c are four contiguous floats.
#pragma unroll
      for (int j = 0; j < 8; ++j)
        *reinterpret_cast<float4*>(dst + (int64_t)(col + j) * E.r + m0) =
            make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (m0 + v < E.r) dst[(int64_t)(col + j) * E.r + m0 + v] = acc[j][v];
    }
  }
  if (E.splits == 1) {
    sq = wave_sum(sq);
    if (lane == 0) args.partials[i * args.P + E.partial_col + chunk] = sq;
  }
}

// Layers with several row ranges: g_i = the ranges' partials added in range
// order, written over range 0, and its squared norm per chunk. One workgroup
// per (layer, example, chunk), numbered as the grad kernel's jobs with one
// range. A chunk's elements are one run of 64 V r floats when the narrow side
// is A (rows of r values) and r runs of 64 V floats when it is G; consecutive
// threads take consecutive groups of four floats (every run starts 16-byte
// aligned and holds a multiple of four).
template <int V>
__global__ __launch_bounds__(kThreads) void skinny_finish_kernel(SkArgs args) {
  __shared__ float red[kSkWaves];
  const uint32_t job = blockIdx.x;
  const SkEntry& E = args.L[sk_find_layer(args, job)];
  const uint32_t w = job - E.job_begin;
  const int chunk = (int)(w % (uint32_t)E.chunks);
  const int64_t i = w / (uint32_t)E.chunks;
  const int64_t per_ex = (int64_t)E.d_w * E.r;
  const int64_t per_split = (int64_t)args.B * per_ex;
  float* g = E.store + i * per_ex;
  const int c0 = chunk * 64 * V;
  const int cw = min(64 * V, E.d_w - c0);   // wide columns of this chunk
  const int64_t run_len = E.narrow_is_a ? (int64_t)cw * E.r : cw;
  const int64_t total = (E.narrow_is_a ? 1 : E.r) * run_len;
  float sq = 0.f;
#pragma unroll 2
  for (int64_t k = 4 * (int64_t)threadIdx.x; k < total; k += 4 * kThreads) {
    const int64_t run = k / run_len;
    const int64_t off = (E.narrow_is_a ? (int64_t)c0 * E.r : run * E.d_w + c0) + (k - run * run_len);
    float4 x = *reinterpret_cast<const float4*>(g + off);
    for (int sp = 1; sp < E.splits; ++sp) {
      const float4 y = *reinterpret_cast<const float4*>(g + sp * per_split + off);
      x.x += y.x;
      x.y += y.y;
      x.z += y.z;
      x.w += y.w;
    }
    *reinterpret_cast<float4*>(g + off) = x;
    sq = fmaf(x.x, x.x, sq);
    sq = fmaf(x.y, x.y, sq);
    sq = fmaf(x.z, x.z, sq);
    sq = fmaf(x.w, x.w, sq);
  }
  sq = block_sum(sq, red);
  if (threadIdx.x == 0) args.partials[i * args.P + E.partial_col + chunk] = sq;
}

// out[e] = (accumulate ? out[e] : 0) + sum_i c_i g_i[e]; examples with
// c_i == 0 add nothing. A workgroup owns 64 groups of four elements; wave w
// sums examples w, w + 4, w + 8, ... in order and the four wave sums are added
// as (w0 + w1) + (w2 + w3), a fixed order (results do not depend on timing).
struct SkClipEntry {
  const float* store;   // [B][n] per-example gradients
  float* out;
  int64_t n;            // d_out * d_in
  uint32_t wg_begin;
};
struct SkClipArgs {
  SkClipEntry L[kMaxLayersPerLaunch];
  int32_t n_layers;
  int32_t B;
  const float* factors;
  int32_t accumulate;
};

__global__ __launch_bounds__(kThreads) void skinny_clip_kernel(SkClipArgs args) {
  __shared__ float red[kSkWaves - 1][64][4];
  int lo = 0, hi = args.n_layers - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
  }
  const SkClipEntry& E = args.L[lo];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t e0 = ((int64_t)(blockIdx.x - E.wg_begin) * 64 + lane) * 4;
  const int cnt = e0 >= E.n ? 0 : (E.n - e0 < 4 ? (int)(E.n - e0) : 4);
  float sum[4] = {0.f, 0.f, 0.f, 0.f};
  if (cnt == 4 && (E.n & 3) == 0) {
    // Whole groups of a layer with n % 4 == 0: 16-byte loads (every example's
    // gradient starts 16-byte aligned), four examples in flight.
#pragma unroll 4
    for (int i = wave; i < args.B; i += kSkWaves) {
      const float c = args.factors[i];
      const float4 g = *reinterpret_cast<const float4*>(E.store + (int64_t)i * E.n + e0);
      if (c != 0.0f) {
        sum[0] = fmaf(c, g.x, sum[0]);
        sum[1] = fmaf(c, g.y, sum[1]);
        sum[2] = fmaf(c, g.z, sum[2]);
        sum[3] = fmaf(c, g.w, sum[3]);
      }
    }
  } else if (cnt > 0) {
    for (int i = wave; i < args.B; i += kSkWaves) {
      const float c = args.factors[i];
      if (c == 0.0f) continue;
      const float* g = E.store + (int64_t)i * E.n + e0;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q < cnt) sum[q] = fmaf(c, g[q], sum[q]);
    }
  }
  if (wave > 0)
#pragma unroll
    for (int q = 0; q < 4; ++q) red[wave - 1][lane][q] = sum[q];
  __syncthreads();
  if (wave == 0 && cnt > 0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < cnt) {
        const float v = (sum[q] + red[0][lane][q]) + (red[1][lane][q] + red[2][lane][q]);
        E.out[e0 + q] = args.accumulate ? E.out[e0 + q] + v : v;
      }
    }
  }
}

int64_t sk_rank(const dpsgd_layer& L) { return L.d_in <= L.d_out ? L.d_in : L.d_out; }
// Narrow side rounded up to the kernel's R.
int sk_rpad(const dpsgd_layer& L) { return sk_rank(L) <= 4 ? 4 : (sk_rank(L) <= 8 ? 8 : 16); }
// Wide elements per lane: four (16 bytes of float32, 8 of bf16). Chunks of
// 256 columns divide the usual model widths (768, 2304, 4096) exactly, and
// R x 4 accumulators leave room for four or more waves per SIMD.
int sk_vec(const dpsgd_layer& L) {
  (void)L;
  return 4;
}
int64_t sk_wide(const dpsgd_layer& L) { return L.d_in <= L.d_out ? L.d_out : L.d_in; }
double sk_grad_bytes(const dpsgd_layer& L) { return 4.0 * (double)L.d_in * (double)L.d_out; }
double sk_input_bytes(const dpsgd_layer& L) {
  return (double)L.T * (double)(L.d_in + L.d_out) * (L.dtype == DPSGD_BF16 ? 2.0 : 4.0);
}

template <typename TIn, int R, int V>
void launch_grad(const SkArgs& args, hipStream_t stream) {
  const uint32_t wgs = (args.jobs + kSkWaves - 1) / kSkWaves;
  hipLaunchKernelGGL((skinny_grad_kernel<TIn, R, V>), dim3(wgs), dim3(kThreads), 0, stream, args);
}

}  // namespace

bool skinny_ok(const dpsgd_layer& L) {
  if (sk_rank(L) > kSkinnyMaxRank) return false;
  // Lane column indices are 32-bit: keep the wide side well inside int32.
  if (sk_wide(L) % sk_vec(L) != 0 || sk_wide(L) > (INT64_C(1) << 30)) return false;
  // The stored gradients must be much smaller than the inputs they replace.
  return 4.0 * sk_grad_bytes(L) <= sk_input_bytes(L);
}

// bf16 layers whose wide side is a multiple of 8 take the MFMA kernel.
bool sk_mfma(const dpsgd_layer& L) { return L.dtype == DPSGD_BF16 && sk_wide(L) % 8 == 0; }

int64_t skinny_chunks(const dpsgd_layer& L) {
  return ceil_div(sk_wide(L), sk_mfma(L) ? kSkmCols : 64 * sk_vec(L));
}

void plan_skinny(const dpsgd_layer* layers, const int* idx, int n, int cus, int64_t* splits) {
  int64_t base = 0;
  for (int k = 0; k < n; ++k) base += layers[idx[k]].B * skinny_chunks(layers[idx[k]]);
  // Enough waves for about eight per CU, with at most 16 ranges, ranges of at
  // least 64 rows and range partials at most 1/4 of the layer's input bytes.
  int64_t target = 1;
  while (target < 16 && base * target < 8 * (int64_t)cus) target *= 2;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    int64_t s = 1;
    while (2 * s <= target && L.T / (2 * s) >= 64 &&
           4.0 * (double)(2 * s) * sk_grad_bytes(L) <= sk_input_bytes(L))
      s *= 2;
    splits[k] = s;
  }
}

size_t skinny_store_bytes(const dpsgd_layer& L, int64_t splits) {
  return round_up((size_t)splits * (size_t)L.B * (size_t)(L.d_in * L.d_out) * sizeof(float), 256);
}

// One pair of launches (grad, then finish when a layer has several row
// ranges) per class and per kMaxLayersPerLaunch layers: the MFMA class
// (class 0), then the VALU kernel's classes of padded rank R, which fix its R
// and V.
int launch_skinny_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                        const int64_t* splits, float* const* stores, float* partials, int64_t P,
                        hipStream_t stream) {
  if (n <= 0) return DPSGD_OK;
  const bool bf16 = layers[idx[0]].dtype == DPSGD_BF16;
  for (int R : {0, 4, 8, 16}) {
    int pos[kMaxLayersPerLaunch];
    int k0 = 0;
    while (k0 < n) {
      // The next up to kMaxLayersPerLaunch layers of this class.
      int m = 0;
      for (; k0 < n && m < kMaxLayersPerLaunch; ++k0) {
        const dpsgd_layer& L = layers[idx[k0]];
        if ((sk_mfma(L) ? 0 : sk_rpad(L)) == R) pos[m++] = k0;
      }
      if (m == 0) break;
      SkArgs ga{}, fa{};
      ga.n = fa.n = m;
      ga.B = fa.B = (int32_t)layers[idx[0]].B;
      ga.P = fa.P = P;
      ga.partials = fa.partials = partials;
      int64_t gjobs = 0, fjobs = 0;
      for (int k = 0; k < m; ++k) {
        const dpsgd_layer& L = layers[idx[pos[k]]];
        SkEntry E{};
        E.narrow_is_a = L.d_in <= L.d_out ? 1 : 0;
        E.wide = E.narrow_is_a ? L.G : L.A;
        E.narrow = E.narrow_is_a ? L.A : L.G;
        E.store = stores[pos[k]];
        E.T = (int32_t)L.T;
        E.d_w = (int32_t)sk_wide(L);
        E.r = (int32_t)sk_rank(L);
        E.chunks = (int32_t)skinny_chunks(L);
        E.splits = (int32_t)splits[pos[k]];
        E.partial_col = (int32_t)cols[idx[pos[k]]];
        ga.L[k] = E;
        fa.L[k] = E;
        ga.L[k].job_begin = (uint32_t)gjobs;
        fa.L[k].job_begin = (uint32_t)fjobs;
        gjobs += L.B * E.chunks * E.splits;
        // Layers with one range are finished by the grad kernel; the finish
        // kernel gives them no jobs (a layer with none starts where the next
        // one does and is never the one found for a job).
        if (E.splits > 1) fjobs += L.B * E.chunks;
      }
      if (gjobs > 0x7FFFFFFF || fjobs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
      ga.jobs = (uint32_t)gjobs;
      fa.jobs = (uint32_t)fjobs;
      if (R == 0) {
        hipLaunchKernelGGL(skinny_mfma_kernel, dim3((ga.jobs + kSkWaves - 1) / kSkWaves),
                           dim3(kThreads), 0, stream, ga);
      } else if (bf16) {
        if (R == 4) launch_grad<uint16_t, 4, 4>(ga, stream);
        else if (R == 8) launch_grad<uint16_t, 8, 4>(ga, stream);
        else launch_grad<uint16_t, 16, 4>(ga, stream);
      } else {
        if (R == 4) launch_grad<float, 4, 4>(ga, stream);
        else if (R == 8) launch_grad<float, 8, 4>(ga, stream);
        else launch_grad<float, 16, 4>(ga, stream);
      }
      if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
      if (fjobs > 0) {
        // Chunks of 64 V wide columns: 128 for the MFMA class, 256 otherwise.
        if (R == 0)
          hipLaunchKernelGGL(skinny_finish_kernel<kSkmCols / 64>, dim3(fa.jobs), dim3(kThreads), 0,
                             stream, fa);
        else
          hipLaunchKernelGGL(skinny_finish_kernel<4>, dim3(fa.jobs), dim3(kThreads), 0, stream, fa);
        if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
      }
    }
  }
  return DPSGD_OK;
}

int launch_skinny_clip(const dpsgd_layer* layers, const int* idx, int n, float* const* stores,
                       const float* factors, float* const* outs, int accumulate,
                       hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    SkClipArgs a{};
    a.n_layers = m;
    a.B = (int32_t)layers[idx[base]].B;
    a.factors = factors;
    a.accumulate = accumulate;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const dpsgd_layer& L = layers[idx[base + k]];
      SkClipEntry& E = a.L[k];
      E.store = stores[base + k];
      E.out = outs[base + k];
      E.n = L.d_in * L.d_out;
      E.wg_begin = (uint32_t)wgs;
      wgs += ceil_div(E.n, 4 * 64);
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL(skinny_clip_kernel, dim3((uint32_t)wgs), dim3(kThreads), 0, stream, a);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

}  // namespace dpsgd
