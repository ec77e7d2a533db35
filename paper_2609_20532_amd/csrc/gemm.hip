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
#include "lds_dma.h"
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

// ------------------------------------------- float32, k-major slices in LDS
//
// Float32 layers with T % 32 == 0 and both widths multiples of 4. A 32-row
// slice of both operands is copied to LDS unchanged, row-major [k][cols], by
// direct 16-byte global-to-LDS copies. v_mfma_f32_32x32x2f32 takes lane l's
// operand at row (first operand) or column (second) l % 32 and k = l / 32, so
// one wave reads 32 consecutive words of rows k and k + 1 per operand block:
// no transpose anywhere. Odd rows are stored rotated by 32 columns, so the two
// half-waves (rows k and k + 1, same columns) hit different LDS banks.
// The tile is 128 x 128 (2 x 2 waves) or, for d_out <= 64, 64 x 256 (1 x 4
// waves), so a narrow G side does not leave half of every tile empty; each
// wave owns 64 x 64 as 2 x 2 blocks of 32 x 32. Two slice buffers of up to
// 40 KB let two workgroups share a CU. Clip weights are applied on the
// accumulator (T % 32 == 0 makes every step lie inside one example); an
// example whose factor is 0 is neither copied nor multiplied.

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kK32Rows = 32;                                  // k rows per slice
constexpr int kK32StageFloats = kK32Rows * (64 + 256);        // largest slice (64 x 256 tile)
constexpr int kK32MaxCopies = kK32StageFloats / 256 / 4;      // 1 KB copies per wave (10)

struct K32Entry {
  const float* Xm;       // G: [B*T][M]
  const float* Xn;       // A: [B*T][N]
  float* out;            // EPI_STORE: grad (splits == 1) or this layer's split partials
  int32_t M, N, T;
  int32_t tm;            // tile rows (along M): 64 or 128
  int32_t tn;            // tile columns (along N): 256 or 128
  int32_t tiles_n;
  int32_t splits, q_per_split;
  uint32_t wg_begin;
  int32_t partial_col;   // EPI_SUMSQ
  int32_t accumulate;    // EPI_STORE, splits == 1
  int32_t ex_per_job;    // EPI_SUMSQ: consecutive examples of one job
};

struct K32Args {
  K32Entry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  const float* factors;
  float* partials;
  int64_t P;
};

template <int SCALE, int EPI>
__global__ __launch_bounds__(kThreads, 2) void tgemm_k32_kernel(K32Args args) {
  __shared__ __attribute__((aligned(16))) float lds[2 * kK32StageFloats];

  int l = 0;
  {
    int lo = 0, hi = args.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
    }
    l = lo;
  }
  const K32Entry& E = args.L[l];
  const int TM = E.tm, TN = E.tn;
  const int tiles_mn = ((E.M + TM - 1) / TM) * E.tiles_n;
  // Within a layer, consecutive jobs (the tiles of one K range) run on one XCD
  // and share its L2. All jobs of a layer cost the same, while layers differ
  // (a layer's K range per job can be 32 times another's), so every XCD takes
  // an equal share of each layer rather than a contiguous part of the grid.
  const int n_outer = EPI == EPI_SUMSQ ? (args.B + E.ex_per_job - 1) / E.ex_per_job : E.splits;
  const uint32_t n_l = (uint32_t)tiles_mn * (uint32_t)n_outer;
  const uint32_t w = xcd_two_class_index(blockIdx.x - E.wg_begin, n_l, n_l);
  const int outer = (int)(w / (uint32_t)tiles_mn);  // split (STORE) or example group (SUMSQ)
  const int tile = (int)(w % (uint32_t)tiles_mn);
  const int tmi = tile / E.tiles_n, tni = tile % E.tiles_n;

  const int spe = E.T / kK32Rows;
  int64_t q0, q1;
  if (EPI == EPI_SUMSQ) {
    // A job runs the copy pipeline across ex_per_job consecutive examples of
    // one tile, so a short T does not leave the workgroup mostly in its
    // prologue and epilogue.
    q0 = (int64_t)outer * E.ex_per_job * spe;
    q1 = (int64_t)min((outer + 1) * E.ex_per_job, args.B) * spe;
  } else {
    q0 = (int64_t)outer * E.q_per_split;
    q1 = min(q0 + (int64_t)E.q_per_split, (int64_t)args.B * spe);
  }

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wc = TN / 64;
  const int wm = wave / wc, wn = wave % wc;
  const int h = lane >> 5, c32 = lane & 31;

  // Clip factors through the scalar cache (constant address space), so they
  // never count against vmcnt, which tracks the slice copies.
  typedef __attribute__((address_space(4))) const float const_float;
  const const_float* fac = (const const_float*)args.factors;

  // Copy p of this wave moves 1 KB chunk c = wave + 4 p of the slice: chunks
  // [0, TM / 8) hold the G rows (TM columns each), the rest the A rows (TN
  // columns). Lane i writes words 4 i .. 4 i + 3 of its chunk; the source
  // column undoes the odd-row rotation and is clamped into the row (columns
  // past the edge feed only outputs that are never stored).
  const int nm = TM / 8, ncopy = (TM + TN) / 8;   // 1 KB chunks: G side, whole slice
  uint32_t voff[kK32MaxCopies];
  uint32_t inside = 0;   // bit p: copy p's columns lie inside the row
#pragma unroll
  for (int p = 0; p < kK32MaxCopies; ++p) {
    const int c = wave + 4 * p;
    const bool mside = c < nm;
    const int W = mside ? TM : TN, R = mside ? E.M : E.N;
    const int f = 256 * (mside ? c : c - nm) + 4 * lane;
    const int k = f / W, pc = f & (W - 1);
    const int col = ((mside ? tmi * TM : tni * TN) + ((pc + W - 32 * (k & 1)) & (W - 1)));
    voff[p] = (uint32_t)k * (uint32_t)R * 4u + (uint32_t)min(col, R - 4) * 4u;
    if (col < R) inside |= 1u << p;
  }
  const uint32_t lds0 = lds_address(lds);
  const char* Gb = reinterpret_cast<const char*>(E.Xm);
  const char* Ab = reinterpret_cast<const char*>(E.Xn);
  const int64_t gslice = (int64_t)kK32Rows * E.M * 4, aslice = (int64_t)kK32Rows * E.N * 4;

  auto issue = [&](int64_t qq, int slot) {
    if (SCALE == SCALE_ACC && fac[(int)(qq / spe)] == 0.0f) return;
    const char* gs = Gb + qq * gslice;
    const char* as = Ab + qq * aslice;
    const uint32_t dst = lds0 + (uint32_t)slot * (kK32StageFloats * 4);
#pragma unroll
    for (int p = 0; p < kK32MaxCopies; ++p) {
      const int c = wave + 4 * p;
      // For the norms, a lane whose columns lie past the edge copies nothing:
      // its LDS words keep the zeros written at the start, so rows and
      // columns outside the tile's valid part contribute exactly 0.
      // (The LDS address is made wave-uniform before the per-lane branch.)
      const uint32_t la = __builtin_amdgcn_readfirstlane(dst + 1024u * (uint32_t)c);
      if (c < ncopy && (EPI != EPI_SUMSQ || ((inside >> p) & 1u)))
        copy16_to_lds(c < nm ? gs : as, voff[p], la);
    }
  };

  // Operand words of this lane: row k = 2 kp + h of block a (G side) or b (A side).
  int offa[2], offb[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    offa[a] = h * TM + ((wm * 64 + 32 * a + 32 * h) & (TM - 1)) + c32;
    offb[a] = kK32Rows * TM + h * TN + ((wn * 64 + 32 * a + 32 * h) & (TN - 1)) + c32;
  }

  f32x16_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;
  float c_cur = 1.0f;    // accumulator unit (SCALE_ACC): acc * c_cur is the weighted sum
  bool started = false;

  // Output v of block (a, b) in this lane: row 8 (v / 4) + 4 h + v % 4 and
  // column l % 32 of the block.
  const int m_base = tmi * TM + wm * 64, n_base = tni * TN + wn * 64;

  if (EPI == EPI_SUMSQ && ((tmi + 1) * TM > E.M || (tni + 1) * TN > E.N)) {
    // Edge tile: clear both slice buffers once (see issue()).
    for (int i = threadIdx.x * 4; i < 2 * kK32StageFloats; i += kThreads * 4)
      *reinterpret_cast<float4*>(lds + i) = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();
  }
  if (q0 < q1) issue(q0, 0);
  for (int64_t q = q0; q < q1; ++q) {
    // Slice q is complete for this wave once none of its vector-memory
    // operations is outstanding (its copies, and a partial stored at the end
    // of the previous example); the barrier makes every wave's copies visible
    // and guarantees that slice q - 1, whose buffer is refilled next, is no
    // longer read.
    wait_vmcnt<0>();
    barrier_no_wait();
    if (q + 1 < q1) issue(q + 1, (int)((q + 1 - q0) & 1));
    bool skip = false;
    if (SCALE == SCALE_ACC) {
      const float c_new = fac[(int)(q / spe)];
      skip = c_new == 0.0f;
      if (!skip) {
        if (started && c_cur != c_new) {
          const float sc = c_cur / c_new;
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) acc[a][b] *= sc;
        }
        c_cur = c_new;
        started = true;
      }
    }
    if (skip) continue;
    // A wave whose 64 x 64 block lies wholly past the output's edge (the
    // last tile of a width that is not a multiple of the tile) has nothing
    // to multiply: its accumulators stay 0 and its SIMD serves the other
    // workgroup. It still takes part in the copies, barriers and partials.
    if (m_base < E.M && n_base < E.N) {
      const float* S = lds + (int)((q - q0) & 1) * kK32StageFloats;
      const float* pa0 = S + offa[0];
      const float* pa1 = S + offa[1];
      const float* pb0 = S + offb[0];
      const float* pb1 = S + offb[1];
#pragma unroll
      for (int kp = 0; kp < kK32Rows / 2; ++kp) {
        const float a0 = pa0[2 * kp * TM], a1 = pa1[2 * kp * TM];
        const float b0 = pb0[2 * kp * TN], b1 = pb1[2 * kp * TN];
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
      }
    }
    if (EPI == EPI_SUMSQ && (q + 1) % spe == 0) {
      // End of an example: this wave's share of ||G_i^T A_i||_F^2 over the
      // tile (entries past the edges are exactly 0), one partial per wave.
      float s = 0.f;
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            s = fmaf(acc[a][b][v], acc[a][b][v], s);
            acc[a][b][v] = 0.0f;
          }
      s = wave_sum(s);
      if (lane == 0)
        args.partials[(q / spe) * args.P + E.partial_col + 4 * tile + wave] = s;
    }
  }

  if (EPI == EPI_STORE) {
    float* out = E.out + (E.splits > 1 ? (int64_t)outer * E.M * E.N : 0);
    const bool add = E.splits == 1 && E.accumulate;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int n = n_base + 32 * b + c32;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int m = m_base + 32 * a + 8 * (v >> 2) + 4 * h + (v & 3);
          if (m < E.M && n < E.N) {
            float* p = out + (int64_t)m * E.N + n;
            const float r = SCALE == SCALE_ACC ? acc[a][b][v] * c_cur : acc[a][b][v];
            *p = add ? *p + r : r;
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

constexpr int kSplitElemsPerWG = kThreads * 4;  // one float4 per thread

// Adds the partials in split order. A layer can have tens of splits, so the
// loads of eight consecutive splits are issued before their adds (the order
// of the additions does not change) and each thread owns one float4, which
// gives enough workgroups to cover the GPU.
__global__ __launch_bounds__(kThreads) void split_reduce_kernel(SplitArgs args) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
  }
  const SplitEntry& E = args.L[lo];
  const int64_t e = (int64_t)(blockIdx.x - E.wg_begin) * kSplitElemsPerWG + (int64_t)threadIdx.x * 4;
  if (e >= E.numel) return;
  const int S = E.splits;
  if (E.vec) {
    float4 v = E.accumulate ? *reinterpret_cast<const float4*>(E.grad + e)
                            : make_float4(0.f, 0.f, 0.f, 0.f);
    const float* part = E.part + e;
    int s = 0;
    for (; s + 8 <= S; s += 8) {
      float4 p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) p[u] = *reinterpret_cast<const float4*>(part + (int64_t)(s + u) * E.numel);
#pragma unroll
      for (int u = 0; u < 8; ++u) { v.x += p[u].x; v.y += p[u].y; v.z += p[u].z; v.w += p[u].w; }
    }
    for (; s < S; ++s) {
      const float4 p = *reinterpret_cast<const float4*>(part + (int64_t)s * E.numel);
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    *reinterpret_cast<float4*>(E.grad + e) = v;
  } else {
    for (int k = 0; k < 4 && e + k < E.numel; ++k) {
      float v = E.accumulate ? E.grad[e + k] : 0.f;
      for (int s = 0; s < S; ++s) v += E.part[(int64_t)s * E.numel + e + k];
      E.grad[e + k] = v;
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

// ------------------------------------------------------ tiny layers (VALU)
//
// Layers with at most kTinyMaxOut entries in g_i = G_i^T A_i (a stem
// convolution's 16 x 27, a small head) would leave an MFMA tile almost empty,
// so each example's gradient is formed directly: its rows are staged in LDS a
// chunk at a time and thread t accumulates entries t and t + 256 of g_i in
// float32. The norm variant sums g_i's squares per example; the clip variant
// adds c_i g_i to the job's partial sum (an example with c_i = 0 is skipped,
// its rows are never read).

constexpr int kTinyMaxOut = 2 * kThreads;     // d_in * d_out
constexpr int kTinyLdsFloats = 16384;         // 64 KB of staged rows
constexpr int kTinyBatch = 16;                // loads in flight per thread while staging

struct TinyEntry {
  const void* A;          // [B*T][N]
  const void* G;          // [B*T][M]
  float* out;             // EPI_STORE: grad (one job) or this layer's per-job partials
  int32_t M, N, T;
  int32_t ex_per_job;
  int32_t jobs;
  uint32_t wg_begin;
  int32_t partial_col;    // EPI_SUMSQ
  int32_t accumulate;     // EPI_STORE, jobs == 1
};

struct TinyArgs {
  TinyEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  const float* factors;
  float* partials;
  int64_t P;
};

template <typename TIn, int EPI>
__global__ __launch_bounds__(kThreads) void tiny_kernel(TinyArgs args) {
  __shared__ float rows[kTinyLdsFloats];
  __shared__ float red[4];
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
  }
  const TinyEntry& E = args.L[lo];
  const int job = (int)(blockIdx.x - E.wg_begin);
  const int M = E.M, N = E.N, T = E.T, W = M + N;
  const int rc = kTinyLdsFloats / W;   // rows per chunk
  const TIn* A = static_cast<const TIn*>(E.A);
  const TIn* G = static_cast<const TIn*>(E.G);
  const int tid = threadIdx.x;
  const int n_out = M * N;
  const int o0 = tid, o1 = tid + kThreads;
  const int m0 = o0 / N, n0 = o0 - m0 * N, m1 = o1 / N, n1 = o1 - m1 * N;
  float sum0 = 0.f, sum1 = 0.f;   // EPI_STORE: sum over this job's examples of c_i g_i
  const int ex_begin = job * E.ex_per_job;
  const int ex_end = min(ex_begin + E.ex_per_job, args.B);
  for (int ex = ex_begin; ex < ex_end; ++ex) {
    const float c = EPI == EPI_STORE ? args.factors[ex] : 1.0f;
    if (EPI == EPI_STORE && c == 0.0f) continue;   // uniform over the workgroup
    float g0 = 0.f, g1 = 0.f;
    for (int r0 = 0; r0 < T; r0 += rc) {
      const int nr = min(rc, T - r0);
      const int64_t row = (int64_t)ex * T + r0;
      // Staged chunk: rows [r][0, M) hold G, [r][M, M + N) hold A.
      __syncthreads();   // the previous chunk is no longer read
      // kTinyBatch independent loads per thread, then their LDS stores, so the
      // staging waits for one memory latency per batch rather than per element.
      const int n_el = nr * W;
      for (int i0 = 0; i0 < n_el; i0 += kThreads * kTinyBatch) {
        float v[kTinyBatch];
#pragma unroll
        for (int u = 0; u < kTinyBatch; ++u) {
          const int i = i0 + u * kThreads + tid;
          v[u] = 0.f;
          if (i < n_el) {
            const int r = i / W, k = i - r * W;
            v[u] = k < M ? load_elem(G + (row + r) * M + k) : load_elem(A + (row + r) * N + (k - M));
          }
        }
#pragma unroll
        for (int u = 0; u < kTinyBatch; ++u) {
          const int i = i0 + u * kThreads + tid;
          if (i < n_el) rows[i] = v[u];
        }
      }
      __syncthreads();
      if (o0 < n_out)
        for (int r = 0; r < nr; ++r) g0 = fmaf(rows[r * W + m0], rows[r * W + M + n0], g0);
      if (o1 < n_out)
        for (int r = 0; r < nr; ++r) g1 = fmaf(rows[r * W + m1], rows[r * W + M + n1], g1);
    }
    if (EPI == EPI_SUMSQ) {
      const float s = block_sum(g0 * g0 + g1 * g1, red);
      if (tid == 0) args.partials[(int64_t)ex * args.P + E.partial_col] = s;
    } else {
      sum0 = fmaf(c, g0, sum0);
      sum1 = fmaf(c, g1, sum1);
    }
  }
  if (EPI == EPI_STORE) {
    float* out = E.out + (E.jobs > 1 ? (int64_t)job * n_out : 0);
    const bool add = E.jobs == 1 && E.accumulate;
    if (o0 < n_out) out[o0] = add ? out[o0] + sum0 : sum0;
    if (o1 < n_out) out[o1] = add ? out[o1] + sum1 : sum1;
  }
}

template <typename TIn, int EPI>
int launch_tiny_group(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                      float* const* outs, const int* jobs, const int* accumulate,
                      const int64_t* cols, float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    TinyArgs args{};
    args.n = m;
    args.B = (int32_t)layers[idx[base]].B;
    args.factors = factors;
    args.partials = partials;
    args.P = P;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const int li = idx[base + k];
      const dpsgd_layer& L = layers[li];
      TinyEntry& E = args.L[k];
      E.A = L.A;
      E.G = L.G;
      E.M = (int32_t)L.d_out;
      E.N = (int32_t)L.d_in;
      E.T = (int32_t)L.T;
      E.wg_begin = (uint32_t)wgs;
      if (EPI == EPI_STORE) {
        E.out = outs[base + k];
        E.jobs = jobs[base + k];
        E.accumulate = accumulate ? accumulate[base + k] : 0;
      } else {
        E.jobs = (int32_t)L.B;
        E.partial_col = (int32_t)cols[li];
      }
      // A job past the last example writes zeros, so the count may overshoot.
      E.ex_per_job = (int32_t)ceil_div(L.B, E.jobs);
      wgs += E.jobs;
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL((tiny_kernel<TIn, EPI>), dim3((uint32_t)wgs), dim3(kThreads), 0, stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

template <int SCALE, int EPI>
int launch_k32_group(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                     float* const* outs, const int* splits, const int* accumulate,
                     const int64_t* cols, float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    K32Args args{};
    args.n = m;
    args.B = (int32_t)layers[idx[base]].B;
    args.factors = factors;
    args.partials = partials;
    args.P = P;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const int li = idx[base + k];
      const dpsgd_layer& L = layers[li];
      K32Entry& E = args.L[k];
      E.Xm = static_cast<const float*>(L.G);
      E.Xn = static_cast<const float*>(L.A);
      E.M = (int32_t)L.d_out;
      E.N = (int32_t)L.d_in;
      E.T = (int32_t)L.T;
      E.tm = k32_tile_m(L);
      E.tn = k32_tile_n(L);
      E.tiles_n = (int32_t)ceil_div(L.d_in, E.tn);
      const int64_t tiles = ceil_div(L.d_out, E.tm) * E.tiles_n;
      E.wg_begin = (uint32_t)wgs;
      if (EPI == EPI_STORE) {
        E.out = outs[base + k];
        E.splits = splits[base + k];
        E.q_per_split = (int32_t)ceil_div(L.B * (L.T / kK32Rows), E.splits);
        E.accumulate = accumulate ? accumulate[base + k] : 0;
        wgs += tiles * E.splits;
      } else {
        E.partial_col = (int32_t)cols[li];
        E.ex_per_job = k32_ex_per_job(L);
        wgs += tiles * ceil_div(L.B, E.ex_per_job);
      }
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL((tgemm_k32_kernel<SCALE, EPI>), dim3((uint32_t)wgs), dim3(kThreads), 0,
                       stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

}  // namespace

bool k32_ok(const dpsgd_layer& L) {
  // The copies address a slice with 32-bit per-lane offsets: 32 rows of d * 4
  // bytes must stay below 2^32.
  return L.dtype == DPSGD_F32 && L.T % kK32Rows == 0 && L.d_in % 4 == 0 && L.d_out % 4 == 0 &&
         L.d_in <= (INT64_C(1) << 24) && L.d_out <= (INT64_C(1) << 24);
}
int k32_tile_m(const dpsgd_layer& L) { return L.d_out <= 64 ? 64 : 128; }
int k32_tile_n(const dpsgd_layer& L) { return L.d_out <= 64 ? 256 : 128; }
int k32_ex_per_job(const dpsgd_layer& L) {
  // About 16 K steps (512 rows) per materialised-norm job, at most 8 examples.
  const int64_t e = 16 / (L.T / kK32Rows);
  return (int)(e < 1 ? 1 : e > 8 ? 8 : e);
}
bool tiny_ok(const dpsgd_layer& L) { return L.d_in * L.d_out <= kTinyMaxOut; }
int tiny_jobs(const dpsgd_layer& L) {
  // About two workgroups per CU, each over ceil(B / jobs) consecutive examples.
  const int64_t want = L.B < 2 * (int64_t)tr_cu_count() ? L.B : 2 * (int64_t)tr_cu_count();
  return (int)ceil_div(L.B, ceil_div(L.B, want));
}
int64_t mat_tile_count(const dpsgd_layer& L) {
  if (tr_tile_ok(L)) return (L.d_out / 256) * (L.d_in / 256);
  if (k32_ok(L)) return ceil_div(L.d_out, k32_tile_m(L)) * ceil_div(L.d_in, k32_tile_n(L));
  return ceil_div(L.d_out, kTile) * ceil_div(L.d_in, kTile);
}

void plan_clip(const dpsgd_layer* layers, int n_layers, ClipPlan* plan) {
  // Layers on the 256- and 384x256-tile kernels are balanced by their own
  // plans (whole tiles, then a split tail). The 128-tile layers split their K
  // range so that every workgroup of the launch gets about the same number of
  // K steps: the layers of one call can differ by orders of magnitude in
  // B * T (a convolution's positions) and in output tiles, and a layer with
  // few output tiles but a long K range would otherwise run on a handful of
  // CUs.
  // The balance is per launch: layers of different kernel instances (vector
  // or element loads, weight on the accumulator or on the operand, k-major
  // float32) run in separate launches, one after the other, so each launch
  // fills the GPU on its own.
  const int cus = tr_cu_count();
  int tr_idx[kMaxLayersPerLaunch], n_tr = 0, wd_idx[kMaxLayersPerLaunch], n_wd = 0;
  // output tiles x K steps per launch: 128-tile variants 0..3, k-major float32 4
  int64_t work[5] = {0, 0, 0, 0, 0};
  auto group = [](const dpsgd_layer& L) {
    if (k32_ok(L)) return 4;
    const bool vec = L.dtype == DPSGD_BF16 ? tgemm_vec_ok<uint16_t>(L) : tgemm_vec_ok<float>(L);
    return (vec ? 0 : 1) + (clip_scale_mode(L) == SCALE_ACC ? 0 : 2);
  };
  // Layers on the 128-tile and k-major kernels (the others have their own plans).
  auto split_k = [](const dpsgd_layer& L) { return !wide_tile_ok(L) && !tr_tile_ok(L) && !tiny_ok(L); };
  for (int l = 0; l < n_layers; ++l) {
    const dpsgd_layer& L = layers[l];
    if (wide_tile_ok(L)) wd_idx[n_wd++] = l;
    else if (tr_tile_ok(L)) tr_idx[n_tr++] = l;
    else if (split_k(L)) work[group(L)] += mat_tile_count(L) * clip_q_total(L, clip_scale_mode(L));
  }
  constexpr int64_t kMinStepsPerSplit = 4;
  constexpr int64_t kMaxSplits = 1024;
  auto split_count = [](int64_t q_total, int64_t chunk) {
    int64_t s = ceil_div(q_total, chunk);
    if (s > q_total / kMinStepsPerSplit) s = q_total / kMinStepsPerSplit;
    if (s > kMaxSplits) s = kMaxSplits;
    return s < 1 ? (int64_t)1 : s;
  };
  // Both kernels hold two workgroups per CU. A launch runs in rounds of that
  // many workgroups, and a round that is only partly filled costs as much as
  // a full one, so the chunk (K steps per workgroup) is chosen per launch:
  // for r = 1 .. 8 rounds, the smallest chunk whose workgroups fit r rounds,
  // keeping the r with the least r x (longest workgroup in K steps).
  const int64_t slots = 2 * (int64_t)cus;
  int64_t chunk_of[5] = {1, 1, 1, 1, 1};
  for (int g = 0; g < 5; ++g) {
    if (work[g] == 0) continue;
    int64_t q_max = 1;
    for (int l = 0; l < n_layers; ++l)
      if (split_k(layers[l]) && group(layers[l]) == g) {
        const int64_t q = clip_q_total(layers[l], clip_scale_mode(layers[l]));
        if (q > q_max) q_max = q;
      }
    // Workgroups of the launch and its longest K range, for a given chunk.
    auto eval = [&](int64_t chunk, int64_t* longest) {
      int64_t wgs = 0, lg = 0;
      for (int l = 0; l < n_layers; ++l) {
        const dpsgd_layer& L = layers[l];
        if (!split_k(L) || group(L) != g) continue;
        const int64_t q = clip_q_total(L, clip_scale_mode(L));
        const int64_t sp = split_count(q, chunk);
        wgs += mat_tile_count(L) * sp;
        const int64_t len = ceil_div(q, sp);
        if (len > lg) lg = len;
      }
      if (longest) *longest = lg;
      return wgs;
    };
    int64_t best_chunk = q_max, best_cost = -1;
    for (int64_t r = 1; r <= 8; ++r) {
      if (eval(q_max, nullptr) > r * slots) continue;   // not even one split per layer fits
      int64_t lo = kMinStepsPerSplit < q_max ? kMinStepsPerSplit : q_max, hi = q_max;
      while (lo < hi) {   // smallest chunk with at most r rounds of workgroups
        const int64_t mid = (lo + hi) / 2;
        if (eval(mid, nullptr) <= r * slots) hi = mid; else lo = mid + 1;
      }
      int64_t longest = 0;
      eval(lo, &longest);
      const int64_t cost = r * longest;
      if (best_cost < 0 || cost < best_cost) { best_cost = cost; best_chunk = lo; }
    }
    chunk_of[g] = best_chunk;
  }
  size_t off = 0;
  for (int l = 0; l < n_layers; ++l) {
    const dpsgd_layer& L = layers[l];
    int64_t s = 1;
    if (split_k(L)) s = split_count(clip_q_total(L, clip_scale_mode(L)), chunk_of[group(L)]);
    else if (tiny_ok(L)) s = tiny_jobs(L);   // one partial per job of consecutive examples
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
  int idx[8][kMaxLayersPerLaunch];
  float* outs[8][kMaxLayersPerLaunch];
  int spl[8][kMaxLayersPerLaunch];
  int acc[8][kMaxLayersPerLaunch];
  int cnt[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int l = 0; l < n_layers; ++l) {
    const dpsgd_layer& L = layers[l];
    const bool vec = bf16 ? tgemm_vec_ok<uint16_t>(L) : tgemm_vec_ok<float>(L);
    const int g = wide_tile_ok(L) ? 5
                  : tr_tile_ok(L) ? 4
                  : tiny_ok(L)    ? 7
                  : k32_ok(L)     ? 6
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
  if (st == DPSGD_OK && cnt[6])
    st = launch_k32_group<SCALE_ACC, EPI_STORE>(layers, idx[6], cnt[6], factors, outs[6], spl[6],
                                                acc[6], nullptr, nullptr, 0, stream);
  if (st == DPSGD_OK && cnt[7])
    st = bf16 ? launch_tiny_group<uint16_t, EPI_STORE>(layers, idx[7], cnt[7], factors, outs[7], spl[7],
                                                       acc[7], nullptr, nullptr, 0, stream)
              : launch_tiny_group<float, EPI_STORE>(layers, idx[7], cnt[7], factors, outs[7], spl[7],
                                                    acc[7], nullptr, nullptr, 0, stream);
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
  int iv[256], is[256], ib[256], ik[256], it[256], nv = 0, ns = 0, nb = 0, nk = 0, nt = 0;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    const bool vec = bf16 ? tgemm_vec_ok<uint16_t>(L) : tgemm_vec_ok<float>(L);
    if (tr_tile_ok(L)) ib[nb++] = idx[k];
    else if (tiny_ok(L)) it[nt++] = idx[k];
    else if (k32_ok(L)) ik[nk++] = idx[k];
    else if (vec) iv[nv++] = idx[k];
    else is[ns++] = idx[k];
  }
  int st = DPSGD_OK;
  if (nb) st = launch_tr_mat_norms(layers, ib, nb, cols, partials, P, stream);
  if (st == DPSGD_OK && nk)
    st = launch_k32_group<SCALE_NONE, EPI_SUMSQ>(layers, ik, nk, nullptr, nullptr, nullptr, nullptr,
                                                 cols, partials, P, stream);
  if (st == DPSGD_OK && nt)
    st = bf16 ? launch_tiny_group<uint16_t, EPI_SUMSQ>(layers, it, nt, nullptr, nullptr, nullptr,
                                                       nullptr, cols, partials, P, stream)
              : launch_tiny_group<float, EPI_SUMSQ>(layers, it, nt, nullptr, nullptr, nullptr, nullptr,
                                                    cols, partials, P, stream);
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
