// 256x256-tile transposed-operand MFMA GEMM for bf16 layers (clip-weighted sum
// and materialised norms), built on two CDNA4 features:
//
//  * global_load_lds_dwordx4: every K slice of G [k][m] and A [k][n] is copied
//    from HBM straight into LDS in its natural k-major layout, 16 bytes per
//    lane, with no VGPR staging and no ALU work. A four-slot ring of 32-row
//    slices keeps three slices in flight while the fourth is consumed.
//  * ds_read_b64_tr_b16: the MFMA operand (8 consecutive k of one row m) is read
//    transposed out of that k-major tile. Within a 16-lane group, lane d
//    receives element d % 4 of the 8-byte chunks addressed by lanes
//    4r + d/4, r = 0..3, so pointing lane s at X[k0 + s/4][m0 + 4(s%4)] hands
//    lane d the four values X[k0..k0+3][m0 + d].
//
// LDS layout of a slice: 32 rows of 512 bytes (256 bf16). A 32-byte segment
// sg of row k is stored at segment sg ^ f(k), f(k) = (k & 3) | ((k >> 1) & 4),
// so the 8 rows read together by one half-wave fall on 8 different 32-byte
// bank groups (conflict-free transposed reads). The direct loads apply the
// same permutation when choosing which global chunk each lane fetches.
//
// Eight wave64s per workgroup in a 2 x 4 grid own 128 x 64 sub-tiles; their
// accumulators (128 fp32 per lane) stay in ordinary VGPRs, so the clip weight
// can be applied exactly: the accumulator is kept in units of the current
// example's factor and multiplied by c_prev / c_next at each example boundary
// (paper: Section 2.2, g_bar_i = c_i g_i summed over the batch).
#include "mma.h"

namespace dpsgd {
namespace {

constexpr int kTrTile = 256;             // workgroup tile edge
constexpr int kTrBK = 32;                // k rows per slice
constexpr int kTrStages = 4;             // LDS ring slots
constexpr int kTrThreads = 512;          // 8 wave64s
constexpr int kTrRowBytes = kTrTile * 2; // 512
constexpr int kTrOpBytes = kTrBK * kTrRowBytes;       // 16 KB per operand slice
constexpr int kTrStageBytes = 2 * kTrOpBytes;         // G slice then A slice
constexpr int kTrLdsBytes = kTrStages * kTrStageBytes; // 128 KB

enum TrEpi : int { TR_STORE = 0, TR_SUMSQ = 1 };

struct TrEntry {
  const void* G;          // [B*T][M]
  const void* A;          // [B*T][N]
  float* out;             // STORE: grad (splits == 1) or split partials
  int32_t M, N, T;
  int32_t tiles_n;
  int32_t splits;
  int32_t q_per_split;    // K slices per split (STORE)
  uint32_t wg_begin;
  int32_t partial_col;    // SUMSQ
  int32_t accumulate;
  int32_t pad;
};
struct TrArgs {
  TrEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  const float* factors;
  float* partials;
  int64_t P;
};

__device__ __forceinline__ int seg_swizzle(int k) { return (k & 3) | ((k >> 1) & 4); }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef short v4i16_t __attribute__((ext_vector_type(4)));

// One 16-byte-per-lane copy from global memory into LDS at lds_addr + 16 * lane.
// Issued as inline assembly so the compiler does not treat later LDS reads as
// aliasing an in-flight copy (it would otherwise wait for every outstanding
// copy before each read); completion is tracked with explicit vmcnt waits.
__device__ __forceinline__ void copy16_to_lds(const void* gptr, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_addr)
               : "m0", "memory");
}

__device__ __forceinline__ bf16x8_t read_frag_tr(const char* lds_base, uint32_t off0, uint32_t off1) {
  typedef __attribute__((address_space(3))) v4i16_t lds_v4i16;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(lds_base + off0));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(lds_base + off1));
  typedef short v8i16_t __attribute__((ext_vector_type(8)));
  const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

template <int EPI>
__global__ __launch_bounds__(kTrThreads, 1) void tgemm_tr_kernel(TrArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[kTrLdsBytes];
  __shared__ float red[8];

  const uint32_t wgl = xcd_logical_index(blockIdx.x, gridDim.x);
  int l = 0;
  {
    int lo = 0, hi = args.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (args.L[mid].wg_begin <= wgl) lo = mid; else hi = mid - 1;
    }
    l = lo;
  }
  const TrEntry& E = args.L[l];
  const int M = E.M, N = E.N, T = E.T, B = args.B;
  const int tiles_n = E.tiles_n;
  const int tiles_mn = (M / kTrTile) * tiles_n;
  const uint32_t w = wgl - E.wg_begin;
  const int outer = (int)(w / (uint32_t)tiles_mn);   // split (STORE) or example (SUMSQ)
  const int tile = (int)(w % (uint32_t)tiles_mn);
  const int tm = tile / tiles_n, tn = tile % tiles_n;
  const int spe = T / kTrBK;                          // slices per example

  int64_t q0, q1;
  if (EPI == TR_SUMSQ) {
    q0 = (int64_t)outer * spe;
    q1 = q0 + spe;
  } else {
    const int64_t q_total = (int64_t)B * spe;
    q0 = (int64_t)outer * E.q_per_split;
    q1 = min(q0 + (int64_t)E.q_per_split, q_total);
  }

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;           // 2 x 4 waves: 128 x 64 each

  // ---- direct-load assignment: wave w fills row pairs w and w + 8 of both operands.
  const uint16_t* Gt = static_cast<const uint16_t*>(E.G) + tm * kTrTile;
  const uint16_t* At = static_cast<const uint16_t*>(E.A) + tn * kTrTile;
  int ld_k[2];          // row within the slice
  int ld_chunk[2];      // global 16-byte chunk (0..31) within the 256-wide row
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int k = 2 * (wave + 8 * p) + (lane >> 5);
    const int pos = lane & 31;
    ld_k[p] = k;
    ld_chunk[p] = 2 * (((pos >> 1) ^ seg_swizzle(k))) + (pos & 1);
  }

  // ---- transposed-read offsets (bytes within an operand slice), per half h.
  const int s = lane & 15, grp = lane >> 4;
  uint32_t offA[8][2], offB[4][2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = 8 * grp + 4 * h + (s >> 2);
    const int f = seg_swizzle(k);
    const int q = (s & 3) >> 1, half = (s & 1) * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int blk = wm * 8 + i;  // 16-wide block index along M
      offA[i][h] = k * kTrRowBytes + (2 * (blk ^ f) + q) * 16 + half;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int blk = wn * 4 + j;
      offB[j][h] = kTrOpBytes + k * kTrRowBytes + (2 * (blk ^ f) + q) * 16 + half;
    }
  }

  // LDS byte address of the ring (M0 holds LDS addresses for the copies).
  const uint32_t lds_addr0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto issue = [&](int64_t qq, int slot) {
    const int ex = (int)(qq / spe);
    const int ls = (int)(qq - (int64_t)ex * spe);
    const int64_t row0 = (int64_t)ex * T + ls * kTrBK;
    const uint32_t dst = lds_addr0 + (uint32_t)slot * kTrStageBytes;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int64_t row = row0 + ld_k[p];
      const uint32_t pair = wave_u + 8u * p;
      copy16_to_lds(Gt + row * M + ld_chunk[p] * 8, dst + pair * 1024u);
      copy16_to_lds(At + row * N + ld_chunk[p] * 8, dst + kTrOpBytes + pair * 1024u);
    }
  };

  // Clip factors through the scalar cache (constant address space): these loads
  // then never count against vmcnt, which tracks the slice copies.
  typedef __attribute__((address_space(4))) const float const_float;
  const const_float* fac = (const const_float*)args.factors;

  f32x4_t acc[8][4];
  zero_acc_t(acc);
  float c_cur = 1.0f;
  bool started = false;

  // Prologue: slices q0, q0+1, q0+2 in flight.
#pragma unroll
  for (int d = 0; d < kTrStages - 1; ++d)
    if (q0 + d < q1) issue(q0 + d, d);

  int ex = (int)(q0 / spe);
  int ls = (int)(q0 - (int64_t)ex * spe);
  for (int64_t q = q0; q < q1; ++q) {
    // This wave's loads of slice q are done once at most the later slices' loads
    // (4 instructions per slice) are outstanding; the barrier then makes every
    // wave's part visible and guarantees slice q-1 is no longer being read.
    const int64_t later = q1 - 1 - q;
    if (later >= 2) wait_vmcnt<8>();
    else if (later == 1) wait_vmcnt<4>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (q + kTrStages - 1 < q1) issue(q + kTrStages - 1, (int)((q - q0 + kTrStages - 1) % kTrStages));

    bool skip = false;
    if (EPI == TR_STORE && (ls == 0 || q == q0)) {
      const float c_new = fac[ex];
      if (c_new != 0.0f) {
        if (started && c_cur != c_new) scale_acc_t(acc, c_cur / c_new);
        c_cur = c_new;
        started = true;
      }
    }
    if (EPI == TR_STORE) skip = fac[ex] == 0.0f;  // example contributes nothing

    if (!skip) {
      const char* base = lds + (int)((q - q0) % kTrStages) * kTrStageBytes;
      bf16x8_t b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = read_frag_tr(base, offB[j][0], offB[j][1]);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bf16x8_t a = read_frag_tr(base, offA[i][0], offA[i][1]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[j], acc[i][j], 0, 0, 0);
      }
    }
    if (++ls == spe) { ls = 0; ++ex; }
  }

  if (EPI == TR_SUMSQ) {
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) sum = fmaf(acc[i][j][v], acc[i][j][v], sum);
    sum = wave_sum(sum);
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
      for (int k = 0; k < 8; ++k) t += red[k];
      args.partials[(int64_t)outer * args.P + E.partial_col + tile] = t;
    }
  } else {
    float* out = E.out + (E.splits > 1 ? (int64_t)outer * M * N : 0);
    const bool add = E.splits == 1 && E.accumulate;
    float* col0 = out + (int64_t)(tm * kTrTile + wm * 128 + 4 * (lane >> 4)) * N + tn * kTrTile +
                  wn * 64 + (lane & 15);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float* p = col0 + (int64_t)(i * 16 + v) * N;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float x = acc[i][j][v] * c_cur;
          p[j * 16] = add ? p[j * 16] + x : x;
        }
      }
  }
}

}  // namespace

bool tr_tile_ok(const dpsgd_layer& L) {
  return L.dtype == DPSGD_BF16 && L.d_in % kTrTile == 0 && L.d_out % kTrTile == 0 &&
         L.T % kTrBK == 0;
}

int64_t tr_q_total(const dpsgd_layer& L) { return L.B * (L.T / kTrBK); }

template <int EPI>
static int launch_tr_group(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                           float* const* outs, const int* splits, const int* accumulate,
                           const int64_t* cols, float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    TrArgs args{};
    args.n = m;
    args.B = (int32_t)layers[idx[base]].B;
    args.factors = factors;
    args.partials = partials;
    args.P = P;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const int li = idx[base + k];
      const dpsgd_layer& L = layers[li];
      TrEntry& E = args.L[k];
      E.G = L.G;
      E.A = L.A;
      E.M = (int32_t)L.d_out;
      E.N = (int32_t)L.d_in;
      E.T = (int32_t)L.T;
      E.tiles_n = (int32_t)(L.d_in / kTrTile);
      const int64_t tiles = (L.d_out / kTrTile) * E.tiles_n;
      E.wg_begin = (uint32_t)wgs;
      if (EPI == TR_STORE) {
        E.out = outs[base + k];
        E.splits = splits[base + k];
        E.q_per_split = (int32_t)ceil_div(tr_q_total(L), E.splits);
        E.accumulate = accumulate ? accumulate[base + k] : 0;
        wgs += tiles * E.splits;
      } else {
        E.partial_col = (int32_t)cols[li];
        wgs += tiles * L.B;
      }
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL(tgemm_tr_kernel<EPI>, dim3((uint32_t)wgs), dim3(kTrThreads), 0, stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

int launch_tr_clip(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                   float* const* outs, const int* splits, const int* accumulate,
                   hipStream_t stream) {
  return launch_tr_group<TR_STORE>(layers, idx, n, factors, outs, splits, accumulate, nullptr,
                                   nullptr, 0, stream);
}

int launch_tr_mat_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                        float* partials, int64_t P, hipStream_t stream) {
  return launch_tr_group<TR_SUMSQ>(layers, idx, n, nullptr, nullptr, nullptr, nullptr, cols,
                                   partials, P, stream);
}

}  // namespace dpsgd
