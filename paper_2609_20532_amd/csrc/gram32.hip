// Gram-form per-example norms for float32 layers with short examples
// (T <= 64): the norm in Gram form of Section 2.2,
//
//   ||G_i^T A_i||_F^2 = sum_{t,s} (A_i A_i^T)[t][s] (G_i G_i^T)[t][s].
//
// With T <= 64 both Gram matrices fit one 64 x 64 tile, so an example costs
// 64 * 64 * (d_in + d_out) multiply-adds against 128 * 128 * T on the tiles of
// the materialised form (WRN-16-4's 8 x 8 feature maps: T = 64, d_in up to
// 2304, d_out = 256).
//
// One workgroup per example. The example's rows are streamed through LDS in
// 64-column slices (first the A columns, then the G columns) by direct
// 16-byte global-to-LDS copies into two slots (the next slice is copied
// while the current one is multiplied); rows past T are never copied and
// stay zero. Each of the four waves owns one 32 x 32 block
// of the 64 x 64 Gram and accumulates it with v_mfma_f32_32x32x2f32, whose
// operands are lane l's row l % 32 at k = l / 32: a transposed read of the
// row-major slice. Row t of a slice is stored rotated by t 16-byte units, so
// the 32 rows a half-wave reads at one column spread over the LDS banks. The
// A and G blocks sit in two accumulators with the same layout, so the
// element-wise product is formed in registers.
#include "lds_dma.h"
#include "mma.h"

namespace dpsgd {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kG64Rows = 64;                               // rows of the Gram tile (T <= 64)
constexpr int kG64Cols = 64;                               // d columns per slice
constexpr int kG64SliceFloats = kG64Rows * kG64Cols;       // 16 KB
constexpr int kG64Slots = 2;
constexpr int kG64Copies = kG64SliceFloats / 256 / 4;      // 1 KB copies per wave per slice (4)

struct G64Entry {
  const float* A;          // [B*T][d_in]
  const float* G;          // [B*T][d_out]
  int32_t d_in, d_out, T;
  uint32_t wg_begin;       // first workgroup (example 0) of this layer
  int32_t partial_col;     // partial slot of the layer
  int32_t pad;
};

struct G64Args {
  G64Entry L[kMaxLayersPerLaunch];
  int32_t n;
  float* partials;         // [B][P]
  int64_t P;
};

// Word offset of (row t, column k) inside a slice.
__device__ __forceinline__ int g64_word(int t, int k) {
  return t * kG64Cols + 4 * (((k >> 2) + t) & 15) + (k & 3);
}

__global__ __launch_bounds__(kThreads, 2) void gram64_kernel(G64Args args) {
  __shared__ __attribute__((aligned(16))) float lds[kG64Slots * kG64SliceFloats];
  __shared__ float red[4];

  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].wg_begin <= blockIdx.x) lo = mid; else hi = mid - 1;
  }
  const G64Entry& E = args.L[lo];
  const int64_t ex = blockIdx.x - E.wg_begin;
  const int T = E.T;
  const int na = E.d_in / kG64Cols, ns = na + E.d_out / kG64Cols;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = lane >> 5, c32 = lane & 31;
  const int bm = wave >> 1, bn = wave & 1;   // this wave's 32 x 32 block

  // Copy p of this wave moves 1 KB chunk c = wave + 4 p: rows 4c .. 4c + 3.
  // Lane i writes physical unit i % 16 of row 4c + i / 16, which holds the
  // row's logical columns 4 ((u - t) mod 16) .. +3. Rows past T copy nothing.
  uint32_t va[kG64Copies], vg[kG64Copies];
  uint32_t active = 0;
#pragma unroll
  for (int p = 0; p < kG64Copies; ++p) {
    const int c = wave + 4 * p;
    const int t = 4 * c + (lane >> 4), u = lane & 15;
    const int col = 4 * ((u - t) & 15);
    va[p] = (uint32_t)t * (uint32_t)E.d_in * 4u + (uint32_t)col * 4u;
    vg[p] = (uint32_t)t * (uint32_t)E.d_out * 4u + (uint32_t)col * 4u;
    if (t < T) active |= 1u << p;
  }
  const char* Ab = reinterpret_cast<const char*>(E.A + ex * T * (int64_t)E.d_in);
  const char* Gb = reinterpret_cast<const char*>(E.G + ex * T * (int64_t)E.d_out);
  const uint32_t lds0 = lds_address(lds);

  auto issue = [&](int s, int slot) {
    const bool is_a = s < na;
    const char* base = is_a ? Ab + (int64_t)s * kG64Cols * 4 : Gb + (int64_t)(s - na) * kG64Cols * 4;
#pragma unroll
    for (int p = 0; p < kG64Copies; ++p) {
      const int c = wave + 4 * p;
      const uint32_t la = __builtin_amdgcn_readfirstlane(
          lds0 + (uint32_t)slot * (kG64SliceFloats * 4) + 1024u * (uint32_t)c);
      if ((active >> p) & 1u) copy16_to_lds(base, is_a ? va[p] : vg[p], la);
    }
  };

  if (T < kG64Rows) {
    // Rows past T are never copied: clear the whole ring once.
    for (int i = threadIdx.x * 4; i < kG64Slots * kG64SliceFloats; i += kThreads * 4)
      *reinterpret_cast<float4*>(lds + i) = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();
  }

  f32x16_t acc_a, acc_g;
#pragma unroll
  for (int v = 0; v < 16; ++v) { acc_a[v] = 0.f; acc_g[v] = 0.f; }

  // Operand words of this lane: row 32 bm + l % 32 (first) and 32 bn + l % 32
  // (second) at k = 2 kp + l / 32.
  const int ta = 32 * bm + c32, tb = 32 * bn + c32;

  if (ns > 0) issue(0, 0);
  for (int s = 0; s < ns; ++s) {
    // Slice s is complete for this wave once nothing is outstanding (how many
    // copies a wave issues depends on T, so no partial count is used); the
    // barrier makes every wave's copies visible and guarantees that slice
    // s - 1, whose slot is refilled next, is no longer read.
    wait_vmcnt<0>();
    barrier_no_wait();
    if (s + 1 < ns) issue(s + 1, (s + 1) % kG64Slots);

    const float* S = lds + (s % kG64Slots) * kG64SliceFloats;
    if (s < na) {
#pragma unroll
      for (int kp = 0; kp < kG64Cols / 2; ++kp) {
        const int k = 2 * kp + h;
        acc_a = __builtin_amdgcn_mfma_f32_32x32x2f32(S[g64_word(ta, k)], S[g64_word(tb, k)], acc_a, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kp = 0; kp < kG64Cols / 2; ++kp) {
        const int k = 2 * kp + h;
        acc_g = __builtin_amdgcn_mfma_f32_32x32x2f32(S[g64_word(ta, k)], S[g64_word(tb, k)], acc_g, 0, 0, 0);
      }
    }
  }

  // Both accumulators hold the same (row, column) in each register, and rows
  // and columns past T are exactly 0.
  float v = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) v = fmaf(acc_a[i], acc_g[i], v);
  v = block_sum(v, red);
  if (threadIdx.x == 0) args.partials[ex * args.P + E.partial_col] = v;
}

}  // namespace

bool gram64_ok(const dpsgd_layer& L) {
  // 32-bit per-lane copy offsets: 64 rows of d * 4 bytes stay below 2^32.
  return L.dtype == DPSGD_F32 && L.T >= 2 && L.T <= kG64Rows && L.d_in % kG64Cols == 0 &&
         L.d_out % kG64Cols == 0 && L.d_in <= (INT64_C(1) << 24) && L.d_out <= (INT64_C(1) << 24);
}

int launch_gram64(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                  float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    G64Args args{};
    args.n = m;
    args.partials = partials;
    args.P = P;
    int64_t wgs = 0;
    for (int k = 0; k < m; ++k) {
      const int li = idx[base + k];
      const dpsgd_layer& L = layers[li];
      G64Entry& E = args.L[k];
      E.A = static_cast<const float*>(L.A);
      E.G = static_cast<const float*>(L.G);
      E.d_in = (int32_t)L.d_in;
      E.d_out = (int32_t)L.d_out;
      E.T = (int32_t)L.T;
      E.wg_begin = (uint32_t)wgs;
      E.partial_col = (int32_t)cols[li];
      wgs += L.B;
    }
    if (wgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL(gram64_kernel, dim3((uint32_t)wgs), dim3(kThreads), 0, stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

}  // namespace dpsgd
