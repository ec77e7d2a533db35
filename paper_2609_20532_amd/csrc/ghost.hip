// Ghost-norm (Gram form) kernels for bf16 layers whose widths are multiples
// of 64 (paper: Section 2.2, per-example clipping by the L2 norm of g_i; the
// squared Frobenius norm of g_i = G_i^T A_i equals <A_i A_i^T, G_i G_i^T>_F).
//
// A workgroup owns one example i and one 128 x 128 tile (p, q), p <= q, of
// the T x T upper triangle (or, see below, three of them). It accumulates the
// activation Gram tile
//   GA[t][s] = sum_j A_i[128p + t][j] A_i[128q + s][j]   over the d_in columns
// and then the output-gradient Gram tile GG over the d_out columns, both in
// registers with the same layout, and returns sum_{t,s} GA[t][s] GG[t][s]
// (times 2 off the diagonal). Rows past T are read as a copy of the last row
// (in-bounds) and masked out of the sum.
//
// The contraction runs along the contiguous dimension of A and G, so the
// MFMA operand (8 consecutive columns of one row) is a plain 16-byte LDS
// read: slices of 32 columns of the p and q row blocks are copied from HBM
// straight into LDS (global_load_lds_dwordx4, a four-slot ring, three slices
// in flight) and multiplied with v_mfma_f32_32x32x16_bf16. In LDS a row takes
// 64 bytes and its 16-byte chunk c sits at slot c ^ ((row >> 2) & 3), which
// makes the 16-lane operand reads conflict-free; the copies choose which
// global chunk each lane fetches accordingly.
//
// The pass is close to HBM-bound: every element of A and G takes part in only
// 128 (or 256) multiply-adds per tile. When T spans two row blocks (128 < T <=
// 256) one workgroup owns all three tiles, (0, 0), (0, 1) and (1, 1), so each
// row of the example is fetched once: eight waves in a 2 x 4 grid each own a
// 64 x 32 piece of all three tiles, and slices are 64 columns wide (whole
// 128-byte lines). Otherwise every tile has its own four-wave workgroup (2 x 2
// grid of 64 x 64 sub-tiles, two workgroups per CU), and the tiles of one
// example run on one XCD so the rows they share come from its L2.
#include <algorithm>

#include "lds_dma.h"
#include "mma.h"

namespace dpsgd {
namespace {

constexpr int kGhRows = 128;                        // tile edge along T
constexpr int kGhBK = 32;                           // columns per slice
constexpr int kGhStages = 4;
constexpr int kGhThreads = 256;
constexpr int kGhBlockBytes = kGhRows * kGhBK * 2;  // 8 KB: one row block of a slice
constexpr int kGhStageBytes = 2 * kGhBlockBytes;    // p block, q block
constexpr int kGhLdsBytes = kGhStages * kGhStageBytes;

struct GhEntry {
  const void* A;
  const void* G;
  int32_t d_in, d_out, T;
  int32_t nt;          // 128-row tiles along T
  int32_t pairs;       // nt (nt + 1) / 2
  uint32_t wg_begin;   // first workgroup of this layer in the launch
  int32_t partial_col;
  int32_t groups;      // nt / 2 three-tile groups
  int32_t singles;     // pairs - 3 groups tiles outside them
  int32_t jpe;         // 256-row tiles: jobs per example of a launch without a split
  int32_t halves;      // 256-row tiles: off-diagonal tiles run as two row halves
};
struct GhArgs {
  GhEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int64_t P;
  float* partials;
};

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Position of tile (p, q), p <= q, in the row-major list of the upper triangle.
__host__ __device__ inline int pair_index(int nt, int p, int q) {
  return p * nt - p * (p - 1) / 2 + (q - p);
}
// Tile (p, q) belongs to the three-tile group of row blocks 0 and 1, which
// exists when T spans exactly two row blocks.
__host__ __device__ inline bool in_group(int nt, int p, int q) {
  return nt == 2 && p <= 1 && q <= 1;
}

// s_waitcnt vmcnt(per * min(later, 6)).
template <int PER>
__device__ __forceinline__ void wait_copies_upto6(int later) {
  switch (later < 6 ? later : 6) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<PER>(); break;
    case 2: wait_vmcnt<2 * PER>(); break;
    case 3: wait_vmcnt<3 * PER>(); break;
    case 4: wait_vmcnt<4 * PER>(); break;
    case 5: wait_vmcnt<5 * PER>(); break;
    default: wait_vmcnt<6 * PER>(); break;
  }
}

// sum_{t<rows_p, s<rows_q} GA[t][s] GG[t][s] of tile (p, q) of example i.
template <bool DIAG>
__device__ float ghost_tile(const GhEntry& E, int64_t i, int p, int q, char* lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int wm = wave >> 1, wn = wave & 1;
  const int T = E.T;
  const int rows_p = min(kGhRows, T - kGhRows * p);
  const int rows_q = min(kGhRows, T - kGhRows * q);
  const int nA = E.d_in / kGhBK, n = nA + E.d_out / kGhBK;
  const char* Ab = static_cast<const char*>(E.A) + i * (int64_t)T * E.d_in * 2;
  const char* Gb = static_cast<const char*>(E.G) + i * (int64_t)T * E.d_out * 2;
  const uint32_t lds0 = lds_address(lds);

  // Copy u of this wave moves rows 16 j .. 16 j + 15 (j = wave + 4 u) of a row
  // block: lane l takes row 16 j + l / 4 and the global chunk that belongs in
  // its slot l % 4.
  constexpr int kCopies = DIAG ? 2 : 4;  // per wave per slice
  uint32_t offA[kCopies], offG[kCopies];
#pragma unroll
  for (int u = 0; u < kCopies; ++u) {
    const int blk = u < 2 ? p : q;
    const int j = (int)wave_u + 4 * (u & 1);
    const int rvalid = u < 2 ? rows_p : rows_q;
    const int r = min(16 * j + (lane >> 2), rvalid - 1);
    const int row = kGhRows * blk + r;
    const int chunk = (lane & 3) ^ ((lane >> 4) & 3);
    offA[u] = (uint32_t)row * (uint32_t)E.d_in * 2u + 16u * chunk;
    offG[u] = (uint32_t)row * (uint32_t)E.d_out * 2u + 16u * chunk;
  }
  auto issue = [&](int s, int slot) {
    const bool a = s < nA;
    const char* src = a ? Ab + (int64_t)s * kGhBK * 2 : Gb + (int64_t)(s - nA) * kGhBK * 2;
    const uint32_t dst = lds0 + (uint32_t)slot * kGhStageBytes;
#pragma unroll
    for (int u = 0; u < kCopies; ++u) {
      const int j = (int)wave_u + 4 * (u & 1);
      copy16_to_lds(src, a ? offA[u] : offG[u], dst + (u < 2 ? 0u : (uint32_t)kGhBlockBytes) + 1024u * j);
    }
  };

  // Operand reads: lane l supplies row (l % 32) of a 32-row block and chunk
  // 2 st + l / 32 (k step st of the slice).
  const int f = (lane >> 2) & 3, g = lane >> 5;
  uint32_t rd[2];
#pragma unroll
  for (int st = 0; st < 2; ++st) rd[st] = (lane & 31) * 64 + 16 * ((2 * st + g) ^ f);
  const uint32_t rowA = 64 * wm * 64, rowB = (DIAG ? 0 : kGhBlockBytes) + 64 * wn * 64;

  f32x16_t accA[2][2], accG[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) accA[a][b] = accG[a][b] = f32x16_t{};

  // All waves must be done with the ring before a new tile overwrites it.
  __syncthreads();
#pragma unroll
  for (int d = 0; d < kGhStages - 1; ++d)
    if (d < n) issue(d, d);

  auto slice = [&](int s, f32x16_t (&acc)[2][2]) {
    // This wave's copies of slice s have landed once at most the later
    // slices' copies are outstanding; the barrier makes every wave's part
    // visible and guarantees slice s - 1, whose slot is refilled next, is no
    // longer read.
    const int later = n - 1 - s;
    if (later >= kGhStages - 2) wait_vmcnt<kCopies * (kGhStages - 2)>();
    else if (later == 1) wait_vmcnt<kCopies>();
    else wait_vmcnt<0>();
    barrier_no_wait();
    if (s + kGhStages - 1 < n) issue(s + kGhStages - 1, (s + kGhStages - 1) % kGhStages);
    typedef __attribute__((address_space(3))) const bf16x8_t lds_frag;
    const char* base = lds + (s % kGhStages) * kGhStageBytes;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      bf16x8_t fa[2], fb[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        fa[b] = *(lds_frag*)(base + rowA + 2048 * b + rd[st]);
        fb[b] = *(lds_frag*)(base + rowB + 2048 * b + rd[st]);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
  };
  for (int s = 0; s < nA; ++s) slice(s, accA);
  for (int s = nA; s < n; ++s) slice(s, accG);

  // Element v of block (a, b) in lane l: tile row 64 wm + 32 a + 8 (v / 4) +
  // 4 (l / 32) + v % 4, column 64 wn + 32 b + l % 32.
  float sum = 0.f;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = 64 * wn + 32 * b + (lane & 31);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = 64 * wm + 32 * a + 8 * (v >> 2) + 4 * g + (v & 3);
        const float x = accA[a][b][v] * accG[a][b][v];
        sum += (row < rows_p && col < rows_q) ? x : 0.f;
      }
    }
  return sum;
}

__global__ __launch_bounds__(kGhThreads, 2) void ghost_dma_kernel(GhArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[kGhLdsBytes];
  // Consecutive logical indices (the tiles of one example) run on one XCD, so
  // the rows that two tiles share are fetched from HBM into that XCD's L2 once.
  const uint32_t job = xcd_logical_index(blockIdx.x, gridDim.x);
  int l = 0;
  {
    int lo = 0, hi = args.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (args.L[mid].wg_begin <= job) lo = mid; else hi = mid - 1;
    }
    l = lo;
  }
  const GhEntry& E = args.L[l];
  const uint32_t w = job - E.wg_begin;
  // Jobs of a layer: example-major over the tiles outside the three-tile groups.
  const int64_t i = w / (uint32_t)E.singles;
  int single = (int)(w % (uint32_t)E.singles);
  int p = 0, q = 0;
  for (;; ++q) {
    if (q == E.nt) { ++p; q = p; }
    if (in_group(E.nt, p, q)) continue;
    if (single-- == 0) break;
  }
  const int pr = pair_index(E.nt, p, q);
  float s = p == q ? ghost_tile<true>(E, i, p, q, lds) : 2.0f * ghost_tile<false>(E, i, p, q, lds);
  s = wave_sum(s);
  __syncthreads();   // the ring is free again
  float* red = reinterpret_cast<float*>(lds);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = s;
  __syncthreads();
  if (threadIdx.x == 0)
    args.partials[i * args.P + E.partial_col + pr] = (red[0] + red[1]) + (red[2] + red[3]);
}

// ------------------------------------------------------- three-tile groups
//
// Slices of 64 columns: every row of a slice is one whole 128-byte line of A
// or G. In LDS a row takes 128 bytes and its 16-byte chunk c sits at slot
// c ^ ((row >> 1) & 7), which keeps the 16-lane operand reads conflict-free.

constexpr int kGgWaves = 8;                          // 4 column groups x kGgWavesM row groups
constexpr int kGgThreads = 64 * kGgWaves;
constexpr int kGgWavesM = kGgWaves / 4;
constexpr int kGgRB = kGhRows / 32 / kGgWavesM;     // 32-row blocks per wave
constexpr int kGgBK = 64;
constexpr int kGgStages = 4;
constexpr int kGgBlockBytes = kGhRows * kGgBK * 2;   // 16 KB: one row block of a slice
constexpr int kGgStageBytes = 2 * kGgBlockBytes;     // row blocks a = 2k and b = 2k + 1
constexpr int kGgLdsBytes = kGgStages * kGgStageBytes;

__global__ __launch_bounds__(kGgThreads, 1) void ghost_group_kernel(GhArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[kGgLdsBytes];
  // One job reads all rows of its (example, layer) and no job shares them, so
  // L2 locality does not matter here: the plain order deals every eighth
  // example of each layer to each XCD, which keeps the XCDs' work equal even
  // though the layers' widths differ.
  const uint32_t job = blockIdx.x;
  int l = 0;
  {
    int lo = 0, hi = args.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (args.L[mid].wg_begin <= job) lo = mid; else hi = mid - 1;
    }
    l = lo;
  }
  const GhEntry& E = args.L[l];
  const uint32_t w = job - E.wg_begin;
  const int64_t i = w / (uint32_t)E.groups;
  const int a = 2 * (int)(w % (uint32_t)E.groups), b = a + 1;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(wave);
  // The two diagonal tiles need only their 32 x 32 blocks on or above the
  // diagonal (row block <= column block; a block below it has the sum of its
  // mirror), which leaves more work to the right-hand column groups. Waves w
  // and w + 4 share a SIMD: pairing row group 0 with column group w % 4 and
  // row group 1 with column group 3 - w % 4 gives the SIMDs 10, 10, 8 and 8
  // blocks per k step instead of 6, 8, 10 and 12.
  static_assert(kGgWaves == 8 && kGgRB == 2, "the pairing assumes a 2 x 4 wave grid");
  const int wm = (int)(wave_u >> 2);
  const int wn = wm == 0 ? (int)(wave_u & 3u) : 3 - (int)(wave_u & 3u);
  const int T = E.T;
  const int rows_a = min(kGhRows, T - kGhRows * a);
  const int rows_b = min(kGhRows, T - kGhRows * b);
  const int nA = E.d_in / kGgBK, n = nA + E.d_out / kGgBK;
  const char* Ab = static_cast<const char*>(E.A) + i * (int64_t)T * E.d_in * 2;
  const char* Gb = static_cast<const char*>(E.G) + i * (int64_t)T * E.d_out * 2;
  const uint32_t lds0 = lds_address(lds);

  // Copy u of this wave moves rows 8 j .. 8 j + 7 (j = wave + waves u) of the
  // 256-row window of blocks a and b: lane l takes row 8 j + l / 8 and the
  // global chunk that belongs in its slot l % 8. Rows past T repeat the last
  // row (in-bounds; masked out of the sum).
  constexpr int kCopies = 32 / kGgWaves;
  uint32_t offA[kCopies], offG[kCopies];
#pragma unroll
  for (int u = 0; u < kCopies; ++u) {
    const int j = (int)wave_u + kGgWaves * u;
    const int row = min(kGhRows * a + 8 * j + (lane >> 3), T - 1);
    const int chunk = (lane & 7) ^ ((4 * (j & 1) + (lane >> 4)) & 7);
    offA[u] = (uint32_t)row * (uint32_t)E.d_in * 2u + 16u * chunk;
    offG[u] = (uint32_t)row * (uint32_t)E.d_out * 2u + 16u * chunk;
  }
  auto issue = [&](int s, int slot) {
    const bool isA = s < nA;
    const char* src = isA ? Ab + (int64_t)s * kGgBK * 2 : Gb + (int64_t)(s - nA) * kGgBK * 2;
    const uint32_t dst = lds0 + (uint32_t)slot * kGgStageBytes;
#pragma unroll
    for (int u = 0; u < kCopies; ++u)
      copy16_to_lds(src, isA ? offA[u] : offG[u], dst + 1024u * ((int)wave_u + kGgWaves * u));
  };

  // Operand reads: lane l supplies row (l % 32) of a 32-row block and chunk
  // 2 st + l / 32 of k step st (four per slice).
  const int f = (lane >> 1) & 7, g = lane >> 5;
  uint32_t rd[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) rd[st] = (lane & 31) * 128 + 16 * ((2 * st + g) ^ f);
  const uint32_t rowsA = 32 * kGgRB * wm * 128, rowsB = kGgBlockBytes + 32 * kGgRB * wm * 128;
  const uint32_t colA = 32 * wn * 128, colB = kGgBlockBytes + 32 * wn * 128;

  // Tiles t = 0: (a, a), 1: (a, b), 2: (b, b); each wave: rows 32 kGgRB wm ..
  // (kGgRB 32-row blocks r) and columns 32 wn .. +31 of every tile.
  f32x16_t accA[3][kGgRB], accG[3][kGgRB];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int r = 0; r < kGgRB; ++r) accA[t][r] = accG[t][r] = f32x16_t{};

#pragma unroll
  for (int d = 0; d < kGgStages - 1; ++d)
    if (d < n) issue(d, d);

  auto slice = [&](int s, f32x16_t (&acc)[3][kGgRB]) {
    // This wave's copies of slice s have landed once at most the later
    // slices' copies are outstanding; the barrier makes every wave's part
    // visible and guarantees slice s - 1, whose slot is refilled next, is no
    // longer read.
    const int later = n - 1 - s;
    if (later >= kGgStages - 2) wait_vmcnt<kCopies * (kGgStages - 2)>();
    else if (later == 1) wait_vmcnt<kCopies>();
    else wait_vmcnt<0>();
    barrier_no_wait();
    if (s + kGgStages - 1 < n) issue(s + kGgStages - 1, (s + kGgStages - 1) % kGgStages);
    typedef __attribute__((address_space(3))) const bf16x8_t lds_frag;
    const char* base = lds + (s % kGgStages) * kGgStageBytes;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      bf16x8_t fa[kGgRB], fb[kGgRB];
#pragma unroll
      for (int r = 0; r < kGgRB; ++r) {
        fa[r] = *(lds_frag*)(base + rowsA + 4096 * r + rd[st]);
        fb[r] = *(lds_frag*)(base + rowsB + 4096 * r + rd[st]);
      }
      const bf16x8_t ca = *(lds_frag*)(base + colA + rd[st]);
      const bf16x8_t cb = *(lds_frag*)(base + colB + rd[st]);
#pragma unroll
      for (int r = 0; r < kGgRB; ++r) {
        const bool upper = kGgRB * wm + r <= wn;   // wave-uniform
        if (upper) acc[0][r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[r], ca, acc[0][r], 0, 0, 0);
        acc[1][r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[r], cb, acc[1][r], 0, 0, 0);
        if (upper) acc[2][r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[r], cb, acc[2][r], 0, 0, 0);
      }
    }
  };
  for (int s = 0; s < nA; ++s) slice(s, accA);
  for (int s = nA; s < n; ++s) slice(s, accG);

  // Element v of block r in lane l: tile row 32 (kGgRB wm + r) + 8 (v / 4) +
  // 4 (l / 32) + v % 4, column 32 wn + l % 32.
  float sum[3] = {0.f, 0.f, 0.f};
  const int col = 32 * wn + (lane & 31);
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    const int rv = t == 2 ? rows_b : rows_a, cv = t == 0 ? rows_a : rows_b;
#pragma unroll
    for (int r = 0; r < kGgRB; ++r) {
      float blk = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = 32 * (kGgRB * wm + r) + 8 * (v >> 2) + 4 * g + (v & 3);
        const float x = accA[t][r][v] * accG[t][r][v];
        blk += (row < rv && col < cv) ? x : 0.f;
      }
      // Diagonal tiles: a block above the diagonal stands for itself and its
      // mirror; blocks below it were not computed.
      const int R = kGgRB * wm + r;
      const float wgt = t == 1 ? 1.f : (R < wn ? 2.f : (R == wn ? 1.f : 0.f));
      sum[t] += wgt * blk;
    }
    sum[t] = wave_sum(sum[t]);
  }
  __syncthreads();   // the ring is free again
  float* red = reinterpret_cast<float*>(lds);
  if (lane == 0)
#pragma unroll
    for (int t = 0; t < 3; ++t) red[3 * wave + t] = sum[t];
  __syncthreads();
  if (threadIdx.x < 3) {
    const int t = threadIdx.x;
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < kGgThreads / 64; ++k) v += red[3 * k + t];
    const int p = t == 2 ? b : a, q = t == 0 ? a : b;
    args.partials[i * args.P + E.partial_col + pair_index(E.nt, p, q)] = t == 1 ? 2.0f * v : v;
  }
}

// ------------------------------------------------------- 256-row tiles
//
// For T > 256 a workgroup owns one 256 x 256 tile (p, q), p <= q, of the upper
// triangle. Every row copied into LDS then takes part in 256 multiply-adds per
// column instead of 128, so a tile moves half the bytes per FLOP of the
// 128-row kernel above. The two float32 Gram tiles of a 256 x 256 tile
// (512 KB) would fill the whole register file; instead GA is accumulated
// first and each lane parks its accumulators in the workspace (written and
// read back only by that lane), GG reuses the same registers, and the lanes
// read GA back for the elementwise product. WAVES waves form a (WAVES / 2) x 2
// grid of sub-tiles of kMB x 4 blocks of 32 x 32: 64 x 128 for eight waves,
// 128 x 128 for four. A diagonal tile is symmetric, so its two sub-tiles
// below the 128-row diagonal are skipped and the two above it count twice;
// an off-diagonal tile may run as two jobs, one per 128-row half of block p
// (the four waves of that half multiply, all eight copy and synchronise).
// The loop is bound by LDS bandwidth, so what such a skipped sub-tile saves
// is mostly its operand reads. The grid is capped at
// kGhost256MaxGrid workgroups, each with a park slot of its own; workgroup b
// takes jobs b, b + grid, ... .

constexpr int kG4Rows = 256;
constexpr int kG4ParkFloats = kG4Rows * kG4Rows;   // per workgroup
constexpr int kG4BK = 64;                          // columns per slice
constexpr int kG4Waves = 8;

template <int BK, int WAVES>
struct G4Cfg {
  static constexpr int kThreads = 64 * WAVES;
  static constexpr int kMB = 2 * 8 / WAVES;                 // 32-row blocks per wave along p
  static constexpr int kNB = 4;                             // 32-row blocks per wave along q
  static constexpr int kRowBytes = 2 * BK;                  // one row of a slice
  static constexpr int kChunks = BK / 8;                    // 16-byte chunks per row
  static constexpr int kRowsPerCopy = 1024 / kRowBytes;     // rows per copy instruction
  static constexpr int kBlockBytes = kG4Rows * kRowBytes;   // one 256-row block of a slice
  static constexpr int kStageBytes = 2 * kBlockBytes;       // blocks p and q
  static constexpr int kStages = BK == 64 ? 2 : 4;
  static constexpr int kLdsBytes = kStages * kStageBytes;   // 128 KB
  static constexpr int kCopiesPerBlock = kG4Rows / kRowsPerCopy / WAVES;   // per wave
  static constexpr int kSteps = BK / 16;                    // MFMA k steps per slice
  static constexpr int kParkPerWave = kG4ParkFloats / WAVES;
  // LDS slot of chunk c of row r is c ^ swz(r): the 16-lane operand reads
  // (16 consecutive rows, one chunk) then touch 16 distinct 16-byte bank groups.
  __host__ __device__ static constexpr int swz(int r) {
    return BK == 64 ? ((r >> 1) & 7) : ((r >> 2) & 3);
  }
};

// split == 1: job = tile; park holds kG4ParkFloats per workgroup of the grid.
// split > 1: job = (tile, part), part p taking slices [n p / split,
// n (p + 1) / split) of the tile's n = (d_in + d_out) / 64 column slices (A's
// first, then G's); park holds two slots of kG4ParkFloats per job (its
// partial GA, masked to the tile's valid rows and columns, and its partial
// GG), which ghost256_combine_kernel adds and multiplies.
struct G4Args {
  GhEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t split;
  uint32_t jobs;
  int64_t P;
  float* partials;
  float* park;
};

// This wave's part of sum_{t<rows_p, s<rows_q} GA[t][s] GG[t][s] over 256 x 256
// tile (p, q) of example i: the sum over its sub-tile, doubled when the wave
// is in w2_mask, 0 when it is not in act_mask; park is a kG4ParkFloats scratch
// slot of this workgroup. SPLIT: the column slices [s_lo, s_hi) (A's slices
// first, then G's) are part of the tile and every wave takes part; the
// partial GA (masked) goes to park_a and the partial GG to park_g instead,
// and the result is 0.
template <int BK, int WAVES, bool DIAG, bool SPLIT>
__device__ float ghost_tile256(const GhEntry& E, int64_t i, int p, int q, char* lds, float* park,
                               int s_lo_arg, int s_hi_arg, float* park_a, float* park_g,
                               uint32_t act_mask, uint32_t w2_mask) {
  using C = G4Cfg<BK, WAVES>;
  constexpr int MB = C::kMB, NB = C::kNB;
  const int lane = threadIdx.x & 63;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // A wave outside act_mask still copies and takes part in every barrier but
  // reads no operands and multiplies nothing (its sub-tile adds 0).
  const bool active = SPLIT || ((act_mask >> wave_u) & 1u) != 0u;
  const int wm = (int)(wave_u >> 1), wn = (int)(wave_u & 1u);
  const int T = E.T;
  const int rows_p = min(kG4Rows, T - kG4Rows * p);
  const int rows_q = min(kG4Rows, T - kG4Rows * q);
  const int nA = E.d_in / BK, n = nA + E.d_out / BK;
  // A whole tile runs every slice (bounds known to the compiler).
  const int s_lo = SPLIT ? s_lo_arg : 0, s_hi = SPLIT ? s_hi_arg : n;
  const char* Ab = static_cast<const char*>(E.A) + i * (int64_t)T * E.d_in * 2;
  const char* Gb = static_cast<const char*>(E.G) + i * (int64_t)T * E.d_out * 2;
  const uint32_t lds0 = lds_address(lds);

  // Copy u of this wave fills the kRowsPerCopy rows starting at kRowsPerCopy j
  // (j = wave + WAVES (u % kPer)) of block p (u < kPer) or block q: lane l
  // takes row kRowsPerCopy j + l / kChunks and the global chunk that belongs
  // in its slot l % kChunks. The slot swizzle of that row does not depend on
  // u (kRowsPerCopy WAVES is a multiple of the swizzle period), so a lane's
  // chunk is fixed; its row is clamped to the block's last valid row (rows
  // past T repeat it, in bounds, and are masked out of the sum).
  constexpr int kPer = C::kCopiesPerBlock;
  constexpr int kCopies = DIAG ? kPer : 2 * kPer;
  static_assert((C::kRowsPerCopy * WAVES) % 16 == 0, "both swizzles repeat every 16 rows");
  const int r0 = C::kRowsPerCopy * (int)wave_u + lane / C::kChunks;   // row of copy u = 0
  const uint32_t chunk16 = 16u * (uint32_t)((lane % C::kChunks) ^ C::swz(r0));
  auto issue = [&](int s, int slot) {
    const bool a = s < nA;
    const char* src = a ? Ab + (int64_t)s * BK * 2 : Gb + (int64_t)(s - nA) * BK * 2;
    const uint32_t stride = (uint32_t)(a ? E.d_in : E.d_out) * 2u;
    const uint32_t dst = lds0 + (uint32_t)slot * C::kStageBytes;
#pragma unroll
    for (int u = 0; u < kCopies; ++u) {
      const bool second = u >= kPer;
      const int r = r0 + C::kRowsPerCopy * WAVES * (u % kPer);
      const int row = kG4Rows * (second ? q : p) + min(r, (second ? rows_q : rows_p) - 1);
      const uint32_t dst_off = (second ? (uint32_t)C::kBlockBytes : 0u) +
                               1024u * ((uint32_t)wave_u + WAVES * (u % kPer));
      copy16_to_lds(src, (uint32_t)row * stride + chunk16, dst + dst_off);
    }
  };

  // Operand reads: lane l supplies row (l % 32) of a 32-row block and chunk
  // 2 st + l / 32 of k step st.
  const int g = lane >> 5;
  uint32_t rd[C::kSteps];
#pragma unroll
  for (int st = 0; st < C::kSteps; ++st)
    rd[st] = (uint32_t)((lane & 31) * C::kRowBytes + 16 * ((2 * st + g) ^ C::swz(lane & 31)));
  const uint32_t rowA = (uint32_t)(32 * MB * wm * C::kRowBytes);
  const uint32_t rowB = (DIAG ? 0u : (uint32_t)C::kBlockBytes) + (uint32_t)(32 * NB * wn * C::kRowBytes);

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = f32x16_t{};

  // All waves must be done with the ring (and the previous job's reduction
  // slots) before this tile overwrites it.
  __syncthreads();
#pragma unroll
  for (int d = 0; d < C::kStages - 1; ++d)
    if (s_lo + d < s_hi) issue(s_lo + d, d);

  auto slice = [&](int s) {
    // This wave's copies of slice s have landed once at most the later
    // slices' copies are outstanding (at the first GG slice the park stores
    // are outstanding too, so that wait is for everything); the barrier makes
    // every wave's part visible and guarantees slice s - 1, whose slot is
    // refilled next, is no longer read.
    const int later = s_hi - 1 - s;
    if (s == nA) wait_vmcnt<0>();
    else if (later >= C::kStages - 2) wait_vmcnt<kCopies * (C::kStages - 2)>();
    else if (later == 1) wait_vmcnt<kCopies>();
    else wait_vmcnt<0>();
    barrier_no_wait();
    if (s + C::kStages - 1 < s_hi)
      issue(s + C::kStages - 1, (s - s_lo + C::kStages - 1) % C::kStages);
    if (!active) return;
    typedef __attribute__((address_space(3))) const bf16x8_t lds_frag;
    const char* base = lds + ((s - s_lo) % C::kStages) * C::kStageBytes;
    // Operands of k step st + 1 are read while the MFMAs of step st run; the
    // scheduling barrier keeps the reads of later steps from being hoisted
    // further (which would hold every step's operands in registers at once).
    bf16x8_t fa[2][MB], fb[2][NB];
    auto load = [&](int st, int buf) {
#pragma unroll
      for (int a = 0; a < MB; ++a) fa[buf][a] = *(lds_frag*)(base + rowA + 32 * a * C::kRowBytes + rd[st]);
#pragma unroll
      for (int b = 0; b < NB; ++b) fb[buf][b] = *(lds_frag*)(base + rowB + 32 * b * C::kRowBytes + rd[st]);
    };
    load(0, 0);
#pragma unroll
    for (int st = 0; st < C::kSteps; ++st) {
      if (st + 1 < C::kSteps) load(st + 1, (st + 1) & 1);
#pragma unroll
      for (int a = 0; a < MB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[st & 1][a], fb[st & 1][b], acc[a][b], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Park slot of this lane: float4 k (k = 4 (NB a + b) + c holds elements
  // 4 c .. 4 c + 3 of block (a, b)) at float offset kParkPerWave wave + 256 k +
  // 4 lane, so every store and load instruction covers 1 KB contiguously.
  // Element v of block (a, b) in lane l: tile row 32 (MB wm + a) + 8 (v / 4) +
  // 4 (l / 32) + v % 4, column 32 (NB wn + b) + l % 32.
  const int lane_off = C::kParkPerWave * (int)wave_u + 4 * lane;
  auto park_acc = [&](float* dst, bool masked) {
#pragma unroll
    for (int a = 0; a < MB; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int col = 32 * (NB * wn + b) + (lane & 31);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          f32x4_t v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = 32 * (MB * wm + a) + 8 * c + 4 * g + e;
            const float x = acc[a][b][4 * c + e];
            v4[e] = !masked || (row < rows_p && col < rows_q) ? x : 0.f;
          }
          *reinterpret_cast<f32x4_t*>(dst + lane_off + 256 * (4 * (NB * a + b) + c)) = v4;
        }
        acc[a][b] = f32x16_t{};
        __builtin_amdgcn_sched_barrier(0);   // one block's values in flight at a time
      }
  };
  const int a_end = min(s_hi, nA);
  for (int s = s_lo; s < a_end; ++s) slice(s);
  if (s_lo < nA && active) park_acc(SPLIT ? park_a : park, SPLIT);
  for (int s = max(s_lo, nA); s < s_hi; ++s) slice(s);
  if constexpr (SPLIT) {
    if (s_hi > nA) park_acc(park_g, false);
    return 0.f;
  }
  if (!active) return 0.f;
  float* mine = park + lane_off;

  // Element v of block (a, b) in lane l: tile row 32 (MB wm + a) + 8 (v / 4) +
  // 4 (l / 32) + v % 4, column 32 (NB wn + b) + l % 32. A diagonal tile is
  // computed whole, so its sum is the plain sum over the tile as well.
  float sum = 0.f;
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      f32x4_t ga[4];
#pragma unroll
      for (int c = 0; c < 4; ++c)
        ga[c] = *reinterpret_cast<const f32x4_t*>(mine + 256 * (4 * (NB * a + b) + c));
      const int col = 32 * (NB * wn + b) + (lane & 31);
      float blk = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = 32 * (MB * wm + a) + 8 * (v >> 2) + 4 * g + (v & 3);
        const float x = ga[v >> 2][v & 3] * acc[a][b][v];
        blk += (row < rows_p && col < rows_q) ? x : 0.f;
      }
      sum += blk;
      __builtin_amdgcn_sched_barrier(0);   // one block's parked values in flight at a time
    }
  return ((w2_mask >> wave_u) & 1u) ? 2.0f * sum : sum;
}

// Layer of a job (the last layer starting at or before it).
__device__ __forceinline__ int g4_find_layer(const G4Args& args, uint32_t job) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].wg_begin <= job) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Tile pr of the upper triangle of an nt x nt block grid (row-major order).
__device__ __forceinline__ void g4_tile_pq(int nt, int pr, int& p, int& q) {
  p = 0;
  while (pr >= nt - p) {
    pr -= nt - p;
    ++p;
  }
  q = p + pr;
}

// Off-diagonal tile o (row-major over p < q) of an nt x nt block grid, and
// the inverse.
__device__ __forceinline__ void g4_off_pq(int nt, int o, int& p, int& q) {
  p = 0;
  while (o >= nt - 1 - p) {
    o -= nt - 1 - p;
    ++p;
  }
  q = p + 1 + o;
}
__device__ __forceinline__ int g4_off_index(int nt, int p, int q) {
  return p * (nt - 1) - p * (p - 1) / 2 + (q - p - 1);
}

// Waves of a diagonal tile: sub-tiles (wm, wn) = (wave / 2, wave % 2) cover
// rows 64 wm .. +63 and columns 128 wn .. +127. The tile is symmetric: the two
// sub-tiles below its 128-row diagonal (waves 4, 6) are skipped and the two
// above it (waves 1, 3) count twice.
constexpr uint32_t kG4DiagAct = 0xAFu, kG4DiagW2 = 0x0Au;

// SPLIT: the launch's tiles are split into args.split parts (a separate
// instantiation, so that the whole-tile kernel's code is not shared with it).
template <int BK, int WAVES, bool SPLIT>
__global__ __launch_bounds__(64 * WAVES, 1) void ghost_tile256_kernel(G4Args args) {
  __shared__ __attribute__((aligned(1024))) char lds[G4Cfg<BK, WAVES>::kLdsBytes];
  float* park = args.park + (size_t)blockIdx.x * kG4ParkFloats;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int S = SPLIT ? args.split : 1;
  // Consecutive logical indices (the tiles of one example, and the parts of
  // one tile) run on one XCD, so the rows that they share are fetched from HBM
  // into that XCD's L2 once.
  for (uint32_t job = xcd_logical_index(blockIdx.x, gridDim.x); job < args.jobs; job += gridDim.x) {
    const GhEntry& E = args.L[g4_find_layer(args, job)];
    const uint32_t w = job - E.wg_begin;
    const int n = (E.d_in + E.d_out) / BK;
    int p, q;
    if constexpr (SPLIT) {
      const uint32_t tile = w / (uint32_t)S;
      const int part = (int)(w % (uint32_t)S);
      const int64_t i = tile / (uint32_t)E.pairs;
      g4_tile_pq(E.nt, (int)(tile % (uint32_t)E.pairs), p, q);
      const int s_lo = (int)((int64_t)n * part / S), s_hi = (int)((int64_t)n * (part + 1) / S);
      float* pa = args.park + (size_t)job * 2 * kG4ParkFloats;
      if (p == q) ghost_tile256<BK, WAVES, true, true>(E, i, p, q, lds, park, s_lo, s_hi, pa, pa + kG4ParkFloats, 0u, 0u);
      else ghost_tile256<BK, WAVES, false, true>(E, i, p, q, lds, park, s_lo, s_hi, pa, pa + kG4ParkFloats, 0u, 0u);
      continue;
    }
    // Jobs of an example: with halves, diagonal tile k (k < nt), then the two
    // row halves of every off-diagonal tile; otherwise the tiles of the upper
    // triangle in row-major order. Columns: diagonal tile p, then a pair per
    // off-diagonal tile o (one per half; a whole tile writes the second as 0).
    const int64_t i = w / (uint32_t)E.jpe;
    const int k = (int)(w % (uint32_t)E.jpe);
    int half = -1;
    if (E.halves) {
      if (k < E.nt) {
        p = q = k;
      } else {
        g4_off_pq(E.nt, (k - E.nt) >> 1, p, q);
        half = (k - E.nt) & 1;
      }
    } else {
      g4_tile_pq(E.nt, k, p, q);
    }
    float s;
    if (p == q) {
      s = ghost_tile256<BK, WAVES, true, false>(E, i, p, q, lds, park, 0, n, nullptr, nullptr,
                                                kG4DiagAct, kG4DiagW2);
    } else {
      // Half h: the waves of rows 128 h .. +127 of block p (waves 4 h .. 4 h + 3).
      const uint32_t act = half < 0 ? 0xFFu : 0x0Fu << (4 * half);
      s = ghost_tile256<BK, WAVES, false, false>(E, i, p, q, lds, park, 0, n, nullptr, nullptr,
                                                 act, 0xFFu);
    }
    s = wave_sum(s);
    __syncthreads();   // the ring is free again
    float* red = reinterpret_cast<float*>(lds);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
      float v = 0.f;
#pragma unroll
      for (int k2 = 0; k2 < WAVES; k2 += 2) v += red[k2] + red[k2 + 1];
      float* col = args.partials + i * args.P + E.partial_col;
      if (p == q) {
        col[p] = v;
      } else {
        const int c = E.nt + 2 * g4_off_index(E.nt, p, q);
        if (half < 0) {
          col[c] = v;
          col[c + 1] = 0.f;
        } else {
          col[c + half] = v;
        }
      }
    }
  }
}

// Split tiles: one workgroup per tile adds the parts' partial Gram tiles in
// part order and writes (p == q ? 1 : 2) sum GA GG (GA is zero outside the
// tile's valid rows and columns). The parked positions of every part follow
// the same lane layout, so the product is elementwise over the slots. Each of
// the 1024 threads takes 16 float4 positions, loaded four at a time from
// every slot before they are multiplied (the pass is bound by load latency).
constexpr int kCbThreads = 1024;
template <int S>
__global__ __launch_bounds__(kCbThreads) void ghost256_combine_kernel(G4Args args) {
  __shared__ float red[kCbThreads / 64];
  const uint32_t job0 = blockIdx.x * (uint32_t)S;   // part 0 of this tile
  const GhEntry& E = args.L[g4_find_layer(args, job0)];
  const uint32_t tile = (job0 - E.wg_begin) / (uint32_t)S;
  const int64_t i = tile / (uint32_t)E.pairs;
  const int pr = (int)(tile % (uint32_t)E.pairs);
  int p, q;
  g4_tile_pq(E.nt, pr, p, q);
  const int nA = E.d_in / kG4BK, n = nA + E.d_out / kG4BK;
  const float* base = args.park + (size_t)job0 * 2 * kG4ParkFloats;
  // The parts holding A slices are a prefix (parts 0 .. pa - 1), those holding
  // G slices a suffix (pg .. S - 1). Every load is issued unconditionally from
  // a slot that was written (the part index clamped into the prefix or the
  // suffix), and a select keeps only the parts' own slots, so the loads of a
  // batch are all in flight at once.
  int pa = 0, pg = S;
#pragma unroll
  for (int part = 0; part < S; ++part) {
    if ((int64_t)n * part / S < nA) pa = part + 1;
    if ((int64_t)n * (part + 1) / S > nA && pg == S) pg = part;
  }
  constexpr int kIters = kG4ParkFloats / (4 * kCbThreads);   // 16
  constexpr int kBatch = 4;
  float sum = 0.f;
  for (int k0 = 0; k0 < kIters; k0 += kBatch) {
    f32x4_t ga[kBatch], gg[kBatch];
#pragma unroll
    for (int kk = 0; kk < kBatch; ++kk) ga[kk] = gg[kk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int part = 0; part < S; ++part) {
      const float* sa = base + (size_t)min(part, pa - 1) * 2 * kG4ParkFloats;
      const float* sg = base + (size_t)max(part, pg) * 2 * kG4ParkFloats + kG4ParkFloats;
      const bool use_a = part < pa, use_g = part >= pg;
#pragma unroll
      for (int kk = 0; kk < kBatch; ++kk) {
        const int pos = 4 * ((k0 + kk) * kCbThreads + (int)threadIdx.x);
        const f32x4_t va = *reinterpret_cast<const f32x4_t*>(sa + pos);
        const f32x4_t vg = *reinterpret_cast<const f32x4_t*>(sg + pos);
        const f32x4_t z = f32x4_t{0.f, 0.f, 0.f, 0.f};
        ga[kk] += use_a ? va : z;
        gg[kk] += use_g ? vg : z;
      }
    }
#pragma unroll
    for (int kk = 0; kk < kBatch; ++kk)
      sum += (ga[kk][0] * gg[kk][0] + ga[kk][1] * gg[kk][1]) + (ga[kk][2] * gg[kk][2] + ga[kk][3] * gg[kk][3]);
  }
  sum = wave_sum(sum);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kCbThreads / 64; w += 2) v += red[w] + red[w + 1];
    float* col = args.partials + i * args.P + E.partial_col;
    if (p == q) {
      col[p] = v;
    } else {
      const int c = E.nt + 2 * g4_off_index(E.nt, p, q);
      col[c] = 2.0f * v;
      col[c + 1] = 0.f;
    }
  }
}

}  // namespace

bool ghost_dma_ok(const dpsgd_layer& L) {
  return L.dtype == DPSGD_BF16 && L.d_in % kGgBK == 0 && L.d_out % kGgBK == 0 &&
         L.T * L.d_in * 2 < (INT64_C(1) << 31) && L.T * L.d_out * 2 < (INT64_C(1) << 31);
}

bool ghost256_ok(const dpsgd_layer& L) { return L.T > kG4Rows && ghost_dma_ok(L); }

// Park floats of an unsplit launch: one slot per workgroup of the capped grid.
static size_t ghost256_park_floats_per_grid(int64_t jobs) {
  const int64_t grid = jobs < kGhost256MaxGrid ? jobs : kGhost256MaxGrid;
  return (size_t)grid * kG4ParkFloats;
}

// Tiles of the upper triangle (p <= q) of an example's T x T Gram matrix.
static int64_t ghost256_pairs(const dpsgd_layer& L) {
  const int64_t nt = ceil_div(L.T, kG4Rows);
  return nt * (nt + 1) / 2;
}

int64_t ghost256_cols(const dpsgd_layer& L) {
  const int64_t nt = ceil_div(L.T, kG4Rows);
  return nt * nt;
}

namespace {

// Plan of one launch of 256-row tiles (at most kMaxLayersPerLaunch layers).
// A job runs on one CU and a tile's time is set by its column slices, so with
// fewer tiles than CUs the chip idles. Splitting every tile's slices into S
// parts (at least 16 slices each) runs S times as many shorter jobs, at the
// cost of parking about S + 1 partial Gram tiles per tile for a combine pass.
// S is the largest (at most 4) whose jobs still fit one round on the CUs:
// with a second round the per-slice time rises by about a third when every
// CU copies at once and the parked traffic grows, and the split measured
// slower (c4's shape, B T = 32768: 0.79 against 0.71 ms), while within one
// round it measured 1.2-2.6 times faster (B T = 1024 ... 12288). Without a
// split, when nt^2 jobs per example (diagonal tiles whole, off-diagonal tiles
// as two row halves) still fit one round, the halves run: no parked partials
// and no combine pass (T = 1024, 4096 -> 11008, B = 16: 256 jobs, 0.370-0.375
// ms against 0.391-0.396 for the 160 whole tiles; T = 512, 768 -> 3072, B =
// 64: 0.099-0.102 against 0.109-0.116 ms).
struct G4Plan {
  int split = 1;
  bool halves = false;
  int64_t tiles = 0;
  int64_t jobs = 0;
  size_t park_bytes = 0;
};

G4Plan plan_ghost256(const dpsgd_layer* layers, const int* idx, int n, int64_t cus) {
  G4Plan plan;
  int64_t slices = 0, cols = 0;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    plan.tiles += L.B * ghost256_pairs(L);
    cols += L.B * ghost256_cols(L);
    slices = std::max<int64_t>(slices, (L.d_in + L.d_out) / kG4BK);
  }
  for (int S = 4; S >= 2; --S)
    if (plan.tiles * S <= cus && slices / S >= 16) {
      plan.split = S;
      break;
    }
  plan.halves = plan.split == 1 && cols > plan.tiles && cols <= cus;
  plan.jobs = plan.split > 1 ? plan.tiles * plan.split : (plan.halves ? cols : plan.tiles);
  plan.park_bytes = plan.split == 1
                        ? ghost256_park_floats_per_grid(plan.jobs) * sizeof(float)
                        : (size_t)plan.tiles * plan.split * 2 * kG4ParkFloats * sizeof(float);
  return plan;
}

}  // namespace

size_t ghost256_park_bytes(const dpsgd_layer* layers, const int* idx, int n) {
  size_t bytes = 0;
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    bytes = std::max(bytes, plan_ghost256(layers, idx + base, m, tr_cu_count()).park_bytes);
  }
  return bytes;
}

int launch_ghost256(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                    float* partials, int64_t P, float* park, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    const G4Plan plan = plan_ghost256(layers, idx + base, m, tr_cu_count());
    G4Args a{};
    a.n = m;
    a.split = plan.split;
    a.P = P;
    a.partials = partials;
    a.park = park;
    int64_t jobs = 0;
    for (int k = 0; k < m; ++k) {
      const dpsgd_layer& L = layers[idx[base + k]];
      GhEntry E{};
      E.A = L.A;
      E.G = L.G;
      E.d_in = (int32_t)L.d_in;
      E.d_out = (int32_t)L.d_out;
      E.T = (int32_t)L.T;
      E.nt = (int32_t)ceil_div(L.T, kG4Rows);
      E.pairs = E.nt * (E.nt + 1) / 2;
      E.jpe = plan.halves ? E.nt * E.nt : E.pairs;
      E.halves = plan.halves ? 1 : 0;
      E.partial_col = (int32_t)cols[idx[base + k]];
      E.wg_begin = (uint32_t)jobs;
      a.L[k] = E;
      jobs += L.B * (int64_t)(plan.split > 1 ? E.pairs * plan.split : E.jpe);
    }
    if (jobs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    a.jobs = (uint32_t)jobs;
    // The launches of one call run in stream order, so they share the park
    // area (sized for the largest plan).
    const int64_t grid = jobs < kGhost256MaxGrid ? jobs : kGhost256MaxGrid;
    if (plan.split > 1)
      hipLaunchKernelGGL((ghost_tile256_kernel<kG4BK, kG4Waves, true>), dim3((uint32_t)grid),
                         dim3(64 * kG4Waves), 0, stream, a);
    else
      hipLaunchKernelGGL((ghost_tile256_kernel<kG4BK, kG4Waves, false>), dim3((uint32_t)grid),
                         dim3(64 * kG4Waves), 0, stream, a);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
    if (plan.split > 1) {
      auto combine = plan.split == 2 ? ghost256_combine_kernel<2>
                     : plan.split == 3 ? ghost256_combine_kernel<3>
                                       : ghost256_combine_kernel<4>;
      hipLaunchKernelGGL(combine, dim3((uint32_t)plan.tiles), dim3(kCbThreads), 0, stream, a);
      if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
    }
  }
  return DPSGD_OK;
}

int launch_ghost_dma(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                     float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    GhArgs ga{}, ta{};
    ga.n = ta.n = m;
    ga.P = ta.P = P;
    ga.partials = ta.partials = partials;
    int64_t gwgs = 0, twgs = 0;
    for (int k = 0; k < m; ++k) {
      const dpsgd_layer& L = layers[idx[base + k]];
      GhEntry E{};
      E.A = L.A;
      E.G = L.G;
      E.d_in = (int32_t)L.d_in;
      E.d_out = (int32_t)L.d_out;
      E.T = (int32_t)L.T;
      E.nt = (int32_t)ceil_div(L.T, kGhRows);
      E.pairs = E.nt * (E.nt + 1) / 2;
      // Three-tile groups pay off when they cover the whole triangle (two row
      // blocks); with more blocks most tiles are off-diagonal singles anyway.
      E.groups = E.nt == 2 ? 1 : 0;
      E.singles = E.pairs - 3 * E.groups;
      E.partial_col = (int32_t)cols[idx[base + k]];
      ga.L[k] = E;
      ta.L[k] = E;
      ga.L[k].wg_begin = (uint32_t)gwgs;
      ta.L[k].wg_begin = (uint32_t)twgs;
      gwgs += L.B * (int64_t)E.groups;
      twgs += L.B * (int64_t)E.singles;
    }
    if (gwgs > 0x7FFFFFFF || twgs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    // A layer with no workgroups in a launch starts where the next one does;
    // the kernels pick the last layer starting at or before their job, which
    // is never an empty one.
    if (gwgs > 0) {
      hipLaunchKernelGGL(ghost_group_kernel, dim3((uint32_t)gwgs), dim3(kGgThreads), 0, stream, ga);
      if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
    }
    if (twgs > 0) {
      hipLaunchKernelGGL(ghost_dma_kernel, dim3((uint32_t)twgs), dim3(kGhThreads), 0, stream, ta);
      if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
    }
  }
  return DPSGD_OK;
}

}  // namespace dpsgd
