// 384x256-tile transposed-operand MFMA GEMM for the clip-weighted sum of bf16
// layers with d_in % 256 == 0 and d_out a multiple of 32 (the last row tile
// may hold fewer than 384 rows: its G copies repeat the last valid 64-byte
// column block, and the rows past d_out are not stored):
//   out[m][n] = sum_k c(k) G[k][m] A[k][n],  k over the B*T rows, c = c_i of
//   the example i = k / T (paper: Section 2.2, the clipped per-example
//   gradients c_i g_i summed over the batch).
//
// Why a second tile shape: per FLOP a 384 x 256 workgroup tile copies 17 %
// fewer bytes into LDS than a 256 x 256 one. Sixteen waves (four per SIMD) own
// 96 x 64 sub-tiles (96 fp32 accumulators each), so a wave that waits on LDS
// reads or the slice barrier leaves three others to keep its SIMD's matrix
// core busy; the transposed reads per FLOP (ds_read_b64_tr_b16, 8 consecutive
// k of one row) are 12 % more than with 128 x 64 sub-tiles, but the LDS is far
// from saturated in this loop (the LDS-activity counter reads about two
// cycles per transposed read). On the 48 layers of a 12-block transformer
// step (d = 768 / 3072, B = 128, T = 256): 5.56-5.58 ms against 5.73 ms for
// eight waves with 96 x 128 sub-tiles and 6.0-6.2 ms for the 256 x 256
// kernel; with the whole tiles and the split-K tail spread evenly over the
// XCDs (xcd_two_class_index) 4.92-4.98 ms. Measured bounds: the MFMA issue of
// the eight-wave loop on its own reached about 1.35 PFLOP/s, and with random
// bf16 data the matrix cores sustain about 1.9 PFLOP/s at the power limit
// rather than the nominal 2.5.
//
// Layout of one ring slot (80 KB): the G slice (64 k-rows of 384 bf16) then
// the A slice (64 k-rows of 256 bf16). Both are stored in 256-byte units that
// hold one 64-byte column block of four consecutive k-rows (k-row 4 q + r at
// byte 64 r of the unit); units run along the columns, then along q. Each
// global_load_lds_dwordx4 fills 1 KB of the slot (four units) in order: lane
// i writes slot byte 1024 t + 16 i.
//
// MFMA: v_mfma_f32_32x32x16_bf16. Operand lane l carries row (l % 32) and k
// 8 (l / 32) .. +7 of a 16-k step; two transposed reads supply it: within a
// 16-lane group, lane s points at k-row k0 + s / 4, column c0 + 4 (s % 4), and
// lane d receives the four values of column c0 + d at k0 .. k0 + 3. Group g
// of the wave takes columns 16 (g & 1) of the 32-wide block and k 8 (g / 2),
// so a half-wave reads four k-rows of one 64-byte column block: exactly one
// 256-byte unit, which covers every LDS bank once (no conflicts; with plain
// row-major rows the four rows fall on the same banks and conflict 4-way).
//
// Exact fp32 clip weights: the accumulator is kept in units of the current
// example's factor and multiplied by c_prev / c_next at each example boundary.
#include "lds_dma.h"
#include "mma.h"

namespace dpsgd {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWdTM = 384;                      // tile rows (d_out)
constexpr int kWdTN = 256;                      // tile columns (d_in)
constexpr int kWdBK = 64;                       // k rows per slice
constexpr int kWdWaves = 16;                    // 4 (M) x 4 (N) waves
constexpr int kWdWavesN = 4;
constexpr int kWdThreads = 64 * kWdWaves;
constexpr int kWdMB = 3;                        // 32-row blocks per wave
constexpr int kWdNB = 2;                        // 32-column blocks per wave
constexpr int kWdGGroup = 4 * kWdTM * 2;        // 3 KB: four G k-rows (12 units)
constexpr int kWdAGroup = 4 * kWdTN * 2;        // 2 KB: four A k-rows (8 units)
constexpr int kWdGBytes = kWdBK / 4 * kWdGGroup;   // 48 KB
constexpr int kWdABytes = kWdBK / 4 * kWdAGroup;   // 32 KB
constexpr int kWdStageBytes = kWdGBytes + kWdABytes;
// Two ring slots: the next slice's copies run while the current one is
// multiplied. With eight waves and 32-row slices, two 40 KB slots measured
// 5.63 ms on the 48-layer step against 6.04 for three and 5.78-5.83 for four
// (more bytes in flight did not help).
constexpr int kWdStages = 2;
constexpr int kWdLdsBytes = kWdStages * kWdStageBytes;   // 160 KB
constexpr int kWdGCopies = kWdGBytes / 1024;             // 48
constexpr int kWdCopies = kWdStageBytes / 1024 / kWdWaves;  // 5 per wave per slice
constexpr int kWdTileElems = kWdTM * kWdTN;
static_assert(kWdGCopies % kWdWaves == 0, "G copies split evenly over the waves");
static_assert((kWdStageBytes / 1024) % kWdWaves == 0, "copies split evenly over the waves");
static_assert(kWdWaves / kWdWavesN * kWdMB * 32 == kWdTM && kWdWavesN * kWdNB * 32 == kWdTN,
              "the wave grid covers the tile");
static_assert(kWdLdsBytes <= 160 * 1024, "LDS budget");
static_assert(kWdStages >= 2, "the ring needs a slot being filled and one being read");

struct WdEntry {
  const void* G;          // [B*T][M]
  const void* A;          // [B*T][N]
  float* out;             // [M][N]
  int32_t M, N, T;
  int32_t tiles_n;
  uint32_t tile_begin;
  int64_t q_total;        // K slices of the layer (B * T / 32)
};

// Jobs [0, n_full) are whole tiles; the n_tail jobs after them split each
// remaining tile's Q K slices into tail_w ranges and write partial tiles that
// wide_fixup_kernel adds in range order.
struct WdArgs {
  WdEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t accumulate;
  const float* factors;
  float* partials;        // [n_tail][384 * 256]
  uint32_t n_full, n_tail, n_tiles;
  int32_t Q;
  int32_t tail_w;
};

// 1 KB of zeros: the copy source for examples whose clip factor is 0.
__device__ const uint4 kWdZero[64] = {};

__device__ __forceinline__ int wd_find_layer(const WdArgs& args, uint32_t tile) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].tile_begin <= tile) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Operand of one 32x32x16 MFMA from two transposed reads (k 0..3, k 4..7 of
// the lane's eight); off is a compile-time immediate.
__device__ __forceinline__ bf16x8_t wd_frag(const char* p0, const char* p1, uint32_t off) {
  typedef short v4i16_t __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16_t lds_v4i16;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + off));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p1 + off));
  typedef short v8i16_t __attribute__((ext_vector_type(8)));
  const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

typedef f32x16_t WdAcc[kWdMB][kWdNB];

// acc = sum over K slices [q0, q1) of tile (tm, tn) of layer E, weighted by the
// clip factors; returns the factor the accumulator must be multiplied by.
// ZA: slices of examples with factor 0 are copied from zeros.
template <bool ZA>
__device__ float wd_segment(const WdEntry& E, int tm, int tn, int64_t q0, int64_t q1,
                            const float* factors, char* lds, WdAcc& acc) {
  const int M = E.M, N = E.N, T = E.T;
  const int spe = T / kWdBK;
  // 32-column blocks of G inside the matrix (12 except in a ragged last row tile).
  const uint32_t nvb = (uint32_t)min(kWdTM / 32, (M - tm * kWdTM) / 32);
  const int lane = threadIdx.x & 63;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const char* Gt = static_cast<const char*>(E.G) + (int64_t)tm * kWdTM * 2;
  const char* At = static_cast<const char*>(E.A) + (int64_t)tn * kWdTN * 2;
  const uint32_t lds_addr0 = lds_address(lds);
  typedef __attribute__((address_space(4))) const float const_float;
  const const_float* fac = (const const_float*)factors;

  // Copy p of this wave is copy t = wave + 16 p of the slot. For G (t < 48)
  // it fills row group t / 3, column blocks 4 (t % 3) .. +3; for A (u = t - 48)
  // row group u / 2, column blocks 4 (u % 2) .. +3. Lane i writes unit i / 16,
  // k-row (i % 16) / 4 of the group, bytes 16 (i % 4) .. +15 of the block.
  const uint32_t l_unit = (uint32_t)lane >> 4, l_row = ((uint32_t)lane >> 2) & 3u,
                 l_byte = 16u * ((uint32_t)lane & 3u);
  uint32_t voff[kWdCopies];
#pragma unroll
  for (int p = 0; p < kWdCopies; ++p) {
    const uint32_t t = wave_u + (uint32_t)(kWdWaves * p);
    if (p < kWdGCopies / kWdWaves) {
      const uint32_t row = 4u * (t / 3u) + l_row, blk = 4u * (t % 3u) + l_unit;
      voff[p] = row * (uint32_t)M * 2u + 64u * min(blk, nvb - 1u) + l_byte;
    } else {
      const uint32_t u = t - (uint32_t)kWdGCopies;
      const uint32_t row = 4u * (u / 2u) + l_row, blk = 4u * (u % 2u) + l_unit;
      voff[p] = row * (uint32_t)N * 2u + 64u * blk + l_byte;
    }
  }
  // Any 16 bytes of the zero buffer serve: lane i copies its bytes 16 i.
  const uint32_t zoff = 16u * (uint32_t)lane;
  const int64_t gslice = (int64_t)kWdBK * M * 2, aslice = (int64_t)kWdBK * N * 2;

  int iex = (int)(q0 / spe);
  int ils = (int)(q0 - (int64_t)iex * spe);
  const char* zsrc = reinterpret_cast<const char*>(kWdZero);
  auto issue = [&](int64_t qq, int slot) {
    const bool zero = ZA && fac[iex] == 0.0f;
    const char* gs = zero ? zsrc : Gt + qq * gslice;
    const char* as = zero ? zsrc : At + qq * aslice;
    const uint32_t dst = lds_addr0 + (uint32_t)slot * kWdStageBytes;
#pragma unroll
    for (int p = 0; p < kWdCopies; ++p) {
      const int t = (int)wave_u + kWdWaves * p;
      // t < 48 exactly for p < 3 (48 = 3 * 16): the operand is known per p.
      if (p < kWdGCopies / kWdWaves)
        copy16_to_lds(gs, zero ? zoff : voff[p], dst + 1024u * (uint32_t)t);
      else
        copy16_to_lds(as, zero ? zoff : voff[p], dst + 1024u * (uint32_t)t);
    }
    if (++ils == spe) { ils = 0; ++iex; }
  };

  // Per-lane read bases: group g = lane / 16, s = lane % 16 addresses k-row
  // 8 (g / 2) + 4 h + s / 4, i.e. row group 2 (g / 2) + h and row s / 4 of
  // it, at byte 32 (g & 1) + 8 (s % 4) of the wave's first column block. Block
  // i and k-step ks add 256 i and 16 rows (4 row groups) as immediates.
  const int wave = (int)wave_u, wm = wave / kWdWavesN, wn = wave % kWdWavesN;
  const int g = lane >> 4, s = lane & 15;
  uint32_t rg[2], ra[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int grp = 2 * (g >> 1) + h;
    const int in_unit = 64 * (s >> 2) + 32 * (g & 1) + 8 * (s & 3);
    rg[h] = (uint32_t)(grp * kWdGGroup + 256 * (kWdMB * wm) + in_unit);
    ra[h] = (uint32_t)(kWdGBytes + grp * kWdAGroup + 256 * (kWdNB * wn) + in_unit);
  }

#pragma unroll
  for (int i = 0; i < kWdMB; ++i)
#pragma unroll
    for (int j = 0; j < kWdNB; ++j) acc[i][j] = f32x16_t{};
  float c_cur = 1.0f;
  bool started = false;
  int ex = (int)(q0 / spe);
  int ls = (int)(q0 - (int64_t)ex * spe);

  __syncthreads();   // the ring may still be read by a previous user

#pragma unroll
  for (int d = 0; d < kWdStages - 1; ++d)
    if (q0 + d < q1) issue(q0 + d, d);

  for (int64_t q = q0; q < q1; ++q) {
    // This wave's copies of slice q are done once at most the later slices'
    // copies are outstanding; the barrier then makes every wave's part
    // visible and guarantees that slice q - 1, whose slot is refilled next,
    // is no longer read.
    const int64_t later = q1 - 1 - q;
    if (later >= kWdStages - 2) wait_vmcnt<kWdCopies * (kWdStages - 2)>();
    else if (later == 1) wait_vmcnt<kWdCopies>();
    else wait_vmcnt<0>();
    barrier_no_wait();
    if (q + kWdStages - 1 < q1) issue(q + kWdStages - 1, (int)((q - q0 + kWdStages - 1) % kWdStages));

    if (ls == 0 || q == q0) {
      const float c_new = fac[ex];
      if (c_new != 0.0f) {
        if (started && c_cur != c_new) {
          const float sc = c_cur / c_new;
#pragma unroll
          for (int i = 0; i < kWdMB; ++i)
#pragma unroll
            for (int j = 0; j < kWdNB; ++j) acc[i][j] *= sc;
        }
        c_cur = c_new;
        started = true;
      }
    }

    const char* base = lds + (int)((q - q0) % kWdStages) * kWdStageBytes;
    const char* g0 = base + rg[0];
    const char* g1 = base + rg[1];
    const char* a0 = base + ra[0];
    const char* a1 = base + ra[1];
#pragma unroll
    for (int ks = 0; ks < kWdBK / 16; ++ks) {
      bf16x8_t b[kWdNB];
#pragma unroll
      for (int j = 0; j < kWdNB; ++j) b[j] = wd_frag(a0, a1, ks * 4 * kWdAGroup + 256 * j);
#pragma unroll
      for (int i = 0; i < kWdMB; ++i) {
        const bf16x8_t a = wd_frag(g0, g1, ks * 4 * kWdGGroup + 256 * i);
#pragma unroll
        for (int j = 0; j < kWdNB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[j], acc[i][j], 0, 0, 0);
      }
    }
    if (++ls == spe) { ls = 0; ++ex; }
  }
  return c_cur;
}

// Writes scale * acc into a 384 x 256 row-major destination (row stride ld),
// adding what is there when add; only the first nvb 32-row blocks (the rows
// inside the matrix). Register v of block (i, j) in lane l is tile row
// 32 (kWdMB wm + i) + 8 (v / 4) + 4 (l / 32) + v % 4, column 32 (kWdNB wn + j) + l % 32.
__device__ __forceinline__ void wd_store(float* dst, int64_t ld, const WdAcc& acc, float scale,
                                         bool add, int nvb) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / kWdWavesN, wn = wave % kWdWavesN;
  float* p0 = dst + (int64_t)(wm * kWdMB * 32 + 4 * (lane >> 5)) * ld + wn * kWdNB * 32 +
              (lane & 31);
#pragma unroll
  for (int i = 0; i < kWdMB; ++i) {
    if (wm * kWdMB + i >= nvb) break;   // wave-uniform
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float* p = p0 + (int64_t)(32 * i + 8 * (v >> 2) + (v & 3)) * ld;
#pragma unroll
      for (int j = 0; j < kWdNB; ++j) {
        const float x = acc[i][j][v] * scale;
        p[32 * j] = add ? p[32 * j] + x : x;
      }
    }
  }
}

__device__ __forceinline__ uint32_t wd_range_begin(uint32_t k, uint32_t Q, uint32_t w) {
  return (uint32_t)(((uint64_t)Q * k) / w);
}

__global__ __launch_bounds__(kWdThreads, 1) void tgemm_wide_kernel(WdArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[kWdLdsBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  WdAcc acc;
  const uint32_t job = xcd_two_class_index(blockIdx.x, gridDim.x, args.n_full);
  const bool whole = job < args.n_full;
  uint32_t tile_g = job, qa = 0, qb = 0;
  if (!whole) {
    const uint32_t p = job - args.n_full, w = (uint32_t)args.tail_w;
    tile_g = args.n_full + p / w;
    qa = wd_range_begin(p % w, (uint32_t)args.Q, w);
    qb = wd_range_begin(p % w + 1, (uint32_t)args.Q, w);
  }
  const int l = wd_find_layer(args, tile_g);
  const WdEntry& E = args.L[l];
  const int tile = (int)(tile_g - E.tile_begin);
  const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
  const int spe = E.T / kWdBK;
  const int64_t q_end = whole ? E.q_total : (int64_t)qb;
  int zero_here = 0;
  {
    const int e1 = (int)((q_end - 1) / spe);
    for (int e = (int)(qa / spe) + tid; e <= e1; e += kWdThreads) zero_here |= args.factors[e] == 0.0f;
  }
  int* flags = reinterpret_cast<int*>(lds);
  const bool wave_zero = __builtin_amdgcn_ballot_w64(zero_here != 0) != 0;
  if (lane == 0) flags[wave] = wave_zero ? 1 : 0;
  __syncthreads();
  bool any_zero = false;
#pragma unroll
  for (int w = 0; w < kWdWaves; ++w) any_zero |= flags[w] != 0;
  const float c = any_zero ? wd_segment<true>(E, tm, tn, qa, q_end, args.factors, lds, acc)
                           : wd_segment<false>(E, tm, tn, qa, q_end, args.factors, lds, acc);
  float* dst = whole ? E.out + (int64_t)tm * kWdTM * E.N + tn * kWdTN
                     : args.partials + (int64_t)(job - args.n_full) * kWdTileElems;
  const int64_t ld = whole ? (int64_t)E.N : (int64_t)kWdTN;
  wd_store(dst, ld, acc, c, whole && args.accumulate, min(kWdTM / 32, (E.M - tm * kWdTM) / 32));
}

// Adds the tail_w partials of every tail tile in range order (deterministic)
// and writes grad = (accumulate ? grad : 0) + sum; 96 workgroups of 1024
// elements per tile.
__global__ __launch_bounds__(256) void wide_fixup_kernel(WdArgs args) {
  constexpr uint32_t kChunks = kWdTileElems / 1024;
  const uint32_t n_tail_tiles = args.n_tiles - args.n_full;
  const uint32_t t_local = blockIdx.x / kChunks;
  if (t_local >= n_tail_tiles) return;
  const uint32_t tile_g = args.n_full + t_local;
  const int l = wd_find_layer(args, tile_g);
  const WdEntry& E = args.L[l];
  const int tile = (int)(tile_g - E.tile_begin);
  const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
  const int e = (int)(blockIdx.x % kChunks) * 1024 + threadIdx.x * 4;
  const int r = e / kWdTN, c = e % kWdTN;
  if (tm * kWdTM + r >= E.M) return;   // rows past d_out of a ragged last row tile
  const float* src = args.partials + (int64_t)t_local * args.tail_w * kWdTileElems + e;
  float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k = 0; k < args.tail_w; ++k) {
    const float4 v = *reinterpret_cast<const float4*>(src + (int64_t)k * kWdTileElems);
    sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
  }
  float4* dst = reinterpret_cast<float4*>(E.out + (int64_t)(tm * kWdTM + r) * E.N + tn * kWdTN + c);
  if (args.accumulate) {
    const float4 gv = *dst;
    sum = make_float4(gv.x + sum.x, gv.y + sum.y, gv.z + sum.z, gv.w + sum.w);
  }
  *dst = sum;
}

}  // namespace

// Row tiles of a layer (the last one may be ragged).
int64_t wide_tiles_m(const dpsgd_layer& L) { return ceil_div(L.d_out, kWdTM); }

bool wide_tile_ok(const dpsgd_layer& L) {
  // Per-lane copy offsets are 32-bit: 32 k-rows of d * 2 bytes stay below 2^32.
  // A ragged last row tile is taken when it pads at most 6 % of d_out and the
  // layer has at least one round of tiles: with fewer, every tile would be
  // split along K, and the 256 x 256 kernel, whose tiles fill the round, was
  // faster (4096 x 4096, B T = 16384: 0.53 against 0.66 ms), while with
  // several rounds the 384-row tile wins (11008 x 4096: 1.30 against 1.35 ms).
  const int64_t tm = wide_tiles_m(L), pad = tm * kWdTM - L.d_out;
  const bool whole = L.d_out % kWdTM == 0;
  const bool ragged = L.d_out % 32 == 0 && 50 * pad <= 3 * L.d_out &&
                      tm * (L.d_in / kWdTN) >= tr_cu_count();
  return L.dtype == DPSGD_BF16 && (whole || ragged) && L.d_in % kWdTN == 0 && L.T % kWdBK == 0 &&
         L.d_in <= (INT64_C(1) << 24) && L.d_out <= (INT64_C(1) << 24);
}

void plan_wide_clip(const dpsgd_layer* layers, const int* idx, int n, int cus, TrClipPlan* plan) {
  int64_t tiles = 0, Q = -1;
  bool uniform = true;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    tiles += wide_tiles_m(L) * (L.d_in / kWdTN);
    const int64_t q = L.B * (L.T / kWdBK);
    if (Q >= 0 && q != Q) uniform = false;
    Q = q;
  }
  plan->n_tiles = tiles;
  plan->Q = Q;
  plan->n_full = tiles;
  plan->n_tail = 0;
  plan->tail_w = 1;
  const int64_t rem = tiles % cus;
  if (uniform && n > 0 && rem != 0) {
    const double tile_flops = 2.0 * kWdTM * kWdTN * (double)(Q * kWdBK);
    const int64_t w = choose_tail_split(rem, cus, Q, tile_flops, 4.0 * kWdTileElems);
    if (w > 1) {
      plan->n_full = tiles - rem;
      plan->tail_w = w;
      plan->n_tail = rem * w;
    }
  }
  plan->tail_bytes = (size_t)plan->n_tail * kWdTileElems * sizeof(float);
}

int launch_wide_clip(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                     float* const* outs, int accumulate, const TrClipPlan& plan, float* tail_ws,
                     hipStream_t stream) {
  if (n > kMaxLayersPerLaunch) return DPSGD_ERR_INVALID_ARG;
  WdArgs args{};
  args.n = n;
  args.accumulate = accumulate;
  args.factors = factors;
  args.partials = tail_ws;
  args.n_full = (uint32_t)plan.n_full;
  args.n_tail = (uint32_t)plan.n_tail;
  args.n_tiles = (uint32_t)plan.n_tiles;
  args.Q = (int32_t)plan.Q;
  args.tail_w = (int32_t)plan.tail_w;
  int64_t tb = 0;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    WdEntry& E = args.L[k];
    E.G = L.G;
    E.A = L.A;
    E.out = outs[k];
    E.M = (int32_t)L.d_out;
    E.N = (int32_t)L.d_in;
    E.T = (int32_t)L.T;
    E.tiles_n = (int32_t)(L.d_in / kWdTN);
    E.tile_begin = (uint32_t)tb;
    E.q_total = L.B * (L.T / kWdBK);
    tb += wide_tiles_m(L) * E.tiles_n;
  }
  const int64_t jobs = plan.n_full + plan.n_tail;
  if (jobs <= 0) return DPSGD_OK;
  if (jobs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
  hipLaunchKernelGGL(tgemm_wide_kernel, dim3((uint32_t)jobs), dim3(kWdThreads), 0, stream, args);
  if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  if (plan.n_tail > 0) {
    const int64_t wgs = (plan.n_tiles - plan.n_full) * (kWdTileElems / 1024);
    hipLaunchKernelGGL(wide_fixup_kernel, dim3((uint32_t)wgs), dim3(256), 0, stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

}  // namespace dpsgd
