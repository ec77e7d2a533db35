// 256x256-tile transposed-operand MFMA GEMM for bf16 layers (clip-weighted sum
// and materialised norms): out[m][n] = sum_k w(k) G[k][m] A[k][n], where k runs
// over the B*T rows (example i = k / T, w = c_i or 1).
//
// Loads: every K slice of G [k][m] and A [k][n] (32 rows) is copied from HBM
// straight into LDS in its natural k-major layout with global_load_lds_dwordx4
// (16 bytes per lane, no VGPR staging, no ALU work). A four-slot ring keeps
// three slices in flight while the fourth is consumed.
//
// Operands: ds_read_b64_tr_b16 reads the MFMA operand (8 consecutive k of
// one row m) transposed out of the k-major tile. Within a 16-lane group, lane
// d receives element d % 4 of the 8-byte chunks addressed by lanes 4r + d/4,
// r = 0..3, so pointing lane s at X[k0 + s/4][m0 + 4(s%4)] hands lane d the
// four values X[k0..k0+3][m0 + d]; two such reads give k0..k0+7.
//
// LDS layout of an operand slice (32 rows of 512 bytes): block j (j = 0..15)
// holds rows j and j + 16 (one 1 KB copy instruction) at byte offset
// j * 1280 + 32 * g(j), g(j) = (j & 3) + 4 * ((j >> 3) & 1): the 8 rows one
// half-wave reads in a transposed read start on 8 different 32-byte bank
// groups (conflict-free), and every read offset is a per-lane base plus a
// compile-time immediate.
//
// Eight wave64s per workgroup in a 2 x 4 grid own 128 x 64 sub-tiles (8 x 4
// blocks of the 16 x 16 MFMA output); their accumulators (128 fp32 per lane)
// stay in VGPRs, so the clip weight is applied exactly: the accumulator is
// kept in units of the current example's factor and multiplied by
// c_prev / c_next at each example boundary
// (paper: Section 2.2, g_bar_i = c_i g_i summed over the batch).
#include "lds_dma.h"
#include "mma.h"

namespace dpsgd {
namespace {

constexpr int kTrTile = 256;             // workgroup tile edge
constexpr int kTrBK = 32;                // k rows per slice
#ifndef DPSGD_TR_STAGES
#define DPSGD_TR_STAGES 4
#endif
constexpr int kTrStages = DPSGD_TR_STAGES;  // LDS ring slots
constexpr int kTrWaves = 8;                            // 2 x 4 grid of 128 x 64 sub-tiles
constexpr int kTrThreads = 64 * kTrWaves;
constexpr int kTrMB = 8;                               // 16-row blocks per wave along M
constexpr int kTrNB = 4;                               // 16-column blocks per wave along N
constexpr int kTrPairs = 16 / kTrWaves;                // row pairs per wave per operand
constexpr int kTrLdPerSlice = 2 * kTrPairs;            // copies per wave per slice
constexpr int kTrRowBytes = kTrTile * 2;              // 512
constexpr int kTrBlockStride = 1280;                   // 1 KB block + room for the bank shift
constexpr int kTrOpBytes = 16 * kTrBlockStride;        // 20 KB per operand slice
constexpr int kTrStageBytes = 2 * kTrOpBytes;          // G slice then A slice
constexpr int kTrLdsBytes = kTrStages * kTrStageBytes; // 160 KB

enum TrEpi : int { TR_STORE = 0, TR_SUMSQ = 1 };

struct TrEntry {
  const void* G;          // [B*T][M]
  const void* A;          // [B*T][N]
  float* out;             // STORE: grad
  int32_t M, N, T;
  int32_t tiles_n;
  uint32_t tile_begin;    // first tile of this layer in the launch's tile list
  int32_t partial_col;    // SUMSQ
  int32_t pad[2];
};
// STORE launches: jobs [0, n_full) are whole tiles (tile = job); the
// n_tail = (n_tiles - n_full) * tail_w jobs after them split each remaining
// tile's Q K slices into tail_w equal ranges (worker p: tile n_full + p /
// tail_w, range p % tail_w) and write partial tiles that tr_fixup_kernel adds
// in range order. SUMSQ launches: job = example * tiles + tile of its layer
// (jobs per layer = B * tiles).
struct TrArgs {
  TrEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  const float* factors;
  float* partials;        // SUMSQ partials, or STORE tail partials [n_tail][256 * 256]
  int64_t P;              // SUMSQ partial row length
  uint32_t n_full, n_tail, n_tiles;
  int32_t Q;              // K slices per tile (STORE)
  int32_t accumulate;
  int32_t tail_w;         // tail workers per tail tile
};

// 512 zero bytes in global memory: the copy source for examples whose clip
// factor is 0.
__device__ const uint4 kZeroRow[32] = {};

// Byte offset of copy block j (rows j and j + 16) within an operand slice.
__host__ __device__ constexpr int block_offset(int j) {
  return j * kTrBlockStride + 32 * ((j & 3) + 4 * ((j >> 3) & 1));
}

// MFMA operand (8 consecutive k of one row) from two transposed 8-byte reads at
// p0 + off (k 0..3) and p1 + off (k 4..7); off is a compile-time immediate.
__device__ __forceinline__ bf16x8_t read_frag_tr(const char* p0, const char* p1, uint32_t off) {
  typedef short v4i16_t __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16_t lds_v4i16;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + off));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p1 + off));
  typedef short v8i16_t __attribute__((ext_vector_type(8)));
  const v8i16_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ int find_layer(const TrArgs& args, uint32_t tile) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].tile_begin <= tile) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Per-lane transposed-read bases (bytes within a stage), fixed for the whole
// kernel: lane 16 grp + s addresses slice row k = 8 grp + 4 h + s / 4 (h = 0
// for k 0..3 of its 8, 1 for 4..7) at column 4 (s % 4) of a 16-wide block.
struct TrLane {
  uint32_t rd[2];
};

__device__ __forceinline__ void init_lane(TrLane& ln, int lane) {
  const int s = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = 8 * grp + 4 * h + (s >> 2);
    ln.rd[h] = block_offset(k & 15) + (k >> 4) * kTrRowBytes + (s & 3) * 8;
  }
}

// Byte offset of the 16-wide column block blk within a slice row.
__device__ __forceinline__ constexpr uint32_t col_block(int blk) { return 32u * blk; }

typedef f32x4_t TrAcc[kTrMB][kTrNB];

// acc = sum over K slices [q0, q1) of tile (tm, tn) of layer E, each slice's
// example weighted by its clip factor when WEIGHTED (exact fp32 weights: the
// accumulator is kept in units of the current factor and rescaled at example
// boundaries). Returns the factor the accumulator must finally be multiplied by.
template <bool WEIGHTED, bool ZA>
__device__ float tr_segment(const TrEntry& E, int tm, int tn, int64_t q0, int64_t q1,
                            const float* factors, char* lds, const TrLane& ln,
                            TrAcc& acc) {
  const int M = E.M, N = E.N, T = E.T;
  const int spe = T / kTrBK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const char* Gt = static_cast<const char*>(E.G) + (int64_t)tm * kTrTile * 2;
  const char* At = static_cast<const char*>(E.A) + (int64_t)tn * kTrTile * 2;
  const uint32_t lds_addr0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(wave);
  // Clip factors through the scalar cache (constant address space): these loads
  // then never count against vmcnt, which tracks the slice copies.
  typedef __attribute__((address_space(4))) const float const_float;
  const const_float* fac = (const const_float*)factors;

  // Copy p of this wave moves block j = wave + p * waves of the slice: lanes
  // 0..31 row j, lanes 32..63 row j + 16, 16 bytes each. The per-lane byte
  // offsets within a slice are fixed; the slice base is uniform.
  const int crow = 16 * (lane >> 5), ccol = (lane & 31) * 16;
  uint32_t goff[kTrPairs], aoff[kTrPairs];
#pragma unroll
  for (int p = 0; p < kTrPairs; ++p) {
    const int j = (int)wave_u + kTrWaves * p;
    goff[p] = (uint32_t)(j + crow) * (uint32_t)M * 2u + ccol;
    aoff[p] = (uint32_t)(j + crow) * (uint32_t)N * 2u + ccol;
  }
  const int64_t gslice = (int64_t)kTrBK * M * 2, aslice = (int64_t)kTrBK * N * 2;

  // Slices are issued in order, one at a time; (iex, ils) is the example and
  // chunk of the next one. T is a multiple of the slice height, so slice qq
  // starts at row qq * 32 of the [B*T] rows.
  int iex = (int)(q0 / spe);
  int ils = (int)(q0 - (int64_t)iex * spe);
  // An example whose clip factor is 0 contributes nothing. With ZA, its slices
  // are copied from a row of zeros instead of G and A, so the MFMA loop needs
  // no branch and non-finite inputs of that example cannot reach the sum; the
  // kernel uses that instance only for a segment that has such an example.
  const char* zrow = reinterpret_cast<const char*>(kZeroRow);
  auto issue = [&](int64_t qq, int slot) {
    const bool zero = ZA && fac[iex] == 0.0f;
    const char* gs = zero ? zrow : Gt + qq * gslice;
    const char* as = zero ? zrow : At + qq * aslice;
    const uint32_t dst = lds_addr0 + (uint32_t)slot * kTrStageBytes;
#pragma unroll
    for (int p = 0; p < kTrPairs; ++p) {
      const uint32_t off = (uint32_t)block_offset((int)wave_u + kTrWaves * p);
      copy16_to_lds(gs, zero ? (uint32_t)ccol : goff[p], dst + off);
      copy16_to_lds(as, zero ? (uint32_t)ccol : aoff[p], dst + kTrOpBytes + off);
    }
    if (++ils == spe) { ils = 0; ++iex; }
  };

#pragma unroll
  for (int ii = 0; ii < kTrMB; ++ii)
#pragma unroll
    for (int jj = 0; jj < kTrNB; ++jj) acc[ii][jj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float c_cur = 1.0f;
  bool started = false;
  int ex = (int)(q0 / spe);
  int ls = (int)(q0 - (int64_t)ex * spe);
  const int wm = wave >> 2, wn = wave & 3;

  // All waves must be done with the ring before a new segment overwrites it.
  __syncthreads();

#pragma unroll
  for (int d = 0; d < kTrStages - 1; ++d)
    if (q0 + d < q1) issue(q0 + d, d);

  for (int64_t q = q0; q < q1; ++q) {
    // This wave's copies of slice q are done once at most the later slices'
    // copies are outstanding; the barrier then makes every wave's part
    // visible and guarantees that slice q - 1, whose slot is refilled next,
    // is no longer read.
    const int64_t later = q1 - 1 - q;
    if (later >= kTrStages - 2) wait_vmcnt<kTrLdPerSlice * (kTrStages - 2)>();
    else if (later == 1) wait_vmcnt<kTrLdPerSlice>();
    else wait_vmcnt<0>();
    barrier_no_wait();
    if (q + kTrStages - 1 < q1) issue(q + kTrStages - 1, (int)((q - q0 + kTrStages - 1) % kTrStages));

    if (WEIGHTED && (ls == 0 || q == q0)) {
      const float c_new = fac[ex];
      if (c_new != 0.0f) {
        if (started && c_cur != c_new) {
          const float sc = c_cur / c_new;
#pragma unroll
          for (int ii = 0; ii < kTrMB; ++ii)
#pragma unroll
            for (int jj = 0; jj < kTrNB; ++jj) acc[ii][jj] *= sc;
        }
        c_cur = c_new;
        started = true;
      }
    }

    const char* base = lds + (int)((q - q0) % kTrStages) * kTrStageBytes;
    const char* b0 = base + ln.rd[0];
    const char* b1 = base + ln.rd[1];
    bf16x8_t b[kTrNB];
#pragma unroll
    for (int jj = 0; jj < kTrNB; ++jj) b[jj] = read_frag_tr(b0, b1, kTrOpBytes + col_block(wn * kTrNB + jj));
#pragma unroll
    for (int ii = 0; ii < kTrMB; ++ii) {
      const bf16x8_t a = read_frag_tr(b0, b1, col_block(wm * kTrMB + ii));
#pragma unroll
      for (int jj = 0; jj < kTrNB; ++jj)
        acc[ii][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[jj], acc[ii][jj], 0, 0, 0);
    }
    if (++ls == spe) { ls = 0; ++ex; }
  }
  return c_cur;
}

// Writes scale * acc to a 256x256 row-major destination with row stride ld
// (adding what is there when add). Element v of block (i, j) in lane l is
// tile row 128 wm + 16 i + 4 (l / 16) + v and column 64 wn + 16 j + l % 16.
__device__ __forceinline__ void store_tile(float* dst, int64_t ld, const TrAcc& acc, float scale,
                                           bool add) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  float* col0 = dst + (int64_t)(wm * 128 + 4 * (lane >> 4)) * ld + wn * 64 + (lane & 15);
#pragma unroll
  for (int i = 0; i < kTrMB; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float* p = col0 + (int64_t)(i * 16 + v) * ld;
#pragma unroll
      for (int j = 0; j < kTrNB; ++j) {
        const float x = acc[i][j][v] * scale;
        p[j * 16] = add ? p[j * 16] + x : x;
      }
    }
}

// First K slice of range k of the w ranges a tile's Q slices are split into.
__device__ __forceinline__ uint32_t tail_range_begin(uint32_t k, uint32_t Q, uint32_t w) {
  return (uint32_t)(((uint64_t)Q * k) / w);
}

template <int EPI>
__global__ __launch_bounds__(kTrThreads, 1) void tgemm_tr_kernel(TrArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[kTrLdsBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  TrLane ln;
  init_lane(ln, lane);
  TrAcc acc;
  const uint32_t job = xcd_two_class_index(blockIdx.x, gridDim.x, args.n_full);

  if (EPI == TR_SUMSQ) {
    // job -> (layer, example, tile); jobs of a layer are B * tiles, laid out from tile_begin * B
    int l = 0;
    {
      int lo = 0, hi = args.n - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (args.L[mid].tile_begin * (uint32_t)args.B <= job) lo = mid; else hi = mid - 1;
      }
      l = lo;
    }
    const TrEntry& E = args.L[l];
    const int tiles_mn = (E.M / kTrTile) * E.tiles_n;
    const uint32_t w = job - E.tile_begin * (uint32_t)args.B;
    const int ex = (int)(w / (uint32_t)tiles_mn);
    const int tile = (int)(w % (uint32_t)tiles_mn);
    const int spe = E.T / kTrBK;
    tr_segment<false, false>(E, tile / E.tiles_n, tile % E.tiles_n, (int64_t)ex * spe,
                      (int64_t)(ex + 1) * spe, nullptr, lds, ln, acc);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < kTrMB; ++i)
#pragma unroll
      for (int j = 0; j < kTrNB; ++j) {
#pragma unroll
        for (int v = 0; v < 4; ++v) sum = fmaf(acc[i][j][v], acc[i][j][v], sum);
      }
    sum = wave_sum(sum);
    float* red = reinterpret_cast<float*>(lds);  // the ring is free after the segment
    __syncthreads();
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
      for (int k = 0; k < kTrWaves; ++k) t += red[k];
      args.partials[(int64_t)ex * args.P + E.partial_col + tile] = t;
    }
    return;
  }

  // Jobs below n_full own a whole tile: all its K slices, stored into the
  // gradient. Tail worker p = job - n_full owns range p % tail_w of tail tile
  // p / tail_w and stores a partial tile.
  const bool whole = job < args.n_full;
  uint32_t tile_g = job, qa = 0, qb = 0;
  if (!whole) {
    const uint32_t p = job - args.n_full, w = (uint32_t)args.tail_w;
    tile_g = args.n_full + p / w;
    qa = tail_range_begin(p % w, (uint32_t)args.Q, w);
    qb = tail_range_begin(p % w + 1, (uint32_t)args.Q, w);
  }
  const int l = find_layer(args, tile_g);
  const TrEntry& E = args.L[l];
  const int tile = (int)(tile_g - E.tile_begin);
  const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
  const int64_t q_end = whole ? (int64_t)args.B * (E.T / kTrBK) : (int64_t)qb;
  // Segments with an example whose factor is 0 take the zero-aware instance
  // (each thread tests a few of the segment's examples).
  int zero_here = 0;
  {
    const int spe = E.T / kTrBK;
    const int e1 = (int)((q_end - 1) / spe);
    for (int e = (int)(qa / spe) + tid; e <= e1; e += kTrThreads) zero_here |= args.factors[e] == 0.0f;
  }
  // Workgroup OR through the (still unused) ring; the segment starts with a
  // barrier before the ring is written.
  int* flags = reinterpret_cast<int*>(lds);
  const bool wave_zero = __builtin_amdgcn_ballot_w64(zero_here != 0) != 0;
  if (lane == 0) flags[wave] = wave_zero ? 1 : 0;
  __syncthreads();
  bool any_zero = false;
#pragma unroll
  for (int w = 0; w < kTrWaves; ++w) any_zero |= flags[w] != 0;
  const float c = any_zero ? tr_segment<true, true>(E, tm, tn, qa, q_end, args.factors, lds, ln, acc)
                           : tr_segment<true, false>(E, tm, tn, qa, q_end, args.factors, lds, ln, acc);
  // One store for both cases (two inlined copies raise register pressure).
  float* dst = whole ? E.out + (int64_t)tm * kTrTile * E.N + tn * kTrTile
                     : args.partials + (int64_t)(job - args.n_full) * kTrTile * kTrTile;
  const int64_t ld = whole ? (int64_t)E.N : (int64_t)kTrTile;
  store_tile(dst, ld, acc, c, whole && args.accumulate);
}

// Adds the tail_w partials of every tail tile in range order (deterministic)
// and writes grad = (accumulate ? grad : 0) + sum. One workgroup per 1024
// elements (256 threads x 4 consecutive elements), 64 workgroups per tile.
__global__ __launch_bounds__(256) void tr_fixup_kernel(TrArgs args) {
  const uint32_t n_tail_tiles = args.n_tiles - args.n_full;
  const uint32_t chunk = blockIdx.x;                 // 64 chunks of 1024 elements per tile
  const uint32_t t_local = chunk >> 6;
  if (t_local >= n_tail_tiles) return;
  const uint32_t tile_g = args.n_full + t_local;
  const int l = find_layer(args, tile_g);
  const TrEntry& E = args.L[l];
  const int tile = (int)(tile_g - E.tile_begin);
  const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
  const int e = (int)(chunk & 63) * 1024 + threadIdx.x * 4;   // 4 consecutive elements
  const int r = e >> 8, c = e & 255;
  const float* src = args.partials + (int64_t)t_local * args.tail_w * kTrTile * kTrTile + e;
  float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k = 0; k < args.tail_w; ++k) {
    const float4 v = *reinterpret_cast<const float4*>(src + (int64_t)k * kTrTile * kTrTile);
    sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
  }
  float4* dst = reinterpret_cast<float4*>(E.out + (int64_t)(tm * kTrTile + r) * E.N + tn * kTrTile + c);
  if (args.accumulate) {
    const float4 g = *dst;
    sum = make_float4(g.x + sum.x, g.y + sum.y, g.z + sum.z, g.w + sum.w);
  }
  *dst = sum;
}

}  // namespace

bool tr_tile_ok(const dpsgd_layer& L) {
  // The copies address a slice with 32-bit per-lane offsets: 32 rows of d * 2
  // bytes must stay below 2^32.
  return L.dtype == DPSGD_BF16 && L.d_in % kTrTile == 0 && L.d_out % kTrTile == 0 &&
         L.T % kTrBK == 0 && L.d_in <= (INT64_C(1) << 24) && L.d_out <= (INT64_C(1) << 24);
}

int64_t tr_q_total(const dpsgd_layer& L) { return L.B * (L.T / kTrBK); }

int tr_cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  return cus;
}

void plan_tr_clip(const dpsgd_layer* layers, const int* idx, int n, int cus, TrClipPlan* plan) {
  int64_t tiles = 0;
  int64_t Q = -1;
  bool uniform = true;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    tiles += (L.d_out / kTrTile) * (L.d_in / kTrTile);
    const int64_t q = tr_q_total(L);
    if (Q >= 0 && q != Q) uniform = false;
    Q = q;
  }
  plan->n_tiles = tiles;
  plan->Q = Q;
  plan->n_full = tiles;
  plan->n_tail = 0;
  plan->tail_w = 1;
  // Whole tiles for the full rounds over the CUs; the last partial round's
  // tiles are each split along K into tail_w ranges so that the round fills
  // the CUs (only when every tile has the same Q).
  const int64_t rem = tiles % cus;
  if (uniform && n > 0 && rem != 0) {
    const double tile_flops = 2.0 * kTrTile * kTrTile * (double)(Q * kTrBK);
    const int64_t w = choose_tail_split(rem, cus, Q, tile_flops, 4.0 * kTrTile * kTrTile);
    if (w > 1) {
      plan->n_full = tiles - rem;
      plan->tail_w = w;
      plan->n_tail = rem * w;
    }
  }
  plan->tail_bytes = (size_t)plan->n_tail * kTrTile * kTrTile * sizeof(float);
}

int launch_tr_clip(const dpsgd_layer* layers, const int* idx, int n, const float* factors,
                   float* const* outs, int accumulate, const TrClipPlan& plan, float* tail_ws,
                   hipStream_t stream) {
  if (n > kMaxLayersPerLaunch) return DPSGD_ERR_INVALID_ARG;
  TrArgs args{};
  args.n = n;
  args.B = (int32_t)layers[idx[0]].B;
  args.factors = factors;
  args.partials = tail_ws;
  args.n_full = (uint32_t)plan.n_full;
  args.n_tail = (uint32_t)plan.n_tail;
  args.n_tiles = (uint32_t)plan.n_tiles;
  args.Q = (int32_t)plan.Q;
  args.accumulate = accumulate;
  args.tail_w = (int32_t)plan.tail_w;
  int64_t tb = 0;
  for (int k = 0; k < n; ++k) {
    const dpsgd_layer& L = layers[idx[k]];
    TrEntry& E = args.L[k];
    E.G = L.G;
    E.A = L.A;
    E.out = outs[k];
    E.M = (int32_t)L.d_out;
    E.N = (int32_t)L.d_in;
    E.T = (int32_t)L.T;
    E.tiles_n = (int32_t)(L.d_in / kTrTile);
    E.tile_begin = (uint32_t)tb;
    tb += (L.d_out / kTrTile) * E.tiles_n;
  }
  const int64_t jobs = plan.n_full + plan.n_tail;
  if (jobs <= 0) return DPSGD_OK;
  if (jobs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
  hipLaunchKernelGGL(tgemm_tr_kernel<TR_STORE>, dim3((uint32_t)jobs), dim3(kTrThreads), 0, stream,
                     args);
  if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  if (plan.n_tail > 0) {
    const int64_t wgs = (plan.n_tiles - plan.n_full) * 64;
    hipLaunchKernelGGL(tr_fixup_kernel, dim3((uint32_t)wgs), dim3(256), 0, stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

int launch_tr_mat_norms(const dpsgd_layer* layers, const int* idx, int n, const int64_t* cols,
                        float* partials, int64_t P, hipStream_t stream) {
  for (int base = 0; base < n; base += kMaxLayersPerLaunch) {
    const int m = n - base < kMaxLayersPerLaunch ? n - base : kMaxLayersPerLaunch;
    TrArgs args{};
    args.n = m;
    args.B = (int32_t)layers[idx[base]].B;
    args.partials = partials;
    args.P = P;
    int64_t tb = 0;
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
      E.tile_begin = (uint32_t)tb;
      E.partial_col = (int32_t)cols[li];
      tb += (L.d_out / kTrTile) * E.tiles_n;
    }
    const int64_t jobs = tb * args.B;
    if (jobs > 0x7FFFFFFF) return DPSGD_ERR_INVALID_ARG;
    hipLaunchKernelGGL(tgemm_tr_kernel<TR_SUMSQ>, dim3((uint32_t)jobs), dim3(kTrThreads), 0,
                       stream, args);
    if (check_launch() != DPSGD_OK) return DPSGD_ERR_HIP;
  }
  return DPSGD_OK;
}

}  // namespace dpsgd
