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
#ifndef DPSGD_TR_STAGES
#define DPSGD_TR_STAGES 4
#endif
constexpr int kTrStages = DPSGD_TR_STAGES;  // LDS ring slots
constexpr int kTrThreads = 512;          // 8 wave64s
constexpr int kTrRowBytes = kTrTile * 2; // 512
constexpr int kTrOpBytes = kTrBK * kTrRowBytes;       // 16 KB per operand slice
constexpr int kTrStageBytes = 2 * kTrOpBytes;         // G slice then A slice
constexpr int kTrLdsBytes = kTrStages * kTrStageBytes; // 128 KB

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
// STORE launches: jobs [0, n_full) are whole tiles (tile = job); jobs
// [n_full, n_full + n_tail) are tail workers that split the K slices of tiles
// n_full .. n_tiles-1 evenly (stream-K) and write partials that
// tr_fixup_kernel adds in worker order. SUMSQ launches: job = example * tiles
// + tile of its layer (jobs per layer = B * tiles).
struct TrArgs {
  TrEntry L[kMaxLayersPerLaunch];
  int32_t n;
  int32_t B;
  const float* factors;
  float* partials;        // SUMSQ partials, or STORE tail partials [2 * n_tail][256 * 256]
  int64_t P;              // SUMSQ partial row length
  uint32_t n_full, n_tail, n_tiles;
  int32_t Q;              // K slices per tile (STORE)
  int32_t accumulate;
  int32_t pad;
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

__device__ __forceinline__ int find_layer(const TrArgs& args, uint32_t tile) {
  int lo = 0, hi = args.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (args.L[mid].tile_begin <= tile) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Per-lane LDS offsets and copy assignment, fixed for the whole kernel.
struct TrLane {
  int ld_k[2];            // slice row of the lane's two copies
  int ld_chunk[2];        // global 16-byte chunk (0..31) within the 256-wide row
  uint32_t offA[8][2];    // transposed-read offsets (bytes within the stage), M side
  uint32_t offB[4][2];    // N side
};

__device__ __forceinline__ void init_lane(TrLane& ln, int wave, int lane) {
  const int wm = wave >> 2, wn = wave & 3;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int k = 2 * (wave + 8 * p) + (lane >> 5);
    const int pos = lane & 31;
    ln.ld_k[p] = k;
    ln.ld_chunk[p] = 2 * (((pos >> 1) ^ seg_swizzle(k))) + (pos & 1);
  }
  const int s = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = 8 * grp + 4 * h + (s >> 2);
    const int f = seg_swizzle(k);
    const int q = (s & 3) >> 1, half = (s & 1) * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int blk = wm * 8 + i;  // 16-wide block index along M
      ln.offA[i][h] = k * kTrRowBytes + (2 * (blk ^ f) + q) * 16 + half;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int blk = wn * 4 + j;
      ln.offB[j][h] = kTrOpBytes + k * kTrRowBytes + (2 * (blk ^ f) + q) * 16 + half;
    }
  }
}

// acc = sum over K slices [q0, q1) of tile (tm, tn) of layer E, each slice's
// example weighted by its clip factor when WEIGHTED (exact fp32 weights: the
// accumulator is kept in units of the current factor and rescaled at example
// boundaries). Returns the factor the accumulator must finally be multiplied by.
template <bool WEIGHTED>
__device__ float tr_segment(const TrEntry& E, int tm, int tn, int64_t q0, int64_t q1,
                            const float* factors, char* lds, const TrLane& ln,
                            f32x4_t (&acc)[8][4]) {
  const int M = E.M, N = E.N, T = E.T;
  const int spe = T / kTrBK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint16_t* Gt = static_cast<const uint16_t*>(E.G) + tm * kTrTile;
  const uint16_t* At = static_cast<const uint16_t*>(E.A) + tn * kTrTile;
  const uint32_t lds_addr0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(wave);
  // Clip factors through the scalar cache (constant address space): these loads
  // then never count against vmcnt, which tracks the slice copies.
  typedef __attribute__((address_space(4))) const float const_float;
  const const_float* fac = (const const_float*)factors;
  (void)lane;

  // T is a multiple of the slice height, so slice qq (example qq / spe, chunk
  // qq % spe) starts at row qq * 32 of the [B*T] rows: no division needed.
  auto issue = [&](int64_t qq, int slot) {
    const int64_t row0 = qq * kTrBK;
    const uint32_t dst = lds_addr0 + (uint32_t)slot * kTrStageBytes;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int64_t row = row0 + ln.ld_k[p];
      const uint32_t pair = wave_u + 8u * p;
      copy16_to_lds(Gt + row * M + ln.ld_chunk[p] * 8, dst + pair * 1024u);
      copy16_to_lds(At + row * N + ln.ld_chunk[p] * 8, dst + kTrOpBytes + pair * 1024u);
    }
  };

  zero_acc_t(acc);
  float c_cur = 1.0f;
  bool started = false;

  // All waves must be done with the ring before a new segment overwrites it.
  __syncthreads();
#pragma unroll
  for (int d = 0; d < kTrStages - 1; ++d)
    if (q0 + d < q1) issue(q0 + d, d);

  int ex = (int)(q0 / spe);
  int ls = (int)(q0 - (int64_t)ex * spe);
  for (int64_t q = q0; q < q1; ++q) {
    // This wave's copies of slice q are done once at most the later slices'
    // copies (4 instructions per slice) are outstanding; the barrier then makes
    // every wave's part visible and guarantees slice q-1 is no longer read.
    const int64_t later = q1 - 1 - q;
    if (later >= kTrStages - 2) wait_vmcnt<4 * (kTrStages - 2)>();
    else if (later == 3) wait_vmcnt<12>();
    else if (later == 2) wait_vmcnt<8>();
    else if (later == 1) wait_vmcnt<4>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (q + kTrStages - 1 < q1) issue(q + kTrStages - 1, (int)((q - q0 + kTrStages - 1) % kTrStages));

    bool skip = false;
    if (WEIGHTED) {
      const float c_new = fac[ex];
      if (ls == 0 || q == q0) {
        if (c_new != 0.0f) {
          if (started && c_cur != c_new) scale_acc_t(acc, c_cur / c_new);
          c_cur = c_new;
          started = true;
        }
      }
      skip = c_new == 0.0f;  // the example contributes nothing
    }
    if (!skip) {
      const char* base = lds + (int)((q - q0) % kTrStages) * kTrStageBytes;
      bf16x8_t b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = read_frag_tr(base, ln.offB[j][0], ln.offB[j][1]);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bf16x8_t a = read_frag_tr(base, ln.offA[i][0], ln.offA[i][1]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[j], acc[i][j], 0, 0, 0);
      }
    }
    if (++ls == spe) { ls = 0; ++ex; }
  }
  return c_cur;
}

// Writes scale * acc to a 256x256 row-major destination with row stride ld
// (adding what is there when add).
__device__ __forceinline__ void store_tile(float* dst, int64_t ld, const f32x4_t (&acc)[8][4],
                                           float scale, bool add) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  float* col0 = dst + (int64_t)(wm * 128 + 4 * (lane >> 4)) * ld + wn * 64 + (lane & 15);
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float* p = col0 + (int64_t)(i * 16 + v) * ld;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float x = acc[i][j][v] * scale;
        p[j * 16] = add ? p[j * 16] + x : x;
      }
    }
}

__device__ __forceinline__ uint32_t tail_unit_begin(uint32_t p, uint64_t units, uint32_t workers) {
  return (uint32_t)((units * p) / workers);
}

template <int EPI>
__global__ __launch_bounds__(kTrThreads, 1) void tgemm_tr_kernel(TrArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[kTrLdsBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  TrLane ln;
  init_lane(ln, wave, lane);
  f32x4_t acc[8][4];
  const uint32_t job = xcd_logical_index(blockIdx.x, gridDim.x);

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
    tr_segment<false>(E, tile / E.tiles_n, tile % E.tiles_n, (int64_t)ex * spe,
                      (int64_t)(ex + 1) * spe, nullptr, lds, ln, acc);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) sum = fmaf(acc[i][j][v], acc[i][j][v], sum);
    sum = wave_sum(sum);
    float* red = reinterpret_cast<float*>(lds);  // the ring is free after the segment
    __syncthreads();
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
      for (int k = 0; k < 8; ++k) t += red[k];
      args.partials[(int64_t)ex * args.P + E.partial_col + tile] = t;
    }
    return;
  }

  if (job < args.n_full) {
    const int l = find_layer(args, job);
    const TrEntry& E = args.L[l];
    const int tile = (int)(job - E.tile_begin);
    const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
    const int64_t q_layer = (int64_t)args.B * (E.T / kTrBK);
    const float c = tr_segment<true>(E, tm, tn, 0, q_layer, args.factors, lds, ln, acc);
    store_tile(E.out + (int64_t)tm * kTrTile * E.N + tn * kTrTile, E.N, acc, c, args.accumulate);
    return;
  }

  // Tail worker p: units [u0, u1) of the tail's n_tiles - n_full tiles x Q slices.
  const uint32_t p = job - args.n_full;
  const uint64_t units = (uint64_t)(args.n_tiles - args.n_full) * (uint32_t)args.Q;
  const uint32_t u0 = tail_unit_begin(p, units, args.n_tail);
  const uint32_t u1 = tail_unit_begin(p + 1, units, args.n_tail);
  uint32_t u = u0;
  for (int k = 0; k < 2 && u < u1; ++k) {
    const uint32_t t_local = u / (uint32_t)args.Q;
    const uint32_t seg_end = min(u1, (t_local + 1) * (uint32_t)args.Q);
    const uint32_t tile_g = args.n_full + t_local;
    const int l = find_layer(args, tile_g);
    const TrEntry& E = args.L[l];
    const int tile = (int)(tile_g - E.tile_begin);
    const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
    const uint32_t qa = u - t_local * (uint32_t)args.Q, qb = seg_end - t_local * (uint32_t)args.Q;
    const float c = tr_segment<true>(E, tm, tn, qa, qb, args.factors, lds, ln, acc);
    store_tile(args.partials + (int64_t)(2 * p + k) * kTrTile * kTrTile, kTrTile, acc, c, false);
    u = seg_end;
  }
}

// Adds the tail partials of every tail tile in worker order (deterministic) and
// writes grad = (accumulate ? grad : 0) + sum. One workgroup per 1024 elements
// (256 threads x 4 consecutive elements), 64 workgroups per tile.
__global__ __launch_bounds__(256) void tr_fixup_kernel(TrArgs args) {
  const uint32_t n_tail_tiles = args.n_tiles - args.n_full;
  const uint32_t chunk = blockIdx.x;                 // 64 chunks of 1024 elements per tile
  const uint32_t t_local = chunk >> 6;
  if (t_local >= n_tail_tiles) return;
  const uint32_t Q = (uint32_t)args.Q;
  const uint64_t units = (uint64_t)n_tail_tiles * Q;
  const uint32_t tb = t_local * Q, te = tb + Q;
  // Contributing workers: ranges [u0(p), u0(p+1)) that intersect [tb, te).
  uint32_t p_first = 0;
  {
    uint32_t lo = 0, hi = args.n_tail - 1;
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) >> 1;
      if (tail_unit_begin(mid, units, args.n_tail) <= tb) lo = mid; else hi = mid - 1;
    }
    p_first = lo;
  }
  const uint32_t tile_g = args.n_full + t_local;
  const int l = find_layer(args, tile_g);
  const TrEntry& E = args.L[l];
  const int tile = (int)(tile_g - E.tile_begin);
  const int tm = tile / E.tiles_n, tn = tile % E.tiles_n;
  const int e = (int)(chunk & 63) * 1024 + threadIdx.x * 4;   // 4 consecutive elements
  const int r = e >> 8, c = e & 255;
  float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
  for (uint32_t p = p_first; p < args.n_tail; ++p) {
    const uint32_t pb = tail_unit_begin(p, units, args.n_tail);
    const uint32_t pe = tail_unit_begin(p + 1, units, args.n_tail);
    if (pb >= te) break;
    if (pe <= tb || pb == pe) continue;
    const int k = pb >= tb ? 0 : 1;                   // first or second segment of worker p
    const float4 v = *reinterpret_cast<const float4*>(
        args.partials + (int64_t)(2 * p + k) * kTrTile * kTrTile + e);
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
  return L.dtype == DPSGD_BF16 && L.d_in % kTrTile == 0 && L.d_out % kTrTile == 0 &&
         L.T % kTrBK == 0;
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
  // Whole tiles for the full rounds over the CUs, then the last partial round's
  // K slices spread evenly over the CUs (only when every tile has the same Q).
  const int64_t rem = tiles % cus;
  if (uniform && n > 0 && rem != 0) {
    plan->n_full = tiles - rem;
    const int64_t units = rem * Q;
    plan->n_tail = units < cus ? units : cus;
  }
  plan->tail_bytes = (size_t)plan->n_tail * 2 * kTrTile * kTrTile * sizeof(float);
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
