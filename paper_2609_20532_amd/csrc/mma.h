// MFMA tile machinery shared by the Gram (ghost-norm) and the transposed-operand
// GEMM kernels (clip-weighted sum, materialised norm).
//
// A workgroup computes a 128x128 fp32 tile with 4 wave64s in a 2x2 grid; each
// wave owns a 64x64 sub-tile as 4x4 blocks of the 16x16 MFMA output.
//
// Both operands of a K step sit in LDS as [row][k] with k contiguous (row
// stride SK = BK + pad elements, 144 bytes for both dtypes), which is the
// layout the 16x16 MFMA operand wants: lane l supplies row (l % 16) and the
// k-slice 8*(l / 16) .. +8 of a 32-wide k chunk.
//   bf16: v_mfma_f32_16x16x32_bf16, one instruction per 16x16 block and k32.
//   fp32: v_mfma_f32_16x16x4_f32, eight instructions per block and k32; the
//         j-th instruction takes element j of each lane's 8-wide k-slice, so
//         the eight together cover the 32 k values once.
// Output element acc[bm][bn][v] of lane l is row bm*16 + 4*(l/16) + v and
// column bn*16 + l%16 of the wave's sub-tile (rows index the first operand).
#pragma once

#include "common.h"

namespace dpsgd {

template <typename TIn> struct TileCfg;
template <> struct TileCfg<uint16_t> {   // bf16 storage
  static constexpr int BK = 64;          // k per step
  static constexpr int SK = 72;          // LDS row stride (elements): 144 bytes
  static constexpr int E = 8;            // elements per 16-byte chunk
};
template <> struct TileCfg<float> {
  static constexpr int BK = 32;
  static constexpr int SK = 36;
  static constexpr int E = 4;
};

constexpr int kTile = 128;                       // workgroup tile edge
template <typename TIn>
constexpr int lds_operand_elems() { return kTile * TileCfg<TIn>::SK; }

__device__ __forceinline__ void zero_acc(f32x4_t (&acc)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
}

__device__ __forceinline__ void scale_acc(f32x4_t (&acc)[4][4], float s) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] *= s;
}

// acc += As[64 rows] . Bs[64 rows]^T over one K step held in LDS.
// As / Bs point at the wave's first row in LDS.
__device__ __forceinline__ void mma_step(const uint16_t* __restrict__ As,
                                         const uint16_t* __restrict__ Bs,
                                         f32x4_t (&acc)[4][4], int lane) {
  constexpr int SK = TileCfg<uint16_t>::SK;
  const int r = lane & 15;
  const int ko = (lane >> 4) * 8;
#pragma unroll
  for (int kc = 0; kc < TileCfg<uint16_t>::BK / 32; ++kc) {
    bf16x8_t a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = *reinterpret_cast<const bf16x8_t*>(As + (i * 16 + r) * SK + kc * 32 + ko);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b[j] = *reinterpret_cast<const bf16x8_t*>(Bs + (j * 16 + r) * SK + kc * 32 + ko);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
}

__device__ __forceinline__ void mma_step(const float* __restrict__ As, const float* __restrict__ Bs,
                                         f32x4_t (&acc)[4][4], int lane) {
  constexpr int SK = TileCfg<float>::SK;
  const int r = lane & 15;
  const int ko = (lane >> 4) * 8;
#pragma unroll
  for (int kc = 0; kc < TileCfg<float>::BK / 32; ++kc) {
    float4 a[4][2], b[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float* p = As + (i * 16 + r) * SK + kc * 32 + ko;
      a[i][0] = *reinterpret_cast<const float4*>(p);
      a[i][1] = *reinterpret_cast<const float4*>(p + 4);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float* p = Bs + (j * 16 + r) * SK + kc * 32 + ko;
      b[j][0] = *reinterpret_cast<const float4*>(p);
      b[j][1] = *reinterpret_cast<const float4*>(p + 4);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][h].x, b[j][h].x, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][h].y, b[j][h].y, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][h].z, b[j][h].z, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][h].w, b[j][h].w, acc[i][j], 0, 0, 0);
        }
    }
  }
}

// Generic bf16 wave tile: acc[MB][NB] += As[MB*16 rows] . Bs[NB*16 rows]^T over one
// K step of BK = 64 in LDS (same operand and output layout as mma_step above).
// With RESCALE, every accumulator block is multiplied by `s` just before its
// first MFMA of the step, so only a few blocks are in flight in VGPRs at a time.
template <int MB, int NB, bool RESCALE = false>
__device__ __forceinline__ void mma_tile_bf16(const uint16_t* __restrict__ As,
                                              const uint16_t* __restrict__ Bs,
                                              f32x4_t (&acc)[MB][NB], int lane, float s = 1.0f) {
  constexpr int SK = TileCfg<uint16_t>::SK;
  const int r = lane & 15;
  const int ko = (lane >> 4) * 8;
#pragma unroll
  for (int kc = 0; kc < TileCfg<uint16_t>::BK / 32; ++kc) {
    bf16x8_t b[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
      b[j] = *reinterpret_cast<const bf16x8_t*>(Bs + (j * 16 + r) * SK + kc * 32 + ko);
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(As + (i * 16 + r) * SK + kc * 32 + ko);
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const f32x4_t c = (RESCALE && kc == 0) ? acc[i][j] * s : acc[i][j];
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[j], c, 0, 0, 0);
      }
    }
  }
}

template <int MB, int NB>
__device__ __forceinline__ void zero_acc_t(f32x4_t (&acc)[MB][NB]) {
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
}

// Multiplies the accumulators by s one block row at a time; the scheduling
// barriers keep the compiler from reading every accumulator register into
// VGPRs at once (the accumulators of large wave tiles live in AGPRs).
template <int MB, int NB>
__device__ __forceinline__ void scale_acc_t(f32x4_t (&acc)[MB][NB], float s) {
#pragma unroll
  for (int i = 0; i < MB; ++i) {
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] *= s;
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Workgroup index remapped so that consecutive logical indices run on the same
// XCD. Workgroups are dispatched round-robin over the 8 XCDs (workgroup b to
// XCD b % 8); this gives XCD x the contiguous logical range of its share, so
// tiles that read the same operand rows share that XCD's L2.
__device__ __forceinline__ uint32_t xcd_logical_index(uint32_t bid, uint32_t nwg) {
  const uint32_t per = nwg >> 3, rem = nwg & 7u, xcd = bid & 7u, idx = bid >> 3;
  return xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}

// xcd_logical_index for a job list of n_first jobs of one kind (whole tiles)
// followed by jobs of another (split tail ranges): every XCD receives an even
// share of each kind, its first-kind jobs as one contiguous range and
// dispatched first, then its share of the rest. With a plain contiguous split
// the first XCDs would hold only whole tiles and finish last.
__device__ __forceinline__ uint32_t xcd_two_class_index(uint32_t bid, uint32_t nwg,
                                                        uint32_t n_first) {
  const uint32_t xcd = bid & 7u, idx = bid >> 3;
  const uint32_t per = nwg >> 3, rem = nwg & 7u;
  const uint32_t fper = n_first >> 3, frem = n_first & 7u;
  const uint32_t f_cnt = fper + (xcd < frem ? 1u : 0u);
  const uint32_t f_begin = xcd * fper + (xcd < frem ? xcd : frem);
  if (idx < f_cnt) return f_begin + idx;
  const uint32_t begin = xcd * per + (xcd < rem ? xcd : rem);
  return n_first + (begin - f_begin) + (idx - f_cnt);
}

// Element loads for the non-vector paths.
__device__ __forceinline__ float load_elem(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ float load_elem(const float* p) { return *p; }

}  // namespace dpsgd
