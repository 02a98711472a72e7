// Shared device helpers for the gfx950 paged-attention kernels.
//
// Matrix-core operand layouts (v_mfma_f32_16x16x32_bf16 and
// v_mfma_f32_32x32x16_bf16, wave64), as used throughout:
//   16x16x32: A[m][k]: lane l holds m = l%16, k = 8*(l/16) + j (j = 0..7)
//             B[k][n]: lane l holds n = l%16, k = 8*(l/16) + j
//             D[m][n]: lane l holds n = l%16, m = 4*(l/16) + i (i = 0..3)
//   32x32x16: A[m][k]: m = l%32, k = 8*(l/32) + j
//             B[k][n]: n = l%32, k = 8*(l/32) + j
//             D[m][n]: n = l%32, m = 8*(i/4) + 4*(l/32) + i%4 (i = 0..15)
// Both kernels compute the transposed score tile S^T = K Q^T, so that one
// lane owns one query row (column n) and row max / row sum reduce mostly
// inside a lane, finishing with permlane16/permlane32 swaps.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace pa {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Butterfly exchanges across lane halves (xor 32) and 16-lane rows (xor 16).
__device__ __forceinline__ float xor32_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor16_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor16_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// fp32 -> bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

// 4 OCP e4m3fn bytes -> 4 bf16 (exact), packed in two dwords.
__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t w) {
  bf16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  bf16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
  u32x2 r;
  r[0] = __builtin_bit_cast(uint32_t, lo);
  r[1] = __builtin_bit_cast(uint32_t, hi);
  return r;
}

// 16 fp8 bytes -> two bf16x8 operands (first 8 values, last 8 values).
__device__ __forceinline__ void fp8x16_to_bf16(const u32x4& w, bf16x8& a, bf16x8& b) {
  u32x2 p0 = fp8x4_to_bf16x4(w[0]), p1 = fp8x4_to_bf16x4(w[1]);
  u32x2 p2 = fp8x4_to_bf16x4(w[2]), p3 = fp8x4_to_bf16x4(w[3]);
  u32x4 ua = {p0[0], p0[1], p1[0], p1[1]};
  u32x4 ub = {p2[0], p2[1], p3[0], p3[1]};
  a = __builtin_bit_cast(bf16x8, ua);
  b = __builtin_bit_cast(bf16x8, ub);
}

__device__ __forceinline__ u32x4 ld16(const void* p) {
  return __builtin_nontemporal_load((const u32x4*)p);
}
__device__ __forceinline__ u32x4 ld16_cached(const void* p) { return *(const u32x4*)p; }

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Physical block holding logical key position p of a sequence, read from its
// block-table row and clamped into [0, num_blocks) so that a corrupt table
// can never address memory outside the cache.
__device__ __forceinline__ int page_of(const int32_t* bt_row, int p, const BlockDiv& bd, int num_blocks) {
  int b = bt_row[bd.block(p)];
  b = b < 0 ? 0 : b;
  return b >= num_blocks ? num_blocks - 1 : b;
}

// Block-wide exclusive scan of NV values per thread (NT threads, a multiple
// of 64), all in one pass; tot[] receives the block totals.  Every thread of
// the block must call it (it synchronises the block).
template <int NV, int NT>
__device__ void block_scan(const int (&v)[NV], int (&ex)[NV], int (&tot)[NV]) {
  __shared__ int wsum[NV][NT / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) x[i] = v[i];
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int y = __shfl_up(x[i], o);
      if (lane >= o) x[i] += y;
    }
  }
  if (lane == 63)
#pragma unroll
    for (int i = 0; i < NV; ++i) wsum[i][w] = x[i];
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int t = lane < NT / 64 ? wsum[i][lane] : 0;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(t, o);
        if (lane >= o) t += y;
      }
      if (lane < NT / 64) wsum[i][lane] = t;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    ex[i] = (w > 0 ? wsum[i][w - 1] : 0) + x[i] - v[i];
    tot[i] = wsum[i][NT / 64 - 1];
  }
  __syncthreads();
}

}  // namespace pa
