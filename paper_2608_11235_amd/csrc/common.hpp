// Shared device helpers for the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cora.h"

constexpr int CORA_MAX_BLOCK = CORA_MAX_BLOCK_LEN;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 bits (lo in the low half), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// float -> bf16 bits, round to nearest even.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) { return __builtin_bit_cast(bf16x8_t, v); }

// Map a linear workgroup id so that each XCD (workgroups are dealt to the 8
// XCDs round-robin) receives a contiguous range of logical tiles: tiles that
// share an operand then share one L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int xcd = bid & 7, slot = bid >> 3;
  const int per = nblocks >> 3, rem = nblocks & 7;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---- softmax statistics of a row (Eq. 1) ---------------------------------------------------
// Partial (max, sum of exp(l - max), lowest index holding the max) over a set of logits;
// an empty set is (-inf, 0, INT_MAX).
struct TopState {
  float m, s;
  int arg;
};

constexpr float LOG2E = 1.4426950408889634f;

// 2^x with the hardware v_exp_f32: results below 2^-126 flush to zero, which cannot change
// a softmax sum that already holds the max term (1.0)
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Union of two partials; on equal maxima the lower index wins, so folding partials in any
// fixed order gives the first occurrence of the maximum.
__device__ __forceinline__ TopState merge(TopState x, TopState y) {
  TopState r;
  r.m = fmaxf(x.m, y.m);
  const float sx = x.m == -INFINITY ? 0.f : x.s * fast_exp2((x.m - r.m) * LOG2E);
  const float sy = y.m == -INFINITY ? 0.f : y.s * fast_exp2((y.m - r.m) * LOG2E);
  r.s = sx + sy;
  r.arg = x.m > y.m ? x.arg : (y.m > x.m ? y.arg : min(x.arg, y.arg));
  return r;
}
