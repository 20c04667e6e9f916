// Device-side helpers shared by the rollout-attention kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ra {

constexpr int kPage = 16;        // tokens per page
constexpr int kHeadDim = 128;    // head dimension
constexpr int kWave = 64;        // CDNA wavefront width

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte global load of 8 bf16 (one dwordx4 per lane).
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ u32x4 load_u32x4(const uint16_t *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

// 16-byte global load marked nontemporal (the load's nt bit): for data read
// once, whose cache lines are each taken whole by one load instruction.
__device__ __forceinline__ u32x4 load_stream_u32x4(const void *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ void store_u32x4(uint16_t *p, u32x4 v) {
  *reinterpret_cast<u32x4 *>(p) = v;
}

// D(16x16, fp32) += A(16x32, bf16) * B(32x16, bf16) on the matrix cores.
// Lane l supplies A row (l % 16) and B column (l % 16), eight consecutive
// contraction slots each (slot group l / 16); it receives D rows
// 4 * (l / 16) + 0..3 of column l % 16.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Round 8 fp32 values to bf16 (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 to_bf16x8(f32x8 v) {
  return __builtin_convertvector(v, bf16x8);
}

__device__ __forceinline__ f32x8 to_f32x8(bf16x8 v) {
  return __builtin_convertvector(v, f32x8);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Rotary position embedding of eight dims of a 128-dim head row, pairing dim
// i with dim i + 64: for the lower dims (upper = false) x c - y s, for the
// upper ones x c + y s, where x are the eight dims, y their partners and
// c, s the cosines and sines of the pairs' angles. Each product and the sum
// are rounded to fp32 separately (no fused multiply-add), the result to bf16
// (round to nearest even).
__device__ __forceinline__ bf16x8 rope8(bf16x8 x, bf16x8 y, f32x8 c, f32x8 s, bool upper) {
#pragma clang fp contract(off)
  const f32x8 xf = to_f32x8(x), yf = to_f32x8(y);
  const f32x8 a = xf * c, b = yf * s;
  return to_bf16x8(upper ? a + b : a - b);
}

// Max / sum over the four lanes that share a matrix column (lanes l, l^16,
// l^32, l^48).
__device__ __forceinline__ float col_max4(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

__device__ __forceinline__ float col_sum4(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// ---- fp8 pools: OCP E4M3 codes ----
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Eight E4M3 codes (byte i of the pair of words = element i) -> bf16, exact:
// every E4M3 value is a bf16 value.
__device__ __forceinline__ bf16x8 fp8x8_to_bf16x8(u32x2 w) {
  const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, false);
  const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], 1.0f, true);
  const bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, false);
  const bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], 1.0f, true);
  return bf16x8{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// E4M3 codes of two fp32 values in the low 16 bits (element 0 in byte 0):
// round to nearest even, saturated to +-448 (infinities included), NaN ->
// 0x7F.
__device__ __forceinline__ uint32_t fp8_pair(float x, float y) {
  const float cx = fminf(fmaxf(x, -448.f), 448.f), cy = fminf(fmaxf(y, -448.f), 448.f);
  uint32_t w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(cx, cy, 0, false) & 0xffffu;
  w = x != x ? ((w & 0xff00u) | 0x7fu) : w;
  w = y != y ? ((w & 0x00ffu) | 0x7f00u) : w;
  return w;
}

// Eight bf16 values (16 bytes) -> eight E4M3 codes of x * inv_scale (the
// product rounded to fp32).
__device__ __forceinline__ u32x2 quantize8(u32x4 v, float inv_scale) {
  u32x2 r;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t lo = fp8_pair(__uint_as_float(v[2 * h] << 16) * inv_scale,
                                 __uint_as_float(v[2 * h] & 0xffff0000u) * inv_scale);
    const uint32_t hi = fp8_pair(__uint_as_float(v[2 * h + 1] << 16) * inv_scale,
                                 __uint_as_float(v[2 * h + 1] & 0xffff0000u) * inv_scale);
    r[h] = lo | (hi << 16);
  }
  return r;
}

__device__ __forceinline__ int clamp_page(int id, int num_pages) {
  return min(max(id, 0), num_pages - 1);
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace ra
