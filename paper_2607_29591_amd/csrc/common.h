// Device helpers shared by the ResKV kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reskv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

// Storage element of a bf16 tensor: the upper 16 bits of an fp32.
struct bf16s {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// 8 consecutive elements of a row converted to fp32.
__device__ __forceinline__ void load8_f32(const uint16_t* p, float (&x)[8]) {
  uint4 w = *reinterpret_cast<const uint4*>(p);
  x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x);
  x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
  x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z);
  x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
}
__device__ __forceinline__ void load8_f32(const float* p, float (&x)[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 w) {
  return __builtin_bit_cast(bf16x8_t, w);
}

// wave64 butterflies over the lanes selected by the xor masks
__device__ __forceinline__ float wave_xor_max(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, 64));
}
__device__ __forceinline__ float wave_xor_add(float v, int mask) {
  return v + __shfl_xor(v, mask, 64);
}

// Reductions over the 16 lanes of one DPP row (lanes 16g .. 16g+15) with DPP
// moves: swap neighbours, swap pairs, mirror within 8, mirror within 16. Each
// step combines a lane with a partner that holds the same partial set size,
// and fp32 add and max are commutative, so all 16 lanes end with the same
// bits.
template <int Ctrl>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), Ctrl, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_move<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_move<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_move<0x141>(v));  // row_half_mirror
  return fmaxf(v, dpp_move<0x140>(v));  // row_mirror
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_move<0xB1>(v);
  v += dpp_move<0x4E>(v);
  v += dpp_move<0x141>(v);
  return v + dpp_move<0x140>(v);
}

// 2^x on the hardware exponential unit (no denormal rescaling); 2^-inf = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int clampi(int x, int lo, int hi) {
  return x < lo ? lo : (x > hi ? hi : x);
}

// ---- 16x16 MFMA tiles over a full row of D elements ------------------------
// C[16 x 16] = A[16 x D] . B[16 x D]^T. Lane l supplies A row (l % 16) and B
// row (l % 16); lane group g = l / 16 takes the 16-byte pieces g, g + 4,
// g + 8, ... of the row, so that one load instruction of the wave reads 64
// contiguous bytes of each of 16 rows (whole cache segments). The MFMA k-steps
// walk those pieces in the same order for A and B, so the sum covers every
// element of the row once.
// Result layout: lane l holds C[4*(l/16) + i][l % 16] for i = 0..3.
template <typename T, int D>
struct Frag;

template <int D>
struct Frag<uint16_t, D> {        // bf16: 16x16x32 steps, 8 elements per step
  static constexpr int kSteps = D / 32;
  uint4 w[kSteps];
  __device__ __forceinline__ void load(const uint16_t* row, int grp) {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) w[i] = *reinterpret_cast<const uint4*>(row + 8 * grp + 32 * i);
  }
  __device__ __forceinline__ void store(uint16_t* row, int grp) const {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) *reinterpret_cast<uint4*>(row + 8 * grp + 32 * i) = w[i];
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) w[i] = make_uint4(0, 0, 0, 0);
  }
};

template <int D>
struct Frag<float, D> {           // fp32: 16x16x4 steps, 1 element per step
  static constexpr int kSteps = D / 16;  // float4 groups
  float4 w[kSteps];
  __device__ __forceinline__ void load(const float* row, int grp) {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) w[i] = *reinterpret_cast<const float4*>(row + 4 * grp + 16 * i);
  }
  __device__ __forceinline__ void store(float* row, int grp) const {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) *reinterpret_cast<float4*>(row + 4 * grp + 16 * i) = w[i];
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < kSteps; ++i) w[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
};

template <int D>
__device__ __forceinline__ f32x4_t mma(const Frag<uint16_t, D>& a, const Frag<uint16_t, D>& b, f32x4_t acc) {
#pragma unroll
  for (int i = 0; i < Frag<uint16_t, D>::kSteps; ++i)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a.w[i]), as_bf16x8(b.w[i]), acc, 0, 0, 0);
  return acc;
}

template <int D>
__device__ __forceinline__ f32x4_t mma(const Frag<float, D>& a, const Frag<float, D>& b, f32x4_t acc) {
#pragma unroll
  for (int i = 0; i < Frag<float, D>::kSteps; ++i) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w[i].x, b.w[i].x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w[i].y, b.w[i].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w[i].z, b.w[i].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w[i].w, b.w[i].w, acc, 0, 0, 0);
  }
  return acc;
}

__device__ __forceinline__ f32x4_t zero4() { return f32x4_t{0.f, 0.f, 0.f, 0.f}; }

}  // namespace reskv
