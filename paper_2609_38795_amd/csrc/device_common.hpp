// Device-side helpers shared by the gfx950 kernels: bf16 storage, MFMA
// operand vectors, wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace alr {

typedef uint16_t bf16;  // bfloat16 bit pattern (storage type)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16 x) { return __uint_as_float(((uint32_t)x) << 16); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// float -> bf16, round to nearest, ties to even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16 f2bf(float f) { return __builtin_bit_cast(bf16, (__bf16)f); }

__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
}

// fp16 storage (partial results whose range is known): two values per word,
// round to nearest even.
typedef _Float16 f16x2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2h(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2v));
}
__device__ __forceinline__ float h_lo(uint32_t w) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
}
__device__ __forceinline__ float h_hi(uint32_t w) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

// Load helpers with a uniform "element type" interface: float or bf16 storage.
template <typename T> struct Elt;
template <> struct Elt<float> {
  __device__ static __forceinline__ float ld(const float* p) { return *p; }
  __device__ static __forceinline__ void st(float* p, float v) { *p = v; }
};
template <> struct Elt<bf16> {
  __device__ static __forceinline__ float ld(const bf16* p) { return bf2f(*p); }
  __device__ static __forceinline__ void st(bf16* p, float v) { *p = f2bf(v); }
};

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// max / sum of v over lanes i and i ^ 32: v_permlane32_swap exchanges the two
// 32-lane halves of the wave in registers (no LDS round trip); the pair it
// returns holds both halves' values in every lane.  All lanes must be active.
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// 2^x on the hardware exp unit (v_exp_f32): results below 2^-126 flush to 0,
// which softmax weights can afford; -inf gives 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Sum / max over each aligned group of LPH (8 or 16) lanes with DPP lane
// permutations inside the 16-lane rows (no LDS round trip): the row (half)
// mirror pairs lane i with its reflection, then the two quad swaps finish the
// group.  Every lane of a group ends with the same bits (each step combines
// a lane with its partner symmetrically).
template <int CTRL>
__device__ __forceinline__ float dpp_perm(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int LPH>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(LPH == 8 || LPH == 16, "lanes per group");
  if constexpr (LPH == 16) v += dpp_perm<0x140>(v);  // row_mirror
  v += dpp_perm<0x141>(v);                           // row_half_mirror
  v += dpp_perm<0xB1>(v);                            // quad_perm [1,0,3,2]
  v += dpp_perm<0x4E>(v);                            // quad_perm [2,3,0,1]
  return v;
}
template <int LPH>
__device__ __forceinline__ float group_max(float v) {
  static_assert(LPH == 8 || LPH == 16, "lanes per group");
  if constexpr (LPH == 16) v = fmaxf(v, dpp_perm<0x140>(v));
  v = fmaxf(v, dpp_perm<0x141>(v));
  v = fmaxf(v, dpp_perm<0xB1>(v));
  v = fmaxf(v, dpp_perm<0x4E>(v));
  return v;
}

template <int CTRL>
__device__ __forceinline__ int dpp_perm_i(int v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ int group_min16_i(int v) {
  v = min(v, dpp_perm_i<0x140>(v));
  v = min(v, dpp_perm_i<0x141>(v));
  v = min(v, dpp_perm_i<0xB1>(v));
  v = min(v, dpp_perm_i<0x4E>(v));
  return v;
}

// max / sum / min of v over lanes i and i ^ 16 (the two 16-lane rows of each
// 32-lane half): v_permlane16_swap exchanges rows 0 <-> 1 and 2 <-> 3 in
// registers; the pair it returns holds both rows' values in every lane.  Both
// rows of a half must be active.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ int min_xor16_i(int v) {
  const auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
  return min((int)r[0], (int)r[1]);
}

}  // namespace alr
