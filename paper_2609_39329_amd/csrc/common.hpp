// Device-side helpers shared by the PatchKV kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, each with its own L2

#define PKV_LDS __attribute__((address_space(3)))

// f(integral_constant<int, I>) for I = 0..N-1, unrolled at compile time
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// D(32x32, f32) += A(32x16, bf16) * B(16x32, bf16).
// Lane l holds A[row l%32][k (l/32)*8 + t] and B[k (l/32)*8 + t][col l%32], t = 0..7;
// D element 4j+i of lane l is D[8j + 4(l/32) + i][l%32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// D(32x32, f32) += A(32x2, f32) * B(2x32, f32); lane l holds A[l%32][l/32] and
// B[l/32][l%32]; D layout as mfma32.
__device__ __forceinline__ f32x16 mfma32_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Transposing LDS read (ds_read_b64_tr_b16). Within each group of 16 lanes, input
// lane 4r+q points at 4 consecutive 16-bit elements (row r, columns 4q..4q+3 of a
// 4x16 block); output lane j of the group receives column j: element r of the
// result is row r's column j.
__device__ __forceinline__ bf16x4 lds_read_tr16(const PKV_LDS __bf16* p) {
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((PKV_LDS i16x4*)(p));
  return __builtin_bit_cast(bf16x4, v);
}

__device__ __forceinline__ bf16x8 cat8(bf16x4 lo, bf16x4 hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Values of lane l and lane l^32, in some order (v_permlane32_swap of x with x).
struct Pair {
  float a, b;
};
__device__ __forceinline__ Pair swap32(float x) {
  unsigned u = __builtin_bit_cast(unsigned, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return {__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1])};
}
__device__ __forceinline__ float pair_max(float x) {
  Pair p = swap32(x);
  return fmaxf(p.a, p.b);
}
__device__ __forceinline__ float pair_sum(float x) {
  Pair p = swap32(x);
  return p.a + p.b;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

// bf16(a) in the low half and bf16(b) in the high half of a dword, rounded to nearest
// even: one v_cvt_pk_bf16_f32, selected by the compiler (which then also inserts the
// wait states an MFMA reading the result needs; an inline-asm conversion hides the
// write from its hazard checks)
__device__ __forceinline__ unsigned pack_bf16(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

__device__ __forceinline__ bf16x8 load_bf16x8(const __bf16* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// Work-item index of this workgroup such that consecutive work items land on the
// same XCD (workgroups are dispatched round-robin over the XCDs).
__device__ __forceinline__ int xcd_item(int per_xcd) {
  int b = blockIdx.x;
  return (b % kXcds) * per_xcd + b / kXcds;
}

}  // namespace pkv
