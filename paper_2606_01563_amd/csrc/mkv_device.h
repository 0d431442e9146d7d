// Device-side building blocks shared by the MomentKV kernels (gfx950 / CDNA4, wave64).
//
//   * element access for fp32 and bf16 (bf16 kept as uint16 bit patterns, RNE rounding)
//   * 8-element MFMA fragments: a lane holds 8 consecutive elements along the
//     contraction index, so fp32 and bf16 operands are loaded the same way
//   * 16x16 MFMA tile product for both element types
//   * 16-lane row reductions through DPP and 64-lane wave reductions
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint16_t bf16_t;  // storage type of bf16 tensors

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf2f(bf16_t x) { return __uint_as_float((uint32_t)x << 16); }

__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);                                             // RNE
  return (bf16_t)(u >> 16);
}

template <class T> __device__ __forceinline__ float to_f(T x);
template <> __device__ __forceinline__ float to_f<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f<bf16_t>(bf16_t x) { return bf2f(x); }

template <class T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float x) { return f2bf(x); }

// ---------------------------------------------------------------- MFMA fragments
template <class T> struct Frag;
template <> struct Frag<bf16_t> { typedef bf16x8 type; };
template <> struct Frag<float> { typedef f32x8 type; };

// 8 consecutive elements starting at p (16-byte aligned for bf16, 32-byte for fp32).
__device__ __forceinline__ bf16x8 load_frag(const bf16_t* p) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  return __builtin_bit_cast(bf16x8, u);
}
__device__ __forceinline__ f32x8 load_frag(const float* p) {
  float4 a = reinterpret_cast<const float4*>(p)[0];
  float4 b = reinterpret_cast<const float4*>(p)[1];
  f32x8 r;
  r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
  r[4] = b.x; r[5] = b.y; r[6] = b.z; r[7] = b.w;
  return r;
}

// The converse of load_frag.
__device__ __forceinline__ void store_frag(bf16_t* p, const bf16x8& f) {
  *reinterpret_cast<uint4*>(p) = __builtin_bit_cast(uint4, f);
}
__device__ __forceinline__ void store_frag(float* p, const f32x8& f) {
  reinterpret_cast<float4*>(p)[0] = make_float4(f[0], f[1], f[2], f[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(f[4], f[5], f[6], f[7]);
}

// Compile-time choice between two types.
template <bool C, class A, class B> struct Pick { typedef A type; };
template <class A, class B> struct Pick<false, A, B> { typedef B type; };

template <class T> __device__ __forceinline__ typename Frag<T>::type zero_frag();
template <> __device__ __forceinline__ bf16x8 zero_frag<bf16_t>() {
  return __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
}
template <> __device__ __forceinline__ f32x8 zero_frag<float>() {
  f32x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = 0.f;
  return r;
}

// Element access.  Elements of a bf16 fragment are read through a bit cast of the whole
// vector to 16-bit integers: a bit cast of a single __bf16 vector element does not select
// the element on this toolchain.
__device__ __forceinline__ bf16_t raw_elem(const bf16x8& f, int e) {
  const u16x8 u = __builtin_bit_cast(u16x8, f);
  return u[e];
}
__device__ __forceinline__ float raw_elem(const f32x8& f, int e) { return f[e]; }
__device__ __forceinline__ float elem_f(const bf16x8& f, int e) { return bf2f(raw_elem(f, e)); }
__device__ __forceinline__ float elem_f(const f32x8& f, int e) { return f[e]; }

// C(16x16) += A(16x32) * B(32x16).  Lane l supplies A[l%16][8*(l/16) + e] and
// B[8*(l/16) + e][l%16], e = 0..7, and holds C[4*(l/16) + i][l%16], i = 0..3.
// bf16: one v_mfma_f32_16x16x32_bf16.  fp32: eight v_mfma_f32_16x16x4f32, the e-th one
// pairing element e of every lane (the 32-long contraction is covered in another order,
// which only changes the summation order).
__device__ __forceinline__ void mma(f32x4& c, const bf16x8& a, const bf16x8& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4& c, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
}

// An MFMA operand fragment read transposed from a row-major bf16 tile in LDS whose rows
// run along the contraction: lane l receives tile[r0 + 8 (l / 16) + e][c0 + l % 16],
// e = 0..7 (the B layout above with the tile's columns as n; the A layout with them as
// m).  ds_read_b64_tr_b16 hands each group of 16 lanes a 4 x 16 block whose row m is read
// by lanes 4m .. 4m + 3 (eight bytes each) and gives lane j the block's column j; two
// such reads cover the eight rows.  ld (elements) and c0 keep every read 8-byte aligned.
__device__ __forceinline__ bf16x8 lds_frag_tr(const bf16_t* tile, int ld, int r0, int c0, int lane) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const int i = lane & 15;
  const bf16_t* p = tile + (r0 + 8 * (lane >> 4) + (i >> 2)) * ld + c0 + 4 * (i & 3);
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * ld));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ f32x4 zero4() {
  f32x4 r;
  r[0] = r[1] = r[2] = r[3] = 0.f;
  return r;
}

// ---------------------------------------------------------------- lane reductions
// DPP row_ror:n rotates within each row of 16 lanes; the butterfly below leaves the
// same value in all 16 lanes of a row (every step combines a commutative pair).
template <int CTRL> __device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int CTRL> __device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f<0x128>(x);
  x += dpp_f<0x124>(x);
  x += dpp_f<0x122>(x);
  x += dpp_f<0x121>(x);
  return x;
}
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_f<0x128>(x));
  x = fmaxf(x, dpp_f<0x124>(x));
  x = fmaxf(x, dpp_f<0x122>(x));
  x = fmaxf(x, dpp_f<0x121>(x));
  return x;
}
// Sum over the lanes of a quad (4 consecutive lanes), same value in all four.
__device__ __forceinline__ float quad_sum(float x) {
  x += dpp_f<0xB1>(x);  // quad_perm [1,0,3,2]
  x += dpp_f<0x4E>(x);  // quad_perm [2,3,0,1]
  return x;
}
// Sum over lanes l, l^16, l^32, l^48 (the four 16-lane rows), same value in each.
__device__ __forceinline__ float cross_row_sum(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}
__device__ __forceinline__ float cross_row_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) { return cross_row_sum(row16_sum(x)); }
__device__ __forceinline__ float wave_max(float x) { return cross_row_max(row16_max(x)); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Online (max, sum) pair in the base-2 domain: represents sum_i 2^(x_i) = l * 2^m.
__device__ __forceinline__ void ml_merge(float& m, float& l, float m2, float l2) {
  float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;  // both empty
  l = l * fast_exp2(m - mn) + l2 * fast_exp2(m2 - mn);
  m = mn;
}

}  // namespace mkv
