// Device-side helpers shared by the prefill and decode kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// 16 bytes as a native vector (not HIP's uint4 struct): arrays of these stay
// in registers, while struct arrays copied element-wise end up in scratch.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_inff();

// Element-type traits: the 8-wide MFMA operand vector, a 32x32x16 MFMA with
// fp32 accumulation, round-to-nearest-even packing of two floats, and the
// fp32 dot product of two packed pairs.
template <typename T> struct Elem;

template <> struct Elem<_Float16> {
  typedef f16x8 vec8;
  typedef f16x2 vec2;
  static __device__ __forceinline__ f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack2(float lo, float hi) {
    vec2 v = {(_Float16)lo, (_Float16)hi};
    return __builtin_bit_cast(uint32_t, v);
  }
  static __device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(vec2, a), __builtin_bit_cast(vec2, b), c, false);
  }
  static __device__ __forceinline__ float lo(uint32_t w) {
    return (float)__builtin_bit_cast(vec2, w)[0];
  }
  static __device__ __forceinline__ float hi(uint32_t w) {
    return (float)__builtin_bit_cast(vec2, w)[1];
  }
};

template <> struct Elem<__bf16> {
  typedef bf16x8 vec8;
  typedef bf16x2 vec2;
  static __device__ __forceinline__ f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack2(float lo, float hi) {
    vec2 v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
  }
  static __device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(vec2, a), __builtin_bit_cast(vec2, b), c, false);
  }
  // bf16 -> f32 is a 16-bit shift: exact.
  static __device__ __forceinline__ float lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
  static __device__ __forceinline__ float hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// SoftCap of a score in log2 units (x = s log2 e): cap tanh(s / cap) log2 e,
// from tanh(y) = 1 - 2 / (1 + e^{2y}) with e^{2y} = 2^(x k2); k2 = 2 / cap,
// cl = cap log2 e.  The exponential saturates to inf or 0 for large |x|, which
// gives +-cl exactly.  `add` replaces the final + cl (cl minus an offset
// folds that offset into the same instruction).
__device__ __forceinline__ float soft_cap(float x, float k2, float cl, float add) {
  const float e = fast_exp2(x * k2);
  return __builtin_fmaf(-2.f * cl, __builtin_amdgcn_rcpf(1.f + e), add);
}
__device__ __forceinline__ float soft_cap(float x, float k2, float cl) { return soft_cap(x, k2, cl, cl); }

// K and V tiles live in LDS row-major, [keys][D], with the 16-byte chunks of
// each row XOR-swizzled: chunk c of row r sits at chunk position c ^ swz(r).
// That keeps the K operand reads (16 consecutive rows at one chunk) and the
// transposing V reads (4 consecutive rows x 4 consecutive chunks per
// half-wave) free of bank conflicts; the copy engine writes whole 1 KB
// blocks, so the swizzle is applied on the global side of the copy.
// swz depends on r % 16 only.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if (D == 128) return 4 * (r & 3) + ((r >> 2) & 3);
  return 4 * ((r >> 1) & 1) + ((r >> 2) & 3);
}

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) void lds_void;

// Transposing LDS read: within each 16-lane group, output lane i element j is
// element (i % 4) of the 8 bytes addressed by lane (i / 4 + 4 j).
__device__ __forceinline__ uint2 lds_read_tr(const void* p) {
  v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p));
  return __builtin_bit_cast(uint2, r);
}

// Cross-lane exchange with lane ^ 32 (the other half of a wave64).
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, 64);
}

}  // namespace attn
