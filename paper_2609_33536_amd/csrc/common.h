// Device-side helpers shared by the libekv kernels (internal header).
//
// Layout constants and the BASE expansion: a BASE byte is executed as the
// 16-bit word with that byte in the high position and a zero low byte
// (paper §3.2; App. B.3).  On gfx950 one v_perm_b32 places two bytes of a
// dword into the high halves of a packed pair of 16-bit words.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ekv {

constexpr int kHeadDim = 128;
constexpr int kPage = 16;
constexpr int kTileWords = kPage * kHeadDim;   // one (plane, head) tile: 2048 words = 4 KiB
constexpr int kTileBytes = 2 * kTileWords;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// v_perm_b32(S0, S1, sel): result byte k is byte sel[k] of the 8-byte value
// {S0:S1} (0..3 from S1, 4..7 from S0); selector 0x0C yields 0x00.
__device__ __forceinline__ uint32_t perm(uint32_t s0, uint32_t s1, uint32_t sel) {
  return __builtin_amdgcn_perm(s0, s1, sel);
}

// Bytes b0 b1 (low half of x) -> words {b0<<8, b1<<8}; high half likewise.
__device__ __forceinline__ uint32_t base_words_lo(uint32_t x) { return perm(0u, x, 0x010C000Cu); }
__device__ __forceinline__ uint32_t base_words_hi(uint32_t x) { return perm(0u, x, 0x030C020Cu); }

// 8 BASE bytes -> 8 executed 16-bit words.
__device__ __forceinline__ u32x4 expand_base8(u32x2 b) {
  return u32x4{base_words_lo(b.x), base_words_hi(b.x), base_words_lo(b.y), base_words_hi(b.y)};
}

struct Bf16 {};
struct Fp16 {};

// Matrix-core operations per element type.
//  qk: 16x16x32 product, A/B = 8 elements per lane.
//  pv: 16x16x16 product, A/B = 4 elements per lane.
template <typename T> struct Mma;

template <> struct Mma<Bf16> {
  static __device__ __forceinline__ f32x4 qk(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
  static __device__ __forceinline__ f32x4 pv(u32x2 a, u32x2 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a),
                                                     __builtin_bit_cast(i16x4, b), c, 0, 0, 0);
  }
  // Round to nearest even; returns the 16-bit word and the value it stands for.
  static __device__ __forceinline__ uint16_t round(float x, float* back) {
    __bf16 h = (__bf16)x;
    *back = (float)h;
    return __builtin_bit_cast(uint16_t, h);
  }
  static __device__ __forceinline__ float widen(uint16_t w) {
    return __builtin_bit_cast(float, (uint32_t)w << 16);
  }
};

template <> struct Mma<Fp16> {
  static __device__ __forceinline__ f32x4 qk(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
  static __device__ __forceinline__ f32x4 pv(u32x2 a, u32x2 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a),
                                                 __builtin_bit_cast(f16x4, b), c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint16_t round(float x, float* back) {
    _Float16 h = (_Float16)x;
    *back = (float)h;
    return __builtin_bit_cast(uint16_t, h);
  }
  static __device__ __forceinline__ float widen(uint16_t w) {
    return (float)__builtin_bit_cast(_Float16, w);
  }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace ekv
