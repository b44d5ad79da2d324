// Device-side building blocks shared by every kernel of the library: slice loads
// and code unpacking for the tile layout declared in include/subspec.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace subspec {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
// Native 128-bit vector (HIP's uint4 is a wrapper struct that register promotion
// does not always split).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Bias added to every unpacked code: the 16-bit field 0x4300 | q is the bf16 value
// 128 + q exactly (exponent 2^7, seven mantissa bits of weight 1), for q < 128.
constexpr uint32_t kPairBias = 0x43004300u;
constexpr float kCodeBias = 128.0f;

// Raw words of one slice (4*BITS bytes, one per lane of a tile).
template <int BITS>
struct Slice {
  uint32_t w[BITS];
};

template <int BITS>
__device__ __forceinline__ Slice<BITS> load_slice(const uint8_t* __restrict__ p) {
  Slice<BITS> s;
  if constexpr (BITS == 4) {
    uint4 v = *reinterpret_cast<const uint4*>(p);
    s.w[0] = v.x; s.w[1] = v.y; s.w[2] = v.z; s.w[3] = v.w;
  } else if constexpr (BITS == 2) {
    uint2 v = *reinterpret_cast<const uint2*>(p);
    s.w[0] = v.x; s.w[1] = v.y;
  } else {
    struct __attribute__((packed, aligned(4))) U3 { uint32_t a, b, c; };
    U3 v = *reinterpret_cast<const U3*>(p);
    s.w[0] = v.a; s.w[1] = v.b; s.w[2] = v.c;
  }
  return s;
}

// Raw buffer resource over `bytes` bytes at p (32-bit offsets from one scalar base,
// so address arithmetic stays in 32 bits).  Word 3 selects the 32-bit data format
// raw buffer accesses need on CDNA; loads at offsets past `bytes` return zeros.
constexpr int kBufferWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes),
                                           kBufferWord3);
}

// Cache policy of the weight stream: non-temporal (every weight byte is read once per
// launch), which keeps the activations and scales that are re-read in the caches.
// Measured on the 7B MLP step: +3-5 % over the default policy.
constexpr int kStreamPolicy = 2;  // nt

template <int BITS>
__device__ __forceinline__ Slice<BITS> load_slice(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  Slice<BITS> s;
  if constexpr (BITS == 4) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kStreamPolicy);
    s.w[0] = v[0]; s.w[1] = v[1]; s.w[2] = v[2]; s.w[3] = v[3];
  } else if constexpr (BITS == 2) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kStreamPolicy);
    s.w[0] = v[0]; s.w[1] = v[1];
  } else {
    const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, off, 0, kStreamPolicy);
    s.w[0] = v[0]; s.w[1] = v[1]; s.w[2] = v[2];
  }
  return s;
}

// (a & mask) | bias in one VALU instruction: gfx950's three-input bitwise
// v_bitop3_b32 with truth table 0xEA (inputs weighted 0xF0, 0xCC, 0xAA).  Through
// the builtin, not inline assembly, so the compiler sees the instruction and keeps
// the wait states a matrix-core read of its result needs.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t mask, uint32_t bias) {
  return __builtin_amdgcn_bitop3_b32(a, mask, bias, 0xEA);
}

// Unpack a slice into its 16 pairs.  pr[p] holds (0x4300 | q_even) in the low and
// (0x4300 | q_odd) in the high 16 bits, i.e. two bf16 values 128 + q; pair p covers
// elements e = 2*(p%4), 2*(p%4)+1 of step p/4.
template <int BITS>
__device__ __forceinline__ void unpack_pairs(const Slice<BITS>& s, uint32_t pr[16]) {
  const uint32_t bias = kPairBias;
  if constexpr (BITS == 4) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t d = s.w[j];
      pr[4 * j + 0] = and_or(d, 0x000F000Fu, bias);
      pr[4 * j + 1] = and_or(d >> 4, 0x000F000Fu, bias);
      pr[4 * j + 2] = and_or(d >> 8, 0x000F000Fu, bias);
      pr[4 * j + 3] = and_or(d >> 12, 0x000F000Fu, bias);
    }
  } else if constexpr (BITS == 2) {
#pragma unroll
    for (int w = 0; w < 2; ++w) {
      const uint32_t d = s.w[w];
#pragma unroll
      for (int t = 0; t < 8; ++t) pr[8 * w + t] = and_or(d >> (2 * t), 0x00030003u, bias);
    }
  } else {
#pragma unroll
    for (int w = 0; w < 3; ++w) {
      const uint32_t d = s.w[w];
#pragma unroll
      for (int t = 0; t < 5; ++t) pr[5 * w + t] = and_or(d >> (3 * t), 0x00070007u, bias);
    }
    uint32_t p15 = and_or(s.w[0] >> 15, 0x00010001u, bias);
    p15 = and_or(s.w[1] >> 14, 0x00020002u, p15);
    pr[15] = and_or(s.w[2] >> 13, 0x00040004u, p15);
  }
}

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, h));
}

// fp32 -> bf16, round to nearest even (hardware conversion on gfx950).
__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

}  // namespace subspec
