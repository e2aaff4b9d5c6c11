// Internal device helpers shared by the MoE kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lancet_moe.h"

namespace lmoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ------------------------------------------------------------------ bf16 <-> f32
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// Two floats to bf16 (lo in bits 0..15), round to nearest, ties to even, NaN
// stays NaN: gfx950's v_cvt_pk_bf16_f32, one instruction for the pair (a
// software rounding with its NaN test compiles to a divergent branch per
// value).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

// A 16-byte vector of 8 bf16 or 4 f32 elements, unpacked to float.
template <typename T> struct Vec;
template <> struct Vec<uint16_t> {       // bf16 storage
  static constexpr int N = 8;
  __device__ static void load(const void* p, float* v) {
    u32x4 r = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(r[i] << 16);
      v[2 * i + 1] = __uint_as_float(r[i] & 0xffff0000u);
    }
  }
  __device__ static void store(void* p, const float* v) {
    u32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    *reinterpret_cast<u32x4*>(p) = r;
  }
};
template <> struct Vec<float> {
  static constexpr int N = 4;
  __device__ static void load(const void* p, float* v) {
    f32x4 r = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = r[i];
  }
  __device__ static void store(void* p, const float* v) {
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = v[i];
    *reinterpret_cast<f32x4*>(p) = r;
  }
};

// ------------------------------------------------------------ blocked layout
// bf16 [E][C][X] buffers of the expert path (X a multiple of 32) are stored in
// 16 x 32 blocks of 1 KiB: within expert e (Cp = C rounded up to 16 rows),
// element (r, c) sits at e * Cp * X + blk_off(r, c, X).  A 16-row x 32-column
// MFMA operand fragment is then one contiguous 1 KiB run, which the loads
// into LDS move several times faster than 16 separate 64-byte row pieces.
// The same blocks serve both GEMM orientations (rows x K and K x columns).
// float buffers stay row-major (Cp = C).
__host__ __device__ __forceinline__ int64_t blk_off(int64_t r, int64_t c, int64_t X) {
  return ((r >> 4) * (X >> 5) + (c >> 5)) * 512 + (r & 15) * 32 + (c & 31);
}
__host__ __device__ __forceinline__ int64_t pad16(int64_t n) { return (n + 15) & ~(int64_t)15; }

// Offset of (row, col) in one expert's [C][X] buffer for storage type T.
template <typename T> __host__ __device__ __forceinline__ int64_t ebuf_off(int64_t r, int64_t c, int64_t X);
template <> __host__ __device__ __forceinline__ int64_t ebuf_off<uint16_t>(int64_t r, int64_t c, int64_t X) {
  return blk_off(r, c, X);
}
template <> __host__ __device__ __forceinline__ int64_t ebuf_off<float>(int64_t r, int64_t c, int64_t X) {
  return r * X + c;
}

// ------------------------------------------------------------------- wave ops
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  return v;
}

// ------------------------------------------------------------------ activation
__device__ __forceinline__ float act_fwd(float h, int act) {
  switch (act) {
    case MOE_ACT_RELU: return h > 0.f ? h : 0.f;
    case MOE_ACT_GELU_TANH: {
      const float c = 0.7978845608028654f;  // sqrt(2/pi)
      return 0.5f * h * (1.f + tanhf(c * (h + 0.044715f * h * h * h)));
    }
    case MOE_ACT_GELU_ERF: return 0.5f * h * (1.f + erff(h * 0.7071067811865476f));
    default: return h;
  }
}

__device__ __forceinline__ float act_bwd(float h, int act) {
  switch (act) {
    case MOE_ACT_RELU: return h > 0.f ? 1.f : 0.f;
    case MOE_ACT_GELU_TANH: {
      const float c = 0.7978845608028654f;
      float u = c * (h + 0.044715f * h * h * h);
      float th = tanhf(u);
      float du = c * (1.f + 3.f * 0.044715f * h * h);
      return 0.5f * (1.f + th) + 0.5f * h * (1.f - th * th) * du;
    }
    case MOE_ACT_GELU_ERF:
      return 0.5f * (1.f + erff(h * 0.7071067811865476f)) + h * expf(-0.5f * h * h) * 0.3989422804014327f;
    default: return 1.f;
  }
}

// Compile-time activation for the bf16 GEMM epilogues, whose outputs are
// rounded to bf16: GELU-tanh is evaluated as h * s, s = sigmoid(2u), the same
// function as 0.5 h (1 + tanh u), u = sqrt(2/pi) (h + 0.044715 h^3), with the
// hardware base-2 exponential and reciprocal (v_exp_f32, v_rcp_f32: about 1 ulp
// each, far below the bf16 rounding of the result; an IEEE division would cost
// about ten instructions per element).  The constants are folded so that
// exp(-2u) = 2^(h (c1 + c2 h^2)), c1 = -2 sqrt(2/pi) log2(e),
// c2 = 0.044715 c1: one multiply-add and one multiply ahead of the exponential.
__device__ __forceinline__ float gelu_tanh_sig(float h, float h2) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(h * fmaf(-0.10294324f, h2, -2.3022082f)));
}

template <int ACT>
__device__ __forceinline__ float act_fwd_t(float h) {
  if constexpr (ACT == MOE_ACT_RELU) return h > 0.f ? h : 0.f;
  else if constexpr (ACT == MOE_ACT_GELU_TANH) {
    return h * gelu_tanh_sig(h, h * h);
  } else if constexpr (ACT == MOE_ACT_GELU_ERF) return 0.5f * h * (1.f + erff(h * 0.7071067811865476f));
  else return h;
}

template <int ACT>
__device__ __forceinline__ float act_bwd_t(float h) {
  if constexpr (ACT == MOE_ACT_RELU) return h > 0.f ? 1.f : 0.f;
  else if constexpr (ACT == MOE_ACT_GELU_TANH) {
    // d/dh [h s] = s + h s (1 - s) (2u)' = s (1 + h (1 - s) (2u)'),
    // (2u)' = 2 sqrt(2/pi) (1 + 3 * 0.044715 h^2)
    const float h2 = h * h;
    const float sg = gelu_tanh_sig(h, h2);
    return sg * fmaf(h * (1.f - sg), fmaf(0.21406445f, h2, 1.5957691f), 1.f);
  } else if constexpr (ACT == MOE_ACT_GELU_ERF)
    return 0.5f * (1.f + erff(h * 0.7071067811865476f)) + h * expf(-0.5f * h * h) * 0.3989422804014327f;
  else return 1.f;
}

}  // namespace lmoe
