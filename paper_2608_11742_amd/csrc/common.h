// Shared device helpers for the gfx950 (CDNA4) kernels: element types,
// 16-byte chunk loads, MFMA wrappers and 64-lane wave reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dllm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// bfloat16 storage is raw 16-bit words
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// float -> bfloat16, round to nearest even (NaN stays NaN)
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

// Element traits: how many elements one 16-byte chunk holds and how an
// element converts to and from float.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int per_chunk = 4;
  static constexpr int bytes = 4;
  __device__ __forceinline__ static float to_f(float v) { return v; }
  __device__ __forceinline__ static float from_f(float v) { return v; }
};
template <> struct Elem<bf16_t> {
  static constexpr int per_chunk = 8;
  static constexpr int bytes = 2;
  __device__ __forceinline__ static float to_f(bf16_t v) { return bf2f(v.bits); }
  __device__ __forceinline__ static bf16_t from_f(float v) { return bf16_t{f2bf(v)}; }
};

// two floats -> two bfloat16 in one word (a in the low half), hardware
// round to nearest even
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {static_cast<__bf16>(a), static_cast<__bf16>(b)};
  return __builtin_bit_cast(uint32_t, v);
}

// two floats -> two IEEE binary16 values in one word (a in the low half),
// hardware round to nearest even
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  const f16x2_t v = {static_cast<_Float16>(a), static_cast<_Float16>(b)};
  return __builtin_bit_cast(uint32_t, v);
}

// the two binary16 halves of a word as floats (exact)
__device__ __forceinline__ float f16_lo(uint32_t w) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xffffu)));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
}

// Attention values (V, stored transposed as V^T) of bf16 models are kept as
// IEEE binary16, saturated to its finite range (+-65504): the P V product
// then runs on fp16 MFMAs with the probabilities in fp16 (11 significant
// bits against bf16's 8).
__device__ __forceinline__ float vt_sat(float v) { return __builtin_amdgcn_fmed3f(v, -65504.0f, 65504.0f); }
__device__ __forceinline__ uint32_t pack_vt2(float a, float b) { return pack_f16x2(vt_sat(a), vt_sat(b)); }
__device__ __forceinline__ void store_vt(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_vt(bf16_t* p, float v) { p->bits = uint16_t(pack_vt2(v, 0.f)); }

// silu(g) = g / (1 + e^-g) with the hardware base-2 exponential and
// reciprocal (about 1 ulp each)
__device__ __forceinline__ float silu_fast(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * g));
}

__device__ __forceinline__ float load_f(const float* p) { return *p; }
__device__ __forceinline__ float load_f(const bf16_t* p) { return bf2f(p->bits); }
__device__ __forceinline__ void store_f(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_f(bf16_t* p, float v) { p->bits = f2bf(v); }

// One MFMA "k-step" over a 16-byte chunk per lane for a 16x16 output block.
// bf16: one v_mfma_f32_16x16x32_bf16 (8 elements per lane, 32 k per step).
// f32:  four v_mfma_f32_16x16x4_f32, element j of every lane's chunk forms
//       step j; A and B use the same lane -> k assignment, so the sum over k
//       is the full dot product regardless of the hardware's k order.
// Output layout of a 16x16 block (both): lane l, element i holds
// D[4 * (l / 16) + i][l % 16].
// 16x16 block, 32 k per step, IEEE binary16 operands (8 per lane)
struct MfmaF16 {
  __device__ __forceinline__ static void run(f32x4& acc, u32x4 a, u32x4 b) {
    typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc, 0,
                                                 0, 0);
  }
};

template <typename T> struct Mfma;
template <> struct Mfma<bf16_t> {
  __device__ __forceinline__ static void run(f32x4& acc, u32x4 a, u32x4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  __device__ __forceinline__ static void run(f32x4& acc, u32x4 a, u32x4 b) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[j]), __uint_as_float(b[j]), acc, 0, 0, 0);
  }
};

// 64-lane reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// (value, id) ordering used by every argmax / top-k: larger value first,
// then smaller id.
__device__ __forceinline__ bool better(float v, int i, float w, int j) {
  return v > w || (v == w && i < j);
}

__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float w = __shfl_xor(v, o, 64);
    int j = __shfl_xor(i, o, 64);
    if (better(w, j, v, i)) { v = w; i = j; }
  }
}

// exp(x) for x <= 0 via the hardware base-2 exponential
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace dllm
