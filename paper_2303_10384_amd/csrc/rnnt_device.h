// Device helpers shared by the three kernels of the RNN-T / W-Transducer path
// (gfx950, wave64).  No host code here.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rnnt {

constexpr float kLog2eF = 1.4426950408889634f;
constexpr float kLn2F = 0.6931471805599453f;
constexpr double kLog2eD = 1.4426950408889634;
constexpr int kWave = 64;

// Per-row record handed from the posterior kernel to the gradient kernel.
// lse2 = ln(sum_v exp z_v) * log2(e); occ_* are the blank / label arc
// posteriors leaving the row's node; label is y_{u+1}, or kNoLabel on the top
// row, or kZeroRow for rows whose gradient is identically zero (padding, bad
// utterances).
struct __attribute__((aligned(16))) RowInfo {
  float lse2;
  float occ_blank;
  float occ_label;
  int32_t label;
};
constexpr int32_t kNoLabel = -1;
constexpr int32_t kZeroRow = -2;

// Lattice scores are kept in log2 units (x * log2 e).  An absent arc, and a
// node that no path reaches, carry kNoArc: finite, so sums and maxima never
// meet -inf - -inf, and so far below any real score that it is exactly
// absorbed by them (kNoArc + any score of magnitude < 1e284 == kNoArc).
constexpr double kNoArc = -0x1p+1000;

// exp2 / log2 on the transcendental unit (v_exp_f32 / v_log_f32, ~1 ulp).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// log2(2^x + 2^y) with float64 operands and result.  The correction term
// log2(1 + 2^-|x-y|) lies in [0, 1] and is formed in float32 (absolute error
// ~1e-7), so the long chains of float64 additions keep their accuracy.  A NaN
// operand gives NaN (|x-y| is NaN); two kNoArc operands give kNoArc.
__device__ __forceinline__ double log_add2(double x, double y) {
  const double m = __builtin_fmax(x, y);
  const float d = static_cast<float>(x - y);
  const float c = fast_log2(1.0f + fast_exp2(-__builtin_fabsf(d)));
  return m + static_cast<double>(c);
}

// ---- element types: 16-byte chunks of logits / gradient -------------------

template <typename T>
struct ElemTraits;

template <>
struct ElemTraits<float> {
  static constexpr int kPerChunk = 4;
  __device__ static __forceinline__ void unpack(const uint4& c, float* f) {
    f[0] = __uint_as_float(c.x);
    f[1] = __uint_as_float(c.y);
    f[2] = __uint_as_float(c.z);
    f[3] = __uint_as_float(c.w);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
  __device__ static __forceinline__ float load1(const float* p) { return *p; }
  __device__ static __forceinline__ void store1(float* p, float v) { *p = v; }
};

// bfloat16 stored as raw uint16 bits; float -> bf16 rounds to nearest even.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t quiet_nan = (u >> 16) | 0x40u;
  return (f != f) ? quiet_nan : rounded;
}

template <>
struct ElemTraits<bf16_t> {
  static constexpr int kPerChunk = 8;
  __device__ static __forceinline__ void unpack(const uint4& c, float* f) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = f32_to_bf16_rne(f[2 * i]) | (f32_to_bf16_rne(f[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static __forceinline__ float load1(const bf16_t* p) { return bf16_to_f32(p->bits); }
  __device__ static __forceinline__ void store1(bf16_t* p, float v) {
    p->bits = static_cast<uint16_t>(f32_to_bf16_rne(v));
  }
};

// IEEE binary16 stored as raw bits; conversions use the hardware (RNE).
struct f16_t {
  uint16_t bits;
};

__device__ __forceinline__ float f16_to_f32(uint32_t bits16) {
  _Float16 h;
  const uint16_t b = static_cast<uint16_t>(bits16);
  __builtin_memcpy(&h, &b, 2);
  return static_cast<float>(h);
}

__device__ __forceinline__ uint32_t f32_to_f16(float f) {
  const _Float16 h = static_cast<_Float16>(f);
  uint16_t b;
  __builtin_memcpy(&b, &h, 2);
  return b;
}

template <>
struct ElemTraits<f16_t> {
  static constexpr int kPerChunk = 8;
  __device__ static __forceinline__ void unpack(const uint4& c, float* f) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = f16_to_f32(w[i] & 0xffffu);
      f[2 * i + 1] = f16_to_f32(w[i] >> 16);
    }
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = f32_to_f16(f[2 * i]) | (f32_to_f16(f[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static __forceinline__ float load1(const f16_t* p) { return f16_to_f32(p->bits); }
  __device__ static __forceinline__ void store1(f16_t* p, float v) { p->bits = static_cast<uint16_t>(f32_to_f16(v)); }
};

}  // namespace rnnt
