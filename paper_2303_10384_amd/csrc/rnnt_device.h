// Device helpers shared by the library's kernels (loss, forced alignment,
// arc-list lattices; gfx950, wave64).  No host code here.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rnnt {

constexpr float kLog2eF = 1.4426950408889634f;
constexpr float kLn2F = 0.6931471805599453f;
constexpr double kLog2eD = 1.4426950408889634;
constexpr int kWave = 64;

// Per-row record handed from the posterior kernel to the gradient kernel.
// lse2 = log2 sum_v 2^(z_v kLog2eF), the normaliser of the exponentials the
// gradient kernel forms (2^(z kLog2eF - lse2)); occ_* are the blank / label arc
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

// Where the posterior kernel computes the row records of the grid lattice
// from: kernel 1's lattice form and the sweeps' scores.
// The lattice form carries each row's lse2f (float32) in the low 16 bits of the
// mantissas of its two float64 weights (low half in lp_blank, high half in
// lp_label), so that the populate kernel writes 16 bytes a row instead of 20.
// The weights move by less than 2^-36 of their value: about 1.5e-9 log2 units
// for a weight of 100, far below what the sweeps resolve; kNoArc stays absorbing
// and a NaN stays a NaN (its top mantissa bit is untouched).
__device__ __forceinline__ double with_low16(double x, uint32_t bits16) {
  const uint64_t v = static_cast<uint64_t>(__double_as_longlong(x));
  return __longlong_as_double(static_cast<long long>((v & ~uint64_t{0xffff}) | bits16));
}
__device__ __forceinline__ double2 pack_lse2f(double2 w, float lse2f) {
  const uint32_t b = __float_as_uint(lse2f);
  w.x = with_low16(w.x, b & 0xffffu);
  w.y = with_low16(w.y, b >> 16);
  return w;
}
__device__ __forceinline__ float unpack_lse2f(double2 w) {
  const uint32_t lo = static_cast<uint32_t>(__double_as_longlong(w.x)) & 0xffffu;
  const uint32_t hi = static_cast<uint32_t>(__double_as_longlong(w.y)) & 0xffffu;
  return __uint_as_float(lo | (hi << 16));
}

struct LatticeRecordSrc {
  int32_t T_max, U_max, u_pad;  // u_pad: row width of alpha / beta
  const int32_t* labels;        // (B, U_max), may be null when U_max == 0
  const int32_t* logit_lens;    // (B)
  const int32_t* label_lens;    // (B)
  const int32_t* status;        // (B) 0: good utterance
  const double2* lp2;           // (B, T_max, U_max+1) {lp_blank, lp_label} * log2 e, lse2f in their low bits
  const double* alpha;          // (B, T_max+U_max+1, u_pad) by diagonal, log2 units
  const double* beta;
  const double* lnp2_fwd;       // (B) log2 P
};

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

// Row record of the valid row r = (b, t, u) (t < T, u <= U) of a good utterance:
//   occ_blank = 2^(alpha(t,u) + lp_blank(t,u) + beta(t+1,u) - log2 P)   (t < T-1)
//   occ_blank = 2^(alpha(T-1,U) + lp_blank(T-1,U) - log2 P)            (closing blank)
//   occ_label = 2^(alpha(t,u) + lp_label(t,u) + beta(t,u+1) - log2 P)   (u < U)
// and 0 for an absent arc.  Every load is issued unconditionally, at an index
// inside the arrays (beta's unit clamped into its row).
__device__ __forceinline__ RowInfo lattice_row_record(const LatticeRecordSrc& s, int b, int t, int u, int64_t r,
                                                      int T, int U, double lnP2) {
  const int d = t + u;
  const int64_t ab0 = static_cast<int64_t>(b) * (s.T_max + s.U_max + 1) * s.u_pad;
  const double al = s.alpha[ab0 + static_cast<int64_t>(d) * s.u_pad + u];
  const double* __restrict__ bt = s.beta + ab0 + static_cast<int64_t>(d + 1) * s.u_pad;
  const double b_down = bt[u];                           // beta(t+1, u)
  const double b_right = bt[min(u + 1, s.u_pad - 1)];    // beta(t, u+1)
  const double2 w = s.lp2[r];
  const float lse2 = unpack_lse2f(w);
  const int y = s.U_max > 0 ? s.labels[static_cast<int64_t>(b) * s.U_max + min(u, s.U_max - 1)] : kNoLabel;
  double xb = kNoArc, xl = kNoArc;
  if (t < T - 1) xb = al + w.x + b_down - lnP2;
  else if (u == U) xb = al + w.x - lnP2;
  if (u < U) xl = al + w.y + b_right - lnP2;
  RowInfo o;
  o.lse2 = lse2;
  o.occ_blank = fast_exp2(static_cast<float>(xb));
  o.occ_label = fast_exp2(static_cast<float>(xl));
  o.label = (u < U) ? y : kNoLabel;
  // Both posteriors underflow float32 (the node lies far from every likely path) and the
  // row's normaliser is finite, so every logit of the row is finite: its gradient
  // p_v (g_b + g_l) - g_b [v = blank] - g_l [v = y] is exactly +0 at every v.  The row
  // goes to the gradient kernel as a zero row, which writes those zeros without reading
  // its logits.
  if (o.occ_blank == 0.f && o.occ_label == 0.f && __builtin_isfinite(lse2)) o = RowInfo{0.f, 0.f, 0.f, kZeroRow};
  return o;
}

// ---- 16-byte global accesses, optionally with the nontemporal (streaming) hint
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ uint4 load16(const uint4* p) {
  if constexpr (NT) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
  } else {
    return *p;
  }
}

template <bool NT>
__device__ __forceinline__ void store16(uint4* p, const uint4& v) {
  if constexpr (NT) {
    const u32x4 w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(p));
  } else {
    *p = v;
  }
}

// ---- reductions over a group of G consecutive lanes (G = 1..64, a power of 2)
// DPP moves inside each 16-lane row (pair swap, quad swap, half-row mirror,
// row mirror), so after the in-row steps every lane holds its group's value;
// across rows: row broadcasts, then the group's last lane is read back.
namespace dpp {
constexpr int kQuadSwap1 = 0xB1;    // quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;    // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;  // lane i <- 7-i within 8 lanes
constexpr int kRowMirror = 0x140;   // lane i <- 15-i within 16 lanes
constexpr int kRowBcast15 = 0x142;  // every lane of row r <- lane 15 of row r-1
constexpr int kRowBcast31 = 0x143;  // every lane of rows 2,3 <- lane 31
}  // namespace dpp

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ float dpp_f32(float x, float fill) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, fill),
                                                               __builtin_bit_cast(int, x), CTRL, ROW_MASK, 0xf,
                                                               false));
}

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ double dpp_f64(double x, double fill) {
  const int lo = __builtin_amdgcn_update_dpp(__double2loint(fill), __double2loint(x), CTRL, ROW_MASK, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(__double2hiint(fill), __double2hiint(x), CTRL, ROW_MASK, 0xf, false);
  return __hiloint2double(hi, lo);
}

struct MaxOp {  // a NaN operand is dropped (callers see NaN through their sums instead)
  template <typename V>
  __device__ static V apply(V a, V b) { return __builtin_fmax(a, b); }
  __device__ static float apply(float a, float b) { return __builtin_fmaxf(a, b); }
};
struct SumOp {
  template <typename V>
  __device__ static V apply(V a, V b) { return a + b; }
};

template <typename V, int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ V dpp_any(V x, V fill) {
  if constexpr (sizeof(V) == 8) return dpp_f64<CTRL, ROW_MASK>(x, fill);
  else return dpp_f32<CTRL, ROW_MASK>(x, fill);
}

// A permutation inside each row of 16 lanes (every lane reads a lane of its own
// row): no fill value, so the compiler may fold the move into the operation
// that uses it.
template <typename V, int CTRL>
__device__ __forceinline__ V dpp_perm(V x) {
  if constexpr (sizeof(V) == 8) {
    const int lo = __builtin_amdgcn_mov_dpp(__double2loint(x), CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(x), CTRL, 0xf, 0xf, false);
    return __hiloint2double(hi, lo);
  } else {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
  }
}

template <typename V>
__device__ __forceinline__ V readlane_any(V x, int lane) {
  if constexpr (sizeof(V) == 8) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(x), lane);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(x), lane);
    return __hiloint2double(hi, lo);
  } else {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), lane));
  }
}

// Every lane of the group receives op over the group's G lanes; `ident` is
// the operation's identity.  All 64 lanes must be active.
template <int G, typename Op, typename V>
__device__ __forceinline__ V group_reduce(V x, V ident) {
  if constexpr (G >= 2) x = Op::apply(x, dpp_perm<V, dpp::kQuadSwap1>(x));
  if constexpr (G >= 4) x = Op::apply(x, dpp_perm<V, dpp::kQuadSwap2>(x));
  if constexpr (G >= 8) x = Op::apply(x, dpp_perm<V, dpp::kHalfMirror>(x));
  if constexpr (G >= 16) x = Op::apply(x, dpp_perm<V, dpp::kRowMirror>(x));
  if constexpr (G >= 32) {
    // rows 1 and 3 add rows 0 and 2: lanes 31 and 63 hold the 32-lane totals
    x = Op::apply(x, dpp_any<V, dpp::kRowBcast15, 0xa>(x, ident));
    if constexpr (G == 32) {
      const V lo = readlane_any(x, 31), hi = readlane_any(x, 63);
      x = (__lane_id() < 32) ? lo : hi;
    } else {
      x = Op::apply(x, dpp_any<V, dpp::kRowBcast31, 0xc>(x, ident));
      x = readlane_any(x, 63);
    }
  }
  return x;
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
  __device__ static __forceinline__ float from_bits(uint32_t b) { return __uint_as_float(b); }
  __device__ static __forceinline__ void store1(float* p, float v) { *p = v; }
};

// bfloat16 stored as raw uint16 bits; float -> bf16 rounds to nearest even.
struct bf16_t {
  uint16_t bits;
};

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// Two floats rounded to nearest even and packed (the first in the low half):
// one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ uint32_t pack2_f16(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2_t));
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

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
    for (int i = 0; i < 4; ++i) w[i] = pack2_bf16(f[2 * i], f[2 * i + 1]);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static __forceinline__ float load1(const bf16_t* p) { return bf16_to_f32(p->bits); }
  __device__ static __forceinline__ float from_bits(uint32_t b) { return bf16_to_f32(b & 0xffffu); }
  __device__ static __forceinline__ void store1(bf16_t* p, float v) {
    p->bits = static_cast<uint16_t>(pack2_bf16(v, 0.f) & 0xffffu);
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
    for (int i = 0; i < 4; ++i) w[i] = pack2_f16(f[2 * i], f[2 * i + 1]);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static __forceinline__ float load1(const f16_t* p) { return f16_to_f32(p->bits); }
  __device__ static __forceinline__ float from_bits(uint32_t b) { return f16_to_f32(b & 0xffffu); }
  __device__ static __forceinline__ void store1(f16_t* p, float v) { p->bits = static_cast<uint16_t>(f32_to_f16(v)); }
};

// ---- raw buffer loads ------------------------------------------------------
// A buffer resource covers [base, base + bytes); a load at an offset at or past
// `bytes` returns zero without a memory access.  Loads issued unconditionally
// with such offsets for lanes that need nothing keep the compiler's wait counts
// exact (a load under a branch makes every later wait a full drain).
constexpr int kBufferWord3 = 0x00020000;               // raw buffer, 32-bit data format (gfx9 family)
constexpr int kOutOfRange = static_cast<int>(0x80000000u);  // past any buffer made here (< 2^31 bytes)
constexpr int kBufferNT = 2;                           // cache-policy bits: nontemporal
constexpr int kBufferSC1 = 16;                         // cache-policy bits: device scope (written through the L2)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_buffer(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), static_cast<int>(bytes),
                                           kBufferWord3);
}

template <bool NT>
__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, NT ? kBufferNT : 0);
}

// A lane's K consecutive float64 scores into a score row, through a buffer:
// `lane_off` the lane's byte offset in the row (per lane, fixed), `row_off` the
// row's byte offset (wave-uniform, in a scalar register), 16-byte stores for
// pairs and an 8-byte store for an odd last score.
template <int K>
__device__ __forceinline__ void store_scores(__amdgpu_buffer_rsrc_t r, int lane_off, int row_off, const double (&x)[K]) {
#pragma unroll
  for (int k = 0; k + 1 < K; k += 2) {
    const uint64_t a = static_cast<uint64_t>(__double_as_longlong(x[k]));
    const uint64_t c = static_cast<uint64_t>(__double_as_longlong(x[k + 1]));
    const u32x4 v = {static_cast<uint32_t>(a), static_cast<uint32_t>(a >> 32), static_cast<uint32_t>(c),
                     static_cast<uint32_t>(c >> 32)};
    __builtin_amdgcn_raw_buffer_store_b128(v, r, lane_off + 8 * k, row_off, 0);
  }
  if constexpr (K % 2 == 1) {
    const uint64_t a = static_cast<uint64_t>(__double_as_longlong(x[K - 1]));
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = {static_cast<uint32_t>(a), static_cast<uint32_t>(a >> 32)};
    __builtin_amdgcn_raw_buffer_store_b64(v, r, lane_off + 8 * (K - 1), row_off, 0);
  }
}

// Lattice-form cell (t, u) of one utterance, t = e - u on diagonal e, through a
// buffer over the utterance's T_max x (U_max+1) cells: its byte offset
// 16 (e U1 - u (U1 - 1)) is one 24-bit multiply-add per lane on top of the
// wave-uniform 16 e U1 (u < 2^11 and 16 (U1 - 1) < 2^15; the span is checked on
// the host to stay under 2^31 bytes).
__device__ __forceinline__ double2 load_lattice_cell(__amdgpu_buffer_rsrc_t r, int e_row_bytes, int u, int neg_step) {
  const u32x4 v = buffer_load16<false>(r, __mul24(u, neg_step) + e_row_bytes);
  double2 w;
  w.x = __hiloint2double(static_cast<int>(v.y), static_cast<int>(v.x));
  w.y = __hiloint2double(static_cast<int>(v.w), static_cast<int>(v.z));
  return w;
}

// One element of type T (4 or 2 bytes) at byte offset `off`, widened to float.
template <typename T>
__device__ __forceinline__ float buffer_load_elem(__amdgpu_buffer_rsrc_t r, int off) {
  if constexpr (sizeof(T) == 4)
    return ElemTraits<T>::from_bits(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
  else
    return ElemTraits<T>::from_bits(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
}

}  // namespace rnnt
