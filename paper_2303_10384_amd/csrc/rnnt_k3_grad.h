// Kernel 3: fused gradient of sum_b loss_b with respect to the logits.
//
// The loss depends on logits row (t, u) only through the two arcs leaving node
// (t, u) (Fig. 1; the wild-card arcs of Fig. 4 carry no parameter), so with
// arc posteriors g_b, g_l and p = softmax(z):
//   d loss / d z_v = p_v (g_b + g_l) - g_b [v = blank] - g_l [v = y_{u+1}]
// The kernel streams the whole gradient tensor once: each 16-byte chunk is
// located in its row(s) by index arithmetic, chunks of zero rows (padding, bad
// utterances) are written as 0 without reading the logits, and every other
// chunk reads the logits once and writes the gradient once.
// p_v = exp2(z_v * kLog2eF - lse2) with lse2 = log2 sum_v 2^(z_v kLog2eF) from the
// row record (the populate kernel's normaliser of the same exponentials).
#pragma once

#include "rnnt_device.h"

#ifndef RNNT_K3_NT_LOAD
#define RNNT_K3_NT_LOAD 1
#endif
#ifndef RNNT_K3_NT_STORE
#define RNNT_K3_NT_STORE 1
#endif

namespace rnnt {

constexpr bool kK3StreamLoads = RNNT_K3_NT_LOAD != 0;
constexpr bool kK3StreamStores = RNNT_K3_NT_STORE != 0;

struct GradParams {
  const void* logits;
  void* grad;
  const RowInfo* rowinfo;
  int64_t n_elem;  // B * T_max * (U_max+1) * V
  int64_t n_rows;  // B * T_max * (U_max+1)
  int32_t V, blank;
};

constexpr int kGradChunksPerThread = 2;
// Threads per block: 128 for float32 logits (HBM-bound: small blocks balance
// best), 256 for 16-bit logits (eight elements per chunk, issue-bound).
template <typename Tin>
constexpr int kGradThreads = sizeof(Tin) == 4 ? 128 : 256;
template <typename Tin>
constexpr int kGradTileChunks = kGradThreads<Tin> * kGradChunksPerThread;

__device__ __forceinline__ float grad_elem(float z, int v, const RowInfo& ri, int blank) {
  const float pr = fast_exp2(fmaf(z, kLog2eF, -ri.lse2));
  float g = pr * (ri.occ_blank + ri.occ_label);
  g = (v == blank) ? g - ri.occ_blank : g;
  g = (v == ri.label) ? g - ri.occ_label : g;
  return (ri.label == kZeroRow) ? 0.f : g;
}

// Gradient elements of one 16-byte input chunk, stored as Tout (one or two
// aligned 16-byte stores).
template <typename Tout, int EPC>
__device__ __forceinline__ void store_chunk(void* dst, int64_t e0, const float* out) {
  constexpr int PER = ElemTraits<Tout>::kPerChunk;
  static_assert(EPC % PER == 0, "input chunk must cover whole output chunks");
  uint4* d = reinterpret_cast<uint4*>(static_cast<Tout*>(dst) + e0);
#pragma unroll
  for (int i = 0; i < EPC / PER; ++i) store16<kK3StreamStores>(d + i, ElemTraits<Tout>::pack(out + i * PER));
}

// The chunks of one block, one at a time (any V; the tensor's final partial
// chunk read and written element by element).  SMALLV: V < elements per chunk,
// so one chunk may cover several rows.  Only small-V tensors and the block
// holding the final partial chunk come here; zero rows' logits are read too
// (and ignored).
template <typename T, typename Tout, bool SMALLV>
__device__ __forceinline__ void grad_chunks_general(const GradParams& p, int64_t tile0, int64_t r_tile,
                                                    uint32_t v_tile) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int kThreads = kGradThreads<T>;
  const uint32_t uV = static_cast<uint32_t>(p.V);
  const uint4* __restrict__ src = static_cast<const uint4*>(p.logits);
  const T* __restrict__ src_e = static_cast<const T*>(p.logits);
  Tout* __restrict__ dst_e = static_cast<Tout*>(p.grad);
  for (int q = 0; q < kGradChunksPerThread; ++q) {
    const int cl = q * kThreads + static_cast<int>(threadIdx.x);
    const int64_t c = tile0 + cl;
    const int64_t e0 = c * EPC;
    if (e0 >= p.n_elem) break;
    const uint32_t off = v_tile + static_cast<uint32_t>(cl) * EPC;
    const uint32_t dr = off / uV;
    int64_t r = r_tile + dr;
    int v = static_cast<int>(off - dr * uV);
    const bool full = e0 + EPC <= p.n_elem;
    float f[EPC], out[EPC];
    RowInfo ri = p.rowinfo[r];
    if (full) {
      ElemTraits<T>::unpack(load16<kK3StreamLoads>(src + c), f);
    } else {
#pragma unroll
      for (int j = 0; j < EPC; ++j) f[j] = (e0 + j < p.n_elem) ? ElemTraits<T>::load1(src_e + e0 + j) : 0.f;
    }
#pragma unroll
    for (int j = 0; j < EPC; ++j) {
      if (v >= p.V) {  // next row (at most once per chunk unless SMALLV)
        v -= p.V;
        ++r;
        if (r < p.n_rows) ri = p.rowinfo[r];
      }
      out[j] = grad_elem(f[j], v, ri, p.blank);
      ++v;
    }
    if (full) {
      store_chunk<Tout, EPC>(p.grad, e0, out);
    } else {
#pragma unroll
      for (int j = 0; j < EPC; ++j)
        if (e0 + j < p.n_elem) ElemTraits<Tout>::store1(dst_e + e0 + j, out[j]);
    }
  }
}

// Tin: logits element type; Tout: gradient element type (Tin or float).
// A block covers kGradTileChunks<Tin> consecutive chunks.  Every block but the one
// holding the tensor's final partial chunk takes the fast path, in three phases
// that keep all of a thread's memory requests in flight together: the row
// records of its chunks; the logits of its chunks, as buffer loads issued
// unconditionally (a chunk whose logits are not needed gets an offset past the
// buffer's end, which reads zero without touching memory); arithmetic and
// stores.
template <typename Tin, typename Tout, bool SMALLV>
__global__ __launch_bounds__(kGradThreads<Tin>) void k3_grad(GradParams p) {
  using T = Tin;
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int kThreads = kGradThreads<Tin>;
  constexpr int kTile = kGradTileChunks<Tin>;
  constexpr int Q = kGradChunksPerThread;
  const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kTile;
  const int64_t e_tile = tile0 * EPC;
  const int64_t r_tile = e_tile / p.V;
  const uint32_t v_tile = static_cast<uint32_t>(e_tile - r_tile * p.V);
  const uint32_t uV = static_cast<uint32_t>(p.V);
  const int64_t n_full = p.n_elem / EPC;  // chunks wholly inside the tensor
  if (SMALLV || (p.n_elem % EPC != 0 && tile0 + kTile > n_full)) {
    grad_chunks_general<T, Tout, SMALLV>(p, tile0, r_tile, v_tile);
    return;
  }

  int64_t r[Q];
  int v[Q];
  RowInfo ri0[Q], ri1[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const uint32_t off = v_tile + static_cast<uint32_t>(q * kThreads + static_cast<int>(threadIdx.x)) * EPC;
    const uint32_t dr = off / uV;
    r[q] = min(r_tile + dr, p.n_rows - 1);  // chunks past the end read a valid record and store nothing
    v[q] = static_cast<int>(off - dr * uV);
    ri0[q] = p.rowinfo[r[q]];
    ri1[q] = p.rowinfo[min(r[q] + 1, p.n_rows - 1)];
  }
  __builtin_amdgcn_sched_barrier(0);  // all record loads issue before any of them is used
  const int64_t tile_bytes = min<int64_t>(kTile, n_full - tile0) * 16;
  const __amdgpu_buffer_rsrc_t rsrc = make_buffer(static_cast<const uint4*>(p.logits) + tile0, tile_bytes);
  u32x4 raw[Q];
  bool store[Q];
  bool any_row[Q];  // some lane's chunk q touches a row with a gradient
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int cl = q * kThreads + static_cast<int>(threadIdx.x);
    const bool live = tile0 + cl < n_full;
    const bool split = v[q] + EPC > p.V;
    const bool zero = ri0[q].label == kZeroRow && (!split || ri1[q].label == kZeroRow);
    store[q] = live;
    any_row[q] = __builtin_amdgcn_ballot_w64(live && !zero) != 0;
    const int off = (live && !zero) ? cl * 16 : kOutOfRange;
    raw[q] = buffer_load16<kK3StreamLoads>(rsrc, off);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    float f[EPC], out[EPC];
    ElemTraits<T>::unpack(make_uint4(raw[q].x, raw[q].y, raw[q].z, raw[q].w), f);
    if (any_row[q] && __builtin_amdgcn_ballot_w64(v[q] + EPC > p.V) == 0) {
      // no chunk q of the wave reaches past its row's end: one record per lane
#pragma unroll
      for (int j = 0; j < EPC; ++j) out[j] = grad_elem(f[j], v[q] + j, ri0[q], p.blank);
    } else if (any_row[q]) {
#pragma unroll
      for (int j = 0; j < EPC; ++j) {
        const int vj = v[q] + j;
        const bool second = vj >= p.V;
        out[j] = second ? grad_elem(f[j], vj - p.V, ri1[q], p.blank) : grad_elem(f[j], vj, ri0[q], p.blank);
      }
    } else {  // the wave's chunks q all lie in zero rows (padding, bad utterances)
#pragma unroll
      for (int j = 0; j < EPC; ++j) out[j] = 0.f;
    }
    if (store[q]) store_chunk<Tout, EPC>(p.grad, (tile0 + q * kThreads + static_cast<int>(threadIdx.x)) * EPC, out);
  }
}

// ---- rows of at least 64 chunks ---------------------------------------------
//
// The 64 consecutive chunks a wavefront takes at once (a "group") then span at
// most two rows, a and a+1, so everything that depends on the row is the same
// across the wave: the two row records (scalar loads), whether a row is a zero
// row, and where the corrected elements -- the blank and the label y_{u+1} of
// each row -- fall.  An element costs one exponential, 2^(z log2 e - s), with
// the row's occupancy g_b + g_l folded into the shift s (one_exp_shift).  In a
// group that reaches into row b, each lane holds two shifts, for the elements
// of its chunk before and after the wave-uniform column where row b starts
// (they differ only in the one lane whose chunk straddles the row end), and an
// element picks one of them by its constant index; where one of the two rows
// is a zero row, that lane's elements of it are set to 0 whatever its logits
// hold (padding logits may be NaN).  The at most four corrections -g_b at
// v = blank and -g_l at v = y_{u+1} are applied by the lane owning the element,
// at a position known to the whole wave.
template <typename Tin>
constexpr int kWideMinV = kWave * ElemTraits<Tin>::kPerChunk - 1;

// out[j] -= corr in lane `owner` for the wave-uniform slot js (no run-time index
// into out: the slot is matched against each constant j)
template <int EPC>
__device__ __forceinline__ void fix_element(float (&out)[EPC], int lane, int owner, int js, float corr) {
#pragma unroll
  for (int j = 0; j < EPC; ++j)
    if (j == js) out[j] = (lane == owner) ? out[j] - corr : out[j];
}

// The correction of column `col` of the group's row a (pos = col - va) or row b
// (pos = V - va + col), if that element lies in the group.
template <int EPC>
__device__ __forceinline__ void fix_column(float (&out)[EPC], int lane, int pos, float corr) {
  if (pos >= 0 && pos < kWave * EPC) fix_element<EPC>(out, lane, pos / EPC, pos % EPC, corr);
}

// The shift s and factor m of a row record such that p_v (g_b + g_l) =
// 2^(z_v log2 e - s) * m.  While |lse2| < kOneExpMaxLse2 the occupancy moves into
// the exponent (s = lse2 - log2(g_b + g_l), m = 1: one exponential and no
// multiply per element); the rounding of s then costs at most 2^-24 |s| ln 2 of
// the element, under 3e-6 of the largest (|s| <= 64 where g_b + g_l is near 1)
// and decaying with the occupancy.  Rows with larger normalisers keep s = lse2
// and m = g_b + g_l, and so do rows whose occupancy lies in (0, 2^-60): the
// exponential unit returns 0 for results below 2^-126, where the product with
// m keeps the subnormal result of the multiply.  A row with no occupancy (zero
// rows included) gets s = +inf: every finite logit then gives exactly 0.
// Returns whether m == 1.
constexpr float kOneExpMaxLse2 = 64.f;
constexpr float kOneExpMinOcc = 0x1p-60f;
__device__ __forceinline__ bool one_exp_shift(const RowInfo& r, float& s, float& m) {
  const float occ = r.occ_blank + r.occ_label;
  const bool one = __builtin_fabsf(r.lse2) < kOneExpMaxLse2 && (occ >= kOneExpMinOcc || occ == 0.f);
  s = one ? r.lse2 - fast_log2(occ) : r.lse2;
  m = one ? 1.f : occ;
  return one;
}

template <typename Tin, typename Tout>
__global__ __launch_bounds__(kGradThreads<Tin>) void k3_grad_wide(GradParams p) {
  using T = Tin;
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int kThreads = kGradThreads<Tin>;
  constexpr int kTile = kGradTileChunks<Tin>;
  constexpr int Q = kGradChunksPerThread;
  const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kTile;
  const int64_t e_tile = tile0 * EPC;
  const int64_t r_tile = e_tile / p.V;
  const int v_tile = static_cast<int>(e_tile - r_tile * p.V);
  const int64_t n_full = p.n_elem / EPC;  // chunks wholly inside the tensor
  if (p.n_elem % EPC != 0 && tile0 + kTile > n_full) {
    grad_chunks_general<T, Tout, false>(p, tile0, r_tile, static_cast<uint32_t>(v_tile));
    return;
  }
  const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
  const RowInfo* __restrict__ rows = p.rowinfo;

  // group q of this wave: chunks tile0 + q*kThreads + 64*wave + lane; its first
  // element is column va of row ra (wave-uniform)
  int va[Q];
  RowInfo Ra[Q], Rb[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int off = v_tile + (q * kThreads + wave * kWave) * EPC;
    const int dr = off / p.V;
    va[q] = off - dr * p.V;
    const int64_t ra = min(r_tile + dr, p.n_rows - 1);  // groups past the end store nothing
    Ra[q] = rows[ra];
    Rb[q] = rows[min(ra + 1, p.n_rows - 1)];
  }
  __builtin_amdgcn_sched_barrier(0);  // all record loads issue before any of them is used
  const int64_t tile_bytes = min<int64_t>(kTile, n_full - tile0) * 16;
  const __amdgpu_buffer_rsrc_t rsrc = make_buffer(static_cast<const uint4*>(p.logits) + tile0, tile_bytes);
  u32x4 raw[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int cl = q * kThreads + static_cast<int>(threadIdx.x);
    const bool live = tile0 + cl < n_full;
    const int v = va[q] + lane * EPC;  // column of the chunk's first element in row a (>= V: in row b)
    const bool za = Ra[q].label == kZeroRow, zb = Rb[q].label == kZeroRow;
    const bool zero = v >= p.V ? zb : (v + EPC > p.V ? za && zb : za);
    raw[q] = buffer_load16<kK3StreamLoads>(rsrc, (live && !zero) ? cl * 16 : kOutOfRange);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int cl = q * kThreads + static_cast<int>(threadIdx.x);
    const int to_b = p.V - va[q];  // the group's first element of row b (>= 64*EPC: none)
    const bool za = Ra[q].label == kZeroRow, zb = Rb[q].label == kZeroRow;
    float out[EPC];
    if (za && (zb || to_b >= kWave * EPC)) {  // the whole group lies in zero rows
#pragma unroll
      for (int j = 0; j < EPC; ++j) out[j] = 0.f;
    } else {
      float f[EPC];
      ElemTraits<T>::unpack(make_uint4(raw[q].x, raw[q].y, raw[q].z, raw[q].w), f);
      // p_v (g_b + g_l) = 2^(z_v log2 e - s) * m per row: s = lse2 - log2(g_b + g_l) and m = 1
      // while |lse2| < kOneExpMaxLse2, else s = lse2 and m = g_b + g_l (see one_exp_shift)
      float sa, ma, sb, mb;
      const bool one_a = one_exp_shift(Ra[q], sa, ma), one_b = one_exp_shift(Rb[q], sb, mb);
      if (to_b >= kWave * EPC) {  // the group lies in row a
        if (one_a) {
#pragma unroll
          for (int j = 0; j < EPC; ++j) out[j] = fast_exp2(fmaf(f[j], kLog2eF, -sa));
        } else {
#pragma unroll
          for (int j = 0; j < EPC; ++j) out[j] = fast_exp2(fmaf(f[j], kLog2eF, -sa)) * ma;
        }
      } else {
        // row b starts at element ks of lane L's chunk: element j of a lane lies in
        // row b from lane L + 1 on (j < ks) or from lane L on (j >= ks)
        const int L = to_b / EPC, ks = to_b % EPC;
        const float s_lo = lane > L ? sb : sa, s_hi = lane >= L ? sb : sa;
        if (one_a && one_b) {
#pragma unroll
          for (int j = 0; j < EPC; ++j) out[j] = fast_exp2(fmaf(f[j], kLog2eF, -(j < ks ? s_lo : s_hi)));
        } else {
          const float m_lo = lane > L ? mb : ma, m_hi = lane >= L ? mb : ma;
#pragma unroll
          for (int j = 0; j < EPC; ++j)
            out[j] = fast_exp2(fmaf(f[j], kLog2eF, -(j < ks ? s_lo : s_hi))) * (j < ks ? m_lo : m_hi);
        }
        if (za != zb) {  // the straddling chunk's elements of a zero row are 0 whatever its logits hold
          const bool z_lo = lane > L ? zb : za, z_hi = lane >= L ? zb : za;
#pragma unroll
          for (int j = 0; j < EPC; ++j) out[j] = (j < ks ? z_lo : z_hi) ? 0.f : out[j];
        }
      }
      if (!za) {
        fix_column<EPC>(out, lane, p.blank - va[q], Ra[q].occ_blank);
        if (Ra[q].label >= 0) fix_column<EPC>(out, lane, Ra[q].label - va[q], Ra[q].occ_label);
      }
      if (!zb && to_b < kWave * EPC) {
        fix_column<EPC>(out, lane, to_b + p.blank, Rb[q].occ_blank);
        if (Rb[q].label >= 0) fix_column<EPC>(out, lane, to_b + Rb[q].label, Rb[q].occ_label);
      }
    }
    if (tile0 + cl < n_full) store_chunk<Tout, EPC>(p.grad, (tile0 + cl) * EPC, out);
  }
}

}  // namespace rnnt
