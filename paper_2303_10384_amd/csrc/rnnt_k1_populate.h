// Kernel 1: row log-normaliser and gather of the blank / label log-probs.
//
// Populate (Section 2.2) selects every arc weight of the grid lattice (Fig. 1)
// from X = log_softmax(logits) by (time, unit_idx, label).  One pass over each
// valid logits row (t < T_b, u <= U_b) computes lse = ln sum_v exp z_v and
// emits only what the lattice needs, formed in float64 from the exact input:
//   lp_blank(t, u) = z[blank] - lse,  lp_label(t, u) = z[y_{u+1}] - lse.
// Padding rows are never touched.
//
// Three output forms (OUT):
//  * kK1Lattice (the fused loss): arc weights in log2 units, stored as
//    {lp_blank, lp_label} pairs per row, (B, T_max, U_max+1) like the logits'
//    rows; absent arcs (the label arc of the top row, the blank arcs of the last
//    frame below the top row) carry kNoArc; lse2f (the log2 normaliser of the
//    kernel's own exponentials, see the results loop) rides as float32 in the
//    low 16 bits of the two weights' mantissas (pack_lse2f) when the loss asks
//    for it.
//  * kK1Dense: natural-log lse / lp_blank / lp_label, (B, T_max, U_max+1)
//    float64 (the populate step on its own);
//  * kK1Rows: lse2f per row, (B, T_max, U_max+1) float64, and no
//    labels read (the loss over arc-list lattices, whose arcs select their own
//    labels).
//
// Mapping: a block owns up to `rows_per_block` consecutive units u of one frame
// t of one utterance, so its rows are consecutive in memory; blocks are numbered
// so that short runs of consecutive blocks go to the same XCD (dispatch deals
// blocks to the 8 XCDs round robin).  A group of
// G lanes reads one row as aligned 16-byte chunks.  The chunks entirely inside
// the row ("interior") are spread NB per lane (G and NB picked from V so that
// G*NB just covers them) and need no element masks: a lane with no chunk of its
// own reloads an interior chunk, which cannot raise the maximum, and drops it
// from the sum with one select.  The elements of the at most two chunks that
// straddle the row's ends are spread over the group, one element per lane
// (two when G is 8), each with its own mask.  Then the sum of
// 2^(z*log2 e - shift) per lane in float32 and across the group by a pairwise
// float32 DPP tree, against a shift taken from the group maximum on the group's
// first row and kept while the rows' sums stay in range (reduce_row).
//
// Fast path (every block whose rows lie in whole chunks): the loads of a
// group's first row are issued before the block stages its labels in LDS, and
// the loads of its next row before its current row is reduced, as buffer
// loads on a per-block buffer resource; a row past the block's last gets
// offsets past the buffer's end (zeros, no memory access), so every load is
// issued unconditionally and the compiler's wait counts stay exact.  Results
// go to LDS and leave the block in one contiguous copy at its end, so no
// global store sits in the row loop either.  Otherwise (rows longer than
// 64 * 5 interior chunks, a block reaching the tensor's final partial chunk,
// or a block spanning 2 GB or more) a general loop with a running (max, sum)
// per lane and element masks.
#pragma once

#include "rnnt_device.h"

#ifndef RNNT_K1_NT_LOAD
#define RNNT_K1_NT_LOAD 1
#endif

namespace rnnt {

constexpr bool kK1StreamLoads = RNNT_K1_NT_LOAD != 0;

constexpr int kK1Dense = 0;
constexpr int kK1Lattice = 1;
constexpr int kK1Rows = 2;

struct PopulateParams {
  const void* logits;
  int32_t B, T_max, U_max, V, blank;
  const int32_t* labels;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  int64_t n_elem;          // B * T_max * (U_max+1) * V
  int32_t n_ublk;          // blocks per frame
  int32_t rows_per_block;  // consecutive units u per block (<= kMaxRowsPerBlock)
  // lattice form
  double2* lp2;            // (B, T_max, U_max+1) {lp_blank, lp_label} * log2(e)
  int32_t pack_lse2f;      // nonzero: lse2f rides in the low bits of each row's two weights (the loss);
                           // zero: the weights as they are (forced alignment, whose ties stay exact)
  // dense form
  double* lse_out;         // (B, T_max, U_max+1) or null
  double* lp_blank_out;
  double* lp_label_out;
  // rows form
  double* lse2_rows;       // (B, T_max, U_max+1): lse2f, as lse2
  int32_t* clear_flags;    // (B) set to 0 by block 0 (the arc-list loss's bad-data flags), or null
};

// (max, sum of exp) of one batch of register-held values, merged into the
// lane's running pair.
template <int N>
__device__ __forceinline__ void merge_batch(const float (&x)[N], float& mloc, float& sloc) {
  const float kNegInf = -__builtin_inff();
  float bm = kNegInf;
#pragma unroll
  for (int i = 0; i < N; ++i) bm = fmaxf(bm, x[i]);
  const float mn = fmaxf(mloc, bm);
  const float sh = (mn == kNegInf) ? 0.f : mn;
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < N; ++i) acc += fast_exp2((x[i] - sh) * kLog2eF);
  sloc = (mloc == kNegInf) ? acc : fmaf(sloc, fast_exp2((mloc - sh) * kLog2eF), acc);
  mloc = mn;
}

__device__ __forceinline__ double clamp_no_arc(double x) { return x < kNoArc ? kNoArc : x; }  // NaN stays NaN

// Geometry of the row a group handles in one iteration of the fast path.
struct RowGeom {
  bool live;   // a row of the block (else: every load is out of range)
  int j;       // number of the row in the block (0 if not live)
  int u;       // unit of the row
  int mis;     // elements of the row's first chunk before the row starts
  int nch;     // chunks touched by the row
  int off0;    // byte offset of the row's first chunk in the block's buffer
  int y;       // label y_{u+1}, or kNoLabel
};

// Elements per lane of a row's (at most two) partial boundary chunks, spread
// over the G lanes of the group.
template <typename T, int G>
constexpr int kBndPerLane = (2 * ElemTraits<T>::kPerChunk + G - 1) / G;

template <typename T, int G, int NB>
struct RowRegs {
  u32x4 raw[NB];                 // interior chunks
  float xb[kBndPerLane<T, G>];   // boundary elements (0 where the slot holds none)
  float zb, zy;                  // z[blank], z[y]
};

// Boundary slot e (0 .. 2*EPC-1) of a row: element e % EPC of its first partial
// chunk (e < EPC) or of its last; the chunk index and the column, and whether
// the slot holds an element of the row.
struct BndSlot {
  int chunk, col;
  bool ok;
};
template <int EPC>
__device__ __forceinline__ BndSlot bnd_slot(const RowGeom& g, int V, int e) {
  const bool first_partial = g.mis != 0;
  const bool last_partial = ((g.mis + V) % EPC) != 0;
  const int kb0 = first_partial ? 0 : -1;
  const int kb1 = (last_partial && g.nch - 1 != kb0) ? g.nch - 1 : -1;
  BndSlot b;
  b.chunk = (e < EPC) ? kb0 : kb1;
  b.col = b.chunk * EPC + (e & (EPC - 1)) - g.mis;
  b.ok = e < 2 * EPC && b.chunk >= 0 && b.col >= 0 && b.col < V;
  return b;
}

// The load of z[y_{u+1}] of one row (same address in every lane of the group).
template <typename T>
__device__ __forceinline__ float issue_label_elem(__amdgpu_buffer_rsrc_t rsrc, const RowGeom& g, int V) {
  const uint32_t rb = g.live ? static_cast<uint32_t>(g.off0) : static_cast<uint32_t>(kOutOfRange);
  const bool y_ok = g.y >= 0 && g.y < V;
  const uint32_t oy = y_ok ? rb + static_cast<uint32_t>(g.mis + g.y) * sizeof(T) : static_cast<uint32_t>(kOutOfRange);
  return buffer_load_elem<T>(rsrc, static_cast<int>(oy));
}

// Issue every load of one row (all lanes, unconditionally); WITH_LABEL false
// leaves z[y] for a later issue_label_elem.  Offsets are unsigned: a row that
// is not live starts at kOutOfRange, and every offset derived from it stays at
// or above 2^31, past the buffer.
template <typename T, int G, int NB, bool WITH_LABEL = true>
__device__ __forceinline__ void issue_row(__amdgpu_buffer_rsrc_t rsrc, const RowGeom& g, int V, int blank, int lg,
                                          RowRegs<T, G, NB>& R) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr uint32_t S = sizeof(T);
  const bool first_partial = g.mis != 0;
  const bool last_partial = ((g.mis + V) % EPC) != 0;
  const int kf = first_partial ? 1 : 0;
  const int kl = g.nch - 1 - (last_partial ? 1 : 0);
  const int kint_lo = kl >= kf ? kf : 0;
  const int kint_hi = kl >= kf ? kl : 0;
  const uint32_t rb = g.live ? static_cast<uint32_t>(g.off0) : static_cast<uint32_t>(kOutOfRange);
#pragma unroll
  for (int q = 0; q < NB; ++q) {
    const int k = min(max(kf + q * G + lg, kint_lo), kint_hi);
    R.raw[q] = buffer_load16<kK1StreamLoads>(rsrc, static_cast<int>(rb + static_cast<uint32_t>(k) * 16u));
  }
  // the partial boundary chunks, one element per lane (their lines come in with the interior loads)
#pragma unroll
  for (int i = 0; i < kBndPerLane<T, G>; ++i) {
    const BndSlot b = bnd_slot<ElemTraits<T>::kPerChunk>(g, V, lg + i * G);
    const uint32_t ob = b.ok ? rb + static_cast<uint32_t>(b.col + g.mis) * S : static_cast<uint32_t>(kOutOfRange);
    R.xb[i] = buffer_load_elem<T>(rsrc, static_cast<int>(ob));
  }
  // the same address in every lane of the group: one request, a line the chunk loads bring in
  R.zb = buffer_load_elem<T>(rsrc, static_cast<int>(rb + static_cast<uint32_t>(g.mis + blank) * S));
  if (WITH_LABEL) R.zy = issue_label_elem<T>(rsrc, g, V);
}

// Accepted range of a row's group sum when the sum used an earlier row's shift.
// A sum of at most 2^16 bounds every term by 2^16 (no element more than 16 log2
// units above the shift, and no overflow); a sum of at least 2^-16 puts the
// largest term within 16 + log2 V units below the shift, so the terms that
// underflow are far below float32 resolution of the sum.  The dominant terms'
// exponents then stay small, which keeps the rounding of their arguments near
// that of the exact-maximum shift.
constexpr float kSumHi = 65536.f;
constexpr float kSumLo = 1.f / 65536.f;

// (shift, group sum of 2^(z log2 e - shift)) of a row from its registers, in
// every lane; the row's lse is ln 2 * (shift + log2 sum).  The shift is the group
// maximum * log2 e on a group's first row (`exact`); later rows sum against the
// shift they inherit, and keep it while every live row of the wave has its group
// sum inside [kSumLo, kSumHi] (a NaN or an empty row fails the test); otherwise
// the whole wave takes its rows' group maxima and sums again from the registers.
// Either shift gives the same lse up to rounding, and a row costs no maximum pass
// unless its range moved far from the shift.
template <typename T, int G, int NB>
__device__ __forceinline__ void reduce_row(const RowRegs<T, G, NB>& R, const RowGeom& g, int V, int lg, bool exact,
                                           float& sh2, double& sg) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  const float kNegInf = -__builtin_inff();
  const bool first_partial = g.mis != 0;
  const bool last_partial = ((g.mis + V) % EPC) != 0;
  const int kf = first_partial ? 1 : 0;
  const int kl = g.nch - 1 - (last_partial ? 1 : 0);
  const int n_int = kl - kf + 1;  // may be <= 0 for tiny rows
  constexpr int BPL = kBndPerLane<T, G>;

  float xb[BPL];
#pragma unroll
  for (int i = 0; i < BPL; ++i) xb[i] = bnd_slot<EPC>(g, V, lg + i * G).ok ? R.xb[i] : kNegInf;
  float x[NB * EPC];
#pragma unroll
  for (int q = 0; q < NB; ++q) ElemTraits<T>::unpack(make_uint4(R.raw[q].x, R.raw[q].y, R.raw[q].z, R.raw[q].w),
                                                     x + q * EPC);
  // group sum of 2^(z log2 e - sh) (interior duplicates masked)
  auto group_sum = [&](float sh) {
    float s = fast_exp2(fmaf(xb[0], kLog2eF, -sh));
#pragma unroll
    for (int i = 1; i < BPL; ++i) s += fast_exp2(fmaf(xb[i], kLog2eF, -sh));
    if (n_int > 0) {
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        float sq = fast_exp2(fmaf(x[q * EPC], kLog2eF, -sh));
#pragma unroll
        for (int j = 1; j < EPC; ++j) sq += fast_exp2(fmaf(x[q * EPC + j], kLog2eF, -sh));
        s += (kf + q * G + lg <= kl) ? sq : 0.f;
      }
    }
    return group_reduce<G, SumOp>(s, 0.f);  // a pairwise tree of the lanes' partial sums
  };
  float sgf = 0.f;
  bool take_max = exact;
  if (!exact) {
    sgf = group_sum(sh2);
    // a row past the block's last is ignored
    const bool bad = g.live && !(sgf >= kSumLo && sgf <= kSumHi);
    take_max = __builtin_amdgcn_ballot_w64(bad) != 0;  // wave-uniform
  }
  if (take_max) {
    // lane maximum (interior duplicates are harmless; no interior chunks -> skip them)
    float m = kNegInf;
#pragma unroll
    for (int i = 0; i < BPL; ++i) m = fmaxf(m, xb[i]);
    if (n_int > 0) {
#pragma unroll
      for (int i = 0; i < NB * EPC; ++i) m = fmaxf(m, x[i]);
    }
    const float mg = group_reduce<G, MaxOp>(m, kNegInf);
    sh2 = (mg == kNegInf) ? 0.f : mg * kLog2eF;
    sgf = group_sum(sh2);
  }
  sg = static_cast<double>(sgf);
}

// Row statistics for any row: batches of NB chunks per lane with a running
// (max, sum) per lane, element masks everywhere, element loads where the row
// reaches into the tensor's final partial chunk.
template <typename T, int G, int NB>
__device__ __forceinline__ void row_stats_general(const T* __restrict__ base, int64_t e0, int64_t c0, int mis,
                                                  int nch, int V, int64_t full_chunks, int lg, float& mg,
                                                  double& sg) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  const float kNegInf = -__builtin_inff();
  const uint4* __restrict__ cbase = reinterpret_cast<const uint4*>(base);
  float mloc = kNegInf, sloc = 0.f;
  if (c0 + nch <= full_chunks) {
    for (int kb = 0; kb < nch; kb += G * NB) {
      uint4 raw[NB];
#pragma unroll
      for (int q = 0; q < NB; ++q) raw[q] = cbase[c0 + min(kb + q * G + lg, nch - 1)];
      float x[NB * EPC];
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        float f[EPC];
        ElemTraits<T>::unpack(raw[q], f);
        const int k = kb + q * G + lg;
#pragma unroll
        for (int j = 0; j < EPC; ++j) {
          const int v = k * EPC + j - mis;
          x[q * EPC + j] = (k < nch && v >= 0 && v < V) ? f[j] : kNegInf;
        }
      }
      merge_batch<NB * EPC>(x, mloc, sloc);
    }
  } else {
    for (int k = lg; k < nch; k += G) {
      float x[EPC];
#pragma unroll
      for (int j = 0; j < EPC; ++j) {
        const int v = k * EPC + j - mis;
        x[j] = (v >= 0 && v < V) ? ElemTraits<T>::load1(base + e0 + v) : kNegInf;
      }
      merge_batch<EPC>(x, mloc, sloc);
    }
  }
  mg = group_reduce<G, MaxOp>(mloc, kNegInf);
  const float scale = (mloc == kNegInf) ? 0.f : fast_exp2((mloc - mg) * kLog2eF);
  sg = static_cast<double>(group_reduce<G, SumOp>(sloc * scale, 0.f));
}

// FAST: blocks whose rows lie in whole chunks take the pipelined path (the
// launcher checks that NB*G covers every row's interior chunks and that a block's
// rows span less than 2 GB); others take row_stats_general.
constexpr int kMaxRowsPerBlock = 256;
constexpr int kXcds = 8;
#ifndef RNNT_K1_XCD_RUN
#define RNNT_K1_XCD_RUN 4
#endif
constexpr int kXcdRun = RNNT_K1_XCD_RUN;  // consecutive blocks per XCD turn


template <typename T, int G, int NB, int OUT, bool FAST>
__global__ __launch_bounds__(256) void k1_populate(PopulateParams p) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int GROUPS = 256 / G;  // rows in flight per block
  // per row: the label, then the group results (shift, sum of exponentials, z[blank], z[y])
  __shared__ int s_label[kMaxRowsPerBlock];
  __shared__ double s_shift2[kMaxRowsPerBlock];
  __shared__ double s_sum[kMaxRowsPerBlock];
  __shared__ float s_zb[kMaxRowsPerBlock];
  __shared__ float s_zy[kMaxRowsPerBlock];

  if (OUT == kK1Rows && p.clear_flags && blockIdx.x == 0)
    for (int i = threadIdx.x; i < p.B; i += blockDim.x) p.clear_flags[i] = 0;
  // block order: runs of kXcdRun consecutive (b, t, ublk) are dealt to the XCDs in
  // turn; XCD x holds physical blocks x, x+8, ..., and its k-th block is element
  // k % kXcdRun of its (k / kXcdRun)-th run
  const int64_t n_blocks = static_cast<int64_t>(p.B) * p.T_max * p.n_ublk;
  const int64_t kx = blockIdx.x / kXcds;
  const int64_t lb = ((kx / kXcdRun) * kXcds + blockIdx.x % kXcds) * kXcdRun + kx % kXcdRun;
  if (lb >= n_blocks) return;
  const int64_t frame = lb / p.n_ublk;  // b * T_max + t
  const int ublk = static_cast<int>(lb - frame * p.n_ublk);
  const int b = static_cast<int>(frame / p.T_max);
  const int t = static_cast<int>(frame - static_cast<int64_t>(b) * p.T_max);
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  if (Tb < 1 || Tb > p.T_max || Ub < 0 || Ub > p.U_max || t >= Tb) return;
  const int u_lo = ublk * p.rows_per_block;
  const int u_hi = min(u_lo + p.rows_per_block, Ub + 1);
  const int U1 = p.U_max + 1;
  if (u_lo >= u_hi) return;
  const int n_rows = u_hi - u_lo;

  const int lg = threadIdx.x % G;  // lane inside the row group
  // a wave's group index (and with it a row's geometry) in scalar registers when
  // a group is the whole wave
  const int grp = (G == kWave) ? __builtin_amdgcn_readfirstlane(threadIdx.x / G) : threadIdx.x / G;
  auto group_uniform = [](int v) { return (G == kWave) ? __builtin_amdgcn_readfirstlane(v) : v; };
  // the block's labels go through LDS, so no label load waits inside the row loop
  auto stage_labels = [&]() {
    for (int i = threadIdx.x; i < n_rows; i += blockDim.x) {
      const int u = u_lo + i;
      s_label[i] = (OUT != kK1Rows && u < Ub) ? p.labels[static_cast<int64_t>(b) * p.U_max + u] : kNoLabel;
    }
    __syncthreads();
  };

  const T* __restrict__ base = static_cast<const T*>(p.logits);
  const int64_t full_chunks = p.n_elem / EPC;
  // row j of the block is unit u_lo + j, V elements after row j - 1
  const int64_t row_lo = frame * U1 + u_lo;
  const int64_t e_first = row_lo * p.V;
  const int64_t c_base = e_first / EPC;
  const int64_t c_end = (e_first + static_cast<int64_t>(n_rows) * p.V + EPC - 1) / EPC;
  const int n_iter = (n_rows + GROUPS - 1) / GROUPS;

  if (FAST && c_end <= full_chunks) {
    const __amdgpu_buffer_rsrc_t rsrc =
        make_buffer(reinterpret_cast<const uint4*>(base) + c_base, (c_end - c_base) * 16);
    // element offset of row j from the block's first chunk (fits 32 bits: the span is checked)
    const int e_rel0 = static_cast<int>(e_first - c_base * EPC);
    // the row's geometry; its label comes from LDS once the labels are staged
    auto geom = [&](int it, bool with_label) {
      RowGeom g;
      const int j = it * GROUPS + grp;
      g.live = j < n_rows;
      g.j = g.live ? j : 0;
      const int e_rel = e_rel0 + g.j * p.V;
      g.mis = e_rel & (EPC - 1);
      g.nch = (g.mis + p.V + EPC - 1) / EPC;
      g.off0 = (e_rel - g.mis) * static_cast<int>(sizeof(T));
      g.y = with_label ? group_uniform(s_label[g.j]) : kNoLabel;
      return g;
    };
    float sh2 = 0.f;  // the group's shift (log2 units), set on its first row
    auto finish = [&](const RowRegs<T, G, NB>& R, const RowGeom& g, bool first) {
      double sg;
      reduce_row<T, G, NB>(R, g, p.V, lg, first, sh2, sg);
      if (g.live && lg == 0) {
        s_shift2[g.j] = sh2;
        s_sum[g.j] = sg;
        s_zb[g.j] = R.zb;
        s_zy[g.j] = R.zy;
      }
    };
    // two register sets in turn (a copy between them would wait for the loads in flight);
    // the first row's chunks go out before the labels are staged, its z[y] after
    RowGeom g0 = geom(0, false), g1;
    RowRegs<T, G, NB> R0, R1;
    issue_row<T, G, NB, false>(rsrc, g0, p.V, p.blank, lg, R0);
    __builtin_amdgcn_sched_barrier(0);
    stage_labels();
    g0.y = group_uniform(s_label[g0.j]);
    R0.zy = issue_label_elem<T>(rsrc, g0, p.V);
    for (int it = 0; it < n_iter; it += 2) {
      g1 = geom(it + 1, true);  // past the block's rows: not live, no memory access
      issue_row<T, G, NB>(rsrc, g1, p.V, p.blank, lg, R1);
      __builtin_amdgcn_sched_barrier(0);  // the next row's loads go out before this row is reduced
      finish(R0, g0, it == 0);
      g0 = geom(it + 2, true);
      issue_row<T, G, NB>(rsrc, g0, p.V, p.blank, lg, R0);
      __builtin_amdgcn_sched_barrier(0);
      finish(R1, g1, false);
    }
  } else {
    stage_labels();
    // all lanes of a wave stay in the loop (the group reductions use every lane);
    // a group past the block's last row computes a row it does not keep
    for (int it = 0; it < n_iter; ++it) {
      const int j_raw = it * GROUPS + grp;
      const bool live = j_raw < n_rows;
      const int j = live ? j_raw : 0;
      const int64_t e0 = e_first + static_cast<int64_t>(j) * p.V;
      const int64_t c0 = e0 / EPC;
      const int mis = static_cast<int>(e0 - c0 * EPC);
      const int nch = (mis + p.V + EPC - 1) / EPC;
      const int y = s_label[j];
      const bool y_ok = (y >= 0 && y < p.V);
      const float zb = ElemTraits<T>::load1(base + e0 + p.blank);
      const float zy = ElemTraits<T>::load1(base + e0 + (y_ok ? y : 0));
      float mg;
      double sg;
      row_stats_general<T, G, NB>(base, e0, c0, mis, nch, p.V, full_chunks, lg, mg, sg);
      if (live && lg == 0) {
        s_shift2[j] = static_cast<double>(mg) * static_cast<double>(kLog2eF);  // the sum is relative to 2^(mg kLog2eF)
        s_sum[j] = sg;
        s_zb[j] = zb;
        s_zy[j] = zy;
      }
    }
  }
  __syncthreads();

  // one thread per row: the arc weights in float64, and the block's results leave
  // in one pass (a contiguous run of rows).  Every exponential above is
  // 2^(z * kLog2eF), so shift + log2(sum) is lse2f = log2 sum 2^(z kLog2eF), the
  // log-normaliser of softmax(c z) with c = kLog2eF / log2(e) = 1 - 1.3e-8.  The
  // gradient kernels exponentiate the same way, so they take lse2f: their softmax
  // then sums to one.  lse2f / kLog2eF = lse(z) + (1 - c) H(softmax z) (H the
  // entropy, at most ln V), so the row's lse is within 1.3e-8 ln V of the exact
  // one, where lse2f / log2(e) would be off by 1.3e-8 |lse|.
  for (int j = threadIdx.x; j < n_rows; j += blockDim.x) {
    const int u = u_lo + j;
    const int64_t row = row_lo + j;
    const int y = s_label[j];
    const bool y_ok = y >= 0 && y < p.V;
    const double lse2f = s_shift2[j] + log2(s_sum[j]);
    const double lse = lse2f / static_cast<double>(kLog2eF);
    const double lpb = static_cast<double>(s_zb[j]) - lse;
    const double lpl = (u < Ub) ? (y_ok ? static_cast<double>(s_zy[j]) - lse : __builtin_nan("")) : -__builtin_inf();
    if (OUT == kK1Lattice) {
      const bool blank_arc = (t < Tb - 1) || (u == Ub);  // absent: last frame below the top row
      double2 w;
      w.x = blank_arc ? clamp_no_arc(lpb * kLog2eD) : kNoArc;
      w.y = (u < Ub) ? clamp_no_arc(lpl * kLog2eD) : kNoArc;
      // device-scope stores, written through the L2 as they are issued: K1's
      // stream of reads then slows less than under the L2's later write-backs
      // (large bf16: K1 0.822 -> 0.812 ms); the block's rows are consecutive
      if (p.pack_lse2f) w = pack_lse2f(w, static_cast<float>(lse2f));  // lse2f rides in the weights' low bits
      const __amdgpu_buffer_rsrc_t r_lp = make_buffer(p.lp2 + row_lo, static_cast<int64_t>(n_rows) * 16);
      const uint64_t wx = static_cast<uint64_t>(__double_as_longlong(w.x));
      const uint64_t wy = static_cast<uint64_t>(__double_as_longlong(w.y));
      const u32x4 v = {static_cast<uint32_t>(wx), static_cast<uint32_t>(wx >> 32), static_cast<uint32_t>(wy),
                       static_cast<uint32_t>(wy >> 32)};
      __builtin_amdgcn_raw_buffer_store_b128(v, r_lp, j * 16, 0, kBufferSC1);
    } else if (OUT == kK1Rows) {
      const __amdgpu_buffer_rsrc_t r_rows = make_buffer(p.lse2_rows + row_lo, static_cast<int64_t>(n_rows) * 8);
      const uint64_t lb = static_cast<uint64_t>(__double_as_longlong(lse2f));
      typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
      const u32x2 v = {static_cast<uint32_t>(lb), static_cast<uint32_t>(lb >> 32)};
      __builtin_amdgcn_raw_buffer_store_b64(v, r_rows, j * 8, 0, kBufferSC1);  // device scope, as above
    } else {
      if (p.lse_out) p.lse_out[row] = lse;
      p.lp_blank_out[row] = lpb;
      p.lp_label_out[row] = lpl;
    }
  }
}

}  // namespace rnnt
