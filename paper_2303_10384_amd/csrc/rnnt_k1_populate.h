// Kernel 1: row log-normaliser and gather of the blank / label log-probs.
//
// Populate (Section 2.2) selects every arc weight of the grid lattice (Fig. 1)
// from X = log_softmax(logits) by (time, unit_idx, label).  One pass over each
// valid logits row (t < T_b, u <= U_b) computes lse = ln sum_v exp z_v and
// emits only what the lattice needs, formed in float64 from the exact input:
//   lp_blank(t, u) = z[blank] - lse,  lp_label(t, u) = z[y_{u+1}] - lse.
// Padding rows are never touched.
//
// Two output forms:
//  * LATTICE (the fused loss): arc weights in log2 units, stored as
//    {lp_blank, lp_label} pairs by anti-diagonal (cell (t, u) of utterance b at
//    (b*(T_max+U_max) + t+u)*(U_max+1) + u), where the lattice kernel reads a
//    diagonal as one contiguous run; absent arcs (the label arc of the top row,
//    the blank arcs of the last frame below the top row) carry kNoArc; plus
//    lse * log2(e) as float32 at the same index.
//  * dense natural-log lse / lp_blank / lp_label, (B, T_max, U_max+1) float64
//    (the populate step on its own).
//
// Mapping: a block owns up to `rows_per_block` consecutive units u of one
// anti-diagonal d of one utterance, so the lattice-form writes of a block are
// one contiguous run.  A group of G lanes reads one row as aligned 16-byte
// chunks.  The chunks entirely inside the row ("interior") are spread NB per
// lane (G and NB picked from V so that G*NB just covers them) and need no
// element masks: a lane with no chunk of its own reloads an interior chunk,
// which cannot raise the maximum, and drops it from the sum with one select.
// The at most two chunks that straddle the row's ends go to lanes 0 and 1 with
// element masks.  All loads are issued, unconditionally, before any value is
// used.  Then two passes over the registers: the group maximum (DPP
// reduction), then the sum of 2^(z*log2 e - max*log2 e) per lane in float32
// and across the group in float64.  Rows longer than 64 * 5 interior chunks
// take a batched path with a running (max, sum) per lane; a row whose last
// chunk runs past the end of the tensor reads element-wise.
#pragma once

#include "rnnt_device.h"

#ifndef RNNT_K1_NT_LOAD
#define RNNT_K1_NT_LOAD 1
#endif

namespace rnnt {

constexpr bool kK1StreamLoads = RNNT_K1_NT_LOAD != 0;

struct PopulateParams {
  const void* logits;
  int32_t B, T_max, U_max, V, blank;
  const int32_t* labels;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  int64_t n_elem;          // B * T_max * (U_max+1) * V
  int32_t n_ublk;          // blocks per anti-diagonal
  int32_t rows_per_block;  // consecutive units u per block (<= kMaxRowsPerBlock)
  // lattice form
  double2* lp2;            // (B, T_max+U_max, U_max+1) {lp_blank, lp_label} * log2(e)
  float* lse2;             // same index: lse * log2(e)
  // dense form
  double* lse_out;         // (B, T_max, U_max+1) or null
  double* lp_blank_out;
  double* lp_label_out;
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

// Row statistics of the common case: the row's interior chunks fit NB per
// lane.  Returns (group max, group sum of exp(z - max)) in every lane.
template <typename T, int G, int NB>
__device__ __forceinline__ void row_stats_fast(const T* __restrict__ base, int64_t c0, int mis, int nch, int V,
                                               int lg, float& mg, double& sg) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  const float kNegInf = -__builtin_inff();
  const uint4* __restrict__ cbase = reinterpret_cast<const uint4*>(base);
  const bool first_partial = mis != 0;
  const bool last_partial = ((mis + V) % EPC) != 0;
  const int kf = first_partial ? 1 : 0;                    // first interior chunk
  const int kl = nch - 1 - (last_partial ? 1 : 0);         // last interior chunk
  const int n_int = kl - kf + 1;                           // may be <= 0 for tiny rows
  // boundary chunks: lane 0 takes the first, lane 1 the last (once if they coincide)
  const int kb0 = first_partial ? 0 : -1;
  const int kb1 = (last_partial && nch - 1 != kb0) ? nch - 1 : -1;
  const int kbnd = (lg == 0) ? kb0 : (lg == 1 ? kb1 : -1);

  uint4 raw[NB];
  const int kint_hi = n_int > 0 ? kl : 0;
  const int kint_lo = n_int > 0 ? kf : 0;
#pragma unroll
  for (int q = 0; q < NB; ++q) {
    const int k = min(max(kf + q * G + lg, kint_lo), kint_hi);
    raw[q] = load16<kK1StreamLoads>(cbase + c0 + k);
  }
  const uint4 rawb = load16<kK1StreamLoads>(cbase + c0 + max(kbnd, 0));

  float xb[EPC];
  {
    float f[EPC];
    ElemTraits<T>::unpack(rawb, f);
#pragma unroll
    for (int j = 0; j < EPC; ++j) {
      const int v = kbnd * EPC + j - mis;
      xb[j] = (kbnd >= 0 && v >= 0 && v < V) ? f[j] : kNegInf;
    }
  }
  float x[NB * EPC];
#pragma unroll
  for (int q = 0; q < NB; ++q) ElemTraits<T>::unpack(raw[q], x + q * EPC);

  // pass 1: maximum (interior duplicates are harmless; no interior chunks -> skip them)
  float m = kNegInf;
#pragma unroll
  for (int j = 0; j < EPC; ++j) m = fmaxf(m, xb[j]);
  if (n_int > 0) {
#pragma unroll
    for (int i = 0; i < NB * EPC; ++i) m = fmaxf(m, x[i]);
  }
  mg = group_reduce<G, MaxOp>(m, kNegInf);
  // pass 2: sum of exp relative to the group maximum
  const float sh = (mg == kNegInf) ? 0.f : mg * kLog2eF;
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < EPC; ++j) s += fast_exp2(fmaf(xb[j], kLog2eF, -sh));
  if (n_int > 0) {
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      float sq = 0.f;
#pragma unroll
      for (int j = 0; j < EPC; ++j) sq += fast_exp2(fmaf(x[q * EPC + j], kLog2eF, -sh));
      s += (kf + q * G + lg <= kl) ? sq : 0.f;
    }
  }
  sg = group_reduce<G, SumOp>(static_cast<double>(s), 0.0);
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
  sg = group_reduce<G, SumOp>(static_cast<double>(sloc * scale), 0.0);
}

// FAST: rows take row_stats_fast (the launcher checks that NB*G covers every
// row's interior chunks); otherwise row_stats_general.
constexpr int kMaxRowsPerBlock = 1024;

template <typename T, int G, int NB, bool LATTICE, bool FAST>
__global__ __launch_bounds__(256) void k1_populate(PopulateParams p) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int GROUPS = 256 / G;      // rows in flight per block
  __shared__ int s_label[kMaxRowsPerBlock];

  const int ND = p.T_max + p.U_max;  // anti-diagonals per utterance
  const int diag = blockIdx.x / p.n_ublk;  // b * ND + d
  const int ublk = blockIdx.x - diag * p.n_ublk;
  const int b = diag / ND;
  const int d = diag - b * ND;
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  if (Tb < 1 || Tb > p.T_max || Ub < 0 || Ub > p.U_max) return;
  const int u_first = ublk * p.rows_per_block;
  const int u_lo = max(u_first, d - (Tb - 1));           // t = d - u <= T_b - 1
  const int u_hi = min(u_first + p.rows_per_block, min(d, Ub) + 1);
  if (u_lo >= u_hi) return;

  const int lg = threadIdx.x % G;  // lane inside the row group
  const int grp = threadIdx.x / G;
  // the block's labels go through LDS, so no label load waits inside the row loop
  for (int i = threadIdx.x; i < u_hi - u_first; i += blockDim.x) {
    const int u = u_first + i;
    s_label[i] = (u < Ub) ? p.labels[static_cast<int64_t>(b) * p.U_max + u] : kNoLabel;
  }
  __syncthreads();

  const T* __restrict__ base = static_cast<const T*>(p.logits);
  const int64_t full_chunks = p.n_elem / EPC;

  // all lanes of a wave stay in the loop (the group reductions use every lane);
  // a group past the block's last row computes a row it does not write
  const int n_iter = (u_hi - u_lo + GROUPS - 1) / GROUPS;
  for (int it = 0; it < n_iter; ++it) {
    const int u_raw = u_lo + it * GROUPS + grp;
    const bool live = u_raw >= u_lo && u_raw < u_hi;
    const int u = live ? u_raw : u_lo;  // dead groups recompute the block's first row
    const int t = d - u;
    const int64_t row = (static_cast<int64_t>(b) * p.T_max + t) * (p.U_max + 1) + u;
    const int64_t e0 = row * p.V;
    const int64_t c0 = e0 / EPC;
    const int mis = static_cast<int>(e0 - c0 * EPC);
    const int nch = (mis + p.V + EPC - 1) / EPC;
    const int y = s_label[u - u_first];
    const bool y_ok = (y >= 0 && y < p.V);
    // z[blank], z[y]: the same address in every lane of the group (one request,
    // a line the row's chunk loads bring in anyway), issued ahead of them
    const float zb = ElemTraits<T>::load1(base + e0 + p.blank);
    const float zy = ElemTraits<T>::load1(base + e0 + (y_ok ? y : 0));

    float mg;
    double sg;
    if (FAST && c0 + nch <= full_chunks)
      row_stats_fast<T, G, NB>(base, c0, mis, nch, p.V, lg, mg, sg);
    else
      row_stats_general<T, G, NB>(base, e0, c0, mis, nch, p.V, full_chunks, lg, mg, sg);

    if (live && lg == 0) {
      const double lse = static_cast<double>(mg) + log(sg);
      const double lpb = static_cast<double>(zb) - lse;
      const double lpl = (u < Ub) ? (y_ok ? static_cast<double>(zy) - lse : __builtin_nan("")) : -__builtin_inf();
      if (LATTICE) {
        const int64_t sc = static_cast<int64_t>(diag) * (p.U_max + 1) + u;
        const bool blank_arc = (t < Tb - 1) || (u == Ub);  // absent: last frame below the top row
        double2 w;
        w.x = blank_arc ? clamp_no_arc(lpb * kLog2eD) : kNoArc;
        w.y = (u < Ub) ? clamp_no_arc(lpl * kLog2eD) : kNoArc;
        p.lp2[sc] = w;
        p.lse2[sc] = static_cast<float>(lse * kLog2eD);
      } else {
        if (p.lse_out) p.lse_out[row] = lse;
        p.lp_blank_out[row] = lpb;
        p.lp_label_out[row] = lpl;
      }
    }
  }
}

}  // namespace rnnt
