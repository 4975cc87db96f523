// Kernel 1: row log-normaliser and gather of the blank / label log-probs.
//
// Populate (Section 2.2) selects every arc weight of the grid lattice (Fig. 1)
// from X = log_softmax(logits) by (time, unit_idx, label).  One pass over each
// valid logits row (t < T_b, u <= U_b) computes lse = ln sum_v exp z_v and
// emits only what the lattice needs:
//   lp_blank(t, u) = z[blank] - lse,  lp_label(t, u) = z[y_{u+1}] - lse
// (float64, formed from the exact input value), plus lse * log2(e) as float32
// for the gradient kernel.  Padding rows are never touched.
//
// Mapping: a block owns `rows_per_block` consecutive rows u of one (b, t)
// segment; a group of G lanes (G = 8..64, chosen from V) reads one row with
// aligned 16-byte loads (the chunks straddling the row's ends are masked, the
// tensor's last partial chunk is read element-wise), reduces max then sum
// within the group, and its lane 0 writes the row's outputs.
#pragma once

#include "rnnt_device.h"

namespace rnnt {

struct PopulateParams {
  const void* logits;
  int32_t B, T_max, U_max, V, blank;
  const int32_t* labels;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  int64_t n_elem;          // B * T_max * (U_max+1) * V
  int32_t n_ublk;          // blocks per (b, t) segment
  int32_t rows_per_block;  // consecutive rows u per block
  RowInfo* rowinfo;        // row records (lse2 filled here) or null
  double* lp_blank;        // element (b,t,u) at b*sb + t*st + u*su (in doubles)
  double* lp_label;
  int64_t sb, st, su;
  double* lse_out;         // dense (B, T_max, U_max+1) or null
};

template <typename T, int G>
__global__ __launch_bounds__(256) void k1_populate(PopulateParams p) {
  constexpr int EPC = ElemTraits<T>::kPerChunk;
  constexpr int NB = 32 / EPC;      // chunks per lane per register batch
  constexpr int GROUPS = 256 / G;   // rows in flight per block
  const float kNegInf = -__builtin_inff();

  const int seg = blockIdx.x / p.n_ublk;  // b * T_max + t
  const int ublk = blockIdx.x - seg * p.n_ublk;
  const int b = seg / p.T_max;
  const int t = seg - b * p.T_max;
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  if (Tb < 1 || Tb > p.T_max || Ub < 0 || Ub > p.U_max || t >= Tb) return;

  const int lg = threadIdx.x % G;  // lane inside the row group
  const int grp = threadIdx.x / G;
  const int u_begin = ublk * p.rows_per_block;
  const int u_end = min(u_begin + p.rows_per_block, Ub + 1);
  const T* __restrict__ base = static_cast<const T*>(p.logits);
  const uint4* __restrict__ cbase = reinterpret_cast<const uint4*>(base);

  for (int u = u_begin + grp; u < u_end; u += GROUPS) {
    const int64_t row = static_cast<int64_t>(seg) * (p.U_max + 1) + u;
    const int64_t e0 = row * p.V;
    const int64_t c0 = e0 / EPC;
    const int mis = static_cast<int>(e0 - c0 * EPC);
    const int nch = (mis + p.V + EPC - 1) / EPC;

    // the two gathered logits, issued before the streaming loads
    float zb = 0.f, zy = 0.f;
    int y = kNoLabel;
    if (lg == 0) {
      zb = ElemTraits<T>::load1(base + e0 + p.blank);
      if (u < Ub) {
        y = p.labels[static_cast<int64_t>(b) * p.U_max + u];
        if (y >= 0 && y < p.V) zy = ElemTraits<T>::load1(base + e0 + y);
      }
    }

    float mloc = kNegInf, sloc = 0.f;
    for (int kb = 0; kb < nch; kb += G * NB) {
      float x[NB * EPC];
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        const int k = kb + q * G + lg;
        float f[EPC];
        if (k < nch) {
          const int64_t ck = c0 + k;
          if ((ck + 1) * EPC <= p.n_elem) {
            ElemTraits<T>::unpack(cbase[ck], f);
          } else {
#pragma unroll
            for (int j = 0; j < EPC; ++j) {
              const int64_t e = ck * EPC + j;
              f[j] = (e < p.n_elem) ? ElemTraits<T>::load1(base + e) : kNegInf;
            }
          }
#pragma unroll
          for (int j = 0; j < EPC; ++j) {
            const int v = k * EPC + j - mis;
            if (v < 0 || v >= p.V) f[j] = kNegInf;
          }
        } else {
#pragma unroll
          for (int j = 0; j < EPC; ++j) f[j] = kNegInf;
        }
#pragma unroll
        for (int j = 0; j < EPC; ++j) x[q * EPC + j] = f[j];
      }
      float bm = kNegInf;
#pragma unroll
      for (int i = 0; i < NB * EPC; ++i) bm = fmaxf(bm, x[i]);
      const float mn = fmaxf(mloc, bm);
      const float sh = (mn == kNegInf) ? 0.f : mn;
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < NB * EPC; ++i) acc += fast_exp2((x[i] - sh) * kLog2eF);
      sloc = (mloc == kNegInf) ? acc : sloc * fast_exp2((mloc - sh) * kLog2eF) + acc;
      mloc = mn;
    }

    // group max, then every lane's partial sum rescaled to it and summed in float64
    float mg = mloc;
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) mg = fmaxf(mg, __shfl_xor(mg, off, G));
    const float scale = (mloc == kNegInf) ? 0.f : fast_exp2((mloc - mg) * kLog2eF);
    double sd = static_cast<double>(sloc * scale);
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) sd += __shfl_xor(sd, off, G);

    if (lg == 0) {
      const double lse = static_cast<double>(mg) + log(sd);
      const int64_t li = static_cast<int64_t>(b) * p.sb + static_cast<int64_t>(t) * p.st +
                         static_cast<int64_t>(u) * p.su;
      p.lp_blank[li] = static_cast<double>(zb) - lse;
      double lpl = -__builtin_inf();
      if (u < Ub) lpl = (y >= 0 && y < p.V) ? static_cast<double>(zy) - lse : __builtin_nan("");
      p.lp_label[li] = lpl;
      if (p.rowinfo) p.rowinfo[row].lse2 = static_cast<float>(lse * kLog2eD);
      if (p.lse_out) p.lse_out[row] = lse;
    }
  }
}

}  // namespace rnnt
