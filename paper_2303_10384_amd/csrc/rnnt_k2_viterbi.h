// Kernel 2v: forced alignment -- the single best path through the grid lattice
// of Fig. 1 (or the W-Transducer lattices of Fig. 4 and Section 4.3), which the
// lattice formulation serves as well as training (Section 2.2).
//
// The forward recursion of kernel 2 with the log-sum replaced by a maximum
// (log2 units, kernel 1's lattice form):
//   delta(t,u) = max(delta(t-1,u) + lp_blank(t-1,u), delta(t,u-1) + lp_label(t,u-1))
// plus, for the W-Transducer, the initial wild-card arc into (t,0) and the final
// wild-card arcs into (T-1,U) (force-final) or into the final state
// (allow-ignore).  Ties go, in this order, to the blank arc, the label arc, the
// initial wild-card arc, the final wild-card arcs (the earliest source frame),
// and at the end of the allow-ignore lattice to the closing blank: a later
// candidate wins only when strictly greater.
//
// One wavefront per utterance sweeps the anti-diagonals as kernel 2's forward
// wave does (lane j owns units K*j .. K*j+K-1).  A node's decision is one bit:
// 1 when it is entered by its label arc, or at u = 0 by the initial wild-card
// arc.  Each step stores, per lane slot k, the wave's ballot of those bits: one
// 64-bit word per (diagonal, k), bit j for unit K*j + k.  The same wave then
// walks back from the path's end one label move at a time, finding each unit's
// entry diagonal among 64 at once (a ballot of that unit's bits over a block of
// diagonals staged in LDS, the next block loaded ahead), and records each unit's
// frame in LDS.
#pragma once

#include "rnnt_device.h"
#include "rnnt_k2_lattice.h"

namespace rnnt {

struct ViterbiParams {
  int32_t B, T_max, U_max, V, blank;
  const int32_t* labels;  // (B, U_max)
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const double2* lp2;      // kernel 1's lattice form (log2 units, (B, T_max, U_max+1))
  uint64_t* decisions;     // (B, T_max+U_max+1, K) ballot words
  float* score_out;        // (B) best path log-probability (natural log), NaN for bad data
  int32_t* label_frames;   // (B, U_max): frame of unit i+1, -1 past U_b or for bad data
  int32_t* span;           // (B, 2) start / end frame, or null
};

constexpr int kViterbiMaxUnits1 = 2048;

template <typename V>
__device__ __forceinline__ V from_lane(V x, int lane) {
  if constexpr (sizeof(V) == 8) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(x), lane);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(x), lane);
    return __hiloint2double(hi, lo);
  } else {
    return __builtin_amdgcn_readlane(x, lane);
  }
}

// VAR: 0 RNN-T, 1 W-Transducer force-final, 2 allow-ignore.
// NW: wavefronts in the sweep, as in kernel 2: wave w owns units 64w .. 64w+63 (one
// per lane), runs a segment of PF steps behind wave w-1 and takes the label-arc term
// of unit 64w-1 from it through LDS.  Its decision word of a diagonal is then word w,
// bit u - 64w (one word per wave and diagonal instead of one per lane slot).  The
// backtrace is wave 0's.
template <int K, int PF, int VAR, int NW = 1>
__global__ __launch_bounds__(64 * NW) void k2_viterbi(ViterbiParams p) {
  static_assert(NW == 1 || K == 1, "several waves take one unit per lane");
  constexpr int kCols = NW > 1 ? NW : K;  // decision words per diagonal
  __shared__ int s_frames[kViterbiMaxUnits1 + 1];  // the last slot takes the stores of blank moves
  __shared__ double s_xch[NW > 1 ? NW - 1 : 1][2][PF];
  __shared__ double s_sink[NW > 1 ? kWave + PF : 1];
  __shared__ double s_end[2];  // the path's end, from the lane owning u = U: delta(T-1, U), acc_top
  __shared__ int s_end_i[2];   // t_star, final_skip
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wv = (NW == 1) ? 0 : __builtin_amdgcn_readfirstlane(tid / kWave);
  const int ub = wv * kWave * K;  // this wave's first unit
  const int T = p.logit_lens[b];
  const int U = p.label_lens[b];
  const int U1 = p.U_max + 1;
  const int ND = p.T_max + p.U_max;

  bool ok = (T >= 1 && T <= p.T_max && U >= 0 && U <= p.U_max);
  int bad = 0;
  if (ok) {
    for (int u = tid; u < U; u += blockDim.x) {
      const int y = p.labels[static_cast<int64_t>(b) * p.U_max + u];
      if (y < 0 || y >= p.V || y == p.blank) bad = 1;
    }
  }
  bad = __syncthreads_or(bad);
  if (!ok || bad) {  // the whole block leaves together
    if (tid == 0) p.score_out[b] = __builtin_nanf("");
    for (int i = tid; i < p.U_max; i += blockDim.x) p.label_frames[static_cast<int64_t>(b) * p.U_max + i] = -1;
    if (p.span && tid < 2) p.span[2 * b + tid] = -1;
    return;
  }

  const int D = T - 1 + U;
  const int owner_top = (U - ub) / K;  // in the wave owning u = U
  const bool owns_top = (U / (kWave * K) == wv) && lane == owner_top;
  const double2* __restrict__ w_utt = p.lp2 + static_cast<int64_t>(b) * p.T_max * U1;
  const __amdgpu_buffer_rsrc_t w_rsrc = make_buffer(w_utt, static_cast<int64_t>(p.T_max) * U1 * 16);
  const int neg_step = -16 * (U1 - 1);
  auto load_w = [&](int e, int k, double& wb, double& wl) {
    const int ec = min(max(e, 0), D);
    const int uc = min(max(ub + lane * K + k, ec - (T - 1)), min(ec, U));
    const double2 w = load_lattice_cell(w_rsrc, 16 * ec * U1, uc, neg_step);  // row (t, u) = (ec - uc, uc)
    wb = w.x;
    wl = w.y;
  };
  uint64_t* __restrict__ dec_utt = p.decisions + static_cast<int64_t>(b) * (ND + 1) * kCols;
  const double w_close = w_utt[(T - 1) * U1 + U].x;

  // ---------------- forward max-plus sweep ----------------
  double a[K];
#pragma unroll
  for (int k = 0; k < K; ++k) a[k] = (ub + lane * K + k == 0) ? 0.0 : kNoArc;
  double a_top = (U == 0) ? 0.0 : kNoArc;  // delta(T-1, U) once the sweep reaches D
  double left_carry = kNoArc;  // lane 0 of wave 0 gets nothing from the shift and keeps kNoArc
  double acc_top = kNoArc;                 // best delta(t', U), t' <= T-2, and its earliest frame
  int t_star = -1;
  if (VAR != 0 && U == 0 && T >= 2) {
    acc_top = 0.0;  // delta(0, U) itself when U = 0
    t_star = 0;
  }
  bool final_skip = false;  // (T-1, U) entered by a final wild-card arc (force-final)

  double rb[PF][K], rl[PF][K];
#pragma unroll
  for (int s = 0; s < PF; ++s) {
#pragma unroll
    for (int k = 0; k < K; ++k) load_w(s, k, rb[s][k], rl[s][k]);
    __builtin_amdgcn_sched_barrier(0);  // issue order = use order (oldest first)
  }

  double x_in[PF];  // lane 0: the fill of each step of a segment (several waves; kNoArc for wave 0)
#pragma unroll
  for (int s = 0; s < PF; ++s) x_in[s] = kNoArc;
  const int n_seg = (D + PF - 1) / PF;
  for (int r = 0; r < n_seg + NW - 1; ++r) {  // every wave passes one barrier per round (several waves)
    const int g = r - wv;  // this wave's segment in round r
    if (g >= 0 && g < n_seg) {
    const int d0 = 1 + g * PF;
    if (NW > 1 && wv > 0) {  // the wave before wrote this segment's values in the previous round
#pragma unroll
      for (int s = 0; s < PF; ++s) x_in[s] = s_xch[max(wv - 1, 0)][(r - 1) & 1][s];
    }
    // lane 63 writes into this round's slots for the next wave, the others into the sink
    double* const x_out = (lane == kWave - 1 && wv < NW - 1) ? &s_xch[min(wv, NW > 1 ? NW - 2 : 0)][r & 1][0]
                                                              : &s_sink[NW > 1 ? lane : 0];
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      const int d = d0 + s;  // slot s holds the weights of diagonal d-1
      double eb[K], el[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        eb[k] = a[k] + rb[s][k];
        el[k] = a[k] + rl[s][k];
      }
      if (NW > 1) x_out[s] = el[K - 1];  // lane 63's for wave wv+1
      double& fill = (NW > 1) ? x_in[s] : left_carry;  // in place: lane 0 keeps the fill
      fill = wave_shift_up(el[K - 1], fill);
      const double left = fill;
      bool dec[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const double cl = (k == 0) ? left : el[k > 0 ? k - 1 : 0];
        dec[k] = cl > eb[k];  // the label arc wins only when strictly greater
        a[k] = dec[k] ? cl : eb[k];
      }
      // wave-uniform conditions on the diagonal; no memory access inside
      if (VAR != 0 && d <= T - 1 && wv == 0 && lane == 0 && 0.0 > a[0]) {  // (0,0)->(d,0), delta(0,0) = 0
        a[0] = 0.0;
        dec[0] = true;
      }
      if (d == D) {
        if (VAR == 1) {
#pragma unroll
          for (int k = 0; k < K; ++k)
            if (ub + lane * K + k == U && acc_top > a[k]) {  // (t*,U)->(T-1,U)
              a[k] = acc_top;
              final_skip = true;
            }
        }
        a_top = at_unit(a, lane, U - ub, a_top);
      }
      if (VAR != 0 && d >= U && d - U <= T - 2) {  // delta(d-U, U), earliest frame on ties
        const double x = at_unit(a, lane, U - ub, kNoArc);
        if (x > acc_top) {
          acc_top = x;
          t_star = d - U;
        }
      }
      // the diagonal's decisions: word k = ballot of slot k, lane l storing word min(l, K-1);
      // several waves: wave w's ballot is word w
      uint64_t word = 0;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const uint64_t m = __ballot(dec[k]);
        word = (lane == k || (k == K - 1 && lane > k)) ? m : word;
      }
      dec_utt[static_cast<int64_t>(min(d, D + 1)) * kCols + (NW > 1 ? wv : min(lane, K - 1))] = word;
#pragma unroll
      for (int k = 0; k < K; ++k) load_w(d - 1 + PF, k, rb[s][k], rl[s][k]);
      __builtin_amdgcn_sched_barrier(0);  // the prefetch stays PF steps ahead of its use
    }
    }
    if (NW > 1) __syncthreads();  // the segment's values reach the next wave
  }

  // the path's end (values of the lane owning u = U; through LDS from another wave)
  bool skip_in;
  if (NW == 1) {
    a_top = from_lane(a_top, owner_top);
    acc_top = from_lane(acc_top, owner_top);
    t_star = from_lane(t_star, owner_top);
    skip_in = from_lane(static_cast<int>(final_skip), owner_top) != 0;
  } else {
    if (owns_top) {
      s_end[0] = a_top;
      s_end[1] = acc_top;
      s_end_i[0] = t_star;
      s_end_i[1] = static_cast<int>(final_skip);
    }
    __syncthreads();
    a_top = s_end[0];
    acc_top = s_end[1];
    t_star = s_end_i[0];
    skip_in = s_end_i[1] != 0;
  }
  double best2 = a_top + w_close;  // closing blank
  int t = T - 1, end_frame = T - 1;
  if (VAR == 1 && skip_in) t = end_frame = t_star;
  if (VAR == 2 && acc_top > best2) {  // (t*,U)->final beats the closing blank
    best2 = acc_top;
    t = end_frame = t_star;
  }

  // ---------------- backtrace ----------------
  __syncthreads();  // the decision words stored above are read back below
  // One step per label move: from node (d - u, u) the path runs down blank arcs (d
  // falls, u stays) to the highest diagonal d' <= d whose node of unit u was entered by
  // its label arc -- at t = 0 it always is -- emits unit u at frame d' - u and goes on
  // from (d' - u, u - 1) on diagonal d' - 1.  Unit u's decision bits over a block of 64
  // diagonals are one ballot: lane l reads the word of diagonal 64 w + l in unit u's
  // column (u % K, or u / 64 with several waves; the block staged in LDS, one column
  // per 64 words) and tests unit u's bit (u / K, or u % 64).  At u = 0 (W-Transducer) a
  // set bit is the initial wild-card arc: the path starts there.  Each step lowers d,
  // so the walk ends after at most U + D/64 + 1 steps.  Wave 0 walks.
  __shared__ uint64_t s_blk[kCols][kWave];
  const __amdgpu_buffer_rsrc_t dec_rsrc = make_buffer(dec_utt, static_cast<int64_t>(ND + 1) * kCols * 8);
  // the words of diagonal 64 w + lane, all columns (0 past the stored rows)
  auto load_block = [&](int w, uint64_t (&x)[kCols]) {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int c = 0; c < kCols; ++c) {
      const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(dec_rsrc, ((kWave * w + lane) * kCols + c) * 8, 0, 0);
      x[c] = (static_cast<uint64_t>(v.y) << 32) | v.x;
    }
  };
  int u = U, d = t + u, start_frame = 0;
  if (wv == 0) {
  int w = d / kWave;
  uint64_t nxt[kCols];
  load_block(w, nxt);
#pragma unroll
  for (int c = 0; c < kCols; ++c) s_blk[c][lane] = nxt[c];
  if (w > 0) load_block(w - 1, nxt);  // the block below, in flight while this one is walked
  while (d > 0 && (VAR != 0 || u > 0)) {
    if (d < kWave * w) {  // one block down (a step lowers the block by at most one)
      w -= 1;
#pragma unroll
      for (int c = 0; c < kCols; ++c) s_blk[c][lane] = nxt[c];
      if (w > 0) load_block(w - 1, nxt);
    }
    const unsigned uu = static_cast<unsigned>(u);
    const uint64_t col = s_blk[NW > 1 ? uu / kWave : uu % K][lane];
    const unsigned bit_of_u = NW > 1 ? uu % kWave : uu / K;
    const uint64_t bits = __ballot(static_cast<int>((col >> bit_of_u) & 1u));  // bit l: diagonal 64 w + l
    const int base = kWave * w;
    const int lo = max(u, 1) - base;  // t >= 0, and never diagonal 0 (node (0,0) has no decision)
    const int hi = d - base;          // lo <= hi <= 63
    const uint64_t m = bits & (~uint64_t{0} >> (63 - hi)) & (~uint64_t{0} << max(lo, 0));
    if (u > 0) {
      int dl;
      if (m != 0) {
        dl = base + 63 - __builtin_clzll(m);
      } else if (u >= base) {
        dl = u;  // t = 0: entered by its label arc
      } else {
        d = base - 1;  // no label move in this block
        continue;
      }
      s_frames[u - 1] = dl - u;  // every lane the same value
      u -= 1;
      d = dl - 1;
    } else {  // u = 0, W-Transducer: the initial wild-card arc into (t, 0), or (0, 0) itself
      if (m != 0) {
        start_frame = base + 63 - __builtin_clzll(m);
        break;
      }
      d = base - 1;
    }
  }
  }
  __syncthreads();
  for (int i = tid; i < p.U_max; i += blockDim.x)
    p.label_frames[static_cast<int64_t>(b) * p.U_max + i] = (i < U) ? s_frames[i] : -1;
  if (tid == 0) {
    p.score_out[b] = static_cast<float>(best2 / kLog2eD);
    if (p.span) {
      p.span[2 * b] = start_frame;
      p.span[2 * b + 1] = end_frame;
    }
  }
}

}  // namespace rnnt
