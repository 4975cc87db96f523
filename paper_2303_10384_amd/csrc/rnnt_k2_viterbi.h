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
// walks back from the path's end, one diagonal per step, reading the words
// through a window of 64 words held one per lane, with the next 64 words loaded
// ahead (so no step waits on memory), and records each unit's frame in LDS.
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

__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(x), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(x >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

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
template <int K, int PF, int VAR>
__global__ __launch_bounds__(64) void k2_viterbi(ViterbiParams p) {
  __shared__ int s_frames[kViterbiMaxUnits1 + 1];  // the last slot takes the stores of blank moves
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int T = p.logit_lens[b];
  const int U = p.label_lens[b];
  const int U1 = p.U_max + 1;
  const int ND = p.T_max + p.U_max;

  bool ok = (T >= 1 && T <= p.T_max && U >= 0 && U <= p.U_max);
  int bad = 0;
  if (ok) {
    for (int u = lane; u < U; u += 64) {
      const int y = p.labels[static_cast<int64_t>(b) * p.U_max + u];
      if (y < 0 || y >= p.V || y == p.blank) bad = 1;
    }
  }
  bad = __syncthreads_or(bad);
  if (!ok || bad) {
    if (lane == 0) p.score_out[b] = __builtin_nanf("");
    for (int i = lane; i < p.U_max; i += 64) p.label_frames[static_cast<int64_t>(b) * p.U_max + i] = -1;
    if (p.span && lane < 2) p.span[2 * b + lane] = -1;
    return;
  }

  const int D = T - 1 + U;
  const int owner_top = U / K;
  const double2* __restrict__ w_utt = p.lp2 + static_cast<int64_t>(b) * p.T_max * U1;
  const __amdgpu_buffer_rsrc_t w_rsrc = make_buffer(w_utt, static_cast<int64_t>(p.T_max) * U1 * 16);
  const int neg_step = -16 * (U1 - 1);
  auto load_w = [&](int e, int k, double& wb, double& wl) {
    const int ec = min(max(e, 0), D);
    const int uc = min(max(lane * K + k, ec - (T - 1)), min(ec, U));
    const double2 w = load_lattice_cell(w_rsrc, 16 * ec * U1, uc, neg_step);  // row (t, u) = (ec - uc, uc)
    wb = w.x;
    wl = w.y;
  };
  uint64_t* __restrict__ dec_utt = p.decisions + static_cast<int64_t>(b) * (ND + 1) * K;
  const double w_close = w_utt[(T - 1) * U1 + U].x;

  // ---------------- forward max-plus sweep ----------------
  double a[K];
#pragma unroll
  for (int k = 0; k < K; ++k) a[k] = (lane * K + k == 0) ? 0.0 : kNoArc;
  double a_top = (U == 0) ? 0.0 : kNoArc;  // delta(T-1, U) once the sweep reaches D
  double left_carry = kNoArc;  // lane 0 gets nothing from the shift and keeps kNoArc
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

  for (int d0 = 1; d0 <= D; d0 += PF) {
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      const int d = d0 + s;  // slot s holds the weights of diagonal d-1
      double eb[K], el[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        eb[k] = a[k] + rb[s][k];
        el[k] = a[k] + rl[s][k];
      }
      left_carry = wave_shift_up(el[K - 1], left_carry);
      const double left = left_carry;
      bool dec[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const double cl = (k == 0) ? left : el[k > 0 ? k - 1 : 0];
        dec[k] = cl > eb[k];  // the label arc wins only when strictly greater
        a[k] = dec[k] ? cl : eb[k];
      }
      // wave-uniform conditions on the diagonal; no memory access inside
      if (VAR != 0 && d <= T - 1 && lane == 0 && 0.0 > a[0]) {  // (0,0)->(d,0), delta(0,0) = 0
        a[0] = 0.0;
        dec[0] = true;
      }
      if (d == D) {
        if (VAR == 1) {
#pragma unroll
          for (int k = 0; k < K; ++k)
            if (lane * K + k == U && acc_top > a[k]) {  // (t*,U)->(T-1,U)
              a[k] = acc_top;
              final_skip = true;
            }
        }
        a_top = at_unit(a, lane, U, a_top);
      }
      if (VAR != 0 && d >= U && d - U <= T - 2) {  // delta(d-U, U), earliest frame on ties
        const double x = at_unit(a, lane, U, kNoArc);
        if (x > acc_top) {
          acc_top = x;
          t_star = d - U;
        }
      }
      // the diagonal's decisions: word k = ballot of slot k; lane l stores word min(l, K-1)
      uint64_t word = 0;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const uint64_t m = __ballot(dec[k]);
        word = (lane == k || (k == K - 1 && lane > k)) ? m : word;
      }
      dec_utt[static_cast<int64_t>(min(d, D + 1)) * K + min(lane, K - 1)] = word;
#pragma unroll
      for (int k = 0; k < K; ++k) load_w(d - 1 + PF, k, rb[s][k], rl[s][k]);
      __builtin_amdgcn_sched_barrier(0);  // the prefetch stays PF steps ahead of its use
    }
  }

  // the path's end (values of the lane owning u = U)
  a_top = from_lane(a_top, owner_top);
  acc_top = from_lane(acc_top, owner_top);
  t_star = from_lane(t_star, owner_top);
  const bool skip_in = from_lane(static_cast<int>(final_skip), owner_top) != 0;
  double best2 = a_top + w_close;  // closing blank
  int t = T - 1, end_frame = T - 1;
  if (VAR == 1 && skip_in) t = end_frame = t_star;
  if (VAR == 2 && acc_top > best2) {  // (t*,U)->final beats the closing blank
    best2 = acc_top;
    t = end_frame = t_star;
  }

  // ---------------- backtrace ----------------
  __syncthreads();  // the decision words stored above are read back below
  int u = U, start_frame = 0;
  // Two windows of 64 words, one per lane, in turn: the walk reads one while the next
  // 64 words below load into the other (a copy between them would wait for that load).
  // A step moves the word index down by at most 2K-1 < 64, so the walk leaves a window
  // only into the next one.
  auto load_window = [&](int lo) { return lo + lane >= 0 ? dec_utt[lo + lane] : uint64_t{0}; };
  // walks while its word lies in [lo, lo + 64); true once (0,0) is reached or the path jumped
  auto walk = [&](const uint64_t& win, int lo) {
    while (t + u > 0) {
      const unsigned uu = static_cast<unsigned>(u);  // u >= 0: unsigned division by K is a shift or a multiply
      const int widx = (t + u) * K + static_cast<int>(uu % K);
      if (widx < lo) return false;
      const uint64_t wd = readlane_u64(win, widx - lo);
      // the move, without branches and in integer 0/1 flags (scalar arithmetic; boolean
      // flags went through a vector select and back): the label arc (t,u-1)->(t,u) (the
      // only way into (0,u)) emits unit u at frame t; at u = 0 a set bit is the initial
      // wild-card arc from (0,0).  t, u >= 0 here.
      const unsigned bit = static_cast<unsigned>(wd >> (uu / K)) & 1u;
      const unsigned u_pos = static_cast<unsigned>(-u) >> 31;      // u > 0
      const unsigned t_zero = static_cast<unsigned>(t - 1) >> 31;  // t == 0
      const int label = static_cast<int>(u_pos & (bit | t_zero));
      const bool jumped = VAR != 0 && (bit & (u_pos ^ 1u)) != 0;
      s_frames[label ? u - 1 : kViterbiMaxUnits1] = t;  // every lane the same value; a spare slot otherwise
      start_frame = jumped ? t : start_frame;
      u -= label;
      t = jumped ? 0 : t - 1 + label;  // a jump ends the walk: (t,u) becomes (0,0)
    }
    return true;
  };
  int lo = (t + u) * K + K - 64;
  uint64_t win_a = load_window(lo);
  uint64_t win_b = load_window(lo - 64);
  while (true) {
    if (walk(win_a, lo)) break;
    lo -= 64;
    win_a = load_window(lo - 64);
    if (walk(win_b, lo)) break;
    lo -= 64;
    win_b = load_window(lo - 64);
  }
  __syncthreads();
  for (int i = lane; i < p.U_max; i += 64)
    p.label_frames[static_cast<int64_t>(b) * p.U_max + i] = (i < U) ? s_frames[i] : -1;
  if (lane == 0) {
    p.score_out[b] = static_cast<float>(best2 / kLog2eD);
    if (p.span) {
      p.span[2 * b] = start_frame;
      p.span[2 * b + 1] = end_frame;
    }
  }
}

}  // namespace rnnt
