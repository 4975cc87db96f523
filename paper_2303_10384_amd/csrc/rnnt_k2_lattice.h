// Kernel 2: forward / backward scores on the grid lattice of one utterance,
// and kernel 2b: arc posteriors of every lattice node.
//
// Eq. 1's Fwd in the log semiring over the lattice of Fig. 1 (Fig. 4 for the
// W-Transducer), and the matching backward scores (log2 units here):
//   alpha(0,0) = 0
//   alpha(t,u) = log2[ 2^{alpha(t-1,u) + lp_blank(t-1,u)} + 2^{alpha(t,u-1) + lp_label(t,u-1)} ]
//   beta(T-1,U) = lp_blank(T-1,U)                               (closing blank)
//   beta(t,u)  = log2[ 2^{lp_blank(t,u) + beta(t+1,u)} + 2^{lp_label(t,u) + beta(t,u+1)} ]
//   log2 P = alpha(T-1,U) + lp_blank(T-1,U) = beta(0,0)
// W-Transducer, force-final (Section 3.2, Fig. 4): weight-0 arcs (0,0)->(t,0)
// for t >= 1 and (t,U)->(T-1,U) for t <= T-2.  Allow-ignore (Section 4.3): the
// latter end in the final state instead.
//
// Schedule: the nodes of an anti-diagonal d = t + u depend only on diagonal
// d-1 (forward) or d+1 (backward).  One wavefront sweeps the diagonals, lane j
// owning the K consecutive units u = K*j .. K*j+K-1, so a step exchanges one
// value with the neighbouring lane (a DPP whole-wave shift); from 65 to 256
// units, two to four wavefronts with one unit per lane do, staggered by a
// segment of steps and exchanging their boundary values through LDS (see the
// kernel's NW parameter).  The forward and
// backward sweeps of an utterance run concurrently, each in a block of its own
// (blockIdx.y), so that the two chains do not share a compute unit.  The weights of
// the next PF diagonals stay in flight in registers (one load per unit and
// diagonal).  No node is masked:
// absent arcs carry kNoArc, so a node outside the utterance accumulates only
// kNoArc or never feeds a node inside it; weights of cells outside the
// utterance are read from a cell clamped into it (a wave-uniform diagonal and
// two per-lane min/max on the unit), so every value stays finite.  Kernel 1
// stores the weights by row, so a diagonal's cells lie U_max rows apart and a
// 128-byte line of them serves eight consecutive diagonals.  alpha and
// beta rows are 64*K wide, one column per lane slot, and the
// steps past the utterance's last diagonal (or before the first) store into
// spare rows, so every load and store goes through a wave-uniform row pointer
// plus a constant lane offset and none sits under a branch.  No wild-card arc
// lengthens a step's chain: the arc into (t,0) is unit 0's second log-add term
// (it has no unit below), the arc out of (t,U) takes the place of unit U's
// absent label arc, and the two log-sums over frames they need (of alpha(t,U)
// and of beta(t,0)) go through LDS to per-lane sums once per segment; the one
// cell each changes is stored again after the sweep.
//
// Kernel 2b, for every padded row (t, u):
//   occ_blank(t,u) = 2^(alpha(t,u) + lp_blank(t,u) + beta(t+1,u) - log2 P)   (t < T-1)
//   occ_blank(T-1,U) = 2^(alpha(T-1,U) + lp_blank(T-1,U) - log2 P)
//   occ_label(t,u) = 2^(alpha(t,u) + lp_label(t,u) + beta(t,u+1) - log2 P)   (u < U)
// written as the row record of the gradient kernel (zero rows for padding and
// for bad utterances), or as dense float64 outputs.
#pragma once

#include "rnnt_device.h"

namespace rnnt {

enum LatticeMode : int {
  kLossOnly = 0,  // forward wave only, nothing stored but ln P and the loss
  kScores = 1,    // forward and backward waves, alpha and beta stored
};

struct LatticeParams {
  int32_t B, T_max, U_max, V, blank;
  const int32_t* labels;  // (B, U_max) or null (lattice-only entry point)
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const double2* lp2;       // kernel 1's lattice form (log2 units, (B, T_max, U_max+1), kNoArc marks), or
  const double* lp_blank;   // dense natural-log weights (B, T_max, U_max+1)
  const double* lp_label;
  double* alpha;  // (B, T_max+U_max+1, u_pad), by diagonal, log2 units; rows past D_b + 1: spare
  double* beta;
  int32_t u_pad;     // row width of alpha / beta: 64 * units per lane
  double* lnp2_fwd;  // (B) log2 P from the forward wave
  double* lnp2_bwd;  // (B) beta(0,0)
  int32_t* status;   // (B) 0: good, 1: bad data
  float* loss_f32;   // (B) or null
};

// Weights of cell (d, u) after clamping it into the utterance's cells (cells
// outside read a valid cell's weights; nothing downstream depends on them).
template <bool DENSE_IN>
__device__ __forceinline__ void load_cell(const LatticeParams& p, int b, int d, int u, int T, int U, int D,
                                          double& wb, double& wl) {
  const int dc = min(max(d, 0), D);
  const int uc = min(max(u, dc - (T - 1)), min(dc, U));
  if (!DENSE_IN) {
    const int64_t row = (static_cast<int64_t>(b) * p.T_max + (dc - uc)) * (p.U_max + 1) + uc;
    const double2 w = p.lp2[row];
    wb = w.x;
    wl = w.y;
  } else {
    const int64_t row = (static_cast<int64_t>(b) * p.T_max + (dc - uc)) * (p.U_max + 1) + uc;
    wb = p.lp_blank[row];
    wl = p.lp_label[row];
  }
}

// Dense natural-log weights turned into the lattice form at their use: log2
// units, kNoArc for absent arcs and for -inf.
__device__ __forceinline__ double to_lattice(double w_ln, bool present) {
  const double w = w_ln * kLog2eD;
  return present ? (w < kNoArc ? kNoArc : w) : kNoArc;
}

__device__ __forceinline__ double wave_shift_up(double x, double fill) {
  // lane i receives lane i-1's value, lane 0 receives `fill` (DPP wave_shr:1)
  const int lo = __builtin_amdgcn_update_dpp(static_cast<int>(__double2loint(fill)),
                                             static_cast<int>(__double2loint(x)), 0x138, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(static_cast<int>(__double2hiint(fill)),
                                             static_cast<int>(__double2hiint(x)), 0x138, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double wave_shift_down(double x, double fill) {
  // lane i receives lane i+1's value, lane 63 receives `fill` (DPP wave_shl:1)
  const int lo = __builtin_amdgcn_update_dpp(static_cast<int>(__double2loint(fill)),
                                             static_cast<int>(__double2loint(x)), 0x130, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(static_cast<int>(__double2hiint(fill)),
                                             static_cast<int>(__double2hiint(x)), 0x130, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}

// Number of units a lane owns so that 64 lanes cover U_max + 1 units.
// Units per lane of the sweeps: the smallest of 1, 2, 3, 4, 6, 8, 12, 16 with 64
// lanes covering U_max + 1 units (a lane's step costs about K cells).
__host__ __device__ constexpr int units_per_lane(int units1) {
  return units1 <= 64 ? 1 : units1 <= 128 ? 2 : units1 <= 192 ? 3 : units1 <= 256 ? 4
       : units1 <= 384 ? 6 : units1 <= 512 ? 8 : units1 <= 768 ? 12 : units1 <= 1024 ? 16
       : units1 <= 1536 ? 24 : 32;
}

// The value of unit u in this lane's slots (x[k] holds unit lane*K + k), or
// `other` in lanes not owning u.  Selecting by the per-lane unit, never by a
// slot number, keeps every index into x static (a run-time slot index would
// move the array out of registers).
template <int K>
__device__ __forceinline__ double at_unit(const double (&x)[K], int lane, int u, double other) {
  double r = other;
#pragma unroll
  for (int k = 0; k < K; ++k) r = (lane * K + k == u) ? x[k] : r;
  return r;
}

// Log-sum (log2 units) over the 64 lanes of a wave; every lane gets the result.
__device__ __forceinline__ double wave_log_sum(double x) {
#pragma unroll
  for (int m = kWave / 2; m >= 1; m /= 2) x = log_add2(x, __shfl_xor(x, m, kWave));
  return x;
}

// VAR: 0 RNN-T, 1 W-Transducer force-final, 2 allow-ignore.
// DENSE_IN: weights from the dense natural-log arrays instead of kernel 1.
// NW: wavefronts per sweep.  Wave w owns units w*64*K .. (w+1)*64*K - 1 (unit u
// still sits in column u of the score rows) and runs the diagonals a whole
// segment of PF steps behind the wave it depends on: the forward wave w after
// wave w-1 (its lane 0 needs the label-arc term of the unit below it), the
// backward wave w after wave w+1 (its lane 63 needs beta of the unit above).
// The neighbouring wave's values of a segment go through LDS, one per step,
// and every wave passes one barrier per segment, active or not, so every wave
// reaches the same barriers.  One unit per lane shortens a step's dependent
// chain to one log-add; the stagger costs NW-1 segments per sweep.
template <int K, int PF, int VAR, int MODE, bool DENSE_IN, int NW = 1>
__global__ __launch_bounds__(64 * NW) void k2_lattice(LatticeParams p) {
  static_assert(NW >= 1 && NW <= 4, "one to four waves per sweep");
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int T = p.logit_lens[b];
  const int U = p.label_lens[b];
  const int U1 = p.U_max + 1;
  const int ND = p.T_max + p.U_max;  // diagonals of the lattice form
  const double kNaN = __builtin_nan("");
  // the neighbouring wave's value of each step of a segment, two segments in turn;
  // every lane writes each step (no exec mask), the lanes without a value to pass
  // into a scratch run of their own (lane + step: no two lanes of a write collide)
  __shared__ double s_xch[NW > 1 ? NW - 1 : 1][2][PF];
  __shared__ double s_sink[NW > 1 || VAR != 0 ? kWave + PF : 1];
  // W-Transducer: the segment's values of the one node whose scores are summed over
  // the sweep (alpha(d-U, U) forward, beta(d, 0) backward), one per step
  __shared__ double s_sum[VAR != 0 ? PF : 1];

  bool ok = (T >= 1 && T <= p.T_max && U >= 0 && U <= p.U_max);
  int bad = 0;
  if (ok && p.labels != nullptr) {
    for (int u = tid; u < U; u += blockDim.x) {
      const int y = p.labels[static_cast<int64_t>(b) * p.U_max + u];
      if (y < 0 || y >= p.V || y == p.blank) bad = 1;
    }
  }
  bad = __syncthreads_or(bad);
  // both sweeps of an utterance reach the same verdict and store the same values
  if (tid == 0) p.status[b] = (ok && !bad) ? 0 : 1;
  if (!ok || bad) {  // the whole block leaves together
    if (tid == 0) {
      p.lnp2_fwd[b] = kNaN;
      p.lnp2_bwd[b] = kNaN;
      if (p.loss_f32) p.loss_f32[b] = __builtin_nanf("");
    }
    return;
  }

  const int sweep = blockIdx.y;  // 0: forward, 1: backward (a block of its own)
  const int lane = tid % kWave;
  const int wv = (NW == 1) ? 0 : __builtin_amdgcn_readfirstlane(tid / kWave);
  const int ub = wv * kWave * K;  // this wave's first unit
  const int D = T - 1 + U;        // last diagonal
  // the lane owning u = U, in the wave owning it
  const bool owns_top = (U / (kWave * K) == wv) && lane == (U - ub) / K;
  // weights of cell (e, u) clamped into the utterance: diagonal into [0, D], then the
  // unit into [e - (T-1), min(e, U)] (t = e - u in [0, T-1]); the row pointer is wave-uniform
  const double2* __restrict__ w_utt = p.lp2 + static_cast<int64_t>(b) * p.T_max * U1;
  const __amdgpu_buffer_rsrc_t w_rsrc = make_buffer(w_utt, static_cast<int64_t>(p.T_max) * U1 * 16);
  // the per-unit factor in a vector register, so the offset's multiply-add takes the
  // row term as its one scalar operand
  int neg_step;
  asm volatile("v_mov_b32 %0, %1" : "=v"(neg_step) : "s"(-16 * (U1 - 1)));
  auto load_w = [&](int e, int k, double& wb, double& wl) {
    if (!DENSE_IN) {
      const int ec = min(max(e, 0), D);
      // the unit's upper clamp as one scalar (a min against two scalars costs a vector move)
      const int hi = __builtin_amdgcn_readfirstlane(min(ec, U));
      const int uc = min(max(ub + lane * K + k, ec - (T - 1)), hi);
      const double2 w = load_lattice_cell(w_rsrc, 16 * ec * U1, uc, neg_step);  // row (t, u) = (ec - uc, uc)
      wb = w.x;
      wl = w.y;
    } else {
      load_cell<true>(p, b, e, ub + lane * K + k, T, U, D, wb, wl);
    }
  };
  // score rows: diagonals 0..D, then spare rows up to ND
  double* __restrict__ a_utt = p.alpha + static_cast<int64_t>(b) * (ND + 1) * p.u_pad;
  double* __restrict__ b_utt = p.beta + static_cast<int64_t>(b) * (ND + 1) * p.u_pad;
  // score rows through per-utterance buffers: the row's byte offset is wave-uniform
  // (the host keeps (T_max + U_max + 1) * u_pad * 8 under 2^31), the lane's fixed
  const __amdgpu_buffer_rsrc_t a_rsrc = make_buffer(a_utt, static_cast<int64_t>(ND + 1) * p.u_pad * 8);
  const __amdgpu_buffer_rsrc_t b_rsrc = make_buffer(b_utt, static_cast<int64_t>(ND + 1) * p.u_pad * 8);
  const int lane_off = (ub + lane * K) * 8;
  const int row_bytes = p.u_pad * 8;
  // segments of PF steps in a sweep of D steps, and the barriers every wave passes
  const int n_seg = (D + PF - 1) / PF;
  const int n_rounds = n_seg + NW - 1;

  // weight of the closing blank, lp_blank(T-1, U)
  double w_close, w_unused;
  if (!DENSE_IN) {
    w_close = w_utt[(T - 1) * U1 + U].x;
  } else {
    load_cell<true>(p, b, D, U, T, U, D, w_close, w_unused);
    w_close = to_lattice(w_close, true);
  }

  if (sweep == 0) {
    // ---------------- forward sweep ----------------
    double a[K];
#pragma unroll
    for (int k = 0; k < K; ++k) a[k] = (ub + lane * K + k == 0) ? 0.0 : kNoArc;
    double a_top = (U == 0) ? 0.0 : kNoArc;    // alpha(T-1, U) once the sweep reaches D
    // the shifted-in neighbour; in RNN-T lane 0 of wave 0 gets none from the shift and
    // keeps kNoArc from here on, so no fill value is set up in each step
    double left_carry = kNoArc;
    // W-Transducer: log-sum of alpha(t, U), t <= T-2, kept per lane (lane s sums the
    // steps s of every segment) in the wave owning unit U and summed over lanes at the
    // end; the owning lane's only work in a step is one LDS store
    const int w_top = U / (kWave * K);
    double acc_lane = kNoArc;
    if (VAR != 0 && U == 0 && T >= 2 && lane == 0) acc_lane = 0.0;  // alpha(0, U) itself when U = 0
    double* const sum_out = owns_top ? &s_sum[0] : &s_sink[VAR != 0 ? lane : 0];
    if (MODE != kLossOnly && wv == 0 && lane == 0) a_utt[0] = 0.0;

    double rb[PF][K], rl[PF][K];
#pragma unroll
    for (int s = 0; s < PF; ++s) {
#pragma unroll
      for (int k = 0; k < K; ++k) load_w(s, k, rb[s][k], rl[s][k]);
      __builtin_amdgcn_sched_barrier(0);  // issue order = use order (oldest first)
    }
    double x_in[PF];  // lane 0: the fill of each step of a segment (several waves)
#pragma unroll
    for (int s = 0; s < PF; ++s) x_in[s] = kNoArc;

    // whole segments of PF steps, no branch around loads or stores; the up to PF-1
    // steps past D touch only nodes outside the utterance and store into spare rows
    for (int r = 0; r < n_rounds; ++r) {
      const int g = r - wv;  // this wave's segment in round r
      if (g >= 0 && g < n_seg) {
        const int d0 = 1 + g * PF;
        // the wave before wrote this segment's values in the previous round: all of them
        // are read at once, so no step waits on the LDS (wave 0 has no wave before it)
        if (NW > 1 && wv > 0) {
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
            double wb = rb[s][k], wl = rl[s][k];
            if (DENSE_IN) {
              const int u = ub + lane * K + k, t = d - 1 - u;
              wb = to_lattice(wb, t < T - 1 || u == U);
              wl = to_lattice(wl, u < U);
            }
            eb[k] = a[k] + wb;
            el[k] = a[k] + wl;
          }
          if (NW > 1) x_out[s] = el[K - 1];  // lane 63's for wave wv+1
          // lane 0 of a later wave takes the unit below it from the wave before, one segment
          // old.  The shift writes over its own fill register, whose lane 0 keeps the fill
          // (the only lane of it ever read), so no copy of the fill precedes it.  Unit 0 has
          // no unit below; in the W-Transducer its second term is the skip arc (0,0)->(d,0)
          // of weight 0 from alpha(0,0) = 0, so no second log-add follows on the chain
          // (log_add2(x, kNoArc) is exactly x)
          double& fill = (NW > 1) ? x_in[s] : left_carry;
          if (VAR != 0 && wv == 0) fill = (d <= T - 1) ? 0.0 : kNoArc;
          fill = wave_shift_up(el[K - 1], fill);
          const double left = fill;
#pragma unroll
          for (int k = 0; k < K; ++k) a[k] = log_add2(eb[k], k == 0 ? left : el[k > 0 ? k - 1 : 0]);
          // once per sweep, wave-uniform: a branch, not selects in every step.  The force-final
          // skip arcs into (T-1, U) are added after the sweep: no later step reads alpha(T-1, U)
          if (__builtin_expect(d == D, 0)) a_top = at_unit(a, lane, U - ub, a_top);
          if (VAR != 0) sum_out[s] = K == 1 ? a[0] : at_unit(a, lane, U - ub, kNoArc);
          if (MODE != kLossOnly)  // the row offset is uniform; readfirstlane keeps it in a scalar register
            store_scores<K>(a_rsrc, lane_off, __builtin_amdgcn_readfirstlane(min(d, D + 1) * row_bytes), a);
#pragma unroll
          for (int k = 0; k < K; ++k) load_w(d - 1 + PF, k, rb[s][k], rl[s][k]);
          __builtin_amdgcn_sched_barrier(0);  // the prefetch stays PF steps ahead of its use
        }
        if (VAR != 0 && wv == w_top) {  // lane s: alpha(d-U, U) of step s, if 0 <= d-U <= T-2
          const int dl = d0 + lane;     // (a wave's LDS accesses complete in order)
          const double x = s_sum[min(lane, PF - 1)];
          acc_lane = log_add2(acc_lane, (lane < PF && dl >= U && dl - U <= T - 2) ? x : kNoArc);
        }
      }
      if (NW > 1) __syncthreads();  // the segment's values reach the next wave
    }
    double acc_top = kNoArc;  // log-sum of alpha(t, U), t <= T-2
    if (VAR != 0 && wv == w_top) acc_top = wave_log_sum(acc_lane);
    if (VAR == 1 && owns_top) {
      a_top = log_add2(a_top, acc_top);  // (t,U)->(T-1,U)
      if (MODE != kLossOnly) {
        // replaces the value the step stored (the fence keeps the compiler from moving that
        // store after this one; one lane's stores to an address complete in order)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        a_utt[static_cast<int64_t>(D) * p.u_pad + U] = a_top;
      }
    }
    if (owns_top) {
      double lnP2 = a_top + w_close;
      if (VAR == 2) lnP2 = log_add2(lnP2, acc_top);  // (t,U)->final
      p.lnp2_fwd[b] = lnP2;
      if (p.loss_f32) p.loss_f32[b] = static_cast<float>(-lnP2 / kLog2eD);
    }
  } else if (MODE != kLossOnly && sweep == 1) {
    // ---------------- backward sweep ----------------
    double bv[K];
#pragma unroll
    for (int k = 0; k < K; ++k) bv[k] = (ub + lane * K + k == U) ? w_close : kNoArc;
    const double b_top = w_close;  // beta(T-1, U)
    // W-Transducer: log-sum of beta(t, 0), t >= 1, kept per lane of wave 0 as in the
    // forward sweep (lane 0 of wave 0 owns unit 0)
    double acc_lane = kNoArc;
    if (VAR != 0 && U == 0 && T >= 2 && wv == 0 && lane == 0) acc_lane = w_close;  // beta(T-1, 0)
    double* const sum_out = (wv == 0 && lane == 0) ? &s_sum[0] : &s_sink[VAR != 0 ? lane : 0];
    if (owns_top) b_utt[static_cast<int64_t>(D) * p.u_pad + U] = w_close;
    double b00 = (D == 0) ? w_close : kNoArc;  // beta(0,0)
    double right_carry = kNoArc;  // lane 63 of the last wave keeps kNoArc (see left_carry)
    const int lag = NW - 1 - wv;  // the last wave goes first

    double rb[PF][K], rl[PF][K];
#pragma unroll
    for (int s = 0; s < PF; ++s) {
#pragma unroll
      for (int k = 0; k < K; ++k) load_w(D - 1 - s, k, rb[s][k], rl[s][k]);
      __builtin_amdgcn_sched_barrier(0);  // issue order = use order (oldest first)
    }
    double x_in[PF];  // lane 63: the fill of each step of a segment (several waves)
#pragma unroll
    for (int s = 0; s < PF; ++s) x_in[s] = kNoArc;

    for (int r = 0; r < n_rounds; ++r) {
      const int g = r - lag;
      if (g >= 0 && g < n_seg) {
        const int d0 = D - 1 - g * PF;
        // the wave after wrote them in the previous round (see the forward sweep)
        if (NW > 1 && wv < NW - 1) {
#pragma unroll
          for (int s = 0; s < PF; ++s) x_in[s] = s_xch[min(wv, NW > 1 ? NW - 2 : 0)][(r - 1) & 1][s];
        }
        double* const x_out = (lane == 0 && wv > 0) ? &s_xch[max(wv - 1, 0)][r & 1][0] : &s_sink[NW > 1 ? lane : 0];
#pragma unroll
        for (int s = 0; s < PF; ++s) {
          const int d = d0 - s;  // slot s holds the weights of diagonal d (d < 0: no node)
          if (NW > 1) x_out[s] = bv[0];  // lane 0's for wave wv-1
          // lane 63 of an earlier wave takes the unit above it from the wave after, one segment
          // old (in place, as in the forward sweep)
          double& fill = (NW > 1) ? x_in[s] : right_carry;
          fill = wave_shift_down(bv[0], fill);
          const double right = fill;
          // W-Transducer: node (d-U, U), t <= T-2, has a skip arc of weight 0 to (T-1, U)
          // (force-final) or to the final node (allow-ignore); it takes the place of the
          // label arc that unit U lacks, so no second log-add follows on the chain
          const bool skip_top = VAR != 0 && d >= U && d - U <= T - 2;  // wave-uniform
          double nb[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            double wb = rb[s][k], wl = rl[s][k];
            if (DENSE_IN) {
              const int u = ub + lane * K + k, t = d - u;
              wb = to_lattice(wb, t < T - 1 || u == U);
              wl = to_lattice(wl, u < U);
            }
            const double xb = wb + bv[k];
            double xl = wl + (k == K - 1 ? right : bv[k + 1 < K ? k + 1 : k]);
            if (VAR != 0) xl = (skip_top && ub + lane * K + k == U) ? (VAR == 1 ? b_top : 0.0) : xl;
            nb[k] = log_add2(xb, xl);
          }
          // wave-uniform, once per sweep: a branch, not selects.  The skip arcs out of (0,0)
          // are added after the sweep: no later step reads beta(0,0)
          if (__builtin_expect(d == 0, 0)) b00 = nb[0];
          if (VAR != 0) sum_out[s] = nb[0];
#pragma unroll
          for (int k = 0; k < K; ++k) bv[k] = nb[k];
          store_scores<K>(b_rsrc, lane_off, __builtin_amdgcn_readfirstlane((d >= 0 ? d : ND) * row_bytes), nb);
#pragma unroll
          for (int k = 0; k < K; ++k) load_w(d - PF, k, rb[s][k], rl[s][k]);
          __builtin_amdgcn_sched_barrier(0);  // the prefetch stays PF steps ahead of its use
        }
        if (VAR != 0 && wv == 0) {  // lane s: beta(d, 0) of step s, if 1 <= d <= T-1
          const int dl = d0 - lane;
          const double x = s_sum[min(lane, PF - 1)];
          acc_lane = log_add2(acc_lane, (lane < PF && dl >= 1 && dl <= T - 1) ? x : kNoArc);
        }
      }
      if (NW > 1) __syncthreads();  // the segment's values reach the previous wave
    }
    if (VAR != 0 && wv == 0) {
      const double acc0 = wave_log_sum(acc_lane);  // log-sum of beta(t, 0), t >= 1
      if (lane == 0) {
        b00 = log_add2(b00, acc0);  // (0,0)->(t,0)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");  // after the step's store of row 0
        b_utt[0] = b00;
      }
    }
    if (wv == 0 && lane == 0) p.lnp2_bwd[b] = b00;
  }
}

// ---------------------------------------------------------------------------
// kernel 2b: arc posteriors per padded row

struct PostParams {
  int32_t B, T_max, U_max;
  const int32_t* labels;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int32_t* status;
  const double2* lp2;  // kernel 1's lattice form (lse2f in the weights' low bits), or
  const double* lp_blank;  // dense natural-log weights
  const double* lp_label;
  const double* alpha;
  const double* beta;
  const double* lnp2_fwd;
  const double* lnp2_bwd;
  int64_t n_rows;
  int32_t u_pad;          // row width of alpha / beta
  RowInfo* rowinfo;       // row records for the gradient kernel, or
  double* alpha_out;      // dense float64 natural-log outputs (each may be null)
  double* beta_out;
  double* occ_blank_out;
  double* occ_label_out;
  double* loss_out;
  double* loss_bwd_out;
};

constexpr int kPostThreads = 1024;
constexpr int kPostTileT = 8;  // frames per block

// One block per (utterance, kPostTileT frames t0 .. t0+7, every unit).  Its
// threads walk the tile's cells diagonal by diagonal (consecutive threads:
// consecutive t, so consecutive cells of one diagonal), which makes the loads
// of alpha and beta contiguous; the tile's rows of lattice weights and of row
// records are one contiguous range of memory each, read and completed by the
// block.
template <bool DENSE>
__global__ __launch_bounds__(kPostThreads) void k2b_posteriors(PostParams p) {
  const int U1 = p.U_max + 1;
  const int n_tiles = (p.T_max + kPostTileT - 1) / kPostTileT;
  const int b = static_cast<int>(blockIdx.x / n_tiles);
  const int t0 = static_cast<int>(blockIdx.x - static_cast<int64_t>(b) * n_tiles) * kPostTileT;
  const int t_end = min(t0 + kPostTileT, p.T_max);
  const int T = p.logit_lens[b];
  const int U = p.label_lens[b];
  const bool good = p.status[b] == 0;
  const int64_t r_utt = static_cast<int64_t>(b) * p.T_max * U1;
  if (DENSE && t0 == 0 && threadIdx.x == 0) {
    const double ln2 = 1.0 / kLog2eD;
    if (p.loss_out) p.loss_out[b] = good ? -p.lnp2_fwd[b] * ln2 : __builtin_nan("");
    if (p.loss_bwd_out) p.loss_bwd_out[b] = good ? -p.lnp2_bwd[b] * ln2 : __builtin_nan("");
  }
  if (!good || t0 >= T) {  // the whole tile is zero rows
    if (!DENSE) {
      const int64_t r0 = r_utt + static_cast<int64_t>(t0) * U1;
      const int n = (t_end - t0) * U1;
      for (int i = threadIdx.x; i < n; i += kPostThreads) p.rowinfo[r0 + i] = RowInfo{0.f, 0.f, 0.f, kZeroRow};
    }
    return;
  }
  const double lnP2 = p.lnp2_fwd[b];
  const int64_t ab0 = static_cast<int64_t>(b) * (p.T_max + p.U_max + 1) * p.u_pad;
  const LatticeRecordSrc src{p.T_max, p.U_max, p.u_pad, p.labels, p.logit_lens, p.label_lens, p.status,
                             p.lp2,   p.alpha, p.beta,  p.lnp2_fwd};

  const int n_items = kPostTileT * (kPostTileT - 1 + U1);
  for (int i = threadIdx.x; i < n_items; i += kPostThreads) {
    const int t = t0 + i % kPostTileT;
    const int d = t0 + i / kPostTileT;  // diagonal
    const int u = d - t;
    if (t >= t_end || u < 0 || u > p.U_max) continue;
    const int64_t r = r_utt + static_cast<int64_t>(t) * U1 + u;
    if (t >= T || u > U) {
      if (!DENSE) p.rowinfo[r] = RowInfo{0.f, 0.f, 0.f, kZeroRow};
      continue;
    }
    if (!DENSE) {
      p.rowinfo[r] = lattice_row_record(src, b, t, u, r, T, U, lnP2);
      continue;
    }
    const double al = p.alpha[ab0 + static_cast<int64_t>(d) * p.u_pad + u];
    const double wb = to_lattice(p.lp_blank[r], true);
    const double wl = to_lattice(u < U ? p.lp_label[r] : 0.0, u < U);
    double xb = kNoArc, xl = kNoArc;
    if (t < T - 1) xb = al + wb + p.beta[ab0 + static_cast<int64_t>(d + 1) * p.u_pad + u] - lnP2;
    else if (u == U) xb = al + wb - lnP2;
    if (u < U) xl = al + wl + p.beta[ab0 + static_cast<int64_t>(d + 1) * p.u_pad + u + 1] - lnP2;
    const double ln2 = 1.0 / kLog2eD;
    if (p.alpha_out) p.alpha_out[r] = al * ln2;
    if (p.beta_out) p.beta_out[r] = p.beta[ab0 + static_cast<int64_t>(d) * p.u_pad + u] * ln2;
    if (p.occ_blank_out) p.occ_blank_out[r] = exp2(xb);
    if (p.occ_label_out) p.occ_label_out[r] = exp2(xl);
  }
}

}  // namespace rnnt
