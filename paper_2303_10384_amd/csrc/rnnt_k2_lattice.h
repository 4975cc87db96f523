// Kernel 2: forward / backward scores on the grid lattice of one utterance.
//
// Eq. 1's Fwd in the log semiring over the lattice of Fig. 1 (and Fig. 4 for
// the W-Transducer), plus the matching backward scores, then the posterior of
// every blank and label arc.
//
//   alpha(0,0) = 0
//   alpha(t,u) = ln[ e^{alpha(t-1,u) + lp_blank(t-1,u)} + e^{alpha(t,u-1) + lp_label(t,u-1)} ]
//   beta(T-1,U) = lp_blank(T-1,U)                         (closing blank)
//   beta(t,u)  = ln[ e^{lp_blank(t,u) + beta(t+1,u)} + e^{lp_label(t,u) + beta(t,u+1)} ]
//   ln P = alpha(T-1,U) + lp_blank(T-1,U) = beta(0,0)
// W-Transducer, force-final (Section 3.2, Fig. 4): weight-0 arcs (0,0)->(t,0)
// for t >= 1 and (t,U)->(T-1,U) for t <= T-2.  Allow-ignore (Section 4.3): the
// latter go to the final state instead.
//
// Schedule: every node on an anti-diagonal d = t + u depends only on diagonal
// d-1 (forward) or d+1 (backward), so one wavefront sweeps the diagonals with
// lane j owning the K consecutive units u = K*j .. K*j+K-1; the only exchange
// per step is one value with the neighbouring lane.  The forward wave and the
// backward wave of an utterance run concurrently in one block; the arc weights
// of the next PF diagonals are kept in flight in registers.  The wild-card arcs
// need two running log-sums (top row for the forward wave, bottom row for the
// backward wave) held by the owning lanes.  After both sweeps the whole block
// turns the scores into arc posteriors:
//   occ_blank(t,u) = exp(alpha(t,u) + lp_blank(t,u) + beta(t+1,u) - ln P)   (t < T-1)
//   occ_blank(T-1,U) = exp(alpha(T-1,U) + lp_blank(T-1,U) - ln P)
//   occ_label(t,u) = exp(alpha(t,u) + lp_label(t,u) + beta(t,u+1) - ln P)   (u < U)
// Scores are float64; the log-add correction term is float32 (see log_add).
#pragma once

#include "rnnt_device.h"

namespace rnnt {

enum LatticeMode : int {
  kLossOnly = 0,   // forward wave only, writes ln P / loss
  kRowRecords = 1, // both waves, then RowInfo for every row (gradient kernel input)
  kDenseOut = 2,   // both waves, then dense float64 scores / posteriors
};

struct LatticeParams {
  int32_t B, T_max, U_max, V, blank, variant;
  const int32_t* labels;  // (B, U_max) or null (lattice-only entry point)
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const double* lp_blank;  // element (b,t,u) at b*sb + t*st + u*su (in doubles)
  const double* lp_label;
  int64_t sb, st, su;
  double* alpha;  // workspace: (b, d, u) at b*sab + d*(U_max+1) + u, plus one scratch row
                  // per utterance after diagonal T_max+U_max-1 (sab >= (T_max+U_max+1)*(U_max+1))
  double* beta;
  int64_t sab;
  double* lnp_fwd;  // (B) workspace
  double* lnp_bwd;  // (B) workspace
  float* loss_f32;  // (B) or null
  RowInfo* rowinfo;  // kRowRecords
  double* alpha_out;  // kDenseOut outputs, dense (B, T_max, U_max+1), each may be null
  double* beta_out;
  double* occ_blank_out;
  double* occ_label_out;
  double* loss_out;      // (B) or null
  double* loss_bwd_out;  // (B) or null
};

// Arc weights of diagonal d for the lane's K cells.  The loads are issued
// unconditionally (cells outside the utterance read its node (0,0), which is
// always written) and nothing touches the registers here, so the loads stay in
// flight until the step that uses them; masking happens at that use.
template <int K, bool IL>
__device__ __forceinline__ void load_diag(const LatticeParams& p, int64_t lp0, int d, int lane, int T, int U,
                                          double (&rb)[K], double (&rl)[K]) {
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int u = lane * K + k;
    const int t = d - u;
    const bool v = (t >= 0) && (t < T) && (u <= U);
    const int64_t idx = v ? lp0 + static_cast<int64_t>(t) * p.st + static_cast<int64_t>(u) * p.su : lp0;
    if (IL) {
      const double2 w = *reinterpret_cast<const double2*>(p.lp_blank + idx);
      rb[k] = w.x;
      rl[k] = w.y;
    } else {
      rb[k] = p.lp_blank[idx];
      rl[k] = p.lp_label[idx];
    }
  }
}

// Neighbour exchange along the wavefront: lane i receives lane i-1's value
// (lane 0 receives `fill`), or lane i+1's (lane 63 receives `fill`), by DPP
// whole-wave shifts.
__device__ __forceinline__ double wave_shift_up(double x, double fill) {
  const int lo = __builtin_amdgcn_update_dpp(static_cast<int>(__double2loint(fill)),
                                             static_cast<int>(__double2loint(x)), 0x138, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(static_cast<int>(__double2hiint(fill)),
                                             static_cast<int>(__double2hiint(x)), 0x138, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double wave_shift_down(double x, double fill) {
  const int lo = __builtin_amdgcn_update_dpp(static_cast<int>(__double2loint(fill)),
                                             static_cast<int>(__double2loint(x)), 0x130, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(static_cast<int>(__double2hiint(fill)),
                                             static_cast<int>(__double2hiint(x)), 0x130, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}

// IL: arc weights interleaved (lp_label == lp_blank + 1), read as one 16-byte load.
template <int K, int PF, int MODE, bool IL>
__global__ __launch_bounds__(MODE == kLossOnly ? 64 : 512) void k2_lattice(LatticeParams p) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int T = p.logit_lens[b];
  const int U = p.label_lens[b];
  const int U1 = p.U_max + 1;
  const double kNaN = __builtin_nan("");

  bool ok = (T >= 1 && T <= p.T_max && U >= 0 && U <= p.U_max);
  int bad = 0;
  if (ok && p.labels != nullptr) {
    for (int u = tid; u < U; u += blockDim.x) {
      const int y = p.labels[static_cast<int64_t>(b) * p.U_max + u];
      if (y < 0 || y >= p.V || y == p.blank) bad = 1;
    }
  }
  bad = __syncthreads_or(bad);
  if (!ok || bad) {
    if (tid == 0) {
      p.lnp_fwd[b] = kNaN;
      p.lnp_bwd[b] = kNaN;
      if (p.loss_f32) p.loss_f32[b] = __builtin_nanf("");
      if (p.loss_out) p.loss_out[b] = kNaN;
      if (p.loss_bwd_out) p.loss_bwd_out[b] = kNaN;
    }
    if (MODE == kRowRecords) {
      const int rows = p.T_max * U1;
      RowInfo* ri = p.rowinfo + static_cast<int64_t>(b) * rows;
      for (int r = tid; r < rows; r += blockDim.x) ri[r] = RowInfo{0.f, 0.f, 0.f, kZeroRow};
    }
    return;
  }

  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int D = T - 1 + U;  // last diagonal
  const int64_t lp0 = static_cast<int64_t>(b) * p.sb;
  const int64_t ab0 = static_cast<int64_t>(b) * p.sab;
  const int variant = p.variant;
  const int owner_top = U / K;  // lane owning u = U
  const int64_t dump = static_cast<int64_t>(p.T_max + p.U_max) * U1;  // scratch row after the last diagonal

  if (wave == 0) {
    // ---------------- forward sweep ----------------
    double a[K];
#pragma unroll
    for (int k = 0; k < K; ++k) a[k] = (lane * K + k == 0) ? 0.0 : neg_inf();
    double acc_top = neg_inf();  // log-sum of alpha(t, U), t <= T-2 (owner lane)
    double a_top = (U == 0) ? 0.0 : neg_inf();  // latest alpha(t, U) (owner lane)
    if (MODE != kLossOnly && lane == 0) p.alpha[ab0] = 0.0;
    if (variant != 0 && U == 0 && T >= 2 && lane == 0) acc_top = 0.0;

    double rb[PF][K], rl[PF][K];
#pragma unroll
    for (int s = 0; s < PF; ++s) load_diag<K, IL>(p, lp0, s, lane, T, U, rb[s], rl[s]);

    // Whole blocks of PF steps with no branch around the loads or stores (a
    // branch would make the wait counters unknown at the join and serialise
    // the prefetch); the up to PF-1 steps past D only see invalid nodes.
    for (int d0 = 1; d0 <= D; d0 += PF) {
#pragma unroll
      for (int s = 0; s < PF; ++s) {
        const int d = d0 + s;  // slot s holds the weights of diagonal d-1
        {
          double eb[K], el[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            eb[k] = a[k] + rb[s][k];
            el[k] = (lane * K + k < U) ? a[k] + rl[s][k] : neg_inf();
          }
          const double left = wave_shift_up(el[K - 1], neg_inf());
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int u = lane * K + k;
            const int t = d - u;
            const bool v = (t >= 0) && (t < T) && (u <= U);
            double n = log_add(eb[k], k == 0 ? left : el[k > 0 ? k - 1 : 0]);
            // wild-card arcs into this node: (0,0)->(t,0) and (t',U)->(T-1,U)
            // (with U = 0 both reach (T-1, 0) and both count)
            double extra = (variant != 0 && u == 0 && t >= 1) ? 0.0 : neg_inf();
            if (variant == 1 && u == U && t == T - 1) extra = log_add(extra, acc_top);
            if (extra != neg_inf()) n = log_add(n, extra);
            n = v ? n : neg_inf();
            a[k] = n;
            // every lane stores (invalid nodes store -inf in place, lanes past
            // U_max into the dump row) so no store sits under a branch
            if (MODE != kLossOnly)
              p.alpha[ab0 + (u <= p.U_max && d <= D ? static_cast<int64_t>(d) * U1 + u : dump)] = n;
            if (u == U && v) a_top = n;
            if (variant != 0 && u == U && v && t <= T - 2) acc_top = log_add(acc_top, n);
          }
          load_diag<K, IL>(p, lp0, d - 1 + PF, lane, T, U, rb[s], rl[s]);
        }
      }
    }
    if (lane == owner_top) {
      const double aU = a_top;  // alpha(T-1, U)
      const int64_t idx = lp0 + static_cast<int64_t>(T - 1) * p.st + static_cast<int64_t>(U) * p.su;
      double lnP = aU + p.lp_blank[idx];
      if (variant == 2) lnP = log_add(lnP, acc_top);  // (t',U)->final
      p.lnp_fwd[b] = lnP;
      if (p.loss_f32) p.loss_f32[b] = static_cast<float>(-lnP);
    }
  } else if (MODE != kLossOnly && wave == 1) {
    // ---------------- backward sweep ----------------
    double bv[K];
#pragma unroll
    for (int k = 0; k < K; ++k) bv[k] = neg_inf();
    double b_top = neg_inf();  // beta(T-1, U) (owner lane)
    double acc0 = neg_inf();   // log-sum of beta(t, 0), t >= 1 (lane 0)
    if (lane == owner_top) {
      const int64_t idx = lp0 + static_cast<int64_t>(T - 1) * p.st + static_cast<int64_t>(U) * p.su;
      const double x = p.lp_blank[idx];
#pragma unroll
      for (int k = 0; k < K; ++k)
        if (lane * K + k == U) bv[k] = x;
      b_top = x;
      p.beta[ab0 + static_cast<int64_t>(D) * U1 + U] = x;
      if (variant != 0 && U == 0 && T >= 2) acc0 = x;
    }

    double rb[PF][K], rl[PF][K];
#pragma unroll
    for (int s = 0; s < PF; ++s) load_diag<K, IL>(p, lp0, D - 1 - s, lane, T, U, rb[s], rl[s]);

    double b00 = bv[0];  // beta(0,0) (lane 0); already final when D == 0
    for (int d0 = D - 1; d0 >= 0; d0 -= PF) {
#pragma unroll
      for (int s = 0; s < PF; ++s) {
        const int d = d0 - s;  // slot s holds the weights of diagonal d (d < 0: no node)
        {
          const double right = wave_shift_down(bv[0], neg_inf());
          double nb[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int u = lane * K + k;
            const int t = d - u;
            const bool v = (t >= 0) && (t < T) && (u <= U);
            const double xb = rb[s][k] + bv[k];
            const double xl = (u < U) ? rl[s][k] + (k == K - 1 ? right : bv[k + 1 < K ? k + 1 : k]) : neg_inf();
            double n = log_add(xb, xl);
            // wild-card arcs out of this node: (t,U)->(T-1,U) or (t,U)->final, and (0,0)->(t',0)
            const double extra = (u == U && t < T - 1 && variant == 1) ? b_top
                                 : (u == U && t < T - 1 && variant == 2) ? 0.0 : neg_inf();
            if (extra != neg_inf()) n = log_add(n, extra);
            if (variant != 0 && u == 0 && t == 0) n = log_add(n, acc0);
            n = v ? n : neg_inf();
            nb[k] = n;
            p.beta[ab0 + (u <= p.U_max && d >= 0 ? static_cast<int64_t>(d) * U1 + u : dump)] = n;
            if (variant != 0 && u == 0 && v && t >= 1) acc0 = log_add(acc0, n);
            if (u == 0 && d == 0) b00 = n;
          }
#pragma unroll
          for (int k = 0; k < K; ++k) bv[k] = nb[k];
          load_diag<K, IL>(p, lp0, d - PF, lane, T, U, rb[s], rl[s]);
        }
      }
    }
    if (lane == 0) p.lnp_bwd[b] = b00;
  }

  if (MODE == kLossOnly) return;
  __syncthreads();

  // ---------------- arc posteriors ----------------
  // RB rows per thread are loaded before any is used (independent loads in
  // flight); cells outside the utterance read node (0,0) and are discarded.
  constexpr int RB = 4;
  const double lnP = p.lnp_fwd[b];
  const int rows = p.T_max * U1;
  const int64_t row0 = static_cast<int64_t>(b) * rows;
  const double* __restrict__ alpha = p.alpha;
  const double* __restrict__ beta = p.beta;
  const int32_t* __restrict__ lab_b = p.labels ? p.labels + static_cast<int64_t>(b) * p.U_max : nullptr;
  if (MODE == kDenseOut && tid == 0) {
    if (p.loss_out) p.loss_out[b] = -lnP;
    if (p.loss_bwd_out) p.loss_bwd_out[b] = -p.lnp_bwd[b];
  }
  for (int rb0 = tid; rb0 < rows; rb0 += blockDim.x * RB) {
    double al[RB], be_b[RB], be_l[RB], lpb[RB], lpl[RB];
    float l2[RB];
    int lab[RB];
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int r = rb0 + i * blockDim.x;
      const int t = r / U1;
      const int u = r - t * U1;
      const bool valid = (r < rows) && (t < T) && (u <= U);
      const int d = t + u;
      const int64_t ai = valid ? ab0 + static_cast<int64_t>(d) * U1 + u : ab0;
      const int64_t bi_b = (valid && t < T - 1) ? ab0 + static_cast<int64_t>(d + 1) * U1 + u : ab0;
      const int64_t bi_l = (valid && u < U) ? ab0 + static_cast<int64_t>(d + 1) * U1 + u + 1 : ab0;
      const int64_t li = valid ? lp0 + static_cast<int64_t>(t) * p.st + static_cast<int64_t>(u) * p.su : lp0;
      al[i] = alpha[ai];
      be_b[i] = beta[bi_b];
      be_l[i] = beta[bi_l];
      if (IL) {
        const double2 w = *reinterpret_cast<const double2*>(p.lp_blank + li);
        lpb[i] = w.x;
        lpl[i] = w.y;
      } else {
        lpb[i] = p.lp_blank[li];
        lpl[i] = p.lp_label[li];
      }
      l2[i] = (MODE == kRowRecords) ? p.rowinfo[valid ? row0 + r : row0].lse2 : 0.f;
      lab[i] = (lab_b != nullptr && U > 0) ? lab_b[u < U ? u : U - 1] : kNoLabel;
    }
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int r = rb0 + i * blockDim.x;
      if (r >= rows) break;
      const int t = r / U1;
      const int u = r - t * U1;
      const bool valid = (t < T) && (u <= U);
      if (MODE == kRowRecords && !valid) {
        p.rowinfo[row0 + r] = RowInfo{0.f, 0.f, 0.f, kZeroRow};
        continue;
      }
      if (!valid) continue;
      double xb = neg_inf(), xl = neg_inf();
      if (t < T - 1) xb = al[i] + lpb[i] + be_b[i] - lnP;
      else if (u == U) xb = al[i] + lpb[i] - lnP;
      if (u < U) xl = al[i] + lpl[i] + be_l[i] - lnP;
      if (MODE == kRowRecords) {
        RowInfo o;
        o.lse2 = l2[i];
        o.occ_blank = fast_exp2(static_cast<float>(xb * kLog2eD));
        o.occ_label = fast_exp2(static_cast<float>(xl * kLog2eD));
        o.label = (u < U) ? lab[i] : kNoLabel;
        p.rowinfo[row0 + r] = o;
      } else {
        const int64_t o = row0 + r;
        if (p.alpha_out) p.alpha_out[o] = al[i];
        if (p.beta_out) p.beta_out[o] = beta[ab0 + static_cast<int64_t>(t + u) * U1 + u];
        if (p.occ_blank_out) p.occ_blank_out[o] = exp(xb);
        if (p.occ_label_out) p.occ_label_out[o] = exp(xl);
      }
    }
  }
}

}  // namespace rnnt
