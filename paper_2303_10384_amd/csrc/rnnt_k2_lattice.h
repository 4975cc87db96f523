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
  double* alpha;  // workspace: (b, d, u) at b*sab + d*(U_max+1) + u
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

template <int K, bool IL>
__device__ __forceinline__ void load_diag(const LatticeParams& p, int64_t lp0, int d, int lane, int T, int U,
                                          double (&rb)[K], double (&rl)[K]) {
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int u = lane * K + k;
    const int t = d - u;
    double xb = neg_inf(), xl = neg_inf();
    if (t >= 0 && t < T && u <= U) {
      const int64_t idx = lp0 + static_cast<int64_t>(t) * p.st + static_cast<int64_t>(u) * p.su;
      if (IL) {
        const double2 w = *reinterpret_cast<const double2*>(p.lp_blank + idx);
        xb = w.x;
        xl = w.y;
      } else {
        xb = p.lp_blank[idx];
        if (u < U) xl = p.lp_label[idx];
      }
      if (u == U) xl = neg_inf();
    }
    rb[k] = xb;
    rl[k] = xl;
  }
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

    for (int d0 = 1; d0 <= D; d0 += PF) {
#pragma unroll
      for (int s = 0; s < PF; ++s) {
        const int d = d0 + s;  // slot s holds the weights of diagonal d-1
        if (d <= D) {
          double eb[K], el[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            eb[k] = a[k] + rb[s][k];
            el[k] = a[k] + rl[s][k];
          }
          double left = __shfl_up(el[K - 1], 1);
          if (lane == 0) left = neg_inf();
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int u = lane * K + k;
            const int t = d - u;
            const bool v = (t >= 0) && (t < T) && (u <= U);
            double n = log_add(eb[k], k == 0 ? left : el[k > 0 ? k - 1 : 0]);
            if (variant != 0 && u == 0 && t >= 1) n = log_add(n, 0.0);            // (0,0)->(t,0)
            if (variant == 1 && u == U && t == T - 1) n = log_add(n, acc_top);      // (t',U)->(T-1,U)
            n = v ? n : neg_inf();
            a[k] = n;
            if (MODE != kLossOnly && v) p.alpha[ab0 + static_cast<int64_t>(d) * U1 + u] = n;
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

    for (int d0 = D - 1; d0 >= 0; d0 -= PF) {
#pragma unroll
      for (int s = 0; s < PF; ++s) {
        const int d = d0 - s;  // slot s holds the weights of diagonal d
        if (d >= 0) {
          double right = __shfl_down(bv[0], 1);
          if (lane == kWave - 1) right = neg_inf();
          double nb[K];
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int u = lane * K + k;
            const int t = d - u;
            const bool v = (t >= 0) && (t < T) && (u <= U);
            const double xb = rb[s][k] + bv[k];
            const double xl = rl[s][k] + (k == K - 1 ? right : bv[k + 1 < K ? k + 1 : k]);
            double n = log_add(xb, xl);
            if (u == U && t < T - 1) {
              if (variant == 1) n = log_add(n, b_top);  // (t,U)->(T-1,U)
              if (variant == 2) n = log_add(n, 0.0);    // (t,U)->final
            }
            if (variant != 0 && u == 0 && t == 0) n = log_add(n, acc0);  // (0,0)->(t',0)
            n = v ? n : neg_inf();
            nb[k] = n;
            if (v) p.beta[ab0 + static_cast<int64_t>(d) * U1 + u] = n;
            if (variant != 0 && u == 0 && v && t >= 1) acc0 = log_add(acc0, n);
          }
#pragma unroll
          for (int k = 0; k < K; ++k) bv[k] = nb[k];
          load_diag<K, IL>(p, lp0, d - PF, lane, T, U, rb[s], rl[s]);
        }
      }
    }
    if (lane == 0) p.lnp_bwd[b] = bv[0];
  }

  if (MODE == kLossOnly) return;
  __syncthreads();

  // ---------------- arc posteriors ----------------
  const double lnP = p.lnp_fwd[b];
  const int rows = p.T_max * U1;
  const int64_t row0 = static_cast<int64_t>(b) * rows;
  if (MODE == kDenseOut && tid == 0) {
    if (p.loss_out) p.loss_out[b] = -lnP;
    if (p.loss_bwd_out) p.loss_bwd_out[b] = -p.lnp_bwd[b];
  }
  for (int r = tid; r < rows; r += blockDim.x) {
    const int t = r / U1;
    const int u = r - t * U1;
    const bool valid = (t < T) && (u <= U);
    if (MODE == kRowRecords && !valid) {
      p.rowinfo[row0 + r] = RowInfo{0.f, 0.f, 0.f, kZeroRow};
      continue;
    }
    if (!valid) continue;
    const int d = t + u;
    const double al = p.alpha[ab0 + static_cast<int64_t>(d) * U1 + u];
    const int64_t li = lp0 + static_cast<int64_t>(t) * p.st + static_cast<int64_t>(u) * p.su;
    double lpb, lpl;
    if (IL) {
      const double2 w = *reinterpret_cast<const double2*>(p.lp_blank + li);
      lpb = w.x;
      lpl = w.y;
    } else {
      lpb = p.lp_blank[li];
      lpl = (u < U) ? p.lp_label[li] : neg_inf();
    }
    double xb = neg_inf(), xl = neg_inf();
    if (t < T - 1) xb = al + lpb + p.beta[ab0 + static_cast<int64_t>(d + 1) * U1 + u] - lnP;
    else if (u == U) xb = al + lpb - lnP;
    if (u < U) xl = al + lpl + p.beta[ab0 + static_cast<int64_t>(d + 1) * U1 + u + 1] - lnP;
    if (MODE == kRowRecords) {
      RowInfo o;
      o.lse2 = p.rowinfo[row0 + r].lse2;
      o.occ_blank = fast_exp2(static_cast<float>(xb * kLog2eD));
      o.occ_label = fast_exp2(static_cast<float>(xl * kLog2eD));
      o.label = (u < U) ? p.labels[static_cast<int64_t>(b) * p.U_max + u] : kNoLabel;
      p.rowinfo[row0 + r] = o;
    } else {
      const int64_t o = row0 + r;
      if (p.alpha_out) p.alpha_out[o] = al;
      if (p.beta_out) p.beta_out[o] = p.beta[ab0 + static_cast<int64_t>(d) * U1 + u];
      if (p.occ_blank_out) p.occ_blank_out[o] = exp(xb);
      if (p.occ_label_out) p.occ_label_out[o] = exp(xl);
    }
  }
}

}  // namespace rnnt
