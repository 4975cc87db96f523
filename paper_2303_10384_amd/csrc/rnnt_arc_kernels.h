// Kernels of the loss over lattices given as arc lists (Section 2.2: a lattice
// graph whose arcs are filled in from X = log_softmax(logits) by indexed
// selection; the loss of Eq. 1 is its negative forward score, the gradient comes
// from its forward and backward scores).  The plan they read is laid out in
// rnnt_arc_layout.h; the row normaliser (kernel 1, rows mode) and the gradient
// kernel (kernel 3) are shared with the grid path.
//
//   populate   one thread per arc: the weight score + z[label] - lse in log2
//              units, stored in the arc orders of both sweeps; NaN for an arc
//              that reads a row outside its utterance's valid rows.
//   sweep      one wavefront per (utterance, direction): the levels in order;
//              per level, one lane per entering arc adds the arc's weight to its
//              source's score (read from LDS), then one lane per state sums its
//              run of those terms in the log semiring.  The next level's arc and
//              state records are loaded while the current one is computed.
//   rows       one thread per logits row: the arc posteriors of the row's label
//              arcs, summed into the row record of kernel 3 (blank occupancy,
//              occupancy of the row's one non-blank label).
//   extra rows one block per row whose arcs carry two or more distinct
//              non-blank labels: the whole gradient row, written after kernel 3.
#pragma once

#include "rnnt_arc_layout.h"
#include "rnnt_device.h"

namespace rnnt {

__device__ __forceinline__ int clamp_index(int i, int n) {  // keeps an index from the plan inside [0, n)
  return static_cast<int>(min(static_cast<unsigned>(i), static_cast<unsigned>(n > 0 ? n - 1 : 0)));
}

// Logits row r = (b * T_max + t) * (U_max+1) + u, split into (b, t, u).
struct RowPos {
  int b, t, u;
};
__device__ __forceinline__ RowPos row_pos(int r, int T_max, int U_max) {
  const int U1 = U_max + 1;
  const int rpu = T_max * U1;
  RowPos q;
  q.b = r / rpu;
  const int rem = r - q.b * rpu;
  q.t = rem / U1;
  q.u = rem - q.t * U1;
  return q;
}

__device__ __forceinline__ bool lengths_ok(int Tb, int Ub, int T_max, int U_max) {
  return Tb >= 1 && Tb <= T_max && Ub >= 0 && Ub <= U_max;
}

// ---------------------------------------------------------------- populate

struct ArcPopulateParams {
  const void* logits;
  int32_t B, T_max, U_max, V;
  int32_t n_arcs, n_rows;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int4* arcs;        // graph-0 order
  const float* score;
  const int32_t* perm;     // graph-0 position -> graph-1 position
  const double* lse2_rows; // lse * log2(e) per valid row
  double* w0;              // weights, graph-0 order (log2 units)
  double* w1;              // weights, graph-1 order
};

template <typename T>
__global__ __launch_bounds__(256) void k_arc_populate(ArcPopulateParams p) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= p.n_arcs) return;
  const int4 a = p.arcs[i];
  double w = static_cast<double>(p.score[i]) * kLog2eD;
  if (a.w >= 0) {
    const RowPos q = row_pos(a.z, p.T_max, p.U_max);
    const int Tb = p.logit_lens[clamp_index(q.b, p.B)];
    const int Ub = p.label_lens[clamp_index(q.b, p.B)];
    const bool ok = a.z >= 0 && a.z < p.n_rows && lengths_ok(Tb, Ub, p.T_max, p.U_max) && q.t < Tb && q.u <= Ub &&
                    a.w < p.V;
    if (ok) {
      const float z = ElemTraits<T>::load1(static_cast<const T*>(p.logits) + static_cast<int64_t>(a.z) * p.V + a.w);
      w += static_cast<double>(z) * kLog2eD - p.lse2_rows[a.z];
    } else {
      w = __builtin_nan("");
    }
  }
  p.w0[i] = w;
  p.w1[clamp_index(p.perm[i], p.n_arcs)] = w;
}

// ---------------------------------------------------------------- sweep

struct ArcSweepParams {
  int32_t B, T_max, U_max;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int4* utt;
  const int4* ends;
  const int4* level[2];
  const int32_t* seg[2];
  const int32_t* pin[2];
  const int32_t* loc[2];
  const double* w[2];
  double* val[2];   // scores per state, graph g's numbering (log2 units)
  double* lnp2;     // (2, B): log2 P from the forward sweep, then from the backward one
  int32_t* status;  // (B): 0 scores valid, 1 bad data, 2 no path reaches the final state
  float* loss;      // (B) or null
};

// Records of one level held in registers: the first NC chunks of 64 entering
// arcs and the first NS chunks of 64 states.
template <int NC, int NS>
struct SweepRegs {
  int4 info;  // {first state, states, first arc, arcs | max in-degree << 16}
  int32_t loc[NC];
  double w[NC];
  int32_t seg[NS];
  int32_t pin[NS];
};

__device__ __forceinline__ double buffer_load_f64(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));  // two dwords
}
__device__ __forceinline__ int buffer_load_i32(__amdgpu_buffer_rsrc_t r, int off) {
  return static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

__device__ __forceinline__ double lane_value(double x, int lane) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(x), lane);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(x), lane);
  return __hiloint2double(hi, lo);
}

template <int NC, int NS>
__global__ __launch_bounds__(64) void k_arc_sweep(ArcSweepParams p) {
  __shared__ double s_val[kArcDummy + 1];    // ring of recent scores, pinned scores, a dummy slot
  __shared__ double s_x[kArcLevelArcs];      // source score + arc weight, one per entering arc of the level
  __shared__ int4 s_lvl[kArcLevelWindow];    // level records
  const int b = blockIdx.x >> 1;
  const int g = blockIdx.x & 1;
  const int lane = threadIdx.x;
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  double* lnp_out = p.lnp2 + g * p.B + b;
  if (!lengths_ok(Tb, Ub, p.T_max, p.U_max)) {
    if (lane == 0) {
      *lnp_out = __builtin_nan("");
      if (g == 0) {
        p.status[b] = 1;
        if (p.loss) p.loss[b] = __builtin_nanf("");
      }
    }
    return;
  }
  const int4 ut = p.utt[b];
  const int4 en = p.ends[b];
  const int s_begin = ut.x, n_states = ut.y - ut.x, l_begin = ut.z, l_end = ut.w;
  const int a_begin = en.z, n_arcs = en.w - en.z;
  const int start = g ? en.y : s_begin;   // the sweep's start state (score 0)
  const int fin = g ? ut.y - 1 : en.x;    // the state whose score is ln P
  // every record of the plan is read through a buffer bounded to this utterance
  const __amdgpu_buffer_rsrc_t rs_loc = make_buffer(p.loc[g] + a_begin, static_cast<int64_t>(n_arcs) * 4);
  const __amdgpu_buffer_rsrc_t rs_w = make_buffer(p.w[g] + a_begin, static_cast<int64_t>(n_arcs) * 8);
  const __amdgpu_buffer_rsrc_t rs_seg = make_buffer(p.seg[g] + s_begin, static_cast<int64_t>(n_states) * 4);
  const __amdgpu_buffer_rsrc_t rs_pin = make_buffer(p.pin[g] + s_begin, static_cast<int64_t>(n_states) * 4);
  const __amdgpu_buffer_rsrc_t rs_val = make_buffer(p.val[g] + s_begin, static_cast<int64_t>(n_states) * 8);
  const __amdgpu_buffer_rsrc_t rs_lvl = make_buffer(p.level[g] + l_begin, static_cast<int64_t>(l_end - l_begin) * 16);

  int win = l_begin;  // first level staged in s_lvl
  auto load_window = [&](int base) {
    for (int i = lane; i < kArcLevelWindow; i += kWave) {
      const u32x4 r = buffer_load16<false>(rs_lvl, (base - l_begin + i) * 16);
      s_lvl[i] = make_int4(static_cast<int>(r.x), static_cast<int>(r.y), static_cast<int>(r.z),
                           static_cast<int>(r.w));
    }
  };
  load_window(win);

  // every load is issued unconditionally; a lane without a record reads past the buffer (zero)
  auto issue = [&](int k, SweepRegs<NC, NS>& R) {
    const int4 info = s_lvl[min(max(k - win, 0), kArcLevelWindow - 1)];
    R.info = (k < l_end) ? info : make_int4(0, 0, 0, 0);
    const int ns = R.info.y;
    const int na = R.info.w & 0xffff;
    const int arel = R.info.z - a_begin;
    const int srel = R.info.x - s_begin;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int i = c * kWave + lane;
      R.loc[c] = buffer_load_i32(rs_loc, i < na ? (arel + i) * 4 : kOutOfRange);
      R.w[c] = buffer_load_f64(rs_w, i < na ? (arel + i) * 8 : kOutOfRange);
    }
#pragma unroll
    for (int c = 0; c < NS; ++c) {
      const int j = c * kWave + lane;
      R.seg[c] = buffer_load_i32(rs_seg, j < ns ? (srel + j) * 4 : kOutOfRange);
      R.pin[c] = buffer_load_i32(rs_pin, j < ns ? (srel + j) * 4 : kOutOfRange);
    }
  };

  double lnp = kNoArc;
  bool have = false;  // this lane computed the score of `fin`
  bool bad = false;   // an arc weight is NaN (a row outside the valid region, NaN logits)

  auto arc_term = [&](int i, int na, int loc, double w) {
    const double src = s_val[min(static_cast<unsigned>(loc), static_cast<unsigned>(kArcDummy))];
    s_x[i & (kArcLevelArcs - 1)] = src + w;
    bad = bad || (i < na && __builtin_isnan(w));
  };
  auto state_sum = [&](int s_lo, int ns, int maxdeg, int j, int seg, int pin) {
    const bool ok = j < ns;
    const int s = s_lo + j;
    const int rel = seg & 0xffff;
    const int cnt = static_cast<int>(static_cast<unsigned>(seg) >> 16);
    double v = kNoArc;
    for (int q = 0; q < maxdeg; ++q) {
      const double x = s_x[(rel + q) & (kArcLevelArcs - 1)];
      v = log_add2(v, q < cnt ? x : kNoArc);
    }
    v = (s == start) ? 0.0 : v;
    s_val[ok ? ((s - s_begin) & (kArcRing - 1)) : kArcDummy] = v;
    s_val[ok ? min(static_cast<unsigned>(pin), static_cast<unsigned>(kArcDummy)) : kArcDummy] = v;
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), rs_val,
                                          ok ? (s - s_begin) * 8 : kOutOfRange, 0, 0);
    const bool f = ok && s == fin;
    lnp = f ? v : lnp;
    have = have || f;
  };
  auto process = [&](const SweepRegs<NC, NS>& R) {
    const int s_lo = R.info.x, ns = R.info.y;
    const int na = R.info.w & 0xffff;
    const int maxdeg = static_cast<int>(static_cast<unsigned>(R.info.w) >> 16);
#pragma unroll
    for (int c = 0; c < NC; ++c) arc_term(c * kWave + lane, na, R.loc[c], R.w[c]);
    if (na > NC * kWave) {  // a level with more arcs than the registers hold
      const int arel = R.info.z - a_begin;
      for (int c = NC; c * kWave < na; ++c) {
        const int i = c * kWave + lane;
        const int loc = buffer_load_i32(rs_loc, i < na ? (arel + i) * 4 : kOutOfRange);
        const double w = buffer_load_f64(rs_w, i < na ? (arel + i) * 8 : kOutOfRange);
        arc_term(i, na, loc, w);
      }
    }
#pragma unroll
    for (int c = 0; c < NS; ++c) state_sum(s_lo, ns, maxdeg, c * kWave + lane, R.seg[c], R.pin[c]);
    if (ns > NS * kWave) {  // a level with more states than the registers hold
      const int srel = s_lo - s_begin;
      for (int c = NS; c * kWave < ns; ++c) {
        const int j = c * kWave + lane;
        const int seg = buffer_load_i32(rs_seg, j < ns ? (srel + j) * 4 : kOutOfRange);
        const int pin = buffer_load_i32(rs_pin, j < ns ? (srel + j) * 4 : kOutOfRange);
        state_sum(s_lo, ns, maxdeg, j, seg, pin);
      }
    }
  };

  // two register sets in turn: level k+1's records load while level k is summed
  SweepRegs<NC, NS> RA, RB;
  issue(l_begin, RA);
  for (int k = l_begin; k < l_end; k += 2) {
    if (k + 2 >= win + kArcLevelWindow) {
      win = k;
      load_window(win);
    }
    issue(k + 1, RB);
    __builtin_amdgcn_sched_barrier(0);
    process(RA);
    issue(k + 2, RA);
    __builtin_amdgcn_sched_barrier(0);
    process(RB);
  }

  const uint64_t holder = __ballot(have);
  lnp = lane_value(lnp, holder ? __builtin_ctzll(holder) : 0);
  const bool any_bad = __ballot(bad) != 0;
  if (lane == 0) {
    *lnp_out = lnp;
    if (g == 0) {
      const int st = (any_bad || __builtin_isnan(lnp)) ? 1 : (lnp > 0.5 * kNoArc ? 0 : 2);
      p.status[b] = st;
      if (p.loss)
        p.loss[b] = st == 1 ? __builtin_nanf("")
                            : (st == 2 ? __builtin_inff() : static_cast<float>(-lnp / kLog2eD));
    }
  }
}

// ---------------------------------------------------------------- row records

struct ArcRowParams {
  int32_t T_max, U_max, blank;
  int32_t n_rows, n_arcs, n_row_arcs, n_states;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int4* utt;
  const int4* arcs;
  const int32_t* row_seg;
  const int32_t* row_arc;
  const double* w0;
  const double* val0;
  const double* val1;
  const double* lnp2;
  const int32_t* status;
  const double* lse2_rows;
  RowInfo* rowinfo;
};

// Posterior of graph-0 arc i of utterance b (mirror = s_begin + s_end - 1).
__device__ __forceinline__ float arc_occupancy(const ArcRowParams& p, int i, int mirror, double lnp, int& label) {
  const int4 a = p.arcs[i];
  label = a.w;
  const double e = p.val0[clamp_index(a.x, p.n_states)] + p.w0[i] + p.val1[clamp_index(mirror - a.y, p.n_states)] -
                   lnp;
  return fast_exp2(static_cast<float>(e));
}

__global__ __launch_bounds__(256) void k_arc_rows(ArcRowParams p) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= p.n_rows) return;
  const RowPos q = row_pos(r, p.T_max, p.U_max);
  RowInfo ri;
  ri.lse2 = 0.f;
  ri.occ_blank = 0.f;
  ri.occ_label = 0.f;
  ri.label = kZeroRow;
  if (p.status[q.b] == 0 && q.t < p.logit_lens[q.b] && q.u <= p.label_lens[q.b]) {
    const double lnp = p.lnp2[q.b];
    const int4 ut = p.utt[q.b];
    const int mirror = ut.x + ut.y - 1;
    const int j0 = p.row_seg[r], j1 = p.row_seg[r + 1];
    float ob = 0.f, ol = 0.f;
    int primary = kNoLabel;
    bool extra = false;
    for (int j = j0; j < j1; ++j) {
      int label;
      const float occ = arc_occupancy(p, clamp_index(p.row_arc[clamp_index(j, p.n_row_arcs)], p.n_arcs), mirror,
                                      lnp, label);
      if (label == p.blank) {
        ob += occ;
      } else if (primary == kNoLabel || primary == label) {
        primary = label;
        ol += occ;
      } else {
        extra = true;  // a second non-blank label: the extra-rows kernel writes this row
      }
    }
    if (!extra) {
      ri.lse2 = static_cast<float>(p.lse2_rows[r]);
      ri.occ_blank = ob;
      ri.occ_label = ol;
      ri.label = primary;
    }
  }
  p.rowinfo[r] = ri;
}

// ---------------------------------------------------------------- extra rows

struct ArcExtraParams {
  ArcRowParams rows;
  const void* logits;
  void* grad;
  const int32_t* xrows;
  int32_t V;
};

template <typename Tin, typename Tout>
__global__ __launch_bounds__(256) void k_arc_extra_rows(ArcExtraParams p) {
  __shared__ int s_label[kArcRowArcsMax];
  __shared__ float s_occ[kArcRowArcsMax];
  __shared__ float s_tot;
  const ArcRowParams& rp = p.rows;
  const int r = clamp_index(p.xrows[blockIdx.x], rp.n_rows);
  const RowPos q = row_pos(r, rp.T_max, rp.U_max);
  if (!(rp.status[q.b] == 0 && q.t < rp.logit_lens[q.b] && q.u <= rp.label_lens[q.b])) return;  // stays zero
  const double lnp = rp.lnp2[q.b];
  const int4 ut = rp.utt[q.b];
  const int mirror = ut.x + ut.y - 1;
  const int j0 = rp.row_seg[r];
  const int n = min(rp.row_seg[r + 1] - j0, kArcRowArcsMax);
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    int label;
    s_occ[k] = arc_occupancy(rp, clamp_index(rp.row_arc[clamp_index(j0 + k, rp.n_row_arcs)], rp.n_arcs), mirror,
                             lnp, label);
    s_label[k] = label;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.f;
    for (int k = 0; k < n; ++k) tot += s_occ[k];
    s_tot = tot;
  }
  __syncthreads();
  const float lse2 = static_cast<float>(rp.lse2_rows[r]);
  const float tot = s_tot;
  const Tin* zr = static_cast<const Tin*>(p.logits) + static_cast<int64_t>(r) * p.V;
  Tout* gr = static_cast<Tout*>(p.grad) + static_cast<int64_t>(r) * p.V;
  for (int v = threadIdx.x; v < p.V; v += blockDim.x) {
    const float pr = fast_exp2(fmaf(ElemTraits<Tin>::load1(zr + v), kLog2eF, -lse2));
    float gv = pr * tot;
    for (int k = 0; k < n; ++k) gv = (s_label[k] == v) ? gv - s_occ[k] : gv;
    ElemTraits<Tout>::store1(gr + v, gv);
  }
}

}  // namespace rnnt
