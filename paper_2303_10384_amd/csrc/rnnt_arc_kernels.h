// Kernels of the loss over lattices given as arc lists (Section 2.2: a lattice
// graph whose arcs are filled in from X = log_softmax(logits) by indexed
// selection; the loss of Eq. 1 is its negative forward score, the gradient comes
// from its forward and backward scores).  The plan they read is laid out in
// rnnt_arc_layout.h; the row normaliser (kernel 1, rows mode) and the gradient
// kernel (kernel 3) are shared with the grid path.
//
//   populate   one thread per arc slot: the weight score + z[label] - lse in log2
//              units, stored with the source's LDS slot in the slot records of
//              both sweeps; NaN for an arc that reads a row outside its
//              utterance's valid rows, which flags the utterance.
//   sweep      one workgroup per (utterance, direction), a wavefront per chunk of
//              64 states of a level: the levels in order, one barrier each, in
//              blocks whose slot records and pins are first copied to LDS (every
//              load issued, then one wait), one lane per state.  On a padded level
//              a lane reads its state's slot records and each source score from
//              LDS and sums the terms in the log semiring; on a generic level one
//              lane per entering arc first forms the terms in LDS, then one lane
//              per state sums its run.
//   posteriors one thread per arc slot: the posterior of each label arc, in
//              slot order, with its label.
//   rows       one thread per logits row: the posteriors of the row's label
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

// Arc slot records, written by the populate kernel for both sweeps: three
// int32 per slot, the arc's weight in log2 units (a double, low word first) and
// the LDS slot of its source score (-1 for padding), so the sweep fetches a
// slot with one 12-byte load.
constexpr int kSlotWords = 3;

__device__ __forceinline__ void store_slot(int32_t* rec, int i, double w, int loc) {
  int32_t* r = rec + static_cast<int64_t>(i) * kSlotWords;
  r[0] = __double2loint(w);
  r[1] = __double2hiint(w);
  r[2] = loc;
}
__device__ __forceinline__ double slot_weight(const int32_t* rec, int i) {
  const int32_t* r = rec + static_cast<int64_t>(i) * kSlotWords;
  return __hiloint2double(r[1], r[0]);
}

struct ArcPopulateParams {
  const void* logits;
  int32_t B, T_max, U_max, V;
  int32_t n_slots0, n_slots1, n_rows;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int4* arcs;        // per graph-0 slot
  const float* score;
  const int32_t* perm;     // graph-0 slot -> graph-1 slot
  const int32_t* loc0;     // LDS slot of the source score, per graph-0 slot
  const int32_t* loc1;     // the same per graph-1 slot
  const double* lse2_rows; // log2 sum_v 2^(z_v kLog2eF) per valid row (the populate kernel's lse2f)
  int32_t* bad;            // (B): set to 1 for an utterance with a NaN arc weight (cleared by kernel 1)
  int32_t* rec0;           // slot records of graph 0
  int32_t* rec1;           // slot records of graph 1
};

// One thread per slot index: graph-0 slot i (a padding record, or the arc's
// weight stored for both sweeps) and, if graph-1 slot i is padding, its record.
template <typename T>
__global__ __launch_bounds__(256) void k_arc_populate(ArcPopulateParams p) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < p.n_slots1 && p.loc1[i] < 0) store_slot(p.rec1, i, 0.0, -1);
  if (i >= p.n_slots0) return;
  const int4 a = p.arcs[i];
  if (a.x < 0) {
    store_slot(p.rec0, i, 0.0, -1);
    return;
  }
  double w = static_cast<double>(p.score[i]) * kLog2eD;
  if (a.w >= 0) {
    const RowPos q = row_pos(a.z, p.T_max, p.U_max);
    const int Tb = p.logit_lens[clamp_index(q.b, p.B)];
    const int Ub = p.label_lens[clamp_index(q.b, p.B)];
    const bool ok = a.z >= 0 && a.z < p.n_rows && lengths_ok(Tb, Ub, p.T_max, p.U_max) && q.t < Tb && q.u <= Ub &&
                    a.w < p.V;
    if (ok) {
      const float z = ElemTraits<T>::load1(static_cast<const T*>(p.logits) + static_cast<int64_t>(a.z) * p.V + a.w);
      // (z - lse) log2(e), with lse = lse2f / kLog2eF
      w += (static_cast<double>(z) - p.lse2_rows[a.z] / static_cast<double>(kLog2eF)) * kLog2eD;
    } else {
      w = __builtin_nan("");
    }
    if (__builtin_isnan(w)) p.bad[clamp_index(q.b, p.B)] = 1;  // every writer stores the same value
  }
  store_slot(p.rec0, i, w, p.loc0[i]);
  const int j = clamp_index(p.perm[i], p.n_slots1);
  store_slot(p.rec1, j, w, p.loc1[j]);
}

// ---------------------------------------------------------------- sweep

struct ArcSweepParams {
  int32_t B, T_max, U_max;
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int4* utt;
  const int4* ends;
  const int4* slots;
  const int4* level[2];
  const int32_t* seg[2];
  const int32_t* pin[2];
  const int32_t* rec[2];  // slot records (weight, source LDS slot)
  double* val[2];   // scores per state, graph g's numbering (log2 units)
  double* lnp2;     // (2, B): log2 P from the forward sweep, then from the backward one
  const int32_t* bad;  // (B): an arc weight is NaN (flagged by the populate kernel)
  int32_t* status;  // (B): 0 scores valid, 1 bad data, 2 no path reaches the final state
  float* loss;      // (B) or null
};

__device__ __forceinline__ int buffer_load_i32(__amdgpu_buffer_rsrc_t r, int off) {
  return static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

__device__ __forceinline__ double lane_value(double x, int lane) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(x), lane);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(x), lane);
  return __hiloint2double(hi, lo);
}

// LDS stage of a block of consecutive levels: their slot records (raw bytes,
// from the 16-byte boundary at or below the block's first record) and the
// pinned LDS slots of their states.  Both are filled by direct-to-LDS buffer
// loads, 64 lanes x 16 (records) or 4 (pins) bytes per load, so the stages are
// whole numbers of such batches.
constexpr int kStageBatch = kWave * 16;
constexpr int kStageBytes = (kArcLevelArcs * kSlotWords * 4 + 16 + kStageBatch - 1) / kStageBatch * kStageBatch;
constexpr int kStageStates = kArcRing;  // any level's states (the planner bounds a level by the ring)
constexpr int kStageLevels = 64;  // levels per block: one level record per lane
static_assert(kStageStates % kWave == 0, "pins are staged 64 at a time");

typedef __attribute__((address_space(3))) void lds_void;

// vmcnt(0), expcnt and lgkmcnt left at their maxima (gfx9 encoding)
constexpr int kWaitVmcnt0 = 0x0F70;

// Barrier for LDS traffic between the wavefronts of a workgroup: the fences order
// LDS accesses only, so this wave's global stores stay in flight (a full
// __syncthreads() would wait for them at every level).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// NW wavefronts per (utterance, direction), wave w taking chunk w of 64 states of
// each level (one barrier per level: a level reads only earlier levels), and DM
// slots per state: the shape of the levels taken in three phases (all reads, all
// sums, all stores); other levels take a loop over their chunks.
template <int NW, int DM>
__global__ __launch_bounds__(kWave * NW) void k_arc_sweep(ArcSweepParams p) {
  __shared__ double s_val[kArcDummy + 1];                    // ring of recent scores, pinned scores, a dummy slot
  __shared__ double s_x[kArcLevelArcs];                      // terms of a generic level, one per entering arc
  __shared__ __attribute__((aligned(16))) int32_t s_rec[kStageBytes / 4];  // staged slot records
  __shared__ int32_t s_pin[kStageStates];                    // staged pinned LDS slots
  __shared__ double s_lnp;                                   // the score of the final state
  const int b = blockIdx.x >> 1;
  const int g = blockIdx.x & 1;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);  // this wavefront's chunk of each level
  const int Tb = p.logit_lens[b];
  const int Ub = p.label_lens[b];
  double* lnp_out = p.lnp2 + g * p.B + b;
  if (!lengths_ok(Tb, Ub, p.T_max, p.U_max)) {
    if (tid == 0) {
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
  const int4 sr = p.slots[b];
  const int s_begin = ut.x, n_states = ut.y - ut.x, l_begin = ut.z, l_end = ut.w;
  const int slot_begin = g ? sr.z : sr.x;
  const int n_slots = g ? sr.w - sr.z : sr.y - sr.x;
  const int start = g ? en.y : s_begin;   // the sweep's start state (score 0)
  const int fin = g ? ut.y - 1 : en.x;    // the state whose score is ln P
  // every record of the plan is read through a buffer bounded to this utterance; the
  // slot records' buffer starts at the 16-byte boundary at or below the first one
  const int32_t* rec_first = p.rec[g] + static_cast<int64_t>(slot_begin) * kSlotWords;
  const int rec_skew = static_cast<int>(reinterpret_cast<uintptr_t>(rec_first) & 15);  // bytes
  const __amdgpu_buffer_rsrc_t rs_rec = make_buffer(reinterpret_cast<const char*>(rec_first) - rec_skew,
                                                    static_cast<int64_t>(n_slots) * 12 + rec_skew);
  const __amdgpu_buffer_rsrc_t rs_seg = make_buffer(p.seg[g] + s_begin, static_cast<int64_t>(n_states) * 4);
  const __amdgpu_buffer_rsrc_t rs_pin = make_buffer(p.pin[g] + s_begin, static_cast<int64_t>(n_states) * 4);
  const __amdgpu_buffer_rsrc_t rs_val = make_buffer(p.val[g] + s_begin, static_cast<int64_t>(n_states) * 8);
  const __amdgpu_buffer_rsrc_t rs_lvl = make_buffer(p.level[g] + l_begin, static_cast<int64_t>(l_end - l_begin) * 16);

  // the level records of a block sit one per lane (lane i: level k0 + i), so a level's
  // record is four readlanes; past the utterance's levels a lane holds zeros
  auto load_records = [&](int k0) {
    return buffer_load16<false>(rs_lvl, (k0 - l_begin + lane) * 16);
  };
  auto record_of = [&](const u32x4& r, int i) {  // i uniform, < 64
    return make_int4(__builtin_amdgcn_readlane(static_cast<int>(r.x), i),
                     __builtin_amdgcn_readlane(static_cast<int>(r.y), i),
                     __builtin_amdgcn_readlane(static_cast<int>(r.z), i),
                     __builtin_amdgcn_readlane(static_cast<int>(r.w), i));
  };
  auto wave_prefix_sum = [&](int x) {  // inclusive, over the wave's lanes
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const int y = __shfl_up(x, d, kWave);
      x += (lane >= d) ? y : 0;
    }
    return x;
  };
  if (tid == 0) s_lnp = kNoArc;

  // source score + weight of one arc slot; kNoArc for padding and idle lanes
  auto term = [&](bool use, int loc, double w) {
    const double src = s_val[use ? min(static_cast<unsigned>(loc), static_cast<unsigned>(kArcDummy)) : kArcDummy];
    return use ? src + w : kNoArc;
  };
  // a state's score into its ring slot and its pinned slot; a lane without a state
  // writes the dummy slot (index arithmetic, so the stores are not branched around)
  auto finish = [&](int s, bool ok, double v, int pin) {
    v = (s == start) ? 0.0 : v;
    const int keep = -static_cast<int>(ok);
    const int ring = (s - s_begin) & (kArcRing - 1);
    const int pinned = static_cast<int>(min(static_cast<unsigned>(pin), static_cast<unsigned>(kArcDummy)));
    s_val[kArcDummy + ((ring - kArcDummy) & keep)] = v;
    s_val[kArcDummy + ((pinned - kArcDummy) & keep)] = v;
  };

  static_assert(kStageLevels == kWave, "a block's level records sit one per lane");
  u32x4 recs = load_records(l_begin);
  for (int k0 = l_begin; k0 < l_end;) {
    // the block: levels k0 .. k1-1 whose slot records and states fit the stage (at least
    // one level), from prefix sums over the lanes' records
    const int ps = wave_prefix_sum(static_cast<int>(recs.w & 0xffffu));
    const int pn = wave_prefix_sum(static_cast<int>(recs.y & (kArcGenericLevel - 1)));
    const bool fits = k0 + lane < l_end && (lane == 0 || (ps <= kArcLevelArcs && pn <= kStageStates));
    const int n_lv = __popcll(__ballot(fits));  // the fitting lanes are a prefix
    const int k1 = k0 + n_lv;
    const int slots = __builtin_amdgcn_readlane(ps, n_lv - 1);
    const int states = __builtin_amdgcn_readlane(pn, n_lv - 1);
    const int4 first = record_of(recs, 0);
    const u32x4 recs_next = load_records(k1);  // arrives with the stage below
    // copy the block's records and pins to LDS with direct-to-LDS loads, the waves
    // taking turns: every load issued, then one wait and a barrier (lane i of a load
    // fills bytes 16 i (records) or 4 i (pins))
    const int byte_lo = (first.z - slot_begin) * 12 + rec_skew;  // in the records' buffer
    const int byte_lo16 = byte_lo & ~15;
    const int skew = byte_lo - byte_lo16;
    const int n16 = (skew + slots * 12 + 15) / 16;
    for (int m = wv; m * kWave < n16; m += NW) {
      const int i = m * kWave + lane;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_rec, (lds_void*)(s_rec + m * (kStageBatch / 4)), 16,
                                               i < n16 ? byte_lo16 + i * 16 : kOutOfRange, 0, 0, 0);
    }
    const int srel0 = first.x - s_begin;
    for (int m = wv; m * kWave < states; m += NW) {
      const int i = m * kWave + lane;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_pin, (lds_void*)(s_pin + m * kWave), 4,
                                               i < states ? (srel0 + i) * 4 : kOutOfRange, 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    lds_barrier();
    // the block's levels, in order, from LDS; the next level's record and this wave's
    // slot records of it are read while the current level is summed (they do not
    // depend on any score), so a level waits only on its sources' scores
    auto level_info = [&](int k) { return record_of(recs, k - k0); };
    struct Pre {
      int4 li;
      bool fast;  // padded, one chunk per wave, at most DM slots per state
      double w[DM];
      int loc[DM];
      int pin;
    };
    auto read_pre = [&](int k) {
      Pre r;
      r.li = level_info(k);
      const int ns = r.li.y & (kArcGenericLevel - 1);
      const int D = static_cast<int>(static_cast<unsigned>(r.li.w) >> 16);
      r.fast = (r.li.y & kArcGenericLevel) == 0 && ns <= NW * kWave && D <= DM;
      const int j = wv * kWave + lane;
      const int rel_rec = skew / 4 + (r.li.z - first.z) * kSlotWords;
      r.pin = s_pin[min(max(r.li.x - first.x + j, 0), kStageStates - 1)];
#pragma unroll
      for (int q = 0; q < DM; ++q) {
        const bool use = r.fast && j < ns && q < D;
        // 24-bit multiplies (full rate): slots of a level stay below kArcLevelArcs
        const int at = use ? min(rel_rec + static_cast<int>(__umul24(__umul24(j, D) + q, kSlotWords)),
                                 kStageBytes / 4 - kSlotWords)
                           : 0;
        r.w[q] = __hiloint2double(s_rec[at + 1], s_rec[at]);
        r.loc[q] = use ? s_rec[at + 2] : -1;
      }
      return r;
    };
    Pre cur = read_pre(k0);
    for (int k = k0; k < k1; ++k) {
      Pre nxt;
      const int4 li = cur.li;
      const int s_lo = li.x;
      const int ns = li.y & (kArcGenericLevel - 1);
      const bool padded = (li.y & kArcGenericLevel) == 0;
      const int nslots = li.w & 0xffff;
      const int D = static_cast<int>(static_cast<unsigned>(li.w) >> 16);
      const int rel_rec = skew / 4 + (li.z - first.z) * kSlotWords;  // first record of the level in s_rec (words)
      const int srel = s_lo - s_begin;
      auto pin_of = [&](int j) { return s_pin[min(max(s_lo - first.x + j, 0), kStageStates - 1)]; };
      auto rec_term = [&](bool ok, int r) {  // slot record r of the level
        const int w0 = rel_rec + r * kSlotWords;
        const int at = ok ? min(max(w0, 0), kStageBytes / 4 - kSlotWords) : 0;
        const double w = __hiloint2double(s_rec[at + 1], s_rec[at]);
        const int loc = s_rec[at + 2];
        return term(ok && loc >= 0, loc, w);
      };
      if (cur.fast) {
        // one chunk per wave; no state of a level reads another state of it
        const int j = wv * kWave + lane;
        double src[DM];
#pragma unroll
        for (int q = 0; q < DM; ++q)
          src[q] = s_val[cur.loc[q] >= 0 ? min(static_cast<unsigned>(cur.loc[q]), static_cast<unsigned>(kArcDummy))
                                         : kArcDummy];
        // the sources' reads go out first: LDS answers in order, and the next level's
        // records are not needed before the barrier
        __builtin_amdgcn_sched_barrier(0);
        nxt = read_pre(k + 1 < k1 ? k + 1 : k);
        double v = kNoArc;
#pragma unroll
        for (int q = 0; q < DM; ++q) {
          const double x = cur.loc[q] >= 0 ? src[q] + cur.w[q] : kNoArc;
          v = (q == 0) ? x : log_add2(v, x);
        }
        finish(s_lo + j, j < ns, v, cur.pin);
      } else if (padded) {
        nxt = read_pre(k + 1 < k1 ? k + 1 : k);
        for (int c = wv; c * kWave < ns; c += NW) {
          const int j = c * kWave + lane;
          const bool ok = j < ns;
          double v = rec_term(ok && D > 0, j * D);
          for (int q = 1; q < D; ++q) v = log_add2(v, rec_term(ok, j * D + q));
          finish(s_lo + j, ok, v, pin_of(j));
        }
      } else {
        nxt = read_pre(k + 1 < k1 ? k + 1 : k);
        // generic level: one lane per entering arc forms its term, then one lane per state sums its run
        for (int c = wv; c * kWave < nslots; c += NW) {
          const int i = c * kWave + lane;
          s_x[i & (kArcLevelArcs - 1)] = rec_term(i < nslots, i);
        }
        lds_barrier();
        for (int c = wv; c * kWave < ns; c += NW) {
          const int j = c * kWave + lane;
          const bool ok = j < ns;
          const int seg = buffer_load_i32(rs_seg, ok ? (srel + j) * 4 : kOutOfRange);
          const int rel = seg & 0xffff;
          const int cnt = static_cast<int>(static_cast<unsigned>(seg) >> 16);
          double v = kNoArc;
          for (int q = 0; q < D; ++q) {
            const double x = s_x[(rel + q) & (kArcLevelArcs - 1)];
            v = log_add2(v, q < cnt ? x : kNoArc);
          }
          finish(s_lo + j, ok, v, pin_of(j));
        }
      }
      lds_barrier();  // the level's scores are in LDS before the next level reads them
      cur = nxt;
    }
    // the block's scores leave for global memory in one coalesced pass, from the ring
    // (a block's states all fit it); the next block's levels write the ring only after
    // the barrier that follows its stage copy
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    for (int i = tid; i < states; i += kWave * NW) {
      const int s = first.x + i;
      const double v = s_val[(s - s_begin) & (kArcRing - 1)];
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), rs_val, (s - s_begin) * 8, 0, 0);
      if (s == fin) s_lnp = v;
    }
    recs = recs_next;
    k0 = k1;
  }

  lds_barrier();
  if (tid == 0) {
    const double lp = s_lnp;
    *lnp_out = lp;
    if (g == 0) {
      const int st = (p.bad[b] != 0 || __builtin_isnan(lp)) ? 1 : (lp > 0.5 * kNoArc ? 0 : 2);
      p.status[b] = st;
      if (p.loss)
        p.loss[b] = st == 1 ? __builtin_nanf("")
                            : (st == 2 ? __builtin_inff() : static_cast<float>(-lp / kLog2eD));
    }
  }
}

// ---------------------------------------------------------------- row records

struct ArcRowParams {
  int32_t T_max, U_max, blank;
  int32_t n_rows, n_arcs, n_row_arcs, n_states;  // n_arcs: graph-0 slots
  const int32_t* logit_lens;
  const int32_t* label_lens;
  const int4* utt;
  const int4* arcs;
  const int32_t* row_seg;
  const int32_t* row_arc;
  const int32_t* rec0;    // graph-0 slot records
  const double* val0;
  const double* val1;
  const double* lnp2;
  const int32_t* status;
  const double* lse2_rows;
  int2* occ;        // per graph-0 slot: {posterior bits, label}, written by the posterior kernel
  RowInfo* rowinfo;
};

// Posterior of every graph-0 label arc, exp2(alpha(src) + w + beta(dst) - log2 P),
// computed in slot order: the slot's arc and record are read where consecutive
// threads read consecutive slots, and the scores of consecutive states mostly lie
// together too.  The row kernels then read one 8-byte pair per arc.  Padding,
// wild-card arcs and arcs of utterances without valid scores get {0, kNoLabel}.
template <int NT>
__global__ __launch_bounds__(NT) void k_arc_occ(ArcRowParams p) {
  const int i = blockIdx.x * NT + threadIdx.x;
  if (i >= p.n_arcs) return;
  const int4 a = p.arcs[i];
  int2 out = make_int2(0, kNoLabel);
  if (a.x >= 0 && a.w >= 0) {
    const int b = row_pos(clamp_index(a.z, p.n_rows), p.T_max, p.U_max).b;
    if (p.status[b] == 0) {
      const int4 ut = p.utt[b];
      const double e = p.val0[clamp_index(a.x, p.n_states)] + slot_weight(p.rec0, i) +
                       p.val1[clamp_index(ut.x + ut.y - 1 - a.y, p.n_states)] - p.lnp2[b];
      out = make_int2(__float_as_int(fast_exp2(static_cast<float>(e))), a.w);
    }
  }
  p.occ[i] = out;
}

// Posterior and label of graph-0 arc i (from the posterior kernel).
__device__ __forceinline__ float arc_occupancy(const ArcRowParams& p, int i, int& label) {
  const int2 o = p.occ[i];
  label = o.y;
  return __int_as_float(o.x);
}

template <int NT>
__global__ __launch_bounds__(NT) void k_arc_rows(ArcRowParams p) {
  const int r = blockIdx.x * NT + threadIdx.x;
  if (r >= p.n_rows) return;
  const RowPos q = row_pos(r, p.T_max, p.U_max);
  RowInfo ri;
  ri.lse2 = 0.f;
  ri.occ_blank = 0.f;
  ri.occ_label = 0.f;
  ri.label = kZeroRow;
  if (p.status[q.b] == 0 && q.t < p.logit_lens[q.b] && q.u <= p.label_lens[q.b]) {
    const int j0 = p.row_seg[r], j1 = p.row_seg[r + 1];
    float ob = 0.f, ol = 0.f;
    int primary = kNoLabel;
    bool extra = false;
    for (int j = j0; j < j1; ++j) {
      int label;
      const float occ = arc_occupancy(p, clamp_index(p.row_arc[clamp_index(j, p.n_row_arcs)], p.n_arcs), label);
      if (label == p.blank) {
        ob += occ;
      } else if (primary == kNoLabel || primary == label) {
        primary = label;
        ol += occ;
      } else {
        extra = true;  // a second non-blank label: the extra-rows kernel writes this row
      }
    }
    const float lse2 = static_cast<float>(p.lse2_rows[r]);
    // no posterior left in float32 and finite logits: the row's gradient is exactly +0 at
    // every v, written as a zero row without reading its logits (as for the grid lattice)
    if (!extra && !(ob == 0.f && ol == 0.f && __builtin_isfinite(lse2))) {
      ri.lse2 = lse2;
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
  const int j0 = rp.row_seg[r];
  const int n = min(rp.row_seg[r + 1] - j0, kArcRowArcsMax);
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    int label;
    s_occ[k] = arc_occupancy(rp, clamp_index(rp.row_arc[clamp_index(j0 + k, rp.n_row_arcs)], rp.n_arcs), label);
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
