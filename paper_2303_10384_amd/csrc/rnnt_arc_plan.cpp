// Host planner of arc-list lattices: rnnt_arc_plan and rnnt_arc_plan_bytes_bound
// (declared in include/rnnt_mi355x.h; the image layout is in rnnt_arc_layout.h).
//
// For each utterance the planner
//   1. checks the arc list (0 <= src < dst < n, labels in [-1, V), rows inside
//      the logits shape, finite scores);
//   2. gives every state its topological level (0 without entering arcs, else
//      one more than the highest level among its arcs' sources) and renumbers
//      the states level by level (ties by the original number, so the start
//      state comes first);
//   3. for the forward sweep (graph 0) and the backward one (graph 1, the
//      reversed lattice with mirrored numbers), sorts the arcs by destination,
//      records each level's state and arc ranges, each state's run of entering
//      arcs, and the LDS slot each arc reads its source score from: the ring
//      slot when the source lies within kArcRing states before the level, else
//      a pinned slot given to that source once;
//   4. groups the label arcs by logits row (blank arcs first, then by label)
//      for the gradient kernels, and lists the rows that carry two or more
//      distinct non-blank labels.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

#include "rnnt_arc_layout.h"
#include "rnnt_mi355x.h"

namespace rnnt {
namespace {

struct I4 {
  int32_t x, y, z, w;
};
static_assert(sizeof(I4) == 16, "int4 records");
static_assert(sizeof(rnnt_arc_t) == 24, "rnnt_arc_t is six 4-byte fields");

constexpr int64_t kMax32 = 0x7fffffff;
// states or arcs of one utterance: the sweep addresses an utterance's records
// through buffers of fewer than 2^31 bytes (8-byte scores)
constexpr int64_t kMaxPerUtterance = int64_t{1} << 27;

int64_t align_up(int64_t x) { return (x + 255) & ~int64_t{255}; }

struct Counts {
  int64_t B, L, S, A0, A1, N, R, X;  // A0 / A1: slots of the two sweeps
};

int64_t array_bytes(int i, const Counts& c) {
  switch (i) {
    case kImgUtt:
    case kImgEnds:
    case kImgSlots: return c.B * 16;
    case kImgLevel0:
    case kImgLevel1: return c.L * 16;
    case kImgSeg0:
    case kImgSeg1:
    case kImgPin0:
    case kImgPin1: return c.S * 4;
    case kImgArcs: return c.A0 * 16;
    case kImgScore:
    case kImgLoc0:
    case kImgPerm: return c.A0 * 4;
    case kImgLoc1: return c.A1 * 4;
    case kImgRowSeg: return (c.R + 1) * 4;
    case kImgRowArc: return c.N * 4;
    default: return c.X * 4;
  }
}

int64_t layout(const Counts& c, int64_t* off) {
  int64_t o = 0;
  for (int i = 0; i < kImgCount; ++i) {
    off[i] = o;
    o = align_up(o + array_bytes(i, c));
  }
  return o;
}

// One sweep (one graph) of one utterance, in local numbers: states 0..n-1 in
// level order, level k = states [first[k], first[k+1]).
struct Sweep {
  std::vector<int32_t> slot_arc;  // arc id per slot, -1 for padding
  std::vector<I4> level;          // {first state, states | generic << 30, first slot, slots | D << 16}, local
  std::vector<int32_t> seg, pin;  // per state
  std::vector<int32_t> loc;       // per slot (-1 for padding)
  int pins = 0;
  int max_deg = 0;
  int max_pad_deg = 0;            // largest D of a padded level
};

// Slots of a level: padded (D slots per state, state j's q-th entering arc at
// slot j*D + q) when D is at most kArcPadDegree and the padding at most doubles
// the level (or adds 64 slots); otherwise the entering arcs in destination order
// ("generic").
rnnt_status_t build_sweep(int n, const std::vector<int32_t>& first, const std::vector<int32_t>& src,
                          const std::vector<int32_t>& dst, Sweep& sw) {
  const int A = static_cast<int>(src.size());
  const int L = static_cast<int>(first.size()) - 1;
  std::vector<int32_t> order(A);
  for (int i = 0; i < A; ++i) order[i] = i;
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    if (dst[a] != dst[b]) return dst[a] < dst[b];
    if (src[a] != src[b]) return src[a] < src[b];
    return a < b;
  });
  sw.level.assign(L, I4{0, 0, 0, 0});
  sw.seg.assign(n, 0);
  sw.pin.assign(n, kArcDummy);
  sw.slot_arc.clear();
  std::vector<int32_t> first_arc(n + 1, 0);  // entering arcs of state s: order[first_arc[s] .. first_arc[s+1])
  for (int i = 0; i < A; ++i) ++first_arc[dst[i] + 1];
  for (int s = 0; s < n; ++s) first_arc[s + 1] += first_arc[s];
  for (int k = 0; k < L; ++k) {
    const int s_lo = first[k], s_hi = first[k + 1];
    const int ns = s_hi - s_lo;
    if (ns > kArcRing) return RNNT_ERR_UNSUPPORTED;
    const int na = first_arc[s_hi] - first_arc[s_lo];
    int deg = 0;
    for (int s = s_lo; s < s_hi; ++s) deg = std::max(deg, first_arc[s + 1] - first_arc[s]);
    const int64_t padded_slots = static_cast<int64_t>(ns) * deg;
    const bool padded = deg <= kArcPadDegree && padded_slots <= na + std::max(na, 64) &&
                        padded_slots <= kArcLevelArcs;
    if (!padded && na > kArcLevelArcs) return RNNT_ERR_UNSUPPORTED;
    const int slot_lo = static_cast<int>(sw.slot_arc.size());
    for (int s = s_lo; s < s_hi; ++s) {
      const int a0 = first_arc[s], cnt = first_arc[s + 1] - a0;
      const int rel = padded ? (s - s_lo) * deg : static_cast<int>(sw.slot_arc.size()) - slot_lo;
      sw.seg[s] = rel | (cnt << 16);
      for (int q = 0; q < (padded ? deg : cnt); ++q) sw.slot_arc.push_back(q < cnt ? order[a0 + q] : -1);
    }
    const int nslots = static_cast<int>(sw.slot_arc.size()) - slot_lo;
    sw.level[k] = I4{s_lo, ns | (padded ? 0 : kArcGenericLevel), slot_lo, nslots | (deg << 16)};
    sw.max_deg = std::max(sw.max_deg, deg);
    if (padded) sw.max_pad_deg = std::max(sw.max_pad_deg, deg);
  }
  // where each slot reads its source score: the ring when no state of the slot's
  // level shares the source's ring slot (the sweep may store a level's first
  // states before it reads the sources of its last ones), i.e. the source lies
  // within kArcRing states before the level's end; else a pinned slot given once
  sw.loc.assign(sw.slot_arc.size(), -1);
  for (int k = 0; k < L; ++k) {
    const int s_hi = sw.level[k].x + (sw.level[k].y & (kArcGenericLevel - 1));
    const int slot_lo = sw.level[k].z, nslots = sw.level[k].w & 0xffff;
    for (int p = slot_lo; p < slot_lo + nslots; ++p) {
      if (sw.slot_arc[p] < 0) continue;
      const int s = src[sw.slot_arc[p]];
      if (s >= s_hi - kArcRing) {
        sw.loc[p] = s & (kArcRing - 1);
      } else {
        if (sw.pin[s] == kArcDummy) {
          if (sw.pins == kArcPins) return RNNT_ERR_UNSUPPORTED;
          sw.pin[s] = kArcRing + sw.pins++;
        }
        sw.loc[p] = sw.pin[s];
      }
    }
  }
  return RNNT_OK;
}

int pick_chunks(std::vector<int>& sizes) {
  // the smallest register chunk count (64 lanes each) that holds all but ~1 % of the levels
  if (sizes.empty()) return 1;
  std::sort(sizes.begin(), sizes.end());
  const int v = sizes[(sizes.size() - 1) * 99 / 100];
  for (int c : {1, 2, 4, 8})
    if (c * 64 >= v) return c;
  return 8;
}

}  // namespace
}  // namespace rnnt

using namespace rnnt;

extern "C" {

size_t rnnt_arc_plan_bytes_bound(int32_t B, int32_t T_max, int32_t U_max, int64_t num_states, int64_t num_arcs) {
  if (B < 1 || T_max < 1 || U_max < 0 || num_states < 0 || num_arcs < 0) return 0;
  const int64_t R = static_cast<int64_t>(B) * T_max * (static_cast<int64_t>(U_max) + 1);
  if (R >= kMax32 || num_states > kMax32 || num_arcs > kMax32 || 2 * num_arcs + 64 * num_states > kMax32) return 0;
  // padding adds at most max(a level's arcs, 64) slots per level, and there are at most num_states levels
  const int64_t slots = 2 * num_arcs + 64 * num_states;
  const Counts c{B, num_states, num_states, slots, slots, num_arcs, R, std::min(R, num_arcs)};
  int64_t off[kImgCount];
  return static_cast<size_t>(layout(c, off));
}

rnnt_status_t rnnt_arc_plan(int32_t B, int32_t T_max, int32_t U_max, int32_t V, int32_t blank,
                            const int32_t* num_states, const int64_t* arc_begin, const rnnt_arc_t* arcs,
                            void* image, size_t image_bytes, rnnt_arc_plan_t* plan) {
  if (!num_states || !arc_begin || !image || !plan) return RNNT_ERR_NULL_PTR;
  if (B < 1 || T_max < 1 || U_max < 0 || V < 2) return RNNT_ERR_BAD_SHAPE;
  if (blank < 0 || blank >= V) return RNNT_ERR_BAD_BLANK;
  const int64_t U1 = static_cast<int64_t>(U_max) + 1;
  const int64_t R = static_cast<int64_t>(B) * T_max * U1;
  if (R >= kMax32) return RNNT_ERR_UNSUPPORTED;
  if (arc_begin[0] != 0) return RNNT_ERR_BAD_LATTICE;
  int64_t S = 0;
  for (int b = 0; b < B; ++b) {
    if (num_states[b] < 1 || arc_begin[b + 1] < arc_begin[b]) return RNNT_ERR_BAD_LATTICE;
    S += num_states[b];
  }
  const int64_t A = arc_begin[B];
  if (S > kMax32 || A > kMax32) return RNNT_ERR_UNSUPPORTED;
  if (A > 0 && !arcs) return RNNT_ERR_NULL_PTR;
  for (int b = 0; b < B; ++b) {
    for (int64_t i = arc_begin[b]; i < arc_begin[b + 1]; ++i) {
      const rnnt_arc_t& a = arcs[i];
      if (a.src < 0 || a.src >= a.dst || a.dst >= num_states[b]) return RNNT_ERR_BAD_LATTICE;
      if (a.label < -1 || a.label >= V || !std::isfinite(a.score)) return RNNT_ERR_BAD_LATTICE;
      if (a.label >= 0 && (a.t < 0 || a.t >= T_max || a.u < 0 || a.u > U_max)) return RNNT_ERR_BAD_LATTICE;
    }
  }

  std::vector<I4> utt(B), ends(B), slot_rng(B), level0, level1;
  std::vector<int32_t> seg0(S), seg1(S), pin0(S), pin1(S), loc0, loc1, perm, row_of;
  std::vector<I4> arc_img;
  std::vector<float> score;
  std::vector<int> level_states;
  int max_level_states = 0, max_level_arcs = 0, max_deg = 0, max_pad_deg = 0, max_pins = 0;

  int64_t s_base = 0;
  for (int b = 0; b < B; ++b) {
    const int n = num_states[b];
    const int64_t a_base = arc_begin[b];
    if (n > kMaxPerUtterance || arc_begin[b + 1] - a_base > kMaxPerUtterance) return RNNT_ERR_UNSUPPORTED;
    const int na = static_cast<int>(arc_begin[b + 1] - a_base);
    const rnnt_arc_t* ua = arcs + a_base;
    // levels, visiting the arcs by destination (sources are final by then: src < dst)
    std::vector<int32_t> by_dst(na);
    for (int i = 0; i < na; ++i) by_dst[i] = i;
    std::stable_sort(by_dst.begin(), by_dst.end(), [&](int x, int y) { return ua[x].dst < ua[y].dst; });
    std::vector<int32_t> lvl(n, 0);
    for (int i : by_dst) lvl[ua[i].dst] = std::max(lvl[ua[i].dst], lvl[ua[i].src] + 1);
    const int L = *std::max_element(lvl.begin(), lvl.end()) + 1;
    // level-order numbering (stable in the original number)
    std::vector<int32_t> first(L + 1, 0), newid(n);
    for (int s = 0; s < n; ++s) ++first[lvl[s] + 1];
    for (int k = 0; k < L; ++k) first[k + 1] += first[k];
    {
      std::vector<int32_t> fill(first.begin(), first.end() - 1);
      for (int s = 0; s < n; ++s) newid[s] = fill[lvl[s]]++;
    }
    std::vector<int32_t> src0(na), dst0(na), src1(na), dst1(na);
    for (int i = 0; i < na; ++i) {
      src0[i] = newid[ua[i].src];
      dst0[i] = newid[ua[i].dst];
      src1[i] = n - 1 - dst0[i];
      dst1[i] = n - 1 - src0[i];
    }
    std::vector<int32_t> first1(L + 1);
    for (int k = 0; k <= L; ++k) first1[k] = n - first[L - k];
    Sweep g0, g1;
    rnnt_status_t st = build_sweep(n, first, src0, dst0, g0);
    if (st != RNNT_OK) return st;
    st = build_sweep(n, first1, src1, dst1, g1);
    if (st != RNNT_OK) return st;

    const int64_t l_base = static_cast<int64_t>(level0.size());
    const int64_t p0 = static_cast<int64_t>(arc_img.size()), p1 = static_cast<int64_t>(loc1.size());
    const int64_t n0 = static_cast<int64_t>(g0.slot_arc.size()), n1 = static_cast<int64_t>(g1.slot_arc.size());
    if (p0 + n0 > kMax32 || p1 + n1 > kMax32 || n0 > kMaxPerUtterance || n1 > kMaxPerUtterance)
      return RNNT_ERR_UNSUPPORTED;
    utt[b] = I4{static_cast<int32_t>(s_base), static_cast<int32_t>(s_base + n), static_cast<int32_t>(l_base),
                static_cast<int32_t>(l_base + L)};
    const int fin = newid[n - 1];
    ends[b] = I4{static_cast<int32_t>(s_base + fin), static_cast<int32_t>(s_base + (n - 1 - fin)), 0, 0};
    slot_rng[b] = I4{static_cast<int32_t>(p0), static_cast<int32_t>(p0 + n0), static_cast<int32_t>(p1),
                     static_cast<int32_t>(p1 + n1)};
    for (int pass = 0; pass < 2; ++pass) {
      const Sweep& g = pass ? g1 : g0;
      const int64_t pb = pass ? p1 : p0;
      std::vector<I4>& lv = pass ? level1 : level0;
      for (const I4& r : g.level) {
        const int ns = r.y & 0x3fffffff;
        lv.push_back(I4{static_cast<int32_t>(s_base + r.x), r.y, static_cast<int32_t>(pb + r.z), r.w});
        level_states.push_back(ns);
        max_level_states = std::max(max_level_states, ns);
        max_level_arcs = std::max(max_level_arcs, r.w & 0xffff);
      }
      std::vector<int32_t>& sg = pass ? seg1 : seg0;
      std::vector<int32_t>& pn = pass ? pin1 : pin0;
      for (int s = 0; s < n; ++s) {
        sg[s_base + s] = g.seg[s];
        pn[s_base + s] = g.pin[s];
      }
      max_deg = std::max(max_deg, g.max_deg);
      max_pad_deg = std::max(max_pad_deg, g.max_pad_deg);
      max_pins = std::max(max_pins, g.pins);
    }
    loc1.insert(loc1.end(), g1.loc.begin(), g1.loc.end());
    std::vector<int32_t> pos1(na, -1);
    for (int64_t q = 0; q < n1; ++q)
      if (g1.slot_arc[q] >= 0) pos1[g1.slot_arc[q]] = static_cast<int32_t>(p1 + q);
    for (int64_t q = 0; q < n0; ++q) {
      const int id = g0.slot_arc[q];
      loc0.push_back(g0.loc[q]);
      if (id < 0) {  // padding
        arc_img.push_back(I4{-1, -1, -1, -2});
        score.push_back(0.f);
        perm.push_back(-1);
        row_of.push_back(-1);
        continue;
      }
      const rnnt_arc_t& a = ua[id];
      const int64_t row = a.label >= 0 ? (static_cast<int64_t>(b) * T_max + a.t) * U1 + a.u : -1;
      arc_img.push_back(I4{static_cast<int32_t>(s_base + src0[id]), static_cast<int32_t>(s_base + dst0[id]),
                           static_cast<int32_t>(row), a.label});
      score.push_back(a.score);
      perm.push_back(pos1[id]);
      row_of.push_back(static_cast<int32_t>(row));
    }
    s_base += n;
  }
  const int64_t A0 = static_cast<int64_t>(arc_img.size()), A1 = static_cast<int64_t>(loc1.size());

  // label arcs grouped by row (as graph-0 slots): blank first, then by label, then by slot
  std::vector<int32_t> row_seg(R + 1, 0);
  int64_t N = 0;
  for (int64_t q = 0; q < A0; ++q)
    if (row_of[q] >= 0) {
      ++row_seg[row_of[q] + 1];
      ++N;
    }
  for (int64_t r = 0; r < R; ++r) row_seg[r + 1] += row_seg[r];
  std::vector<int32_t> row_arc(N);
  {
    std::vector<int32_t> fill(row_seg.begin(), row_seg.end() - 1);
    for (int64_t q = 0; q < A0; ++q)
      if (row_of[q] >= 0) row_arc[fill[row_of[q]]++] = static_cast<int32_t>(q);
  }
  std::vector<int32_t> xrows;
  for (int64_t r = 0; r < R; ++r) {
    const int lo = row_seg[r], hi = row_seg[r + 1];
    if (hi - lo < 2) continue;
    std::sort(row_arc.begin() + lo, row_arc.begin() + hi, [&](int x, int y) {
      const int lx = arc_img[x].w, ly = arc_img[y].w;
      const bool bx = lx == blank, by = ly == blank;
      if (bx != by) return bx;
      if (lx != ly) return lx < ly;
      return x < y;
    });
    int distinct = 0, prev = -1;
    for (int j = lo; j < hi; ++j) {
      const int l = arc_img[row_arc[j]].w;
      if (l != blank && l != prev) {
        ++distinct;
        prev = l;
      }
    }
    if (distinct >= 2) {
      if (hi - lo > kArcRowArcsMax) return RNNT_ERR_UNSUPPORTED;
      xrows.push_back(static_cast<int32_t>(r));
    }
  }

  const int64_t L_total = static_cast<int64_t>(level0.size());
  const Counts c{B, L_total, S, A0, A1, N, R, static_cast<int64_t>(xrows.size())};
  int64_t off[kImgCount];
  const int64_t total = layout(c, off);
  if (static_cast<int64_t>(image_bytes) < total) return RNNT_ERR_WORKSPACE;
  char* img = static_cast<char*>(image);
  std::memset(img, 0, static_cast<size_t>(total));
  auto put = [&](int i, const void* src, int64_t bytes) {
    if (bytes > 0) std::memcpy(img + off[i], src, static_cast<size_t>(bytes));
  };
  put(kImgUtt, utt.data(), B * 16);
  put(kImgEnds, ends.data(), B * 16);
  put(kImgSlots, slot_rng.data(), B * 16);
  put(kImgLevel0, level0.data(), L_total * 16);
  put(kImgLevel1, level1.data(), L_total * 16);
  put(kImgSeg0, seg0.data(), S * 4);
  put(kImgSeg1, seg1.data(), S * 4);
  put(kImgPin0, pin0.data(), S * 4);
  put(kImgPin1, pin1.data(), S * 4);
  put(kImgArcs, arc_img.data(), A0 * 16);
  put(kImgScore, score.data(), A0 * 4);
  put(kImgLoc0, loc0.data(), A0 * 4);
  put(kImgLoc1, loc1.data(), A1 * 4);
  put(kImgPerm, perm.data(), A0 * 4);
  put(kImgRowSeg, row_seg.data(), (R + 1) * 4);
  put(kImgRowArc, row_arc.data(), N * 4);
  put(kImgXrows, xrows.data(), static_cast<int64_t>(xrows.size()) * 4);

  rnnt_arc_plan_t out{};
  out.B = B;
  out.T_max = T_max;
  out.U_max = U_max;
  out.V = V;
  out.blank = blank;
  out.num_states = static_cast<int32_t>(S);
  out.num_levels = static_cast<int32_t>(L_total);
  out.num_arcs = static_cast<int32_t>(A);
  out.num_row_arcs = static_cast<int32_t>(N);
  out.num_extra_rows = static_cast<int32_t>(xrows.size());
  out.num_slots[0] = static_cast<int32_t>(A0);
  out.num_slots[1] = static_cast<int32_t>(A1);
  out.max_level_states = max_level_states;
  out.max_level_arcs = max_level_arcs;
  out.max_in_degree = max_deg;
  out.max_pins = max_pins;
  out.state_chunks = pick_chunks(level_states);
  out.slots_per_state = max_pad_deg <= 1 ? 1 : (max_pad_deg <= 2 ? 2 : 4);
  out.image_bytes = total;
  for (int i = 0; i < kImgCount; ++i) out.off[i] = off[i];
  *plan = out;
  return RNNT_OK;
}

}  // extern "C"
