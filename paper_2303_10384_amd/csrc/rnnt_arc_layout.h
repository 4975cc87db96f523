// Layout of an arc-list lattice plan: the device image written by the host
// planner (rnnt_arc_plan.cpp) and read by the arc-list kernels
// (rnnt_arc_kernels.h).  Host and device code both include it.
//
// A batch's states are renumbered level by level: level 0 holds the states with
// no entering arc (the start first), and a state's level is one more than the
// highest level among its arcs' sources, so every arc climbs at least one level.
// The forward sweep ("graph 0") visits the levels upwards; the backward sweep
// runs the same algorithm on the reversed lattice ("graph 1"), whose states are
// the mirror images s' = s_begin + s_end - 1 - s and whose levels come in the
// opposite order.
//
// Each sweep keeps the scores of the last kArcRing states it computed in an LDS
// ring (state s at slot (s - s_begin) mod kArcRing); a source further back than
// that has its score pinned in one of kArcPins further LDS slots, chosen by the
// planner.  The planner also writes, per arc, the LDS slot its source is read
// from, so the sweep itself makes no such decision.
#pragma once

#include <stdint.h>

namespace rnnt {

constexpr int kArcRing = 4096;                     // ring of recent state scores (a power of 2)
constexpr int kArcPins = 2048;                     // pinned state scores, per sweep
constexpr int kArcDummy = kArcRing + kArcPins;     // LDS slot that takes stores with nowhere to go
constexpr int kArcLevelArcs = 4096;                // arcs entering one level (a power of 2)
constexpr int kArcLevelWindow = 512;               // level records staged in LDS at a time
constexpr int kArcRowArcsMax = 1024;               // arcs of a row that carries several labels

// Arrays of the image, in order; each starts 256-byte aligned.
//   utt      B x int4 {s_begin, s_end, l_begin, l_end}
//   ends     B x int4 {final state (graph 0), start state (graph 1), arc_begin, arc_end}
//   level_g  L x int4 {first state, states, first arc, arcs | max in-degree << 16}, graph g
//   seg_g    S x int  entering arcs of a state: (offset from the level's first arc) | count << 16
//   pin_g    S x int  LDS slot that also keeps the state's score (kArcDummy: none)
//   arcs     A x int4 {src, dst, row, label}, graph 0 order (sorted by destination);
//            row = (b * T_max + t) * (U_max + 1) + u, or -1 when label == -1
//   score    A x float natural-log arc scores, graph 0 order
//   loc_g    A x int  LDS slot of the arc's source score, in graph g's arc order
//   perm     A x int  position in graph 1's order of each graph-0 arc
//   row_seg  (R+1) x int  label arcs of logits row r: row_arc[row_seg[r] .. row_seg[r+1])
//   row_arc  N x int  graph-0 arc indices, per row blank arcs first, then by label
//   xrows    X x int  rows whose arcs carry two or more distinct non-blank labels
enum ArcImageArray {
  kImgUtt = 0,
  kImgEnds,
  kImgLevel0,
  kImgLevel1,
  kImgSeg0,
  kImgSeg1,
  kImgPin0,
  kImgPin1,
  kImgArcs,
  kImgScore,
  kImgLoc0,
  kImgLoc1,
  kImgPerm,
  kImgRowSeg,
  kImgRowArc,
  kImgXrows,
  kImgCount
};

}  // namespace rnnt
