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
// ring (state s at slot (s - s_begin) mod kArcRing).  An arc reads its source
// from the ring only when the source lies within kArcRing states before the end
// of the arc's level, so no state of that level overwrites it whatever order
// the level's states are stored in; a source further back has its score pinned
// in one of kArcPins further LDS slots, chosen by the planner.  The planner also writes, per arc, the LDS slot its source is read
// from, so the sweep itself makes no such decision.
//
// The arcs entering a level occupy a run of "arc slots".  A padded level gives
// each of its states D slots (D the level's largest in-degree, at most
// kArcPadDegree), state j's q-th entering arc in slot j*D + q and unused slots
// marked as padding, so a lane finds its state's arcs by arithmetic; a generic
// level (a larger D, or padding that would more than double it) lists its
// entering arcs in destination order and each state records where its run
// starts.
#pragma once

#include <stdint.h>

namespace rnnt {

constexpr int kArcRing = 4096;                     // ring of recent state scores (a power of 2)
constexpr int kArcPins = 2048;                     // pinned state scores, per sweep
constexpr int kArcDummy = kArcRing + kArcPins;     // LDS slot that takes stores with nowhere to go
constexpr int kArcLevelArcs = 4096;                // arcs entering one level (a power of 2)
constexpr int kArcRowArcsMax = 1024;               // arcs of a row that carries several labels
constexpr int kArcPadDegree = 4;                   // largest in-degree of a padded level
constexpr int kArcGenericLevel = 1 << 30;          // flag in a level record's state count

// Arrays of the image, in order; each starts 256-byte aligned.
//   utt      B x int4 {s_begin, s_end, l_begin, l_end}
//   ends     B x int4 {final state (graph 0), start state (graph 1), 0, 0}
//   slots    B x int4 {first, end arc slot of graph 0, first, end arc slot of graph 1}
//   level_g  L x int4 {first state, states | kArcGenericLevel if generic, first slot, slots | D << 16}
//   seg_g    S x int  a state's entering arcs: (first slot - the level's first slot) | count << 16
//   pin_g    S x int  LDS slot that also keeps the state's score (kArcDummy: none)
//   arcs     A0 x int4 {src, dst, row, label} per graph-0 slot, padding {-1, -1, -1, -2};
//            row = (b * T_max + t) * (U_max + 1) + u, or -1 when label == -1
//   score    A0 x float natural-log arc scores
//   loc0     A0 x int  LDS slot of the slot's source score, -1 for padding
//   loc1     A1 x int  the same for graph 1's slots
//   perm     A0 x int  graph-1 slot of each graph-0 slot's arc (-1 for padding)
//   row_seg  (R+1) x int  label arcs of logits row r: row_arc[row_seg[r] .. row_seg[r+1])
//   row_arc  N x int  graph-0 slots, per row blank arcs first, then by label
//   xrows    X x int  rows whose arcs carry two or more distinct non-blank labels
enum ArcImageArray {
  kImgUtt = 0,
  kImgEnds,
  kImgSlots,
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
