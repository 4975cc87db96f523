"""Best alignment (forced alignment) on the grid lattice, float64, CPU.

TEST INFRASTRUCTURE ONLY -- the product path never imports this module.

The lattice of Fig. 1 (Grid-Transducer, Section 2.3) and its W-Transducer forms
(Section 3.2, Fig. 4; allow-ignore, Section 4.3) serve forced alignment as
well as training (Section 2.2: the lattice formulations agree for both).  Forced
alignment picks the single path of highest probability instead of summing over
all paths: the forward recursion of ``rnnt_ref.forward_scores`` with the
log-sum replaced by a maximum, plus back-pointers.

Result for one utterance:
* ``score``: the best path's log-probability (natural log, closing blank
  included where the path takes it);
* ``label_frames[i]``: the frame t at which unit y_{i+1} is emitted, i.e. the
  path takes the label arc (t, i) -> (t, i+1);
* ``start_frame``: 0, or s when the path enters (s, 0) from (0, 0) by an
  initial wild-card arc;
* ``end_frame``: T-1, or e when the path leaves (e, U), e <= T-2, by a final
  wild-card arc.

Ties are broken in a fixed order, so the result is unique: at a node the
candidates are taken in the order blank arc, label arc, initial wild-card arc,
final wild-card arcs, and a later candidate replaces the current one only when
strictly greater; among the final wild-card arcs the earliest source frame wins;
at the end of the allow-ignore lattice the closing blank wins a tie with the
jump to the final state.  The same order is written into the GPU kernel.
"""
import math

import numpy as np

NEG_INF = -math.inf

# back-pointer codes
FROM_BLANK, FROM_LABEL, FROM_START_SKIP, FROM_FINAL_SKIP = 0, 1, 2, 3


def best_alignment(lp_blank, lp_label, variant="rnnt"):
    """Max-plus recursion over the (T, U+1) grid, t-outer / u-inner.

    lp_blank, lp_label: (T, U+1) arc log-probabilities (lp_label[:, U] unused).
    Returns dict(score, label_frames (list of U ints), start_frame, end_frame).
    """
    assert variant in ("rnnt", "wrnnt", "wrnnt_allow_ignore")
    lp_blank = np.asarray(lp_blank, dtype=np.float64)
    lp_label = np.asarray(lp_label, dtype=np.float64)
    T, U1 = lp_blank.shape
    U = U1 - 1
    delta = np.full((T, U1), NEG_INF)
    back = np.full((T, U1), -1, dtype=np.int64)
    delta[0, 0] = 0.0
    skip_src = -1  # source frame of the final wild-card arc into (T-1, U), when taken
    for t in range(T):
        for u in range(U1):
            if t == 0 and u == 0:
                continue
            best, arg = NEG_INF, -1
            if t > 0:  # blank arc (t-1, u) -> (t, u)
                best, arg = delta[t - 1, u] + lp_blank[t - 1, u], FROM_BLANK
            if u > 0:  # label arc (t, u-1) -> (t, u)
                c = delta[t, u - 1] + lp_label[t, u - 1]
                if arg < 0 or c > best:
                    best, arg = c, FROM_LABEL
            if variant != "rnnt" and u == 0 and t >= 1:  # initial wild-card arc (0, 0) -> (t, 0)
                c = delta[0, 0]
                if arg < 0 or c > best:
                    best, arg = c, FROM_START_SKIP
            if variant == "wrnnt" and u == U and t == T - 1 and T >= 2:
                # final wild-card arcs (t', U) -> (T-1, U), t' <= T-2; the earliest best source
                src = max(range(T - 1), key=lambda tp: (delta[tp, U], -tp))
                c = delta[src, U]
                if arg < 0 or c > best:
                    best, arg = c, FROM_FINAL_SKIP
                    skip_src = src
            delta[t, u] = best
            back[t, u] = arg

    # the end of the path
    score = delta[T - 1, U] + lp_blank[T - 1, U]  # closing blank from (T-1, U)
    t, u = T - 1, U
    end_frame = T - 1
    if variant == "wrnnt_allow_ignore" and T >= 2:
        src = max(range(T - 1), key=lambda tp: (delta[tp, U], -tp))
        if delta[src, U] > score:  # (src, U) -> final state, weight 0
            score = delta[src, U]
            t, end_frame = src, src
    if variant == "wrnnt" and back[T - 1, U] == FROM_FINAL_SKIP:
        t, end_frame = skip_src, skip_src

    # walk the back-pointers to (0, 0)
    label_frames = [-1] * U
    start_frame = 0
    while (t, u) != (0, 0):
        b = back[t, u]
        if b == FROM_BLANK:
            t -= 1
        elif b == FROM_LABEL:
            label_frames[u - 1] = t
            u -= 1
        elif b == FROM_START_SKIP:
            start_frame = t
            break
        else:
            raise AssertionError("final wild-card back-pointer inside the walk")
    return {"score": float(score), "label_frames": label_frames, "start_frame": start_frame,
            "end_frame": end_frame}


def alignment_score(lp_blank, lp_label, label_frames, start_frame, end_frame, variant="rnnt"):
    """Log-probability of the one path described by (label_frames, start, end).

    The path: (0, 0), a jump to (start_frame, 0) if start_frame > 0, then from
    frame start_frame on, blanks and the units at their frames, until (end_frame,
    U); then, if end_frame < T-1, the final jump; then the closing blank unless the
    allow-ignore jump ended the path.  Returns -inf for an impossible description.
    """
    lp_blank = np.asarray(lp_blank, dtype=np.float64)
    lp_label = np.asarray(lp_label, dtype=np.float64)
    T, U1 = lp_blank.shape
    U = U1 - 1
    frames = list(label_frames)
    if len(frames) != U or not (0 <= start_frame <= end_frame <= T - 1):
        return NEG_INF
    if variant == "rnnt" and (start_frame != 0 or end_frame != T - 1):
        return NEG_INF
    if any(f < start_frame or f > end_frame for f in frames) or frames != sorted(frames):
        return NEG_INF
    score = 0.0
    t, u = start_frame, 0
    while True:
        # units emitted at this frame, in order
        while u < U and frames[u] == t:
            score += lp_label[t, u]
            u += 1
        if t == end_frame:
            break
        score += lp_blank[t, u]
        t += 1
    if u != U:
        return NEG_INF
    if end_frame < T - 1:
        if variant == "rnnt":
            return NEG_INF
        if variant == "wrnnt":
            score += lp_blank[T - 1, U]
        return score
    return score + lp_blank[T - 1, U]


def utterance_alignment(z, labels, blank=0, variant="rnnt"):
    """Forced alignment of one utterance from its logits (T, U+1, V)."""
    from .rnnt_ref import lattice_weights
    _, lp_b, lp_l = lattice_weights(z, labels, blank)
    return best_alignment(lp_b, lp_l, variant)
