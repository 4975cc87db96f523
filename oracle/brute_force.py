"""Enumeration of every alignment on tiny lattices (float64, CPU).

TEST INFRASTRUCTURE ONLY -- the product path never imports this module.

An RNN-T alignment (Section 1: exactly one non-blank output per unit, blank
moves to the next frame) of U units over T frames is a sequence of emissions
walked from frame 0, unit 0: a blank emitted at (t, u) moves to frame t+1, the
unit y_{u+1} emitted at (t, u) moves to unit u+1; the sequence holds all U units
in order and exactly T blanks, the last emission being a blank at frame T-1
(Fig. 1).  Its probability is the product of the emitted symbols'
probabilities at the (t, u) where they are emitted.

The W-Transducer (Section 3.2, Fig. 4) adds probability-one skips: the walk may
start at any frame s (a jump from (0, 0) to (s, 0), s >= 1) and, once all units
are emitted at (e, U) with e <= T-2, may jump to (T-1, U) and then must emit the
closing blank.  The allow-ignore variant (Section 4.3) jumps to the end instead
and needs no closing blank.

This enumerator walks those sequences directly (no lattice, no recursion over
nodes) and sums path probabilities; it is exponential, for T <= 5, U <= 3.
"""
import math


def path_log_scores(lp_blank, lp_label, variant="rnnt"):
    """Log-scores of every alignment (one entry per distinct arc sequence)."""
    T = len(lp_blank)
    U = len(lp_blank[0]) - 1
    out = []
    starts = [0] if variant == "rnnt" else list(range(T))
    for s in starts:
        _walk_from(s, T, U, lp_blank, lp_label, variant, out)
    return out


def _walk_from(s, T, U, lp_blank, lp_label, variant, out):
    # after a jump to (s, 0) (or the plain start s = 0) walk as usual; the flag
    # ``jumped`` marks a walk that took the final jump and now owes the closing blank
    stack = [(s, 0, 0.0, False)]
    while stack:
        t, u, score, jumped = stack.pop()
        if jumped:
            out.append(score + lp_blank[T - 1][U])
            continue
        if t == T - 1 and u == U:
            out.append(score + lp_blank[t][u])
        if t < T - 1:
            stack.append((t + 1, u, score + lp_blank[t][u], False))
        if u < U:
            stack.append((t, u + 1, score + lp_label[t][u], False))
        if u == U and t < T - 1:
            if variant == "wrnnt":
                stack.append((T - 1, U, score, True))
            elif variant == "wrnnt_allow_ignore":
                out.append(score)


def path_alignments(lp_blank, lp_label, variant="rnnt"):
    """Every alignment as (log-score, label frames, start frame, end frame).

    Label frame i is the frame at which unit y_{i+1} is emitted; the start frame
    is the frame the walk starts from (after an initial jump, or 0); the end frame
    is the frame of the last emitted unit's node (e, U) left by a final jump, or
    T-1 when the walk reaches (T-1, U) by itself.  The walk is the one of
    ``path_log_scores``, recording where each unit is emitted.
    """
    T = len(lp_blank)
    U = len(lp_blank[0]) - 1
    out = []
    starts = [0] if variant == "rnnt" else list(range(T))
    for s in starts:
        stack = [(s, 0, 0.0, ())]
        while stack:
            t, u, score, frames = stack.pop()
            if t == T - 1 and u == U:
                out.append((score + lp_blank[t][u], frames, s, T - 1))
            if t < T - 1:
                stack.append((t + 1, u, score + lp_blank[t][u], frames))
            if u < U:
                stack.append((t, u + 1, score + lp_label[t][u], frames + (t,)))
            if u == U and t < T - 1:
                if variant == "wrnnt":
                    out.append((score + lp_blank[T - 1][U], frames, s, t))
                elif variant == "wrnnt_allow_ignore":
                    out.append((score, frames, s, t))
    return out


def brute_force_log_prob(lp_blank, lp_label, variant="rnnt"):
    """ln of the summed probability of every alignment."""
    scores = path_log_scores(lp_blank, lp_label, variant)
    m = max(scores)
    return m + math.log(sum(math.exp(x - m) for x in scores))


def count_paths(T, U, variant="rnnt"):
    zeros = [[0.0] * (U + 1) for _ in range(T)]
    return len(path_log_scores(zeros, zeros, variant))


def graph_paths(arcs, start, final):
    """Every start->final path of an explicit weighted graph, by depth-first search.

    arcs: list of (src, dst, weight); parallel arcs are distinct entries.
    Returns a list of (log-score, tuple of arc indices).
    """
    out_arcs = {}
    for i, (s, d, w) in enumerate(arcs):
        out_arcs.setdefault(s, []).append((i, d, w))
    paths = []
    stack = [(start, 0.0, ())]
    while stack:
        n, sc, used = stack.pop()
        if n == final:
            paths.append((sc, used))
            continue
        for i, d, w in out_arcs.get(n, []):
            stack.append((d, sc + w, used + (i,)))
    return paths


def graph_paths_log_prob(arcs, start, final):
    """ln of the summed path probability and the number of paths."""
    paths = graph_paths(arcs, start, final)
    m = max(sc for sc, _ in paths)
    return m + math.log(sum(math.exp(sc - m) for sc, _ in paths)), len(paths)


def graph_arc_posteriors(arcs, start, final):
    """Share of the total path probability that passes through each arc."""
    paths = graph_paths(arcs, start, final)
    total = sum(math.exp(sc) for sc, _ in paths)
    post = [0.0] * len(arcs)
    for sc, used in paths:
        for i in used:
            post[i] += math.exp(sc) / total
    return post
