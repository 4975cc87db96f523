"""Pins of the forced-alignment oracle (oracle/viterbi.py), CPU only.

The best path is pinned by enumeration: every alignment of a tiny lattice
(brute_force.path_alignments, a walk over emission sequences with no lattice
recursion) and every path of the graphs transcribed from Fig. 1 and Fig. 4
(brute_force.graph_paths).  The tie rule is pinned by all-zero weights, where
every path scores the same.
"""
import math

import numpy as np
import pytest

from figures import allow_ignore_from_fig4, grid_weights, load_figure
from oracle import brute_force as BF
from oracle import rnnt_ref as R
from oracle import viterbi as VB

VARIANTS = R.VARIANTS


def random_weights(rng, T, U):
    return -rng.exponential(1.0, size=(T, U + 1)), -rng.exponential(1.5, size=(T, U + 1))


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("U", [0, 1, 2, 3])
def test_best_path_is_the_enumerated_maximum(variant, T, U):
    rng = np.random.default_rng(100 * T + 10 * U + VARIANTS.index(variant))
    for _ in range(4):
        lp_b, lp_l = random_weights(rng, T, U)
        paths = BF.path_alignments(lp_b.tolist(), lp_l.tolist(), variant)
        scores = np.array([p[0] for p in paths])
        best = scores.max()
        r = VB.best_alignment(lp_b, lp_l, variant)
        assert abs(r["score"] - best) <= 1e-12
        # the returned description is a path of that score
        own = VB.alignment_score(lp_b, lp_l, r["label_frames"], r["start_frame"], r["end_frame"], variant)
        assert abs(own - best) <= 1e-12
        # with a unique maximum it is the enumerated best path
        order = np.sort(scores)
        if len(order) == 1 or order[-1] - order[-2] > 1e-9:
            s, fr, st, en = paths[int(np.argmax(scores))]
            assert (tuple(r["label_frames"]), r["start_frame"], r["end_frame"]) == (fr, st, en)


@pytest.mark.parametrize("variant", VARIANTS)
def test_enumerated_descriptions_score_themselves(variant):
    rng = np.random.default_rng(7)
    lp_b, lp_l = random_weights(rng, 4, 3)
    for sc, fr, st, en in BF.path_alignments(lp_b.tolist(), lp_l.tolist(), variant):
        assert abs(VB.alignment_score(lp_b, lp_l, list(fr), st, en, variant) - sc) <= 1e-12


def figure_best(fig):
    """Best path of a transcribed figure graph: score and the frames of its unit arcs."""
    arcs = [(s, d, w) for (s, d, sym, w) in fig["arcs"]]
    paths = BF.graph_paths(arcs, 0, fig["final"])
    sc, used = max(paths, key=lambda p: p[0])
    frames = [fig["nodes"][fig["arcs"][i][0]][0] for i in used if fig["arcs"][i][2] in fig["units"]]
    return sc, frames


@pytest.mark.parametrize("variant,loader", [
    ("rnnt", lambda: load_figure("fig1_rnnt_lattice.txt")),
    ("wrnnt", lambda: load_figure("fig4_wrnnt_lattice.txt")),
    ("wrnnt_allow_ignore", lambda: allow_ignore_from_fig4(load_figure("fig4_wrnnt_lattice.txt"))),
])
def test_printed_lattices(variant, loader):
    fig = loader()
    lp_b, lp_l = map(np.array, grid_weights(fig))
    sc, frames = figure_best(fig)
    r = VB.best_alignment(lp_b, lp_l, variant)
    assert abs(r["score"] - sc) <= 1e-9
    assert r["label_frames"] == frames


def test_fig1_best_path_by_hand():
    # Fig. 1: the best alignment emits A at frame 1 and C at frame 1 (weights read off the figure:
    # <b>(0,0) -0.17, A(1,0) -1.55, C(1,1) -1.86, then blanks at (1,2), (2,2) and the closing (3,2))
    fig = load_figure("fig1_rnnt_lattice.txt")
    lp_b, lp_l = map(np.array, grid_weights(fig))
    r = VB.best_alignment(lp_b, lp_l, "rnnt")
    expect = lp_b[0, 0] + lp_l[1, 0] + lp_l[1, 1] + lp_b[1, 2] + lp_b[2, 2] + lp_b[3, 2]
    assert r["label_frames"] == [1, 1]
    assert abs(r["score"] - expect) <= 1e-12


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("T,U", [(1, 0), (3, 0), (1, 3), (4, 2), (6, 3)])
def test_tie_rule_on_equal_weights(variant, T, U):
    # all arcs weigh 0: every path scores 0 and the fixed order decides: walking back from
    # (T-1, U) the blank arc wins every tie, so all units sit on frame 0 and no skip is taken
    z = np.zeros((T, U + 1))
    r = VB.best_alignment(z, z, variant)
    assert r["score"] == 0.0
    assert r["label_frames"] == [0] * U
    assert (r["start_frame"], r["end_frame"]) == (0, T - 1)


@pytest.mark.parametrize("variant", VARIANTS)
def test_max_below_sum(variant):
    rng = np.random.default_rng(11)
    for T, U in [(5, 3), (9, 4), (12, 7)]:
        lp_b, lp_l = random_weights(rng, T, U)
        r = VB.best_alignment(lp_b, lp_l, variant)
        _, lnP = R.forward_scores(lp_b, np.where(np.arange(U + 1) < U, lp_l, -np.inf), variant)
        n = BF.count_paths(T, U, variant) if T * U <= 40 else None
        assert r["score"] <= lnP + 1e-12
        if n is not None:
            assert r["score"] >= lnP - math.log(n) - 1e-12


def test_single_path_cases():
    rng = np.random.default_rng(3)
    lp_b, lp_l = random_weights(rng, 6, 0)  # U = 0: blanks only
    r = VB.best_alignment(lp_b, lp_l, "rnnt")
    assert abs(r["score"] - lp_b[:, 0].sum()) <= 1e-12 and r["label_frames"] == []
    lp_b, lp_l = random_weights(rng, 1, 4)  # T = 1: all units, then the closing blank
    r = VB.best_alignment(lp_b, lp_l, "rnnt")
    assert abs(r["score"] - (lp_l[0, :4].sum() + lp_b[0, 4])) <= 1e-12 and r["label_frames"] == [0, 0, 0, 0]


def test_skips_are_taken_when_they_pay():
    # W-Transducer: frames before the first unit and after the last are expensive as blanks,
    # so the best path jumps over them
    T, U = 8, 2
    lp_b = np.full((T, U + 1), -5.0)
    lp_l = np.full((T, U + 1), -5.0)
    lp_l[3, 0], lp_l[4, 1] = -0.1, -0.1   # units at frames 3 and 4
    lp_b[3, 1] = -0.1                      # the blank between them
    lp_b[T - 1, U] = -0.1                  # the closing blank
    r = VB.best_alignment(lp_b, lp_l, "wrnnt")
    assert (r["label_frames"], r["start_frame"], r["end_frame"]) == ([3, 4], 3, 4)
    assert abs(r["score"] - (-0.4)) <= 1e-12
    r = VB.best_alignment(lp_b, lp_l, "wrnnt_allow_ignore")
    assert (r["label_frames"], r["start_frame"], r["end_frame"]) == ([3, 4], 3, 4)
    assert abs(r["score"] - (-0.3)) <= 1e-12
    r = VB.best_alignment(lp_b, lp_l, "rnnt")
    assert r["start_frame"] == 0 and r["end_frame"] == T - 1


@pytest.mark.parametrize("variant", ["wrnnt", "wrnnt_allow_ignore"])
def test_final_skip_tie_takes_the_earliest_source(variant):
    # every node (t', U), t' <= T-2, is reached with score 0 and the ends through frame T-1 cost
    # -5, so the final wild-card arc wins and its sources tie: the earliest frame is taken
    T, U = 5, 1
    lp_b = np.zeros((T, U + 1))
    lp_l = np.zeros((T, U + 1))
    lp_b[:, U] = -5.0      # blanks after the unit
    lp_l[T - 1, 0] = -5.0  # the unit at the last frame
    r = VB.best_alignment(lp_b, lp_l, variant)
    assert (r["label_frames"], r["start_frame"], r["end_frame"]) == ([0], 0, 0)
    assert r["score"] == (-5.0 if variant == "wrnnt" else 0.0)


def test_logits_entry_matches_weights_entry():
    rng = np.random.default_rng(5)
    z = rng.standard_normal((6, 4, 9)) * 2.0
    labels = np.array([3, 1, 7])
    r1 = VB.utterance_alignment(z, labels, 0, "wrnnt")
    _, lp_b, lp_l = R.lattice_weights(z, labels, 0)
    r2 = VB.best_alignment(lp_b, lp_l, "wrnnt")
    assert r1 == r2


# planted mistakes in the forced-alignment oracle must fail the pins above
VB_MUTATIONS = {
    "label_wins_ties": ("if arg < 0 or c > best:\n                    best, arg = c, FROM_LABEL",
                        "if arg < 0 or c >= best:\n                    best, arg = c, FROM_LABEL"),
    "no_initial_skip": ("if variant != \"rnnt\" and u == 0 and t >= 1:", "if False:"),
    "latest_final_source": ("key=lambda tp: (delta[tp, U], -tp))\n                c = delta[src, U]",
                            "key=lambda tp: (delta[tp, U], tp))\n                c = delta[src, U]"),
    "label_frame_off_by_one": ("label_frames[u - 1] = t", "label_frames[u - 1] = t - 1"),
    "blank_weight_wrong_frame": ("delta[t - 1, u] + lp_blank[t - 1, u]", "delta[t - 1, u] + lp_blank[t, u]"),
}


@pytest.mark.parametrize("name", sorted(VB_MUTATIONS))
def test_mutants_are_caught(name, monkeypatch):
    import types
    src = open(VB.__file__).read()
    old, new = VB_MUTATIONS[name]
    assert src.count(old) == 1, name
    mod = types.ModuleType("viterbi_mutant")
    mod.__dict__["__package__"] = "oracle"
    exec(compile(src.replace(old, new), VB.__file__ + ":" + name, "exec"), mod.__dict__)
    monkeypatch.setattr(VB, "best_alignment", mod.best_alignment)
    caught = False
    for check in (lambda: test_best_path_is_the_enumerated_maximum("wrnnt", 4, 2),
                  lambda: test_best_path_is_the_enumerated_maximum("rnnt", 3, 2),
                  lambda: test_tie_rule_on_equal_weights("wrnnt", 4, 2),
                  lambda: test_printed_lattices("rnnt", lambda: load_figure("fig1_rnnt_lattice.txt")),
                  lambda: test_skips_are_taken_when_they_pay(),
                  lambda: test_final_skip_tie_takes_the_earliest_source("wrnnt"),
                  lambda: test_tie_rule_on_equal_weights("wrnnt", 3, 0)):
        try:
            check()
        except AssertionError:
            caught = True
            break
    assert caught, name
