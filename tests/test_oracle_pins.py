"""Pins of the float64 oracle against what the paper and the mathematics fix.

Every check here is independent of the oracle's own arithmetic: the paper's
printed lattices (Fig. 1, Fig. 4), path enumeration, closed forms for uniform
logits, special cases that reduce to a single path, finite differences,
library autograd and conservation laws of the arc posteriors.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from figures import allow_ignore_from_fig4, grid_weights, load_figure
from oracle import brute_force as BF
from oracle import lattice_dag as DAG
from oracle import rnnt_ref as R

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def expected():
    with open(os.path.join(GOLDEN, "fig_expected.json")) as f:
        return json.load(f)


# ----------------------------------------------------------------------------
# Worked examples printed in the paper
# ----------------------------------------------------------------------------

FIGS = [
    ("rnnt", "rnnt_fig1", lambda: load_figure("fig1_rnnt_lattice.txt")),
    ("wrnnt", "wrnnt_fig4", lambda: load_figure("fig4_wrnnt_lattice.txt")),
    ("wrnnt_allow_ignore", "wrnnt_allow_ignore_fig4_redirected",
     lambda: allow_ignore_from_fig4(load_figure("fig4_wrnnt_lattice.txt"))),
]


def test_golden_values_are_the_hand_computed_pins():
    """Stored losses equal the values computed from the printed weights."""
    e = expected()
    assert e["rnnt_fig1"]["loss"] == pytest.approx(4.2574511041, abs=1e-10)
    assert e["wrnnt_fig4"]["loss"] == pytest.approx(2.2070452674, abs=1e-10)
    assert e["wrnnt_allow_ignore_fig4_redirected"]["loss"] == pytest.approx(1.9385100266, abs=1e-10)
    assert e["rnnt_fig1"]["n_paths"] == math.comb(4 - 1 + 2, 2)


@pytest.mark.parametrize("variant,key,loader", FIGS)
def test_grid_recursion_reproduces_figure(variant, key, loader):
    """Grid alpha/beta on the printed weights == enumeration of the drawn graph."""
    fig = loader()
    lp_b, lp_l = grid_weights(fig)
    lp_b, lp_l = np.array(lp_b), np.array(lp_l)
    alpha, lnP = R.forward_scores(lp_b, lp_l, variant)
    beta, lnP_b = R.backward_scores(lp_b, lp_l, variant)
    exp_loss = expected()[key]["loss"]
    assert -lnP == pytest.approx(exp_loss, abs=1e-12)
    assert -lnP_b == pytest.approx(exp_loss, abs=1e-12)
    # figure graph enumerated here directly as well (the golden file could be stale)
    arcs = [(s, d, w) for (s, d, _sym, w) in fig["arcs"]]
    assert -BF.graph_paths_log_prob(arcs, 0, fig["final"])[0] == pytest.approx(exp_loss, abs=1e-12)
    # per-arc posteriors of every blank and unit arc
    occ_b, occ_l = R.arc_posteriors(alpha, beta, lp_b, lp_l, lnP)
    for (s, d, sym, p) in expected()[key]["arc_posteriors"]:
        if sym == "<eps>":
            continue
        t, u = fig["nodes"][s]
        got = occ_b[t, u] if sym == "<b>" else occ_l[t, u]
        assert got == pytest.approx(p, abs=1e-12), (s, d, sym)


def test_fig1_printed_occupancy_pins():
    fig = load_figure("fig1_rnnt_lattice.txt")
    lp_b, lp_l = map(np.array, grid_weights(fig))
    alpha, lnP = R.forward_scores(lp_b, lp_l, "rnnt")
    beta, _ = R.backward_scores(lp_b, lp_l, "rnnt")
    ob, ol = R.arc_posteriors(alpha, beta, lp_b, lp_l, lnP)
    assert ob[0, 0] == pytest.approx(0.6692677774, abs=1e-10)
    assert ol[0, 0] == pytest.approx(0.3307322226, abs=1e-10)
    assert ob[3, 2] == pytest.approx(1.0, abs=1e-14)
    assert ol[3, 1] == pytest.approx(0.1082525647, abs=1e-10)
    assert ob.sum() == pytest.approx(4.0, abs=1e-12)
    assert ol.sum() == pytest.approx(2.0, abs=1e-12)


def test_fig4_printed_occupancy_pins():
    fig = load_figure("fig4_wrnnt_lattice.txt")
    lp_b, lp_l = map(np.array, grid_weights(fig))
    alpha, lnP = R.forward_scores(lp_b, lp_l, "wrnnt")
    beta, _ = R.backward_scores(lp_b, lp_l, "wrnnt")
    ob, ol = R.arc_posteriors(alpha, beta, lp_b, lp_l, lnP)
    assert ob[0, 0] == pytest.approx(0.3439563866, abs=1e-10)
    assert ol[0, 0] == pytest.approx(0.2123980526, abs=1e-10)
    assert ob[3, 2] == pytest.approx(1.0, abs=1e-14)
    assert ol[3, 1] == pytest.approx(0.0608619270, abs=1e-10)
    assert ob.sum() == pytest.approx(2.2280408132, abs=1e-10)
    assert ol.sum() == pytest.approx(2.0, abs=1e-12)


@pytest.mark.parametrize("variant,key,loader", FIGS)
def test_arc_list_builder_matches_figure(variant, key, loader):
    """The arc-list formulation draws exactly the figure's arcs (as multisets)."""
    fig = loader()
    T, U = fig["frames"], len(fig["units"])
    inv = {v: k for k, v in fig["nodes"].items()}
    inv[DAG.FINAL] = fig["final"]
    built = sorted((inv[s], inv[d], {"blank": "<b>", "skip": "<eps>"}.get(kind, fig["units"][u] if kind == "label" else None))
                   for (s, d, kind, t, u) in DAG.grid_arcs(T, U, variant))
    drawn = sorted((s, d, sym) for (s, d, sym, _w) in fig["arcs"])
    assert built == drawn


# ----------------------------------------------------------------------------
# Enumeration of alignments
# ----------------------------------------------------------------------------

def random_weights(rng, T, U):
    lp_b = rng.normal(size=(T, U + 1)) - 1.0
    lp_l = rng.normal(size=(T, U + 1)) - 1.0
    lp_l[:, U] = -np.inf
    return lp_b, lp_l


@pytest.mark.parametrize("variant", R.VARIANTS)
def test_grid_equals_alignment_enumeration(variant):
    rng = np.random.default_rng(11)
    for T in range(1, 5):
        for U in range(0, 4):
            lp_b, lp_l = random_weights(rng, T, U)
            _, lnP = R.forward_scores(lp_b, lp_l, variant)
            _, lnP_b = R.backward_scores(lp_b, lp_l, variant)
            bf = BF.brute_force_log_prob(lp_b.tolist(), lp_l.tolist(), variant)
            assert lnP == pytest.approx(bf, abs=1e-12), (T, U)
            assert lnP_b == pytest.approx(bf, abs=1e-12), (T, U)


def test_rnnt_path_count():
    for T in range(1, 5):
        for U in range(0, 4):
            assert BF.count_paths(T, U, "rnnt") == math.comb(T - 1 + U, U)


def wrnnt_path_count(T, U, allow_ignore=False):
    """Paths of the W-lattices counted by (start frame s, frame e where the
    final jump is taken, or e = T-1 for none)."""
    n = 0
    for s in range(T):
        for e in range(s, T):
            n += math.comb(e - s + U, U)
    return n


@pytest.mark.parametrize("variant", ["wrnnt", "wrnnt_allow_ignore"])
def test_wrnnt_path_count(variant):
    for T in range(1, 5):
        for U in range(0, 4):
            assert BF.count_paths(T, U, variant) == wrnnt_path_count(T, U)


# ----------------------------------------------------------------------------
# Closed forms for uniform logits (every arc probability q = 1/V)
# ----------------------------------------------------------------------------

def uniform_loss_rnnt(T, U, V):
    # C(T-1+U, U) alignments, each T blanks and U units of probability 1/V
    return (T + U) * math.log(V) - math.log(math.comb(T - 1 + U, U))


def uniform_loss_wrnnt(T, U, V, allow_ignore=False):
    # start frame s, last grid node (e, U) before the final jump (e = T-1: no jump)
    q = 1.0 / V
    P = 0.0
    for s in range(T):
        for e in range(s, T):
            grid = math.comb(e - s + U, U) * q ** (e - s + U)
            if allow_ignore and e < T - 1:
                P += grid  # jump straight to the final state
            else:
                P += grid * q  # closing blank
    return -math.log(P)


def uniform_loss_wrnnt_by_last_unit(T, U, V):
    """The same total decomposed by the frame e of the last unit emission
    (U >= 1): C(e-s+U-1, U-1) ways to reach it, then k blanks on the top row
    before the jump or the end (a second derivation, not the first re-typed)."""
    q = 1.0 / V
    P = 0.0
    for s in range(T):
        for e in range(s, T):
            tail = sum(q ** k for k in range(T - e))
            P += math.comb(e - s + U - 1, U - 1) * q ** (e - s + U) * tail * q
    return -math.log(P)


def test_uniform_closed_form_values():
    assert uniform_loss_rnnt(4, 2, 4) == pytest.approx(6.015181073725, abs=1e-11)
    assert uniform_loss_rnnt(20, 8, 16) == pytest.approx(63.019432685652, abs=1e-10)
    assert uniform_loss_rnnt(250, 80, 1025) == pytest.approx(2108.184478674, abs=1e-8)
    assert uniform_loss_wrnnt(4, 2, 4) == pytest.approx(2.190896982605, abs=1e-11)
    assert uniform_loss_wrnnt(20, 8, 16) == pytest.approx(21.407178743851, abs=1e-10)
    for T, U, V in [(1, 1, 3), (2, 1, 5), (4, 2, 4), (7, 3, 6), (20, 8, 16)]:
        assert uniform_loss_wrnnt(T, U, V) == pytest.approx(uniform_loss_wrnnt_by_last_unit(T, U, V), rel=1e-13)


@pytest.mark.parametrize("variant", R.VARIANTS)
@pytest.mark.parametrize("T,U,V", [(1, 0, 3), (1, 3, 5), (4, 0, 7), (4, 2, 4), (9, 5, 6), (20, 8, 16)])
def test_uniform_logits_closed_form(variant, T, U, V):
    z = np.zeros((T, U + 1, V))
    labels = np.arange(U) % (V - 1) + 1
    r = R.utterance_loss_grad(z, labels, 0, variant)
    if variant == "rnnt":
        ref = uniform_loss_rnnt(T, U, V)
    else:
        ref = uniform_loss_wrnnt(T, U, V, allow_ignore=(variant == "wrnnt_allow_ignore"))
    assert r["loss"] == pytest.approx(ref, rel=1e-13, abs=1e-13)


def test_uniform_closed_form_at_bpe_shape():
    """T=250, U=80, V=1025 through the recursion on uniform weights."""
    T, U, V = 250, 80, 1025
    lp = np.full((T, U + 1), -math.log(V))
    lp_l = lp.copy()
    lp_l[:, U] = -np.inf
    _, lnP = R.forward_scores(lp, lp_l, "rnnt")
    assert -lnP == pytest.approx(uniform_loss_rnnt(T, U, V), rel=1e-13)
    _, lnPw = R.forward_scores(lp, lp_l, "wrnnt")
    assert -lnPw == pytest.approx(555.928071792, abs=1e-8)
    assert -lnPw == pytest.approx(uniform_loss_wrnnt(T, U, V), rel=1e-12)


# ----------------------------------------------------------------------------
# Special cases that reduce to one alignment
# ----------------------------------------------------------------------------

def test_no_units_is_all_blanks():
    rng = np.random.default_rng(3)
    T, V = 6, 5
    z = rng.normal(size=(T, 1, V))
    r = R.utterance_loss_grad(z, [], 0, "rnnt")
    ls = z - np.log(np.exp(z).sum(-1, keepdims=True))
    assert r["loss"] == pytest.approx(-ls[:, 0, 0].sum(), abs=1e-12)


def test_single_frame_is_all_units_then_blank():
    rng = np.random.default_rng(4)
    U, V = 4, 6
    z = rng.normal(size=(1, U + 1, V))
    labels = [1, 3, 5, 2]
    ls = z - np.log(np.exp(z).sum(-1, keepdims=True))
    ref = -(sum(ls[0, u, labels[u]] for u in range(U)) + ls[0, U, 0])
    for variant in R.VARIANTS:  # no skip arc exists at T = 1
        assert R.utterance_loss_grad(z, labels, 0, variant)["loss"] == pytest.approx(ref, abs=1e-12)


# ----------------------------------------------------------------------------
# Gradient
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("variant", R.VARIANTS)
@pytest.mark.parametrize("T,U,V,blank", [(3, 2, 4, 0), (4, 3, 5, 2), (2, 0, 3, 1), (1, 2, 4, 3)])
def test_gradient_central_differences(variant, T, U, V, blank):
    rng = np.random.default_rng(100 + T * 10 + U)
    z = rng.normal(size=(T, U + 1, V)) * 1.5
    labels = [v for v in rng.permutation([x for x in range(V) if x != blank]).tolist()][:U]
    while len(labels) < U:
        labels.append([x for x in range(V) if x != blank][0])
    g = R.utterance_loss_grad(z, labels, blank, variant)["grad"]
    h = 1e-6
    fd = np.zeros_like(z)
    for idx in itertools.product(range(T), range(U + 1), range(V)):
        zp = z.copy()
        zm = z.copy()
        zp[idx] += h
        zm[idx] -= h
        fd[idx] = (R.utterance_loss_grad(zp, labels, blank, variant, need_grad=False)["loss"]
                   - R.utterance_loss_grad(zm, labels, blank, variant, need_grad=False)["loss"]) / (2 * h)
    np.testing.assert_allclose(g, fd, atol=1e-7)


@pytest.mark.parametrize("variant", R.VARIANTS)
def test_gradient_matches_torch_autograd(variant):
    rng = np.random.default_rng(7)
    T, U, V = 4, 3, 6
    z = rng.normal(size=(T, U + 1, V)) * 2
    labels = [2, 5, 1]
    loss_t, g_t = DAG.torch_autograd_loss_grad(z, labels, 0, variant)
    r = R.utterance_loss_grad(z, labels, 0, variant)
    assert r["loss"] == pytest.approx(loss_t, abs=1e-12)
    np.testing.assert_allclose(r["grad"], g_t, atol=1e-12)


@pytest.mark.parametrize("variant", R.VARIANTS)
def test_posterior_conservation(variant):
    rng = np.random.default_rng(8)
    T, U, V = 12, 5, 9
    z = rng.normal(size=(T, U + 1, V)) * 3
    labels = rng.integers(1, V, size=U)
    r = R.utterance_loss_grad(z, labels, 0, variant)
    # every alignment emits each unit exactly once
    assert r["occ_label"].sum() == pytest.approx(U, abs=1e-10)
    # every gradient row sums to zero over the vocabulary
    np.testing.assert_allclose(r["grad"].sum(-1), 0.0, atol=1e-12)
    assert r["lnP"] == pytest.approx(r["lnP_backward"], abs=1e-12 * max(1, abs(r["lnP"])))
    if variant != "wrnnt_allow_ignore":
        # every alignment ends with the closing blank
        assert r["occ_blank"][T - 1, U] == pytest.approx(1.0, abs=1e-12)
    if variant == "rnnt":
        # exactly T blanks per alignment
        assert r["occ_blank"].sum() == pytest.approx(T, abs=1e-10)
        # each alignment crosses every anti-diagonal t+u = d exactly once
        node = np.exp(r["alpha"] + r["beta"] - r["lnP"])
        for d in range(T + U):
            s = sum(node[t, d - t] for t in range(T) if 0 <= d - t <= U)
            assert s == pytest.approx(1.0, abs=1e-12), d


def test_row_normalizer_matches_scipy():
    from scipy.special import logsumexp
    rng = np.random.default_rng(9)
    z = rng.normal(size=(5, 4, 1025)) * 3
    np.testing.assert_allclose(R.row_log_normalizer(z), logsumexp(z, axis=-1), rtol=0, atol=1e-12)


@pytest.mark.parametrize("variant", R.VARIANTS)
def test_shift_invariance(variant):
    rng = np.random.default_rng(10)
    T, U, V = 5, 3, 7
    z = rng.normal(size=(T, U + 1, V))
    shift = rng.normal(size=(T, U + 1, 1)) * 10
    labels = [3, 1, 6]
    a = R.utterance_loss_grad(z, labels, 0, variant)
    b = R.utterance_loss_grad(z + shift, labels, 0, variant)
    assert a["loss"] == pytest.approx(b["loss"], abs=1e-11)
    np.testing.assert_allclose(a["grad"], b["grad"], atol=1e-12)


@settings(max_examples=60, deadline=None)
@given(T=st.integers(1, 4), U=st.integers(0, 3), V=st.integers(2, 6), blank_pos=st.integers(0, 5),
       variant=st.sampled_from(R.VARIANTS), seed=st.integers(0, 2**31 - 1))
def test_property_three_formulations_agree(T, U, V, blank_pos, variant, seed):
    rng = np.random.default_rng(seed)
    blank = blank_pos % V
    non_blank = [x for x in range(V) if x != blank]
    labels = [non_blank[i] for i in rng.integers(0, len(non_blank), size=U)]
    z = rng.normal(size=(T, U + 1, V)) * 2
    r = R.utterance_loss_grad(z, labels, blank, variant)
    d = DAG.dag_loss_grad(z, labels, blank, variant)
    bf = -BF.brute_force_log_prob(r["lp_blank"].tolist(), r["lp_label"].tolist(), variant)
    assert r["loss"] == pytest.approx(d["loss"], abs=1e-12)
    assert r["loss"] == pytest.approx(bf, abs=1e-12)
    np.testing.assert_allclose(r["grad"], d["grad"], atol=1e-12)


# ----------------------------------------------------------------------------
# Batched wrapper semantics
# ----------------------------------------------------------------------------

def test_batched_padding_and_bad_data():
    rng = np.random.default_rng(12)
    B, T, U, V = 4, 5, 3, 6
    logits = rng.normal(size=(B, T, U + 1, V)).astype(np.float32)
    labels = rng.integers(1, V, size=(B, U)).astype(np.int32)
    tl = np.array([5, 3, 0, 4], np.int32)      # utterance 2: T_b = 0 is bad data
    ul = np.array([3, 1, 2, 2], np.int32)
    labels[3, 1] = 0                           # utterance 3: a label equal to blank
    logits[1, 3:] = np.nan                     # padding of utterance 1 must not matter
    logits[1, :, 2:] = np.nan
    loss, grad = R.rnnt_loss_grad(logits, labels, tl, ul, 0, "rnnt")
    assert np.isfinite(loss[0]) and np.isfinite(loss[1])
    assert np.isnan(loss[2]) and np.isnan(loss[3])
    assert np.all(grad[2] == 0) and np.all(grad[3] == 0)
    assert np.all(grad[1, 3:] == 0) and np.all(grad[1, :, 2:] == 0)
    one = R.utterance_loss_grad(logits[1, :3, :2].astype(np.float64), labels[1, :1], 0, "rnnt")
    assert loss[1] == pytest.approx(one["loss"], abs=0)
