"""Pins of the arc-list oracle (oracle/arc_lattice.py), CPU only.

The arc-list forward-backward is pinned by:
* enumeration of every start -> final path of small random lattices
  (brute_force.graph_paths: a depth-first walk, no recursion over states),
  for the loss and for each arc's posterior;
* the lattices transcribed from Fig. 1 and Fig. 4 (arc weights as printed),
  whose path sums are the stored figure values;
* the grid recursion of rnnt_ref (itself pinned to the figures and closed
  forms) on the lattices of all three variants, listed arc by arc;
* float64 reverse-mode autograd through the forward recursion alone;
* special cases: one path, no path, duplicated arcs, one state;
* planted mistakes, each of which one of the pins above must catch.
"""
import json
import math
import os
import types

import numpy as np
import pytest
from scipy.special import log_softmax

from figures import allow_ignore_from_fig4, load_figure
from oracle import arc_lattice as AL
from oracle import brute_force as BF
from oracle import lattice_dag as LD
from oracle import rnnt_ref as R
from paper_2303_10384_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
EXPECTED = json.load(open(os.path.join(HERE, "golden", "fig_expected.json")))


def as_tuples(arcs):
    return [(int(a["src"]), int(a["dst"]), int(a["t"]), int(a["u"]), int(a["label"]), float(a["score"]))
            for a in arcs]


def random_case(seed, T=3, U=2, V=5, n_states=7, n_arcs=14):
    rng = np.random.default_rng(seed)
    n, arcs = W.random_arc_lattice(rng, T, U, V, n_states, n_arcs, eps_frac=0.25, long_frac=0.3)
    z = rng.standard_normal((T, U + 1, V)) * 1.5
    return z, n, as_tuples(arcs)


def test_populate_matches_torch_log_softmax():
    import torch
    z, n, arcs = random_case(1)
    w = AL.arc_weights(z, arcs)
    logp = torch.log_softmax(torch.tensor(z), dim=-1).numpy()
    for wi, (_s, _d, t, u, label, score) in zip(w, arcs):
        expect = score + (logp[t, u, label] if label >= 0 else 0.0)
        assert abs(wi - expect) <= 1e-12


@pytest.mark.parametrize("seed", range(12))
def test_loss_and_posteriors_match_path_enumeration(seed):
    z, n, arcs = random_case(seed)
    w = AL.arc_weights(z, arcs)
    graph = [(s, d, wi) for (s, d, *_r), wi in zip(arcs, w)]
    lnP, n_paths = BF.graph_paths_log_prob(graph, 0, n - 1)
    r = AL.arc_lattice_loss_grad(z, arcs, n)
    assert abs(r["loss"] + lnP) <= 1e-10 * max(1.0, abs(lnP))
    post = BF.graph_arc_posteriors(graph, 0, n - 1)
    np.testing.assert_allclose(r["posteriors"], post, rtol=0, atol=1e-12)


def figure_arc_list(fig):
    """The figure graph as an arc list with weights as scores (label -1: no logits),
    states renumbered in (t + u, u) order with the final state last."""
    order = sorted(fig["nodes"], key=lambda s: (sum(fig["nodes"][s]), fig["nodes"][s][1]))
    new = {s: i for i, s in enumerate(order)}
    new[fig["final"]] = len(order)
    arcs = [(new[s], new[d], 0, 0, -1, w) for (s, d, _sym, w) in fig["arcs"]]
    return len(order) + 1, arcs


@pytest.mark.parametrize("key,loader", [
    ("rnnt_fig1", lambda: load_figure("fig1_rnnt_lattice.txt")),
    ("wrnnt_fig4", lambda: load_figure("fig4_wrnnt_lattice.txt")),
    ("wrnnt_allow_ignore_fig4_redirected", lambda: allow_ignore_from_fig4(load_figure("fig4_wrnnt_lattice.txt"))),
])
def test_printed_lattices(key, loader):
    fig = loader()
    n, arcs = figure_arc_list(fig)
    z = np.zeros((1, 1, 2))
    r = AL.arc_lattice_loss_grad(z, arcs, n)
    assert abs(r["loss"] - EXPECTED[key]["loss"]) <= 1e-9
    if key == "rnnt_fig1":
        assert abs(r["loss"] - 4.2574511041) <= 1e-9  # the value stated for Fig. 1's weights


def grid_as_arc_list(T, U, labels, blank, variant):
    """lattice_dag.grid_arcs (the oracle's own listing of Fig. 1 / Fig. 4 arcs) in the
    arc-list form: states numbered t*(U+1)+u, the final state last."""
    def sid(n):
        return T * (U + 1) if n == LD.FINAL else n[0] * (U + 1) + n[1]
    arcs = []
    for (s, d, kind, t, u) in LD.grid_arcs(T, U, variant):
        label = blank if kind == "blank" else (int(labels[u]) if kind == "label" else -1)
        arcs.append((sid(s), sid(d), t, u, label, 0.0))
    return T * (U + 1) + 1, arcs


@pytest.mark.parametrize("variant", R.VARIANTS)
@pytest.mark.parametrize("T,U", [(1, 0), (1, 3), (4, 0), (4, 2), (7, 5)])
def test_grid_lattices_match_the_grid_recursion(variant, T, U):
    rng = np.random.default_rng(10 * T + U)
    V, blank = 6, 2
    z = rng.standard_normal((T, U + 1, V)) * 2
    labels = rng.choice([v for v in range(V) if v != blank], size=U)
    n, arcs = grid_as_arc_list(T, U, labels, blank, variant)
    r = AL.arc_lattice_loss_grad(z, arcs, n)
    g = R.utterance_loss_grad(z, labels, blank, variant)
    assert abs(r["loss"] - g["loss"]) <= 1e-10 * max(1.0, abs(g["loss"]))
    np.testing.assert_allclose(r["grad"], g["grad"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_gradient_matches_autograd(seed):
    z, n, arcs = random_case(100 + seed, T=3, U=2, V=6, n_states=9, n_arcs=20)
    r = AL.arc_lattice_loss_grad(z, arcs, n)
    loss, grad = AL.torch_autograd_loss_grad(z, arcs, n)
    assert abs(r["loss"] - loss) <= 1e-10 * max(1.0, abs(loss))
    np.testing.assert_allclose(r["grad"], grad, rtol=0, atol=1e-12)


def test_single_path_and_shift_invariance():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((3, 2, 5))
    arcs = [(0, 1, 0, 0, 3, 0.25), (1, 2, 1, 1, 0, 0.0), (2, 3, 2, 0, -1, -0.5)]
    r = AL.arc_lattice_loss_grad(z, arcs, 4)
    lp = log_softmax(z, axis=-1)
    assert abs(r["loss"] - -(lp[0, 0, 3] + 0.25 + lp[1, 1, 0] - 0.5)) <= 1e-12
    np.testing.assert_allclose(r["posteriors"], [1.0, 1.0, 1.0], atol=1e-14)
    r2 = AL.arc_lattice_loss_grad(z + rng.standard_normal((3, 2, 1)), arcs, 4)
    assert abs(r2["loss"] - r["loss"]) <= 1e-12
    np.testing.assert_allclose(r2["grad"], r["grad"], atol=1e-12)


def test_no_path_one_state_and_parallel_arcs():
    z = np.random.default_rng(5).standard_normal((2, 2, 4))
    r = AL.arc_lattice_loss_grad(z, [(0, 1, 0, 0, 1, 0.0), (2, 3, 1, 1, 2, 0.0)], 4)  # final unreachable
    assert r["loss"] == math.inf and not r["grad"].any()
    r = AL.arc_lattice_loss_grad(z, [], 1)  # start is final: the empty path, probability 1
    assert r["loss"] == 0.0 and not r["grad"].any()
    one = [(0, 1, 0, 0, 1, 0.0), (1, 2, 1, 0, 3, 0.0)]
    two = one + [(0, 1, 0, 0, 1, 0.0)]  # the first arc doubled: twice the probability
    a = AL.arc_lattice_loss_grad(z, one, 3)["loss"]
    b = AL.arc_lattice_loss_grad(z, two, 3)["loss"]
    assert abs(a - b - math.log(2.0)) <= 1e-12


def test_batch_validity_rules():
    rng = np.random.default_rng(6)
    logits = rng.standard_normal((3, 4, 3, 5))
    lat = [(3, [(0, 1, 3, 2, 1, 0.0), (1, 2, 0, 0, -1, 0.0)])] * 3
    loss, grad = AL.batch_loss_grad(logits, np.array([4, 3, 4]), np.array([2, 2, 1]), lat)
    assert np.isfinite(loss[0]) and np.isnan(loss[1]) and np.isnan(loss[2])  # t = 3 / u = 2 outside
    assert not grad[1:].any()
    assert grad[0, 3, 2].any() and not grad[0, :3].any()


# planted mistakes in the oracle must fail the pins above
MUTATIONS = {
    "max_instead_of_sum": ("alpha[n] = logsumexp([alpha[arcs[i][0]] + w[i] for i in incoming[n]])",
                           "alpha[n] = max([alpha[arcs[i][0]] + w[i] for i in incoming[n]])"),
    "posterior_wrong_beta": ("math.exp(alpha[s] + w[i] + beta[d] - lnP)", "math.exp(alpha[s] + w[i] + beta[s] - lnP)"),
    "gradient_without_softmax": ("grad[t, u, :] += g * p[t, u, :]", "pass"),
    "epsilon_reads_logits": ("(logp[t, u, label] if label >= 0 else 0.0)", "logp[t, u, label]"),
    "score_sign": ("w[i] = float(score) +", "w[i] = -float(score) +"),
    "backward_skips_start": ("for n in range(n_states - 2, -1, -1):", "for n in range(n_states - 2, 0, -1):"),
    "backward_skips_next_to_final": ("for n in range(n_states - 2, -1, -1):", "for n in range(n_states - 3, -1, -1):"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutants_are_caught(name, monkeypatch):
    src = open(AL.__file__).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, name
    mod = types.ModuleType("arc_lattice_mutant")
    mod.__dict__["__package__"] = "oracle"
    exec(compile(src.replace(old, new), AL.__file__ + ":" + name, "exec"), mod.__dict__)
    for fn in ("arc_weights", "forward_backward", "arc_posteriors", "arc_lattice_loss_grad"):
        monkeypatch.setattr(AL, fn, getattr(mod, fn))
    checks = [lambda: test_loss_and_posteriors_match_path_enumeration(3),
              lambda: test_grid_lattices_match_the_grid_recursion("wrnnt", 4, 2),
              lambda: test_gradient_matches_autograd(1),
              lambda: test_single_path_and_shift_invariance()]
    caught = False
    for check in checks:
        try:
            check()
        except AssertionError:
            caught = True
            break
    assert caught, name
