"""Planted mistakes in the oracle must be caught by its pins.

Each case copies the oracle's source, plants one plausible mistake (a dropped
term, a wrong index, a flipped sign), loads the result as a throw-away module
and runs a small battery of the pins from test_oracle_pins against it.  The
battery must fail for every mutant.  Everything runs on the CPU.
"""
import itertools
import math
import os
import types

import numpy as np
import pytest

from figures import allow_ignore_from_fig4, grid_weights, load_figure
from oracle import brute_force as BF

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "rnnt_ref.py")

MUTATIONS = {
    "drop_initial_skip_fwd": ("acc = log_add(acc, alpha[0, 0])", "pass"),
    "drop_final_skips_fwd": ("for tp in range(T - 1):\n                    acc = log_add(acc, alpha[tp, U])",
                             "for tp in range(T - 2):\n                    acc = log_add(acc, alpha[tp, U])"),
    "blank_weight_wrong_frame": ("alpha[t - 1, u] + lp_blank[t - 1, u]", "alpha[t - 1, u] + lp_blank[t, u]"),
    "label_weight_wrong_unit": ("alpha[t, u - 1] + lp_label[t, u - 1]", "alpha[t, u - 1] + lp_label[t - 1, u - 1]"),
    "drop_closing_blank": ("lnP = alpha[T - 1, U] + lp_blank[T - 1, U]  # closing blank",
                           "lnP = alpha[T - 1, U]"),
    "backward_skip_range": ("for tp in range(1, T):", "for tp in range(2, T):"),
    "backward_final_skip_target": ("acc = log_add(acc, beta[T - 1, U])", "acc = log_add(acc, beta[T - 1, U - 1])"),
    "label_index_shift": ("z[:, u, int(labels[u])] - lse[:, u]", "z[:, u, int(labels[u - 1])] - lse[:, u]"),
    "lse_drops_max": ("(m + np.log(np.exp(z - m)", "(np.log(np.exp(z - m)"),
    "grad_blank_sign": ("grad[:, :, blank] -= occ_blank", "grad[:, :, blank] += occ_blank"),
    "grad_softmax_unshifted": ("softmax = np.exp(z - lse[:, :, None])", "softmax = np.exp(z)"),
    "posterior_wrong_beta": ("occ_blank[t, u] = math.exp(alpha[t, u] + lp_blank[t, u] + beta[t + 1, u] - lnP)",
                             "occ_blank[t, u] = math.exp(alpha[t, u] + lp_blank[t, u] + beta[t, u] - lnP)"),
    "label_posterior_wrong_beta": ("lp_label[t, u] + beta[t, u + 1] - lnP", "lp_label[t, u] + beta[t, u] - lnP"),
    "grad_label_row": ("grad[:, u, int(labels[u])] -= occ_label[:, u]", "grad[:, u, int(labels[u])] -= occ_blank[:, u]"),
    "log_add_sign": ("return a + math.log1p(math.exp(b - a))", "return a + math.log1p(math.exp(a - b))"),
}


def load_mutant(name):
    src = open(SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, name
    mod = types.ModuleType("rnnt_ref_mutant_" + name)
    exec(compile(src.replace(old, new), SRC + ":" + name, "exec"), mod.__dict__)
    return mod


def battery(R):
    """Raises AssertionError (or any error) if a pin fails."""
    # printed lattices
    for variant, fig, ref in [
        ("rnnt", load_figure("fig1_rnnt_lattice.txt"), 4.2574511041),
        ("wrnnt", load_figure("fig4_wrnnt_lattice.txt"), 2.2070452674),
        ("wrnnt_allow_ignore", allow_ignore_from_fig4(load_figure("fig4_wrnnt_lattice.txt")), 1.9385100266),
    ]:
        lp_b, lp_l = map(np.array, grid_weights(fig))
        alpha, lnP = R.forward_scores(lp_b, lp_l, variant)
        beta, lnP_b = R.backward_scores(lp_b, lp_l, variant)
        assert abs(-lnP - ref) < 1e-9 and abs(-lnP_b - ref) < 1e-9
    # enumeration and finite differences on a tiny logits case, every variant
    rng = np.random.default_rng(5)
    T, U, V = 3, 2, 4
    z = rng.normal(size=(T, U + 1, V))
    labels = [2, 3]
    for variant in ("rnnt", "wrnnt", "wrnnt_allow_ignore"):
        r = R.utterance_loss_grad(z, labels, 0, variant)
        ls = z - np.log(np.exp(z).sum(-1, keepdims=True))
        lp_b = ls[:, :, 0]
        lp_l = np.full((T, U + 1), -np.inf)
        for u in range(U):
            lp_l[:, u] = ls[:, u, labels[u]]
        bf = BF.brute_force_log_prob(lp_b.tolist(), lp_l.tolist(), variant)
        assert abs(r["loss"] + bf) < 1e-10
        h = 1e-6
        for idx in itertools.product(range(T), range(U + 1), range(V)):
            zp, zm = z.copy(), z.copy()
            zp[idx] += h
            zm[idx] -= h
            fd = (R.utterance_loss_grad(zp, labels, 0, variant, False)["loss"]
                  - R.utterance_loss_grad(zm, labels, 0, variant, False)["loss"]) / (2 * h)
            assert abs(fd - r["grad"][idx]) < 1e-6
    # uniform closed form
    T, U, V = 6, 3, 5
    r = R.utterance_loss_grad(np.zeros((T, U + 1, V)), [1, 2, 3], 0, "rnnt", False)
    assert abs(r["loss"] - ((T + U) * math.log(V) - math.log(math.comb(T - 1 + U, U)))) < 1e-12


def test_battery_passes_on_the_oracle():
    from oracle import rnnt_ref
    battery(rnnt_ref)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name):
    mutant = load_mutant(name)
    with pytest.raises(Exception):
        battery(mutant)
