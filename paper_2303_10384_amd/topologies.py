"""Lattices as arc lists, the input of rnnt_arc_plan (no loss arithmetic here).

An arc is a record (src, dst, t, u, label, score) in ARC_DTYPE, the layout of
rnnt_arc_t: it leaves state src for state dst and weighs score plus, when
label >= 0, the log-probability of `label` in logits row (t, u).  Per utterance,
states are 0 .. n-1, 0 the start and n-1 the final state, and every arc goes
from a lower to a higher state (Section 2.2 builds the training lattice as such
a graph and fills in its weights by indexed selection).

grid_lattice lists the lattice of Fig. 1 (Section 2.3) and its W-Transducer
forms (Fig. 4 / Section 3.2 force-final, Section 4.3 allow-ignore): node (t, u)
is state t*(U+1)+u and the final state is T*(U+1).
"""
import numpy as np

ARC_DTYPE = np.dtype([("src", "<i4"), ("dst", "<i4"), ("t", "<i4"), ("u", "<i4"), ("label", "<i4"),
                      ("score", "<f4")])

VARIANTS = ("rnnt", "wrnnt", "wrnnt_allow_ignore")


def _arcs(src, dst, t, u, label):
    a = np.zeros(len(src), ARC_DTYPE)
    a["src"], a["dst"], a["t"], a["u"], a["label"] = src, dst, t, u, label
    return a


def grid_lattice(T, U, labels, blank=0, variant="rnnt"):
    """(n_states, arcs) of one utterance with T frames and units labels[:U].

    Blank arcs (t, u) -> (t+1, u) for t < T-1; label arcs (t, u) -> (t, u+1)
    carrying labels[u] for u < U; the closing blank (T-1, U) -> final.  The
    W-Transducer adds score-0 arcs that read no logits: (0, 0) -> (t, 0) for
    1 <= t <= T-1, and (t, U) -> (T-1, U) for t <= T-2 (force-final) or
    (t, U) -> final (allow-ignore).
    """
    if variant not in VARIANTS:
        raise ValueError("variant must be one of %s" % (VARIANTS,))
    T, U = int(T), int(U)
    U1 = U + 1
    final = T * U1
    labels = np.asarray(labels, dtype=np.int32)[:U]
    parts = []
    tb, ub = np.meshgrid(np.arange(T - 1), np.arange(U1), indexing="ij")
    tb, ub = tb.ravel(), ub.ravel()
    parts.append(_arcs(tb * U1 + ub, (tb + 1) * U1 + ub, tb, ub, blank))
    tl, ul = np.meshgrid(np.arange(T), np.arange(U), indexing="ij")
    tl, ul = tl.ravel(), ul.ravel()
    parts.append(_arcs(tl * U1 + ul, tl * U1 + ul + 1, tl, ul, labels[ul] if U else np.zeros(0, np.int32)))
    parts.append(_arcs([(T - 1) * U1 + U], [final], [T - 1], [U], [blank]))
    if variant != "rnnt":
        ts = np.arange(1, T)
        parts.append(_arcs(np.zeros(len(ts), np.int32), ts * U1, 0, 0, -1))
        tf = np.arange(T - 1)
        dst = (T - 1) * U1 + U if variant == "wrnnt" else final
        parts.append(_arcs(tf * U1 + U, np.full(len(tf), dst), 0, 0, -1))
    return final + 1, np.concatenate(parts)


def batch_grid_lattices(logit_lens, label_lens, labels, blank=0, variant="rnnt"):
    """grid_lattice for every utterance of a batch (host arrays of lengths and labels)."""
    logit_lens = np.asarray(logit_lens)
    label_lens = np.asarray(label_lens)
    labels = np.asarray(labels)
    return [grid_lattice(int(logit_lens[b]), int(label_lens[b]), labels[b], blank, variant)
            for b in range(len(logit_lens))]
