"""Explicit arc-list formulation of the same lattices (float64, CPU).

TEST INFRASTRUCTURE ONLY -- the product path never imports this module.

Section 2 (Eq. 1) defines the loss as the negative forward score of a lattice
WFST; Section 2.2 builds that lattice by composition and then populates its arcs
by indexed selection from X using each arc's (time, unit_idx, label).  This
module follows that view: it lists every arc of the lattice explicitly, each
with its source, destination, label kind and (time, unit_idx), populates the
weights from log_softmax(logits) (scipy's routine), and runs a generic
topological-order forward/backward over the arc list.  It shares no code with
``rnnt_ref`` (different formulation, different helpers) so that agreement
between the two pins the grid recursion's indexing.

Arc sets (Fig. 1 for RNN-T; Fig. 4 and Section 3.2 for the W-Transducer;
Section 4.3 for the allow-ignore variant) are described in ``grid_arcs``.
"""
import numpy as np
from scipy.special import log_softmax, logsumexp

FINAL = "final"


def grid_arcs(T, U, variant="rnnt"):
    """Arc list of the lattice for T frames and U units.

    Each arc is (src, dst, kind, t, u) with kind in {"blank", "label", "skip"};
    nodes are (t, u) tuples plus FINAL; (t, u) of an arc is its source node
    (the "time:unit_idx" labels of Fig. 4).  Skip arcs carry probability one.
    """
    arcs = []
    for t in range(T):
        for u in range(U + 1):
            if t < T - 1:
                arcs.append(((t, u), (t + 1, u), "blank", t, u))
            if u < U:
                arcs.append(((t, u), (t, u + 1), "label", t, u))
    arcs.append(((T - 1, U), FINAL, "blank", T - 1, U))
    if variant in ("wrnnt", "wrnnt_allow_ignore"):
        for t in range(1, T):
            arcs.append(((0, 0), (t, 0), "skip", 0, 0))
        for t in range(T - 1):
            dst = (T - 1, U) if variant == "wrnnt" else FINAL
            arcs.append(((t, U), dst, "skip", t, U))
    return arcs


def topological_nodes(T, U):
    """Nodes ordered by t+u (every arc, skip arcs included, increases t+u)."""
    nodes = sorted(((t, u) for t in range(T) for u in range(U + 1)), key=lambda n: (n[0] + n[1], n[1]))
    return nodes + [FINAL]


def populate(arcs, logp, labels, blank):
    """Arc weights by indexed selection from logp (T, U+1, V) (Section 2.2 Populate)."""
    w = np.empty(len(arcs))
    for i, (_, _, kind, t, u) in enumerate(arcs):
        if kind == "blank":
            w[i] = logp[t, u, blank]
        elif kind == "label":
            w[i] = logp[t, u, int(labels[u])]
        else:
            w[i] = 0.0
    return w


def dag_forward_backward(nodes, arcs, weights, start):
    """Generic log-semiring forward/backward over an arc list.

    Returns (fwd dict, bwd dict, lnP, arc posteriors array).  Parallel arcs are
    separate list entries and are summed.
    """
    incoming = {n: [] for n in nodes}
    outgoing = {n: [] for n in nodes}
    for i, (s, d, *_rest) in enumerate(arcs):
        incoming[d].append(i)
        outgoing[s].append(i)
    fwd = {}
    for n in nodes:
        if n == start:
            fwd[n] = 0.0
            continue
        terms = [fwd[arcs[i][0]] + weights[i] for i in incoming[n]]
        fwd[n] = logsumexp(terms) if terms else -np.inf
    bwd = {}
    for n in reversed(nodes):
        if n == FINAL:
            bwd[n] = 0.0
            continue
        terms = [weights[i] + bwd[arcs[i][1]] for i in outgoing[n]]
        bwd[n] = logsumexp(terms) if terms else -np.inf
    lnP = fwd[FINAL]
    post = np.array([np.exp(fwd[s] + weights[i] + bwd[d] - lnP) for i, (s, d, *_r) in enumerate(arcs)])
    return fwd, bwd, lnP, post


def dag_loss_grad(z, labels, blank=0, variant="rnnt"):
    """Loss and gradient of one utterance through the arc-list view.

    z: (T, U+1, V) logits.  The gradient is assembled from arc posteriors:
    each blank/label arc with posterior g contributes g * (softmax - onehot) to
    the row of its source node (the derivative of -log_softmax).
    """
    z = np.asarray(z, dtype=np.float64)
    T, U1, V = z.shape
    U = U1 - 1
    logp = log_softmax(z, axis=-1)
    arcs = grid_arcs(T, U, variant)
    nodes = topological_nodes(T, U)
    w = populate(arcs, logp, labels, blank)
    fwd, bwd, lnP, post = dag_forward_backward(nodes, arcs, w, (0, 0))
    p = np.exp(logp)
    grad = np.zeros_like(z)
    for i, (_, _, kind, t, u) in enumerate(arcs):
        if kind == "skip":
            continue
        v = blank if kind == "blank" else int(labels[u])
        grad[t, u, :] += post[i] * p[t, u, :]
        grad[t, u, v] -= post[i]
    return dict(loss=-lnP, lnP=lnP, fwd=fwd, bwd=bwd, arcs=arcs, posteriors=post, grad=grad)


def torch_autograd_loss_grad(z, labels, blank=0, variant="rnnt"):
    """Loss and gradient by float64 autograd through the arc-list forward pass.

    Uses torch's log_softmax / logsumexp and reverse-mode autograd: a gradient
    obtained with no posterior formula at all.
    """
    import torch

    zt = torch.tensor(np.asarray(z, dtype=np.float64), requires_grad=True)
    T, U1, V = zt.shape
    U = U1 - 1
    logp = torch.log_softmax(zt, dim=-1)
    arcs = grid_arcs(T, U, variant)
    nodes = topological_nodes(T, U)
    incoming = {n: [] for n in nodes}
    for a in arcs:
        incoming[a[1]].append(a)
    fwd = {}
    zero = torch.zeros((), dtype=torch.float64)
    for n in nodes:
        if n == (0, 0):
            fwd[n] = zero
            continue
        terms = []
        for (s, _d, kind, t, u) in incoming[n]:
            if kind == "blank":
                w = logp[t, u, blank]
            elif kind == "label":
                w = logp[t, u, int(labels[u])]
            else:
                w = zero
            terms.append(fwd[s] + w)
        fwd[n] = torch.logsumexp(torch.stack(terms), dim=0)
    loss = -fwd[FINAL]
    loss.backward()
    return float(loss.detach()), zt.grad.numpy().copy()
