"""Loss and gradient of a lattice given as a plain list of arcs (float64, CPU).

TEST INFRASTRUCTURE ONLY -- the product path never imports this module.

Section 2.2 builds the training lattice as a graph whose arcs each carry a time
index, a unit index and an input label, and fills in every arc's weight by
indexed selection from the log-probabilities (Populate); the loss is the
negative forward score of that lattice (Eq. 1), and the gradients follow from
its forward and backward scores.  Nothing in that recipe depends on the grid
shape of Fig. 1: any acyclic lattice over the same (T, U+1, V) tensor works,
which is how a new loss such as the W-Transducer (Section 3) is obtained by
changing the graph alone.

This module is that recipe for an arbitrary list of arcs of one utterance:
    arc = (src, dst, t, u, label, score)
    weight = score + log_softmax(z[t, u])[label]   if label >= 0
           = score                                  if label == -1 (reads no logits)
States are 0 .. n-1; state 0 is the start and state n-1 the final state; every
arc goes from a lower to a higher state number, so loops in state order are the
forward and backward recursions.  Parallel arcs are separate entries and their
probabilities add.

    loss = -ln (sum over start -> final paths of exp(sum of the path's weights))
    d loss / d z[t, u, :] = sum over arcs a reading row (t, u) of
                            g_a * (softmax(z[t, u]) - onehot(label_a)),
where g_a is the arc's posterior (the share of the path probability through a).
When no path reaches the final state the loss is +inf and the gradient 0.
"""
import math

import numpy as np
from scipy.special import log_softmax, logsumexp

NEG_INF = -math.inf


def check_arcs(arcs, n_states):
    """Raise ValueError unless the arcs fit the numbering rules above."""
    if n_states < 1:
        raise ValueError("a lattice needs at least one state")
    for (s, d, t, u, label, score) in arcs:
        if not (0 <= s < d < n_states):
            raise ValueError(f"arc {s}->{d} does not go from a lower to a higher state")
        if label < -1:
            raise ValueError(f"bad label {label}")


def arc_weights(z, arcs):
    """Populate: each arc's weight from log_softmax of its row (scipy's routine)."""
    z = np.asarray(z, dtype=np.float64)
    logp = log_softmax(z, axis=-1) if z.size else z
    w = np.empty(len(arcs))
    for i, (_s, _d, t, u, label, score) in enumerate(arcs):
        w[i] = float(score) + (logp[t, u, label] if label >= 0 else 0.0)
    return w


def forward_backward(n_states, arcs, w):
    """alpha, beta (length n_states) and ln P by loops in state order."""
    incoming = [[] for _ in range(n_states)]
    outgoing = [[] for _ in range(n_states)]
    for i, (s, d, *_rest) in enumerate(arcs):
        incoming[d].append(i)
        outgoing[s].append(i)
    alpha = np.full(n_states, NEG_INF)
    alpha[0] = 0.0
    for n in range(1, n_states):
        if incoming[n]:
            alpha[n] = logsumexp([alpha[arcs[i][0]] + w[i] for i in incoming[n]])
    beta = np.full(n_states, NEG_INF)
    beta[n_states - 1] = 0.0
    for n in range(n_states - 2, -1, -1):
        if outgoing[n]:
            beta[n] = logsumexp([w[i] + beta[arcs[i][1]] for i in outgoing[n]])
    lnP = float(alpha[n_states - 1])
    # both recursions sum the same paths
    assert (lnP == NEG_INF and beta[0] == NEG_INF) or abs(beta[0] - lnP) <= 1e-9 * max(1.0, abs(lnP)), (beta[0], lnP)
    return alpha, beta, lnP


def arc_posteriors(alpha, beta, arcs, w, lnP):
    """exp(alpha(src) + w + beta(dst) - ln P) per arc (0 for every arc when ln P = -inf)."""
    if lnP == NEG_INF:
        return np.zeros(len(arcs))
    return np.array([math.exp(alpha[s] + w[i] + beta[d] - lnP) if alpha[s] > NEG_INF and beta[d] > NEG_INF else 0.0
                     for i, (s, d, *_r) in enumerate(arcs)])


def arc_lattice_loss_grad(z, arcs, n_states, need_grad=True):
    """Loss (and gradient w.r.t. z, shape of z) of one utterance's lattice."""
    check_arcs(arcs, n_states)
    z = np.asarray(z, dtype=np.float64)
    w = arc_weights(z, arcs)
    alpha, beta, lnP = forward_backward(n_states, arcs, w)
    post = arc_posteriors(alpha, beta, arcs, w, lnP)
    out = dict(loss=-lnP, lnP=lnP, alpha=alpha, beta=beta, weights=w, posteriors=post)
    if need_grad:
        grad = np.zeros_like(z)
        if z.size:
            p = np.exp(log_softmax(z, axis=-1))
            for g, (_s, _d, t, u, label, _score) in zip(post, arcs):
                if label < 0 or g == 0.0:
                    continue
                grad[t, u, :] += g * p[t, u, :]
                grad[t, u, label] -= g
        out["grad"] = grad
    return out


def utterance_is_valid(T_b, U_b, arcs, T_max, U_max, V):
    """Data checks the device can only make at run time: the lengths, and every
    arc that reads logits reads a row of the utterance's valid region."""
    if not (1 <= T_b <= T_max and 0 <= U_b <= U_max):
        return False
    for (_s, _d, t, u, label, _score) in arcs:
        if label >= 0 and not (0 <= t < T_b and 0 <= u <= U_b and label < V):
            return False
    return True


def batch_loss_grad(logits, logit_lens, label_lens, lattices, need_grad=True):
    """Per-utterance losses and the full gradient tensor of a batch.

    logits: (B, T_max, U_max+1, V); lattices: list of (n_states, arcs) per
    utterance.  Rows outside (t < T_b, u <= U_b) get a zero gradient; an
    utterance that fails `utterance_is_valid` gets loss NaN and a zero gradient.
    """
    logits = np.asarray(logits)
    B, T_max, U1, V = logits.shape
    loss = np.full(B, np.nan)
    grad = np.zeros(logits.shape) if need_grad else None
    for b, (n_states, arcs) in enumerate(lattices):
        T_b, U_b = int(logit_lens[b]), int(label_lens[b])
        if not utterance_is_valid(T_b, U_b, arcs, T_max, U1 - 1, V):
            continue
        r = arc_lattice_loss_grad(logits[b, :T_b, :U_b + 1].astype(np.float64), arcs, n_states, need_grad)
        loss[b] = r["loss"]
        if need_grad:
            grad[b, :T_b, :U_b + 1] = r["grad"]
    return loss, grad


def torch_autograd_loss_grad(z, arcs, n_states):
    """Loss and gradient by float64 reverse-mode autograd through the forward
    recursion alone (torch's log_softmax / logsumexp): a gradient obtained with
    no posterior formula."""
    import torch

    zt = torch.tensor(np.asarray(z, dtype=np.float64), requires_grad=True)
    logp = torch.log_softmax(zt, dim=-1)
    incoming = [[] for _ in range(n_states)]
    for a in arcs:
        incoming[a[1]].append(a)
    alpha = [None] * n_states
    alpha[0] = torch.zeros((), dtype=torch.float64)
    for n in range(1, n_states):
        terms = []
        for (s, _d, t, u, label, score) in incoming[n]:
            if alpha[s] is None:
                continue
            wt = logp[t, u, label] + float(score) if label >= 0 else torch.tensor(float(score), dtype=torch.float64)
            terms.append(alpha[s] + wt)
        alpha[n] = torch.logsumexp(torch.stack(terms), dim=0) if terms else None
    if alpha[n_states - 1] is None:
        return math.inf, np.zeros(zt.shape)
    loss = -alpha[n_states - 1]
    loss.backward()
    return float(loss.detach()), zt.grad.numpy().copy()
