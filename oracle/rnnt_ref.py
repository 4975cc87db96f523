"""Grid-lattice oracle for the RNN-T and W-Transducer losses (float64, CPU).

TEST INFRASTRUCTURE ONLY -- the product path never imports this module.

What is computed (paper: "Powerful and Extensible WFST Framework for
RNN-Transducer Losses", Laptev et al., ICASSP 2023):

* Eq. 1: the loss is the negative forward score of the training lattice,
  ``loss = -Fwd(L)``, i.e. ``-ln P(Y|X)`` summed over all alignments.
* The lattice populates its arcs from a log-probability tensor X of shape
  (T, U+1, V) (Section 2, Eq. 1 text; Populate in Section 2.2).  The API takes
  raw joint logits, so X = log_softmax(logits) over V.
* Fig. 1 / Section 2.3 (Grid-Transducer): node (t, u) for t in [0, T),
  u in [0, U].  A blank arc leaves (t, u) to (t+1, u) for t < T-1; a label arc
  leaves (t, u) to (t, u+1) for u < U carrying unit y_{u+1}; one final blank arc
  leaves (T-1, U) to the final state.  No blank arc leaves (T-1, u < U) (the
  figure draws none).  An arc's time and unit index are those of its source
  node (arc labels "time:unit_idx" in Fig. 3 and Fig. 4).
* Section 3.2 / Fig. 4 (W-Transducer, "force-final"): epsilon arcs of
  probability one from the initial node (0, 0) to every (t, 0), t = 1..T-1, and
  from every (t, U), t = 0..T-2, to the previous-to-final node (T-1, U); the
  closing blank is still required.  Parallel arcs are summed.
* Section 4.3 ("W-RNNT-allow-ignore"): the final epsilon arcs from (t, U),
  t = 0..T-2, go to the final state instead, so the closing blank is optional.

Algorithm: plain t-outer / u-inner forward recursion and the reversed backward
recursion in the log semiring, arc posteriors from alpha + arc weight + beta,
then the chain rule through log_softmax.  No blocking, no diagonal schedule.
"""
import math

import numpy as np

NEG_INF = -math.inf

VARIANTS = ("rnnt", "wrnnt", "wrnnt_allow_ignore")


def log_add(a, b):
    """ln(e^a + e^b) in float64; two -inf operands give -inf, never NaN."""
    if a == NEG_INF:
        return b
    if b == NEG_INF:
        return a
    if a < b:
        a, b = b, a
    return a + math.log1p(math.exp(b - a))


def row_log_normalizer(z):
    """lse over the last axis (the vocabulary), max-shifted, float64."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))[..., 0]


def lattice_weights(z, labels, blank):
    """Populate the grid (Section 2.2 Populate; Fig. 1 arc weights).

    z: (T, U+1, V) logits of ONE utterance (already cut to its lengths).
    labels: (U,) target units y_1..y_U.
    Returns lse (T, U+1), lp_blank (T, U+1), lp_label (T, U+1); lp_label[:, U]
    is -inf (no label arc leaves the top row).
    """
    z = np.asarray(z, dtype=np.float64)
    T, U1, _ = z.shape
    U = U1 - 1
    lse = row_log_normalizer(z)
    lp_blank = z[:, :, blank] - lse
    lp_label = np.full((T, U1), NEG_INF)
    for u in range(U):
        lp_label[:, u] = z[:, u, int(labels[u])] - lse[:, u]
    return lse, lp_blank, lp_label


def forward_scores(lp_blank, lp_label, variant="rnnt"):
    """alpha(t, u) = log-sum of all partial paths from (0, 0) into (t, u).

    Returns (alpha, lnP) with lnP the forward score of the final state.
    """
    assert variant in VARIANTS
    T, U1 = lp_blank.shape
    U = U1 - 1
    alpha = np.full((T, U1), NEG_INF)
    for t in range(T):
        for u in range(U1):
            if t == 0 and u == 0:
                alpha[0, 0] = 0.0
                continue
            acc = NEG_INF
            if t > 0:  # blank arc (t-1, u) -> (t, u)
                acc = log_add(acc, alpha[t - 1, u] + lp_blank[t - 1, u])
            if u > 0:  # label arc (t, u-1) -> (t, u)
                acc = log_add(acc, alpha[t, u - 1] + lp_label[t, u - 1])
            if variant != "rnnt" and u == 0 and t >= 1:
                # initial wild-card arc (0, 0) -> (t, 0), weight ln 1 = 0
                acc = log_add(acc, alpha[0, 0])
            if variant == "wrnnt" and u == U and t == T - 1:
                # final wild-card arcs (t', U) -> (T-1, U), t' < T-1, weight 0
                for tp in range(T - 1):
                    acc = log_add(acc, alpha[tp, U])
            alpha[t, u] = acc
    lnP = alpha[T - 1, U] + lp_blank[T - 1, U]  # closing blank
    if variant == "wrnnt_allow_ignore":
        for tp in range(T - 1):  # (t', U) -> final, weight 0
            lnP = log_add(lnP, alpha[tp, U])
    return alpha, lnP


def backward_scores(lp_blank, lp_label, variant="rnnt"):
    """beta(t, u) = log-sum of all partial paths from (t, u) to the final state.

    Returns (beta, lnP) with lnP = beta(0, 0).
    """
    assert variant in VARIANTS
    T, U1 = lp_blank.shape
    U = U1 - 1
    beta = np.full((T, U1), NEG_INF)
    for t in range(T - 1, -1, -1):
        for u in range(U, -1, -1):
            acc = NEG_INF
            if t == T - 1 and u == U:  # closing blank
                acc = lp_blank[T - 1, U]
            if t < T - 1:  # blank arc (t, u) -> (t+1, u)
                acc = log_add(acc, lp_blank[t, u] + beta[t + 1, u])
            if u < U:  # label arc (t, u) -> (t, u+1)
                acc = log_add(acc, lp_label[t, u] + beta[t, u + 1])
            if u == U and t < T - 1:
                if variant == "wrnnt":  # (t, U) -> (T-1, U), weight 0
                    acc = log_add(acc, beta[T - 1, U])
                elif variant == "wrnnt_allow_ignore":  # (t, U) -> final, weight 0
                    acc = log_add(acc, 0.0)
            if variant != "rnnt" and t == 0 and u == 0:
                for tp in range(1, T):  # (0, 0) -> (t', 0), weight 0
                    acc = log_add(acc, beta[tp, 0])
            beta[t, u] = acc
    return beta, beta[0, 0]


def arc_posteriors(alpha, beta, lp_blank, lp_label, lnP):
    """Posterior mass of every blank and label arc (zero where the arc is absent).

    occ_blank(t, u) = exp(alpha(t,u) + lp_blank(t,u) + beta(t+1,u) - lnP), t < T-1
    occ_blank(T-1, U) = exp(alpha(T-1,U) + lp_blank(T-1,U) - lnP)   (closing blank)
    occ_label(t, u) = exp(alpha(t,u) + lp_label(t,u) + beta(t,u+1) - lnP), u < U
    Wild-card arcs carry no parameter, so they have no entry here.
    """
    T, U1 = lp_blank.shape
    U = U1 - 1
    occ_blank = np.zeros((T, U1))
    occ_label = np.zeros((T, U1))
    for t in range(T):
        for u in range(U1):
            if t < T - 1:
                occ_blank[t, u] = math.exp(alpha[t, u] + lp_blank[t, u] + beta[t + 1, u] - lnP)
            elif u == U:
                occ_blank[t, u] = math.exp(alpha[t, u] + lp_blank[t, u] - lnP)
            if u < U:
                occ_label[t, u] = math.exp(alpha[t, u] + lp_label[t, u] + beta[t, u + 1] - lnP)
    return occ_blank, occ_label


def utterance_loss_grad(z, labels, blank=0, variant="rnnt", need_grad=True):
    """Loss and d(loss)/d(logits) for ONE utterance.

    z: (T, U+1, V) logits cut to this utterance's lengths; labels: (U,).
    Returns dict with loss, lnP (forward), lnP_backward, alpha, beta, lse,
    lp_blank, lp_label, occ_blank, occ_label and grad (T, U+1, V) or None.
    grad = softmax * (occ_blank + occ_label) - occ_blank*[v=blank] - occ_label*[v=y_{u+1}]
    """
    z = np.asarray(z, dtype=np.float64)
    lse, lp_blank, lp_label = lattice_weights(z, labels, blank)
    alpha, lnP = forward_scores(lp_blank, lp_label, variant)
    out = dict(loss=-lnP, lnP=lnP, alpha=alpha, lse=lse, lp_blank=lp_blank, lp_label=lp_label)
    if not need_grad:
        out["grad"] = None
        return out
    beta, lnP_b = backward_scores(lp_blank, lp_label, variant)
    occ_blank, occ_label = arc_posteriors(alpha, beta, lp_blank, lp_label, lnP)
    softmax = np.exp(z - lse[:, :, None])
    grad = softmax * (occ_blank + occ_label)[:, :, None]
    grad[:, :, blank] -= occ_blank
    U = z.shape[1] - 1
    for u in range(U):
        grad[:, u, int(labels[u])] -= occ_label[:, u]
    out.update(beta=beta, lnP_backward=lnP_b, occ_blank=occ_blank, occ_label=occ_label, grad=grad)
    return out


def utterance_is_valid(T_b, U_b, labels_b, T_max, U_max, V, blank):
    """Data checks of the boundary: 1 <= T_b <= T_max, 0 <= U_b <= U_max,
    every used label in [0, V) and different from blank."""
    if not (1 <= T_b <= T_max and 0 <= U_b <= U_max):
        return False
    for u in range(U_b):
        y = int(labels_b[u])
        if y < 0 or y >= V or y == blank:
            return False
    return True


def rnnt_loss_grad(logits, labels, logit_lens, label_lens, blank=0, variant="rnnt",
                   need_grad=True, utterances=None):
    """Batched oracle with the boundary's semantics.

    logits: (B, T_max, U_max+1, V) any float dtype, upcast exactly to float64
    per utterance; labels (B, U_max); logit_lens, label_lens (B,).
    Returns (loss (B,) float64, grad float64 of logits' shape or None).
    Rows outside t < T_b, u <= U_b get an exact zero gradient; an utterance with
    bad data gets loss NaN and zero gradient.  ``utterances`` restricts the work
    to a subset of b (others are left NaN / zero) for large batches.
    """
    logits = np.asarray(logits)
    B, T_max, U1_max, V = logits.shape
    U_max = U1_max - 1
    loss = np.full(B, np.nan)
    grad = np.zeros(logits.shape, dtype=np.float64) if need_grad else None
    for b in (range(B) if utterances is None else utterances):
        T_b, U_b = int(logit_lens[b]), int(label_lens[b])
        if not utterance_is_valid(T_b, U_b, labels[b], T_max, U_max, V, blank):
            continue
        z = logits[b, :T_b, :U_b + 1, :].astype(np.float64)
        r = utterance_loss_grad(z, labels[b][:U_b], blank, variant, need_grad)
        loss[b] = r["loss"]
        if need_grad:
            grad[b, :T_b, :U_b + 1, :] = r["grad"]
    return loss, grad
