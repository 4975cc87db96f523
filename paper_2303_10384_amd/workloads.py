"""Seeded synthetic inputs for the RNN-T / W-RNNT loss (no loss arithmetic here).

The same generator feeds the GPU path and the CPU oracle in tests and in the
benchmark.  Shapes and value distributions follow the workloads the loss is
measured on; joint-network outputs are stood in for by Gaussian logits.

Lengths: T_b uniform in [ceil(0.5 T_max), T_max], U_b uniform in
[ceil(0.3 U_max), U_max], then U_b = min(U_b, T_b); utterance 0 is set to
(T_max, U_max) so the padded shape is the batch maximum, as a collate function
produces.  Labels uniform in [1, V-1] (blank = 0).  The W-Transducer workload
keeps every frame (T_b = T_max) and cuts a uniform 0-20 % prefix and 0-20 %
suffix off a full label sequence of U_max units (words dropped "in a random
left-right proportion", Section 4.1), so U_b is in [0.6 U_max, U_max].
"""
import math
from dataclasses import dataclass

import numpy as np

BASE_SEED = 230310384


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    T_max: int
    U_max: int
    V: int
    sigma: float
    dtype: str          # "f32" | "bf16" | "f16"
    variant: str        # "rnnt" | "wrnnt" | "wrnnt_allow_ignore"
    lengths: str        # "full" | "variable" | "text_drop"
    index: int

    @property
    def seed(self):
        return BASE_SEED + self.index

    def describe(self):
        return ("%s: B=%d T_max=%d U_max=%d V=%d logits~N(0,%g) %s %s lengths=%s"
                % (self.name, self.B, self.T_max, self.U_max, self.V, self.sigma, self.dtype, self.variant,
                   self.lengths))


WORKLOADS = {
    "tiny": Workload("tiny", 2, 20, 8, 16, 1.0, "f32", "rnnt", "full", 0),
    "char": Workload("char", 16, 150, 40, 29, 2.0, "f32", "rnnt", "variable", 1),
    "bpe": Workload("bpe", 32, 250, 80, 1025, 3.0, "f32", "rnnt", "variable", 2),
    "wrnnt": Workload("wrnnt", 32, 250, 80, 1025, 3.0, "f32", "wrnnt", "text_drop", 3),
    "large": Workload("large", 64, 500, 150, 1025, 3.0, "bf16", "rnnt", "variable", 4),
}


def make_lengths_labels(w, seed=None):
    """(logit_lens int32 (B,), label_lens int32 (B,), labels int32 (B, U_max)) as numpy arrays."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    B, T, U, V = w.B, w.T_max, w.U_max, w.V
    if w.lengths == "full":
        tl = np.full(B, T, np.int32)
        ul = np.full(B, U, np.int32)
        labels = rng.integers(1, V - 1, size=(B, U), endpoint=True).astype(np.int32)
    elif w.lengths == "variable":
        tl = rng.integers(math.ceil(0.5 * T), T, size=B, endpoint=True).astype(np.int32)
        ul = rng.integers(math.ceil(0.3 * U), U, size=B, endpoint=True).astype(np.int32)
        ul = np.minimum(ul, tl).astype(np.int32)
        tl[0], ul[0] = T, min(U, T)
        labels = rng.integers(1, V - 1, size=(B, U), endpoint=True).astype(np.int32)
        for b in range(B):
            labels[b, ul[b]:] = 0
    elif w.lengths == "text_drop":
        tl = np.full(B, T, np.int32)
        full = rng.integers(1, V - 1, size=(B, U), endpoint=True).astype(np.int32)
        r = rng.random(size=(B, 2))
        labels = np.zeros((B, U), np.int32)
        ul = np.zeros(B, np.int32)
        for b in range(B):
            pre = int(math.floor(r[b, 0] * 0.2 * U))
            suf = int(math.floor(r[b, 1] * 0.2 * U))
            keep = full[b, pre:U - suf]
            ul[b] = len(keep)
            labels[b, :len(keep)] = keep
        ul[0] = U  # one complete transcript keeps the padded shape at U_max
        labels[0] = full[0]
    else:
        raise ValueError(w.lengths)
    return tl, ul, labels


def torch_dtype(name):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[name]


def make_logits(w, device, seed=None, dtype=None):
    """Logits (B, T_max, U_max+1, V) ~ N(0, sigma^2) in w.dtype, or in `dtype` when given
    (rounded to nearest even from float32), drawn by torch's generator on `device`."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(w.seed if seed is None else seed)
    shape = (w.B, w.T_max, w.U_max + 1, w.V)
    dtype = dtype or w.dtype
    out = torch.empty(shape, dtype=torch_dtype(dtype), device=device)
    if dtype == "f32":
        out.normal_(0.0, w.sigma, generator=g)
    else:
        # draw in float32 slabs to bound the temporary memory, then round
        for b in range(w.B):
            tmp = torch.empty(shape[1:], dtype=torch.float32, device=device)
            tmp.normal_(0.0, w.sigma, generator=g)
            out[b].copy_(tmp)
    return out


def poison_padding(logits, logit_lens, label_lens, value=float("nan")):
    """Fill every logits row outside t < T_b, u <= U_b with `value` (in place)."""
    for b in range(logits.shape[0]):
        T_b, U_b = int(logit_lens[b]), int(label_lens[b])
        logits[b, T_b:] = value
        logits[b, :, U_b + 1:] = value
    return logits


def small_case(B, T_max, U_max, V, seed, sigma=1.5, dtype="f32", full=False, blank=0):
    """A seeded random case of any shape (numpy): logits float32 array, lengths, labels.

    Used for parity sweeps over shapes; blank may be any index (labels avoid it)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if full:
        tl = np.full(B, T_max, np.int32)
        ul = np.full(B, U_max, np.int32)
    else:
        tl = rng.integers(1, T_max, size=B, endpoint=True).astype(np.int32)
        ul = rng.integers(0, U_max, size=B, endpoint=True).astype(np.int32)
        tl[0], ul[0] = T_max, U_max
    non_blank = np.array([v for v in range(V) if v != blank], np.int32)
    labels = non_blank[rng.integers(0, len(non_blank), size=(B, U_max))].astype(np.int32)
    logits = (rng.standard_normal(size=(B, T_max, U_max + 1, V)) * sigma).astype(np.float32)
    return logits, tl, ul, labels


from .topologies import ARC_DTYPE  # noqa: E402  (the record layout of an arc)


def random_arc_lattice(rng, T_b, U_b, V, n_states, n_arcs, eps_frac=0.2, score_sigma=0.5, long_frac=0.1):
    """A seeded random acyclic lattice over one utterance's rows (structure only).

    States 0 .. n_states-1 (0 the start, n_states-1 the final state).  A chain
    0 -> 1 -> ... -> n_states-1 guarantees a complete path; the other arcs join
    random pairs src < dst, mostly between nearby states, a share `long_frac`
    anywhere.  Each arc reads a random row (t < T_b, u <= U_b) and label, or,
    with probability eps_frac, no logits (label -1); scores are N(0, score_sigma).
    Returns (n_states, arcs) with arcs a numpy array of ARC_DTYPE.
    """
    n_states = max(1, int(n_states))
    pairs = [(s, s + 1) for s in range(n_states - 1)]
    while len(pairs) < n_arcs and n_states >= 2:
        s = int(rng.integers(0, n_states - 1))
        if rng.random() < long_frac:
            d = int(rng.integers(s + 1, n_states))
        else:
            d = min(n_states - 1, s + 1 + int(rng.integers(0, 3)))
        pairs.append((s, d))
    arcs = np.zeros(len(pairs), ARC_DTYPE)
    for i, (s, d) in enumerate(pairs):
        eps = rng.random() < eps_frac
        arcs[i] = (s, d, 0 if eps else rng.integers(0, T_b), 0 if eps else rng.integers(0, U_b + 1),
                   -1 if eps else rng.integers(0, V), rng.standard_normal() * score_sigma)
    return n_states, arcs[rng.permutation(len(arcs))]
