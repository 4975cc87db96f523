"""The arc-list planner (rnnt_arc_plan, host code in the library), CPU only.

The plan image is replayed here the way the device kernels read it: the
level records in order; per level, each entering arc's source score read from
the LDS slot the plan names (a ring of recent states that later states
overwrite, plus pinned slots); each state's run of entering arcs; the
reversed lattice through the mirror numbering and the arc permutation; the
label arcs grouped by logits row.  Unwritten LDS slots hold NaN, so a slot read
before it is written, or after the ring has overwritten it, shows up.  The
losses and gradients of the replay must match the arc-list oracle.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest
from scipy.special import log_softmax, logsumexp

from oracle import arc_lattice as AL
from paper_2303_10384_amd import topologies as TP
from paper_2303_10384_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LAYOUT = open(os.path.join(ROOT, "paper_2303_10384_amd", "csrc", "rnnt_arc_layout.h")).read()


def const(name):
    return int(re.search(r"constexpr int %s = (\w+)" % name, LAYOUT).group(1))


RING, PINS, LEVEL_ARCS = const("kArcRing"), const("kArcPins"), const("kArcLevelArcs")
PAD_DEGREE = const("kArcPadDegree")
DUMMY = RING + PINS


# When RNNT_ARC_PLAN_SANITIZED names a build of rnnt_arc_plan.cpp alone with the
# address and undefined-behaviour sanitizers (test_arc_plan_sanitized_cpu.py makes
# one and reruns this file in a process that preloads the sanitizer runtime), every
# planner call below goes to that build.
SANITIZED = os.environ.get("RNNT_ARC_PLAN_SANITIZED")


class SanitizedPlanner:
    """The planner's entry points from the sanitizer build, standing in for the library
    (the planner tests call nothing else; status strings come from the binding's names)."""

    def __init__(self, path, BD):
        lib = ctypes.CDLL(path)
        i32, i64, vp, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
        lib.rnnt_arc_plan_bytes_bound.argtypes = [i32, i32, i32, i64, i64]
        lib.rnnt_arc_plan_bytes_bound.restype = sz
        lib.rnnt_arc_plan.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, sz, ctypes.POINTER(BD.ArcPlanDesc)]
        lib.rnnt_arc_plan.restype = ctypes.c_int
        self.rnnt_arc_plan = lib.rnnt_arc_plan
        self.rnnt_arc_plan_bytes_bound = lib.rnnt_arc_plan_bytes_bound
        self.names = BD.STATUS_NAMES

    def rnnt_status_string(self, status):
        return self.names.get(int(status), "unknown status").encode()


@pytest.fixture(scope="module")
def binding():
    from paper_2303_10384_amd import binding as BD
    if SANITIZED:
        saved, BD._lib = BD._lib, SanitizedPlanner(SANITIZED, BD)
        yield BD
        BD._lib = saved
        return
    if not os.path.exists(BD.LIB_PATH):
        from paper_2303_10384_amd import build
        build.build(verbose=False)
    BD.load_library()
    yield BD


GENERIC = 1 << 30


def unpack(plan):
    d, img = plan.desc, plan.image.numpy()
    B, S, L, N, X = d.B, d.num_states, d.num_levels, d.num_row_arcs, d.num_extra_rows
    A0, A1 = d.num_slots[0], d.num_slots[1]
    R = B * d.T_max * (d.U_max + 1)

    def arr(i, dtype, n, width=1):
        return np.frombuffer(img, dtype=dtype, count=n * width, offset=d.off[i]).reshape((n, width) if width > 1
                                                                                       else (n,))
    return dict(
        utt=arr(0, np.int32, B, 4), ends=arr(1, np.int32, B, 4), slots=arr(2, np.int32, B, 4),
        level=[arr(3, np.int32, L, 4), arr(4, np.int32, L, 4)],
        seg=[arr(5, np.int32, S), arr(6, np.int32, S)], pin=[arr(7, np.int32, S), arr(8, np.int32, S)],
        arcs=arr(9, np.int32, A0, 4), score=arr(10, np.float32, A0), loc=[arr(11, np.int32, A0), arr(12, np.int32, A1)],
        perm=arr(13, np.int32, A0), row_seg=arr(14, np.int32, R + 1), row_arc=arr(15, np.int32, N),
        xrows=arr(16, np.int32, X))


def replay_sweep(P, g, b, w):
    """Scores of every state of utterance b in graph g, read as the sweep reads them."""
    s_begin, s_end, l_begin, l_end = (int(x) for x in P["utt"][b])
    fin0, start1 = int(P["ends"][b][0]), int(P["ends"][b][1])
    start = start1 if g else s_begin
    lds = np.full(DUMMY + 1, np.nan)
    val = np.full(s_end - s_begin, np.nan)

    def term(slot):
        loc = int(P["loc"][g][slot])
        if loc < 0:
            return -math.inf
        assert loc <= DUMMY
        v = lds[loc] + w[slot]
        assert not np.isnan(v), "a source score read from an unwritten or overwritten slot"
        return v

    for k in range(l_begin, l_end):
        s_lo, ns_flag, slot_lo, packed = (int(x) for x in P["level"][g][k])
        ns, generic = ns_flag & (GENERIC - 1), bool(ns_flag & GENERIC)
        nslots, D = packed & 0xFFFF, packed >> 16
        assert ns <= RING and nslots <= LEVEL_ARCS
        if not generic:
            assert nslots == ns * D and D <= PAD_DEGREE
        # a generic level reads every source before it stores a score; a padded level
        # takes its states 64 at a time, each group read and then stored
        groups = [range(s_lo, s_lo + ns)] if generic else [range(c, min(c + 64, s_lo + ns))
                                                           for c in range(s_lo, s_lo + ns, 64)]
        for group in groups:
            out = []
            for s in group:
                seg = int(P["seg"][g][s])
                rel, cnt = seg & 0xFFFF, seg >> 16
                assert cnt <= D
                if generic:
                    terms = [term(slot_lo + rel + q) for q in range(cnt)]
                else:
                    j = s - s_lo
                    assert rel == j * D
                    terms = [term(slot_lo + j * D + q) for q in range(D)]
                    assert all(int(P["loc"][g][slot_lo + j * D + q]) < 0 for q in range(cnt, D))  # padding
                v = logsumexp(terms) if terms and max(terms) > -math.inf else -math.inf
                out.append(0.0 if s == start else v)
            for s, v in zip(group, out):
                lds[(s - s_begin) & (RING - 1)] = v
                lds[P["pin"][g][s]] = v
                val[s - s_begin] = v
    assert not np.isnan(val).any()
    return val


def replay(plan, logits, logit_lens, label_lens, blank):
    """Losses and gradient of the batch from the plan image (float64)."""
    P = unpack(plan)
    d = plan.desc
    B, T_max, U1, V = logits.shape
    logp = log_softmax(logits.astype(np.float64), axis=-1).reshape(-1, V)
    A0, A1 = d.num_slots[0], d.num_slots[1]
    w0 = np.full(A0, np.nan)
    bad = np.zeros(B, bool)
    real = 0
    for q in range(A0):
        src, dst, row, label = (int(x) for x in P["arcs"][q])
        if src < 0:  # padding
            assert (dst, row, label) == (-1, -1, -2) and P["perm"][q] == -1 and P["loc"][0][q] == -1
            continue
        real += 1
        w0[q] = float(P["score"][q])
        if label >= 0:
            b, rem = divmod(row, T_max * U1)
            t, u = divmod(rem, U1)
            if t >= logit_lens[b] or u > label_lens[b]:
                bad[b] = True
            w0[q] += logp[row, label]
    assert real == d.num_arcs
    w1 = np.full(A1, np.nan)
    used = P["perm"][P["perm"] >= 0]
    w1[used] = w0[P["perm"] >= 0]
    assert len(set(used.tolist())) == real  # one graph-1 slot per arc
    assert np.all((P["loc"][1] >= 0) == ~np.isnan(w1))  # the other graph-1 slots are padding
    loss = np.full(B, np.nan)
    grad = np.zeros(logits.shape).reshape(-1, V)
    for b in range(B):
        if bad[b]:
            continue
        alpha = replay_sweep(P, 0, b, w0)
        beta = replay_sweep(P, 1, b, w1)
        s_begin, s_end = int(P["utt"][b][0]), int(P["utt"][b][1])
        fin = int(P["ends"][b][0]) - s_begin
        lnP = alpha[fin]
        assert lnP == beta[-1] == -math.inf or abs(beta[-1] - lnP) <= 1e-9 * max(1.0, abs(lnP))
        loss[b] = -lnP
        if lnP == -math.inf:
            continue
        rows = range(b * T_max * U1, (b + 1) * T_max * U1)
        for r in rows:
            j0, j1 = int(P["row_seg"][r]), int(P["row_seg"][r + 1])
            if j0 == j1:
                continue
            occ, labels = [], []
            for j in range(j0, j1):
                q = int(P["row_arc"][j])
                src, dst, row, label = (int(x) for x in P["arcs"][q])
                assert row == r and label >= 0
                e = alpha[src - s_begin] + w0[q] + beta[s_end - 1 - dst] - lnP
                occ.append(math.exp(e) if e > -math.inf else 0.0)
                labels.append(label)
            non_blank = [l for l in labels if l != blank]
            assert labels == sorted(labels, key=lambda l: (l != blank, l))  # blank first, then by label
            assert (len(set(non_blank)) >= 2) == (r in set(P["xrows"].tolist()))
            p = np.exp(logp[r])
            grad[r] += p * sum(occ)
            for o, l in zip(occ, labels):
                grad[r, l] -= o
    return loss, grad.reshape(logits.shape)


def as_tuples(arcs):
    return [(int(a["src"]), int(a["dst"]), int(a["t"]), int(a["u"]), int(a["label"]), float(a["score"])) for a in arcs]


def check_against_oracle(binding, lattices, logits, tl, ul, blank, grad_atol=1e-11):
    B, T_max, U1, V = logits.shape
    plan = binding.arc_plan(lattices, T_max, U1 - 1, V, blank)
    loss, grad = replay(plan, logits, tl, ul, blank)
    ref_loss, ref_grad = AL.batch_loss_grad(logits, tl, ul, [(n, as_tuples(a)) for n, a in lattices])
    np.testing.assert_allclose(loss, ref_loss, rtol=1e-10, atol=0)
    np.testing.assert_allclose(grad, ref_grad, rtol=0, atol=grad_atol)
    return plan


@pytest.mark.parametrize("variant", TP.VARIANTS)
def test_grid_lattices_replay(binding, variant):
    logits, tl, ul, labels = W.small_case(3, 7, 4, 6, seed=3, blank=1)
    lattices = TP.batch_grid_lattices(tl, ul, labels, 1, variant)
    check_against_oracle(binding, lattices, logits, tl, ul, 1)


@pytest.mark.parametrize("seed", range(6))
def test_random_lattices_replay(binding, seed):
    rng = np.random.default_rng(seed)
    B, T_max, U_max, V = 3, 5, 3, 7
    logits = rng.standard_normal((B, T_max, U_max + 1, V)) * 2
    tl = np.array([5, 3, 4])
    ul = np.array([3, 2, 3])
    lattices = [W.random_arc_lattice(rng, tl[b], ul[b], V, 6 + 5 * b, 20 + 12 * b, long_frac=0.3) for b in range(B)]
    check_against_oracle(binding, lattices, logits, tl, ul, 0)


def test_long_arcs_use_pinned_slots(binding):
    # more states than the ring holds, with arcs from the start and into the final
    # state spanning all of them (the W-Transducer's wild-card arcs, scaled up)
    T, U, V = 100, 90, 5
    rng = np.random.default_rng(9)
    logits = rng.standard_normal((1, T, U + 1, V))
    labels = rng.integers(1, V, size=(1, U))
    for variant in ("wrnnt", "wrnnt_allow_ignore"):
        lattices = TP.batch_grid_lattices([T], [U], labels, 0, variant)
        assert lattices[0][0] > RING
        # float64 sums in another order over ~190 levels: ~1e-10 apart, where a lost arc shows as >= 1e-3
        plan = check_against_oracle(binding, lattices, logits, np.array([T]), np.array([U]), 0, grad_atol=1e-9)
        assert 0 < plan.max_pins <= PINS


def test_rows_with_several_labels(binding):
    # two label arcs with different labels on the same row: the extra-rows kernel's rows
    rng = np.random.default_rng(2)
    logits = rng.standard_normal((2, 3, 2, 5))
    arcs = np.zeros(6, TP.ARC_DTYPE)
    for i, a in enumerate([(0, 1, 0, 0, 2, 0.1), (0, 1, 0, 0, 3, -0.2), (0, 1, 0, 0, 0, 0.0), (1, 2, 1, 1, 4, 0.0),
                           (1, 2, 1, 0, 1, 0.3), (2, 3, 2, 1, -1, 0.0)]):
        arcs[i] = a
    lattices = [(4, arcs), (4, arcs)]
    plan = check_against_oracle(binding, lattices, logits, np.array([3, 3]), np.array([1, 1]), 0)
    assert plan.num_extra_rows == 2


def test_degenerate_lattices(binding):
    logits = np.random.default_rng(1).standard_normal((3, 2, 2, 4))
    one = (1, np.zeros(0, TP.ARC_DTYPE))                     # start is final: loss 0
    cut = np.zeros(2, TP.ARC_DTYPE)                          # the final state unreachable: loss inf
    cut[0] = (0, 1, 0, 0, 1, 0.0)
    cut[1] = (2, 3, 1, 1, 2, 0.0)
    outside = np.zeros(1, TP.ARC_DTYPE)                      # reads row t = 1 of a one-frame utterance
    outside[0] = (0, 1, 1, 0, 1, 0.0)
    check_against_oracle(binding, [one, (4, cut), (2, outside)], logits, np.array([2, 2, 1]), np.array([1, 1, 1]), 0)


def test_planner_rejects_bad_lists(binding):
    def plan_status(n, arcs, T=3, U=2, V=5, blank=0):
        a = np.zeros(len(arcs), TP.ARC_DTYPE)
        for i, x in enumerate(arcs):
            a[i] = x
        try:
            binding.arc_plan([(n, a)], T, U, V, blank)
            return 0
        except binding.RNNTError as e:
            return e.status
    assert plan_status(3, [(0, 1, 0, 0, 1, 0.0), (1, 2, 0, 0, 1, 0.0)]) == 0
    assert plan_status(3, [(1, 1, 0, 0, 1, 0.0)]) == 10     # not increasing
    assert plan_status(3, [(2, 1, 0, 0, 1, 0.0)]) == 10
    assert plan_status(3, [(0, 3, 0, 0, 1, 0.0)]) == 10     # state out of range
    assert plan_status(3, [(0, 1, 0, 0, 5, 0.0)]) == 10     # label >= V
    assert plan_status(3, [(0, 1, 0, 0, -2, 0.0)]) == 10
    assert plan_status(3, [(0, 1, 3, 0, 1, 0.0)]) == 10     # t >= T_max
    assert plan_status(3, [(0, 1, 0, 3, 1, 0.0)]) == 10     # u > U_max
    assert plan_status(3, [(0, 1, 9, 9, -1, 0.0)]) == 0     # an arc without a label reads no row
    assert plan_status(3, [(0, 1, 0, 0, 1, float("nan"))]) == 10  # scores must be finite
    assert plan_status(3, [(0, 1, 0, 0, -1, float("inf"))]) == 10
    assert plan_status(0, []) == 10
    assert plan_status(3, [(0, 1, 0, 0, 1, 0.0)], blank=5) == 3
    # a level with more entering arcs than the sweep holds
    wide = [(0, 1, 0, 0, 1, 0.0)] * (LEVEL_ARCS + 1)
    assert plan_status(2, wide) == 9


def test_plan_descriptor_and_bound(binding):
    lib = binding.load_library()
    lattices = TP.batch_grid_lattices([4, 2], [2, 1], [[1, 2], [3, 0]], 0, "wrnnt")
    plan = binding.arc_plan(lattices, 4, 2, 5, 0)
    d = plan.desc
    assert d.num_states == sum(n for n, _ in lattices) and d.num_arcs == sum(len(a) for _, a in lattices)
    assert d.image_bytes <= lib.rnnt_arc_plan_bytes_bound(2, 4, 2, d.num_states, d.num_arcs)
    assert all(o % 256 == 0 for o in d.off) and list(d.off) == sorted(d.off)
    # too small an image buffer
    buf = (ctypes.c_uint8 * 64)()
    desc = binding.ArcPlanDesc()
    arcs = np.concatenate([a for _, a in lattices])
    st = lib.rnnt_arc_plan(2, 4, 2, 5, 0, np.array([n for n, _ in lattices], np.int32).ctypes.data,
                           np.array([0, len(lattices[0][1]), len(arcs)], np.int64).ctypes.data, arcs.ctypes.data,
                           ctypes.cast(buf, ctypes.c_void_p), 64, ctypes.byref(desc))
    assert st == 6


def test_padded_and_generic_levels(binding):
    # the W-Transducer's final level gathers T-1 wild-card arcs: a generic level; all
    # other levels of the grid have in-degree <= 2 and are padded
    rng = np.random.default_rng(4)
    logits = rng.standard_normal((2, 9, 4, 6))
    labels = rng.integers(1, 6, size=(2, 3))
    lattices = TP.batch_grid_lattices([9, 7], [3, 2], labels, 0, "wrnnt")
    plan = check_against_oracle(binding, lattices, logits, np.array([9, 7]), np.array([3, 2]), 0)
    P = unpack(plan)
    generic = [(int(r[1]) & GENERIC) != 0 for r in P["level"][0]]
    assert sum(generic) == 2  # one per utterance, forward sweep
    assert plan.slots_per_state == 2


def test_sources_near_the_ring_edge(binding):
    # levels of more than 64 states (stored in two groups) whose arcs reach back
    # almost kArcRing states: the W-Transducer's wild-card arcs on a 250 x 68 grid
    rng = np.random.default_rng(12)
    T, U, V = 250, 67, 5
    logits = rng.standard_normal((1, T, U + 1, V))
    labels = rng.integers(1, V, size=(1, U))
    lattices = TP.batch_grid_lattices([T], [U], labels, 0, "wrnnt")
    check_against_oracle(binding, lattices, logits, np.array([T]), np.array([U]), 0, grad_atol=1e-9)


def raw_plan(binding, B, T, U, V, blank, num_states, arc_begin, arcs, image_bytes=None):
    """rnnt_arc_plan on raw host arrays (any arc_begin, even a malformed one); returns
    (status, descriptor)."""
    lib = binding.load_library()
    num_states = np.ascontiguousarray(num_states, np.int32)
    arc_begin = np.ascontiguousarray(arc_begin, np.int64)
    arcs = np.ascontiguousarray(arcs, TP.ARC_DTYPE)
    if image_bytes is None:
        bound = lib.rnnt_arc_plan_bytes_bound(B, T, U, int(max(0, num_states.sum())), int(max(0, len(arcs))))
        image_bytes = int(bound) if bound else 256
    image = np.zeros(max(image_bytes, 1), np.uint8)
    desc = binding.ArcPlanDesc()
    st = lib.rnnt_arc_plan(B, T, U, V, blank, num_states.ctypes.data, arc_begin.ctypes.data,
                           arcs.ctypes.data if len(arcs) else None, image.ctypes.data, image_bytes,
                           ctypes.byref(desc))
    return st, desc


MUTATIONS = ("src_not_below_dst", "dst_past_end", "negative_src", "label_past_vocab", "label_below_minus_one",
             "row_t_past_end", "row_u_past_end", "score_nan", "score_inf", "no_states", "arc_begin_not_zero",
             "arc_begin_decreasing", "image_short", "bad_shape", "bad_blank")


def test_planner_fuzz_random_and_malformed(binding):
    """Seeded fuzz: random valid batches of lattices must plan (every 8th one is also
    replayed against the oracle); each planted defect must give its status code and
    nothing else.  Stops at the first failure (the seed and the defect are in the
    assertion message)."""
    n_valid = 0
    for seed in range(240):
        rng = np.random.default_rng(10_000 + seed)
        B = int(rng.integers(1, 4))
        T_max, U_max, V = int(rng.integers(1, 6)), int(rng.integers(0, 4)), int(rng.integers(2, 9))
        blank = int(rng.integers(0, V))
        tl = rng.integers(1, T_max, size=B, endpoint=True)
        ul = rng.integers(0, U_max, size=B, endpoint=True)
        lattices = [W.random_arc_lattice(rng, int(tl[b]), int(ul[b]), V, int(rng.integers(1, 12)),
                                         int(rng.integers(0, 30)), long_frac=0.3) for b in range(B)]
        num_states = np.array([n for n, _ in lattices], np.int32)
        counts = np.array([len(a) for _, a in lattices], np.int64)
        arc_begin = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
        arcs = np.concatenate([a for _, a in lattices]) if counts.sum() else np.zeros(0, TP.ARC_DTYPE)
        st, _ = raw_plan(binding, B, T_max, U_max, V, blank, num_states, arc_begin, arcs)
        assert st == 0, ("valid batch refused", seed, st)
        n_valid += 1
        if seed % 8 == 0:
            logits = rng.standard_normal((B, T_max, U_max + 1, V))
            check_against_oracle(binding, lattices, logits, tl, ul, blank)
        # one planted defect per seed
        kind = MUTATIONS[seed % len(MUTATIONS)]
        ns, ab, ar = num_states.copy(), arc_begin.copy(), arcs.copy()
        T2, U2, V2, blank2, img = T_max, U_max, V, blank, None
        expect = 10
        have_arc = len(ar) > 0
        i = int(rng.integers(0, len(ar))) if have_arc else 0
        b_of_i = int(np.searchsorted(arc_begin, i, side="right") - 1) if have_arc else 0
        if kind in ("src_not_below_dst", "dst_past_end", "negative_src", "label_past_vocab", "label_below_minus_one",
                    "row_t_past_end", "row_u_past_end", "score_nan", "score_inf") and not have_arc:
            kind = "no_states"
        if kind == "src_not_below_dst":
            ar[i]["src"] = ar[i]["dst"]
        elif kind == "dst_past_end":
            ar[i]["dst"] = ns[b_of_i]
        elif kind == "negative_src":
            ar[i]["src"] = -1
        elif kind == "label_past_vocab":
            ar[i]["label"] = V
        elif kind == "label_below_minus_one":
            ar[i]["label"] = -2
        elif kind == "row_t_past_end":
            ar[i]["label"], ar[i]["t"] = blank, T_max
        elif kind == "row_u_past_end":
            ar[i]["label"], ar[i]["u"] = blank, U_max + 1
        elif kind == "score_nan":
            ar[i]["score"] = np.nan
        elif kind == "score_inf":
            ar[i]["score"] = -np.inf
        elif kind == "no_states":
            ns[int(rng.integers(0, B))] = 0
        elif kind == "arc_begin_not_zero":
            ab[0] = 1
        elif kind == "arc_begin_decreasing":
            ab[int(rng.integers(1, B + 1))] = -1
        elif kind == "image_short":
            img, expect = 255, 6
        elif kind == "bad_shape":
            T2, expect = 0, 2
        elif kind == "bad_blank":
            blank2, expect = V, 3
        st, _ = raw_plan(binding, B, T2, U2, V2, blank2, ns, ab, ar, image_bytes=img)
        assert st == expect, ("defect", kind, "seed", seed, "status", st, "expected", expect)
    assert n_valid == 240
