"""GPU parity of the loss over arc-list lattices (rnnt_arc_plan + rnnt_arc_loss
through the C-ABI) against the float64 arc-list oracle (oracle/arc_lattice.py).

Tolerances as for the grid path, with the loss's relative error taken against
max(1, |L_ref|): fp32 logits, |L - L_ref| <= 1e-5 max(1, |L_ref|) and every
gradient element within 1e-5; half-precision logits, 2e-3 max(1, |L_ref|) and
the gradient bounds of test_gpu_parity.grad_bound.  The absolute 1e-5 term of a
gradient bound grows to 1e-5 max(1, S) on a row whose arcs' posteriors sum to S:
a general lattice may read one row many times over on a path, which a grid never
does (S <= 1 there, so the grid's bounds are unchanged).  An utterance whose final state
no path reaches has loss +inf and a zero gradient; one with bad data, loss NaN
and a zero gradient.  On the lattices of Fig. 1 / Fig. 4 the arc-list path also
agrees with the grid kernels (rnnt_loss) on the same logits.
"""
import sys

import numpy as np
import pytest

from oracle import arc_lattice as AL
from paper_2303_10384_amd import topologies as TP
from paper_2303_10384_amd import workloads as W
from test_gpu_parity import grad_bound

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def announce(request):
    sys.__stderr__.write("\n[gpu-test] %s\n" % request.node.nodeid)
    sys.__stderr__.flush()
    yield


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "GPU tests need a GPU"
    return _t


@pytest.fixture(scope="module")
def pkg(torch):
    import paper_2303_10384_amd as P
    P.load_library()
    return P


def to_dev(torch, x):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def as_tuples(arcs):
    return [(int(a["src"]), int(a["dst"]), int(a["t"]), int(a["u"]), int(a["label"]), float(a["score"])) for a in arcs]


def run_arc(torch, pkg, logits_np, tl, ul, lattices, blank=0, dtype="f32", need_grad=True, poison=True):
    """GPU arc-list loss on the given inputs; returns (loss, grad or None, logits as seen, float64)."""
    B, T_max, U1, V = logits_np.shape
    lg = to_dev(torch, logits_np).to(W.torch_dtype(dtype))
    if poison:
        W.poison_padding(lg, tl, ul)
    plan = pkg.arc_plan(lattices, T_max, U1 - 1, V, blank, device="cuda:0")
    grad_out = torch.full(lg.shape, float("nan"), dtype=lg.dtype, device=lg.device) if need_grad else None
    loss, grad = pkg.arc_loss(lg, to_dev(torch, np.asarray(tl, np.int32)), to_dev(torch, np.asarray(ul, np.int32)),
                              plan, need_grad=need_grad, grad_out=grad_out)
    torch.cuda.synchronize()
    seen = lg.float().cpu().numpy().astype(np.float64)
    g = grad.float().cpu().numpy().astype(np.float64) if grad is not None else None
    return loss.cpu().numpy().astype(np.float64), g, seen


def reference(seen, tl, ul, lattices, need_grad):
    """Oracle losses and gradient of the batch (as AL.batch_loss_grad), plus each row's
    occupancy: the summed posteriors of the arcs that read it."""
    B, T_max, U1, V = seen.shape
    ref_loss = np.full(B, np.nan)
    ref_grad = np.zeros(seen.shape) if need_grad else None
    occ = np.zeros(seen.shape[:3])
    for b, (n, a) in enumerate(lattices):
        arcs = as_tuples(a)
        T_b, U_b = int(tl[b]), int(ul[b])
        if not AL.utterance_is_valid(T_b, U_b, arcs, T_max, U1 - 1, V):
            continue
        r = AL.arc_lattice_loss_grad(seen[b, :T_b, :U_b + 1], arcs, n, need_grad)
        ref_loss[b] = r["loss"]
        if need_grad:
            ref_grad[b, :T_b, :U_b + 1] = r["grad"]
        for g, (_s, _d, t, u, label, _w) in zip(r["posteriors"], arcs):
            if label >= 0:
                occ[b, t, u] += g
    return ref_loss, ref_grad, occ


def check(loss, grad, seen, tl, ul, lattices, dtype="f32"):
    ref_loss, ref_grad, occ = reference(seen, tl, ul, lattices, grad is not None)
    assert np.array_equal(np.isnan(loss), np.isnan(ref_loss)), (loss, ref_loss)
    assert np.array_equal(np.isinf(loss), np.isinf(ref_loss)), (loss, ref_loss)
    good = np.isfinite(ref_loss)
    # relative to max(1, |L_ref|): each log-semiring addition carries ~1e-7 of absolute error
    # (its float32 correction term), which a loss near 0 cannot absorb relatively
    rel = np.abs(loss[good] - ref_loss[good]) / np.maximum(np.abs(ref_loss[good]), 1.0)
    lim = 1e-5 if dtype == "f32" else 2e-3
    assert np.all(rel <= lim), (rel.max(), loss, ref_loss)
    if grad is not None:
        err = np.abs(grad - ref_grad)
        # a row read by arcs of total posterior S has elements p_v S - occ_v, formed in float32:
        # the absolute term of the bound scales with max(1, S) (S <= 1 on every grid lattice)
        bound = grad_bound(ref_grad, dtype, dtype) + 1e-5 * (np.maximum(occ, 1.0) - 1.0)[..., None]
        bad = ~(err <= bound)
        assert not bad.any(), (err.max(), np.argwhere(bad)[:5])
        for b in range(len(tl)):
            assert np.all(grad[b, int(tl[b]):] == 0) and np.all(grad[b, :, int(ul[b]) + 1:] == 0)
            if not good[b]:
                assert np.all(grad[b] == 0)
    return ref_loss


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("variant", TP.VARIANTS)
@pytest.mark.parametrize("B,T,U,V,blank,seed", [(3, 9, 5, 11, 0, 1), (2, 17, 70, 33, 4, 2), (4, 6, 0, 7, 2, 3),
                                                (2, 5, 130, 9, 0, 4)])
def test_grid_lattices_match_oracle_and_grid_kernels(torch, pkg, dtype, variant, B, T, U, V, blank, seed):
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=seed, sigma=2.0, blank=blank)
    lattices = TP.batch_grid_lattices(tl, ul, labels, blank, variant)
    loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, blank, dtype)
    check(loss, grad, seen, tl, ul, lattices, dtype)
    # the grid kernels on the same logits
    lg = to_dev(torch, seen).to(W.torch_dtype(dtype))
    l2, g2 = pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), blank=blank,
                           variant=variant)
    torch.cuda.synchronize()
    l2 = l2.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(loss - l2) <= (1e-5 if dtype == "f32" else 2e-3) * np.maximum(np.abs(l2), 1.0))
    g2 = g2.float().cpu().numpy().astype(np.float64)
    # each path rounds its own float32 gradient: one bf16 step (2^-8) apart at most, twice the bound
    lim = {"f32": 1e-5, "bf16": 2.0 ** -7 * np.abs(g2) + 2e-5, "f16": 2e-3 * np.abs(g2) + 2e-5}[dtype]
    assert np.all(np.abs(grad - g2) <= lim)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", range(8))
def test_random_lattices(torch, pkg, dtype, seed):
    rng = np.random.default_rng(100 + seed)
    B, T_max, U_max, V = 4, 7, 5, 37
    logits = (rng.standard_normal((B, T_max, U_max + 1, V)) * 2).astype(np.float32)
    tl = np.array([7, 4, 6, 7], np.int32)
    ul = np.array([5, 3, 5, 2], np.int32)
    lattices = [W.random_arc_lattice(rng, tl[b], ul[b], V, 10 + 9 * b, 30 + 25 * b, long_frac=0.2)
                for b in range(B)]
    loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, 0, dtype)
    check(loss, grad, seen, tl, ul, lattices, dtype)


@pytest.mark.parametrize("chunk", range(4))
def test_arc_seeded_random_sweep(torch, pkg, chunk):
    # 12 seeded random batches per chunk: random padded shape and lengths, random acyclic
    # lattices (up to ~4000 states, dense or sparse, arcs without logits, long arcs),
    # any blank index, every logits dtype
    rng = np.random.default_rng(9500 + chunk)
    for i in range(12):
        B = int(rng.integers(1, 5))
        T_max = int(rng.choice([1, 2, int(rng.integers(1, 20)), int(rng.integers(20, 80))]))
        U_max = int(rng.choice([0, 1, int(rng.integers(0, 12)), int(rng.integers(12, 50))]))
        V = int(rng.choice([2, int(rng.integers(2, 40)), int(rng.integers(40, 400))]))
        blank = int(rng.integers(0, V))
        dtype = str(rng.choice(["f32", "bf16", "f16"]))
        tl = rng.integers(1, T_max, endpoint=True, size=B).astype(np.int32)
        ul = rng.integers(0, U_max, endpoint=True, size=B).astype(np.int32)
        sizes = [int(rng.choice([2, int(rng.integers(2, 60)), int(rng.integers(60, 800)), int(rng.integers(800, 4000))]))
                 for _ in range(B)]
        # within the planner's limits: no more than ~700 arcs reading one row on average
        # (a row carrying several labels takes at most 1024)
        sizes = [max(2, min(n, 700 * int(tl[b]) * (int(ul[b]) + 1))) for b, n in enumerate(sizes)]
        dens = [float(rng.choice([1.0, 2.0, 4.0])) for _ in range(B)]
        long_frac = float(rng.choice([0.0, 0.05, 0.3]))
        eps_frac = float(rng.choice([0.0, 0.2, 0.6]))
        print("[arc-random %d.%d] B=%d T_max=%d U_max=%d V=%d blank=%d %s states=%s density=%s long=%g eps=%g"
              % (chunk, i, B, T_max, U_max, V, blank, dtype, sizes, dens, long_frac, eps_frac), flush=True)
        logits = (rng.standard_normal((B, T_max, U_max + 1, V)) * float(rng.choice([1.0, 2.0, 3.0]))).astype(np.float32)
        arcs = [min(int(dens[b] * sizes[b]), 700 * int(tl[b]) * (int(ul[b]) + 1)) for b in range(B)]
        lattices = [W.random_arc_lattice(rng, int(tl[b]), int(ul[b]), V, sizes[b], arcs[b], eps_frac=eps_frac,
                                         long_frac=long_frac) for b in range(B)]
        loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, blank, dtype)
        check(loss, grad, seen, tl, ul, lattices, dtype)


def test_long_arcs_and_many_levels(torch, pkg):
    # more states than the sweep's LDS window (long arcs read pinned slots), and more
    # levels than one staged window of level records
    rng = np.random.default_rng(7)
    T, U, V = 100, 90, 17
    logits = (rng.standard_normal((3, T, U + 1, V)) * 2).astype(np.float32)
    tl = np.array([T, T, 80], np.int32)
    ul = np.array([U, U, 60], np.int32)
    labels = rng.integers(1, V, size=(3, U)).astype(np.int32)
    lattices = [TP.grid_lattice(T, U, labels[0], 0, "wrnnt"), TP.grid_lattice(T, U, labels[1], 0, "wrnnt_allow_ignore")]
    n = 1500  # a chain of 1500 states: 1500 levels, one state each, with a few long arcs
    chain = np.zeros(n - 1 + 40, TP.ARC_DTYPE)
    for s in range(n - 1):
        chain[s] = (s, s + 1, s % 80, (s // 80) % 61, 1 + s % (V - 1), 0.0)
    for i in range(40):
        s = int(rng.integers(0, n - 600))
        chain[n - 1 + i] = (s, s + 500 + i, 3, 7, 2, -0.5)
    lattices.append((n, chain))
    loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, 0, "f32")
    check(loss, grad, seen, tl, ul, lattices)


def test_wide_levels_and_rows_with_several_labels(torch, pkg):
    rng = np.random.default_rng(8)
    V = 29
    logits = (rng.standard_normal((2, 6, 4, V)) * 2).astype(np.float32)
    tl = np.array([6, 6], np.int32)
    ul = np.array([3, 3], np.int32)
    # a fan: start -> 300 states -> a chain of 250 states -> final; the fan level holds
    # more states and arcs than the sweep keeps in registers
    fan = []
    for i in range(300):
        fan.append((0, 1 + i, i % 6, i % 4, 1 + i % (V - 1), 0.01 * (i % 7)))
        fan.append((1 + i, 301, (i + 1) % 6, (i + 2) % 4, -1 if i % 3 else 5, 0.0))
    for s in range(301, 551):
        fan.append((s, s + 1, s % 6, s % 4, 1 + s % 5, 0.0))
    fan_arcs = np.array(fan, TP.ARC_DTYPE)
    # alternatives: two or three labels on the same row (the extra-rows kernel)
    alt = [(0, 1, 0, 0, 3, 0.0), (0, 1, 0, 0, 4, -0.3), (0, 1, 0, 0, 0, 0.2), (1, 2, 1, 1, 7, 0.0),
           (1, 2, 1, 1, 8, 0.0), (1, 2, 1, 1, 9, 0.0), (2, 3, 2, 1, 0, 0.0), (2, 3, 3, 2, 11, 0.1)]
    lattices = [(552, fan_arcs), (4, np.array(alt, TP.ARC_DTYPE))]
    loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, 0, "f32")
    check(loss, grad, seen, tl, ul, lattices)
    for dtype in ("bf16", "f16"):
        loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, 0, dtype)
        check(loss, grad, seen, tl, ul, lattices, dtype)


def test_degenerate_and_bad_utterances(torch, pkg):
    rng = np.random.default_rng(9)
    V = 6
    logits = rng.standard_normal((6, 3, 3, V)).astype(np.float32)
    tl = np.array([3, 3, 1, 3, 0, 3], np.int32)
    ul = np.array([2, 2, 2, 1, 1, 2], np.int32)
    one = (1, np.zeros(0, TP.ARC_DTYPE))                                        # the empty path: loss 0
    cut = (4, np.array([(0, 1, 0, 0, 1, 0.0), (2, 3, 1, 1, 2, 0.0)], TP.ARC_DTYPE))  # no path: +inf
    outside = (2, np.array([(0, 1, 2, 0, 1, 0.0)], TP.ARC_DTYPE))              # reads t = 2 with T_b = 1: NaN
    deep = (2, np.array([(0, 1, 1, 2, 1, 0.0)], TP.ARC_DTYPE))                 # reads u = 2 with U_b = 1: NaN
    ok = TP.grid_lattice(3, 1, [4], 0, "rnnt")                                 # lengths T_b = 0: NaN
    good = TP.grid_lattice(3, 2, [4, 5], 0, "wrnnt")
    lattices = [one, cut, outside, deep, ok, good]
    loss, grad, seen = run_arc(torch, pkg, logits, tl, ul, lattices, 0, "f32")
    assert loss[0] == 0.0 and np.isinf(loss[1]) and loss[1] > 0
    assert np.isnan(loss[2:5]).all() and np.isfinite(loss[5])
    check(loss, grad, seen, tl, ul, lattices)


def test_loss_only_and_determinism(torch, pkg):
    logits, tl, ul, labels = W.small_case(5, 20, 12, 40, seed=13)
    lattices = TP.batch_grid_lattices(tl, ul, labels, 0, "wrnnt")
    a = run_arc(torch, pkg, logits, tl, ul, lattices)
    b = run_arc(torch, pkg, logits, tl, ul, lattices)
    c = run_arc(torch, pkg, logits, tl, ul, lattices, need_grad=False)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[0], c[0])


def test_plan_shape_mismatch_is_refused(torch, pkg):
    logits, tl, ul, labels = W.small_case(2, 5, 3, 9, seed=1)
    plan = pkg.arc_plan(TP.batch_grid_lattices(tl, ul, labels), 5, 3, 10, 0, device="cuda:0")  # V = 10, not 9
    with pytest.raises(pkg.RNNTError) as e:
        pkg.arc_loss(to_dev(torch, logits), to_dev(torch, tl), to_dev(torch, ul), plan)
    assert e.value.status == 10


@pytest.mark.parametrize("name,utts", [("bpe", [0, 21]), ("wrnnt", [0, 30])])
def test_full_size_grid_lattices(torch, pkg, name, utts):
    # the benchmark's workloads as arc lists: every utterance against the grid kernels,
    # sampled utterances against the oracle
    w = W.WORKLOADS[name]
    tl, ul, labels = W.make_lengths_labels(w)
    lg = W.make_logits(w, "cuda:0")
    lattices = TP.batch_grid_lattices(tl, ul, labels, 0, w.variant)
    plan = pkg.arc_plan(lattices, w.T_max, w.U_max, w.V, 0, device="cuda:0")
    loss, grad = pkg.arc_loss(lg, to_dev(torch, tl), to_dev(torch, ul), plan)
    l2, g2 = pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), variant=w.variant)
    torch.cuda.synchronize()
    assert torch.all((loss - l2).abs() <= 1e-5 * l2.abs())
    assert float((grad - g2).abs().max()) <= 1e-5
    loss = loss.cpu().numpy().astype(np.float64)
    for b in utts:
        T_b, U_b = int(tl[b]), int(ul[b])
        z = lg[b:b + 1].float().cpu().numpy().astype(np.float64)
        ref_loss, ref_grad = AL.batch_loss_grad(z, tl[b:b + 1], ul[b:b + 1],
                                                [(lattices[b][0], as_tuples(lattices[b][1]))])
        assert abs(loss[b] - ref_loss[0]) <= 1e-5 * abs(ref_loss[0])
        gb = grad[b].float().cpu().numpy().astype(np.float64)
        assert np.abs(gb - ref_grad[0]).max() <= 1e-5
        assert T_b >= 1 and U_b >= 0
