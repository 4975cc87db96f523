"""GPU parity: the HIP path (through the C-ABI) against the float64 oracle.

Tolerances.  fp32 logits: per-utterance |L - L_ref| <= 1e-5 |L_ref| and every
gradient element |g - g_ref| <= 1e-5.  bf16 / fp16 logits: |L - L_ref| <=
2e-3 |L_ref|; gradient stored as float32 or fp16: |g - g_ref| <= 2e-3 |g_ref| +
1e-5; gradient stored as bf16: its own rounding reaches 2^-8 relative, so the
bound is (2^-8 + 1e-5) |g_ref| + 1e-5 and the stored value must equal the
correctly rounded g_ref except next to ties.  g_ref is computed from the same
half-precision values upcast exactly.  Padding rows must be exactly 0 and NaN
logits in the padding must not leak.
"""
import dataclasses
import os
import sys

import numpy as np
import pytest

from figures import allow_ignore_from_fig4, grid_weights, load_figure
from oracle import rnnt_ref as R
from paper_2303_10384_amd import workloads as W

pytestmark = pytest.mark.gpu

VARIANTS = ("rnnt", "wrnnt", "wrnnt_allow_ignore")


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


def to_dev(torch, x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")
    return t.to(dtype) if dtype is not None else t


BF16_U = 2.0 ** -8  # unit roundoff of bfloat16 storage (8-bit significand)


def grad_bound(grad_ref, logits_dtype, grad_dtype):
    """Per-element bound on |g - g_ref|.

    fp32 logits: 1e-5 absolute.  Half-precision logits with a float32 gradient,
    or an fp16 gradient: 2e-3 |g_ref| + 1e-5.  A bf16 gradient is float32
    arithmetic rounded once to bf16, whose own rounding reaches 2^-8 relative, so
    its bound is that rounding plus the float32 slack: (2^-8 + 1e-5) |g_ref| + 1e-5.
    """
    if logits_dtype == "f32":
        return 1e-5
    if grad_dtype == "bf16":
        return (BF16_U + 1e-5) * np.abs(grad_ref) + 1e-5
    return 2e-3 * np.abs(grad_ref) + 1e-5


def bf16_round(x):
    import torch as _t
    return _t.from_numpy(np.asarray(x, dtype=np.float32)).to(_t.bfloat16).float().numpy().astype(np.float64)


def tol_check(loss, grad, loss_ref, grad_ref, logits_dtype="f32", tl=None, ul=None, grad_dtype=None):
    """Assert the stated tolerances; returns (max loss rel err, max grad abs err)."""
    grad_dtype = grad_dtype or logits_dtype
    half = logits_dtype != "f32"
    good = np.isfinite(loss_ref)
    assert np.array_equal(np.isnan(loss), ~good), (loss, loss_ref)
    rel = np.abs(loss[good] - loss_ref[good]) / np.maximum(np.abs(loss_ref[good]), 1e-30)
    lrt = 2e-3 if half else 1e-5
    assert np.all(rel <= lrt), ("loss", rel.max(), loss[good], loss_ref[good])
    gerr = 0.0
    if grad is not None:
        err = np.abs(grad.astype(np.float64) - grad_ref)
        bad = ~(err <= grad_bound(grad_ref, logits_dtype, grad_dtype))  # NaN counts as bad
        assert not bad.any(), ("grad", err.max(), np.argwhere(bad)[:5])
        gerr = float(err.max())
        if grad_dtype == "bf16":
            # float32 arithmetic: the stored value is the correctly rounded g_ref, or its
            # neighbour where g_ref sits next to a tie or is a cancelling small difference
            rn = bf16_round(grad_ref)
            differ = grad != rn
            assert np.all(np.abs(grad - rn)[differ] <= 2.0 ** -7 * np.abs(rn[differ]) + 1e-5)
            if differ.size >= 10000:
                assert differ.mean() <= 1e-2, differ.mean()
        if tl is not None:
            for b in range(len(tl)):
                if not good[b]:
                    assert np.all(grad[b] == 0)
                    continue
                assert np.all(grad[b, tl[b]:] == 0)
                assert np.all(grad[b, :, ul[b] + 1:] == 0)
    return float(rel.max()) if rel.size else 0.0, gerr


def run_case(torch, pkg, logits_np, tl, ul, labels, blank=0, variant="rnnt", dtype="f32", poison=True,
             need_grad=True, grad_dtype=None):
    """GPU call on the given inputs (logits rounded to dtype on the device);
    returns (loss, grad as float64 numpy or None, the exact logits the GPU saw as float64).
    The gradient buffer starts out NaN, so an element the kernels never write shows."""
    lg = to_dev(torch, logits_np).to(W.torch_dtype(dtype))
    if poison:
        W.poison_padding(lg, tl, ul)
    grad_out = None
    if need_grad:
        gdt = W.torch_dtype(grad_dtype or dtype)
        grad_out = torch.full(lg.shape, float("nan"), dtype=gdt, device=lg.device)
    loss, grad = pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), blank=blank,
                               variant=variant, need_grad=need_grad, grad_out=grad_out,
                               grad_dtype=None if grad_dtype is None else W.torch_dtype(grad_dtype))
    torch.cuda.synchronize()
    seen = lg.float().cpu().numpy().astype(np.float64)
    g = grad.float().cpu().numpy().astype(np.float64) if grad is not None else None
    return loss.cpu().numpy().astype(np.float64), g, seen


# ---------------------------------------------------------------------------
# the library that runs is the in-tree HIP build
# ---------------------------------------------------------------------------

def test_native_library_loaded(torch, pkg):
    logits, tl, ul, labels = W.small_case(1, 3, 2, 5, seed=1)
    run_case(torch, pkg, logits, tl, ul, labels)
    maps = open("/proc/self/maps").read()
    assert "librnnt_mi355x.so" in maps
    assert "gfx950" in pkg.version()


# ---------------------------------------------------------------------------
# lattice kernel on the paper's printed lattices
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("variant,loader,ref", [
    ("rnnt", lambda: load_figure("fig1_rnnt_lattice.txt"), 4.2574511041),
    ("wrnnt", lambda: load_figure("fig4_wrnnt_lattice.txt"), 2.2070452674),
    ("wrnnt_allow_ignore", lambda: allow_ignore_from_fig4(load_figure("fig4_wrnnt_lattice.txt")), 1.9385100266),
])
def test_lattice_kernel_on_printed_figures(torch, pkg, variant, loader, ref):
    fig = loader()
    lp_b, lp_l = map(np.array, grid_weights(fig))
    lp_l[:, -1] = np.nan  # never read
    T, U1 = lp_b.shape
    out = pkg.lattice_scores(to_dev(torch, lp_b[None]), to_dev(torch, lp_l[None]),
                             to_dev(torch, np.array([T], np.int32)), to_dev(torch, np.array([U1 - 1], np.int32)),
                             variant)
    loss = float(out["loss"][0])
    assert abs(loss - ref) <= 1e-6 * ref
    assert abs(float(out["loss_bwd"][0]) - ref) <= 1e-6 * ref
    alpha, lnP = R.forward_scores(lp_b, np.where(np.isnan(lp_l), -np.inf, lp_l), variant)
    beta, _ = R.backward_scores(lp_b, np.where(np.isnan(lp_l), -np.inf, lp_l), variant)
    ob, ol = R.arc_posteriors(alpha, beta, lp_b, np.where(np.isnan(lp_l), -np.inf, lp_l), lnP)
    np.testing.assert_allclose(out["alpha"][0].cpu().numpy(), alpha, atol=1e-6)
    np.testing.assert_allclose(out["beta"][0].cpu().numpy(), beta, atol=1e-6)
    np.testing.assert_allclose(out["occ_blank"][0].cpu().numpy(), ob, atol=1e-6)
    np.testing.assert_allclose(out["occ_label"][0].cpu().numpy(), ol, atol=1e-6)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("B,T,U", [(3, 7, 5), (2, 40, 70), (2, 6, 200), (1, 3, 300), (1, 2, 700), (1, 3, 1500),
                                   (1, 2, 2047), (4, 1, 0), (3, 9, 0)])
def test_lattice_kernel_random_weights(torch, pkg, variant, B, T, U):
    rng = np.random.default_rng(B * 1000 + T * 10 + U)
    lp_b = -rng.exponential(1.0, size=(B, T, U + 1))
    lp_l = -rng.exponential(1.5, size=(B, T, U + 1))
    tl = rng.integers(1, T, size=B, endpoint=True).astype(np.int32)
    ul = rng.integers(0, U, size=B, endpoint=True).astype(np.int32)
    tl[0], ul[0] = T, U
    out = pkg.lattice_scores(to_dev(torch, lp_b), to_dev(torch, lp_l), to_dev(torch, tl), to_dev(torch, ul), variant)
    for b in range(B):
        Tb, Ub = tl[b], ul[b]
        pb = lp_b[b, :Tb, :Ub + 1]
        pl = lp_l[b, :Tb, :Ub + 1].copy()
        pl[:, Ub] = -np.inf
        alpha, lnP = R.forward_scores(pb, pl, variant)
        beta, lnPb = R.backward_scores(pb, pl, variant)
        ob, ol = R.arc_posteriors(alpha, beta, pb, pl, lnP)
        scale = max(1.0, abs(lnP))
        assert abs(float(out["loss"][b]) + lnP) <= 1e-9 * scale + 2e-6 * np.sqrt(Tb + Ub), (b, lnP)
        assert abs(float(out["loss_bwd"][b]) + lnPb) <= 1e-9 * scale + 2e-6 * np.sqrt(Tb + Ub)
        np.testing.assert_allclose(out["occ_blank"][b, :Tb, :Ub + 1].cpu().numpy(), ob, atol=1e-5)
        np.testing.assert_allclose(out["occ_label"][b, :Tb, :Ub + 1].cpu().numpy(), ol, atol=1e-5)


# ---------------------------------------------------------------------------
# populate kernel (lse and gathered log-probs), tested on its own
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("V,blank", [(2, 0), (3, 2), (5, 1), (16, 0), (29, 0), (257, 100), (1025, 0), (4100, 4099)])
def test_populate_kernel(torch, pkg, dtype, V, blank):
    logits, tl, ul, labels = W.small_case(3, 6, 5, V, seed=V + blank, sigma=3.0, blank=blank)
    lg = to_dev(torch, logits).to(W.torch_dtype(dtype))
    W.poison_padding(lg, tl, ul)
    lse, lpb, lpl = pkg.log_softmax_gather(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), blank)
    torch.cuda.synchronize()
    z = lg.float().cpu().numpy().astype(np.float64)
    for b in range(3):
        T_b, U_b = tl[b], ul[b]
        lse_r, pb_r, pl_r = R.lattice_weights(z[b, :T_b, :U_b + 1], labels[b, :U_b], blank)
        np.testing.assert_allclose(lse[b, :T_b, :U_b + 1].cpu().numpy(), lse_r, rtol=0, atol=1e-6)
        np.testing.assert_allclose(lpb[b, :T_b, :U_b + 1].cpu().numpy(), pb_r, rtol=0, atol=1e-6)
        np.testing.assert_allclose(lpl[b, :T_b, :U_b].cpu().numpy(), pl_r[:, :U_b], rtol=0, atol=1e-6)
        assert np.all(np.isneginf(lpl[b, :T_b, U_b].cpu().numpy()))
        # rows outside the utterance are not written
        assert np.all(np.isnan(lse[b, T_b:].cpu().numpy()))
        assert np.all(np.isnan(lse[b, :, U_b + 1:].cpu().numpy()))


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("V", [300, 1025, 4100])
def test_populate_kernel_rows_far_apart(torch, pkg, dtype, V):
    # a frame's rows at offsets up to 150 nats apart and with spreads from 0.3 to 20:
    # rows whose range leaves the shift a wave carries from row to row, so the
    # populate kernel must notice and take their maxima again
    B, T, U = 2, 5, 40
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=V + 7, sigma=1.0, full=True)
    rng = np.random.Generator(np.random.PCG64(V))
    offset = rng.choice([-90.0, -40.0, 0.0, 0.0, 0.0, 35.0, 120.0], size=(B, T, U + 1, 1))
    spread = rng.choice([0.3, 1.0, 3.0, 3.0, 20.0], size=(B, T, U + 1, 1))
    if dtype == "f16":  # inside the float16 range
        offset, spread = offset / 4, np.minimum(spread, 5.0)
    logits = (logits * spread + offset).astype(np.float32)
    lg = to_dev(torch, logits).to(W.torch_dtype(dtype))
    lse, lpb, lpl = pkg.log_softmax_gather(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), 0)
    torch.cuda.synchronize()
    z = lg.float().cpu().numpy().astype(np.float64)
    for b in range(B):
        lse_r, pb_r, pl_r = R.lattice_weights(z[b], labels[b], 0)
        np.testing.assert_allclose(lse[b].cpu().numpy(), lse_r, rtol=0, atol=1e-6)
        np.testing.assert_allclose(lpb[b].cpu().numpy(), pb_r, rtol=0, atol=1e-6)
        np.testing.assert_allclose(lpl[b, :, :U].cpu().numpy(), pl_r[:, :U], rtol=0, atol=1e-6)


# ---------------------------------------------------------------------------
# end to end: rnnt_loss against the oracle
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,gdt", [("f32", "f32"), ("bf16", "f32")])
@pytest.mark.parametrize("variant", ["rnnt", "wrnnt"])
def test_loss_rows_far_apart(torch, pkg, dtype, gdt, variant):
    # the loss and gradient over rows far apart in offset and spread (the row
    # normaliser's shift is taken again wherever a row leaves its range); lse stays
    # under ~110 nats, where the gradient kernel's float32 normaliser (log2 units)
    # keeps the softmax within 5.3e-6 relative
    B, T, U, V = 3, 6, 30, 1025
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=31, sigma=1.0)
    rng = np.random.Generator(np.random.PCG64(32))
    offset = rng.choice([-60.0, -25.0, 0.0, 0.0, 25.0, 60.0], size=(B, T, U + 1, 1))
    spread = rng.choice([0.3, 1.0, 3.0, 10.0], size=(B, T, U + 1, 1))
    logits = (logits * spread + offset).astype(np.float32)
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, variant=variant, dtype=dtype, grad_dtype=gdt)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, variant)
    tol_check(loss, grad, loss_ref, grad_ref, dtype, tl, ul, grad_dtype=gdt)


@pytest.mark.parametrize("variant", VARIANTS)
def test_tiny_workload(torch, pkg, variant):
    w = W.WORKLOADS["tiny"]
    tl, ul, labels = W.make_lengths_labels(w)
    logits = W.make_logits(w, "cuda:0").cpu().numpy()
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, variant=variant)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, variant)
    tol_check(loss, grad, loss_ref, grad_ref, "f32", tl, ul)


@pytest.mark.parametrize("variant", ["rnnt", "wrnnt"])
def test_char_workload(torch, pkg, variant):
    w = W.WORKLOADS["char"]
    tl, ul, labels = W.make_lengths_labels(w)
    logits = W.make_logits(w, "cuda:0").cpu().numpy()
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, variant=variant)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, variant)
    tol_check(loss, grad, loss_ref, grad_ref, "f32", tl, ul)


@pytest.mark.parametrize("dtype,gdt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f16", "f16"),
                                       ("f16", "f32")])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("B,T,U,V,blank,seed", [
    (4, 9, 6, 7, 0, 1), (3, 17, 70, 33, 5, 2), (2, 5, 130, 11, 10, 3), (5, 13, 3, 1030, 1029, 4),
    (2, 4, 2, 3, 1, 5), (3, 6, 4, 2, 0, 6), (1, 1, 5, 9, 0, 7), (2, 11, 0, 6, 2, 8)])
def test_random_shapes(torch, pkg, dtype, gdt, variant, B, T, U, V, blank, seed):
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=seed, sigma=2.0, blank=blank)
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, blank=blank, variant=variant, dtype=dtype,
                                grad_dtype=gdt)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, blank, variant)
    tol_check(loss, grad, loss_ref, grad_ref, dtype, tl, ul, grad_dtype=gdt)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("B,T,U,V,seed", [
    (2, 5, 150, 7, 24),    # 3 units per lane of the sweep
    (2, 4, 300, 6, 21),    # 6 units per lane; a diagonal split over two populate blocks
    (1, 3, 700, 5, 22),    # 12 units per lane
    (1, 2, 1023, 3, 23),   # 16 units per lane (U_max + 1 = 1024)
    (1, 3, 1535, 4, 25),   # 24 units per lane
    (1, 2, 2047, 3, 26),   # the widest label axis the sweep takes (U_max + 1 = 2048)
])
def test_wide_label_axis(torch, pkg, dtype, variant, B, T, U, V, seed):
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=seed, sigma=2.0)
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, variant=variant, dtype=dtype,
                                grad_dtype="f32")
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, variant)
    tol_check(loss, grad, loss_ref, grad_ref, dtype, tl, ul, grad_dtype="f32")


@pytest.mark.parametrize("variant", VARIANTS)
def test_sweep_wave_boundaries(torch, pkg, variant):
    # U_max + 1 = 151: three sweep waves of 64 units.  The utterances put u = U at and around
    # the waves' edges (63, 64, 65, 127, 128) and at the ends (0, 1, 150), with one, two and
    # several frames, so the last unit and the closing blank sit in every wave and lane 0 / 63
    # of each wave exchange across the boundary.
    logits, _, _, labels = W.small_case(12, 7, 150, 9, seed=31, sigma=2.0)
    ul = np.array([0, 1, 63, 64, 65, 127, 128, 150, 64, 127, 0, 150], np.int32)
    tl = np.array([7, 1, 2, 7, 3, 1, 7, 2, 1, 7, 1, 7], np.int32)
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, variant=variant)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, variant)
    tol_check(loss, grad, loss_ref, grad_ref, "f32", tl, ul)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rows_of_underflowed_posteriors_are_exact_zeros(torch, pkg, dtype):
    # long lattices with sharp logits: many valid rows lie so far from every likely path that
    # both arc posteriors underflow float32; the gradient kernel writes them as zero rows
    # without reading their logits, so their gradient must be exactly +0 (and the rest match)
    logits, tl, ul, labels = W.small_case(2, 120, 40, 300, seed=41, sigma=3.0, full=True)
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, dtype=dtype, grad_dtype="f32")
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, "rnnt")
    tol_check(loss, grad, loss_ref, grad_ref, dtype, tl, ul, grad_dtype="f32")
    n_far = 0
    for b in range(2):
        _, lp_b, lp_l = R.lattice_weights(seen[b], labels[b], 0)
        alpha, lnP = R.forward_scores(lp_b, lp_l, "rnnt")
        beta, _ = R.backward_scores(lp_b, lp_l, "rnnt")
        ob, ol = R.arc_posteriors(alpha, beta, lp_b, lp_l, lnP)
        far = np.maximum(ob, ol) < 2.0 ** -140  # well below float32's range: 0 on the device too
        n_far += int(far.sum())
        assert np.all(grad[b][far] == 0) and not np.any(np.signbit(grad[b][far]))
    assert n_far >= 0.1 * 2 * 120 * 41, n_far  # the case exercises the skipped rows


def random_case(rng):
    """Shape, variant, dtypes, blank and logit scale of one seeded random case (up to 2e7 logits)."""
    B = int(rng.integers(1, 5))
    T = int(rng.choice([1, 2, 3, int(rng.integers(1, 40)), int(rng.integers(40, 260))]))
    U = int(rng.choice([0, 1, int(rng.integers(0, 70)), int(rng.integers(60, 260)), int(rng.integers(250, 700))]))
    V = int(rng.choice([2, 3, int(rng.integers(2, 64)), int(rng.integers(64, 700))]))
    while B * T * (U + 1) * V > 20_000_000:
        if U > 0 and rng.random() < 0.5:
            U //= 2
        elif T > 1:
            T = max(1, T // 2)
        else:
            V = max(2, V // 2)
    variant = str(rng.choice(VARIANTS))
    dtype = str(rng.choice(["f32", "f32", "bf16", "f16"]))
    gdt = dtype if dtype == "f32" else str(rng.choice([dtype, "f32"]))
    return dict(B=B, T=T, U=U, V=V, variant=variant, dtype=dtype, gdt=gdt, blank=int(rng.integers(0, V)),
                sigma=float(rng.choice([1.0, 2.0, 3.0, 4.0])), full=bool(rng.random() < 0.3),
                seed=int(rng.integers(0, 1 << 30)))


@pytest.mark.parametrize("chunk", range(8))
def test_seeded_random_sweep(torch, pkg, chunk):
    # 50 seeded random cases per chunk: any blank index, U from 0 to ~700 (one to four
    # waves, or 6-12 units per lane), T from 1, V from 2, every variant and dtype.
    # The loss is held to the relative bound against max(1, |L_ref|): a W-Transducer
    # loss with U = 0 can sit near 0 (P may exceed 1), where each log-add's float32
    # correction term leaves ~1e-8 of absolute error.  The share of bf16-stored
    # elements off the correctly rounded value is checked for V >= 32 only: with two
    # or three classes most elements are cancelling differences p*occ - occ, whose
    # float32 value need not round like the exact one (each is still within the bound).
    rng = np.random.default_rng(9100 + chunk)
    for i in range(50):
        c = random_case(rng)
        sys.__stderr__.write("[random-case %d.%d] %s\n" % (chunk, i, c))
        sys.__stderr__.flush()
        logits, tl, ul, labels = W.small_case(c["B"], c["T"], c["U"], c["V"], seed=c["seed"], sigma=c["sigma"],
                                              full=c["full"], blank=c["blank"])
        loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, blank=c["blank"], variant=c["variant"],
                                    dtype=c["dtype"], grad_dtype=c["gdt"])
        loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, c["blank"], c["variant"])
        good = np.isfinite(loss_ref)
        assert np.array_equal(np.isnan(loss), ~good), (c, loss, loss_ref)
        lrel = np.abs(loss[good] - loss_ref[good]) / np.maximum(np.abs(loss_ref[good]), 1.0)
        assert np.all(lrel <= (1e-5 if c["dtype"] == "f32" else 2e-3)), (c, lrel.max())
        err = np.abs(grad - grad_ref)
        assert np.all(err <= grad_bound(grad_ref, c["dtype"], c["gdt"])), (c, float(np.nanmax(err)))
        if c["gdt"] == "bf16":
            rn = bf16_round(grad_ref)
            differ = grad != rn
            assert np.all(np.abs(grad - rn)[differ] <= 2.0 ** -7 * np.abs(rn[differ]) + 1e-5), c
            if differ.size >= 10000 and c["V"] >= 32:
                assert differ.mean() <= 1e-2, (c, differ.mean())
        for b in range(c["B"]):
            if not good[b]:
                assert np.all(grad[b] == 0), c
                continue
            assert np.all(grad[b, tl[b]:] == 0) and np.all(grad[b, :, ul[b] + 1:] == 0), c


@pytest.mark.parametrize("dtype,V,blank", [("f32", 4100, 17), ("bf16", 8200, 8199), ("f16", 2600, 0)])
def test_large_vocabulary(torch, pkg, dtype, V, blank):
    # rows longer than the populate kernel's register path (64 lanes x 5 chunks) take its batched path
    logits, tl, ul, labels = W.small_case(3, 7, 5, V, seed=V, sigma=3.0, blank=blank)
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, blank=blank, dtype=dtype)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, blank, "rnnt")
    tol_check(loss, grad, loss_ref, grad_ref, dtype, tl, ul)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("B,T,U,seed", [(4, 12, 9, 11), (3, 9, 100, 13), (2, 7, 150, 14), (2, 5, 230, 15)])
def test_loss_only_matches_fused(torch, pkg, variant, B, T, U, seed):
    # one sweep wave, and two, three and four waves per sweep (65 to 256 units)
    logits, tl, ul, labels = W.small_case(B, T, U, 40, seed=seed)
    a, _, seen = run_case(torch, pkg, logits, tl, ul, labels, variant=variant, need_grad=False)
    b, g, _ = run_case(torch, pkg, logits, tl, ul, labels, variant=variant, need_grad=True)
    assert g is not None
    np.testing.assert_array_equal(a, b)
    loss_ref, _ = R.rnnt_loss_grad(seen, labels, tl, ul, 0, variant, need_grad=False)
    tol_check(a, None, loss_ref, None, "f32")


def test_bad_data_is_isolated(torch, pkg):
    logits, tl, ul, labels = W.small_case(6, 8, 5, 12, seed=12)
    tl[1] = 0          # no frames
    ul[2] = 6          # more units than U_max
    labels[3, 1] = 0   # a unit equal to blank
    labels[4, 0] = 12  # a unit outside the vocabulary
    tl[5] = 9          # more frames than T_max
    loss, grad, seen = run_case(torch, pkg, logits, tl, ul, labels, poison=False)
    assert np.isfinite(loss[0])
    assert np.all(np.isnan(loss[1:]))
    assert np.all(grad[1:] == 0)
    loss_ref, grad_ref = R.rnnt_loss_grad(seen, labels, tl, ul, 0, "rnnt")
    tol_check(loss, grad, loss_ref, grad_ref, "f32")


def test_batch_permutation_and_determinism(torch, pkg):
    logits, tl, ul, labels = W.small_case(5, 10, 7, 50, seed=13)
    l1, g1, _ = run_case(torch, pkg, logits, tl, ul, labels)
    l2, g2, _ = run_case(torch, pkg, logits, tl, ul, labels)
    np.testing.assert_array_equal(l1, l2)
    np.testing.assert_array_equal(g1, g2)
    perm = np.array([3, 0, 4, 2, 1])
    lp, gp, _ = run_case(torch, pkg, logits[perm], tl[perm], ul[perm], labels[perm])
    np.testing.assert_array_equal(lp, l1[perm])
    np.testing.assert_array_equal(gp, g1[perm])


def test_no_write_past_gradient(torch, pkg):
    logits, tl, ul, labels = W.small_case(3, 7, 4, 13, seed=14)
    lg = to_dev(torch, logits)
    n = lg.numel()
    buf = torch.full((n + 4096,), 12345.0, dtype=torch.float32, device="cuda:0")
    grad = buf[:n].view(lg.shape)
    pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), grad_out=grad)
    torch.cuda.synchronize()
    assert torch.all(buf[n:] == 12345.0)


def test_preallocated_workspace_and_autograd(torch, pkg):
    logits, tl, ul, labels = W.small_case(3, 8, 5, 21, seed=15)
    lg = to_dev(torch, logits)
    nbytes = pkg.loss_workspace_bytes(3, 8, 5, 21)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    l1, g1 = pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), workspace=ws)
    l2, g2 = pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul))
    assert torch.equal(l1, l2) and torch.equal(g1, g2)
    x = lg.clone().requires_grad_(True)
    out = pkg.rnnt_loss_autograd(x, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), reduction="mean")
    out.backward()
    assert torch.allclose(out, l2.mean())
    assert torch.allclose(x.grad, g2 / 3, atol=1e-7)


# ---------------------------------------------------------------------------
# full-size workloads (the sizes the benchmark times): the loss of every
# utterance, and the gradient of several (always the shortest and the longest),
# against the oracle, run per utterance in a pool of worker processes
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def oracle_pool():
    import oracle_pool as OP
    pool = OP.make_pool()
    yield pool
    pool.close()
    pool.join()


def utterance_bits(torch, lg, b, T_b, U_b):
    """The valid rows of utterance b as the GPU consumed them: float32 values, or the
    16-bit patterns of bfloat16 / float16 (widened exactly by the worker)."""
    x = lg[b, :T_b, :U_b + 1].contiguous()
    if x.dtype == torch.float32:
        return x.cpu().numpy()
    return x.view(torch.int16).cpu().numpy().view(np.uint16)


def full_size_case(torch, pkg, pool, name, grad_utts, grad_dtype=None, logits_dtype=None, variant=None):
    import oracle_pool as OP
    w = W.WORKLOADS[name]
    if variant is not None:
        w = dataclasses.replace(w, variant=variant)  # same seed: the same lengths, labels and logits
    ldt = logits_dtype or w.dtype
    gdt = grad_dtype or ldt
    tl, ul, labels = W.make_lengths_labels(w)
    lg = W.make_logits(w, "cuda:0", dtype=ldt)
    # NaN everywhere first: every element must be written (padding rows as exact zeros)
    grad_out = torch.full(lg.shape, float("nan"), dtype=W.torch_dtype(gdt), device=lg.device)
    loss, grad = pkg.rnnt_loss(lg, to_dev(torch, labels), to_dev(torch, tl), to_dev(torch, ul), variant=w.variant,
                               grad_out=grad_out, grad_dtype=W.torch_dtype(gdt))
    torch.cuda.synchronize()
    loss = loss.cpu().numpy().astype(np.float64)
    size = tl.astype(np.int64) * (ul.astype(np.int64) + 1)
    grad_set = set(grad_utts) | {int(np.argmax(size)), int(np.argmin(size))}
    jobs = ((b, utterance_bits(torch, lg, b, int(tl[b]), int(ul[b])), ldt, labels[b, :int(ul[b])], 0, w.variant,
             b in grad_set) for b in range(w.B))
    results = OP.run_batched(pool, jobs)
    assert sorted(r[0] for r in results) == list(range(w.B))
    loss_ref = np.full(w.B, np.nan)
    for b, lref, _ in results:
        loss_ref[b] = lref
    lrel, _ = tol_check(loss, None, loss_ref, None, ldt)  # every utterance's loss
    gmax, gratio = 0.0, 0.0
    for b, _, gref_v in results:
        if gref_v is None:
            continue
        T_b, U_b = int(tl[b]), int(ul[b])
        g = grad[b].float().cpu().numpy().astype(np.float64)
        gref = np.zeros(g.shape)
        gref[:T_b, :U_b + 1] = gref_v
        _, gerr = tol_check(loss[b:b + 1], g[None], loss_ref[b:b + 1], gref[None], ldt, tl[b:b + 1], ul[b:b + 1],
                            grad_dtype=gdt)
        gmax = max(gmax, gerr)
        gratio = max(gratio, float(np.max(np.abs(g - gref) / grad_bound(gref, ldt, gdt))))
    sys.__stderr__.write("[full-size] %s (%s) logits %s grad %s: loss max rel err %.2e over %d utterances; grad max "
                         "abs err %.2e, max err / bound %.3f over utterances %s\n"
                         % (name, w.variant, ldt, gdt, lrel, w.B, gmax, gratio, sorted(grad_set)))
    sys.__stderr__.flush()
    # properties that hold at any size, on every utterance
    for b in range(w.B):
        gb = grad[b, :int(tl[b]), :int(ul[b]) + 1].float()
        rs = gb.sum(dim=-1).abs()
        if gdt == "bf16":
            # each stored element is within 2^-8 of its exact value, whose row sums to 0
            assert bool((rs <= 2.0 ** -8 * (1 + 2.0 ** -8) * gb.abs().sum(dim=-1) + 1e-5).all())
        elif gdt == "f16":
            # 2^-11 relative per stored element, plus at most half the subnormal spacing 2^-24
            # for each of the V elements that fall below the normal range
            slack = gb.shape[-1] * 2.0 ** -25 + 2e-5
            assert bool((rs <= 2.0 ** -11 * (1 + 2.0 ** -11) * gb.abs().sum(dim=-1) + slack).all())
        else:
            assert float(rs.max()) < 2e-5
        assert torch.all(grad[b, int(tl[b]):] == 0)
        assert torch.all(grad[b, :, int(ul[b]) + 1:] == 0)
    assert np.all(np.isfinite(loss)) and np.all(loss > 0)


def test_bpe_workload_full_size(torch, pkg, oracle_pool):
    full_size_case(torch, pkg, oracle_pool, "bpe", grad_utts=[0, 5, 17])


def test_wrnnt_workload_full_size(torch, pkg, oracle_pool):
    full_size_case(torch, pkg, oracle_pool, "wrnnt", grad_utts=[0, 9, 20])


def test_large_bf16_workload_full_size(torch, pkg, oracle_pool):
    full_size_case(torch, pkg, oracle_pool, "large", grad_utts=[0, 21, 40])


def test_large_bf16_workload_float32_gradient(torch, pkg, oracle_pool):
    full_size_case(torch, pkg, oracle_pool, "large", grad_utts=[5, 33, 50], grad_dtype="f32")


def test_wrnnt_workload_allow_ignore_full_size(torch, pkg, oracle_pool):
    # the wrnnt batch's shape, lengths and logits under the allow-ignore arcs (Section 4.3)
    full_size_case(torch, pkg, oracle_pool, "wrnnt", grad_utts=[0, 14, 27], variant="wrnnt_allow_ignore")


def test_large_shape_float16_logits(torch, pkg, oracle_pool):
    # the large batch's shape and lengths with IEEE half logits (Section 4.2's precision)
    full_size_case(torch, pkg, oracle_pool, "large", grad_utts=[3, 44], logits_dtype="f16")
