"""rnnt_loss_noalloc (the allocation-free entry point, workspace in the library's
static device array) against rnnt_loss with a caller-given workspace: two calls
in a row on one GPU, the second with a smaller input, each giving exactly the
bits of the workspace entry point (the same kernels on the same inputs)."""
import sys

import numpy as np
import pytest

from paper_2303_10384_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def announce(request):
    sys.__stderr__.write("\n[gpu-test] %s\n" % request.node.nodeid)
    sys.__stderr__.flush()
    yield


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def _inputs(torch, name):
    w = W.WORKLOADS[name]
    tl, ul, labels = W.make_lengths_labels(w)
    return w, W.make_logits(w, "cuda:0"), _dev(torch, labels), _dev(torch, tl), _dev(torch, ul)


def _reference(torch, pkg, lg, labels, tl, ul, variant):
    ws = torch.empty(pkg.loss_workspace_bytes(*lg.shape[:2], lg.shape[2] - 1, lg.shape[3],
                                              pkg.binding.dtype_code(lg.dtype)), dtype=torch.uint8, device="cuda:0")
    return pkg.rnnt_loss(lg, labels, tl, ul, variant=variant, workspace=ws)


def _noalloc(torch, pkg, lg, labels, tl, ul, variant, poison):
    # outputs pre-filled with a value no result takes, so an unwritten element shows
    loss = torch.full((lg.shape[0],), poison, dtype=torch.float32, device="cuda:0")
    grad = torch.full(lg.shape, poison, dtype=lg.dtype, device="cuda:0")
    return pkg.rnnt_loss_noalloc(lg, labels, tl, ul, loss, grad, variant=variant)


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    import torch
    import paper_2303_10384_amd as P
    assert torch.cuda.is_available()
    P.load_library()
    # first call: the bpe batch (B=32, T_max=250, U_max=80, V=1025, fp32), the benchmark's shape
    w1, lg1, lab1, tl1, ul1 = _inputs(torch, "bpe")
    assert P.loss_workspace_bytes(w1.B, w1.T_max, w1.U_max, w1.V) <= P.binding.NOALLOC_SCRATCH_BYTES
    loss_a, grad_a = _noalloc(torch, P, lg1, lab1, tl1, ul1, w1.variant, 12345.0)
    torch.cuda.synchronize()
    loss_r, grad_r = _reference(torch, P, lg1, lab1, tl1, ul1, w1.variant)
    torch.cuda.synchronize()
    assert torch.equal(loss_a, loss_r), (loss_a, loss_r)
    assert torch.equal(grad_a, grad_r)
    assert bool(torch.isfinite(loss_a).all())
    del grad_a, grad_r
    # second call, right after: a smaller batch (char, B=16, T_max=150, U_max=40, V=29) on the
    # W-Transducer lattice; the scratch still holds the first call's contents
    w2, lg2, lab2, tl2, ul2 = _inputs(torch, "char")
    loss_b, grad_b = _noalloc(torch, P, lg2, lab2, tl2, ul2, "wrnnt", -777.0)
    torch.cuda.synchronize()
    loss_s, grad_s = _reference(torch, P, lg2, lab2, tl2, ul2, "wrnnt")
    torch.cuda.synchronize()
    assert torch.equal(loss_b, loss_s), (loss_b, loss_s)
    assert torch.equal(grad_b, grad_s)
    assert bool(torch.isfinite(loss_b).all())


def test_noalloc_refuses_a_shape_beyond_the_scratch():
    import torch
    import paper_2303_10384_amd as P
    # the large bf16 batch needs ~316 MiB of workspace: refused on the host, nothing launched
    w = W.WORKLOADS["large"]
    lg = torch.empty((w.B, w.T_max, w.U_max + 1, w.V), dtype=torch.bfloat16, device="cuda:0")
    labels = torch.ones((w.B, w.U_max), dtype=torch.int32, device="cuda:0")
    lens = torch.ones((w.B,), dtype=torch.int32, device="cuda:0")
    loss = torch.empty((w.B,), dtype=torch.float32, device="cuda:0")
    with pytest.raises(P.RNNTError, match="static scratch") as e:
        P.rnnt_loss_noalloc(lg, labels, lens, lens, loss, None)
    assert e.value.status == 11
