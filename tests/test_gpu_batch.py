"""GPU: a batch is the sum of its utterances, and rnnt_loss can be captured.

Every kernel computes an utterance from that utterance's inputs alone.  Where
T_max (U_max+1) V is a multiple of the 16-byte chunk width (8 elements covers
float32 and the 16-bit types), every utterance also starts on a chunk boundary,
so each row is reduced in the same order wherever its utterance sits, and the
batch must give exactly the bits of one-utterance calls.  A captured graph of
the call must give the eager call's bits on every replay, with eager work in
between.
"""
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


def dev(torch, x):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def call(torch, pkg, lg, labels, tl, ul, variant):
    grad = torch.full(lg.shape, float("nan"), dtype=lg.dtype, device=lg.device)
    loss, grad = pkg.rnnt_loss(lg, dev(torch, labels), dev(torch, tl), dev(torch, ul), variant=variant,
                               grad_out=grad)
    torch.cuda.synchronize()
    return loss.cpu(), grad.cpu()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant", ["rnnt", "wrnnt", "wrnnt_allow_ignore"])
@pytest.mark.parametrize("B,T,U,V,seed", [(2, 6, 3, 16, 1), (3, 9, 5, 24, 2), (7, 12, 7, 40, 3),
                                          (5, 16, 15, 64, 4)])
def test_batch_matches_one_utterance_calls(torch, pkg, dtype, variant, B, T, U, V, seed):
    assert (T * (U + 1) * V) % 8 == 0
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=seed, sigma=2.0)
    lg = dev(torch, logits).to(W.torch_dtype(dtype))
    W.poison_padding(lg, tl, ul)
    loss, grad = call(torch, pkg, lg, labels, tl, ul, variant)
    for b in range(B):
        lb, gb = call(torch, pkg, lg[b:b + 1].clone(), labels[b:b + 1], tl[b:b + 1], ul[b:b + 1], variant)
        assert torch.equal(loss[b:b + 1], lb), (b, loss[b].item(), lb.item())
        assert torch.equal(grad[b:b + 1], gb), b


def test_captured_graph_replays_the_eager_bits(torch, pkg):
    B, T, U, V = 6, 20, 9, 48
    logits, tl, ul, labels = W.small_case(B, T, U, V, seed=8, sigma=2.0)
    lg = dev(torch, logits)
    W.poison_padding(lg, tl, ul)
    lab_d, tl_d, ul_d = dev(torch, labels), dev(torch, tl), dev(torch, ul)
    ws = torch.empty(pkg.loss_workspace_bytes(B, T, U, V), dtype=torch.uint8, device="cuda:0")
    grad = torch.empty_like(lg)
    loss = torch.empty(B, dtype=torch.float32, device="cuda:0")

    def step():
        pkg.rnnt_loss(lg, lab_d, tl_d, ul_d, variant="wrnnt", workspace=ws, grad_out=grad, loss_out=loss)

    step()
    torch.cuda.synchronize()
    loss_ref, grad_ref = loss.clone(), grad.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for k in range(3):
        grad.fill_(float("nan"))
        loss.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(loss, loss_ref), k
        assert torch.equal(grad, grad_ref), k
        step()  # eager work between the replays
        torch.cuda.synchronize()
        assert torch.equal(loss, loss_ref) and torch.equal(grad, grad_ref), k
