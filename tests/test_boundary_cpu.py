"""The C-ABI library without a GPU: it loads, exports every declared symbol,
sizes its workspace as documented, and rejects bad arguments with the right
status before touching the device (no compute call is made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rnnt_mi355x.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2303_10384_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2303_10384_amd import build
        build.build(verbose=False)
    return binding.load_library()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rnnt_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_documented_entry_points():
    names = declared_functions()
    assert names == sorted(["rnnt_loss_workspace_bytes", "rnnt_loss", "rnnt_loss_timed", "rnnt_log_softmax_gather",
                            "rnnt_lattice_workspace_bytes", "rnnt_lattice_scores", "rnnt_status_string",
                            "rnnt_version", "rnnt_viterbi_workspace_bytes", "rnnt_viterbi",
                            "rnnt_viterbi_timed", "rnnt_arc_plan_bytes_bound", "rnnt_arc_plan",
                            "rnnt_arc_loss_workspace_bytes", "rnnt_arc_loss", "rnnt_arc_loss_timed",
                            "rnnt_loss_noalloc"])


def test_every_declared_symbol_is_exported(lib):
    from paper_2303_10384_amd import binding
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert sorted(binding.EXPORTED) == declared_functions()


def test_status_strings_and_version(lib):
    from paper_2303_10384_amd import binding
    for code in range(12):
        assert binding.status_string(code) and binding.status_string(code) != "unknown status"
    assert binding.status_string(12) == "unknown status"
    assert binding.status_string(0) == "ok"
    assert "gfx950" in binding.version()


def shape(B=2, T=5, U=3, V=7, dt=0, gdt=None):
    from paper_2303_10384_amd.binding import Shape
    return Shape(B, T, U, V, dt, dt if gdt is None else gdt)


def expected_workspace(B, T, U, V):
    a = lambda x: (x + 255) // 256 * 256  # noqa: E731
    rows = B * T * (U + 1)
    cells = B * T * (U + 1)                  # lattice cells, one per logits row
    K = next(k for k in (1, 2, 3, 4, 6, 8, 12, 16, 24, 32) if U + 1 <= 64 * k or k == 32)  # units per lane of the sweep
    score_cells = B * (T + U + 1) * 64 * K  # rows 64*K wide, plus one spare diagonal per utterance
    o = a(rows * 16)               # row records
    o = a(o + cells * 16)          # {lp_blank, lp_label}, lse2f in their low bits
    o = a(o + score_cells * 8)     # alpha
    o = a(o + score_cells * 8)     # beta
    o = a(o + 2 * B * 8)           # log P forward / backward
    return a(o + B * 4)            # status


@pytest.mark.parametrize("B,T,U,V", [(1, 1, 0, 2), (2, 20, 8, 16), (32, 250, 80, 1025), (64, 500, 150, 1025),
                                     (1, 3, 1535, 4), (1, 2, 2047, 3)])
def test_workspace_size(lib, B, T, U, V):
    assert lib.rnnt_loss_workspace_bytes(shape(B, T, U, V)) == expected_workspace(B, T, U, V)


def test_workspace_size_of_bad_shape_is_zero(lib):
    assert lib.rnnt_loss_workspace_bytes(shape(B=0)) == 0
    assert lib.rnnt_loss_workspace_bytes(shape(V=1)) == 0
    assert lib.rnnt_loss_workspace_bytes(shape(dt=7)) == 0


FAKE = 1 << 20  # aligned, never dereferenced: every call below fails validation first


def call_loss(lib, sh, logits=FAKE, labels=FAKE, tl=FAKE, ul=FAKE, blank=0, variant=0, loss=FAKE, grad=FAKE,
              ws=0, ws_bytes=0):
    vp = ctypes.c_void_p
    return lib.rnnt_loss(vp(logits), sh, vp(labels), vp(tl), vp(ul), blank, variant, vp(loss), vp(grad), vp(ws),
                         ws_bytes, vp(0))


def test_rnnt_loss_host_errors(lib):
    assert call_loss(lib, shape(B=0)) == 2
    assert call_loss(lib, shape(T=0)) == 2
    assert call_loss(lib, shape(U=-1)) == 2
    assert call_loss(lib, shape(V=1)) == 2
    assert call_loss(lib, shape(dt=3)) == 4
    assert call_loss(lib, shape(dt=0, gdt=1)) == 4   # fp32 logits, bf16 gradient: not offered
    assert call_loss(lib, shape(dt=1, gdt=2)) == 4
    assert call_loss(lib, shape(), logits=0) == 1
    assert call_loss(lib, shape(), labels=0) == 1
    assert call_loss(lib, shape(), tl=0) == 1
    assert call_loss(lib, shape(), ul=0) == 1
    assert call_loss(lib, shape(), loss=0) == 1
    assert call_loss(lib, shape(), blank=-1) == 3
    assert call_loss(lib, shape(), blank=7) == 3
    assert call_loss(lib, shape(), variant=3) == 5
    assert call_loss(lib, shape(), logits=FAKE + 4) == 7
    assert call_loss(lib, shape(), grad=FAKE + 8) == 7
    assert call_loss(lib, shape(U=2048)) == 9
    assert call_loss(lib, shape(B=1, T=65536, U=2047, V=2)) == 9  # the lattice form's 2^31-byte buffer
    assert call_loss(lib, shape(B=1, T=65535, U=2047, V=2), ws=FAKE, ws_bytes=0) == 6  # fits: on to the workspace
    need = lib.rnnt_loss_workspace_bytes(shape())
    assert call_loss(lib, shape(), ws=FAKE, ws_bytes=need - 1) == 6
    assert call_loss(lib, shape(), ws=FAKE + 16, ws_bytes=need) == 7


def call_noalloc(lib, sh, logits=FAKE, labels=FAKE, tl=FAKE, ul=FAKE, blank=0, variant=0, loss=FAKE, grad=FAKE):
    vp = ctypes.c_void_p
    return lib.rnnt_loss_noalloc(vp(logits), sh, vp(labels), vp(tl), vp(ul), blank, variant, vp(loss), vp(grad),
                                 vp(0))


def test_noalloc_scratch_size_matches_header():
    from paper_2303_10384_amd import binding
    m = re.search(r"#define RNNT_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == binding.NOALLOC_SCRATCH_BYTES


def test_noalloc_host_errors(lib):
    # every check below returns before any HIP call (there is no device here)
    from paper_2303_10384_amd import binding
    assert call_noalloc(lib, shape(B=0)) == 2
    assert call_noalloc(lib, shape(dt=3)) == 4
    assert call_noalloc(lib, shape(), logits=0) == 1
    assert call_noalloc(lib, shape(), loss=0) == 1
    assert call_noalloc(lib, shape(), blank=7) == 3
    assert call_noalloc(lib, shape(), variant=3) == 5
    assert call_noalloc(lib, shape(), grad=FAKE + 8) == 7
    assert call_noalloc(lib, shape(U=2048)) == 9
    # the largest batch of bpe rows that fits, and one utterance more
    cap = binding.NOALLOC_SCRATCH_BYTES
    assert lib.rnnt_loss_workspace_bytes(shape(32, 250, 80, 1025)) <= cap
    B = 32
    while lib.rnnt_loss_workspace_bytes(shape(B + 1, 250, 80, 1025)) <= cap:
        B += 1
    assert call_noalloc(lib, shape(B + 1, 250, 80, 1025)) == 11
    assert call_noalloc(lib, shape(64, 500, 150, 1025, dt=1)) == 11  # the large bf16 batch needs ~0.4 GB
    assert "static scratch" in binding.status_string(11)


def test_other_entry_points_host_errors(lib):
    vp = ctypes.c_void_p
    st = lib.rnnt_log_softmax_gather(vp(FAKE), shape(), vp(FAKE), vp(FAKE), vp(FAKE), 9, vp(FAKE), vp(FAKE),
                                     vp(FAKE), vp(0))
    assert st == 3
    st = lib.rnnt_log_softmax_gather(vp(FAKE), shape(), vp(FAKE), vp(FAKE), vp(FAKE), 0, vp(FAKE), vp(0),
                                     vp(FAKE), vp(0))
    assert st == 1
    st = lib.rnnt_lattice_scores(vp(FAKE), vp(FAKE), shape(), vp(FAKE), vp(FAKE), 4, vp(0), vp(0), vp(0), vp(0),
                                 vp(0), vp(0), vp(0), 0, vp(0))
    assert st == 5
    st = lib.rnnt_lattice_scores(vp(0), vp(FAKE), shape(), vp(FAKE), vp(FAKE), 0, vp(0), vp(0), vp(0), vp(0),
                                 vp(0), vp(0), vp(0), 0, vp(0))
    assert st == 1
    need = lib.rnnt_lattice_workspace_bytes(shape())
    st = lib.rnnt_lattice_scores(vp(FAKE), vp(FAKE), shape(), vp(FAKE), vp(FAKE), 0, vp(0), vp(0), vp(0), vp(0),
                                 vp(0), vp(0), vp(FAKE), need - 1, vp(0))
    assert st == 6


def expected_viterbi_workspace(B, T, U, V):
    a = lambda x: (x + 255) // 256 * 256  # noqa: E731
    cells = B * T * (U + 1)
    K = next(k for k in (1, 2, 3, 4, 6, 8, 12, 16, 24, 32) if U + 1 <= 64 * k or k == 32)
    o = a(cells * 16)                    # {lp_blank, lp_label}, lse2f in their low bits
    return a(o + B * (T + U + 1) * K * 8)  # decision words


@pytest.mark.parametrize("B,T,U,V", [(1, 1, 0, 2), (32, 250, 80, 1025), (3, 7, 200, 9), (2, 5, 1023, 3),
                                     (2, 5, 2047, 3)])
def test_viterbi_workspace_size(lib, B, T, U, V):
    assert lib.rnnt_viterbi_workspace_bytes(shape(B, T, U, V)) == expected_viterbi_workspace(B, T, U, V)
    assert lib.rnnt_viterbi_workspace_bytes(shape(B=0)) == 0


def call_viterbi(lib, sh, logits=FAKE, labels=FAKE, tl=FAKE, ul=FAKE, blank=0, variant=0, score=FAKE,
                 frames=FAKE, span=0, ws=None, ws_bytes=None):
    vp = ctypes.c_void_p
    if ws is None:  # a workspace one byte short: every call stops before any device work
        ws, ws_bytes = FAKE, max(0, lib.rnnt_viterbi_workspace_bytes(sh) - 1)
    return lib.rnnt_viterbi(vp(logits), sh, vp(labels), vp(tl), vp(ul), blank, variant, vp(score), vp(frames),
                            vp(span), vp(ws), ws_bytes, vp(0))


def test_viterbi_host_errors(lib):
    assert call_viterbi(lib, shape(B=0)) == 2
    assert call_viterbi(lib, shape(V=1)) == 2
    assert call_viterbi(lib, shape(dt=3)) == 4
    assert call_viterbi(lib, shape(), logits=0) == 1
    assert call_viterbi(lib, shape(), labels=0) == 1
    assert call_viterbi(lib, shape(), score=0) == 1
    assert call_viterbi(lib, shape(), frames=0) == 1
    assert call_viterbi(lib, shape(), blank=7) == 3
    assert call_viterbi(lib, shape(), variant=3) == 5
    assert call_viterbi(lib, shape(), logits=FAKE + 4) == 7
    assert call_viterbi(lib, shape(U=2048)) == 9
    assert call_viterbi(lib, shape(B=1, T=65536, U=2047, V=2)) == 9
    assert call_viterbi(lib, shape()) == 6  # workspace one byte short
    need = lib.rnnt_viterbi_workspace_bytes(shape())
    assert call_viterbi(lib, shape(), ws=FAKE + 16, ws_bytes=need) == 7


def test_binding_refuses_cpu_tensors(lib):
    import torch
    from paper_2303_10384_amd import rnnt_loss
    x = torch.zeros(1, 2, 2, 3)
    with pytest.raises(ValueError, match="GPU"):
        rnnt_loss(x, torch.zeros(1, 1, dtype=torch.int32), torch.ones(1, dtype=torch.int32),
                  torch.ones(1, dtype=torch.int32))


def test_arc_loss_host_errors(lib):
    from paper_2303_10384_amd import binding, topologies
    plan = binding.arc_plan(topologies.batch_grid_lattices([5, 4], [3, 2], [[1, 2, 3], [4, 5, 0]]), 5, 3, 7, 0)
    d = plan.desc
    vp = ctypes.c_void_p
    need = lib.rnnt_arc_loss_workspace_bytes(ctypes.byref(d))
    assert need > 0 and lib.rnnt_arc_loss_workspace_bytes(None) == 0

    def call(sh, logits=FAKE, tl=FAKE, ul=FAKE, desc=d, image=FAKE, loss=FAKE, grad=FAKE, ws=FAKE, ws_bytes=None):
        return lib.rnnt_arc_loss(vp(logits), sh, vp(tl), vp(ul), ctypes.byref(desc) if desc is not None else None,
                                 vp(image), vp(loss), vp(grad), vp(ws), need - 1 if ws_bytes is None else ws_bytes,
                                 vp(0))
    sh = shape(2, 5, 3, 7)
    assert call(sh) == 6                        # everything right but a workspace one byte short
    assert call(shape(B=0)) == 2
    assert call(sh, logits=0) == 1
    assert call(sh, desc=None) == 1
    assert call(sh, image=0) == 1
    assert call(sh, loss=0) == 1
    assert call(shape(2, 5, 3, 8)) == 10        # the plan was made for V = 7
    assert call(shape(3, 5, 3, 7)) == 10
    assert call(sh, image=FAKE + 8) == 7
    assert call(sh, ws=FAKE + 16, ws_bytes=need) == 7
    bad = binding.ArcPlanDesc.from_buffer_copy(d)
    bad.off[3] = bad.off[2] - 256               # offsets out of order
    assert call(sh, desc=bad) == 10
