"""ctypes binding of librnnt_mi355x.so (argument marshalling only).

Every step of the loss runs in the HIP library; torch is used for device
memory and the current stream.  There is no CPU fallback: if the library is
missing or the tensors are not on a GPU, the calls raise.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# another build of the same library may be named by RNNT_MI355X_LIBRARY
LIB_PATH = os.environ.get("RNNT_MI355X_LIBRARY") or os.path.join(PKG, "librnnt_mi355x.so")

RNNT_OK = 0
STATUS_NAMES = {
    0: "RNNT_OK", 1: "RNNT_ERR_NULL_PTR", 2: "RNNT_ERR_BAD_SHAPE", 3: "RNNT_ERR_BAD_BLANK",
    4: "RNNT_ERR_BAD_DTYPE", 5: "RNNT_ERR_BAD_VARIANT", 6: "RNNT_ERR_WORKSPACE", 7: "RNNT_ERR_ALIGNMENT",
    8: "RNNT_ERR_HIP", 9: "RNNT_ERR_UNSUPPORTED", 10: "RNNT_ERR_BAD_LATTICE", 11: "RNNT_ERR_SCRATCH",
}
# bytes of rnnt_loss_noalloc's static device scratch (RNNT_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 64 << 20
VARIANTS = {"rnnt": 0, "wrnnt": 1, "wrnnt_allow_ignore": 2}
DTYPE_F32, DTYPE_BF16, DTYPE_F16 = 0, 1, 2

# every symbol declared in include/rnnt_mi355x.h
EXPORTED = ("rnnt_loss_workspace_bytes", "rnnt_loss", "rnnt_loss_timed", "rnnt_log_softmax_gather", "rnnt_lattice_workspace_bytes",
            "rnnt_lattice_scores", "rnnt_status_string", "rnnt_version", "rnnt_viterbi_workspace_bytes", "rnnt_viterbi",
            "rnnt_viterbi_timed", "rnnt_arc_plan_bytes_bound", "rnnt_arc_plan", "rnnt_arc_loss_workspace_bytes",
            "rnnt_arc_loss", "rnnt_arc_loss_timed", "rnnt_loss_noalloc")


class Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T_max", ctypes.c_int32), ("U_max", ctypes.c_int32),
                ("V", ctypes.c_int32), ("dtype", ctypes.c_int), ("grad_dtype", ctypes.c_int)]


class ArcPlanDesc(ctypes.Structure):
    """rnnt_arc_plan_t."""
    _fields_ = ([(n, ctypes.c_int32) for n in (
        "B", "T_max", "U_max", "V", "blank", "num_states", "num_levels", "num_arcs", "num_row_arcs",
        "num_extra_rows")] + [("num_slots", ctypes.c_int32 * 2)] + [(n, ctypes.c_int32) for n in (
            "max_level_states", "max_level_arcs", "max_in_degree", "max_pins", "state_chunks",
            "slots_per_state")] + [("image_bytes", ctypes.c_int64), ("off", ctypes.c_int64 * 17)])


class RNNTError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s failed: %s (%s)" % (where, STATUS_NAMES.get(status, status), status_string(status)))


_lib = None


def load_library():
    """Load the in-tree library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("librnnt_mi355x.so is not built (run __graft_entry__.build() or "
                           "python -m paper_2303_10384_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.rnnt_loss_workspace_bytes.argtypes = [Shape]
    lib.rnnt_loss_workspace_bytes.restype = sz
    lib.rnnt_lattice_workspace_bytes.argtypes = [Shape]
    lib.rnnt_lattice_workspace_bytes.restype = sz
    lib.rnnt_loss.argtypes = [vp, Shape, vp, vp, vp, i32, ctypes.c_int, vp, vp, vp, sz, vp]
    lib.rnnt_loss.restype = ctypes.c_int
    lib.rnnt_loss_timed.argtypes = [vp, Shape, vp, vp, vp, i32, ctypes.c_int, vp, vp, vp, sz, vp, vp]
    lib.rnnt_loss_timed.restype = ctypes.c_int
    lib.rnnt_loss_noalloc.argtypes = [vp, Shape, vp, vp, vp, i32, ctypes.c_int, vp, vp, vp]
    lib.rnnt_loss_noalloc.restype = ctypes.c_int
    lib.rnnt_log_softmax_gather.argtypes = [vp, Shape, vp, vp, vp, i32, vp, vp, vp, vp]
    lib.rnnt_log_softmax_gather.restype = ctypes.c_int
    lib.rnnt_lattice_scores.argtypes = [vp, vp, Shape, vp, vp, ctypes.c_int, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.rnnt_lattice_scores.restype = ctypes.c_int
    lib.rnnt_viterbi_workspace_bytes.argtypes = [Shape]
    lib.rnnt_viterbi_workspace_bytes.restype = sz
    lib.rnnt_viterbi.argtypes = [vp, Shape, vp, vp, vp, i32, ctypes.c_int, vp, vp, vp, vp, sz, vp]
    lib.rnnt_viterbi.restype = ctypes.c_int
    lib.rnnt_viterbi_timed.argtypes = [vp, Shape, vp, vp, vp, i32, ctypes.c_int, vp, vp, vp, vp, sz, vp, vp]
    lib.rnnt_viterbi_timed.restype = ctypes.c_int
    i64 = ctypes.c_int64
    lib.rnnt_arc_plan_bytes_bound.argtypes = [i32, i32, i32, i64, i64]
    lib.rnnt_arc_plan_bytes_bound.restype = sz
    lib.rnnt_arc_plan.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, sz, ctypes.POINTER(ArcPlanDesc)]
    lib.rnnt_arc_plan.restype = ctypes.c_int
    lib.rnnt_arc_loss_workspace_bytes.argtypes = [ctypes.POINTER(ArcPlanDesc)]
    lib.rnnt_arc_loss_workspace_bytes.restype = sz
    lib.rnnt_arc_loss.argtypes = [vp, Shape, vp, vp, ctypes.POINTER(ArcPlanDesc), vp, vp, vp, vp, sz, vp]
    lib.rnnt_arc_loss.restype = ctypes.c_int
    lib.rnnt_arc_loss_timed.argtypes = [vp, Shape, vp, vp, ctypes.POINTER(ArcPlanDesc), vp, vp, vp, vp, sz, vp, vp]
    lib.rnnt_arc_loss_timed.restype = ctypes.c_int
    lib.rnnt_status_string.argtypes = [ctypes.c_int]
    lib.rnnt_status_string.restype = ctypes.c_char_p
    lib.rnnt_version.argtypes = []
    lib.rnnt_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status):
    return load_library().rnnt_status_string(int(status)).decode()


def version():
    return load_library().rnnt_version().decode()


def _torch():
    import torch
    return torch


def dtype_code(dtype):
    torch = _torch()
    codes = {torch.float32: DTYPE_F32, torch.bfloat16: DTYPE_BF16, torch.float16: DTYPE_F16}
    if dtype not in codes:
        raise TypeError("logits must be float32, bfloat16 or float16, got %s" % dtype)
    return codes[dtype]


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _check_gpu(name, t, dtype=None):
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor (no CPU path exists)" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))


def _stream_handle(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def shape_of(logits, grad_dtype=None):
    B, T, U1, V = logits.shape
    dt = dtype_code(logits.dtype)
    return Shape(B, T, U1 - 1, V, dt, dt if grad_dtype is None else dtype_code(grad_dtype))


def loss_workspace_bytes(B, T_max, U_max, V, dtype_code_=DTYPE_F32):
    return load_library().rnnt_loss_workspace_bytes(Shape(B, T_max, U_max, V, dtype_code_, dtype_code_))


def rnnt_loss(logits, labels, logit_lens, label_lens, blank=0, variant="rnnt", need_grad=True,
              workspace=None, grad_out=None, loss_out=None, events=None, grad_dtype=None):
    """Per-utterance loss (float32, shape (B,)) and gradient (logits' shape and dtype, or None).

    logits (B, T_max, U_max+1, V) float32/bfloat16/float16 on the GPU; labels (B, U_max) int32;
    logit_lens, label_lens (B,) int32.  workspace: optional uint8 GPU tensor of at least
    loss_workspace_bytes(...) bytes; grad_out / loss_out: optional preallocated outputs;
    events: optional ctypes array of 5 hipEvent_t recorded around the kernels;
    grad_dtype: None (the logits' dtype) or torch.float32.
    """
    torch = _torch()
    lib = load_library()
    _check_gpu("logits", logits)
    _check_gpu("labels", labels, torch.int32)
    _check_gpu("logit_lens", logit_lens, torch.int32)
    _check_gpu("label_lens", label_lens, torch.int32)
    if logits.dim() != 4:
        raise ValueError("logits must be (B, T_max, U_max+1, V)")
    if grad_out is not None and grad_dtype is None:
        grad_dtype = grad_out.dtype
    shape = shape_of(logits, grad_dtype)
    if labels.shape != (shape.B, shape.U_max) or logit_lens.shape != (shape.B,) or label_lens.shape != (shape.B,):
        raise ValueError("labels must be (B, U_max) and the length vectors (B,)")
    if variant not in VARIANTS:
        raise ValueError("variant must be one of %s" % sorted(VARIANTS))
    dev = logits.device
    loss = loss_out if loss_out is not None else torch.empty(shape.B, dtype=torch.float32, device=dev)
    _check_gpu("loss_out", loss, torch.float32)
    grad = None
    if need_grad:
        gdt = logits.dtype if grad_dtype is None else grad_dtype
        grad = grad_out if grad_out is not None else torch.empty(logits.shape, dtype=gdt, device=dev)
        _check_gpu("grad_out", grad, gdt)
        if grad.shape != logits.shape:
            raise ValueError("grad_out must have the logits' shape")
    ws_ptr, ws_bytes = ctypes.c_void_p(0), 0
    if workspace is not None:
        _check_gpu("workspace", workspace)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    if events is None:
        st = lib.rnnt_loss(_ptr(logits), shape, _ptr(labels), _ptr(logit_lens), _ptr(label_lens), int(blank),
                           VARIANTS[variant], _ptr(loss), _ptr(grad), ws_ptr, ws_bytes, _stream_handle(dev))
    else:  # host array of 5 hipEvent_t handles
        st = lib.rnnt_loss_timed(_ptr(logits), shape, _ptr(labels), _ptr(logit_lens), _ptr(label_lens),
                                 int(blank), VARIANTS[variant], _ptr(loss), _ptr(grad), ws_ptr, ws_bytes,
                                 _stream_handle(dev), events)
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_loss")
    return loss, grad


def rnnt_loss_noalloc(logits, labels, logit_lens, label_lens, loss_out, grad_out=None, blank=0, variant="rnnt"):
    """rnnt_loss with the library's static device scratch as workspace (no device allocation
    in the library): the caller passes every output, loss_out (B,) float32 and grad_out
    (logits' shape, the logits' dtype or float32) or None for the loss alone.  Returns
    (loss_out, grad_out)."""
    torch = _torch()
    lib = load_library()
    _check_gpu("logits", logits)
    _check_gpu("labels", labels, torch.int32)
    _check_gpu("logit_lens", logit_lens, torch.int32)
    _check_gpu("label_lens", label_lens, torch.int32)
    _check_gpu("loss_out", loss_out, torch.float32)
    if logits.dim() != 4:
        raise ValueError("logits must be (B, T_max, U_max+1, V)")
    shape = shape_of(logits, None if grad_out is None else grad_out.dtype)
    if labels.shape != (shape.B, shape.U_max) or logit_lens.shape != (shape.B,) or label_lens.shape != (shape.B,):
        raise ValueError("labels must be (B, U_max) and the length vectors (B,)")
    if loss_out.shape != (shape.B,):
        raise ValueError("loss_out must be (B,)")
    if grad_out is not None:
        _check_gpu("grad_out", grad_out)
        if grad_out.shape != logits.shape:
            raise ValueError("grad_out must have the logits' shape")
    if variant not in VARIANTS:
        raise ValueError("variant must be one of %s" % sorted(VARIANTS))
    st = lib.rnnt_loss_noalloc(_ptr(logits), shape, _ptr(labels), _ptr(logit_lens), _ptr(label_lens), int(blank),
                               VARIANTS[variant], _ptr(loss_out), _ptr(grad_out), _stream_handle(logits.device))
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_loss_noalloc")
    return loss_out, grad_out


def log_softmax_gather(logits, labels, logit_lens, label_lens, blank=0):
    """(lse, lp_blank, lp_label) float64 (B, T_max, U_max+1); entries outside the valid rows are NaN."""
    torch = _torch()
    lib = load_library()
    _check_gpu("logits", logits)
    shape = shape_of(logits)
    dev = logits.device
    outs = [torch.full((shape.B, shape.T_max, shape.U_max + 1), float("nan"), dtype=torch.float64, device=dev)
            for _ in range(3)]
    st = lib.rnnt_log_softmax_gather(_ptr(logits), shape, _ptr(labels), _ptr(logit_lens), _ptr(label_lens),
                                     int(blank), _ptr(outs[0]), _ptr(outs[1]), _ptr(outs[2]), _stream_handle(dev))
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_log_softmax_gather")
    return tuple(outs)


def lattice_scores(lp_blank, lp_label, logit_lens, label_lens, variant="rnnt"):
    """GPU forward/backward on given float64 lattice weights (B, T_max, U_max+1).

    Returns dict with alpha, beta, occ_blank, occ_label (NaN outside the valid
    nodes), loss and loss_bwd (B,) float64.
    """
    torch = _torch()
    lib = load_library()
    for n, t in (("lp_blank", lp_blank), ("lp_label", lp_label)):
        _check_gpu(n, t, torch.float64)
    B, T, U1 = lp_blank.shape
    shape = Shape(B, T, U1 - 1, 2, DTYPE_F32, DTYPE_F32)
    dev = lp_blank.device
    nan = float("nan")
    out = {k: torch.full((B, T, U1), nan, dtype=torch.float64, device=dev)
           for k in ("alpha", "beta", "occ_blank", "occ_label")}
    out["loss"] = torch.full((B,), nan, dtype=torch.float64, device=dev)
    out["loss_bwd"] = torch.full((B,), nan, dtype=torch.float64, device=dev)
    st = lib.rnnt_lattice_scores(_ptr(lp_blank), _ptr(lp_label), shape, _ptr(logit_lens), _ptr(label_lens),
                                 VARIANTS[variant], _ptr(out["alpha"]), _ptr(out["beta"]), _ptr(out["loss"]),
                                 _ptr(out["loss_bwd"]), _ptr(out["occ_blank"]), _ptr(out["occ_label"]),
                                 ctypes.c_void_p(0), 0, _stream_handle(dev))
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_lattice_scores")
    return out


def viterbi_workspace_bytes(B, T_max, U_max, V, dtype_code_=DTYPE_F32):
    return load_library().rnnt_viterbi_workspace_bytes(Shape(B, T_max, U_max, V, dtype_code_, dtype_code_))


def viterbi_align(logits, labels, logit_lens, label_lens, blank=0, variant="rnnt", workspace=None, outputs=None,
                  events=None):
    """Forced alignment (best path) of every utterance.

    Returns (score (B,) float32 natural-log best path log-probability,
    label_frames (B, U_max) int32 frame of each unit or -1, span (B, 2) int32
    first / last frame of the path).  outputs: optional preallocated (score,
    label_frames, span); events: optional ctypes array of 3 hipEvent_t recorded
    around the two kernels.
    """
    torch = _torch()
    lib = load_library()
    _check_gpu("logits", logits)
    _check_gpu("labels", labels, torch.int32)
    _check_gpu("logit_lens", logit_lens, torch.int32)
    _check_gpu("label_lens", label_lens, torch.int32)
    if logits.dim() != 4:
        raise ValueError("logits must be (B, T_max, U_max+1, V)")
    shape = shape_of(logits)
    if labels.shape != (shape.B, shape.U_max) or logit_lens.shape != (shape.B,) or label_lens.shape != (shape.B,):
        raise ValueError("labels must be (B, U_max) and the length vectors (B,)")
    if variant not in VARIANTS:
        raise ValueError("variant must be one of %s" % sorted(VARIANTS))
    dev = logits.device
    if outputs is None:
        score = torch.empty(shape.B, dtype=torch.float32, device=dev)
        frames = torch.empty((shape.B, shape.U_max), dtype=torch.int32, device=dev)
        span = torch.empty((shape.B, 2), dtype=torch.int32, device=dev)
    else:
        score, frames, span = outputs
        _check_gpu("score", score, torch.float32)
        _check_gpu("label_frames", frames, torch.int32)
        _check_gpu("span", span, torch.int32)
        if score.shape != (shape.B,) or frames.shape != (shape.B, shape.U_max) or span.shape != (shape.B, 2):
            raise ValueError("outputs must be (B,), (B, U_max) and (B, 2)")
    ws_ptr, ws_bytes = ctypes.c_void_p(0), 0
    if workspace is not None:
        _check_gpu("workspace", workspace)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    args = (_ptr(logits), shape, _ptr(labels), _ptr(logit_lens), _ptr(label_lens), int(blank), VARIANTS[variant],
            _ptr(score), _ptr(frames), _ptr(span), ws_ptr, ws_bytes, _stream_handle(dev))
    st = lib.rnnt_viterbi(*args) if events is None else lib.rnnt_viterbi_timed(*args, events)
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_viterbi")
    return score, frames, span


class ArcPlan:
    """A batch of arc-list lattices planned by rnnt_arc_plan: the descriptor
    (`desc`, host) and the image (`image`, a uint8 tensor, on the device once
    `to()` has copied it there)."""

    def __init__(self, desc, image):
        self.desc = desc
        self.image = image

    def to(self, device):
        return ArcPlan(self.desc, self.image.to(device))

    def __getattr__(self, name):  # the descriptor's sizes
        if name in ("desc", "image"):
            raise AttributeError(name)
        return getattr(self.desc, name)


def arc_plan(lattices, T_max, U_max, V, blank=0, device=None):
    """Plan a batch of lattices given as arc lists (host work, in the library).

    lattices: one (n_states, arcs) per utterance, arcs a numpy array of
    topologies.ARC_DTYPE (states local to the utterance).  Returns an ArcPlan,
    its image moved to `device` when given.
    """
    import numpy as np
    from .topologies import ARC_DTYPE
    torch = _torch()
    lib = load_library()
    B = len(lattices)
    num_states = np.array([int(n) for n, _ in lattices], np.int32)
    arc_lists = [np.ascontiguousarray(np.asarray(a, dtype=ARC_DTYPE)) for _, a in lattices]
    counts = np.array([len(a) for a in arc_lists], np.int64)
    arc_begin = np.zeros(B + 1, np.int64)
    np.cumsum(counts, out=arc_begin[1:])
    arcs = np.concatenate(arc_lists) if B else np.zeros(0, ARC_DTYPE)
    arcs = np.ascontiguousarray(arcs, dtype=ARC_DTYPE)
    bound = lib.rnnt_arc_plan_bytes_bound(B, int(T_max), int(U_max), int(num_states.sum()), int(arc_begin[-1]))
    if bound == 0:
        raise RNNTError(2, "rnnt_arc_plan_bytes_bound")
    image = torch.empty(bound, dtype=torch.uint8)
    desc = ArcPlanDesc()
    st = lib.rnnt_arc_plan(B, int(T_max), int(U_max), int(V), int(blank), num_states.ctypes.data,
                           arc_begin.ctypes.data, arcs.ctypes.data if len(arcs) else None,
                           ctypes.c_void_p(image.data_ptr()), bound, ctypes.byref(desc))
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_arc_plan")
    plan = ArcPlan(desc, image[:desc.image_bytes].clone())
    return plan.to(device) if device is not None else plan


def arc_loss_workspace_bytes(plan):
    return load_library().rnnt_arc_loss_workspace_bytes(ctypes.byref(plan.desc))


def arc_loss(logits, logit_lens, label_lens, plan, need_grad=True, workspace=None, grad_out=None, loss_out=None,
             events=None, grad_dtype=None):
    """Per-utterance loss (float32 (B,)) and gradient of a batch of arc-list lattices.

    logits (B, T_max, U_max+1, V) on the GPU; logit_lens, label_lens (B,) int32;
    plan: an ArcPlan whose image is on the logits' device.  events: optional
    ctypes array of 6 hipEvent_t recorded around the kernels.
    """
    torch = _torch()
    lib = load_library()
    _check_gpu("logits", logits)
    _check_gpu("logit_lens", logit_lens, torch.int32)
    _check_gpu("label_lens", label_lens, torch.int32)
    _check_gpu("plan image", plan.image, torch.uint8)
    if logits.dim() != 4:
        raise ValueError("logits must be (B, T_max, U_max+1, V)")
    if grad_out is not None and grad_dtype is None:
        grad_dtype = grad_out.dtype
    shape = shape_of(logits, grad_dtype)
    if logit_lens.shape != (shape.B,) or label_lens.shape != (shape.B,):
        raise ValueError("the length vectors must be (B,)")
    dev = logits.device
    loss = loss_out if loss_out is not None else torch.empty(shape.B, dtype=torch.float32, device=dev)
    _check_gpu("loss_out", loss, torch.float32)
    grad = None
    if need_grad:
        gdt = logits.dtype if grad_dtype is None else grad_dtype
        grad = grad_out if grad_out is not None else torch.empty(logits.shape, dtype=gdt, device=dev)
        _check_gpu("grad_out", grad, gdt)
        if grad.shape != logits.shape:
            raise ValueError("grad_out must have the logits' shape")
    ws_ptr, ws_bytes = ctypes.c_void_p(0), 0
    if workspace is not None:
        _check_gpu("workspace", workspace)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    args = (_ptr(logits), shape, _ptr(logit_lens), _ptr(label_lens), ctypes.byref(plan.desc), _ptr(plan.image),
            _ptr(loss), _ptr(grad), ws_ptr, ws_bytes, _stream_handle(dev))
    st = lib.rnnt_arc_loss(*args) if events is None else lib.rnnt_arc_loss_timed(*args, events)
    if st != RNNT_OK:
        raise RNNTError(st, "rnnt_arc_loss")
    return loss, grad
