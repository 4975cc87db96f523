#!/usr/bin/env python3
"""Benchmark of the fused RNN-T loss + gradient on one MI355X.

One step = one rnnt_loss call with a gradient output (kernel 1 log-normaliser
and gather, kernel 2 lattice sweep and arc posteriors, kernel 3 gradient) over
one batch of the workload, inputs already resident in HBM.  The step time comes
from plain calls with one HIP event at each step boundary; the per-kernel times
from a second loop of the timed entry point, whose events between the kernels
add a few microseconds per step.  Prints ONE JSON
line: throughput in joint-logit elements/s (padded tensor B*T_max*(U_max+1)*V
per step), the achieved HBM bandwidth of the dominant kernel against the
MI355X peak, and the CPU oracle timed on a bounded sample.  With --mode viterbi
a step is one forced alignment of the batch (populate kernel, alignment kernel)
and the line reports that path the same way.  With --mode arc a step is one
rnnt_arc_loss call with a gradient, the workload's lattices given as arc lists
(planned once on the host before timing, like the labels).

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload bpe] [--mode loss|viterbi|arc]
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
ROWREC_BYTES = 16      # per-row record written by kernel 2b and read by kernel 3
PROFILE_DIR = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles through the HIP runtime torch already loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, n):
        arr = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(h)) == 0
            arr[i] = h
        return arr

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) == 0
        return ms.value

    def destroy(self, arr):
        for h in arr:
            self.hip.hipEventDestroy(ctypes.c_void_p(h))


def profiled_traffic(workload, kernel="k3_grad", path_kind="loss"):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter record
    of the path, if it was taken on the kernel sources as they are now; else None."""
    from paper_2303_10384_amd.profiling import SOURCES, source_digest
    path = os.path.join(PROFILE_DIR, "k3_grad_%s_traffic.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_digest") != source_digest(SOURCES[path_kind]):
        return None
    if kernel == "k3_grad":
        return rec.get("hbm_bytes_per_launch")
    return rec.get("kernels", {}).get(kernel, {}).get("hbm_bytes")


def step_times(ev, events, last):
    """(median, mean) step time in ms: the median of each step's own span (its first
    event to its last), and the span of all steps over their number."""
    import numpy as np
    per_step = [ev.elapsed_ms(e[0], e[last]) for e in events]
    mean = ev.elapsed_ms(events[0][0], events[-1][last]) / len(events)
    return float(np.median(per_step)), mean


def plain_step_times(torch, ev, call, steps):
    """(median, mean) step time in ms of `steps` calls with no event inside a call:
    one event at each step boundary on the launch stream; a step's span runs from
    its boundary event to the next."""
    import numpy as np
    hip = ev.hip
    hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    marks = ev.create(steps + 1)
    torch.cuda.synchronize()
    for k in range(steps):
        assert hip.hipEventRecord(ctypes.c_void_p(marks[k]), stream) == 0
        call()
    assert hip.hipEventRecord(ctypes.c_void_p(marks[steps]), stream) == 0
    torch.cuda.synchronize()
    spans = [ev.elapsed_ms(marks[k], marks[k + 1]) for k in range(steps)]
    mean = ev.elapsed_ms(marks[0], marks[steps]) / steps
    ev.destroy(marks)
    return float(np.median(spans)), mean


def algorithmic_bytes(w, tl, ul, s_in, s_out, r_grad=None):
    """Bytes each streaming kernel must move at the least, per launch.

    Kernel 1 reads the logits of the valid rows (t < T_b, u <= U_b) once.
    Kernel 3 reads the logits of the valid rows whose gradient is not identically
    zero (r_grad of them; a row whose arc posteriors both underflow float32 has an
    exactly zero gradient and needs no logits) and the per-row record of every
    padded row, and writes the whole gradient (zeros in the padding rows).  The
    lattice arrays of kernels 2 / 2b (a few MB) are left out.  The step as a whole
    must read the valid logits once for the normalisers and those r_grad rows a
    second time (the arc posteriors depend on every row's normaliser), and write
    the whole gradient once.  r_grad defaults to every valid row."""
    import numpy as np
    r_valid = int(np.sum(tl.astype(np.int64) * (ul.astype(np.int64) + 1)))
    r_total = w.B * w.T_max * (w.U_max + 1)
    r_grad = r_valid if r_grad is None else int(r_grad)
    V = w.V
    return {
        "valid_rows": r_valid,
        "padded_rows": r_total,
        "gradient_rows": r_grad,
        "k1_populate": r_valid * V * s_in,
        "k3_grad": r_grad * V * s_in + r_total * V * s_out + r_total * ROWREC_BYTES,
        "step": (r_valid + r_grad) * V * s_in + r_total * V * s_out,
    }


def gradient_rows(torch, grad, tl, ul):
    """Valid rows whose gradient holds a nonzero element (the rows whose logits the
    gradient needs), counted on the device one utterance at a time."""
    n = 0
    for b in range(grad.shape[0]):
        g = grad[b, :int(tl[b]), :int(ul[b]) + 1]
        n += int((g != 0).any(dim=-1).sum().item())
    return n


def gradient_rows_f32(torch, grad, tl, ul, call_f32):
    """gradient_rows, counted on a float32 gradient: a 16-bit store can round all of a
    row's tiny but nonzero elements to 0 (fp16's range ends at 6e-8), though the row's
    logits were read to form them.  call_f32(g32) runs the step once more (untimed)
    with a float32 gradient into g32."""
    if grad.dtype == torch.float32:
        return gradient_rows(torch, grad, tl, ul)
    g32 = torch.empty(grad.shape, dtype=torch.float32, device=grad.device)
    call_f32(g32)
    if g32.is_cuda:
        torch.cuda.synchronize()
    n = gradient_rows(torch, g32, tl, ul)
    del g32
    return n


def cpu_oracle_worker(args):
    import numpy as np

    from oracle import arc_lattice, rnnt_ref, viterbi
    from paper_2303_10384_amd import topologies
    T_b, U_b, V, sigma, seed, labels, variant, mode = args
    z = np.random.default_rng(seed).standard_normal((T_b, U_b + 1, V), dtype=np.float32) * np.float32(sigma)
    if mode == "arc":
        n, arcs = topologies.grid_lattice(T_b, U_b, labels, 0, variant)
        arcs = [(int(a["src"]), int(a["dst"]), int(a["t"]), int(a["u"]), int(a["label"]), float(a["score"]))
                for a in arcs]
    t0 = time.perf_counter()
    if mode == "viterbi":
        viterbi.utterance_alignment(z.astype(np.float64), labels, 0, variant)
    elif mode == "arc":
        arc_lattice.arc_lattice_loss_grad(z.astype(np.float64), arcs, n)
    else:
        rnnt_ref.utterance_loss_grad(z.astype(np.float64), labels, 0, variant, need_grad=True)
    return time.perf_counter() - t0


def cpu_baseline(w, tl, ul, labels, budget_s, mode="loss"):
    """Time the float64 oracle (loss + gradient) on utterances of this workload
    (same lengths and labels, logits freshly drawn on the host with the same
    distribution), spread over a process pool.  Runs before the GPU is touched,
    so the workers are plain forks.  The pool takes the process's CPUs up to 16,
    the CPU share that goes with one GPU on the machines this is measured on."""
    import multiprocessing as mp

    available = len(os.sched_getaffinity(0))
    cores = max(1, min(16, available))
    per_utt_elems = w.T_max * (w.U_max + 1) * w.V
    jobs = [(int(tl[b]), int(ul[b]), w.V, w.sigma, w.seed * 1000 + b, labels[b, :int(ul[b])].copy(), w.variant,
             mode) for b in range(w.B)]
    ctx = mp.get_context("fork")
    with ctx.Pool(cores) as pool:
        pool.map(cpu_oracle_worker, jobs[:cores])  # warm-up round (worker start-up, first imports)
        # one pass over the batch sizes the sample: the mean of the evaluations' own times
        t_eval = sum(pool.map(cpu_oracle_worker, jobs)) / len(jobs)
        # cycle through the batch's utterances until about budget_s of work per worker is queued
        n_eval = max(min(cores, len(jobs)), int(budget_s * min(cores, len(jobs)) / max(t_eval, 1e-4)))
        sample = [jobs[i % len(jobs)] for i in range(n_eval)]
        log("[bench] cpu oracle: %.3f s per utterance evaluation; timing %d evaluations" % (t_eval, len(sample)))
        t0 = time.perf_counter()
        per_eval = pool.map(cpu_oracle_worker, sample)  # each evaluation's own time, in its worker
        wall = time.perf_counter() - t0
    n = len(sample)
    used = min(cores, n)
    busy = sum(per_eval) / used  # oracle time per worker, the logits' drawing excluded
    return {
        "value": n * per_utt_elems / busy,
        "unit": "joint-logit elements/s",
        "cores": used,
        "cores_available": available,
        "kind": "oracle",
        "single_core_value": n * per_utt_elems / sum(per_eval),
        "sample": "%d utterance evaluations cycling through the %d utterances of the batch (their lengths and "
                  "labels; logits freshly drawn on the host from N(0,%g), the workload's distribution, not copied "
                  "from the GPU's tensor), float64 %s, %d worker processes running at once, %.1f s of oracle "
                  "time per worker (%.1f s wall, which also draws the logits); elements counted as padded rows x V "
                  "like the GPU value" % (n, w.B, w.sigma,
                                          {"viterbi": "forced alignment",
                                           "arc": "arc-list loss + gradient (oracle/arc_lattice.py)"}.get(
                                              mode, "loss + gradient"),
                                          used, busy, wall),
    }


def copy_probe(torch, w, steps):
    """Plain device-to-device copies of a known size (the gradient tensor's bytes):
    the reference reading for the FETCH_SIZE / WRITE_SIZE counters."""
    nbytes = w.B * w.T_max * (w.U_max + 1) * w.V * 4
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "copies": steps}), flush=True)


def viterbi_bench(args, w, tl, ul, logits, labels_d, tl_d, ul_d, cpu):
    """Forced alignment of the workload's batch: populate kernel + alignment kernel
    (sweep and backtrace) per step, timed with HIP events on the launch stream."""
    import numpy as np
    import torch

    from paper_2303_10384_amd import binding
    dev = logits.device
    outs = (torch.empty(w.B, dtype=torch.float32, device=dev),
            torch.empty((w.B, w.U_max), dtype=torch.int32, device=dev),
            torch.empty((w.B, 2), dtype=torch.int32, device=dev))
    ws = torch.empty(binding.viterbi_workspace_bytes(w.B, w.T_max, w.U_max, w.V, binding.dtype_code(logits.dtype)),
                     dtype=torch.uint8, device=dev)
    call = lambda ev=None: binding.viterbi_align(logits, labels_d, tl_d, ul_d, 0, w.variant, ws, outs, ev)  # noqa: E731
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    log("[bench] warmup done")
    ev = HipEvents()
    events = [ev.create(3) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        call(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    k_ms = [[ev.elapsed_ms(e[i], e[i + 1]) for i in range(2)] for e in events]
    ms_inst, _ = step_times(ev, events, 2)
    for e in events:
        ev.destroy(e)
    ms_per_step, ms_mean = plain_step_times(torch, ev, call, args.steps)
    k1_ms, kv_ms = (float(np.mean([r[i] for r in k_ms])) for i in range(2))
    log("[bench] per step %.4f ms median, %.4f mean (instrumented %.4f, wall %.4f ms): k1 %.4f  k2_viterbi %.4f ms"
        % (ms_per_step, ms_mean, ms_inst, wall * 1e3 / args.steps, k1_ms, kv_ms))
    ab = algorithmic_bytes(w, tl, ul, logits.element_size(), logits.element_size())
    elems = ab["padded_rows"] * w.V
    k1_gbs = ab["k1_populate"] / (k1_ms * 1e-3) / 1e9
    result = {
        "metric": "forced-alignment joint-logit elements/sec (best path and its frames) and achieved HBM GB/s vs peak",
        "value": elems / (ms_per_step * 1e-3),
        "valid_elements_per_s": ab["valid_rows"] * w.V / (ms_per_step * 1e-3),
        "unit": "joint-logit elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_mean": round(ms_mean, 5),
        "ms_per_step_instrumented": round(ms_inst, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.describe() + " forced alignment",
            "B": w.B, "T_max": w.T_max, "U_max": w.U_max, "V": w.V, "variant": w.variant,
            "valid_rows": ab["valid_rows"], "padded_rows": ab["padded_rows"],
            "lattice_scores": "f64", "softmax": "f32",
        },
        "hbm_gbs_step": round(ab["k1_populate"] / (ms_per_step * 1e-3) / 1e9, 1),
        "hbm_frac_step": round(ab["k1_populate"] / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "kernel_ms": {"k1_populate": round(k1_ms, 5), "k2_viterbi": round(kv_ms, 5)},
        "kernel_gbs": {"k1_populate": round(k1_gbs, 1)},
        "algorithmic_bytes": {"k1_populate": ab["k1_populate"], "step": ab["k1_populate"]},
        "roofline": {
            "bound": "hbm",
            "kernel": "k1_populate (row log-normaliser and gather)",
            "achieved": round(k1_gbs, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(k1_gbs / PEAK_HBM_GBS, 4),
            "traffic": profiled_traffic(args.workload, "k1_populate") if args.traffic_ok else None,
            "bytes_per_launch": ab["k1_populate"],
            "launch_ms": round(k1_ms, 5),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


def arc_bench(args, w, tl, ul, labels, logits, tl_d, ul_d, cpu):
    """The loss over the workload's lattices given as arc lists: kernel 1 (rows form),
    arc populate, the two level sweeps, row records, kernel 3 (+ rows with several
    labels) per step, timed with HIP events on the launch stream."""
    import numpy as np
    import torch

    from paper_2303_10384_amd import binding, topologies
    dev = logits.device
    t0 = time.perf_counter()
    lattices = topologies.batch_grid_lattices(tl, ul, labels, 0, w.variant)
    plan = binding.arc_plan(lattices, w.T_max, w.U_max, w.V, 0, device=dev)
    plan_s = time.perf_counter() - t0
    log("[bench] arc lists: %d states, %d arcs, %d levels; planned in %.2f s (host)"
        % (plan.num_states, plan.num_arcs, plan.num_levels, plan_s))
    grad = torch.empty_like(logits)
    loss = torch.empty(w.B, dtype=torch.float32, device=dev)
    ws = torch.empty(binding.arc_loss_workspace_bytes(plan), dtype=torch.uint8, device=dev)
    call = lambda ev=None: binding.arc_loss(logits, tl_d, ul_d, plan, True, ws, grad, loss, ev)  # noqa: E731
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    log("[bench] warmup done")
    ev = HipEvents()
    events = [ev.create(6) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        call(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    k_ms = [[ev.elapsed_ms(e[i], e[i + 1]) for i in range(5)] for e in events]
    ms_inst, _ = step_times(ev, events, 5)
    for e in events:
        ev.destroy(e)
    ms_per_step, ms_mean = plain_step_times(torch, ev, call, args.steps)
    k1_ms, kp_ms, ks_ms, kr_ms, k3_ms = (float(np.mean([r[i] for r in k_ms])) for i in range(5))
    log("[bench] per step %.4f ms median, %.4f mean (instrumented %.4f, wall %.4f ms): k1 %.4f  populate %.4f  "
        "sweep %.4f  rows %.4f  k3 %.4f ms" % (ms_per_step, ms_mean, ms_inst, wall * 1e3 / args.steps, k1_ms, kp_ms,
                                               ks_ms, kr_ms, k3_ms))
    r_grad = gradient_rows_f32(torch, grad, tl, ul,
                               lambda g32: binding.arc_loss(logits, tl_d, ul_d, plan, True, ws, g32, loss))
    ab = algorithmic_bytes(w, tl, ul, logits.element_size(), grad.element_size(), r_grad)
    elems = ab["padded_rows"] * w.V
    k3_gbs = ab["k3_grad"] / (k3_ms * 1e-3) / 1e9
    result = {
        "metric": "arc-list lattice loss+grad joint-logit elements/sec and achieved HBM GB/s vs peak",
        "value": elems / (ms_per_step * 1e-3),
        "valid_elements_per_s": ab["valid_rows"] * w.V / (ms_per_step * 1e-3),
        "unit": "joint-logit elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_mean": round(ms_mean, 5),
        "ms_per_step_instrumented": round(ms_inst, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.describe() + " as arc lists",
            "B": w.B, "T_max": w.T_max, "U_max": w.U_max, "V": w.V, "variant": w.variant,
            "valid_rows": ab["valid_rows"], "padded_rows": ab["padded_rows"], "gradient_rows": ab["gradient_rows"],
            "states": plan.num_states, "arcs": plan.num_arcs, "levels": plan.num_levels,
            "plan": "built once on the host before timing (%.2f s), image %d bytes on the device"
                    % (plan_s, plan.image_bytes),
            "lattice_scores": "f64", "softmax": "f32",
        },
        "hbm_gbs_step": round(ab["step"] / (ms_per_step * 1e-3) / 1e9, 1),
        "hbm_frac_step": round(ab["step"] / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "kernel_ms": {"k1_populate": round(k1_ms, 5), "arc_populate": round(kp_ms, 5), "arc_sweep": round(ks_ms, 5),
                      "arc_rows": round(kr_ms, 5), "k3_grad": round(k3_ms, 5)},
        "kernel_gbs": {"k1_populate": round(ab["k1_populate"] / (k1_ms * 1e-3) / 1e9, 1), "k3_grad": round(k3_gbs, 1)},
        "algorithmic_bytes": {"k1_populate": ab["k1_populate"], "k3_grad": ab["k3_grad"], "step": ab["step"]},
        "roofline": {
            "bound": "hbm",
            "kernel": "k3_grad (fused gradient)",
            "achieved": round(k3_gbs, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(k3_gbs / PEAK_HBM_GBS, 4),
            "traffic": profiled_traffic(args.workload + "_arc", "k3_grad", "arc") if args.traffic_ok else None,
            "bytes_per_launch": ab["k3_grad"],
            "launch_ms": round(k3_ms, 5),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="bpe", choices=["tiny", "char", "bpe", "wrnnt", "large"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle work per worker to time")
    ap.add_argument("--dtype", default=None, choices=["f32", "bf16", "f16"],
                    help="logits dtype in place of the workload's own (same draws, rounded)")
    ap.add_argument("--mode", default="loss", choices=["loss", "viterbi", "arc"],
                    help="loss: the fused loss + gradient (the headline metric); viterbi: forced alignment; "
                         "arc: the loss + gradient over the workload's lattices given as arc lists")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run --steps device-to-device copies of the workload's gradient size (the "
                         "known-size copy that calibrates the HBM byte counters), then exit")
    args = ap.parse_args()
    args.traffic_ok = True  # cleared when --dtype changes the workload's logits dtype
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (utterances are "
              "independent, so a batch shards by utterance across processes). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2303_10384_amd import binding
    from paper_2303_10384_amd import workloads as W

    w = W.WORKLOADS[args.workload]
    if args.dtype is not None and args.dtype != w.dtype:
        # the same shapes, lengths, labels and normal draws, rounded to another logits dtype;
        # the committed counter records are of the workload's own dtype, so no traffic is reported
        import dataclasses
        w = dataclasses.replace(w, dtype=args.dtype)
        args.traffic_ok = False
    if args.copy_probe:
        copy_probe(torch, w, args.steps)
        return
    log("[bench] workload", w.describe())
    tl, ul, labels = W.make_lengths_labels(w)
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle (budget %.0f s)" % args.cpu_budget)
        cpu = cpu_baseline(w, tl, ul, labels, args.cpu_budget, args.mode)
        log("[bench] cpu oracle: %.3g elements/s on %d cores" % (cpu["value"], cpu["cores"]))

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    binding.load_library()
    logits = W.make_logits(w, dev)
    labels_d = torch.from_numpy(labels).to(dev)
    tl_d = torch.from_numpy(tl).to(dev)
    ul_d = torch.from_numpy(ul).to(dev)
    if args.mode == "viterbi":
        viterbi_bench(args, w, tl, ul, logits, labels_d, tl_d, ul_d, cpu)
        return
    if args.mode == "arc":
        arc_bench(args, w, tl, ul, labels, logits, tl_d, ul_d, cpu)
        return
    grad = torch.empty_like(logits)
    loss = torch.empty(w.B, dtype=torch.float32, device=dev)
    ws = torch.empty(binding.loss_workspace_bytes(w.B, w.T_max, w.U_max, w.V, binding.dtype_code(logits.dtype)),
                     dtype=torch.uint8, device=dev)
    call = lambda ev=None: binding.rnnt_loss(logits, labels_d, tl_d, ul_d, 0, w.variant, True, ws, grad,  # noqa: E731
                                             loss, ev)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    log("[bench] warmup done")

    ev = HipEvents()
    events = [ev.create(5) for _ in range(args.steps)]
    torch.cuda.synchronize()  # barrier: one process, one GPU
    t0 = time.perf_counter()
    for k in range(args.steps):
        call(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    k_ms = [[ev.elapsed_ms(e[i], e[i + 1]) for i in range(4)] for e in events]
    ms_inst, _ = step_times(ev, events, 4)
    for e in events:
        ev.destroy(e)
    ms_per_step, ms_mean = plain_step_times(torch, ev, call, args.steps)
    k1_ms, k2_ms, k2b_ms, k3_ms = (float(np.mean([r[i] for r in k_ms])) for i in range(4))
    log("[bench] per step %.4f ms median, %.4f mean (instrumented %.4f, wall %.4f ms): k1 %.4f  k2 %.4f  k2b %.4f  "
        "k3 %.4f ms" % (ms_per_step, ms_mean, ms_inst, wall * 1e3 / args.steps, k1_ms, k2_ms, k2b_ms, k3_ms))

    r_grad = gradient_rows_f32(torch, grad, tl, ul, lambda g32: binding.rnnt_loss(
        logits, labels_d, tl_d, ul_d, 0, w.variant, True, ws, g32, loss))
    ab = algorithmic_bytes(w, tl, ul, logits.element_size(), grad.element_size(), r_grad)
    r_valid, r_total, V = ab["valid_rows"], ab["padded_rows"], w.V
    elems = r_total * V
    k1_bytes, k3_bytes, step_bytes = ab["k1_populate"], ab["k3_grad"], ab["step"]
    k3_gbs = k3_bytes / (k3_ms * 1e-3) / 1e9
    traffic = profiled_traffic(args.workload) if args.traffic_ok else None
    roofline = {
        "bound": "hbm",
        "kernel": "k3_grad (fused gradient)",
        "achieved": round(k3_gbs, 1),
        "peak": PEAK_HBM_GBS,
        "unit": "GB/s",
        "frac": round(k3_gbs / PEAK_HBM_GBS, 4),
        "traffic": traffic,
        "bytes_per_launch": k3_bytes,
        "launch_ms": round(k3_ms, 5),
    }
    result = {
        "metric": "joint-logit elements/sec (loss+grad fwd/bwd) and achieved HBM GB/s vs peak",
        "value": elems / (ms_per_step * 1e-3),
        "valid_elements_per_s": r_valid * V / (ms_per_step * 1e-3),
        "unit": "joint-logit elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_mean": round(ms_mean, 5),
        "ms_per_step_instrumented": round(ms_inst, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "bf16": "bf16", "f16": "f16"}[w.dtype],
        "data": "synthetic",
        "config": {
            "workload": w.describe(),
            "B": w.B, "T_max": w.T_max, "U_max": w.U_max, "V": V, "variant": w.variant,
            "valid_rows": r_valid, "padded_rows": r_total, "gradient_rows": ab["gradient_rows"],
            "lattice_scores": "f64", "softmax": "f32",
        },
        "hbm_gbs_step": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "hbm_frac_step": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "kernel_ms": {"k1_populate": round(k1_ms, 5), "k2_lattice": round(k2_ms, 5),
                      "k2b_posteriors": round(k2b_ms, 5), "k3_grad": round(k3_ms, 5)},
        "kernel_gbs": {"k1_populate": round(k1_bytes / (k1_ms * 1e-3) / 1e9, 1), "k3_grad": round(k3_gbs, 1)},
        "algorithmic_bytes": {"k1_populate": k1_bytes, "k3_grad": k3_bytes, "step": step_bytes},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
