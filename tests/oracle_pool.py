"""Worker side of the full-size parity tests: the float64 oracle on one utterance
at a time, in a pool of processes started by spawn (they import numpy and the
oracle only, never torch or the GPU library).

An utterance travels as the raw element bits the GPU consumed: float32 values,
or the 16-bit patterns of bfloat16 / float16, widened here exactly to float64.
"""
import multiprocessing
import os

import numpy as np

from oracle import rnnt_ref


def widen(bits, kind):
    """Exact float64 values of logits given as float32 values or 16-bit patterns."""
    if kind == "f32":
        return np.asarray(bits, dtype=np.float32).astype(np.float64)
    if kind == "bf16":
        return (np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if kind == "f16":
        return np.asarray(bits).astype(np.uint16).view(np.float16).astype(np.float64)
    raise ValueError(kind)


def utterance_ref(job):
    """job = (b, bits (T_b, U_b+1, V), kind, labels (U_b,), blank, variant, need_grad);
    returns (b, loss, grad (T_b, U_b+1, V) float64 or None)."""
    b, bits, kind, labels, blank, variant, need_grad = job
    r = rnnt_ref.utterance_loss_grad(widen(bits, kind), labels, blank, variant, need_grad=need_grad)
    return b, float(r["loss"]), r["grad"]


def workers():
    """Pool size: the process's CPUs, at most 16 (the CPU share that goes with one GPU)."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def make_pool():
    return multiprocessing.get_context("spawn").Pool(workers())


def run_batched(pool, jobs, batch=None):
    """Results of utterance_ref over `jobs` (an iterable built lazily), at most `batch`
    jobs in flight, so only a bounded number of utterances sit in memory at once."""
    batch = batch or 2 * workers()
    out, pending = [], []
    for job in jobs:
        pending.append(job)
        if len(pending) == batch:
            out.extend(pool.map(utterance_ref, pending, chunksize=1))
            pending = []
    if pending:
        out.extend(pool.map(utterance_ref, pending, chunksize=1))
    return out
