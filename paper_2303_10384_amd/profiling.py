"""HBM traffic of the kernels from rocprofv3 counter runs.

Two `rocprofv3 --pmc` runs of the benchmark (FETCH_SIZE, then WRITE_SIZE) and
the same two counters on a device-to-device copy of known size
(`bench.py --copy-probe`) give, per kernel, the bytes fetched from and written
to HBM per launch: each counter is scaled by the factor that makes the copy's
reading equal its known size.  The gradient kernel's figure is written, with the
digest of the sources it was measured on, to profiles/k3_grad_<workload>_traffic.json,
which bench.py reports as roofline.traffic while the sources are unchanged.
--path arc reads the kernels of the arc-list loss (bench.py --mode arc).

    python -m paper_2303_10384_amd.profiling --workload bpe [--path loss|arc] \\
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR [--out profiles]
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import statistics

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# the sources whose change invalidates a traffic figure, per path: the two
# streaming kernels whose figures the record serves (the populate kernel and the
# gradient kernel) and the arc-list kernels of that path
SOURCES = {
    "loss": [
        "paper_2303_10384_amd/csrc/rnnt_device.h",
        "paper_2303_10384_amd/csrc/rnnt_k1_populate.h",
        "paper_2303_10384_amd/csrc/rnnt_launch_k1.h",
        "paper_2303_10384_amd/csrc/rnnt_launch_k1_lattice.hip",
        "paper_2303_10384_amd/csrc/rnnt_k3_grad.h",
        "paper_2303_10384_amd/csrc/rnnt_launch_k3.hip",
    ],
    "arc": [
        "paper_2303_10384_amd/csrc/rnnt_device.h",
        "paper_2303_10384_amd/csrc/rnnt_k1_populate.h",
        "paper_2303_10384_amd/csrc/rnnt_launch_k1.h",
        "paper_2303_10384_amd/csrc/rnnt_launch_k1_rows.hip",
        "paper_2303_10384_amd/csrc/rnnt_k3_grad.h",
        "paper_2303_10384_amd/csrc/rnnt_launch_k3.hip",
        "paper_2303_10384_amd/csrc/rnnt_arc_layout.h",
        "paper_2303_10384_amd/csrc/rnnt_arc_kernels.h",
    ],
}
KERNEL_SOURCES = SOURCES["loss"]

KERNEL_SETS = {  # short name -> substring of the demangled kernel name
    "loss": {
        "k1_populate": "rnnt::k1_populate",
        "k2_lattice": "rnnt::k2_lattice",
        "k2b_posteriors": "rnnt::k2b_posteriors",
        "k3_grad": "rnnt::k3_grad",
    },
    "arc": {
        "k1_populate": "rnnt::k1_populate",
        "arc_populate": "rnnt::k_arc_populate",
        "arc_sweep": "rnnt::k_arc_sweep",
        "arc_rows": "rnnt::k_arc_rows",
        "k3_grad": "rnnt::k3_grad",
    },
}
KERNELS = KERNEL_SETS["loss"]
COPY_KERNEL = "copyBuffer"


def source_digest(paths, root=ROOT):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(root, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_counter(path_or_dir, counter):
    """[(kernel name, value in KiB)] per dispatch from a rocprofv3 counter_collection.csv."""
    path = path_or_dir
    if os.path.isdir(path):
        found = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
        if len(found) != 1:
            raise FileNotFoundError("expected one counter_collection.csv under %s, found %d" % (path, len(found)))
        path = found[0]
    out = []
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            if row["Counter_Name"] == counter:
                out.append((row["Kernel_Name"], float(row["Counter_Value"])))
    return out


def per_kernel_kib(rows, substr):
    vals = [v for name, v in rows if substr in name]
    if not vals:
        raise ValueError("no dispatch of a kernel matching %r" % substr)
    return statistics.median(vals), len(vals)


def copy_scale(rows, copy_bytes, counter):
    """Bytes per counted KiB: the copy kernel's dispatches that moved the probe's
    size (the largest readings) against the known size."""
    vals = sorted((v for name, v in rows if COPY_KERNEL in name), reverse=True)
    if not vals:
        raise ValueError("no %s dispatch in the copy probe's %s run" % (COPY_KERNEL, counter))
    big = [v for v in vals if v >= 0.5 * vals[0]]
    return copy_bytes / statistics.median(big), statistics.median(big), len(big)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", required=True)
    ap.add_argument("--path", default="loss", choices=sorted(SOURCES))
    ap.add_argument("--fetch", required=True, help="rocprofv3 --pmc FETCH_SIZE output of bench.py")
    ap.add_argument("--write", required=True, help="rocprofv3 --pmc WRITE_SIZE output of bench.py")
    ap.add_argument("--copy-fetch", required=True, help="FETCH_SIZE output of bench.py --copy-probe")
    ap.add_argument("--copy-write", required=True, help="WRITE_SIZE output of bench.py --copy-probe")
    ap.add_argument("--copy-bytes", type=int, required=True, help="bytes per copy of the probe")
    ap.add_argument("--algorithmic", help="JSON line of bench.py (kernel algorithmic bytes), optional")
    ap.add_argument("--commands", default="", help="text naming the commands that made the runs")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    a = ap.parse_args(argv)

    f_scale, f_copy, f_n = copy_scale(read_counter(a.copy_fetch, "FETCH_SIZE"), a.copy_bytes, "FETCH_SIZE")
    w_scale, w_copy, w_n = copy_scale(read_counter(a.copy_write, "WRITE_SIZE"), a.copy_bytes, "WRITE_SIZE")
    fetch = read_counter(a.fetch, "FETCH_SIZE")
    write = read_counter(a.write, "WRITE_SIZE")
    algo = {}
    if a.algorithmic:
        with open(a.algorithmic) as f:
            line = [ln for ln in f if ln.strip().startswith("{")][-1]
        algo = json.loads(line).get("algorithmic_bytes", {})
    kernels = {}
    for short, substr in KERNEL_SETS[a.path].items():
        fk, nf = per_kernel_kib(fetch, substr)
        wk, nw = per_kernel_kib(write, substr)
        kernels[short] = {
            "fetch_bytes": round(fk * f_scale),
            "write_bytes": round(wk * w_scale),
            "hbm_bytes": round(fk * f_scale + wk * w_scale),
            "fetch_kib_raw": fk,
            "write_kib_raw": wk,
            "dispatches": [nf, nw],
            "algorithmic_bytes": algo.get(short),
        }
    rec = {
        "workload": a.workload,
        "kernel": "k3_grad",
        "hbm_bytes_per_launch": kernels["k3_grad"]["hbm_bytes"],
        "kernels": kernels,
        "calibration": {
            "copy_bytes": a.copy_bytes,
            "fetch_kib_raw": f_copy, "fetch_bytes_per_kib": f_scale, "fetch_dispatches": f_n,
            "write_kib_raw": w_copy, "write_bytes_per_kib": w_scale, "write_dispatches": w_n,
        },
        "commands": a.commands,
        "path": a.path,
        "sources": SOURCES[a.path],
        "source_digest": source_digest(SOURCES[a.path]),
    }
    os.makedirs(a.out, exist_ok=True)
    path = os.path.join(a.out, "k3_grad_%s_traffic.json" % a.workload)
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(path)
    for k, v in kernels.items():
        alg = v["algorithmic_bytes"]
        print("%-15s fetch %8.1f MB  write %8.1f MB  total %8.1f MB  algorithmic %s" % (
            k, v["fetch_bytes"] / 1e6, v["write_bytes"] / 1e6, v["hbm_bytes"] / 1e6,
            "%.1f MB (x%.3f)" % (alg / 1e6, v["hbm_bytes"] / alg) if alg else "-"))
    return rec


if __name__ == "__main__":
    main()
