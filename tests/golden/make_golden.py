"""Writes fig_expected.json from the transcribed figures, using only oracle/.

The expected losses and arc posteriors come from enumerating every path of the
transcribed graphs (oracle.brute_force.graph_paths); no GPU code is involved.
Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, HERE)

from oracle.brute_force import graph_arc_posteriors, graph_paths_log_prob  # noqa: E402
from figures import allow_ignore_from_fig4, load_figure  # noqa: E402


def summarize(fig):
    arcs = [(s, d, w) for (s, d, _sym, w) in fig["arcs"]]
    lnP, n_paths = graph_paths_log_prob(arcs, 0, fig["final"])
    post = graph_arc_posteriors(arcs, 0, fig["final"])
    return dict(loss=-lnP, n_paths=n_paths,
                arc_posteriors=[[s, d, sym, p] for (s, d, sym, _w), p in zip(fig["arcs"], post)])


def main():
    fig1 = load_figure("fig1_rnnt_lattice.txt")
    fig4 = load_figure("fig4_wrnnt_lattice.txt")
    out = {
        "source": "paths of the graphs transcribed from the paper's Fig. 1 and Fig. 4, enumerated by oracle.brute_force",
        "rnnt_fig1": summarize(fig1),
        "wrnnt_fig4": summarize(fig4),
        "wrnnt_allow_ignore_fig4_redirected": summarize(allow_ignore_from_fig4(fig4)),
    }
    with open(os.path.join(HERE, "fig_expected.json"), "w") as f:
        json.dump(out, f, indent=1)
    for k in ("rnnt_fig1", "wrnnt_fig4", "wrnnt_allow_ignore_fig4_redirected"):
        print(k, "%.10f" % out[k]["loss"], out[k]["n_paths"], "paths")


if __name__ == "__main__":
    main()
