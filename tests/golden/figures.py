"""Reader for the lattice fixtures transcribed from the paper's Fig. 1 and Fig. 4."""
import os

HERE = os.path.dirname(os.path.abspath(__file__))


def load_figure(name):
    """Parse a fixture: returns dict(units, frames, nodes {state: (t, u)}, final, arcs [(src, dst, sym, w)])."""
    fig = dict(nodes={}, arcs=[])
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, *rest = line.split()
            if k == "units":
                fig["units"] = rest
            elif k == "frames":
                fig["frames"] = int(rest[0])
            elif k == "node":
                fig["nodes"][int(rest[0])] = (int(rest[1]), int(rest[2]))
            elif k == "final":
                fig["final"] = int(rest[0])
            elif k == "arc":
                fig["arcs"].append((int(rest[0]), int(rest[1]), rest[2], float(rest[3])))
    return fig


def allow_ignore_from_fig4(fig4):
    """The allow-ignore reading (Section 4.3): Fig. 4's final skip arcs redirected
    to the final state; everything else unchanged."""
    top = {s for s, (t, u) in fig4["nodes"].items() if u == len(fig4["units"])}
    prev_final = [s for s, tu in fig4["nodes"].items() if tu == (fig4["frames"] - 1, len(fig4["units"]))][0]
    arcs = []
    for (s, d, sym, w) in fig4["arcs"]:
        if sym == "<eps>" and s in top and d == prev_final:
            d = fig4["final"]
        arcs.append((s, d, sym, w))
    return dict(fig4, arcs=arcs)


def grid_weights(fig):
    """lp_blank / lp_label (T x (U+1) lists, -inf where no arc) read off the
    figure's blank and unit arcs through the node map."""
    T, U = fig["frames"], len(fig["units"])
    ninf = float("-inf")
    lp_b = [[ninf] * (U + 1) for _ in range(T)]
    lp_l = [[ninf] * (U + 1) for _ in range(T)]
    for (s, d, sym, w) in fig["arcs"]:
        if sym == "<eps>":
            continue
        t, u = fig["nodes"][s]
        if sym == "<b>":
            lp_b[t][u] = w
        else:
            assert sym == fig["units"][u], (sym, u)
            lp_l[t][u] = w
    return lp_b, lp_l
