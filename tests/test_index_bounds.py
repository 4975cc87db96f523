"""Host-side model of the kernels' grids and index arithmetic (no GPU).

Before any launch, this checks for every workload shape that each block of
each kernel only addresses memory inside the buffers it is given, that the
gradient kernel's chunk -> (row, column) mapping reproduces the flat index
exactly, and that 32-bit intermediates cannot overflow.  The formulas mirror
the launch code in csrc/rnnt_api.hip and the kernels' index expressions.
"""
import os
import re

import numpy as np
import pytest

from paper_2303_10384_amd.workloads import WORKLOADS

_CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2303_10384_amd", "csrc")
_K1_SRC = os.path.join(_CSRC, "rnnt_k1_populate.h")
# consecutive populate blocks per XCD turn, as the kernel source defines it
K1_XCD_RUN = int(re.search(r"#define RNNT_K1_XCD_RUN (\d+)", open(_K1_SRC).read()).group(1))
# whether sweeps of 65..256 units run one unit per lane over several wavefronts
K2_MULTI_WAVE = int(re.search(r"#define RNNT_K2_MULTI_WAVE (\d+)",
                              open(os.path.join(_CSRC, "rnnt_launch_k2.h")).read()).group(1))


def units_per_lane(U1):
    return next(k for k in (1, 2, 3, 4, 6, 8, 12, 16, 24, 32) if U1 <= 64 * k)


def sweep_shape(U1):
    """(wavefronts per sweep, units per lane) of the lattice sweeps."""
    K = units_per_lane(U1)
    return (K, 1) if K2_MULTI_WAVE and K in (2, 3, 4) else (1, K)

EPC = {"f32": 4, "bf16": 8, "f16": 8}
SHAPES = [(w.B, w.T_max, w.U_max, w.V, w.dtype) for w in WORKLOADS.values()] + [
    (3, 7, 0, 2, "f32"), (2, 5, 4, 3, "bf16"), (1, 1, 1023, 5, "f32"), (4, 9, 63, 4097, "f16"),
    (5, 3, 64, 7, "bf16"), (2, 2, 127, 8, "f32"), (2, 4, 300, 6, "f32"), (1, 3, 700, 5, "bf16"),
    (1, 2, 1023, 3, "bf16"), (1, 3, 1535, 4, "f32"), (1, 2, 2047, 3, "bf16"), (3, 7, 5, 4100, "f32"), (3, 7, 5, 8200, "bf16"), (3, 7, 5, 2600, "f16")]


def k1_shape(V, epc):
    interior = V // epc
    best, best_slots = (64, 5, False), 1 << 30
    for g in (8, 16, 32, 64):
        for nb in range(1, 6):
            if g * nb >= interior and g * nb <= best_slots:
                best, best_slots = (g, nb, True), g * nb
    return best


@pytest.mark.parametrize("run", sorted({1, K1_XCD_RUN, 16}))
@pytest.mark.parametrize("B,T,U,V,dt", SHAPES)
def test_populate_kernel_addresses(B, T, U, V, dt, run):
    epc = EPC[dt]
    esz = {"f32": 4, "bf16": 2, "f16": 2}[dt]
    n_elem = B * T * (U + 1) * V
    G, NB, fast = k1_shape(V, epc)
    cap = 32 if dt == "f32" else 256  # consecutive units of one frame per block, at most
    n_ublk = -(-(U + 1) // cap)
    rows_per_block = -(-(U + 1) // n_ublk)  # equal blocks up to one unit
    assert rows_per_block <= cap and (n_ublk - 1) * rows_per_block < U + 1
    blocks = B * T * n_ublk
    grid = -(-(-(-blocks // run)) // 8) * 8 * run
    assert grid < 2**31
    # XCD-major numbering: physical block i (XCD i % 8, its k-th block, k = i // 8) ->
    # logical ((k // run) * 8 + i % 8) * run + k % run, a bijection onto [0, blocks) once
    # the logical numbers >= blocks (the grid's round-up) are dropped
    i = np.arange(grid, dtype=np.int64)
    k = i // 8
    lb = ((k // run) * 8 + i % 8) * run + k % run
    kept = np.sort(lb[lb < blocks])
    assert np.array_equal(kept, np.arange(blocks))
    fast = fast and rows_per_block * V * esz + 64 < 0x7fffffff
    # every row a block can reach with full lengths (t < T, u <= U)
    b, t, u = np.meshgrid(np.arange(B), np.arange(T), np.arange(U + 1), indexing="ij")
    b, t, u = b.ravel(), t.ravel(), u.ravel()
    row = (b.astype(np.int64) * T + t) * (U + 1) + u
    e0 = row * V
    c0 = e0 // epc
    mis = e0 - c0 * epc
    nch = (mis + V + epc - 1) // epc
    assert np.all((c0 + nch - 1) * epc < n_elem)
    assert np.all(e0 + V <= n_elem)
    whole = c0 + nch <= n_elem // epc
    assert np.all(((c0 + nch) * epc <= n_elem)[whole])
    if fast:
        # interior chunks [kf, kl] fit G*NB lanes-chunks; every clamped index stays in [0, nch)
        first_partial = mis != 0
        last_partial = (mis + V) % epc != 0
        kf = first_partial.astype(np.int64)
        kl = nch - 1 - last_partial.astype(np.int64)
        assert np.all(kl - kf + 1 <= G * NB)
        assert np.all(np.maximum(kl, 0) < nch) and np.all(kf <= nch)
    # only rows reaching into the tensor's final partial chunk read element-wise
    assert np.all((e0 + V > (n_elem // epc) * epc)[~whole])
    if fast:
        # per-block buffer: from the first chunk of the block's first row (unit u_lo) to
        # the end of its last row; row j of the block at element e_rel0 + j * V
        ublk = u // rows_per_block
        u_lo = ublk * rows_per_block
        n_rows = np.minimum(rows_per_block, U + 1 - u_lo)
        j = u - u_lo
        row_lo = (b.astype(np.int64) * T + t) * (U + 1) + u_lo
        e_first = row_lo * V
        c_base = e_first // epc
        c_end = (e_first + n_rows * V + epc - 1) // epc
        assert np.all((c_end - c_base) * 16 < 2**31)
        e_rel = (e_first - c_base * epc) + j * V
        assert np.array_equal(e_rel, e0 - c_base * epc)
        off0 = (e_rel - mis) * esz
        assert np.all(off0 >= 0) and np.all(off0 + nch * 16 <= (c_end - c_base) * 16)
        assert np.all(e_rel * esz < 2**31)
        # rows per block fit the LDS arrays
        assert n_rows.max() <= 256
    # lattice-form writes at the row index, inside the B * T * (U+1) cell arrays
    assert row.max() < B * T * (U + 1) and row.min() >= 0


@pytest.mark.parametrize("B,T,U,V,dt", SHAPES)
def test_gradient_kernel_chunk_mapping(B, T, U, V, dt):
    epc = EPC[dt]
    n_elem = B * T * (U + 1) * V
    n_rows = B * T * (U + 1)
    tile = (128 if dt == "f32" else 256) * 2  # threads x chunks per thread
    chunks = -(-n_elem // epc)
    blocks = -(-chunks // tile)
    assert blocks < 2**31
    rng = np.random.default_rng(0)
    blk = np.unique(np.concatenate([np.arange(min(blocks, 64)), np.arange(max(0, blocks - 64), blocks),
                                    rng.integers(0, blocks, size=256)])).astype(np.int64)
    tile0 = blk * tile
    e_tile = tile0 * epc
    r_tile = e_tile // V
    v_tile = e_tile - r_tile * V
    assert np.all(v_tile < V)
    for cl in (0, 1, tile // 2 - 1, tile // 2, tile - 1):
        c = tile0 + cl
        e0 = c * epc
        live = e0 < n_elem
        off = v_tile + cl * epc
        assert np.all(off < 2**32)
        dr = off // V
        r = r_tile + dr
        v = off - dr * V
        assert np.all((r * V + v)[live] == e0[live])
        assert np.all(r[live] < n_rows)
        if V >= epc:
            split = v + epc > V
            # the second row of a split chunk exists unless the chunk runs past the end
            assert np.all(((r + 1 < n_rows) | (e0 + epc > n_elem))[live & split])


@pytest.mark.parametrize("B,T,U,V,dt", SHAPES)
def test_lattice_kernel_addresses(B, T, U, V, dt):
    """Sweep kernel: weights of any step e read at the cell clamped into the utterance,
    diagonal ec = clamp(e, 0, D), unit clamp(u, ec - (T_b-1), min(ec, U_b)), a valid cell,
    stored at its row (b, ec - u, u);
    alpha stored in row min(d, D+1), beta in row d (or the spare row ND when d < 0), each row
    u_pad = 64*K wide; the posterior kernel reads alpha, beta only at diagonals <= D."""
    U1 = U + 1
    ND = T + U
    NW, K = sweep_shape(U1)
    u_pad = 64 * units_per_lane(U1)
    assert NW * 64 * K == u_pad  # unit u in column u whatever the waves
    n_cells = B * T * U1  # kernel 1's lattice form: one cell per logits row
    n_scores = B * (ND + 1) * u_pad
    lanes = np.concatenate([w * 64 * K + np.arange(64) * K for w in range(NW)])  # each lane's first unit
    for Tb, Ub in [(T, U), (1, 0), (max(1, T // 2), U // 2), (1, U), (T, 0)]:
        D = Tb - 1 + Ub
        PF = 1 if K >= 24 else 2 if K >= 16 else min(24, 48 // K)
        for bb in {0, B - 1}:
            for e in range(-PF - 2, D + PF + 2):  # every diagonal a load or store step can name
                ec = min(max(e, 0), D)
                for k in range(K):
                    uc = np.minimum(np.maximum(lanes + k, ec - (Tb - 1)), min(ec, Ub))
                    tc = ec - uc
                    assert np.all((tc >= 0) & (tc < Tb) & (uc >= 0) & (uc <= Ub))  # a cell kernel 1 wrote
                    w = (bb * T + tc) * U1 + uc  # row (t, u) of utterance bb
                    assert np.all(w >= 0) and np.all(w < n_cells)
                    rows = []
                    if 1 <= e <= D + PF - 1:  # forward steps d = 1 .. (last block's end)
                        rows.append(min(e, D + 1))
                    if -PF + 1 <= e <= D - 1:  # backward steps d = D-1 .. (last block's end)
                        rows.append(e if e >= 0 else ND)
                    for row in rows:
                        a = (bb * (ND + 1) + row) * u_pad + lanes + k
                        assert np.all(a >= 0) and np.all(a < n_scores)
        # spare rows never overlap the rows the posterior kernel reads (d <= D)
        assert D + 1 <= ND


@pytest.mark.parametrize("NW", [2, 3, 4])
@pytest.mark.parametrize("D", [0, 1, 23, 24, 25, 47, 48, 330, 649])
def test_lattice_multi_wave_schedule(NW, D):
    """Several wavefronts per sweep: wave w runs segment g = r - lag(w) of PF steps in round r
    (lag w forward, NW-1-w backward) and every wave passes one barrier per round.  Each value a
    wave takes from its neighbour (slot [pair][r-1 & 1][s] in round r) was written by that
    neighbour in round r-1 for the same diagonal, and is not overwritten before it is read; the
    LDS slots stay inside [NW-1][2][PF]."""
    PF = 24  # one unit per lane
    n_seg = (D + PF - 1) // PF
    n_rounds = n_seg + NW - 1
    for sweep in ("forward", "backward"):
        writes = {}  # (pair, half, s) -> list of (round, diagonal)
        reads = []   # (round, pair, half, s, diagonal)
        active = {w: 0 for w in range(NW)}
        for r in range(n_rounds):  # the same trip count for every wave: equal barrier counts
            for w in range(NW):
                lag = w if sweep == "forward" else NW - 1 - w
                g = r - lag
                if not (0 <= g < n_seg):
                    continue
                active[w] += 1
                for s in range(PF):
                    d = 1 + g * PF + s if sweep == "forward" else D - 1 - g * PF - s
                    producer = w < NW - 1 if sweep == "forward" else w > 0
                    consumer = w > 0 if sweep == "forward" else w < NW - 1
                    if producer:
                        pair = w if sweep == "forward" else w - 1
                        assert 0 <= pair < NW - 1
                        writes.setdefault((pair, r & 1, s), []).append((r, d))
                    if consumer:
                        pair = w - 1 if sweep == "forward" else w
                        assert 0 <= pair < NW - 1
                        reads.append((r, pair, (r - 1) & 1, s, d))
        assert all(n == n_seg for n in active.values())  # every wave runs every segment once
        for r, pair, half, s, d in reads:
            # the latest write to the slot before round r: made in round r-1, for diagonal d
            before = [(rw, dw) for rw, dw in writes.get((pair, half, s), []) if rw < r]
            assert before and before[-1] == (r - 1, d)
            # and the next write to that slot comes after round r's barrier
            assert all(rw > r for rw, _ in writes[(pair, half, s)] if rw >= r)


@pytest.mark.parametrize("T,U", [(1, 0), (2, 0), (5, 0), (1, 7), (2, 1), (30, 17), (250, 80), (24, 0), (25, 23),
                                 (500, 150), (3, 255), (40, 300), (7, 700), (3, 1000), (2, 1535), (9, 2047)])
def test_wildcard_sums_take_each_frame_once(T, U):
    """W-Transducer sweeps: the owning lane stores the value of step s of a segment in LDS
    slot s, and after the segment lane s adds it to its own sum when the step's diagonal is
    in range.  Every frame's term enters exactly once: alpha(t, U) for t <= T-2 (forward;
    t = 0 from the start when U = 0) and beta(t, 0) for 1 <= t <= T-1 (backward; t = T-1
    from the start when U = 0), and the stash and sink indices stay inside their arrays."""
    nw, K = sweep_shape(U + 1)
    PF = 1 if K >= 24 else 2 if K >= 16 else min(24, 48 // K)
    D = T - 1 + U
    n_seg = (D + PF - 1) // PF
    fwd, bwd = [], []
    if U == 0 and T >= 2:
        fwd.append(0)
        bwd.append(T - 1)
    for g in range(n_seg):
        d0f, d0b = 1 + g * PF, D - 1 - g * PF
        for lane in range(64):
            for s_ in range(PF):
                assert 0 <= lane + s_ < 64 + PF  # the sink of the lanes without a value
            if lane < PF:  # min(lane, PF - 1) is the slot read; lanes >= PF add nothing
                d = d0f + lane
                if U <= d <= U + T - 2:
                    fwd.append(d - U)
                d = d0b - lane
                if 1 <= d <= T - 1:
                    bwd.append(d)
    assert sorted(fwd) == list(range(0, T - 1))
    assert sorted(bwd) == list(range(1, T))


@pytest.mark.parametrize("B,T,U,V,dt", SHAPES)
def test_gradient_kernel_fast_path_buffer(B, T, U, V, dt):
    """Blocks on the buffer-load path: no partial chunk inside, a per-block buffer of at
    most one tile (offsets fit 32 bits), every live chunk's offset inside it, dead chunks
    past its end; the row-record indices of dead chunks are clamped into the records."""
    epc = EPC[dt]
    n_elem = B * T * (U + 1) * V
    n_rows = B * T * (U + 1)
    tile = (128 if dt == "f32" else 256) * 2  # threads x chunks per thread
    n_chunks = -(-n_elem // epc)
    n_full = n_elem // epc
    blocks = -(-n_chunks // tile)
    for blk in sorted(b for b in {0, 1, blocks // 2, blocks - 2, blocks - 1} if 0 <= b < blocks):
        tile0 = blk * tile
        general = V < epc or (n_elem % epc != 0 and tile0 + tile > n_full)
        if general:
            # at most the last block holds the partial chunk
            assert V < epc or blk == blocks - 1
            continue
        tile_bytes = min(tile, n_full - tile0) * 16
        assert 0 < tile_bytes <= tile * 16 < 2**31
        cl = np.arange(tile)
        live = tile0 + cl < n_full
        assert np.all((cl * 16 < tile_bytes) == live)
        e_tile = tile0 * epc
        r_tile, v_tile = e_tile // V, e_tile % V
        r = np.minimum(r_tile + (v_tile + cl * epc) // V, n_rows - 1)
        assert np.all(r >= 0) and np.all(np.minimum(r + 1, n_rows - 1) < n_rows)
    assert 0x80000000 > tile * 16  # the out-of-range offset lies past every block's buffer


@pytest.mark.parametrize("B,T,U,V,dt", SHAPES)
def test_posterior_kernel_tiles_cover_every_row_once(B, T, U, V, dt):
    """Posterior kernel: block (b, tile) walks item i -> t = t0 + i % 8, d = t0 + i // 8, u = d - t
    over 8 * (7 + U + 1) items; kept items (t < min(t0+8, T), 0 <= u <= U) are every row once."""
    TT = 8
    U1 = U + 1
    n_tiles = -(-T // TT)
    assert B * n_tiles < 2**31
    seen = np.zeros((T, U1), np.int64)
    for tile in range(n_tiles):
        t0 = tile * TT
        i = np.arange(TT * (TT - 1 + U1))
        t = t0 + i % TT
        d = t0 + i // TT
        u = d - t
        keep = (t < min(t0 + TT, T)) & (u >= 0) & (u <= U)
        np.add.at(seen, (t[keep], u[keep]), 1)
        # consecutive items of one diagonal are consecutive cells (coalesced loads)
        assert np.all(np.diff(u[:TT]) == -1)
    assert np.all(seen == 1)


@pytest.mark.parametrize("B,T,U,V,dt", SHAPES)
def test_viterbi_kernel_addresses(B, T, U, V, dt):
    """Forced-alignment kernel: decision words stored at row min(d, D+1), one per lane slot (K a
    row) or one per wave (NW a row); the backtrace stages blocks of 64 diagonals, lane l loading
    the words of diagonal 64 w + l at byte offset ((64 w + l) cols + c) * 8: never negative, and past
    the utterance's (T_max+U_max+1)*cols words only beyond the last row (a buffer load there reads
    0), under 2^31 bytes."""
    U1 = U + 1
    ND = T + U
    NW, K = sweep_shape(U1)
    cols = units_per_lane(U1)  # decision words per diagonal: one per lane slot, or one per wave
    assert cols == (NW if NW > 1 else K)
    words = (ND + 1) * cols
    lanes = np.arange(64)
    for Tb, Ub in [(T, U), (1, 0), (max(1, T // 2), U // 2), (1, U), (T, 0)]:
        D = Tb - 1 + Ub
        PF = 1 if K >= 24 else 2 if K >= 16 else min(24, 48 // K)
        for d in range(1, D + PF):
            row = min(d, D + 1)
            for wv in range(NW):
                for lane in range(64):
                    assert 0 <= row * cols + (wv if NW > 1 else min(lane, K - 1)) < words
        # unit u's word column and bit: (u % K, u // K) in one wave, (u // 64, u % 64) over several
        for u in range(Ub + 1):
            c, bit = (u // 64, u % 64) if NW > 1 else (u % K, u // K)
            assert 0 <= c < cols and 0 <= bit < 64
        for w in range(D // 64 + 1):
            for k in range(cols):
                idx = (64 * w + lanes) * cols + k
                assert np.all(idx >= 0) and np.all(idx * 8 < 2 ** 31)
                # a word past the stored rows is a diagonal past ND: masked off by the walk (d <= D)
                assert np.all((idx < words) | (64 * w + lanes > ND))


def _walk_by_diagonal(dec, t, U, var):
    """The backtrace one diagonal per step (the plain definition): at node (t, u) a set bit
    means entered by the label arc (or, at u = 0, by the initial wild-card arc)."""
    u, start, frames = U, 0, {}
    while t + u > 0:
        bit = dec[t + u][u]
        label = u > 0 and (bit or t == 0)
        jumped = var != 0 and bit and u == 0
        if label:
            frames[u - 1] = t
            u -= 1
        elif jumped:
            start = t
            break
        else:
            t -= 1
    return frames, start


def _walk_by_label_moves(dec, t, U, var, ND):
    """The kernel's backtrace: one step per label move, unit u's bits over a block of 64
    diagonals taken as one 64-bit mask (the ballot), the highest set bit in [max(u, 1), d]."""
    u, start, frames = U, 0, {}
    d = t + u
    w = d // 64
    steps = 0
    while d > 0 and (var != 0 or u > 0):
        steps += 1
        if d < 64 * w:
            w -= 1
            assert d >= 64 * w  # at most one block down per step
        base = 64 * w
        bits = 0
        for lane in range(64):
            if base + lane <= ND and dec[base + lane][u]:
                bits |= 1 << lane
        lo, hi = max(u, 1) - base, d - base
        assert lo <= hi <= 63
        m = bits & ((1 << (hi + 1)) - 1) & ~((1 << max(lo, 0)) - 1)
        if u > 0:
            if m:
                dl = base + m.bit_length() - 1
            elif u >= base:
                dl = u
            else:
                d = base - 1
                continue
            frames[u - 1] = dl - u
            u -= 1
            d = dl - 1
        else:
            if m:
                start = base + m.bit_length() - 1
                break
            d = base - 1
    assert steps <= U + (t + U) // 64 + 1
    return frames, start


@pytest.mark.parametrize("var", [0, 1, 2])
@pytest.mark.parametrize("T,U,density", [(1, 0, 0.5), (3, 1, 0.5), (7, 5, 0.2), (70, 3, 0.05), (5, 130, 0.9),
                                         (200, 80, 0.3), (150, 150, 0.5), (64, 64, 0.0), (65, 63, 1.0)])
def test_viterbi_walk_by_label_moves(var, T, U, density):
    """The block-ballot backtrace reaches the same frames and start frame as the walk one
    diagonal at a time, on random decision bits (any bits define a valid walk)."""
    rng = np.random.default_rng(T * 1000 + U + var)
    ND = T - 1 + U
    for _ in range(5):
        dec = rng.random((ND + 65, U + 1)) < density
        for t_end in {T - 1, max(0, T // 2)}:
            assert _walk_by_label_moves(dec, t_end, U, var, ND) == _walk_by_diagonal(dec, t_end, U, var)
