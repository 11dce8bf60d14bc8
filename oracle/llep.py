"""CPU oracle of the least-loaded expert-parallel plan and of one rank's
share of the layer under that plan.

TEST INFRASTRUCTURE ONLY: imported by tests/ and the benchmark, never by the
product path.  It shares no code with the HIP library.

Mixture-of-Parallelisms Sec. 3.3 (recap of LLEP): each call measures how
much work every rank holds; a rank above its share hands part of it, with
the weights of the experts concerned, to ranks below their share, which
then compute those token-expert products themselves; the set of products
computed stays the same.  The paper gives no planning steps (they are in
the LLEP paper, which is not available), so the plan below is a reading of
that description, fully specified so that the device planner can be checked
bit for bit:

  * Load is counted in units of g rows (the granule; g = 1 counts rows, g =
    the grouped GEMM's row-tile height counts the tiles a rank's products
    run, since a window of w rows costs ceil(w / g) tiles whatever w is).
  * E experts on E_p ranks, expert e at home on rank e // (E / E_p);
    n_e = assignments of expert e (over all tokens), u_e = ceil(n_e / g) its
    units, U = sum u_e; capacity C = max(ceil(capacity_in / g),
    ceil(U / E_p)) units.
  * Keep at home: every rank walks its experts in ascending index and keeps
    min(u_e, C - load) units of each (its first min(n_e, that * g) rows);
    the rest of expert e, in units, is its spill s_e.
  * Move to the least loaded: experts with s_e > 0, in order of decreasing
    s_e (ties: lower index first), hand their spill in pieces to the rank
    with the smallest load in units (ties: lower rank), each piece as many
    units as that rank's room C - load allows, until nothing is left; a
    piece of t units is t * g rows, or what is left of the expert.
  * Expert e's assignments, in the layer's stable row order (ascending
    assignment index t*k + i), are cut into consecutive windows: the home
    rank's [0, keep_e) first, then the pieces in the order they were handed
    out.  Every piece on a rank other than the home is one weight shipment.
    Every window but an expert's last starts and ends on a multiple of g,
    so no window splits a unit and a rank's unit load is the sum of
    ceil(window / g) over its windows.
"""
from __future__ import annotations

import numpy as np


def llep_plan(counts, E_p: int, capacity: int = 0, granule: int = 1):
    """Returns (lo [E_p, E], hi [E_p, E], load [E_p], n_ship) as int64 numpy
    arrays / int.  Rank r computes rows [lo[r, e], hi[r, e]) of expert e;
    load is each rank's rows (its units are at most the capacity C)."""
    n = [int(c) for c in counts]
    E = len(n)
    g = int(granule)
    assert E_p >= 1 and E % E_p == 0 and g >= 1
    G = E // E_p
    u = [-(-c // g) for c in n]
    C = max(-(-int(capacity) // g), -(-sum(u) // E_p))
    lo = np.zeros((E_p, E), np.int64)
    hi = np.zeros((E_p, E), np.int64)
    load_u = [0] * E_p
    load_rows = [0] * E_p
    spill = [0] * E  # units
    for r in range(E_p):
        for e in range(r * G, (r + 1) * G):
            keep = min(u[e], C - load_u[r])
            hi[r, e] = min(n[e], keep * g)
            load_u[r] += keep
            load_rows[r] += int(hi[r, e])
            spill[e] = u[e] - keep
    order = sorted((e for e in range(E) if spill[e] > 0), key=lambda e: (-spill[e], e))
    n_ship = 0
    for e in order:
        start = (u[e] - spill[e]) * g  # rows kept at home
        while spill[e] > 0:
            r = min(range(E_p), key=lambda q: (load_u[q], q))
            take = min(spill[e], C - load_u[r])
            assert take > 0, "capacity below the total"
            rows = min(n[e] - start, take * g)
            lo[r, e], hi[r, e] = start, start + rows
            load_u[r] += take
            load_rows[r] += rows
            start += rows
            spill[e] -= take
            n_ship += 1
    return lo, hi, np.array(load_rows, np.int64), n_ship


def rank_rows(topk_idx, lo, hi, r: int):
    """The assignments rank r computes under a plan: for every expert e in
    ascending order, the assignments a = t*k + i with topk_idx = e whose
    position among expert e's assignments (ascending a) lies in
    [lo[r, e], hi[r, e]).  Returns (offsets [E + 1], row_src [rows]) with
    the rows of expert e at [offsets[e], offsets[e + 1])."""
    idx = np.asarray(topk_idx, np.int64).reshape(-1)
    E = lo.shape[1]
    offsets = [0]
    rows = []
    for e in range(E):
        a_e = np.nonzero(idx == e)[0]  # ascending assignment index
        sel = a_e[lo[r, e]:hi[r, e]]
        rows.extend(sel.tolist())
        offsets.append(offsets[-1] + len(sel))
    return np.array(offsets, np.int64), np.array(rows, np.int64)
