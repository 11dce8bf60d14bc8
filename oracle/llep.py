"""CPU oracle of the least-loaded expert-parallel plan and of one rank's
share of the layer under that plan.

TEST INFRASTRUCTURE ONLY: imported by tests/ and the benchmark, never by the
product path.  It shares no code with the HIP library.

Mixture-of-Parallelisms Sec. 3.3 (recap of LLEP): at every MoE call the
per-rank token load is measured, excess tokens move from overloaded ranks
to underloaded ones, and the expert weights travel with them so that the
receiving rank computes those token-expert products itself; which products
are computed never changes.  The paper gives no planning steps (they are in
the LLEP paper, which is not available), so the plan below is a reading of
that description, fully specified so that the device planner can be checked
bit for bit:

  * E experts on E_p ranks, expert e at home on rank e // (E / E_p);
    n_e = assignments of expert e (over all tokens); L = sum n_e;
    capacity C = max(capacity_in, ceil(L / E_p)).
  * Keep at home: every rank walks its experts in ascending index and keeps
    min(n_e, C - load) of each; the rest of expert e is its spill s_e.
  * Move to the least loaded: experts with s_e > 0, in order of decreasing
    s_e (ties: lower index first), hand their spill in pieces to the rank
    with the smallest load (ties: lower rank), each piece as large as that
    rank's room C - load allows, until nothing is left.
  * Expert e's assignments, in the layer's stable row order (ascending
    assignment index t*k + i), are cut into consecutive windows: the home
    rank's [0, keep_e) first, then the pieces in the order they were handed
    out.  Every piece on a rank other than the home is one weight shipment.
"""
from __future__ import annotations

import numpy as np


def llep_plan(counts, E_p: int, capacity: int = 0):
    """Returns (lo [E_p, E], hi [E_p, E], load [E_p], n_ship) as int64 numpy
    arrays / int.  Rank r computes rows [lo[r, e], hi[r, e]) of expert e."""
    n = [int(c) for c in counts]
    E = len(n)
    assert E_p >= 1 and E % E_p == 0
    G = E // E_p
    total = sum(n)
    C = max(int(capacity), -(-total // E_p))
    lo = np.zeros((E_p, E), np.int64)
    hi = np.zeros((E_p, E), np.int64)
    load = [0] * E_p
    spill = [0] * E
    for r in range(E_p):
        for e in range(r * G, (r + 1) * G):
            keep = min(n[e], C - load[r])
            hi[r, e] = keep
            load[r] += keep
            spill[e] = n[e] - keep
    order = sorted((e for e in range(E) if spill[e] > 0), key=lambda e: (-spill[e], e))
    n_ship = 0
    for e in order:
        start = n[e] - spill[e]
        while spill[e] > 0:
            r = min(range(E_p), key=lambda q: (load[q], q))
            take = min(spill[e], C - load[r])
            assert take > 0, "capacity below the total"
            lo[r, e], hi[r, e] = start, start + take
            load[r] += take
            start += take
            spill[e] -= take
            n_ship += 1
    return lo, hi, np.array(load, np.int64), n_ship


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
