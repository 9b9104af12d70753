"""Store/recompute selection by exhaustive enumeration (TEST INFRASTRUCTURE ONLY).

The plain definition of the paper's integer program (Sec. IV-A): one binary
v_i per forwarded array (1 = store, 0 = recompute), objective
sum_i c_i (1 - v_i), and a sequence of memory measurements m_j, each an
affine function of v, built from the program's allocation timeline; the
peak t = max_j m_j must not exceed the limit. With control flow, every path
contributes its own sequence and all of them are constraints (Sec. IV-B).

The timeline is a list of events, each adding an affine amount to the
running total of one path and recording a measurement:
  ("alloc", s)            +s
  ("free", s)             -s
  ("produce", i)          +S_i          forward pass creates A_i
  ("drop", i)             -S_i (1-v_i)  after its forward use, unless stored
  ("recompute", i)        +(1-v_i)(R_i + S_i)   backward pass rebuilds A_i
  ("recompute_done", i)   -(1-v_i) R_i  the rebuild's temporaries are freed
  ("release", i)          -S_i          backward use of A_i is over
  ("path",)               starts a new path (running total back to 0)
This enumerates all 2^n assignments and keeps the cheapest feasible one;
ties go to the lower peak, then to the assignment that stores the
lowest-numbered arrays.
"""
from itertools import product


def measurements(arrays, events, v):
    """All measurement sequences (one per path) for the assignment v.
    arrays: list of dicts with keys size, overhead, cost."""
    paths, cur, m = [], [], 0.0
    for ev in events:
        kind = ev[0]
        if kind == "path":
            if cur:
                paths.append(cur)
            cur, m = [], 0.0
            continue
        if kind == "alloc":
            m += ev[1]
        elif kind == "free":
            m -= ev[1]
        else:
            a = arrays[ev[1]]
            keep = v[ev[1]]
            if kind == "produce":
                m += a["size"]
            elif kind == "drop":
                m -= a["size"] * (1 - keep)
            elif kind == "recompute":
                m += (1 - keep) * (a["overhead"] + a["size"])
            elif kind == "recompute_done":
                m -= (1 - keep) * a["overhead"]
            elif kind == "release":
                m -= a["size"]
            else:
                raise ValueError(kind)
        cur.append(m)
    if cur:
        paths.append(cur)
    return paths


def peak(arrays, events, v):
    return max(max(p) for p in measurements(arrays, events, v))


def cost(arrays, v):
    return sum(a["cost"] * (1 - vi) for a, vi in zip(arrays, v))


def solve(arrays, events, limit):
    """(v, cost, peak) of the best feasible assignment, or None."""
    best = None
    for v in product((1, 0), repeat=len(arrays)):
        pk = peak(arrays, events, v)
        if pk > limit:
            continue
        key = (cost(arrays, v), pk, tuple(1 - x for x in v))
        if best is None or key < best[0]:
            best = (key, v, pk)
    if best is None:
        return None
    return list(best[1]), best[0][0], best[2]
