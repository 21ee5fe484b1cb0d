"""Writes the stored fixtures under tests/golden/ that are derived by search.

Calls only the CPU oracle (hash/cell layout) and plain Python logic; nothing
here comes from the GPU path.  Run: python tests/golden/make_golden.py
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402


def fig1_search():
    """Find a tiny sketch whose hypergraph has the structure of the paper's
    Figure 1 (section 3.2): three nonzeros x, y, z; only z owns a cell no other
    nonzero maps to, so z is peeled first; once z is removed, x and y each own
    such a cell and are peeled next."""
    for rows in (4, 5, 6):
        for seed in range(1, 200000):
            g = oracle.Geom(n=3, rows=rows, seed=seed, c=1)
            cl, _ = oracle.cells(g, [0, 1, 2])
            cl = [set(int(v) for v in r) for r in cl]
            deg = {}
            for r in cl:
                for v in r:
                    deg[v] = deg.get(v, 0) + 1
            pure0 = [any(deg[v] == 1 for v in r) for r in cl]
            if sorted(pure0) != [False, False, True]:
                continue
            z = pure0.index(True)
            rest = [i for i in range(3) if i != z]
            deg2 = dict(deg)
            for v in cl[z]:
                deg2[v] -= 1
            if all(any(deg2[v] == 1 for v in cl[i]) for i in rest):
                return rows, seed, z, [sorted(r) for r in cl]
    raise RuntimeError("no Figure-1 geometry found")


def main():
    rows, seed, z, cl = fig1_search()
    with open(os.path.join(HERE, "fig1_example.txt"), "w") as f:
        f.write("# Structure of the worked example of section 3.2 (Figure 1): nonzeros x, y, z;\n")
        f.write("# z alone in one of its counters is peeled in round 1, then x and y in round 2.\n")
        f.write("# The figure's numbers are not available, so only its peeling order is pinned.\n")
        f.write("# Geometry found by tests/golden/make_golden.py (oracle hash, c = 1, n = 3).\n")
        f.write(f"rows {rows}\nseed {seed}\nc 1\nn 3\nz {z}\n")
        for i, r in enumerate(cl):
            f.write(f"cells {i} {' '.join(str(v) for v in r)}\n")
    print("fig1:", rows, seed, z, cl)


if __name__ == "__main__":
    main()
