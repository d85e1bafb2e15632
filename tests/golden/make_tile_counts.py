"""Writes tile_counts.txt: the number of full and partial tiles per (b, h) of every
measured workload, counted by the oracle's brute-force classifier over every
query-tile row (oracle.blockmask.build). Calls nothing but oracle/ and the
workload table (which holds pattern parameters only).

    python tests/golden/make_tile_counts.py
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import workloads as W  # noqa: E402
from oracle import blockmask  # noqa: E402


def main():
    lines = ["# Full and partial tiles per (b, h) of the measured workloads, from the",
             "# oracle's brute-force classifier over every query-tile row",
             "# (written by make_tile_counts.py; not a value the paper prints).",
             "# workload  tile_m tile_n  n_full n_partial"]
    for w in list(W.ATTN_WORKLOADS) + [W.C5]:
        bm = blockmask.build(w.pattern, w.tile_m, w.tile_n)
        lines.append(f"{w.name} {w.tile_m} {w.tile_n} {bm.total_full} {bm.total_part}")
        print(lines[-1], flush=True)
    with open(os.path.join(HERE, "tile_counts.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
