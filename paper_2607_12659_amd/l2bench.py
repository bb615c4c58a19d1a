"""Build and run the L2 / HBM read-rate microbenchmark (csrc/l2bench.hip).

    python -m paper_2607_12659_amd.l2bench --build     # on the build host (hipcc)
    python -m paper_2607_12659_amd.l2bench [--mib 16] [--out FILE]

Prints one markdown table: bytes read per compute unit per second and over
the chip, for plain vector loads and for direct-to-LDS loads, from a 1 MiB
region that stays in L2 and from HBM, per workgroup count, waves per
workgroup and loads in flight per wave.
"""
from __future__ import annotations

import argparse
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "csrc", "l2bench.hip")
EXE = os.path.join(HERE, "l2bench")


def build() -> str:
    from paper_2607_12659_amd import build as b
    b._run([b.HIPCC, *[f for f in b.FLAGS if f != "-fPIC"], SRC, "-o", EXE])
    return EXE


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--build", action="store_true")
    ap.add_argument("--mib", type=int, default=16, help="MiB read by each workgroup from the L2-resident region")
    ap.add_argument("--out", default="")
    args = ap.parse_args()
    if args.build:
        print(build())
        return
    if not os.path.exists(EXE):
        sys.exit("%s is not built: run with --build first" % EXE)
    out = subprocess.run([EXE, str(args.mib)], stdout=subprocess.PIPE, text=True, check=True).stdout
    lines = ["| load | source | workgroups | waves per workgroup | 1 KiB loads in flight per wave | GB/s per unit | TB/s over the chip | ms |",
             "|---|---|---:|---:|---:|---:|---:|---:|"]
    for row in out.splitlines():
        if row.startswith("#"):
            lines.insert(0, row[2:] + "\n")
            continue
        kind, srcname, wgs, waves, u, gbs, tbs, ms = row.split()
        lines.append("| %s | %s | %s | %s | %s | %s | %s | %s |" % (kind, srcname, wgs, waves, u, gbs, tbs, ms))
    text = "\n".join(lines) + "\n"
    print(text)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(HERE))
    main()
