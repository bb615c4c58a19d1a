"""Build and run the link microbenchmark (csrc/linkbench.hip).

    python -m paper_2607_12659_amd.linkbench --build     # on the build host (hipcc)
    python -m paper_2607_12659_amd.linkbench [--phases 400] [--out FILE]

Prints one markdown table: microseconds per phase of a chain of dependent
producer -> consumer links between the workgroups of a persistent kernel
(one per compute unit), per link mode, activation size, producer and
consumer counts and background stream.  Every row's checksums are verified
against the host; a row with errors or mismatches is marked.
"""
from __future__ import annotations

import argparse
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "csrc", "linkbench.hip")
EXE = os.path.join(HERE, "linkbench")


def build() -> str:
    from paper_2607_12659_amd import build as b
    b._run([b.HIPCC, *[f for f in b.FLAGS if f != "-fPIC"], SRC, "-o", EXE])
    return EXE


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--build", action="store_true")
    ap.add_argument("--phases", type=int, default=400)
    ap.add_argument("--out", default="")
    args = ap.parse_args()
    if args.build:
        print(build())
        return
    if not os.path.exists(EXE):
        sys.exit("%s is not built: run with --build first" % EXE)
    out = subprocess.run([EXE, str(args.phases)], stdout=subprocess.PIPE, text=True, check=True).stdout
    lines = ["| link | activation KiB | producers | consumers | background KiB per CU | us per phase | check |",
             "|---|---:|---:|---:|---:|---:|---|"]
    notes = []
    for row in out.splitlines():
        if row.startswith("# CUs"):
            lines.insert(0, row[2:] + "\n")
            continue
        if row.startswith("#"):
            notes.append(row[2:])
            continue
        mode, kb, prod, cons, bg, us, err, bad = row.split()
        ok = "ok" if err == "0" and bad == "0" else "ERROR (err %s, mismatches %s)" % (err, bad)
        lines.append("| %s | %s | %s | %s | %s | %s | %s |" % (mode, kb, prod, cons, bg, us, ok))
    text = "\n".join(lines) + "\n" + "".join("\n" + n + "\n" for n in notes)
    print(text)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(HERE))
    main()
