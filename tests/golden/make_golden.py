"""Write tests/golden/oracle_small_cases.json.

Calls only ``oracle/`` and the seeded generators in ``workloads``: every stored
value is the oracle's fp64 result (as float.hex) on a small seeded case, plus
the sha256 of the generated inputs.  The file pins the generators and the
oracle against silent change; it is rewritten only when a change to either is
justified by the paper.

    python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads  # noqa: E402

CASES = [
    dict(q=3, N=5, K=256, G=128, B=2, seed=0, exp_range=(-8, -2), outlier_fraction=0.0),
    dict(q=2, N=3, K=64, G=8, B=1, seed=1, exp_range=(-10, -3), outlier_fraction=0.05),
    dict(q=4, N=2, K=768, G=768, B=3, seed=2, exp_range=(-12, -3), outlier_fraction=0.01),
]


def compute(spec):
    c = workloads.random_case(spec["q"], spec["N"], spec["K"], spec["G"], spec["B"],
                              seed=spec["seed"], exp_range=tuple(spec["exp_range"]),
                              outlier_fraction=spec["outlier_fraction"])
    y, a = oracle.shiftadd_gemm(c["x"], c["signs"], c["exps"], spec["G"], nthreads=1)
    return dict(spec=spec,
                sha256=dict(signs=workloads.sha256(c["signs"]), exps=workloads.sha256(c["exps"]),
                            x=workloads.sha256(c["x"])),
                y=[[float(v).hex() for v in row] for row in y],
                absterm=[[float(v).hex() for v in row] for row in a])


def main():
    out = dict(about="Written by tests/golden/make_golden.py from oracle/ only (fp64, float.hex).",
               cases=[compute(s) for s in CASES],
               mixed_bits_7b_layer_set=workloads.mixed_bits(0))
    with open(os.path.join(HERE, "oracle_small_cases.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
