"""Writes tiny_case_digest.json: SHA-256 digests of the tiny W8A8 case
(X [64 x 256] with 4 outlier channels x30, W [512 x 256], bias [512], seed 0)
and of every intermediate the CPU oracle computes from it.

It calls only the seeded generator and oracle/. Run from the repository root:
    python tests/golden/make_golden.py
"""
import hashlib
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth   # noqa: E402


def digest(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def main():
    oracle.build()
    c = synth.tiny_case()
    r = oracle.recipe(c["X"], c["W"], c["bias"], c["M"], c["N"], c["K"])
    out = {"X": digest(c["X"]), "W": digest(c["W"]), "bias": digest(c["bias"])}
    out.update({k: digest(v) for k, v in r.items()})
    doc = {"case": "tiny W8A8 linear, M=64 K=256 N=512, seed 0, alpha 0.5",
           "numpy": np.__version__, "sha256": out}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_case_digest.json")
    with open(path, "w") as f:
        json.dump(doc, f, indent=1, sort_keys=True)
        f.write("\n")
    print(path)


if __name__ == "__main__":
    main()
