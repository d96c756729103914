"""Writes tests/golden/brute_tiny.json: tiny FEM-read cases evaluated term by
term at 50 significant digits by the oracle's brute-force evaluator.

The inputs are small fixed decimals written out here so that the fixture is
self-describing; the expected values come only from ``oracle.brute``.
Run from the repository root:  python tests/golden/make_golden.py
"""

import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))

import numpy as np  # noqa: E402

from oracle import brute  # noqa: E402


def case(seed, T, d, D, beta_lo, beta_hi, kind):
    rng = np.random.default_rng(seed)
    # Values rounded to 3 decimals: exact decimal inputs, easy to retype.
    q = np.round(rng.standard_normal((T, d)), 3)
    k = np.round(rng.standard_normal((T, d)), 3)
    v = np.round(rng.standard_normal((T, D)) * 2.0, 3)
    beta = np.round(np.exp(rng.uniform(np.log(beta_lo), np.log(beta_hi), D)), 3)
    fn = brute.brute_fem_softmax if kind == "softmax" else brute.brute_fem_linear
    out = fn(q.tolist(), k.tolist(), v.tolist(), beta.tolist(), dps=50)
    return {
        "kind": kind, "seed": seed, "T": T, "d": d, "D": D,
        "q": q.tolist(), "k": k.tolist(), "v": v.tolist(), "beta": beta.tolist(),
        "out": [[str(x) for x in row] for row in out],
    }


def main():
    cases = [
        case(1, 6, 3, 4, 0.1, 8.0, "softmax"),
        case(2, 12, 4, 3, 0.05, 20.0, "softmax"),
        case(3, 24, 8, 2, 0.5, 4.0, "softmax"),
        case(4, 9, 3, 3, 0.1, 8.0, "linear"),
        case(5, 20, 4, 2, 0.1, 4.0, "linear"),
    ]
    doc = {
        "about": "FEM read, 0-based causal support {0..t}; values are mpmath 50-digit "
                 "term-by-term evaluations of F = log(sum_i p_t(i) exp(beta v_ij))/beta "
                 "(Sec. 2.3, free-energy read) with the softmax prior q.k/sqrt(d) "
                 "(Sec. 1) or the linear prior phi=elu+1 (Appendix, linear attention).",
        "generator": "tests/golden/make_golden.py (calls oracle.brute only)",
        "cases": cases,
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "brute_tiny.json")
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
