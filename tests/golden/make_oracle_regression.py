"""Writes oracle_regression.json: the oracle's outputs on a few tiny seeded
inputs, so that any later change to the oracle's arithmetic shows up as a
failing regression test (and must then be justified by a passage of the
paper).  Calls only the oracle; inputs come from numpy's PCG64 stream.

    python tests/golden/make_oracle_regression.py
"""
import hashlib
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
import oracle  # noqa: E402

CASES = [
    # B, Hq, Hkv, T, W, d, P, G, budget, gamma, tau, lam, mode, seed
    (1, 4, 1, 96, 8, 16, 32, 4, 12, 10.0, 0.95, 1.0, 0, 1),
    (2, 6, 2, 70, 5, 8, 16, 2, 9, 3.0, 0.9, 1.0, 0, 2),
    (1, 2, 2, 33, 4, 8, 8, 8, 5, 10.0, 0.95, 1.0, 1, 3),
]


def inputs(case):
    B, Hq, Hkv, T, W, d = case[:6]
    rng = np.random.Generator(np.random.PCG64(case[-1]))
    q = (rng.standard_normal((B, Hq, W, d)) + rng.standard_normal((B, Hq, 1, d))).astype(np.float32)
    k = rng.standard_normal((B, Hkv, T, d)).astype(np.float32)
    return q, k


def run(case):
    B, Hq, Hkv, T, W, d, P, G, budget, gamma, tau, lam, mode, seed = case
    q, k = inputs(case)
    r = oracle.select_layer(q, k, k, Hkv=Hkv, budget=budget, P=P, G=G, gamma=gamma, tau=tau,
                            lam=lam, seed=seed, layer=seed, mode=mode)
    return {
        "case": list(case),
        "proxies_sha256": hashlib.sha256(r.proxies.tobytes()).hexdigest(),
        "q_last_sha256": hashlib.sha256(r.q_last.tobytes()).hexdigest(),
        "mass_head": [float(x) for x in r.mass.ravel()[:8]],
        "anchor_head": [float(x) for x in r.anchor.ravel()[:8]],
        "votes_sum": int(r.sel.votes.sum()),
        "idx": r.sel.idx.tolist(),
    }


if __name__ == "__main__":
    out = {"note": "written by make_oracle_regression.py from the oracle only", "cases": [run(c) for c in CASES]}
    with open(os.path.join(HERE, "oracle_regression.json"), "w") as f:
        json.dump(out, f, indent=1)
