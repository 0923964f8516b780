"""Write tests/golden/tiny_oracle.json: input hashes and oracle values of the tiny workload.

Calls only the seeded input generator and oracle/ (never the GPU path). The
stored values guard against silent drift of either; they are not a pin of
the oracle's correctness (the pins in tests/test_oracle_pins.py are).
Run from the repository root:  python tests/golden/make_golden.py
"""
import hashlib
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2606_20005_amd import inputs  # noqa: E402


def sha(x):
    return hashlib.sha256(np.ascontiguousarray(x).tobytes()).hexdigest()


def main():
    d = inputs.make("tiny")
    w = d["w"]
    out = {"workload": "tiny", "seed": w.seed,
           "sha256": {k: sha(d[k]) for k in ("Q1", "K1", "Q2", "K2", "g")}}
    for causal in (False, True):
        kl, l1, l2, dQ1, dK1, dQ2, dK2 = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2,
                                                         causal, oracle.kl_oracle.FWD, d["g"])
        out["causal" if causal else "noncausal"] = {
            "kl_rows_0_16": kl[0, 0, :16].tolist(), "lse1_rows_0_16": l1[0, 0, :16].tolist(),
            "lse2_rows_0_16": l2[0, 0, :16].tolist(), "kl_sum": float(kl.sum()),
            "dQ2_norm": float(np.linalg.norm(dQ2)), "dK2_norm": float(np.linalg.norm(dK2)),
            "dQ1_norm": float(np.linalg.norm(dQ1)), "dK1_norm": float(np.linalg.norm(dK1))}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_oracle.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
