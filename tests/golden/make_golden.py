"""Writes the oracle regression fixtures in this folder.

Calls only the oracle and the seeded input generators.  Run from the repo
root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2607_05708_amd import inputs  # noqa: E402


def tiny_retrieval(seed=0):
    """1,024 i.i.d. unit chunk embeddings (d = 256, fp32), 16 queries, top-8."""
    bank = inputs.iid_unit(seed, inputs.TAG_TINY, 2, 1024, 256, "f32")
    q = inputs.iid_unit(seed, inputs.TAG_TINY, 4, 16, 256, "f32")
    r = oracle.retrieve(q, bank, k=8, scale=1.0)
    return {
        "workload": "tiny retrieval: n=1024, d=256, fp32, m=16, k=8, scale=1, seed=%d" % seed,
        "idx": r["idx"].tolist(),
        "score": [[float.hex(float(x)) for x in row] for row in r["score"]],
        "lse": [float.hex(float(x)) for x in r["lse"]],
    }


if __name__ == "__main__":
    with open(os.path.join(HERE, "tiny_retrieval_seed0.json"), "w") as f:
        json.dump(tiny_retrieval(0), f, indent=1)
    print("wrote tiny_retrieval_seed0.json")
