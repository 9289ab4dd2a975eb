"""The scoped parity checker on the CPU: it accepts the oracle's own output
(rounded to the GPU's fp32 outputs) and rejects planted mistakes of the
kinds a scoped kernel could make."""
import numpy as np
import pytest

import oracle
from paper_2607_05708_amd import inputs
from parity import check_topk_scoped


def _case():
    b = inputs.iid_unit(3, 90, 0, 300, 32, "f32")
    q = inputs.iid_unit(3, 90, 4, 24, 32, "f32")
    rns, live, kns = inputs.namespaces(3, 90, 300, 40, 0.2, run=3, m=24)
    kns = kns.copy()
    kns[0] = -1
    ref = oracle.retrieve_scoped(q, b, 12, rns, live, kns, scale=2.0)
    g = {"idx": ref["idx"].copy(), "score": ref["score"].astype(np.float32),
         "prob": ref["prob"].astype(np.float32), "lse": ref["lse"].astype(np.float32)}
    return q, b, rns, live, kns, g


def _check(q, b, rns, live, kns, g):
    return check_topk_scoped("cpu", q, b, np.arange(q.shape[0]), g, 12, 2.0, rns, live, kns)


def test_accepts_oracle_output():
    q, b, rns, live, kns, g = _case()
    assert (g["idx"] == -1).any()             # the case has short rows ...
    assert g["lse"][0] == -np.inf             # ... and an empty one
    r = _check(q, b, rns, live, kns, g)
    assert r["exact_rows"] == int(np.count_nonzero(g["lse"] > -np.inf))   # every non-empty row


@pytest.mark.parametrize("mistake", ["out_of_scope", "tombstoned", "pad_zero", "pad_score", "lse_empty",
                                     "dropped_best"])
def test_rejects_planted_mistakes(mistake):
    q, b, rns, live, kns, g = _case()
    short = int(np.nonzero((g["idx"] == -1).any(axis=1) & (g["idx"][:, 0] >= 0))[0][0])
    full = int(np.nonzero((g["idx"] >= 0).all(axis=1))[0][0])
    if mistake == "out_of_scope":
        other = int(np.nonzero((rns != kns[full]) & (live != 0))[0][0])
        g["idx"][full, -1] = other
    elif mistake == "tombstoned":
        dead = int(np.nonzero((rns == kns[full]) & (live == 0))[0][0])
        g["idx"][full, -1] = dead
    elif mistake == "pad_zero":
        g["idx"][short, -1] = 0
    elif mistake == "pad_score":
        g["score"][short, -1] = 0.0
    elif mistake == "lse_empty":
        g["lse"][0] = 0.0
    else:
        g["idx"][full, :-1] = g["idx"][full, 1:].copy()
        g["score"][full, :-1] = g["score"][full, 1:].copy()
        g["idx"][full, -1] = -1
    with pytest.raises(AssertionError):
        _check(q, b, rns, live, kns, g)
