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
    assert r["exact_rows"] == q.shape[0]          # every row, the empty ones included


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


# ------------------------------------------------------------------ normaliser
# The unscoped checker on the CPU: the oracle's own output (rounded to the
# fp32 the GPU writes) passes; the same output with one split's share of the
# softmax sum dropped from lse and p (as a merge that lost one partial would
# produce) fails the fp32-derived rule, for 1/64 and 1/512 of the bank.

def _unscoped_case():
    from paper_2607_05708_amd import inputs as I
    n, d, m, k = 8192, 128, 12, 16
    cb = I.clustered_bank(5, 90, n, d, 64, 0.3, "bf16", m_queries=m)
    ref = oracle.retrieve(cb.queries, cb.emb, k, scale=1.0)
    g = {"idx": ref["idx"].copy(), "score": ref["score"][:, :k].astype(np.float32),
         "prob": ref["prob"][:, :k].astype(np.float32), "lse": ref["lse"].astype(np.float32)}
    return cb, g, k


def test_unscoped_accepts_oracle_output():
    from parity import check_topk
    cb, g, k = _unscoped_case()
    r = check_topk("cpu", cb.queries, cb.emb, np.arange(cb.queries.shape[0]), g, k, 1.0)
    assert r["exact_rows"] == r["rows"] and r["lse_err_max"] < 1e-5


@pytest.mark.parametrize("share", [64, 512])
def test_dropped_split_partial_fails_the_normaliser_rule(share):
    from parity import RTOL, check_topk
    cb, g, k = _unscoped_case()
    n = cb.emb.shape[0]
    s = oracle.scores(cb.queries, cb.emb)                   # fp64 [m, n]
    # one split of n/share rows holding none of the selected ids
    w = n // share
    start = next(b0 for b0 in range(0, n, w) if not np.any((g["idx"] >= b0) & (g["idx"] < b0 + w)))
    keep = np.ones(n, dtype=bool)
    keep[start:start + w] = False
    mx = s[:, keep].max(axis=1, keepdims=True)
    lse_drop = (mx[:, 0] + np.log(np.exp(s[:, keep] - mx).sum(axis=1)))
    assert np.all(np.isin(g["idx"], np.nonzero(keep)[0]))  # the winners themselves are unchanged
    bad = dict(g)
    bad["lse"] = lse_drop.astype(np.float32)
    # the stated 2e-2 rule alone cannot see it ...
    lse_ref = g["lse"].astype(np.float64)
    assert np.all(np.abs(lse_drop - lse_ref) <= RTOL["bf16"] * np.maximum(1.0, np.abs(lse_ref)))
    # ... the fp32 rule does, through lse and through p
    with pytest.raises(AssertionError, match="lse error .*fp32 rule"):
        check_topk("cpu", cb.queries, cb.emb, np.arange(cb.queries.shape[0]), bad, k, 1.0)
    bad = dict(g)
    bad["lse"] = None
    bad["prob"] = np.exp(g["score"].astype(np.float64) - lse_drop[:, None]).astype(np.float32)
    with pytest.raises(AssertionError, match="prob relative error .*fp32 rule"):
        check_topk("cpu", cb.queries, cb.emb, np.arange(cb.queries.shape[0]), bad, k, 1.0)


def test_doubled_split_partial_fails_the_normaliser_rule():
    from parity import check_topk
    cb, g, k = _unscoped_case()
    n = cb.emb.shape[0]
    s = oracle.scores(cb.queries, cb.emb)
    w = np.ones(n)
    w[:n // 512] = 2.0                                     # one split's partial counted twice
    mx = s.max(axis=1, keepdims=True)
    bad = dict(g)
    bad["lse"] = (mx[:, 0] + np.log((w * np.exp(s - mx)).sum(axis=1))).astype(np.float32)
    with pytest.raises(AssertionError, match="fp32 rule"):
        check_topk("cpu", cb.queries, cb.emb, np.arange(cb.queries.shape[0]), bad, k, 1.0)
