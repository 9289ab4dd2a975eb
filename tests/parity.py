"""Parity rules between the GPU path and the fp64 oracle.

Scores: |s_gpu - s_ref| <= rtol * max(|s_ref|, ||q_i|| ||b_j||), rtol = 2e-2 for
bf16 embeddings and 1e-5 for fp32 (the relative-tolerance reading used where
s is near 0 for unit vectors).
Top-k sets:
  (a) identical wherever the oracle's gap s_(k) - s_(k+1) exceeds rtol;
  (b) identical wherever that gap exceeds eps_i = 2 d 2^-24 ||q_i|| max_j ||b_j||,
      a bound on the fp32 accumulation error of either path, which any
      correct fp32-accumulating kernel meets;
  (c) on every row, an id may only be swapped across the k boundary with
      another id whose oracle score is within eps_i of the boundary.
Ties (equal fp32 scores) resolve to the lower id on both sides, so with
exactly representable scores (integer-grid inputs) ids must match exactly.
Softmax normaliser and probabilities, two rules each:
  (a) the stated score tolerance carried through: |lse - lse_ref| <=
      rtol * max(1, |lse_ref|), and, since p = exp(scale * s - lse), a score
      within rtol * r_i and an lse within that bound give
      |p - p_ref| <= (scale * rtol * r_i + rtol * max(1, |lse_ref|)) * p_ref
      (r_i = ||q_i|| max_j ||b_j||);
  (b) rules derived from the fp32 arithmetic both paths share the inputs of.
      lse is a smooth maximum of scale * s (its derivative in each score is
      that score's p, summing to 1), so a score error of at most eps_i moves it
      by at most scale * eps_i; fp32 summation of the exponentials, the exp2
      approximation and the rounding of scale * log2(e) add a relative error
      far below 1e-5 for the row lengths used here:
        |lse - lse_ref| <= tol_lse_i = scale * eps_i + 1e-5 * max(1, |lse_ref|);
      p = exp(scale * s - lse), so its relative error is bounded by the error
      of the exponent, plus fp32 rounding of the exponent's terms:
        |p - p_ref| <= (scale * eps_i + tol_lse_i + 1e-5 * max(1, scale * r_i)) * p_ref,
      with r_i = ||q_i|| max_j ||b_j|| (so |scale * s| <= scale * r_i).
  A merge that loses one partial's share w of the sum moves lse by ln(1 - w)
  (-0.0157 for a 1/64 share, -0.00195 for 1/512), which (a) misses and (b)
  catches.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2607_05708_amd import inputs

RTOL = {"f32": 1e-5, "bf16": 2e-2}


def decode(a: np.ndarray) -> np.ndarray:
    return inputs.bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


def bank_max_norm(b: np.ndarray, block: int = 65536) -> float:
    """max_j ||b_j|| in fp64, a block of rows at a time (no full fp64 copy of a large bank)."""
    return max(float(np.linalg.norm(decode(b[i:i + block]), axis=1).max()) for i in range(0, b.shape[0], block))


def pair_scores(q: np.ndarray, b: np.ndarray, rows: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Oracle scores s[rows[i], ids[i, r]] without scoring the whole bank."""
    out = np.empty(ids.shape, dtype=np.float64)
    for i, row in enumerate(rows):
        sel = ids[i]
        out[i] = oracle.scores(q[row:row + 1], np.ascontiguousarray(b[sel]))[0]
    return out


def check_topk(name: str, q: np.ndarray, b: np.ndarray, rows: np.ndarray, gpu: dict, k: int, scale: float,
               self_idx=None, exact: bool = False, bmax: float | None = None) -> dict:
    """Compare GPU outputs for query rows `rows` (indices into q) with the oracle.

    gpu: dict of numpy arrays idx [len(rows), k], score, prob, lse.
    bmax: max_j ||b_j|| if the caller has it (computed from b otherwise).
    Returns the row count, the rows whose set is bit-exact (reported, not
    gated beyond the rules above) and the largest lse error.
    """
    dt = "bf16" if q.dtype == np.uint16 else "f32"
    rtol = RTOL[dt]
    d = q.shape[1]
    qs = np.ascontiguousarray(q[rows])
    si = None if self_idx is None else np.asarray(self_idx)[rows]
    kk = min(k + 1, b.shape[0] - (0 if si is None else 1))
    ref = oracle.retrieve(qs, b, kk, scale=scale, self_idx=si)
    ref_idx, ref_s, lse_ref = ref["idx"][:, :k], ref["score"], ref["lse"]
    gi = gpu["idx"].astype(np.int64)
    assert gi.shape == (len(rows), k), name
    assert np.all((gi >= 0) & (gi < b.shape[0])), f"{name}: id out of range"
    if si is not None:
        assert not np.any(gi == si[:, None]), f"{name}: self selected"
    for i in range(len(rows)):
        assert len(set(gi[i].tolist())) == k, f"{name}: duplicate ids in row {rows[i]}"
    s_gpu_ref = pair_scores(q, b, rows, gi)
    qn = np.linalg.norm(decode(qs), axis=1)
    if bmax is None:
        bmax = bank_max_norm(b)
    scale_ij = np.maximum(np.abs(s_gpu_ref), qn[:, None] * np.linalg.norm(decode(b[gi.ravel()]), axis=1).reshape(gi.shape))
    err = np.abs(gpu["score"].astype(np.float64) - s_gpu_ref)
    assert np.all(err <= rtol * scale_ij), f"{name}: score error {err.max():.3g}"
    eps = 2.0 * d * 2.0 ** -24 * qn * bmax
    if exact:
        assert np.array_equal(gi, ref_idx), f"{name}: ids differ on exact inputs"
        assert np.array_equal(gpu["score"].astype(np.float64), ref_s[:, :k]), f"{name}: scores differ on exact inputs"
    kth = ref_s[:, k - 1]
    nxt = ref_s[:, k] if kk > k else np.full(len(rows), -np.inf)
    gap = kth - nxt
    n_exact = 0
    for i in range(len(rows)):
        same = set(gi[i].tolist()) == set(ref_idx[i].tolist())
        n_exact += same
        if gap[i] > rtol or gap[i] > eps[i]:
            assert same, f"{name}: row {rows[i]} set differs with gap {gap[i]:.3g}"
        if not same:
            extra = set(gi[i].tolist()) - set(ref_idx[i].tolist())
            missing = set(ref_idx[i].tolist()) - set(gi[i].tolist())
            se = pair_scores(q, b, rows[i:i + 1], np.array([sorted(extra)]))[0]
            sm = pair_scores(q, b, rows[i:i + 1], np.array([sorted(missing)]))[0]
            assert np.all(se >= kth[i] - eps[i]), f"{name}: row {rows[i]} selected a non-boundary id"
            assert np.all(sm <= nxt[i] + eps[i]), f"{name}: row {rows[i]} dropped a non-boundary id"
    # rank order on the GPU side: scores non-increasing, equal scores by id
    gs = gpu["score"]
    for i in range(len(rows)):
        for r in range(k - 1):
            assert gs[i, r] > gs[i, r + 1] or (gs[i, r] == gs[i, r + 1] and gi[i, r] < gi[i, r + 1]), \
                f"{name}: row {rows[i]} not in rank order"
    tol_lse, tol_p = normaliser_tolerances(scale, eps, lse_ref, qn * bmax)
    if "lse" in gpu and gpu["lse"] is not None:
        lerr = np.abs(gpu["lse"].astype(np.float64) - lse_ref)
        assert np.all(lerr <= rtol * np.maximum(1.0, np.abs(lse_ref))), f"{name}: lse error {lerr.max():.3g}"
        bad = np.nonzero(lerr > tol_lse)[0]
        assert bad.size == 0, \
            f"{name}: lse error {lerr[bad[0]]:.3g} > {tol_lse[bad[0]]:.3g} (fp32 rule) in row {rows[bad[0]]}"
    if "prob" in gpu and gpu["prob"] is not None:
        p_ref = np.exp(scale * s_gpu_ref - lse_ref[:, None])
        perr = np.abs(gpu["prob"].astype(np.float64) - p_ref)
        tol_stated = scale * rtol * qn * bmax + rtol * np.maximum(1.0, np.abs(lse_ref))
        assert np.all(perr <= tol_stated[:, None] * p_ref + 1e-30), f"{name}: prob error {(perr / p_ref).max():.3g}"
        rel = perr / np.maximum(p_ref, 1e-300)
        bad = np.argwhere(rel > tol_p[:, None])
        assert bad.size == 0, \
            f"{name}: prob relative error {rel.max():.3g} > {tol_p[bad[0][0]]:.3g} (fp32 rule) in row {rows[bad[0][0]]}"
    return {"rows": len(rows), "exact_rows": n_exact,
            "lse_err_max": float(np.max(np.abs(gpu["lse"].astype(np.float64) - lse_ref)))
            if gpu.get("lse") is not None else None}


def normaliser_tolerances(scale: float, eps, lse_ref, r):
    """Rule (b) for lse and p (module docstring): per-row absolute lse bound
    and relative p bound from the fp32 score bound eps_i and r_i = ||q_i|| max ||b_j||."""
    eps = np.asarray(eps, dtype=np.float64)
    lse_ref = np.asarray(lse_ref, dtype=np.float64)
    tol_lse = scale * eps + 1e-5 * np.maximum(1.0, np.abs(lse_ref))
    tol_p = scale * eps + tol_lse + 1e-5 * np.maximum(1.0, scale * np.asarray(r, dtype=np.float64))
    return tol_lse, tol_p


def check_topk_scoped(name: str, q: np.ndarray, b: np.ndarray, rows: np.ndarray, gpu: dict, k: int, scale: float,
                      row_ns: np.ndarray, row_live: np.ndarray, key_ns: np.ndarray, self_idx=None) -> dict:
    """check_topk's rules for namespace-scoped selection, on query rows `rows`.

    Candidates of query i: live rows (row_live) with row_ns == key_ns[i], minus
    self_idx[i].  With c_i candidates the first min(k, c_i) slots follow
    check_topk's rules within the candidates; slots past c_i hold id -1,
    score -inf and p 0; lse is -inf when c_i = 0.
    """
    dt = "bf16" if q.dtype == np.uint16 else "f32"
    rtol = RTOL[dt]
    d = q.shape[1]
    n = b.shape[0]
    qs = np.ascontiguousarray(q[rows])
    kns = np.asarray(key_ns)[rows]
    si = None if self_idx is None else np.asarray(self_idx)[rows]
    ref = oracle.retrieve_scoped(qs, b, k + 1, row_ns, row_live, kns, scale=scale, self_idx=si)
    gi = gpu["idx"].astype(np.int64)
    gs = gpu["score"].astype(np.float64)
    assert gi.shape == (len(rows), k), name
    bnorm = np.linalg.norm(decode(b), axis=1)
    qn = np.linalg.norm(decode(qs), axis=1)
    n_exact = 0
    for i in range(len(rows)):
        cand = (np.asarray(row_live) != 0) & (np.asarray(row_ns) == kns[i])
        if si is not None and 0 <= si[i] < n:
            cand[si[i]] = False
        c = int(cand.sum())
        have = min(k, c)
        # padding
        assert np.all(gi[i, have:] == -1), f"{name}: row {rows[i]} not padded with -1"
        assert np.all(gs[i, have:] == -np.inf), f"{name}: row {rows[i]} padding score is not -inf"
        if "prob" in gpu and gpu["prob"] is not None:
            assert np.all(gpu["prob"][i, have:] == 0), f"{name}: row {rows[i]} padding p is not 0"
        if c == 0:
            if "lse" in gpu and gpu["lse"] is not None:
                assert gpu["lse"][i] == -np.inf, f"{name}: row {rows[i]} empty scope, lse {gpu['lse'][i]}"
            n_exact += 1  # all padding, as the oracle's (checked above)
            continue
        ids = gi[i, :have]
        assert np.all((ids >= 0) & (ids < n)), f"{name}: row {rows[i]} id out of range"
        assert np.all(cand[ids]), f"{name}: row {rows[i]} selected a row outside its scope"
        assert len(set(ids.tolist())) == have, f"{name}: row {rows[i]} duplicate ids"
        s_ref = oracle.scores(qs[i:i + 1], np.ascontiguousarray(b[ids]))[0]
        tol = rtol * np.maximum(np.abs(s_ref), qn[i] * bnorm[ids])
        err = np.abs(gs[i, :have] - s_ref)
        assert np.all(err <= tol), f"{name}: row {rows[i]} score error {err.max():.3g}"
        for r in range(have - 1):
            assert gs[i, r] > gs[i, r + 1] or (gs[i, r] == gs[i, r + 1] and ids[r] < ids[r + 1]), \
                f"{name}: row {rows[i]} not in rank order"
        ref_ids = ref["idx"][i, :have].astype(np.int64)
        ref_s = ref["score"][i]
        eps = 2.0 * d * 2.0 ** -24 * qn[i] * bnorm[cand].max()
        kth = ref_s[have - 1]
        nxt = ref_s[have] if ref["idx"][i, have] >= 0 else -np.inf
        gap = kth - nxt
        same = set(ids.tolist()) == set(ref_ids.tolist())
        n_exact += same
        if gap > rtol or gap > eps:
            assert same, f"{name}: row {rows[i]} set differs with gap {gap:.3g}"
        if not same:
            extra = sorted(set(ids.tolist()) - set(ref_ids.tolist()))
            missing = sorted(set(ref_ids.tolist()) - set(ids.tolist()))
            se = oracle.scores(qs[i:i + 1], np.ascontiguousarray(b[extra]))[0]
            sm = oracle.scores(qs[i:i + 1], np.ascontiguousarray(b[missing]))[0]
            assert np.all(se >= kth - eps), f"{name}: row {rows[i]} selected a non-boundary id"
            assert np.all(sm <= nxt + eps), f"{name}: row {rows[i]} dropped a non-boundary id"
        lse_ref = ref["lse"][i]
        tol_lse, tol_p = normaliser_tolerances(scale, eps, lse_ref, qn[i] * bnorm[cand].max())
        if "lse" in gpu and gpu["lse"] is not None:
            lerr = abs(float(gpu["lse"][i]) - lse_ref)
            assert lerr <= rtol * max(1.0, abs(lse_ref)), f"{name}: row {rows[i]} lse error {lerr:.3g}"
            assert lerr <= tol_lse, f"{name}: row {rows[i]} lse error {lerr:.3g} > {float(tol_lse):.3g} (fp32 rule)"
        if "prob" in gpu and gpu["prob"] is not None:
            p_ref = np.exp(scale * s_ref - lse_ref)
            perr = np.abs(gpu["prob"][i, :have].astype(np.float64) - p_ref)
            tol_stated = scale * rtol * qn[i] * bnorm[cand].max() + rtol * max(1.0, abs(lse_ref))
            assert np.all(perr <= tol_stated * p_ref + 1e-30), f"{name}: row {rows[i]} prob error"
            assert np.all(perr <= tol_p * p_ref), f"{name}: row {rows[i]} prob error {(perr / p_ref).max():.3g} (fp32 rule)"
    return {"rows": len(rows), "exact_rows": n_exact}
