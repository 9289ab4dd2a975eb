"""fp64 CPU oracle (ctypes binding over ``oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and
the benchmark's CPU-baseline leg, never by the GPU library or its binding.
It shares no code with the GPU path; both read the bytes the seeded
generators produce.

Definitions follow the paper's Algorithm 1 (relevance selection in its
Dense-only form of Section 5.5, FetchByID, SortByTime, Insert) and the
block directory of Section 4.2; see ``oracle.c`` for the formulas.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16 = 0, 1
ORDER_RANK, ORDER_TIME = 0, 1


def build(force: bool = True, src: str = _SRC, out: str = _LIB, defines=()) -> str:
    """Compile the oracle with gcc (plain C11, OpenMP, no fast-math)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall"]
        cmd += [f"-D{d}" for d in defines]
        subprocess.check_call(cmd + ["-o", tmp, src, "-lm"])
        os.replace(tmp, out)
    return out


def _bind(L):
    p, i64, i32, f64 = C.c_void_p, C.c_int64, C.c_int32, C.c_double
    L.oracle_scores.argtypes = [p, i64, p, i64, i64, i64, i32, i32, p, i32]
    L.oracle_scores.restype = None
    L.oracle_retrieve.argtypes = [p, i64, p, i64, i64, i64, i32, i32, i32, f64, p, p, p, p, p, p, i32]
    L.oracle_retrieve.restype = C.c_int
    L.oracle_retrieve_scoped.argtypes = [p, i64, p, i64, i64, i64, i32, i32, i32, f64, p, p, p, p, p, p, p, p, p, i32]
    L.oracle_retrieve_scoped.restype = C.c_int
    L.oracle_time_order.argtypes = [p, i64, i32, p]
    L.oracle_time_order.restype = None
    L.oracle_gather.argtypes = [p, i64, i64, p, i64, i32, p, i64, i32, i32, p]
    L.oracle_gather.restype = C.c_int
    L.oracle_gather_budget.argtypes = [p, i64, i64, p, i64, i32, p, i32, p, i64, i32, i32, p, p, p]
    L.oracle_gather_budget.restype = C.c_int
    L.oracle_compact.argtypes = [p, i64, i64, p, i64, i32, p, p, i32, i32, f64, i64, p, p, p, p]
    L.oracle_compact.restype = C.c_int
    L.oracle_colocate.argtypes = [p, i64, i64, p, i64, i32, p, p, i64, i32, C.c_float, i32, i64, p, p, p]
    L.oracle_colocate.restype = C.c_int
    L.oracle_payload_page.argtypes = [C.c_uint64, i64, i32, i32, i64, p]
    L.oracle_payload_page.restype = None
    L.oracle_expected_blocks.argtypes = [C.c_uint64, p, i64, i32, i32, i32, i64, p, i64, p, i32]
    L.oracle_expected_blocks.restype = None
    L.oracle_append_table.argtypes = [i64, i32, i64, p]
    L.oracle_append_table.restype = None
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = _bind(C.CDLL(_LIB))
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _dtype_of(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"embeddings must be float32 or uint16 (bf16 bits), got {a.dtype}")


def scores(q: np.ndarray, b: np.ndarray, threads: int = 0, L=None) -> np.ndarray:
    """s_ij = sum_t q_it b_jt in fp64, [m, n]."""
    q = np.ascontiguousarray(q)
    b = np.ascontiguousarray(b)
    dt = _dtype_of(q)
    assert _dtype_of(b) == dt and q.shape[1] == b.shape[1]
    out = np.empty((q.shape[0], b.shape[0]), dtype=np.float64)
    (L or lib()).oracle_scores(_ptr(q), q.shape[1], _ptr(b), b.shape[1], q.shape[0], b.shape[0], q.shape[1], dt,
                        _ptr(out), threads)
    return out


def retrieve(q: np.ndarray, b: np.ndarray, k: int, scale: float = 1.0, self_idx=None, full: bool = False,
             threads: int = 0, L=None) -> dict:
    """Dense relevance selection: top-k ids/scores/probabilities and lse per key."""
    q = np.ascontiguousarray(q)
    b = np.ascontiguousarray(b)
    dt = _dtype_of(q)
    assert _dtype_of(b) == dt and q.shape[1] == b.shape[1]
    m, n = q.shape[0], b.shape[0]
    idx = np.empty((m, k), dtype=np.int32)
    sc = np.empty((m, k), dtype=np.float64)
    pr = np.empty((m, k), dtype=np.float64)
    lse = np.empty(m, dtype=np.float64)
    fp = np.empty((m, n), dtype=np.float64) if full else None
    si = None if self_idx is None else np.ascontiguousarray(self_idx, dtype=np.int64)
    rc = (L or lib()).oracle_retrieve(_ptr(q), q.shape[1], _ptr(b), b.shape[1], m, n, q.shape[1], dt, k, float(scale),
                               _ptr(si), _ptr(idx), _ptr(sc), _ptr(pr), _ptr(lse), _ptr(fp), threads)
    if rc != 0:
        raise ValueError("some key has fewer than k candidates")
    out = {"idx": idx, "score": sc, "prob": pr, "lse": lse}
    if full:
        out["full_prob"] = fp
    return out


def retrieve_scoped(q: np.ndarray, b: np.ndarray, k: int, row_ns, row_live, key_ns, scale: float = 1.0,
                    self_idx=None, full: bool = False, threads: int = 0, L=None) -> dict:
    """Namespace-scoped, tombstone-aware selection: candidates of key i are the
    live bank rows whose namespace equals key_ns[i]; short results are padded
    with id -1, score -inf, p 0 (lse -inf with no candidate)."""
    q = np.ascontiguousarray(q)
    b = np.ascontiguousarray(b)
    dt = _dtype_of(q)
    assert _dtype_of(b) == dt and q.shape[1] == b.shape[1]
    m, n = q.shape[0], b.shape[0]
    rns = np.ascontiguousarray(row_ns, dtype=np.int32)
    rlv = np.ascontiguousarray(row_live, dtype=np.uint8)
    kns = np.ascontiguousarray(key_ns, dtype=np.int32)
    assert rns.shape == (n,) and rlv.shape == (n,) and kns.shape == (m,)
    idx = np.empty((m, k), dtype=np.int32)
    sc = np.empty((m, k), dtype=np.float64)
    pr = np.empty((m, k), dtype=np.float64)
    lse = np.empty(m, dtype=np.float64)
    fp = np.empty((m, n), dtype=np.float64) if full else None
    si = None if self_idx is None else np.ascontiguousarray(self_idx, dtype=np.int64)
    (L or lib()).oracle_retrieve_scoped(_ptr(q), q.shape[1], _ptr(b), b.shape[1], m, n, q.shape[1], dt, k, float(scale),
                                        _ptr(si), _ptr(rns), _ptr(rlv), _ptr(kns), _ptr(idx), _ptr(sc), _ptr(pr),
                                        _ptr(lse), _ptr(fp), threads)
    out = {"idx": idx, "score": sc, "prob": pr, "lse": lse}
    if full:
        out["full_prob"] = fp
    return out


def time_order(ids: np.ndarray, group: int, L=None) -> np.ndarray:
    ids = np.ascontiguousarray(ids, dtype=np.int32).ravel()
    out = np.empty_like(ids)
    (L or lib()).oracle_time_order(_ptr(ids), ids.shape[0], group, _ptr(out))
    return out


def gather(pool: np.ndarray, table: np.ndarray, ids: np.ndarray, order: int = ORDER_RANK,
           group: int = 1, L=None) -> np.ndarray:
    """out[i, p] = pool[table[id'_i, p]] as bytes [count, ppc, page_bytes]."""
    pool = np.ascontiguousarray(pool, dtype=np.uint8)
    table = np.ascontiguousarray(table, dtype=np.int32)
    ids = np.ascontiguousarray(ids, dtype=np.int32).ravel()
    n_pages, page_bytes = pool.shape
    n_chunks, ppc = table.shape
    out = np.empty((ids.shape[0], ppc, page_bytes), dtype=np.uint8)
    rc = (L or lib()).oracle_gather(_ptr(pool), n_pages, page_bytes, _ptr(table), n_chunks, ppc, _ptr(ids), ids.shape[0],
                             order, group, _ptr(out))
    if rc != 0:
        raise ValueError("id or page out of range")
    return out


def gather_budget(pool: np.ndarray, table: np.ndarray, tok_len: np.ndarray, ids: np.ndarray, budget: int,
                  row_bytes: int, L=None):
    """Budget-aware, time-ordered materialisation of rank-ordered ids [m, k]:
    (rows uint8 [m, budget, row_bytes], tokens int32 [m], kept ids int32 [m, k])."""
    pool = np.ascontiguousarray(pool, dtype=np.uint8)
    table = np.ascontiguousarray(table, dtype=np.int32)
    tl = np.ascontiguousarray(tok_len, dtype=np.int32)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    m, k = ids.shape
    n_pages, page_bytes = pool.shape
    n_chunks, ppc = table.shape
    assert tl.shape == (n_chunks,) and page_bytes % row_bytes == 0
    out = np.full((m, budget, row_bytes), 0xA5, dtype=np.uint8)   # so a missing zero tail shows
    tokens = np.empty(m, dtype=np.int32)
    kept = np.empty((m, k), dtype=np.int32)
    rc = (L or lib()).oracle_gather_budget(_ptr(pool), n_pages, page_bytes, _ptr(table), n_chunks, ppc, _ptr(tl),
                                           row_bytes, _ptr(ids), m, k, budget, _ptr(out), _ptr(tokens), _ptr(kept))
    if rc != 0:
        raise ValueError("id, token length or page out of range")
    return out, tokens, kept


def compact(pool: np.ndarray, table: np.ndarray, offsets: np.ndarray, chunks: np.ndarray, pages_per_block: int,
            theta: float, next_free: int, L=None) -> dict:
    """Background block compaction on copies of pool [n_pages, page_bytes]
    and table [n_chunks, ppc]; the per-namespace chunk tables are CSR
    (offsets [n_ns + 1], chunks).  Returns pool, table, phi [n_blocks],
    released [n_blocks], next_free and moved (pages)."""
    pool = np.array(pool, dtype=np.uint8, copy=True, order="C")
    table = np.array(table, dtype=np.int32, copy=True, order="C")
    offs = np.ascontiguousarray(offsets, dtype=np.int32)
    ch = np.ascontiguousarray(chunks, dtype=np.int32)
    n_pages, page_bytes = pool.shape
    n_chunks, ppc = table.shape
    n_blocks = (next_free + pages_per_block - 1) // pages_per_block
    phi = np.empty(n_blocks, dtype=np.float64)
    rel = np.empty(n_blocks, dtype=np.uint8)
    nf = C.c_int64(0)
    mv = C.c_int64(0)
    rc = (L or lib()).oracle_compact(_ptr(pool), n_pages, page_bytes, _ptr(table), n_chunks, ppc, _ptr(offs), _ptr(ch),
                                     offs.shape[0] - 1, pages_per_block, float(theta), next_free, _ptr(phi),
                                     _ptr(rel), C.byref(nf), C.byref(mv))
    if rc != 0:
        raise ValueError("pool too small for the fresh blocks, or chunk ids not ascending")
    return {"pool": pool, "table": table, "phi": phi, "released": rel, "next_free": int(nf.value),
            "moved": int(mv.value)}


def colocate(pool: np.ndarray, table: np.ndarray, ids: np.ndarray, scores: np.ndarray, tau: float, min_group: int,
             next_free: int, L=None) -> dict:
    """Association-aware relocation on copies of pool and table: each key's
    chunks with score >= tau (groups of at least min_group) are rewritten in
    time order to fresh pages.  Returns pool, table, next_free, moved
    (chunks) and groups."""
    pool = np.array(pool, dtype=np.uint8, copy=True, order="C")
    table = np.array(table, dtype=np.int32, copy=True, order="C")
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    sc = np.ascontiguousarray(scores, dtype=np.float32)
    m, k = ids.shape
    nf, mv, gr = C.c_int64(0), C.c_int64(0), C.c_int64(0)
    rc = (L or lib()).oracle_colocate(_ptr(pool), pool.shape[0], pool.shape[1], _ptr(table), table.shape[0],
                                      table.shape[1], _ptr(ids), _ptr(sc), m, k, C.c_float(tau), min_group, next_free,
                                      C.byref(nf), C.byref(mv), C.byref(gr))
    if rc != 0:
        raise ValueError("id out of range or pool too small for the fresh pages")
    return {"pool": pool, "table": table, "next_free": int(nf.value), "moved": int(mv.value),
            "groups": int(gr.value)}


def payload_page(key: int, chunk: int, page: int, ppc: int, page_bytes: int, L=None) -> np.ndarray:
    out = np.empty(page_bytes // 8, dtype=np.uint64)
    (L or lib()).oracle_payload_page(C.c_uint64(key), chunk, page, ppc, page_bytes, _ptr(out))
    return out


def expected_blocks(key: int, ids: np.ndarray, order: int, group: int, ppc: int, page_bytes: int,
                    slots=None, threads: int = 0, L=None) -> np.ndarray:
    """Gathered blocks for a pool holding payload(c, p) at page table[c, p];
    uint64 [len(slots), ppc, page_bytes/8]."""
    ids = np.ascontiguousarray(ids, dtype=np.int32).ravel()
    sl = None if slots is None else np.ascontiguousarray(slots, dtype=np.int64)
    ns = ids.shape[0] if sl is None else sl.shape[0]
    out = np.empty((ns, ppc, page_bytes // 8), dtype=np.uint64)
    (L or lib()).oracle_expected_blocks(C.c_uint64(key), _ptr(ids), ids.shape[0], order, group, ppc, page_bytes, _ptr(sl),
                                 ns, _ptr(out), threads)
    return out


def append_table(m: int, ppc: int, next_free: int, L=None) -> np.ndarray:
    out = np.empty((m, ppc), dtype=np.int32)
    (L or lib()).oracle_append_table(m, ppc, next_free, _ptr(out))
    return out
