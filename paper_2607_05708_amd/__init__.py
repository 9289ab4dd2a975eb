"""Python binding of libmemattn.so: dense MemAttention retrieval and chunk
materialisation on one MI355X.

Argument marshalling only: every step runs in the library's HIP kernels;
PyTorch supplies device memory and the current stream.  The library must
have been built (``python -m paper_2607_05708_amd.build``); nothing here
falls back to another implementation.

Names follow the C ABI in ``include/memattn.h``:

* ``mem_retrieve_topk``   -- query-aware retrieval (LLMSelect of Algorithm 1
  in the Dense-only form of Section 5.5)
* ``mem_build_relations`` -- cross-chunk relations of every bank row
* ``mem_retrieve_topk_scoped`` / ``mem_build_relations_scoped`` -- the same,
  restricted to each key's (user, session) namespace and to live rows
  (T[u][s] of Section 4.1, tombstones of Section 4.2)
* ``mem_retrieve_topk_grouped`` -- the scoped retrieval over per-namespace
  chunk tables, each query scored against its own table only
* ``mem_gather_chunks``   -- FetchByID + SortByTime through the page table
* ``mem_gather_budget``   -- the same within a memory token budget, packed as
  token rows (the prompt prefix of Section 4.3)
* ``mem_append_chunks``   -- Insert with append-only page allocation
* ``mem_compact_blocks``  -- background block compaction (Eq. 2, Algorithm 2)
* ``mem_colocate``        -- association-aware relocation (Algorithm 2, online stage)
"""
from __future__ import annotations

import ctypes as C
import os

import torch  # noqa: F401  (loads the HIP runtime the library binds to)

__all__ = ["MemError", "MEM_F32", "MEM_BF16", "MEM_ORDER_RANK", "MEM_ORDER_TIME", "library_path", "lib",
           "mem_workspace_bytes", "mem_retrieve_topk", "mem_retrieve_topk_noalloc", "mem_scratch_bytes",
           "mem_build_relations", "mem_retrieve_topk_scoped",
           "mem_build_relations_scoped", "mem_workspace_bytes_grouped", "mem_retrieve_topk_grouped", "mem_gather_chunks", "mem_gather_budget", "mem_append_chunks",
           "mem_compact_workspace_bytes", "mem_compact_blocks", "mem_colocate_workspace_bytes", "mem_colocate",
           "BankState"]

_HERE = os.path.dirname(os.path.abspath(__file__))
MEM_F32, MEM_BF16 = 0, 1
MEM_ORDER_RANK, MEM_ORDER_TIME = 0, 1


class MemBank(C.Structure):
    _fields_ = [("emb", C.c_void_p), ("n", C.c_int64), ("d", C.c_int32), ("dtype", C.c_int32),
                ("row_stride", C.c_int64)]


class MemTopkOut(C.Structure):
    _fields_ = [("idx", C.c_void_p), ("score", C.c_void_p), ("prob", C.c_void_p), ("lse", C.c_void_p)]


class MemPages(C.Structure):
    _fields_ = [("pool", C.c_void_p), ("n_pages", C.c_int64), ("page_bytes", C.c_int64), ("table", C.c_void_p),
                ("n_chunks", C.c_int64), ("pages_per_chunk", C.c_int32)]


class MemChunkTables(C.Structure):
    _fields_ = [("offsets", C.c_void_p), ("chunks", C.c_void_p), ("n_ns", C.c_int32), ("n_entries", C.c_int64)]


class MemCompactResult(C.Structure):
    _fields_ = [("moved_pages", C.c_int64), ("released_blocks", C.c_int64), ("next_free_page", C.c_int64)]


class MemColocateResult(C.Structure):
    _fields_ = [("moved_chunks", C.c_int64), ("groups", C.c_int64), ("next_free_page", C.c_int64)]


class MemError(RuntimeError):
    def __init__(self, call: str, status: int, message: str):
        super().__init__(f"{call}: status {status}: {message}")
        self.status = status


_lib = None


def library_path() -> str:
    return os.path.join(_HERE, "libmemattn.so")


def lib():
    """Load libmemattn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m paper_2607_05708_amd.build`")
        L = C.CDLL(path)
        P, i64, i32, f32 = C.c_void_p, C.c_int64, C.c_int32, C.c_float
        L.mem_workspace_bytes.argtypes = [i64, i64, i32, i32, i32]
        L.mem_workspace_bytes.restype = C.c_size_t
        L.mem_retrieve_topk.argtypes = [C.POINTER(MemBank), P, i64, i64, i32, f32, MemTopkOut, P, P, C.c_size_t, P]
        L.mem_retrieve_topk.restype = C.c_int
        L.mem_retrieve_topk_noalloc.argtypes = [C.POINTER(MemBank), P, i64, i64, i32, f32, MemTopkOut, P, P]
        L.mem_retrieve_topk_noalloc.restype = C.c_int
        L.mem_scratch_bytes.argtypes = []
        L.mem_scratch_bytes.restype = C.c_size_t
        L.mem_build_relations.argtypes = [C.POINTER(MemBank), i32, f32, i32, MemTopkOut, P, C.c_size_t, P]
        L.mem_build_relations.restype = C.c_int
        L.mem_retrieve_topk_scoped.argtypes = [C.POINTER(MemBank), P, P, P, i64, i64, i32, f32, MemTopkOut, P, P,
                                               C.c_size_t, P]
        L.mem_retrieve_topk_scoped.restype = C.c_int
        L.mem_build_relations_scoped.argtypes = [C.POINTER(MemBank), P, i32, f32, i32, MemTopkOut, P, C.c_size_t, P]
        L.mem_build_relations_scoped.restype = C.c_int
        L.mem_gather_chunks.argtypes = [C.POINTER(MemPages), P, i64, i32, i32, P, P]
        L.mem_gather_chunks.restype = C.c_int
        L.mem_workspace_bytes_grouped.argtypes = [i64, i32, i64, i32, i32]
        L.mem_workspace_bytes_grouped.restype = C.c_size_t
        L.mem_retrieve_topk_grouped.argtypes = [C.POINTER(MemBank), C.POINTER(MemChunkTables), P, P, i64, i64, i32,
                                                f32, MemTopkOut, P, C.c_size_t, P]
        L.mem_retrieve_topk_grouped.restype = C.c_int
        L.mem_gather_budget.argtypes = [C.POINTER(MemPages), P, i32, P, i64, i32, i32, P, P, P, P]
        L.mem_gather_budget.restype = C.c_int
        L.mem_compact_workspace_bytes.argtypes = [i64, i32, i64, i32, i32]
        L.mem_compact_workspace_bytes.restype = C.c_size_t
        L.mem_compact_blocks.argtypes = [P, i64, i64, P, i64, i32, C.POINTER(MemChunkTables), i32, f32, i64, P, P,
                                         C.POINTER(MemCompactResult), P, C.c_size_t, P]
        L.mem_compact_blocks.restype = C.c_int
        L.mem_colocate_workspace_bytes.argtypes = [i64, i32, i64]
        L.mem_colocate_workspace_bytes.restype = C.c_size_t
        L.mem_colocate.argtypes = [P, i64, i64, P, i64, i32, P, P, i64, i32, f32, i32, i64,
                                   C.POINTER(MemColocateResult), P, C.c_size_t, P]
        L.mem_colocate.restype = C.c_int
        L.mem_append_chunks.argtypes = [C.POINTER(MemBank), i64, P, i64, i64, P, i32, C.POINTER(C.c_int64), i64, P]
        L.mem_append_chunks.restype = C.c_int
        L.mem_status_string.argtypes = [C.c_int]
        L.mem_status_string.restype = C.c_char_p
        L.mem_last_error.argtypes = []
        L.mem_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _check(call: str, status: int) -> None:
    if status != 0:
        L = lib()
        raise MemError(call, status, f"{L.mem_status_string(status).decode()}: {L.mem_last_error().decode()}")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return MEM_F32
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return MEM_BF16
    raise TypeError(f"embeddings must be float32 or bfloat16 (or int16/uint16 bf16 bits), got {t.dtype}")


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    return t


def _rows(t: torch.Tensor, name: str):
    _dev(t, name)
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be 2-D with unit stride along the embedding dimension")
    return t.shape[0], t.shape[1], t.stride(0)


def _stream(stream):
    return (stream if stream is not None else torch.cuda.current_stream()).cuda_stream


def _bank(emb: torch.Tensor, n: int | None = None) -> MemBank:
    rows, d, stride = _rows(emb, "bank")
    return MemBank(emb.data_ptr(), rows if n is None else n, d, _dtype_code(emb), stride)


def mem_workspace_bytes(m: int, n: int, d: int, k: int, dtype: int) -> int:
    return int(lib().mem_workspace_bytes(m, n, d, k, dtype))


def _topk_out(m, k, device, out):
    if out is None:
        out = (torch.empty((m, k), dtype=torch.int32, device=device),
               torch.empty((m, k), dtype=torch.float32, device=device),
               torch.empty((m, k), dtype=torch.float32, device=device),
               torch.empty((m,), dtype=torch.float32, device=device))
    if len(out) != 4:
        raise ValueError("out must be a tuple (idx, score, prob, lse)")
    idx, score, prob, lse = out
    if idx is None:
        raise ValueError("out.idx is required")
    # the kernels write m*k int32/float values (m for lse) through these
    # pointers, so dtype and shape are checked here, before any launch
    for t, nm, dt, shape in ((idx, "idx", torch.int32, (m, k)), (score, "score", torch.float32, (m, k)),
                             (prob, "prob", torch.float32, (m, k)), (lse, "lse", torch.float32, (m,))):
        if t is None:
            continue
        if not isinstance(t, torch.Tensor) or t.dtype != dt or tuple(t.shape) != shape:
            got = f"{t.dtype} {list(t.shape)}" if isinstance(t, torch.Tensor) else type(t).__name__
            raise ValueError(f"out.{nm} must be {dt} of shape {list(shape)}, got {got}")
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"out.{nm} must be a contiguous GPU tensor")
    ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    return out, MemTopkOut(ptr(idx), ptr(score), ptr(prob), ptr(lse))


def _workspace(nbytes, device, workspace):
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
    _dev(workspace, "workspace")
    return workspace, workspace.numel() * workspace.element_size()


def _full_prob(full_prob, m, n):
    if full_prob is None:
        return None
    _dev(full_prob, "full_prob")
    if full_prob.dtype != torch.float32 or not full_prob.is_contiguous() or tuple(full_prob.shape) != (m, n):
        raise ValueError("full_prob must be a contiguous float32 [m, n] GPU tensor")
    return full_prob.data_ptr()


def _ns(t: torch.Tensor, length: int, name: str) -> int:
    _dev(t, name)
    if t.dtype != torch.int32 or t.dim() != 1 or not t.is_contiguous() or t.shape[0] != length:
        raise ValueError(f"{name} must be a contiguous int32 [{length}] GPU tensor")
    return t.data_ptr()


def mem_retrieve_topk(bank: torch.Tensor, queries: torch.Tensor, k: int, scale: float = 1.0, *, out=None,
                      full_prob: torch.Tensor | None = None, workspace: torch.Tensor | None = None, stream=None):
    """Top-k chunk ids, scores, probabilities and lse per query: (idx, score, prob, lse)."""
    b = _bank(bank)
    m, d, q_stride = _rows(queries, "queries")
    if d != b.d or _dtype_code(queries) != b.dtype:
        raise ValueError("queries must match the bank's dtype and dimension")
    out, o = _topk_out(m, k, bank.device, out)
    ws, ws_bytes = _workspace(mem_workspace_bytes(m, b.n, b.d, k, b.dtype), bank.device, workspace)
    fp = _full_prob(full_prob, m, b.n)
    _check("mem_retrieve_topk", lib().mem_retrieve_topk(C.byref(b), queries.data_ptr(), m, q_stride, k, scale, o, fp,
                                                        ws.data_ptr(), ws_bytes, _stream(stream)))
    return out


def mem_scratch_bytes() -> int:
    return int(lib().mem_scratch_bytes())


def mem_retrieve_topk_noalloc(bank: torch.Tensor, queries: torch.Tensor, k: int, scale: float = 1.0, *, out,
                              full_prob: torch.Tensor | None = None, stream=None):
    """mem_retrieve_topk with the library's fixed scratch array as workspace: the library allocates nothing.
    ``out`` (idx, score, prob, lse) must be supplied by the caller."""
    b = _bank(bank)
    m, d, q_stride = _rows(queries, "queries")
    if d != b.d or _dtype_code(queries) != b.dtype:
        raise ValueError("queries must match the bank's dtype and dimension")
    if out is None:
        raise ValueError("out must be supplied (this call allocates nothing)")
    out, o = _topk_out(m, k, bank.device, out)
    fp = _full_prob(full_prob, m, b.n)
    _check("mem_retrieve_topk_noalloc", lib().mem_retrieve_topk_noalloc(C.byref(b), queries.data_ptr(), m, q_stride,
                                                                        k, scale, o, fp, _stream(stream)))
    return out


def mem_retrieve_topk_scoped(bank: torch.Tensor, row_ns: torch.Tensor, queries: torch.Tensor,
                             query_ns: torch.Tensor, k: int, scale: float = 1.0, *, out=None,
                             full_prob: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                             stream=None):
    """mem_retrieve_topk over each query's namespace: candidates of query i are the bank rows j with
    row_ns[j] >= 0 and row_ns[j] == query_ns[i] (int32 GPU tensors; negative row_ns = tombstoned).
    Rows with fewer than k candidates are padded with id -1, score -inf, p 0."""
    b = _bank(bank)
    m, d, q_stride = _rows(queries, "queries")
    if d != b.d or _dtype_code(queries) != b.dtype:
        raise ValueError("queries must match the bank's dtype and dimension")
    rn, qn = _ns(row_ns, b.n, "row_ns"), _ns(query_ns, m, "query_ns")
    out, o = _topk_out(m, k, bank.device, out)
    ws, ws_bytes = _workspace(mem_workspace_bytes(m, b.n, b.d, k, b.dtype), bank.device, workspace)
    fp = _full_prob(full_prob, m, b.n)
    _check("mem_retrieve_topk_scoped",
           lib().mem_retrieve_topk_scoped(C.byref(b), rn, queries.data_ptr(), qn, m, q_stride, k, scale, o, fp,
                                          ws.data_ptr(), ws_bytes, _stream(stream)))
    return out


def mem_build_relations(bank: torch.Tensor, k: int, scale: float = 1.0, exclude_self: bool = True, *, out=None,
                        workspace: torch.Tensor | None = None, stream=None):
    """Top-k related chunks of every bank row: (idx, score, prob, lse), each [n, ...]."""
    b = _bank(bank)
    out, o = _topk_out(b.n, k, bank.device, out)
    ws, ws_bytes = _workspace(mem_workspace_bytes(b.n, b.n, b.d, k, b.dtype), bank.device, workspace)
    _check("mem_build_relations", lib().mem_build_relations(C.byref(b), k, scale, 1 if exclude_self else 0, o,
                                                            ws.data_ptr(), ws_bytes, _stream(stream)))
    return out


def mem_workspace_bytes_grouped(m: int, n_ns: int, n_entries: int, d: int, k: int) -> int:
    return int(lib().mem_workspace_bytes_grouped(m, n_ns, n_entries, d, k))


def mem_retrieve_topk_grouped(bank: torch.Tensor, offsets: torch.Tensor, chunks: torch.Tensor,
                              queries: torch.Tensor, query_ns: torch.Tensor, k: int, scale: float = 1.0, *,
                              out=None, workspace: torch.Tensor | None = None, stream=None):
    """Retrieval of each query within its own namespace's chunk table (CSR: ``offsets`` int32 [n_ns + 1],
    ``chunks`` int32 bank rows, ascending within a namespace): (idx, score, prob, lse), padded with -1."""
    b = _bank(bank)
    m, d, q_stride = _rows(queries, "queries")
    if d != b.d or _dtype_code(queries) != b.dtype:
        raise ValueError("queries must match the bank's dtype and dimension")
    n_ns = offsets.shape[0] - 1
    _ns(offsets, n_ns + 1, "offsets")
    qn = _ns(query_ns, m, "query_ns")
    n_entries = chunks.shape[0]
    if n_entries:
        _ns(chunks, n_entries, "chunks")
    T = MemChunkTables(offsets.data_ptr(), chunks.data_ptr() if n_entries else None, n_ns, n_entries)
    out, o = _topk_out(m, k, bank.device, out)
    ws, ws_bytes = _workspace(mem_workspace_bytes_grouped(m, n_ns, n_entries, b.d, k), bank.device, workspace)
    _check("mem_retrieve_topk_grouped",
           lib().mem_retrieve_topk_grouped(C.byref(b), C.byref(T), queries.data_ptr(), qn, m, q_stride, k, scale, o,
                                           ws.data_ptr(), ws_bytes, _stream(stream)))
    return out


def mem_build_relations_scoped(bank: torch.Tensor, row_ns: torch.Tensor, k: int, scale: float = 1.0,
                               exclude_self: bool = True, *, out=None, workspace: torch.Tensor | None = None,
                               stream=None):
    """mem_build_relations with each row's candidates limited to the live rows of its own namespace
    (row_ns int32 [n]; a tombstoned row, row_ns < 0, gets an all-padding result)."""
    b = _bank(bank)
    rn = _ns(row_ns, b.n, "row_ns")
    out, o = _topk_out(b.n, k, bank.device, out)
    ws, ws_bytes = _workspace(mem_workspace_bytes(b.n, b.n, b.d, k, b.dtype), bank.device, workspace)
    _check("mem_build_relations_scoped",
           lib().mem_build_relations_scoped(C.byref(b), rn, k, scale, 1 if exclude_self else 0, o, ws.data_ptr(),
                                            ws_bytes, _stream(stream)))
    return out


def mem_gather_chunks(pool: torch.Tensor, table: torch.Tensor, ids: torch.Tensor, order: int = MEM_ORDER_RANK,
                      group: int = 1, *, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Gathered blocks, uint8 [count, pages_per_chunk, page_bytes].

    ``pool``: uint8 [n_pages, page_bytes]; ``table``: int32 [n_chunks, ppc]; ``ids``: int32, any shape
    (flattened in row-major order; with MEM_ORDER_TIME each consecutive ``group`` ids are time-sorted).
    """
    for t, nm in ((pool, "pool"), (table, "table"), (ids, "ids")):
        _dev(t, nm)
        if not t.is_contiguous():
            raise ValueError(f"{nm} must be contiguous")
    if pool.dim() != 2 or table.dim() != 2 or table.dtype != torch.int32 or ids.dtype != torch.int32:
        raise ValueError("pool must be [n_pages, page_bytes]; table and ids int32")
    n_pages, page_bytes = pool.shape[0], pool.shape[1] * pool.element_size()
    n_chunks, ppc = table.shape
    count = ids.numel()
    if out is None:
        out = torch.empty((count, ppc, page_bytes), dtype=torch.uint8, device=pool.device)
    _dev(out, "out")
    if not out.is_contiguous() or out.numel() * out.element_size() != count * ppc * page_bytes:
        raise ValueError("out must be contiguous with count * ppc * page_bytes bytes")
    pg = MemPages(pool.data_ptr(), n_pages, page_bytes, table.data_ptr(), n_chunks, ppc)
    _check("mem_gather_chunks", lib().mem_gather_chunks(C.byref(pg), ids.data_ptr(), count, order, group,
                                                        out.data_ptr(), _stream(stream)))
    return out


def mem_gather_budget(pool: torch.Tensor, table: torch.Tensor, tok_len: torch.Tensor, ids: torch.Tensor,
                      budget_tokens: int, row_bytes: int, *, out=None, stream=None):
    """Budget-aware time-ordered token rows of rank-ordered ids [m, k]:
    (rows uint8 [m, budget_tokens, row_bytes], tokens int32 [m], kept ids int32 [m, k])."""
    for t, nm in ((pool, "pool"), (table, "table"), (tok_len, "tok_len"), (ids, "ids")):
        _dev(t, nm)
        if not t.is_contiguous():
            raise ValueError(f"{nm} must be contiguous")
    if (pool.dim() != 2 or table.dim() != 2 or ids.dim() != 2 or table.dtype != torch.int32
            or ids.dtype != torch.int32 or tok_len.dtype != torch.int32 or tok_len.shape != (table.shape[0],)):
        raise ValueError("pool [n_pages, page_bytes]; table int32 [n_chunks, ppc]; tok_len int32 [n_chunks]; "
                         "ids int32 [m, k]")
    n_pages, page_bytes = pool.shape[0], pool.shape[1] * pool.element_size()
    n_chunks, ppc = table.shape
    m, k = ids.shape
    if out is None:
        out = (torch.empty((m, budget_tokens, row_bytes), dtype=torch.uint8, device=pool.device),
               torch.empty((m,), dtype=torch.int32, device=pool.device),
               torch.empty((m, k), dtype=torch.int32, device=pool.device))
    rows, tokens, kept = out
    _dev(rows, "out rows")
    if not rows.is_contiguous() or rows.numel() * rows.element_size() != m * budget_tokens * row_bytes:
        raise ValueError("out rows must be contiguous with m * budget_tokens * row_bytes bytes")
    pg = MemPages(pool.data_ptr(), n_pages, page_bytes, table.data_ptr(), n_chunks, ppc)
    _check("mem_gather_budget", lib().mem_gather_budget(
        C.byref(pg), tok_len.data_ptr(), row_bytes, ids.data_ptr(), m, k, budget_tokens,
        rows.data_ptr() if rows.numel() else None, _dev(tokens, "out tokens").data_ptr(),
        None if kept is None else _dev(kept, "out ids").data_ptr(), _stream(stream)))
    return out


def mem_compact_workspace_bytes(next_free_page: int, pages_per_block: int, n_entries: int, ppc: int,
                                n_ns: int) -> int:
    return int(lib().mem_compact_workspace_bytes(next_free_page, pages_per_block, n_entries, ppc, n_ns))


def mem_compact_blocks(pool: torch.Tensor, table: torch.Tensor, offsets: torch.Tensor, chunks: torch.Tensor,
                       pages_per_block: int, theta: float, next_free_page: int, *, phi: torch.Tensor | None = None,
                       released: torch.Tensor | None = None, workspace: torch.Tensor | None = None, stream=None):
    """Compact blocks whose invalid ratio is >= theta (pool and table updated in place).

    ``offsets`` int32 [n_ns + 1] / ``chunks`` int32: per-namespace live chunk ids (CSR).
    Returns (dict of moved_pages, released_blocks, next_free_page; phi float [n_blocks]; released uint8 [n_blocks]).
    """
    for t, nm in ((pool, "pool"), (table, "table"), (offsets, "offsets"), (chunks, "chunks")):
        _dev(t, nm)
        if not t.is_contiguous():
            raise ValueError(f"{nm} must be contiguous")
    if table.dtype != torch.int32 or offsets.dtype != torch.int32 or chunks.dtype != torch.int32 or pool.dim() != 2:
        raise ValueError("pool [n_pages, page_bytes]; table, offsets and chunks int32")
    n_pages, page_bytes = pool.shape[0], pool.shape[1] * pool.element_size()
    n_chunks, ppc = table.shape
    n_ns, n_entries = offsets.shape[0] - 1, chunks.shape[0]
    n_blocks = (next_free_page + pages_per_block - 1) // pages_per_block
    if phi is None:
        phi = torch.empty(n_blocks, dtype=torch.float32, device=pool.device)
    if released is None:
        released = torch.empty(n_blocks, dtype=torch.uint8, device=pool.device)
    ws, ws_bytes = _workspace(mem_compact_workspace_bytes(next_free_page, pages_per_block, n_entries, ppc, n_ns),
                              pool.device, workspace)
    T = MemChunkTables(offsets.data_ptr(), chunks.data_ptr() if n_entries else None, n_ns, n_entries)
    res = MemCompactResult()
    _check("mem_compact_blocks", lib().mem_compact_blocks(
        pool.data_ptr(), n_pages, page_bytes, table.data_ptr(), n_chunks, ppc, C.byref(T), pages_per_block, theta,
        next_free_page, phi.data_ptr() if n_blocks else None, released.data_ptr() if n_blocks else None,
        C.byref(res), ws.data_ptr(), ws_bytes, _stream(stream)))
    return ({"moved_pages": res.moved_pages, "released_blocks": res.released_blocks,
             "next_free_page": res.next_free_page}, phi, released)


def mem_colocate_workspace_bytes(m: int, k: int, n_chunks: int) -> int:
    return int(lib().mem_colocate_workspace_bytes(m, k, n_chunks))


def mem_colocate(pool: torch.Tensor, table: torch.Tensor, ids: torch.Tensor, scores: torch.Tensor, tau: float,
                 min_group: int, next_free_page: int, *, workspace: torch.Tensor | None = None, stream=None) -> dict:
    """Relocate each key's chunks with score >= tau (groups of at least min_group) into fresh pages, in time
    order; pool and table updated in place.  Returns moved_chunks, groups and next_free_page."""
    for t, nm in ((pool, "pool"), (table, "table"), (ids, "ids"), (scores, "scores")):
        _dev(t, nm)
        if not t.is_contiguous():
            raise ValueError(f"{nm} must be contiguous")
    if (table.dtype != torch.int32 or ids.dtype != torch.int32 or scores.dtype != torch.float32
            or ids.dim() != 2 or scores.shape != ids.shape or pool.dim() != 2):
        raise ValueError("pool [n_pages, page_bytes]; table and ids int32; scores float32 shaped like ids")
    n_pages, page_bytes = pool.shape[0], pool.shape[1] * pool.element_size()
    n_chunks, ppc = table.shape
    m, k = ids.shape
    ws, ws_bytes = _workspace(mem_colocate_workspace_bytes(m, k, n_chunks), pool.device, workspace)
    res = MemColocateResult()
    _check("mem_colocate", lib().mem_colocate(pool.data_ptr(), n_pages, page_bytes, table.data_ptr(), n_chunks, ppc,
                                              ids.data_ptr(), scores.data_ptr(), m, k, tau, min_group,
                                              next_free_page, C.byref(res), ws.data_ptr(), ws_bytes,
                                              _stream(stream)))
    return {"moved_chunks": res.moved_chunks, "groups": res.groups, "next_free_page": res.next_free_page}


class BankState:
    """A bank tensor with spare capacity plus its page table and page allocator.

    ``emb``: [capacity, d] GPU tensor of which the first ``n`` rows are live;
    ``table``: int32 [capacity, ppc] GPU tensor; ``next_free_page``: host counter.
    """

    def __init__(self, emb: torch.Tensor, n: int, table: torch.Tensor, next_free_page: int, n_pages_cap: int):
        self.emb, self.n, self.table = emb, n, table
        self.next_free_page, self.n_pages_cap = next_free_page, n_pages_cap

    @property
    def live(self) -> torch.Tensor:
        return self.emb[: self.n]


def mem_append_chunks(state: BankState, new_emb: torch.Tensor, stream=None) -> BankState:
    """Insert new chunks: bank rows and page-table rows [n, n + m); advances n and the page counter."""
    cap, d, stride = _rows(state.emb, "bank")
    m, d2, new_stride = _rows(new_emb, "new_emb")
    if d2 != d or _dtype_code(new_emb) != _dtype_code(state.emb):
        raise ValueError("new_emb must match the bank's dtype and dimension")
    _dev(state.table, "table")
    if state.table.dtype != torch.int32 or not state.table.is_contiguous() or state.table.shape[0] < cap:
        raise ValueError("table must be a contiguous int32 [capacity, ppc] GPU tensor")
    b = MemBank(state.emb.data_ptr(), state.n, d, _dtype_code(state.emb), stride)
    nfp = C.c_int64(state.next_free_page)
    _check("mem_append_chunks", lib().mem_append_chunks(C.byref(b), cap, new_emb.data_ptr(), m, new_stride,
                                                        state.table.data_ptr(), state.table.shape[1], C.byref(nfp),
                                                        state.n_pages_cap, _stream(stream)))
    state.n, state.next_free_page = int(b.n), int(nfp.value)
    return state
