"""Seeded synthetic inputs shared by the GPU path's tests/benchmark and the oracle.

This module draws random numbers and lays out bytes; it holds none of the
method's arithmetic (no scoring, normalisation of scores, selection or copy).
Both sides consume exactly the bytes produced here.

Workloads (stand-ins for the agent traces of the paper's evaluation, whose
chunks carry text rather than embeddings):

* chunk embeddings are unit vectors in R^d, either i.i.d. Gaussian directions or
  a Gaussian mixture (centroids N(0, I_d), member = centroid + sigma * N(0, I_d),
  then L2-normalised), stored as fp32 or bf16;
* a query is a perturbed cluster member: raw(j) + 0.2 * N(0, I_d) for a
  uniformly drawn bank row j, L2-normalised;
* each chunk owns a block of ``pages_per_chunk`` fixed-size pages (the
  paper's separation of logical chunk identity from physical placement,
  Section 4.2); the page table places 80 % of each cluster's chunks in one
  contiguous run and scatters the other 20 % page by page;
* page contents are the SplitMix64 stream (Steele, Lea and Flood, OOPSLA 2014)
  keyed by a seeded 64-bit key and indexed by (chunk, page, word).

Random streams: ``numpy.random.Generator(PCG64(SeedSequence([seed, tag,
stream, sub])))``. Streams: 0 centroids, 1 cluster ids, 2 bank noise (sub =
4096-row block), 3 query source rows, 4 query noise / i.i.d. query draws,
5 page layout, 6 payload key, 7 appended-chunk cluster ids (sub = round+1),
8 appended-chunk noise (sub = round+1), 9 namespace ids, 10 tombstones,
11 token counts, 12 block live densities, 13 relocated chunks.

Conversion: fp64 draws -> fp32 (round to nearest even) -> bf16 (round to
nearest even on the fp32 bits); bf16 arrays are returned as their uint16 bit
patterns.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

BLOCK_ROWS = 4096
GOLDEN = np.uint64(0x9E3779B97F4A7C15)

# Workload tags: fixed integers mixed into every seed so that workloads never
# share random streams.
TAG_TINY = 1
TAG_RELATION = 2
TAG_BATCHED = 3
TAG_GATHER = 4
TAG_STREAM = 5


def rng(seed: int, tag: int, stream: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag, stream, sub])))


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


# ---------------------------------------------------------------- conversions

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _unit_rows(raw: np.ndarray) -> np.ndarray:
    return raw / np.linalg.norm(raw, axis=1, keepdims=True)


def _encode(unit64: np.ndarray, dtype: str) -> np.ndarray:
    f32 = unit64.astype(np.float32)
    if dtype == "f32":
        return f32
    if dtype == "bf16":
        return f32_to_bf16_bits(f32)
    raise ValueError(dtype)


# ---------------------------------------------------------------- embeddings

def iid_unit(seed: int, tag: int, stream: int, rows: int, d: int, dtype: str = "f32") -> np.ndarray:
    """i.i.d. N(0, I_d) rows, L2-normalised."""
    return _encode(_unit_rows(rng(seed, tag, stream).standard_normal((rows, d))), dtype)


@dataclass
class ClusteredBank:
    emb: np.ndarray                    # [n, d] float32 or uint16 (bf16 bits)
    cluster: np.ndarray                # [n] int64 cluster id per chunk
    centroids: np.ndarray              # [C, d] float64
    queries: np.ndarray | None = None  # [m, d], same encoding as emb
    query_src: np.ndarray | None = None  # [m] bank row each query perturbs
    dtype: str = "bf16"
    extra: dict = field(default_factory=dict)


def clustered_bank(seed: int, tag: int, n: int, d: int, n_clusters: int, sigma: float,
                   dtype: str = "bf16", m_queries: int = 0, query_sigma: float = 0.2,
                   threads: int | None = None) -> ClusteredBank:
    """Gaussian-mixture bank (uniform cluster weights) and optional perturbed queries.

    Bank noise is drawn per 4096-row block so every raw row is reproducible
    without drawing the whole bank; queries perturb the raw (pre-normalisation)
    member vector of their source row.
    """
    centroids = rng(seed, tag, 0).standard_normal((n_clusters, d))
    cluster = rng(seed, tag, 1).integers(0, n_clusters, size=n)
    out_dtype = np.float32 if dtype == "f32" else np.uint16
    emb = np.empty((n, d), dtype=out_dtype)
    src = None
    raw_q = None
    if m_queries:
        src = rng(seed, tag, 3).integers(0, n, size=m_queries)
        raw_q = np.empty((m_queries, d))

    def block(bi: int):
        r0 = bi * BLOCK_ROWS
        r1 = min(n, r0 + BLOCK_ROWS)
        raw = centroids[cluster[r0:r1]] + sigma * rng(seed, tag, 2, bi).standard_normal((r1 - r0, d))
        emb[r0:r1] = _encode(_unit_rows(raw), dtype)
        if src is not None:
            sel = np.nonzero((src >= r0) & (src < r1))[0]
            raw_q[sel] = raw[src[sel] - r0]

    nblocks = (n + BLOCK_ROWS - 1) // BLOCK_ROWS
    with ThreadPoolExecutor(threads or _threads()) as ex:
        list(ex.map(block, range(nblocks)))
    bank = ClusteredBank(emb=emb, cluster=cluster, centroids=centroids, dtype=dtype)
    if m_queries:
        noise = rng(seed, tag, 4).standard_normal((m_queries, d))
        bank.queries = _encode(_unit_rows(raw_q + query_sigma * noise), dtype)
        bank.query_src = src
    return bank


def appended_chunks(seed: int, tag: int, round_idx: int, m: int, centroids: np.ndarray,
                    sigma: float, dtype: str = "bf16") -> np.ndarray:
    """New chunks for one streaming round, drawn from the bank's mixture."""
    c = rng(seed, tag, 7, round_idx + 1).integers(0, centroids.shape[0], size=m)
    raw = centroids[c] + sigma * rng(seed, tag, 8, round_idx + 1).standard_normal((m, centroids.shape[1]))
    return _encode(_unit_rows(raw), dtype)


def namespaces(seed: int, tag: int, n: int, n_ns: int, dead_frac: float, run: int = 1,
               query_src: np.ndarray | None = None, m: int = 0) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(user, session) namespace id per bank row, a live flag per row and a
    namespace per query.

    Rows come in runs of one namespace (a session appends its chunks in a
    burst, and bursts of different sessions interleave): run lengths are
    geometric with mean `run` (run = 1: every row draws its own namespace),
    namespaces uniform over n_ns per run.  A dead_frac share of rows is
    tombstoned (old copies left by out-of-place updates).  A query takes the
    namespace of its source row when `query_src` is given, else a uniform
    one.  Returns (row_ns int32 [n], row_live uint8 [n], key_ns int32 [m])."""
    if run <= 1:
        row_ns = rng(seed, tag, 9).integers(0, n_ns, size=n).astype(np.int32)
    else:
        lengths = rng(seed, tag, 9, 2).geometric(1.0 / run, size=n)  # each >= 1, so they cover n rows
        starts = np.concatenate([[0], np.cumsum(lengths)])
        n_runs = int(np.searchsorted(starts, n, side="left"))
        ids = rng(seed, tag, 9).integers(0, n_ns, size=n_runs).astype(np.int32)
        row_ns = np.repeat(ids, lengths[:n_runs])[:n]
    row_live = (rng(seed, tag, 10).random(n) >= dead_frac).astype(np.uint8)
    if query_src is not None:
        key_ns = row_ns[np.asarray(query_src)].astype(np.int32)
    else:
        key_ns = rng(seed, tag, 9, 1).integers(0, n_ns, size=m).astype(np.int32)
    return row_ns, row_live, key_ns


def token_lengths(seed: int, tag: int, n: int, lo: int, hi: int) -> np.ndarray:
    """Tokens held by each chunk's block (a compacted memory is shorter than
    its block): uniform integers in [lo, hi], int32 [n]."""
    return rng(seed, tag, 11).integers(lo, hi + 1, size=n).astype(np.int32)


def compaction_layout(seed: int, tag: int, n_blocks: int, pages_per_block: int, ppc: int,
                      relocated_frac: float = 0.2, extra_pages: int = 0) -> tuple[np.ndarray, int]:
    """A pool after a history of out-of-place updates, for block compaction.

    Block b keeps a share u_b ~ uniform(0, 1) of its pages live (so about a
    quarter of the blocks have three quarters or more invalid); the live
    pages, taken in ascending order, are dealt to chunks ppc at a time in id
    order (append order), except that a relocated_frac share of chunks swap
    their pages with other chunks (copies written later elsewhere).
    Returns (table int32 [n_chunks, ppc], next_free = n_blocks * P +
    extra_pages); the extra pages are written but hold no live page."""
    P = pages_per_block
    u = rng(seed, tag, 12).random(n_blocks)
    g = rng(seed, tag, 12, 1)
    live = [b * P + np.sort(g.choice(P, int(u[b] * P), replace=False)) for b in range(n_blocks)]
    pages = np.concatenate(live) if live else np.zeros(0, np.int64)
    pages = pages[: (pages.shape[0] // ppc) * ppc]
    table = pages.reshape(-1, ppc).astype(np.int32)
    n_chunks = table.shape[0]
    moved = np.nonzero(rng(seed, tag, 13).random(n_chunks) < relocated_frac)[0]
    table[moved] = table[rng(seed, tag, 13, 1).permutation(moved)]
    return table, n_blocks * P + extra_pages


def chunk_tables(row_ns: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Per-namespace chunk tables T[u][s] as CSR: live chunk ids (row_ns >= 0)
    grouped by namespace, ascending within each.  Returns (offsets int32
    [n_ns + 1], chunks int32)."""
    row_ns = np.asarray(row_ns)
    live = np.nonzero(row_ns >= 0)[0]
    n_ns = int(row_ns.max()) + 1 if live.size else 0
    order = live[np.argsort(row_ns[live], kind="stable")]
    counts = np.bincount(row_ns[live], minlength=n_ns)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return offsets, order.astype(np.int32)


def scoped_row_ns(row_ns: np.ndarray, row_live: np.ndarray) -> np.ndarray:
    """The library's one-array encoding: the namespace of a live row, -1 for a
    tombstoned one."""
    return np.where(row_live != 0, row_ns, -1).astype(np.int32)


def integer_grid(seed: int, tag: int, rows: int, d: int, dtype: str = "bf16") -> np.ndarray:
    """Entries in {-1, 0, +1} * 2^-5: every product and partial sum of a
    length-d dot product (d <= 2^14) is exactly representable in fp32."""
    v = rng(seed, tag, 4, rows).integers(-1, 2, size=(rows, d)).astype(np.float64) / 32.0
    return _encode(v, dtype)


# ---------------------------------------------------------------- page layout

def page_layout(seed: int, tag: int, cluster: np.ndarray, pages_per_chunk: int = 2,
                run_fraction: float = 0.8) -> np.ndarray:
    """Page table int32 [n, pages_per_chunk] over physical pages [0, n * ppc).

    For each cluster a seeded floor(run_fraction * size) subset of its chunks
    forms one run (ascending chunk id, consecutive pages); every page of the
    remaining chunks is a unit of its own. All units are shuffled and laid
    out back to back.
    """
    n = cluster.shape[0]
    g = rng(seed, tag, 5)
    order = np.argsort(cluster, kind="stable")
    counts = np.bincount(cluster, minlength=int(cluster.max()) + 1 if n else 0)
    starts = np.concatenate([[0], np.cumsum(counts)])
    in_run = np.zeros(n, dtype=bool)
    run_members = []
    for c in range(counts.shape[0]):
        members = order[starts[c]:starts[c + 1]]
        take = int(np.floor(run_fraction * members.shape[0]))
        chosen = np.sort(g.permutation(members)[:take]) if take else members[:0]
        in_run[chosen] = True
        run_members.append(chosen)
    scattered = np.nonzero(~in_run)[0]
    # units: runs first (one per non-empty run), then (chunk, page) singles
    run_units = [r for r in run_members if r.shape[0]]
    n_units = len(run_units) + scattered.shape[0] * pages_per_chunk
    lengths = np.empty(n_units, dtype=np.int64)
    lengths[:len(run_units)] = [r.shape[0] * pages_per_chunk for r in run_units]
    lengths[len(run_units):] = 1
    perm = g.permutation(n_units)
    offsets = np.empty(n_units, dtype=np.int64)
    offsets[perm] = np.concatenate([[0], np.cumsum(lengths[perm])[:-1]])
    table = np.full((n, pages_per_chunk), -1, dtype=np.int64)
    for u, r in enumerate(run_units):
        base = offsets[u] + np.arange(r.shape[0])[:, None] * pages_per_chunk
        table[r] = base + np.arange(pages_per_chunk)[None, :]
    single = offsets[len(run_units):].reshape(scattered.shape[0], pages_per_chunk)
    table[scattered] = single
    assert (table >= 0).all()
    return table.astype(np.int32)


def identity_layout(n: int, pages_per_chunk: int = 2) -> np.ndarray:
    return np.arange(n * pages_per_chunk, dtype=np.int32).reshape(n, pages_per_chunk)


# ---------------------------------------------------------------- payload

def payload_key(seed: int, tag: int) -> int:
    return int(rng(seed, tag, 6).integers(0, 2**63 - 1, dtype=np.int64))


def splitmix64(key: int, counter: np.ndarray) -> np.ndarray:
    """SplitMix64 output number ``counter`` (0-based) of the stream seeded with ``key``."""
    with np.errstate(over="ignore"):
        z = np.uint64(key) + (counter.astype(np.uint64) + np.uint64(1)) * GOLDEN
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def payload_words(key: int, chunk: int, page: int, pages_per_chunk: int, page_bytes: int) -> np.ndarray:
    """The uint64 words of logical page ``page`` of chunk ``chunk``."""
    wpp = page_bytes // 8
    base = (np.int64(chunk) * pages_per_chunk + page) * wpp
    return splitmix64(key, base + np.arange(wpp, dtype=np.int64))


def host_pool(key: int, table: np.ndarray, page_bytes: int, n_pages: int | None = None) -> np.ndarray:
    """Small page pool on the host: physical page table[c, p] holds payload(c, p)."""
    n, ppc = table.shape
    n_pages = n * ppc if n_pages is None else n_pages
    pool = np.zeros((n_pages, page_bytes // 8), dtype=np.uint64)
    for c in range(n):
        for p in range(ppc):
            pool[table[c, p]] = payload_words(key, c, p, ppc, page_bytes)
    return pool.view(np.uint8).reshape(n_pages, page_bytes)


# ---------------------------------------------------------------- device fill

_fill_lib = None


def _inputs_lib():
    global _fill_lib
    import ctypes as C
    if _fill_lib is None:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmeminputs.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m paper_2607_05708_amd.build`")
        L = C.CDLL(path)
        L.meminputs_fill_payload.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_void_p, C.c_int64, C.c_int32,
                                             C.c_uint64, C.c_void_p]
        L.meminputs_fill_payload.restype = C.c_int
        L.meminputs_copy_probe.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]
        L.meminputs_copy_probe.restype = C.c_int
        L.meminputs_mfma_probe.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p]
        L.meminputs_mfma_probe.restype = C.c_int
        _fill_lib = L
    return _fill_lib


def fill_payload_device(pool, table, key: int, stream=None) -> None:
    """Fill a GPU page pool (torch uint8 [n_pages, page_bytes]) so that physical
    page table[c, p] holds payload(c, p); ``table`` is an int32 GPU tensor.
    Uses libmeminputs.so (SplitMix64 on the device); large pools are filled
    without a host round trip."""
    import ctypes as C

    import torch
    L = _inputs_lib()
    assert pool.is_cuda and table.is_cuda and table.dtype == torch.int32 and table.is_contiguous()
    s = (stream if stream is not None else torch.cuda.current_stream()).cuda_stream
    rc = L.meminputs_fill_payload(pool.data_ptr(), pool.shape[0], pool.shape[1] * pool.element_size(),
                                  table.data_ptr(), table.shape[0], table.shape[1], C.c_uint64(key), s)
    if rc != 0:
        raise RuntimeError(f"meminputs_fill_payload failed with {rc}")


def measured_peaks(torch, reps: int = 5) -> dict:
    """Rates this GPU sustains on two probe kernels of libmeminputs.so: a 4 GiB
    streaming device copy (HBM read + write bytes per second) and a
    register-only bf16 MFMA loop over every CU (FLOP/s).  Measurement only."""
    L = _inputs_lib()
    s = torch.cuda.current_stream().cuda_stream
    nbytes = 4 << 30
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    def copy():
        if L.meminputs_copy_probe(a.data_ptr(), b.data_ptr(), nbytes, s) != 0:
            raise RuntimeError("meminputs_copy_probe failed")
    t_copy = timed(copy)
    del a, b
    blocks, iters = 256 * 4, 4096
    out = torch.empty(blocks * 512, dtype=torch.float32, device="cuda")

    def mfma():
        if L.meminputs_mfma_probe(blocks, iters, out.data_ptr(), s) != 0:
            raise RuntimeError("meminputs_mfma_probe failed")
    t_mfma = timed(mfma)
    flops = blocks * 8 * iters * 8 * 2.0 * 32 * 32 * 16
    return {"hbm_copy_GBps": 2.0 * nbytes / t_copy / 1e9, "mfma_bf16_TFLOPs": flops / t_mfma / 1e12,
            "copy": "4 GiB device-to-device, 1,024-thread workgroups of 128 KiB, 4 x 16 B non-temporal loads in flight per lane",
            "mfma": "v_mfma_f32_32x32x16_bf16 on register operands, 8 waves per CU, 1024 workgroups"}
