"""The C ABI without a GPU: the library loads, exports what include/memattn.h
declares, and rejects bad arguments on the host before launching anything."""
import ctypes as C
import os
import re

import pytest

import paper_2607_05708_amd as pm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "memattn.h")
FAKE = 0x100000  # never dereferenced: every call below fails validation first

needs_lib = pytest.mark.skipif(not os.path.exists(pm.library_path()), reason="libmemattn.so not built")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"MEMATTN_API\s+[\w\s\*]+?\b(mem_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(["mem_workspace_bytes", "mem_retrieve_topk", "mem_build_relations",
                                           "mem_retrieve_topk_noalloc", "mem_scratch_bytes",
                                           "mem_retrieve_topk_scoped", "mem_build_relations_scoped",
                                           "mem_workspace_bytes_grouped", "mem_retrieve_topk_grouped",
                                           "mem_gather_chunks", "mem_gather_budget",
                                           "mem_compact_workspace_bytes", "mem_compact_blocks",
                                           "mem_colocate_workspace_bytes", "mem_colocate", "mem_append_chunks", "mem_status_string",
                                           "mem_last_error"])


@needs_lib
def test_library_exports_every_declared_symbol():
    L = C.CDLL(pm.library_path())
    for name in declared_functions():
        assert hasattr(L, name), name


@needs_lib
def test_status_strings():
    L = pm.lib()
    assert L.mem_status_string(0) == b"ok"
    assert L.mem_status_string(-1) == b"invalid argument"
    assert L.mem_status_string(-3) == b"workspace missing or too small"
    assert L.mem_status_string(7) == b"unknown status"


@needs_lib
def test_workspace_bytes():
    L = pm.lib()
    assert L.mem_workspace_bytes(16, 1024, 256, 8, pm.MEM_F32) > 0
    big = L.mem_workspace_bytes(1024, 1 << 20, 1024, 32, pm.MEM_BF16)
    assert 1024 * 32 * 8 <= big < 1 << 30
    assert L.mem_workspace_bytes(16, 1024, 256, 0, pm.MEM_F32) == 0
    assert L.mem_workspace_bytes(16, 1024, 256, 65, pm.MEM_F32) == 0
    assert L.mem_workspace_bytes(16, 0, 256, 8, pm.MEM_F32) == 0
    assert L.mem_workspace_bytes(16, 1024, 256, 8, 7) == 0
    assert L.mem_workspace_bytes(0, 1024, 256, 8, pm.MEM_F32) >= 0


def _bank(n=1024, d=256, dtype=pm.MEM_BF16, stride=None, emb=FAKE):
    return pm.MemBank(emb, n, d, dtype, d if stride is None else stride)


def _out(idx=FAKE):
    return pm.MemTopkOut(idx, None, None, None)


def _retrieve(bank, q=FAKE, m=16, q_stride=256, k=8, scale=1.0, out=None, ws=FAKE, ws_bytes=1 << 30):
    L = pm.lib()
    b = C.byref(bank) if bank is not None else None
    return L.mem_retrieve_topk(b, q, m, q_stride, k, scale, out or _out(), None, ws, ws_bytes, None)


@needs_lib
@pytest.mark.parametrize("case,expect", [
    ("null_bank", -1), ("null_emb", -1), ("bad_dtype", -1), ("d0", -1), ("d_big", -1), ("stride", -1),
    ("k0", -1), ("k65", -1), ("k_gt_n", -1), ("scale0", -1), ("scale_nan", -1), ("scale_inf", -1),
    ("null_q", -1), ("q_stride", -1), ("null_idx", -1), ("null_ws", -3), ("small_ws", -3), ("m_neg", -1),
])
def test_retrieve_validation(case, expect):
    L = pm.lib()
    args = {}
    bank = _bank()
    if case == "null_bank":
        bank = None
    elif case == "null_emb":
        bank = _bank(emb=None)
    elif case == "bad_dtype":
        bank = _bank(dtype=3)
    elif case == "d0":
        bank = _bank(d=0)
    elif case == "d_big":
        bank = _bank(d=8193, stride=8193)
    elif case == "stride":
        bank = _bank(stride=100)
    elif case == "k0":
        args["k"] = 0
    elif case == "k65":
        args["k"] = 65
    elif case == "k_gt_n":
        bank = _bank(n=4)
        args["k"] = 5
    elif case == "scale0":
        args["scale"] = 0.0
    elif case == "scale_nan":
        args["scale"] = float("nan")
    elif case == "scale_inf":
        args["scale"] = float("inf")
    elif case == "null_q":
        args["q"] = None
    elif case == "q_stride":
        args["q_stride"] = 255
    elif case == "null_idx":
        args["out"] = _out(idx=None)
    elif case == "null_ws":
        args["ws"] = None
    elif case == "small_ws":
        args["ws_bytes"] = 16
    elif case == "m_neg":
        args["m"] = -1
    assert _retrieve(bank, **args) == expect
    assert L.mem_last_error() != b""


def _retrieve_noalloc(bank, q=FAKE, m=16, q_stride=256, k=8, scale=1.0, out=None):
    L = pm.lib()
    b = C.byref(bank) if bank is not None else None
    return L.mem_retrieve_topk_noalloc(b, q, m, q_stride, k, scale, out or _out(), None, None)


@needs_lib
def test_noalloc_validates_like_the_workspace_call():
    # argument errors come back before the scratch array is looked up (no
    # device is touched here)
    L = pm.lib()
    assert _retrieve_noalloc(None) == -1
    assert _retrieve_noalloc(_bank(), k=0) == -1
    assert _retrieve_noalloc(_bank(), q=None) == -1
    assert _retrieve_noalloc(_bank(), out=_out(idx=None)) == -1
    assert _retrieve_noalloc(_bank(), scale=0.0) == -1
    assert _retrieve_noalloc(_bank(), m=0, q=None) == 0
    assert L.mem_scratch_bytes() == 128 << 20


@needs_lib
def test_noalloc_rejects_calls_beyond_the_scratch():
    # 4,096 queries against a 1,310,720-row bank need more workspace than the
    # scratch array holds: refused with a message naming the limit
    L = pm.lib()
    need = L.mem_workspace_bytes(4096, 1310720, 1024, 32, pm.MEM_BF16)
    assert need > L.mem_scratch_bytes()
    assert _retrieve_noalloc(_bank(n=1310720, d=1024), m=4096, q_stride=1024, k=32) == -3
    assert b"allocation-free" in L.mem_last_error()


@needs_lib
@pytest.mark.parametrize("dtype", [pm.MEM_BF16, pm.MEM_F32])
def test_scratch_holds_any_retrieval_of_up_to_1024_queries(dtype):
    # the header's promise: up to 1,024 queries fit at any bank size and k
    L = pm.lib()
    for m in (1, 16, 64, 65, 128, 129, 256, 257, 512, 1000, 1024):
        for n in (1024, 262144, 1 << 20, 1 << 24, (1 << 31) - 2):
            for k in (1, 8, 16, 32, 33, 64):
                assert 0 < L.mem_workspace_bytes(m, n, 1024, k, dtype) <= L.mem_scratch_bytes(), (m, n, k)


@needs_lib
def test_retrieve_m0_is_noop():
    assert _retrieve(_bank(), m=0, q=None, ws=None, ws_bytes=0) == 0


@needs_lib
def test_build_relations_validation():
    L = pm.lib()
    b = _bank(n=8, d=64, stride=64)
    # exclude_self leaves 7 candidates
    assert L.mem_build_relations(C.byref(b), 8, 1.0, 1, _out(), FAKE, 1 << 30, None) == -1
    assert L.mem_build_relations(C.byref(b), 8, 1.0, 1, _out(), FAKE, 16, None) == -1
    assert L.mem_build_relations(C.byref(b), 7, 1.0, 1, _out(), FAKE, 16, None) == -3


def _retrieve_scoped(bank, row_ns=FAKE, q=FAKE, query_ns=FAKE, m=16, k=8, ws_bytes=1 << 30):
    L = pm.lib()
    return L.mem_retrieve_topk_scoped(C.byref(bank), row_ns, q, query_ns, m, 256, k, 1.0, _out(), None, FAKE,
                                      ws_bytes, None)


@needs_lib
def test_scoped_validation():
    L = pm.lib()
    # namespaces are required and 4-byte aligned
    assert _retrieve_scoped(_bank(), row_ns=None) == -1
    assert _retrieve_scoped(_bank(), query_ns=None) == -1
    assert _retrieve_scoped(_bank(), row_ns=FAKE + 2) == -1
    assert _retrieve_scoped(_bank(), query_ns=FAKE + 1) == -1
    # the bank and k rules still apply ...
    assert _retrieve_scoped(_bank(d=0)) == -1
    assert _retrieve_scoped(_bank(), k=65) == -1
    # ... except k <= n: short rows are padded, so the request gets as far as the workspace check
    assert _retrieve_scoped(_bank(n=4), k=8, ws_bytes=16) == -3
    assert _retrieve_scoped(_bank(), m=0, q=None, query_ns=None) == 0
    b = _bank(n=8, d=64, stride=64)
    assert L.mem_build_relations_scoped(C.byref(b), None, 4, 1.0, 1, _out(), FAKE, 1 << 30, None) == -1
    assert L.mem_build_relations_scoped(C.byref(b), FAKE, 0, 1.0, 1, _out(), FAKE, 1 << 30, None) == -1
    assert L.mem_build_relations_scoped(C.byref(b), FAKE, 8, 1.0, 1, _out(), FAKE, 16, None) == -3
    assert L.mem_last_error() != b""


def _pages(pool=FAKE, n_pages=64, page_bytes=65536, table=FAKE, n_chunks=32, ppc=2):
    return pm.MemPages(pool, n_pages, page_bytes, table, n_chunks, ppc)


@needs_lib
def test_gather_validation():
    L = pm.lib()
    out = 0x7000_0000_0000
    g = lambda p, ids=FAKE, count=4, order=0, group=1, o=out: L.mem_gather_chunks(  # noqa: E731
        C.byref(p) if p is not None else None, ids, count, order, group, o, None)
    assert g(None) == -1
    assert g(_pages(page_bytes=100)) == -1
    assert g(_pages(ppc=0)) == -1
    assert g(_pages(ppc=65)) == -1
    assert g(_pages(), order=2) == -1
    assert g(_pages(), order=1, group=0) == -1
    assert g(_pages(), order=1, group=1025) == -1
    assert g(_pages(), count=-1) == -1
    assert g(_pages(), ids=None) == -1
    assert g(_pages(pool=FAKE + 8)) == -1                   # misaligned pool
    assert g(_pages(), o=FAKE + 65536) == -1                # out overlaps the pool
    assert g(_pages(), count=0, ids=None, o=None) == 0      # empty gather


@needs_lib
def test_gather_budget_validation():
    L = pm.lib()
    out, tok = 0x7000_0000_0000, 0x7100_0000_0000
    g = lambda p, tl=FAKE, rb=256, ids=FAKE, m=4, k=8, budget=1024, o=out, ot=tok: L.mem_gather_budget(  # noqa: E731
        C.byref(p) if p is not None else None, tl, rb, ids, m, k, budget, o, ot, None, None)
    assert g(None) == -1
    assert g(_pages(), rb=0) == -1
    assert g(_pages(), rb=24) == -1                          # not a multiple of 16
    assert g(_pages(page_bytes=65536), rb=48) == -1          # does not divide the page
    assert g(_pages(), k=0) == -1
    assert g(_pages(), k=65) == -1
    assert g(_pages(), m=-1) == -1
    assert g(_pages(), budget=-1) == -1
    assert g(_pages(), tl=None) == -1
    assert g(_pages(), ids=None) == -1
    assert g(_pages(), ot=None) == -1
    assert g(_pages(), o=None) == -1
    assert g(_pages(), o=FAKE + 4096) == -1                  # out overlaps the pool
    assert g(_pages(pool=FAKE + 8)) == -1                    # misaligned pool
    assert g(_pages(), m=0, ids=None, o=None, ot=None) == 0  # nothing to do
    assert L.mem_last_error() == b""


@needs_lib
def test_append_validation_leaves_counters():
    L = pm.lib()
    b = _bank(n=100, d=64, stride=64)
    nfp = C.c_int64(200)
    # capacity exceeded
    assert L.mem_append_chunks(C.byref(b), 101, FAKE, 2, 64, FAKE, 2, C.byref(nfp), 1000, None) == -1
    # page pool exhausted
    assert L.mem_append_chunks(C.byref(b), 1000, FAKE, 2, 64, FAKE, 2, C.byref(nfp), 203, None) == -1
    assert L.mem_append_chunks(C.byref(b), 1000, FAKE, 2, 64, FAKE, 0, C.byref(nfp), 1000, None) == -1
    assert L.mem_append_chunks(C.byref(b), 1000, None, 2, 64, FAKE, 2, C.byref(nfp), 1000, None) == -1
    assert L.mem_append_chunks(C.byref(b), 1000, FAKE, 2, 63, FAKE, 2, C.byref(nfp), 1000, None) == -1
    assert b.n == 100 and nfp.value == 200
    # m = 0 succeeds without touching the device
    assert L.mem_append_chunks(C.byref(b), 1000, None, 0, 64, FAKE, 2, C.byref(nfp), 1000, None) == 0
    assert b.n == 100 and nfp.value == 200


@needs_lib
def test_binding_rejects_host_tensors():
    import torch
    with pytest.raises(ValueError):
        pm.mem_retrieve_topk(torch.zeros(8, 32), torch.zeros(2, 32), 2)


@pytest.mark.parametrize("bad", ["idx_int64", "idx_short", "score_f64", "prob_shape", "lse_shape", "no_idx",
                                 "three"])
def test_topk_out_dtype_and_shape_are_checked(bad):
    # caller-supplied outputs are checked before any launch: an undersized or
    # wrongly typed buffer would otherwise be written past its end on the GPU
    import torch
    m, k = 6, 4
    out = [torch.empty((m, k), dtype=torch.int32), torch.empty((m, k)), torch.empty((m, k)), torch.empty((m,))]
    if bad == "idx_int64":
        out[0] = torch.empty((m, k), dtype=torch.int64)
    elif bad == "idx_short":
        out[0] = torch.empty((m, k - 1), dtype=torch.int32)
    elif bad == "score_f64":
        out[1] = torch.empty((m, k), dtype=torch.float64)
    elif bad == "prob_shape":
        out[2] = torch.empty((k, m))
    elif bad == "lse_shape":
        out[3] = torch.empty((m, 1))
    elif bad == "no_idx":
        out[0] = None
    else:
        out = out[:3]
    with pytest.raises(ValueError, match="out"):
        pm._topk_out(m, k, "cpu", tuple(out))
    # well-typed host tensors pass the dtype and shape checks and are then
    # refused for not being on the GPU
    good = (torch.empty((m, k), dtype=torch.int32), torch.empty((m, k)), None, torch.empty((m,)))
    with pytest.raises(ValueError, match="GPU"):
        pm._topk_out(m, k, "cpu", good)


@needs_lib
def test_compact_validation():
    L = pm.lib()
    T = pm.MemChunkTables(FAKE, FAKE, 4, 100)
    res = pm.MemCompactResult()
    c = lambda pool=FAKE, n_pages=1000, pb=65536, table=FAKE, n_chunks=50, ppc=2, t=T, P=64, theta=0.75, nf=800, \
        r=res, ws=FAKE, wsb=1 << 30: L.mem_compact_blocks(  # noqa: E731
            pool, n_pages, pb, table, n_chunks, ppc, C.byref(t) if t is not None else None, P, theta, nf, None, None,
            C.byref(r) if r is not None else None, ws, wsb, None)
    assert c(r=None) == -1
    assert c(t=None) == -1
    assert c(pool=None) == -1
    assert c(pool=FAKE + 8) == -1
    assert c(pb=100) == -1
    assert c(ppc=0) == -1
    assert c(ppc=65) == -1
    assert c(table=None) == -1
    assert c(nf=1001) == -1                     # frontier past the pool
    assert c(nf=-1) == -1
    assert c(P=0) == -1
    assert c(theta=float("nan")) == -1
    assert c(t=pm.MemChunkTables(None, FAKE, 4, 100)) == -1
    assert c(t=pm.MemChunkTables(FAKE, FAKE, 0, 100)) == -1
    assert c(ws=None) == -3
    assert c(wsb=16) == -3
    assert L.mem_compact_workspace_bytes(800, 64, 100, 2, 4) > 0
    assert L.mem_compact_workspace_bytes(800, 0, 100, 2, 4) == 0


@needs_lib
def test_colocate_validation():
    L = pm.lib()
    res = pm.MemColocateResult()
    c = lambda pool=FAKE, n_pages=1000, pb=65536, table=FAKE, n_chunks=50, ppc=2, ids=FAKE, sc=FAKE, m=8, k=5, \
        tau=0.7, mg=2, nf=100, r=res, ws=FAKE, wsb=1 << 30: L.mem_colocate(  # noqa: E731
            pool, n_pages, pb, table, n_chunks, ppc, ids, sc, m, k, tau, mg, nf,
            C.byref(r) if r is not None else None, ws, wsb, None)
    assert c(r=None) == -1
    assert c(pool=None) == -1
    assert c(pool=FAKE + 4) == -1
    assert c(pb=24) == -1
    assert c(ppc=0) == -1
    assert c(table=None) == -1
    assert c(nf=1001) == -1
    assert c(k=0) == -1
    assert c(k=65) == -1
    assert c(m=-1) == -1
    assert c(mg=0) == -1
    assert c(tau=float("inf")) == -1
    assert c(ids=None) == -1
    assert c(sc=None) == -1
    assert c(ws=None) == -3
    assert c(wsb=16) == -3
    assert L.mem_colocate_workspace_bytes(8, 5, 50) > 0
    assert L.mem_colocate_workspace_bytes(8, 0, 50) == 0


@needs_lib
def test_grouped_validation():
    L = pm.lib()
    T = pm.MemChunkTables(FAKE, FAKE, 4, 100)
    g = lambda bank=None, t=T, q=FAKE, qn=FAKE, m=16, qs=256, k=8, ws=FAKE, wsb=1 << 30: L.mem_retrieve_topk_grouped(  # noqa: E731
        C.byref(bank or _bank()), C.byref(t) if t is not None else None, q, qn, m, qs, k, 1.0, _out(), ws, wsb, None)
    assert g(t=None) == -1
    assert g(t=pm.MemChunkTables(None, FAKE, 4, 100)) == -1
    assert g(t=pm.MemChunkTables(FAKE, None, 4, 100)) == -1
    assert g(k=33) == -1                                     # the matrix-core path only
    assert g(qn=None) == -1
    assert g(qn=FAKE + 2) == -1
    assert g(bank=_bank(dtype=pm.MEM_F32)) == -2             # unsupported shapes point to the scoped call
    assert g(bank=_bank(d=64, stride=64), qs=64) == -2       # fewer than 3 k-blocks per tile
    assert g(bank=_bank(n=3 << 20, d=1024, stride=1024), qs=1024) == -2   # more than 4 GiB of rows
    assert g(wsb=16) == -3
    assert g(m=0, q=None, qn=None) == 0
    assert L.mem_workspace_bytes_grouped(16, 4, 100, 256, 8) > 0
    assert L.mem_workspace_bytes_grouped(16, 4, 100, 256, 33) == 0


@needs_lib
def test_workspace_size_never_decreases_with_the_bank():
    # a workspace sized for a bank also serves every smaller bank (streaming
    # appends size it once for the bank's capacity)
    L = pm.lib()
    # (more than 64 query tiles, from 16,385 queries on, allow more splits)
    for m in (1, 16, 65, 300, 1024, 4096, 16640, 40000, 100000):
        for d, k, dt in ((1024, 32, pm.MEM_BF16), (256, 8, pm.MEM_F32), (128, 64, pm.MEM_BF16)):
            prev = 0
            for n in list(range(1, 3000, 13)) + list(range(3000, 2_500_000, 9973)):
                w = L.mem_workspace_bytes(m, n, d, k, dt)
                assert w >= prev, (m, d, k, dt, n)
                prev = w
