"""GPU path vs the fp64 oracle at sizes the oracle finishes in seconds
(several tiles, ragged tails), plus exact and edge cases.  Calls go through
the C ABI (the ctypes binding)."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs
from parity import check_topk, decode

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def up(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_retrieve(bank, q, k, scale=1.0, full=False):
    b, qq = up(bank), up(q)
    fp = torch.empty((q.shape[0], bank.shape[0]), dtype=torch.float32, device="cuda") if full else None
    idx, score, prob, lse = pm.mem_retrieve_topk(b, qq, k, scale, full_prob=fp)
    torch.cuda.synchronize()
    out = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
           "lse": lse.cpu().numpy()}
    if full:
        out["full_prob"] = fp.cpu().numpy()
    return out


def test_tiny_retrieval_fp32_full_probabilities(dev):
    say("case: tiny retrieval fp32 n=1024 d=256 m=16 k=8 full_prob")
    bank = inputs.iid_unit(0, inputs.TAG_TINY, 2, 1024, 256, "f32")
    q = inputs.iid_unit(0, inputs.TAG_TINY, 4, 16, 256, "f32")
    g = run_retrieve(bank, q, 8, full=True)
    check_topk("tiny", q, bank, np.arange(16), g, 8, 1.0)
    ref = oracle.retrieve(q, bank, 8, full=True)
    assert np.allclose(g["full_prob"].sum(axis=1), 1.0, rtol=0, atol=1e-5)
    assert np.all(np.abs(g["full_prob"] - ref["full_prob"]) <= 1e-5 * ref["full_prob"] + 1e-12)


@pytest.mark.parametrize("k", [5, 16, 32])
@pytest.mark.parametrize("scale", [1.0, 20.0])
def test_bf16_clustered_matrix_core(dev, k, scale):
    say(f"case: bf16 clustered n=3000 d=256 m=300 k={k} scale={scale}")
    cb = inputs.clustered_bank(1, 60, 3000, 256, 16, 0.3, "bf16", m_queries=300)
    g = run_retrieve(cb.emb, cb.queries, k, scale)
    r = check_topk("bf16", cb.queries, cb.emb, np.arange(300), g, k, scale)
    assert r["exact_rows"] >= 0.95 * r["rows"]


@pytest.mark.parametrize("d", [64, 40])
def test_integer_grid_exact_with_ties(dev, d):
    say(f"case: integer grid exact d={d}")
    base = inputs.integer_grid(2, 61, 350, d)
    bank = np.concatenate([base, base])          # every row duplicated: exact ties
    q = inputs.integer_grid(3, 61, 70, d)
    g = run_retrieve(bank, q, 16, 2.0)
    check_topk("grid", q, bank, np.arange(70), g, 16, 2.0, exact=True)


@pytest.mark.parametrize("d,pad", [(160, 24), (32, 8), (96, 0)])
def test_strided_rows_odd_k_blocks(dev, d, pad):
    # rows padded to a wider row stride; d/32 odd or 1 k-blocks per tile
    say(f"case: strided rows d={d} pad={pad}")
    cb = inputs.clustered_bank(13, 65, 1300, d, 8, 0.3, "bf16", m_queries=270)
    wide_b = np.zeros((1300, d + pad), np.uint16)
    wide_b[:, :d] = cb.emb
    wide_q = np.zeros((270, d + 2 * pad), np.uint16)
    wide_q[:, :d] = cb.queries
    b, q = up(wide_b)[:, :d], up(wide_q)[:, :d]
    idx, score, prob, lse = pm.mem_retrieve_topk(b, q, 16, 2.0)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    check_topk(f"strided-{d}", cb.queries, cb.emb, np.arange(270), g, 16, 2.0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n", [1, 2, 3, 33])
def test_smallest_banks_every_candidate_selected(dev, dtype, n):
    # k equal to the number of candidates: retrieval takes all n rows, a
    # relation build (row itself excluded) all n - 1 others; every id must
    # appear once, in rank order, and the probabilities sum to 1
    say(f"case: smallest banks {dtype} n={n}, k = every candidate")
    bank = inputs.iid_unit(40 + n, 68, 0, n, 64, dtype)
    q = inputs.iid_unit(40 + n, 68, 4, 5, 64, dtype)
    g = run_retrieve(bank, q, n, 1.0)
    check_topk(f"all-n{n}", q, bank, np.arange(5), g, n, 1.0)
    assert np.all(np.sort(g["idx"], axis=1) == np.arange(n)[None, :])
    assert np.allclose(g["prob"].sum(axis=1), 1.0, rtol=0, atol=1e-5)
    if n >= 2:
        r = _relation(up(bank), n - 1, True)
        check_topk(f"all-rel-n{n}", bank, bank, np.arange(n), r, n - 1, 1.0, self_idx=np.arange(n))
        for i in range(n):
            assert sorted(r["idx"][i]) == [j for j in range(n) if j != i]
        assert np.allclose(r["prob"].sum(axis=1), 1.0, rtol=0, atol=1e-5)


def test_largest_dimension_and_row_stride(dev):
    # d = 8192, the largest dimension the boundary takes: on the matrix-core
    # path (256 k-blocks per tile) with bank rows at the largest stride it
    # takes, 65,536 elements, and on the VALU path (fp32, k = 64)
    d = 8192
    say("case: bf16 d=8192 bank row stride 65536, m=70 k=32 (matrix cores)")
    cb = inputs.clustered_bank(33, 65, 1100, d, 8, 0.3, "bf16", m_queries=70)
    wide_b = torch.zeros((1100, 65536), dtype=torch.int16, device="cuda")
    wide_b[:, :d] = torch.from_numpy(cb.emb.view(np.int16)).cuda()
    b = wide_b.view(torch.bfloat16)[:, :d]
    wide_q = np.zeros((70, d + 64), np.uint16)
    wide_q[:, :d] = cb.queries
    idx, score, prob, lse = pm.mem_retrieve_topk(b, up(wide_q)[:, :d], 32, 1.0)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    check_topk("d8192-stride65536", cb.queries, cb.emb, np.arange(70), g, 32, 1.0)
    del wide_b, b
    say("case: f32 d=8192, m=5 k=64 (VALU path)")
    bank = inputs.iid_unit(33, 66, 0, 700, d, "f32")
    q = inputs.iid_unit(33, 66, 4, 5, d, "f32")
    g = run_retrieve(bank, q, 64, 1.0)
    check_topk("d8192-f32", q, bank, np.arange(5), g, 64, 1.0)


@pytest.mark.parametrize("m", [64, 65, 128, 129])
def test_workgroup_shape_boundaries(dev, m):
    # 64 queries use the 64 x 512-row tile, 65..128 the 128 x 256 tile,
    # more the 256 x 256 tile: check each side of both boundaries
    say(f"case: shape boundary m={m} n=5000 d=128 k=16")
    cb = inputs.clustered_bank(15, 67, 5000, 128, 32, 0.3, "bf16", m_queries=m)
    g = run_retrieve(cb.emb, cb.queries, 16, 1.0)
    check_topk(f"shape-m{m}", cb.queries, cb.emb, np.arange(m), g, 16, 1.0)


def test_few_queries_many_partials(dev):
    # 16 queries against 262,144 rows: 256 bank splits x 2 halves = 512 partial
    # lists per query, merged in one wave with more than 64 KiB of LDS
    say("case: m=16 n=262144 d=256 k=32 (512 partials per query)")
    cb = inputs.clustered_bank(14, 66, 262144, 256, 512, 0.3, "bf16", m_queries=16)
    g = run_retrieve(cb.emb, cb.queries, 32, 1.0)
    check_topk("m16-512parts", cb.queries, cb.emb, np.arange(16), g, 32, 1.0)


@pytest.mark.parametrize("m", [1, 2])
def test_generic_merge_many_long_lists(dev, m):
    # fp32, k = 64: 586 (m = 1) or 391 (m = 2) partial lists of 64 keys per
    # query do not fit the LDS of the list-head merges, so the one-workgroup
    # merge inserts them 256 keys at a time
    say(f"case: VALU path f32 n=300000 d=32 m={m} k=64, workgroup merge")
    bank = inputs.iid_unit(32, 64, 0, 300000, 32, "f32")
    q = inputs.iid_unit(32, 64, 4, m, 32, "f32")
    g = run_retrieve(bank, q, 64, 2.0)
    check_topk(f"generic-merge-m{m}", q, bank, np.arange(m), g, 64, 2.0)


@pytest.mark.parametrize("k", [8, 16])
def test_sample_share_by_list_length(dev, k):
    # 98,304 rows, 1,024 queries: a 4,096-row sample is 1/24 of the bank, so
    # k = 16 takes the threshold sample and k = 8 (lists of 8) goes without
    say(f"case: bf16 n=98304 d=128 m=1024 k={k}, sample by list length")
    cb = inputs.clustered_bank(15, 67, 98304, 128, 256, 0.3, "bf16", m_queries=1024)
    g = run_retrieve(cb.emb, cb.queries, k, 1.0)
    rows = np.unique(np.concatenate([np.random.default_rng(16).choice(1024, 96, replace=False), [0, 1023]]))
    r = check_topk(f"share-k{k}", cb.queries, cb.emb, rows, {key: v[rows] for key, v in g.items()}, k, 1.0)
    assert r["exact_rows"] >= 0.95 * r["rows"]


@pytest.mark.parametrize("seed", [1, 2])
def test_seed_reruns(dev, seed):
    # the parity reruns at master seeds 1 and 2: a batched retrieval (65,536 x
    # 1024, 512 queries, k = 16) and a relation build (8,192 x 768, k = 32)
    say(f"case: seed {seed} reruns, batched 65536x1024 m=512 k=16 and relation 8192x768 k=32")
    cb = inputs.clustered_bank(seed, inputs.TAG_BATCHED, 65536, 1024, 256, 0.3, "bf16", m_queries=512)
    g = run_retrieve(cb.emb, cb.queries, 16, 1.0)
    rows = np.unique(np.concatenate([np.random.default_rng(seed).choice(512, 48, replace=False), [0, 511]]))
    check_topk(f"seed{seed}-batched", cb.queries, cb.emb, rows, {key: v[rows] for key, v in g.items()}, 16, 1.0)
    rb = inputs.clustered_bank(seed, inputs.TAG_RELATION, 8192, 768, 64, 0.3, "bf16")
    idx, score, prob, lse = pm.mem_build_relations(up(rb.emb), 32, 1.0, True)
    torch.cuda.synchronize()
    gr = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    rows = np.unique(np.concatenate([np.random.default_rng(seed + 10).choice(8192, 48, replace=False), [0, 8191]]))
    check_topk(f"seed{seed}-relation", rb.emb, rb.emb, rows, {key: v[rows] for key, v in gr.items()}, 32, 1.0,
               self_idx=np.arange(8192))


def test_relation_build_bf16(dev):
    say("case: relation build bf16 n=1500 d=128 k=32 exclude_self")
    cb = inputs.clustered_bank(4, 62, 1500, 128, 8, 0.3, "bf16")
    idx, score, prob, lse = pm.mem_build_relations(up(cb.emb), 32, 1.0, True)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    check_topk("rel-bf16", cb.emb, cb.emb, np.arange(1500), g, 32, 1.0, self_idx=np.arange(1500))


@pytest.mark.parametrize("n", [50, 100, 700])
def test_relation_build_small_banks(dev, n):
    # n <= 64 and <= 128 use the narrow workgroup shapes (one ragged tile,
    # own row masked); 700 the main shape
    say(f"case: relation build bf16 n={n} d=96 k=8 exclude_self")
    cb = inputs.clustered_bank(16, 68, n, 96, 4, 0.3, "bf16")
    idx, score, prob, lse = pm.mem_build_relations(up(cb.emb), 8, 20.0, True)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    check_topk(f"rel-small-{n}", cb.emb, cb.emb, np.arange(n), g, 8, 20.0, self_idx=np.arange(n))


def test_relation_build_fp32_and_keep_self(dev):
    say("case: relation build fp32 n=500 d=64 k=10")
    bank = inputs.iid_unit(5, 63, 0, 500, 64, "f32")
    for excl in (True, False):
        idx, score, prob, lse = pm.mem_build_relations(up(bank), 10, 3.0, excl)
        torch.cuda.synchronize()
        g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
             "lse": lse.cpu().numpy()}
        check_topk(f"rel-f32-{excl}", bank, bank, np.arange(500), g, 10, 3.0,
                   self_idx=np.arange(500) if excl else None)
        if not excl:
            assert np.array_equal(g["idx"][:, 0], np.arange(500))   # unit rows: self is the best match


@pytest.mark.parametrize("case", ["k1", "k_eq_n", "n1", "m1", "k64_bf16", "d32", "small_n_ragged"])
def test_edge_cases(dev, case):
    say(f"case: edge {case}")
    if case == "k1":
        bank, q, k = inputs.clustered_bank(6, 64, 700, 96, 4, 0.3, "bf16").emb, inputs.iid_unit(6, 64, 4, 33, 96, "bf16"), 1
    elif case == "k_eq_n":
        bank, q, k = inputs.iid_unit(7, 64, 0, 40, 48, "f32"), inputs.iid_unit(7, 64, 4, 5, 48, "f32"), 40
    elif case == "n1":
        bank, q, k = inputs.iid_unit(8, 64, 0, 1, 32, "bf16"), inputs.iid_unit(8, 64, 4, 3, 32, "bf16"), 1
    elif case == "m1":
        bank, q, k = inputs.iid_unit(9, 64, 0, 777, 64, "bf16"), inputs.iid_unit(9, 64, 4, 1, 64, "bf16"), 7
    elif case == "k64_bf16":
        bank, q, k = inputs.iid_unit(10, 64, 0, 900, 64, "bf16"), inputs.iid_unit(10, 64, 4, 20, 64, "bf16"), 64
    elif case == "d32":
        bank, q, k = inputs.iid_unit(11, 64, 0, 513, 32, "bf16"), inputs.iid_unit(11, 64, 4, 257, 32, "bf16"), 8
    else:
        bank, q, k = inputs.iid_unit(12, 64, 0, 100, 64, "bf16"), inputs.iid_unit(12, 64, 4, 9, 64, "bf16"), 12
    g = run_retrieve(bank, q, k, 1.5)
    check_topk(case, q, bank, np.arange(q.shape[0]), g, k, 1.5)


@pytest.mark.parametrize("dtype,n,k", [("f32", 6000, 10), ("bf16", 5000, 48), ("f32", 4096, 12), ("f32", 4097, 12)])
def test_valu_path_many_splits(dev, dtype, n, k):
    # the VALU path on banks of 16 to 24 splits of 256 rows (fp32, and bf16
    # with k above the matrix-core limit), full probabilities for fp32
    say(f"case: VALU path {dtype} n={n} d=64 m=20 k={k}")
    bank = inputs.iid_unit(30, 64, 0, n, 64, dtype)
    q = inputs.iid_unit(30, 64, 4, 20, 64, dtype)
    g = run_retrieve(bank, q, k, 2.0, full=(dtype == "f32"))
    check_topk(f"valu-{dtype}-{n}", q, bank, np.arange(20), g, k, 2.0)
    if dtype == "f32":
        ref = oracle.retrieve(q, bank, k, scale=2.0, full=True)
        assert np.all(np.abs(g["full_prob"] - ref["full_prob"]) <= 1e-5 * ref["full_prob"] + 1e-12)


@pytest.mark.parametrize("n", [4096, 4097, 8192])
def test_rank_merge_full_probabilities(dev, n):
    # 300 queries split the bank 4 ways, so the rank merge combines them; it
    # writes the full probability rows itself up to 4,096 rows, and
    # full_prob_kernel does after it for larger banks
    say(f"case: rank merge with full probabilities, f32 n={n} d=64 m=300 k=8")
    bank = inputs.iid_unit(31, 64, 0, n, 64, "f32")
    q = inputs.iid_unit(31, 64, 4, 300, 64, "f32")
    g = run_retrieve(bank, q, 8, 3.0, full=True)
    check_topk(f"rank-full-{n}", q, bank, np.arange(300), g, 8, 3.0)
    ref = oracle.retrieve(q, bank, 8, scale=3.0, full=True)
    assert np.all(np.abs(g["full_prob"] - ref["full_prob"]) <= 1e-5 * ref["full_prob"] + 1e-12)


def test_deterministic_repeat(dev):
    say("case: determinism")
    cb = inputs.clustered_bank(13, 65, 2000, 128, 8, 0.3, "bf16", m_queries=260)
    a = run_retrieve(cb.emb, cb.queries, 16)
    b = run_retrieve(cb.emb, cb.queries, 16)
    for key in a:
        assert np.array_equal(a[key], b[key]), key


# ------------------------------------------------------------------ gather

def _small_pool(seed, n=200, ppc=2, page_bytes=1024):
    cl = np.random.default_rng(seed).integers(0, 7, size=n)
    table = inputs.page_layout(seed, 66, cl, ppc)
    key = inputs.payload_key(seed, 66)
    return table, key, inputs.host_pool(key, table, page_bytes)


@pytest.mark.parametrize("order,group", [(0, 1), (1, 4), (1, 32), (1, 7)])
def test_gather_host_pool_bit_exact(dev, order, group):
    say(f"case: gather host pool order={order} group={group}")
    table, key, pool = _small_pool(14)
    rng = np.random.default_rng(15)
    ids = rng.integers(0, 200, size=61).astype(np.int32)
    ids[[3, 17, 40]] = -1
    ids[5] = ids[6]
    out = pm.mem_gather_chunks(up(pool), up(table), up(ids), order, group)
    torch.cuda.synchronize()
    ref = oracle.gather(pool, table, ids, order=order, group=group)
    assert np.array_equal(out.cpu().numpy(), ref)


@pytest.mark.parametrize("ppc,page_bytes", [(1, 1024), (3, 80000), (1, 65536)])
@pytest.mark.parametrize("order,group", [(0, 1), (1, 7)])
def test_gather_units_across_slots_and_groups(dev, ppc, page_bytes, order, group):
    # a workgroup copies two output pages: with 1 or 3 pages per chunk they
    # can belong to different slots and, in time order, different groups; an
    # odd page count leaves the last workgroup one page; 80,000-byte pages
    # end inside a round of loads
    say(f"case: gather ppc={ppc} page={page_bytes} order={order} group={group}")
    table, key, pool = _small_pool(18, n=120, ppc=ppc, page_bytes=page_bytes)
    rng = np.random.default_rng(19)
    ids = rng.integers(0, 120, size=61).astype(np.int32)
    ids[[2, 30]] = -1
    out = pm.mem_gather_chunks(up(pool), up(table), up(ids), order, group)
    torch.cuda.synchronize()
    ref = oracle.gather(pool, table, ids, order=order, group=group)
    assert np.array_equal(out.cpu().numpy(), ref)


def test_gather_device_filled_pool(dev):
    say("case: gather device-filled pool n=5000 ppc=2 page=4096")
    n, ppc, pb = 5000, 2, 4096
    cl = np.random.default_rng(16).integers(0, 50, size=n)
    table = inputs.page_layout(16, 67, cl, ppc)
    key = inputs.payload_key(16, 67)
    pool = torch.empty((n * ppc, pb), dtype=torch.uint8, device="cuda")
    tdev = up(table)
    inputs.fill_payload_device(pool, tdev, key)
    ids = np.random.default_rng(17).integers(0, n, size=32 * 40).astype(np.int32)
    out = pm.mem_gather_chunks(pool, tdev, up(ids), pm.MEM_ORDER_TIME, 32)
    torch.cuda.synchronize()
    exp = oracle.expected_blocks(key, ids, oracle.ORDER_TIME, 32, ppc, pb)
    assert np.array_equal(out.cpu().numpy().view(np.uint64).reshape(exp.shape), exp)
    # the device fill agrees with the host generator page by page
    hp = inputs.host_pool(key, table[:50], pb, n_pages=n * ppc)
    got = pool.cpu().numpy()
    for c in range(50):
        for p in range(ppc):
            assert np.array_equal(got[table[c, p]], hp[table[c, p]])


def test_append_then_retrieve(dev):
    say("case: append 64 rows then retrieve")
    cb = inputs.clustered_bank(18, 68, 564, 128, 8, 0.3, "bf16")
    cap, ppc = 700, 2
    emb = torch.zeros((cap, 128), dtype=torch.bfloat16, device="cuda")
    emb[:500] = up(cb.emb[:500])
    table = torch.full((cap, ppc), -7, dtype=torch.int32, device="cuda")
    table[:500] = up(inputs.identity_layout(500, ppc))
    st = pm.BankState(emb, 500, table, 1000, 5000)
    pm.mem_append_chunks(st, up(cb.emb[500:564]))
    assert st.n == 564 and st.next_free_page == 1000 + 64 * ppc
    torch.cuda.synchronize()
    assert np.array_equal(table[500:564].cpu().numpy(), oracle.append_table(64, ppc, 1000))
    assert np.all(table[564:].cpu().numpy() == -7)
    assert np.array_equal(emb[:564].view(torch.int16).cpu().numpy().view(np.uint16), cb.emb)
    q = inputs.iid_unit(19, 68, 4, 40, 128, "bf16")
    g = run_retrieve(cb.emb, q, 8)
    idx, score, prob, lse = pm.mem_retrieve_topk(st.live, up(q), 8)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), g["idx"])
    check_topk("append", q, cb.emb, np.arange(40), g, 8, 1.0)


# ------------------------------------------------------------------ threshold-sample path

def test_sampled_threshold_retrieval(dev):
    """m = 2000 queries (8 query tiles) against 70,000 rows: 31 splits of 9
    tiles, the first tile of each sampled, so the full pass starts from a
    sampled lower bound (ragged bank and query tails)."""
    say("case: sampled-threshold retrieval n=70000 d=128 m=2000 k=32")
    cb = inputs.clustered_bank(20, 69, 70000, 128, 64, 0.3, "bf16", m_queries=2000)
    g = run_retrieve(cb.emb, cb.queries, 32)
    rows = np.random.default_rng(21).choice(2000, 160, replace=False)
    rows = np.unique(np.concatenate([rows, [0, 1999, 1791, 1792]]))
    sub = {key: (val[rows] if val.ndim == 2 else val[rows]) for key, val in g.items()}
    check_topk("sampled", cb.queries, cb.emb, rows, sub, 32, 1.0)


def test_relation_build_long_splits_ties(dev):
    """Relation build over 33,000 rows (two splits of 65 tiles) with exact
    duplicate rows: ties resolve to the lowest ids across tiles and splits."""
    say("case: relation build with duplicates n=33000 d=64 k=16")
    base = inputs.integer_grid(22, 70, 16500, 64)
    bank = np.concatenate([base, base])
    idx, score, prob, lse = pm.mem_build_relations(up(bank), 16, 2.0, True)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    rows = np.unique(np.concatenate([np.random.default_rng(23).choice(33000, 60, replace=False), [0, 32999]]))
    sub = {key: val[rows] for key, val in g.items()}
    check_topk("rel-ties", bank, bank, rows, sub, 16, 2.0, self_idx=np.arange(33000), exact=True)


def test_sampled_threshold_exact_ties(dev):
    """Sampled-bound path (31 splits of 9 tiles) on exactly representable
    scores with every bank row duplicated: ties at the bound keep the lowest ids."""
    say("case: sampled-threshold retrieval with duplicates n=70000 d=64 m=2000 k=16")
    base = inputs.integer_grid(24, 71, 35000, 64)
    bank = np.concatenate([base, base])
    q = inputs.integer_grid(25, 71, 2000, 64)
    g = run_retrieve(bank, q, 16, 2.0)
    rows = np.unique(np.concatenate([np.random.default_rng(26).choice(2000, 60, replace=False), [0, 1999]]))
    check_topk("sampled-ties", q, bank, rows, {key: val[rows] for key, val in g.items()}, 16, 2.0, exact=True)


@pytest.mark.parametrize("k,n", [(32, 65536), (16, 65536 + 300), (8, 64000)])
def test_two_launch_splits(dev, k, n):
    # 8,192 queries (32 query tiles of 256) split the bank 8 ways; with
    # 65,536 rows a split spans 32 tiles, so the full pass runs in two
    # launches (first quarter of every split, then the rest bounded by the
    # k-th best over those quarters; a ragged last tile with n = 65,836).
    # With 64,000 rows (k = 8) a split spans 32 tiles too but lists of 8 take
    # no threshold sample, so the pass runs in one launch: the same checks
    # cover both plans.
    m = 8192
    say(f"case: two-launch splits k={k} n={n} m={m}")
    cb = inputs.clustered_bank(4, 91, n, 256, 64, 0.3, "bf16", m_queries=m)
    g = run_retrieve(cb.emb, cb.queries, k)
    starts = np.arange(0, m, 256)
    rows = np.unique(np.concatenate([np.random.default_rng(k).choice(m, 64, replace=False), starts, starts + 255]))
    sub = {key: v[rows] for key, v in g.items()}
    r = check_topk(f"two-launch-{k}", cb.queries, cb.emb, rows, sub, k, 1.0)
    say(f"  bit-exact top-k sets {r['exact_rows']}/{r['rows']}, max |lse - lse_ref| {r['lse_err_max']:.3g}")


def test_two_launch_relation_build_exact_ties(dev):
    # integer-grid rows, every row present twice (exact ties, within and
    # across the two launches): 32,768 rows as keys split the bank 2 ways of
    # 64 tiles, so the pass runs in two launches; ids and scores bit-exact
    n = 32768
    say(f"case: two-launch relation build, integer grid, n={n}")
    b = inputs.integer_grid(8, 91, n, 64)
    b = np.concatenate([b[: n // 2], b[: n // 2]])   # every row twice: ties resolve to the lower id
    idx, score, prob, lse = pm.mem_build_relations(up(b), 32, 1.0, True)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    rows = np.unique(np.concatenate([np.random.default_rng(9).choice(n, 40, replace=False), [0, 255, 256, n - 1]]))
    sub = {key: v[rows] for key, v in g.items()}
    check_topk("two-launch-relation-exact", b, b, rows, sub, 32, 1.0, self_idx=np.arange(n), exact=True)


# A relation build over enough rows to take a threshold sample runs its full
# pass with the queries in clustered order (grouped by the label of their
# best sampled row).  A ragged 32,845-row clustered bank takes that path.
def _clustered_relation_bank():
    return inputs.clustered_bank(8, 92, 32768 + 77, 256, 256, 0.3, "bf16").emb


def _relation(b, k, exclude_self):
    idx, score, prob, lse = pm.mem_build_relations(b, k, 1.0, exclude_self)
    torch.cuda.synchronize()
    return {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
            "lse": lse.cpu().numpy()}


def test_clustered_order_changes_no_result(dev):
    # with the row itself kept, a relation build is the retrieval of every
    # row against the bank; the retrieval of a copy of the rows runs them in
    # their own order, so the two must agree bit for bit
    b = _clustered_relation_bank()
    n = b.shape[0]
    say(f"case: clustered-order relation build (self kept) vs retrieval of a copy, n={n}, d=256, k=32")
    bt = up(b)
    rel = _relation(bt, 32, False)
    idx, score, prob, lse = pm.mem_retrieve_topk(bt, bt.clone(), 32, 1.0)
    torch.cuda.synchronize()
    ret = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
           "lse": lse.cpu().numpy()}
    for key in rel:
        np.testing.assert_array_equal(rel[key], ret[key], err_msg=key)


def test_clustered_order_relation_build(dev):
    b = _clustered_relation_bank()
    n = b.shape[0]
    say(f"case: clustered-order relation build (self excluded), n={n}, d=256, k=32, two calls")
    bt = up(b)
    g = _relation(bt, 32, True)
    again = _relation(bt, 32, True)
    for key in g:
        np.testing.assert_array_equal(g[key], again[key], err_msg=key)
    # the first and last query of every 256-query tile and 64 more
    ends = np.concatenate([np.arange(0, n, 256), np.minimum(np.arange(255, n + 255, 256), n - 1)])
    rows = np.unique(np.concatenate([ends, np.random.default_rng(10).choice(n, 64, replace=False)]))
    sub = {key: v[rows] for key, v in g.items()}
    r = check_topk("clustered-order-relation", b, b, rows, sub, 32, 1.0, self_idx=np.arange(n))
    say(f"  rows {r['rows']}, bit-exact top-k sets {r['exact_rows']}/{r['rows']}, "
        f"max |lse - lse_ref| {r['lse_err_max']:.3g}")
