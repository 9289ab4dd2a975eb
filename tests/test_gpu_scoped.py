"""Namespace-scoped, tombstone-aware selection on the GPU vs the fp64 oracle
(oracle.retrieve_scoped): candidates of key i are the live bank rows of its
(user, session) namespace.  The library takes one int32 array per bank row
(namespace, or -1 for a tombstoned row); the oracle takes namespace and live
flag separately, so the encoding is checked too.  Calls go through the C ABI."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs
from parity import check_topk_scoped

pytestmark = pytest.mark.gpu

TAG_SCOPED = 80


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


def host(out, full=None):
    torch.cuda.synchronize()
    idx, score, prob, lse = out
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(), "lse": lse.cpu().numpy()}
    if full is not None:
        g["full_prob"] = full.cpu().numpy()
    return g


def run_scoped(bank, q, row_ns, row_live, key_ns, k, scale=1.0, full=False):
    fp = torch.empty((q.shape[0], bank.shape[0]), dtype=torch.float32, device="cuda") if full else None
    out = pm.mem_retrieve_topk_scoped(up(bank), up(inputs.scoped_row_ns(row_ns, row_live)), up(q),
                                      up(np.asarray(key_ns, np.int32)), k, scale, full_prob=fp)
    return host(out, fp)


@pytest.mark.parametrize("m", [50, 100, 300])
@pytest.mark.parametrize("run", [1, 40])
def test_scoped_matrix_core(dev, m, run):
    # m = 50, 100, 300 take the three workgroup shapes; run = 1 gives every
    # half block of 16 rows mixed namespaces, run = 40 long same-namespace runs
    say(f"case: scoped bf16 n=3000 d=256 m={m} k=16 run={run}")
    cb = inputs.clustered_bank(30, TAG_SCOPED, 3000, 256, 16, 0.3, "bf16", m_queries=m)
    rns, live, kns = inputs.namespaces(30, TAG_SCOPED, 3000, 6, 0.2, run=run, query_src=cb.query_src)
    g = run_scoped(cb.emb, cb.queries, rns, live, kns, 16, 2.0)
    r = check_topk_scoped(f"scoped-m{m}-run{run}", cb.queries, cb.emb, np.arange(m), g, 16, 2.0, rns, live, kns)
    assert r["exact_rows"] >= 0.9 * r["rows"]


def test_scoped_short_and_empty_namespaces(dev):
    # 400 namespaces over 2000 rows (about 4.5 live rows each, k = 8), plus
    # queries with no namespace (-1) and with a namespace no row has:
    # short rows are padded, empty ones have lse = -inf
    say("case: scoped short namespaces n=2000 d=128 m=260 k=8")
    cb = inputs.clustered_bank(31, TAG_SCOPED, 2000, 128, 8, 0.3, "bf16", m_queries=260)
    rns, live, kns = inputs.namespaces(31, TAG_SCOPED, 2000, 400, 0.1, query_src=cb.query_src)
    kns = kns.copy()
    kns[::13] = -1
    kns[5::17] = 10_000
    g = run_scoped(cb.emb, cb.queries, rns, live, kns, 8, 1.0)
    check_topk_scoped("scoped-short", cb.queries, cb.emb, np.arange(260), g, 8, 1.0, rns, live, kns)
    assert np.any(g["idx"] == -1) and np.any(g["lse"] == -np.inf)


def test_scoped_k_above_bank_size(dev):
    # k may exceed n in a scoped call: every row is padded
    say("case: scoped k=32 > n=20")
    bank = inputs.iid_unit(32, TAG_SCOPED, 0, 20, 64, "bf16")
    q = inputs.iid_unit(32, TAG_SCOPED, 4, 10, 64, "bf16")
    rns, live, kns = inputs.namespaces(32, TAG_SCOPED, 20, 2, 0.25, m=10)
    g = run_scoped(bank, q, rns, live, kns, 32, 1.0)
    check_topk_scoped("scoped-k-gt-n", q, bank, np.arange(10), g, 32, 1.0, rns, live, kns)


@pytest.mark.parametrize("n,m", [(40000, 16), (600, 16), (6000, 300)])
def test_scoped_padding_in_every_merge(dev, n, m):
    # about 9 live rows per namespace with k = 32, so most rows are padded,
    # through each merge kernel: 79 partials per query (multi-wave merge),
    # 2 partials (rank merge) and 24 partials (one-wave tournament)
    say(f"case: scoped padding n={n} d=64 m={m} k=32")
    cb = inputs.clustered_bank(40, TAG_SCOPED, n, 64, 16, 0.3, "bf16", m_queries=m)
    rns, live, kns = inputs.namespaces(40, TAG_SCOPED, n, n // 10, 0.1, run=4, query_src=cb.query_src)
    g = run_scoped(cb.emb, cb.queries, rns, live, kns, 32, 1.0)
    check_topk_scoped(f"scoped-pad-{n}", cb.queries, cb.emb, np.arange(m), g, 32, 1.0, rns, live, kns)
    assert np.any(g["idx"] == -1)


def test_scoped_fp32_full_probabilities(dev):
    # VALU path: full_prob is 0 outside the scope and sums to 1 over it
    say("case: scoped fp32 n=1024 d=256 m=16 k=8 full_prob")
    bank = inputs.iid_unit(33, TAG_SCOPED, 2, 1024, 256, "f32")
    q = inputs.iid_unit(33, TAG_SCOPED, 4, 16, 256, "f32")
    rns, live, kns = inputs.namespaces(33, TAG_SCOPED, 1024, 3, 0.1, run=16, m=16)
    kns = kns.copy()
    kns[3] = -1
    g = run_scoped(bank, q, rns, live, kns, 8, 4.0, full=True)
    check_topk_scoped("scoped-f32", q, bank, np.arange(16), g, 8, 4.0, rns, live, kns)
    import oracle
    ref = oracle.retrieve_scoped(q, bank, 8, rns, live, kns, scale=4.0, full=True)
    fp = g["full_prob"].astype(np.float64)
    assert np.all(np.abs(fp - ref["full_prob"]) <= 1e-5 * ref["full_prob"] + 1e-12)
    sums = fp.sum(axis=1)
    assert np.allclose(sums[kns >= 0], 1.0, rtol=0, atol=1e-5) and sums[3] == 0.0


def test_scoped_integer_grid_exact(dev):
    # exactly representable scores with duplicated rows: ids, scores and
    # padding match the oracle exactly
    say("case: scoped integer grid exact d=64")
    base = inputs.integer_grid(34, TAG_SCOPED, 400, 64)
    bank = np.concatenate([base, base])
    q = inputs.integer_grid(35, TAG_SCOPED, 140, 64)
    rns, live, kns = inputs.namespaces(34, TAG_SCOPED, 800, 5, 0.15, run=8, m=140)
    g = run_scoped(bank, q, rns, live, kns, 16, 2.0)
    check_topk_scoped("scoped-grid", q, bank, np.arange(140), g, 16, 2.0, rns, live, kns)
    import oracle
    ref = oracle.retrieve_scoped(q, bank, 16, rns, live, kns, scale=2.0)
    assert np.array_equal(g["idx"], ref["idx"])
    assert np.array_equal(g["score"].astype(np.float64), ref["score"])


def test_scoped_sampled_threshold(dev):
    """The sampled lower bound must come from in-scope rows only: 2000
    queries against 70,000 rows (the sample pass runs), 8 namespaces, 10%
    tombstones."""
    say("case: scoped sampled-threshold n=70000 d=128 m=2000 k=32")
    cb = inputs.clustered_bank(36, TAG_SCOPED, 70000, 128, 64, 0.3, "bf16", m_queries=2000)
    rns, live, kns = inputs.namespaces(36, TAG_SCOPED, 70000, 8, 0.1, run=64, query_src=cb.query_src)
    g = run_scoped(cb.emb, cb.queries, rns, live, kns, 32, 1.0)
    rows = np.unique(np.concatenate([np.random.default_rng(37).choice(2000, 120, replace=False), [0, 1999]]))
    check_topk_scoped("scoped-sampled", cb.queries, cb.emb, rows, {key: v[rows] for key, v in g.items()}, 32, 1.0,
                      rns, live, kns)


@pytest.mark.parametrize("n", [100, 1500])
def test_scoped_relation_build(dev, n):
    # every row against the live rows of its own namespace; tombstoned rows
    # get all-padding results
    say(f"case: scoped relation build bf16 n={n} d=128 k=16 exclude_self")
    cb = inputs.clustered_bank(38, TAG_SCOPED, n, 128, 8, 0.3, "bf16")
    rns, live, _ = inputs.namespaces(38, TAG_SCOPED, n, 4, 0.2, run=20)
    abi = inputs.scoped_row_ns(rns, live)
    g = host(pm.mem_build_relations_scoped(up(cb.emb), up(abi), 16, 3.0, True))
    check_topk_scoped(f"scoped-rel-{n}", cb.emb, cb.emb, np.arange(n), g, 16, 3.0, rns, live, abi,
                      self_idx=np.arange(n))
    dead = np.nonzero(live == 0)[0]
    assert np.all(g["idx"][dead] == -1) and np.all(g["lse"][dead] == -np.inf)


def test_scoped_one_namespace_equals_unscoped(dev):
    # one namespace, no tombstones: identical to the unscoped call, bit for bit
    say("case: scoped with a single namespace vs unscoped n=5000 d=128 m=300 k=32")
    cb = inputs.clustered_bank(39, TAG_SCOPED, 5000, 128, 32, 0.3, "bf16", m_queries=300)
    zeros_b = np.zeros(5000, np.int32)
    g = run_scoped(cb.emb, cb.queries, zeros_b, np.ones(5000, np.uint8), np.zeros(300, np.int32), 32, 1.0)
    u = host(pm.mem_retrieve_topk(up(cb.emb), up(cb.queries), 32, 1.0))
    for key in u:
        assert np.array_equal(g[key], u[key]), key


# ------------------------------------------------------------------ grouped (per-namespace chunk tables)

def run_grouped(bank, q, row_ns, row_live, key_ns, k, scale=1.0):
    offsets, chunks = inputs.chunk_tables(inputs.scoped_row_ns(row_ns, row_live))
    out = pm.mem_retrieve_topk_grouped(up(bank), up(offsets), up(chunks), up(q), up(np.asarray(key_ns, np.int32)),
                                       k, scale)
    return host(out)


# k = 1 and 5 (lists of 8) and k = 16 on tables of about one tile run without
# the threshold sample; k = 32 runs with it
@pytest.mark.parametrize("m,run,k", [(300, 20, 16), (40, 1, 16), (700, 64, 16), (300, 20, 5), (700, 64, 1),
                                     (700, 64, 32)])
def test_grouped_matches_oracle(dev, m, run, k):
    say(f"case: grouped bf16 n=6000 d=128 m={m} run={run} k={k}")
    cb = inputs.clustered_bank(50, TAG_SCOPED, 6000, 128, 16, 0.3, "bf16", m_queries=m)
    rns, live, kns = inputs.namespaces(50, TAG_SCOPED, 6000, 12, 0.15, run=run, query_src=cb.query_src)
    g = run_grouped(cb.emb, cb.queries, rns, live, kns, k, 2.0)
    r = check_topk_scoped(f"grouped-m{m}-k{k}", cb.queries, cb.emb, np.arange(m), g, k, 2.0, rns, live, kns)
    assert r["exact_rows"] >= 0.9 * r["rows"]


def test_grouped_sampled_lists_of_16(dev):
    # six tables of about 3,400 live rows (more than four 512-row tiles on
    # average): k = 16 takes the threshold sample over each table's first tile
    say("case: grouped n=24000 d=128 m=300 k=16 with the threshold sample")
    cb = inputs.clustered_bank(56, TAG_SCOPED, 24000, 128, 32, 0.3, "bf16", m_queries=300)
    rns, live, kns = inputs.namespaces(56, TAG_SCOPED, 24000, 6, 0.15, run=40, query_src=cb.query_src)
    offsets, _ = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
    assert offsets[-1] / 6 >= 4 * 512
    g = run_grouped(cb.emb, cb.queries, rns, live, kns, 16, 1.0)
    r = check_topk_scoped("grouped-k16-sampled", cb.queries, cb.emb, np.arange(300), g, 16, 1.0, rns, live, kns)
    assert r["exact_rows"] >= 0.9 * r["rows"]


def test_grouped_small_tables_padding(dev):
    # 2,000 namespaces over 20,000 rows (about 9 live rows each) with k = 16,
    # queries without a namespace (-1) or with one past the tables
    say("case: grouped small tables n=20000 d=96 m=500 k=16")
    cb = inputs.clustered_bank(51, TAG_SCOPED, 20000, 96, 64, 0.3, "bf16", m_queries=500)
    rns, live, kns = inputs.namespaces(51, TAG_SCOPED, 20000, 2000, 0.1, run=3, query_src=cb.query_src)
    kns = kns.copy()
    kns[::11] = -1
    kns[4::13] = 5000
    g = run_grouped(cb.emb, cb.queries, rns, live, kns, 16, 1.0)
    check_topk_scoped("grouped-small", cb.queries, cb.emb, np.arange(500), g, 16, 1.0, rns, live, kns)
    assert np.any(g["idx"] == -1) and np.any(g["lse"] == -np.inf)


@pytest.mark.parametrize("n_ns,m", [(5000, 600), (40, 20000)])
def test_grouped_preparation_in_several_launches(dev, n_ns, m):
    # more than 4,096 namespaces or 16,384 queries: the query grouping runs
    # as count, scans and scatter kernels instead of one workgroup
    say(f"case: grouped n=30000 d=96 n_ns={n_ns} m={m} k=8, multi-launch preparation")
    cb = inputs.clustered_bank(57, TAG_SCOPED, 30000, 96, 64, 0.3, "bf16", m_queries=m)
    rns, live, kns = inputs.namespaces(57, TAG_SCOPED, 30000, n_ns, 0.1, run=2, query_src=cb.query_src)
    kns = kns.copy()
    kns[::17] = -1
    g = run_grouped(cb.emb, cb.queries, rns, live, kns, 8, 1.0)
    rows = np.unique(np.concatenate([np.random.default_rng(58).choice(m, min(m, 300), replace=False), [0, m - 1]]))
    r = check_topk_scoped(f"grouped-prep-{n_ns}-{m}", cb.queries, cb.emb, rows, {key: v[rows] for key, v in g.items()},
                          8, 1.0, rns, live, kns)
    assert r["exact_rows"] >= 0.9 * r["rows"]


def test_grouped_large_tables_many_splits(dev):
    # two namespaces of about 31,500 live rows: 31 splits per namespace, many
    # tiles per split, 200 queries (several 64-query tiles per namespace)
    say("case: grouped large tables n=70000 d=128 m=200 k=32")
    cb = inputs.clustered_bank(52, TAG_SCOPED, 70000, 128, 64, 0.3, "bf16", m_queries=200)
    rns, live, kns = inputs.namespaces(52, TAG_SCOPED, 70000, 2, 0.1, run=500, query_src=cb.query_src)
    g = run_grouped(cb.emb, cb.queries, rns, live, kns, 32, 1.0)
    rows = np.unique(np.concatenate([np.random.default_rng(53).choice(200, 60, replace=False), [0, 199]]))
    check_topk_scoped("grouped-large", cb.queries, cb.emb, rows, {key: v[rows] for key, v in g.items()}, 32, 1.0,
                      rns, live, kns)


def test_grouped_integer_grid_exact(dev):
    say("case: grouped integer grid exact d=128")
    base = inputs.integer_grid(54, TAG_SCOPED, 900, 128)
    bank = np.concatenate([base, base])
    q = inputs.integer_grid(55, TAG_SCOPED, 150, 128)
    rns, live, kns = inputs.namespaces(54, TAG_SCOPED, 1800, 5, 0.15, run=8, m=150)
    g = run_grouped(bank, q, rns, live, kns, 16, 2.0)
    import oracle
    ref = oracle.retrieve_scoped(q, bank, 16, rns, live, kns, scale=2.0)
    assert np.array_equal(g["idx"], ref["idx"])
    assert np.array_equal(g["score"].astype(np.float64), ref["score"])


def test_grouped_no_namespaces(dev):
    say("case: grouped with no chunk tables")
    bank = inputs.iid_unit(56, TAG_SCOPED, 0, 300, 128, "bf16")
    q = inputs.iid_unit(56, TAG_SCOPED, 4, 20, 128, "bf16")
    out = pm.mem_retrieve_topk_grouped(up(bank), up(np.zeros(1, np.int32)), up(np.zeros(0, np.int32)), up(q),
                                       up(np.zeros(20, np.int32)), 8, 1.0)
    g = host(out)
    assert np.all(g["idx"] == -1) and np.all(g["lse"] == -np.inf) and np.all(g["prob"] == 0)


def test_grouped_table_entries_outside_bank_are_ignored(dev):
    # entries past the bank are dropped (in the sample as well as the pass)
    say("case: grouped with table entries outside the bank")
    cb = inputs.clustered_bank(57, TAG_SCOPED, 3000, 128, 16, 0.3, "bf16", m_queries=100)
    rns, live, kns = inputs.namespaces(57, TAG_SCOPED, 3000, 3, 0.1, run=10, query_src=cb.query_src)
    offsets, chunks = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
    # append one out-of-range entry at the end of every table (ids stay ascending)
    bad_off = offsets + np.arange(offsets.shape[0], dtype=np.int32)
    bad = np.concatenate([np.append(chunks[offsets[u]:offsets[u + 1]], 3000 + u)
                          for u in range(offsets.shape[0] - 1)]).astype(np.int32)
    out = pm.mem_retrieve_topk_grouped(up(cb.emb), up(bad_off), up(bad), up(cb.queries), up(kns), 16, 1.0)
    g = host(out)
    check_topk_scoped("grouped-oob", cb.queries, cb.emb, np.arange(100), g, 16, 1.0, rns, live, kns)


def test_grouped_offsets_are_clamped_to_the_table(dev):
    # a last offset past the table is read as the table's end
    say("case: grouped with a last offset past the table")
    cb = inputs.clustered_bank(58, TAG_SCOPED, 2000, 128, 8, 0.3, "bf16", m_queries=64)
    rns, live, kns = inputs.namespaces(58, TAG_SCOPED, 2000, 4, 0.1, run=10, query_src=cb.query_src)
    offsets, chunks = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
    bad = offsets.copy()
    bad[-1] += 1000
    g = host(pm.mem_retrieve_topk_grouped(up(cb.emb), up(bad), up(chunks), up(cb.queries), up(kns), 8, 1.0))
    ok = host(pm.mem_retrieve_topk_grouped(up(cb.emb), up(offsets), up(chunks), up(cb.queries), up(kns), 8, 1.0))
    for key in g:
        assert np.array_equal(g[key], ok[key]), key
