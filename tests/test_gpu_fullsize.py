"""Parity at the full workload sizes, in the launch configuration the
benchmark times: the GPU runs every row; the fp64 oracle checks sampled rows
(and sampled gathered blocks, whose expected bytes it generates itself)."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs
from parity import bank_max_norm, check_topk, check_topk_scoped

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def up(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def fetch(out):
    idx, score, prob, lse = out
    torch.cuda.synchronize()
    return {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
            "lse": lse.cpu().numpy()}


def sub(g, rows):
    return {k: v[rows] for k, v in g.items()}


def tile_ends(m, tile):
    """First and last query of every query tile of the launch."""
    starts = np.arange(0, m, tile)
    return np.unique(np.concatenate([starts, np.minimum(starts + tile, m) - 1]))


def report(name, r):
    say(f"  {name}: bit-exact top-k sets {r['exact_rows']}/{r['rows']} rows "
        f"({100.0 * r['exact_rows'] / r['rows']:.1f} %), max |lse - lse_ref| {r['lse_err_max']:.3g}")


_BANK1M = {}


def bank_1m():
    """The 1,048,576 x 1024 bf16 clustered bank with 1,024 queries (drawn once per module)."""
    if not _BANK1M:
        say("  drawing the 1M-chunk bank")
        cb = inputs.clustered_bank(0, inputs.TAG_GATHER, 1 << 20, 1024, 1024, 0.3, "bf16", m_queries=1024)
        _BANK1M["cb"] = cb
        _BANK1M["bmax"] = bank_max_norm(cb.emb)
    return _BANK1M["cb"], _BANK1M["bmax"]


def test_relation_build_32k(dev):
    say("case: relation build 32,768 x 768 bf16 k=32")
    cb = inputs.clustered_bank(0, inputs.TAG_RELATION, 32768, 768, 256, 0.3, "bf16")
    g = fetch(pm.mem_build_relations(up(cb.emb), 32, 1.0, True))
    # the first and last key of each of the 128 query tiles of 256 keys, plus
    # 64 drawn keys
    rows = np.unique(np.concatenate([np.random.default_rng(1).choice(32768, 64, replace=False),
                                     tile_ends(32768, 256)]))
    assert len(rows) >= 256
    r = check_topk("relation-32k", cb.emb, cb.emb, rows, sub(g, rows), 32, 1.0, self_idx=np.arange(32768))
    report("relation-32k", r)


def test_batched_retrieval_262k(dev):
    say("case: batched retrieval 262,144 x 1024 bf16, 512 queries, k=16")
    cb = inputs.clustered_bank(0, inputs.TAG_BATCHED, 262144, 1024, 1024, 0.3, "bf16", m_queries=512)
    g = fetch(pm.mem_retrieve_topk(up(cb.emb), up(cb.queries), 16, 1.0))
    # 2,048-row splits: the queries whose source rows (usually their top-1)
    # sit next to a split boundary, the first and last query of both
    # 256-query tiles, and drawn queries
    off = cb.query_src % 2048
    edge = np.argsort(np.minimum(off, 2047 - off), kind="stable")[:16]
    rows = np.unique(np.concatenate([np.random.default_rng(2).choice(512, 120, replace=False), tile_ends(512, 256),
                                     edge]))
    assert len(rows) >= 128
    r = check_topk("batched-262k", cb.queries, cb.emb, rows, sub(g, rows), 16, 1.0)
    report("batched-262k", r)
    # sanity statistic of the workload: top-1 is usually the perturbed source row
    assert np.mean(g["idx"][:, 0] == cb.query_src) > 0.5


@pytest.mark.timeout(300)
def test_small_batch_streaming_1m(dev):
    # the benchmark's small-batch shapes: the first 16, 64 and 128 queries
    # against the whole 1M-chunk bank (narrow and 128-query workgroups, whose
    # sample passes run 256-row tiles); every row is checked
    cb, bmax = bank_1m()
    bank = up(cb.emb)
    for m in (16, 64, 128):
        say(f"case: small-batch retrieval, {m} queries x 1,048,576 x 1024 bf16, k=32")
        q = np.ascontiguousarray(cb.queries[:m])
        g = fetch(pm.mem_retrieve_topk(bank, up(q), 32, 1.0))
        r = check_topk(f"stream-bank-m{m}", q, cb.emb, np.arange(m), g, 32, 1.0, bmax=bmax)
        report(f"stream-bank-m{m}", r)


@pytest.mark.timeout(400)
def test_retrieval_gather_1m(dev):
    say("case: retrieval + gather 1,048,576 x 1024 bf16, 1,024 queries, k=32, 128 GiB pool")
    n, d, m, k, ppc, page = 1 << 20, 1024, 1024, 32, 2, 65536
    cb, bmax = bank_1m()
    bank = up(cb.emb)
    g = fetch(pm.mem_retrieve_topk(bank, up(cb.queries), k, 1.0))
    # 16,384-row splits: queries whose source rows sit next to a split
    # boundary, the first and last query of each 256-query tile, and drawn
    # queries (the oracle scores each against the whole bank)
    off = cb.query_src % 16384
    edge = np.argsort(np.minimum(off, 16383 - off), kind="stable")[:16]
    rows = np.unique(np.concatenate([np.random.default_rng(3).choice(m, 112, replace=False), tile_ends(m, 256),
                                     edge]))
    assert len(rows) >= 128
    r = check_topk("retrieval-1m", cb.queries, cb.emb, rows, sub(g, rows), k, 1.0, bmax=bmax)
    report("retrieval-1m", r)
    del bank
    table_np = inputs.page_layout(0, inputs.TAG_GATHER, cb.cluster, ppc)
    key = inputs.payload_key(0, inputs.TAG_GATHER)
    table = up(table_np)
    pool = torch.empty((n * ppc, page), dtype=torch.uint8, device="cuda")
    inputs.fill_payload_device(pool, table, key)
    # the gather in the benchmark's launch shape (1,024 groups of 32 ids, time
    # order) on seeded ids -- distinct within a group, as a top-32 is -- so no
    # expected value depends on the GPU's selection
    gen = np.random.default_rng(4)
    sel = np.stack([gen.choice(n, k, replace=False) for _ in range(m)]).astype(np.int32)
    ids = up(sel)
    out = pm.mem_gather_chunks(pool, table, ids, pm.MEM_ORDER_TIME, k)
    torch.cuda.synchronize()
    slots = np.unique(np.concatenate([gen.choice(m * k, 200, replace=False), [0, m * k - 1]]))
    exp = oracle.expected_blocks(key, sel.ravel(), oracle.ORDER_TIME, k, ppc, page, slots=slots)
    got = out[torch.from_numpy(slots).cuda()].cpu().numpy().view(np.uint64).reshape(exp.shape)
    assert np.array_equal(got, exp)
    del out
    # budget-aware gather of the same ids: 3,072-token budget, 256-byte token
    # rows, memories of 128 to 512 tokens
    say("case: budget gather of the same ids, budget 3072")
    tok = inputs.token_lengths(0, inputs.TAG_GATHER, n, 128, 512)
    rows, tokens, kept = pm.mem_gather_budget(pool, table, up(tok), ids, 3072, 256)
    torch.cuda.synchronize()
    for i in np.unique(np.concatenate([np.random.default_rng(5).choice(m, 10, replace=False), [0, m - 1]])):
        # the oracle on a pool of just this key's chunks (ids renumbered in
        # the same order, so admission and time order are unchanged)
        u = np.unique(sel[i])
        sub_pool = np.stack([oracle.payload_page(key, c, p, ppc, page).view(np.uint8) for c in u for p in range(ppc)])
        sub_table = np.arange(len(u) * ppc, dtype=np.int32).reshape(len(u), ppc)
        sub_ids = np.searchsorted(u, sel[i]).astype(np.int32)[None]
        r_rows, r_tok, r_kept = oracle.gather_budget(sub_pool, sub_table, tok[u], sub_ids, 3072, 256)
        assert np.array_equal(rows[i].cpu().numpy(), r_rows[0]), f"rows of key {i}"
        assert int(tokens[i]) == int(r_tok[0])
        assert np.array_equal(kept[i].cpu().numpy(), np.where(r_kept[0] >= 0, u[np.maximum(r_kept[0], 0)], -1))
    del pool, rows


def test_grouped_request_selection_1m(dev):
    # the request path's selection as the benchmark runs it: 1,024 requests,
    # top-5 within each request's own chunk table, 256 (user, session)
    # namespaces in runs of 64 chunks, 10 % of chunks deleted
    say("case: grouped top-5, 1,048,576 x 1024 bf16, 1,024 queries, 256 namespaces")
    n, d, m, k = 1 << 20, 1024, 1024, 5
    cb, _ = bank_1m()
    rns, live, kns = inputs.namespaces(0, inputs.TAG_GATHER, n, 256, 0.1, run=64, query_src=cb.query_src)
    offs, chs = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
    g = fetch(pm.mem_retrieve_topk_grouped(up(cb.emb), up(offs), up(chs), up(cb.queries), up(kns), k, 1.0))
    rows = np.unique(np.concatenate([np.random.default_rng(6).choice(m, 12, replace=False), [0, m - 1]]))
    r = check_topk_scoped("grouped-1m", cb.queries, cb.emb, rows, sub(g, rows), k, 1.0, rns, live, kns)
    say(f"  grouped-1m: bit-exact top-k sets {r['exact_rows']}/{r['rows']} rows")


def test_scoped_retrieval_1m(dev):
    # the dense masked call at the benchmark's size: 256 namespaces in runs of
    # 64 rows, 10 % tombstones, 1,024 queries, top-32
    say("case: scoped top-32, 1,048,576 x 1024 bf16, 1,024 queries, 256 namespaces")
    n, d, m, k = 1 << 20, 1024, 1024, 32
    cb, _ = bank_1m()
    rns, live, kns = inputs.namespaces(0, inputs.TAG_GATHER, n, 256, 0.1, run=64, query_src=cb.query_src)
    row_ns = inputs.scoped_row_ns(rns, live)
    g = fetch(pm.mem_retrieve_topk_scoped(up(cb.emb), up(row_ns), up(cb.queries), up(kns), k, 1.0))
    rows = np.unique(np.concatenate([np.random.default_rng(7).choice(m, 12, replace=False), [0, m - 1]]))
    r = check_topk_scoped("scoped-1m", cb.queries, cb.emb, rows, sub(g, rows), k, 1.0, rns, live, kns)
    say(f"  scoped-1m: bit-exact top-k sets {r['exact_rows']}/{r['rows']} rows")


@pytest.mark.timeout(900)
def test_streaming_append_rounds(dev):
    # the whole streaming workload: 64 rounds of 4,096 new chunks scored
    # against the bank as it stands (1,048,576 rows growing to 1,306,624),
    # then appended; every round checks 8 keys (the first and last new chunk
    # and 6 drawn) against the oracle over the whole current bank, and the
    # appended table and rows bit for bit
    rounds, per = 64, 4096
    say(f"case: streaming append, 1,048,576-chunk bank, {per} new chunks per round, {rounds} rounds")
    n, d, k, ppc = 1 << 20, 1024, 32, 2
    cb, bmax = bank_1m()
    cap = n + per * rounds
    emb = torch.empty((cap, d), dtype=torch.bfloat16, device="cuda")
    emb[:n] = up(cb.emb)
    table = torch.full((cap, ppc), -1, dtype=torch.int32, device="cuda")
    table[:n] = up(inputs.page_layout(0, inputs.TAG_GATHER, cb.cluster, ppc))
    st = pm.BankState(emb, n, table, n * ppc, cap * ppc)
    host_bank = np.empty((cap, d), dtype=np.uint16)
    host_bank[:n] = cb.emb
    exact = checked = 0
    lse_err = 0.0
    for r in range(rounds):
        new = inputs.appended_chunks(0, inputs.TAG_STREAM, r, per, cb.centroids, 0.3)
        g = fetch(pm.mem_retrieve_topk(st.live, up(new), k, 1.0))
        rows = np.unique(np.concatenate([np.random.default_rng(10 + r).choice(per, 6, replace=False), [0, per - 1]]))
        res = check_topk(f"stream-r{r}", new, host_bank[:st.n], rows, sub(g, rows), k, 1.0, bmax=bmax)
        exact += res["exact_rows"]
        checked += res["rows"]
        lse_err = max(lse_err, res["lse_err_max"])
        nf = st.next_free_page
        pm.mem_append_chunks(st, up(new))
        torch.cuda.synchronize()
        assert np.array_equal(table[st.n - per:st.n].cpu().numpy(), oracle.append_table(per, ppc, nf))
        assert np.array_equal(emb[st.n - per:st.n].view(torch.int16).cpu().numpy().view(np.uint16), new)
        host_bank[st.n - per:st.n] = new
        bmax = max(bmax, bank_max_norm(new))
        if r % 8 == 7:
            say(f"  rounds 0-{r} green, bank at {st.n} rows")
    assert st.n == n + per * rounds
    report("stream-64-rounds", {"rows": checked, "exact_rows": exact, "lse_err_max": lse_err})
