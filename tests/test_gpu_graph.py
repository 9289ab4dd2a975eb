"""The retrieval and gather calls captured into HIP graphs (torch.cuda.graph
over the binding, which enqueues on the current stream) and replayed: every
replay must equal the eager call bit for bit, also with eager work and
synchronisations between replays and with the inputs rewritten in place.
No call on these paths records a memset or a host synchronisation."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs

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


def outputs(m, k):
    return (torch.empty((m, k), dtype=torch.int32, device="cuda"), torch.empty((m, k), device="cuda"),
            torch.empty((m, k), device="cuda"), torch.empty(m, device="cuda"))


def replay_and_check(call, results, eager_between, refill=None):
    """call() writes into `results` (tensors); capture it, then replay several
    times with eager work between and compare with an eager call each time."""
    call()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    for rep in range(4):
        if refill is not None:
            refill(rep)
        torch.cuda.synchronize()
        call()                      # eager on the current inputs
        torch.cuda.synchronize()
        want = [t.clone() for t in results]
        for t in results:
            t.fill_(0)
        eager_between()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(results, want):
            assert torch.equal(a, b), f"replay {rep} differs from the eager call"


def test_graph_tiny_fp32_full_probabilities(dev):
    say("case: graph of the tiny fp32 retrieval with full probabilities")
    bank = up(inputs.iid_unit(60, 85, 2, 1024, 256, "f32"))
    q = up(inputs.iid_unit(60, 85, 4, 16, 256, "f32"))
    qs = [up(inputs.iid_unit(61 + r, 85, 4, 16, 256, "f32")) for r in range(4)]
    out, fp = outputs(16, 8), torch.empty((16, 1024), device="cuda")
    ws = torch.empty(pm.mem_workspace_bytes(16, 1024, 256, 8, pm.MEM_F32), dtype=torch.uint8, device="cuda")
    other = up(inputs.iid_unit(70, 85, 4, 16, 256, "f32"))
    replay_and_check(lambda: pm.mem_retrieve_topk(bank, q, 8, 2.0, out=out, full_prob=fp, workspace=ws),
                     list(out) + [fp], lambda: pm.mem_retrieve_topk(bank, other, 8, 1.0),
                     refill=lambda r: q.copy_(qs[r]))


def test_graph_matrix_core_with_sample_pass(dev):
    # 2,000 queries against 70,000 rows: sample pass, k-th search, bound
    # init, full pass and merge all captured
    say("case: graph of the matrix-core retrieval with its sample pass")
    cb = inputs.clustered_bank(62, 85, 70000, 128, 64, 0.3, "bf16", m_queries=2000)
    bank, q = up(cb.emb), up(cb.queries)
    out = outputs(2000, 32)
    ws = torch.empty(pm.mem_workspace_bytes(2000, 70000, 128, 32, pm.MEM_BF16), dtype=torch.uint8, device="cuda")
    replay_and_check(lambda: pm.mem_retrieve_topk(bank, q, 32, 1.0, out=out, workspace=ws), list(out),
                     lambda: torch.matmul(bank[:512].float(), q[:64].float().T.contiguous()))


def test_graph_gathers(dev):
    say("case: graph of the time-ordered and the budget gathers")
    n, ppc, pb = 400, 2, 4096
    cl = np.random.default_rng(63).integers(0, 9, size=n)
    table = up(inputs.page_layout(63, 85, cl, ppc))
    pool = up(inputs.host_pool(inputs.payload_key(63, 85), inputs.page_layout(63, 85, cl, ppc), pb))
    g = np.random.default_rng(64)
    ids = up(np.stack([g.choice(n, 16, replace=False) for _ in range(50)]).astype(np.int32))
    tok = up(inputs.token_lengths(63, 85, n, 0, 2 * pb // 256))
    blocks = torch.empty((50 * 16, ppc, pb), dtype=torch.uint8, device="cuda")
    rows = (torch.empty((50, 300, 256), dtype=torch.uint8, device="cuda"), torch.empty(50, dtype=torch.int32,
            device="cuda"), torch.empty((50, 16), dtype=torch.int32, device="cuda"))

    def call():
        pm.mem_gather_chunks(pool, table, ids, pm.MEM_ORDER_TIME, 16, out=blocks)
        pm.mem_gather_budget(pool, table, tok, ids, 300, 256, out=rows)
    perms = [up(np.stack([g.choice(n, 16, replace=False) for _ in range(50)]).astype(np.int32)) for _ in range(4)]
    replay_and_check(call, [blocks] + list(rows), lambda: torch.cuda.synchronize(),
                     refill=lambda r: ids.copy_(perms[r]))


def test_graph_grouped_retrieval(dev):
    say("case: graph of the grouped retrieval (device scans and scatter included)")
    cb = inputs.clustered_bank(65, 85, 6000, 128, 16, 0.3, "bf16", m_queries=300)
    rns, live, kns = inputs.namespaces(65, 85, 6000, 12, 0.15, run=20, query_src=cb.query_src)
    offs, chs = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
    bank, q, ot, ct, qn = up(cb.emb), up(cb.queries), up(offs), up(chs), up(kns)
    out = outputs(300, 16)
    ws = torch.empty(pm.mem_workspace_bytes_grouped(300, offs.shape[0] - 1, chs.shape[0], 128, 16),
                     dtype=torch.uint8, device="cuda")
    rolled = [up(np.roll(kns, r + 1)) for r in range(4)]
    replay_and_check(lambda: pm.mem_retrieve_topk_grouped(bank, ot, ct, q, qn, 16, 1.0, out=out, workspace=ws),
                     list(out), lambda: pm.mem_retrieve_topk(bank, q, 8, 1.0),
                     refill=lambda r: qn.copy_(rolled[r]))


def test_graph_relation_build_clustered_order(dev):
    # 32,845 rows as keys: sample pass, k-th search with best sampled rows,
    # the clustered order and the query copy, both full-pass launches with
    # the bound search between them, and the merge, all captured; the bank
    # is rewritten in place between replays (other rows in other order), so
    # every replay forms its order from the rows it sees
    say("case: graph of the relation build in clustered key order")
    cb = inputs.clustered_bank(63, 86, 32768 + 77, 128, 256, 0.3, "bf16")
    n = cb.emb.shape[0]
    bank = up(cb.emb)
    variants = [up(np.ascontiguousarray(np.roll(cb.emb, 1000 * (r + 1), axis=0))) for r in range(4)]
    out = outputs(n, 32)
    ws = torch.empty(pm.mem_workspace_bytes(n, n, 128, 32, pm.MEM_BF16), dtype=torch.uint8, device="cuda")
    replay_and_check(lambda: pm.mem_build_relations(bank, 32, 1.0, True, out=out, workspace=ws), list(out),
                     lambda: pm.mem_retrieve_topk(bank, bank[:256].contiguous(), 8, 1.0),
                     refill=lambda r: bank.copy_(variants[r]))
