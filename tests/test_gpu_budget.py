"""Budget-aware, time-ordered materialisation (mem_gather_budget) on the GPU
against the oracle, byte for byte.  Calls go through the C ABI."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs

pytestmark = pytest.mark.gpu

TAG_BUDGET = 81


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def pool_case(seed, n, ppc, page_bytes, n_clusters=7):
    cl = np.random.default_rng(seed).integers(0, n_clusters, size=n)
    table = inputs.page_layout(seed, TAG_BUDGET, cl, ppc)
    key = inputs.payload_key(seed, TAG_BUDGET)
    return table, inputs.host_pool(key, table, page_bytes)


def rank_ids(seed, m, k, n, minus_one_frac=0.0):
    g = np.random.default_rng(seed)
    ids = np.stack([g.choice(n, k, replace=False) for _ in range(m)]).astype(np.int32)
    if minus_one_frac:
        cut = g.random(m) < minus_one_frac
        ids[cut, g.integers(0, k, size=int(cut.sum()))] = -1
    return ids


def run(pool, table, tok, ids, budget, row_bytes):
    rows, tokens, kept = pm.mem_gather_budget(up(pool), up(table), up(tok), up(ids), budget, row_bytes)
    torch.cuda.synchronize()
    return rows.cpu().numpy(), tokens.cpu().numpy(), kept.cpu().numpy()


@pytest.mark.parametrize("budget", [0, 1, 37, 512, 513, 1500])
@pytest.mark.parametrize("row_bytes", [64, 256])
def test_budget_bit_exact(dev, budget, row_bytes):
    # 1 KiB pages, 2 per chunk: 32 or 8 token rows per chunk; budgets below
    # one chunk, across the 512-row block boundary and above every chunk
    say(f"case: budget gather budget={budget} row_bytes={row_bytes}")
    table, pool = pool_case(1, 200, 2, 1024)
    cap = 2 * 1024 // row_bytes
    tok = inputs.token_lengths(1, TAG_BUDGET, 200, 0, cap)
    ids = rank_ids(2, 40, 16, 200, minus_one_frac=0.3)
    got = run(pool, table, tok, ids, budget, row_bytes)
    ref = oracle.gather_budget(pool, table, tok, ids, budget, row_bytes)
    for g, r, nm in zip(got, ref, ("rows", "tokens", "kept")):
        assert np.array_equal(g, r), nm


@pytest.mark.parametrize("budget", [512, 1536, 3072])
def test_budget_paper_shape(dev, budget):
    # 512-token blocks of 128 fp16 dims in two 64 KiB pages; memories of 128
    # to 512 tokens; the budgets of the paper's sweep; 32 ids per key
    say(f"case: budget gather 64 KiB pages, 256 B rows, budget={budget}")
    table, pool = pool_case(3, 300, 2, 65536, n_clusters=20)
    tok = inputs.token_lengths(3, TAG_BUDGET, 300, 128, 512)
    ids = rank_ids(4, 48, 32, 300)
    got = run(pool, table, tok, ids, budget, 256)
    ref = oracle.gather_budget(pool, table, tok, ids, budget, 256)
    for g, r, nm in zip(got, ref, ("rows", "tokens", "kept")):
        assert np.array_equal(g, r), nm
    assert np.all(got[1] <= budget) and np.all(got[1] > 0)


def test_budget_edge_cases(dev):
    # k = 64, zero-length chunks, a repeated id, and ids outside the table,
    # which end admission like -1 (the oracle sees them replaced by -1)
    say("case: budget gather edge cases k=64")
    table, pool = pool_case(5, 150, 3, 512)
    cap = 3 * 512 // 16
    tok = inputs.token_lengths(5, TAG_BUDGET, 150, 0, cap)
    tok[::7] = 0
    ids = rank_ids(6, 9, 64, 150)
    ids[1, 10] = ids[1, 3]
    ids[2, 5] = 150
    ids[3, 0] = -5
    ids[4, :] = -1
    got = run(pool, table, tok, ids, 700, 16)
    clean = ids.copy()
    clean[(clean < 0) | (clean >= 150)] = -1
    ref = oracle.gather_budget(pool, table, tok, clean, 700, 16)
    for g, r, nm in zip(got, ref, ("rows", "tokens", "kept")):
        assert np.array_equal(g, r), nm
    assert got[1][4] == 0 and not got[0][4].any() and np.all(got[2][4] == -1)
