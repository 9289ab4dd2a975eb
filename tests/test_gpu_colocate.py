"""Association-aware relocation (mem_colocate) on the GPU against the oracle:
pool bytes, directory, counts and frontier must match exactly.  Inputs (ids
and scores) come from the seeded generators or from the oracle's own
selection, never from the GPU.  Calls go through the C ABI."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs

pytestmark = pytest.mark.gpu

TAG_COLOC = 84


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


def run_both(pool, table, ids, sc, tau, mg, nf):
    ref = oracle.colocate(pool, table, ids, sc, tau, mg, nf)
    gp, gt = up(pool), up(table)
    res = pm.mem_colocate(gp, gt, up(ids.astype(np.int32)), up(sc.astype(np.float32)), tau, mg, nf)
    torch.cuda.synchronize()
    assert np.array_equal(gt.cpu().numpy(), ref["table"]), "directory"
    assert np.array_equal(gp.cpu().numpy(), ref["pool"]), "pool bytes"
    assert res["moved_chunks"] == ref["moved"] and res["groups"] == ref["groups"]
    assert res["next_free_page"] == ref["next_free"]
    return res


def test_colocate_worked_example(dev):
    say("case: relocation worked example")
    pb = 16
    pool = (np.arange(40 * pb) % 251).astype(np.uint8).reshape(40, pb)
    table = np.arange(20, dtype=np.int32).reshape(10, 2)
    ids = np.array([[7, 2, 5], [5, 9, 1], [3, -1, 8], [9, 4, 0]], np.int32)
    sc = np.array([[0.9, 0.8, 0.6], [0.95, 0.75, 0.7], [0.7, 0.99, 0.2], [0.8, 0.9, 0.1]], np.float32)
    res = run_both(pool, table, ids, sc, 0.7, 2, 20)
    assert res["moved_chunks"] == 6


@pytest.mark.parametrize("tau,mg", [(0.7, 2), (0.5, 1), (0.9, 3), (-2.0, 1), (1.5, 1)])
@pytest.mark.parametrize("ppc", [1, 2, 3])
def test_colocate_random(dev, tau, mg, ppc):
    # 500 chunks in a shuffled layout, 300 keys of k = 12 with 10 % -1
    # entries and some repeated ids, scores uniform in [0.2, 1]
    say(f"case: relocation random tau={tau} min_group={mg} ppc={ppc}")
    g = np.random.default_rng(100 + ppc)
    n, m, k = 500, 300, 12
    table = g.permutation(n * ppc).astype(np.int32).reshape(n, ppc)
    pool = g.integers(0, 256, size=(n * ppc * 2 + 64, 64), dtype=np.uint8)
    ids = np.stack([g.choice(n, k, replace=False) for _ in range(m)]).astype(np.int32)
    ids[g.random((m, k)) < 0.1] = -1
    ids[::7, 3] = ids[::7, 1]
    sc = g.uniform(0.2, 1.0, size=(m, k)).astype(np.float32)
    run_both(pool, table, ids, sc, tau, mg, n * ppc)


def test_colocate_relation_groups(dev):
    # groups from the oracle's own relation lists on a clustered bf16 bank:
    # each chunk's top-8 related chunks scoring >= 0.7
    say("case: relocation of oracle relation groups, 2000 chunks")
    cb = inputs.clustered_bank(41, TAG_COLOC, 2000, 128, 40, 0.3, "bf16")
    rel = oracle.retrieve(cb.emb, cb.emb, 8, self_idx=np.arange(2000))
    ids, sc = rel["idx"].astype(np.int32), rel["score"].astype(np.float32)
    assert (sc >= 0.7).mean() > 0.2
    cl = np.random.default_rng(41).integers(0, 20, size=2000)
    table = inputs.page_layout(41, TAG_COLOC, cl, 2)
    pool = np.random.default_rng(42).integers(0, 256, size=(4000 * 3, 256), dtype=np.uint8)
    res = run_both(pool, table, ids, sc, 0.7, 2, 4000)
    assert res["moved_chunks"] > 500


def test_colocate_ids_outside_table_are_ignored(dev):
    say("case: relocation with ids outside the table")
    g = np.random.default_rng(7)
    table = g.permutation(100).astype(np.int32).reshape(50, 2)
    pool = g.integers(0, 256, size=(300, 32), dtype=np.uint8)
    ids = np.stack([g.choice(50, 6, replace=False) for _ in range(20)]).astype(np.int32)
    sc = g.uniform(0.5, 1.0, size=(20, 6)).astype(np.float32)
    bad = ids.copy()
    bad[::3, 0] = 50
    bad[1::3, 2] = -7
    ref = oracle.colocate(pool, table, np.where((bad < 0) | (bad >= 50), -1, bad), sc, 0.6, 2, 100)
    gp, gt = up(pool), up(table)
    res = pm.mem_colocate(gp, gt, up(bad), up(sc), 0.6, 2, 100)
    torch.cuda.synchronize()
    assert np.array_equal(gt.cpu().numpy(), ref["table"]) and np.array_equal(gp.cpu().numpy(), ref["pool"])
    assert res["moved_chunks"] == ref["moved"]


def test_colocate_entries_outside_the_pool_give_zero_pages(dev):
    # relocated chunks whose directory entries point outside the pool: the
    # fresh pages are zeros, as in the oracle; nothing outside the pool is read
    say("case: relocation with directory entries outside the pool")
    g = np.random.default_rng(13)
    table = g.permutation(200).astype(np.int32).reshape(100, 2)
    table[::9, 1] = 400 + np.arange(12)
    table[5::11, 0] = -1
    pool = g.integers(1, 256, size=(400, 48), dtype=np.uint8)
    ids = np.stack([g.choice(100, 8, replace=False) for _ in range(30)]).astype(np.int32)
    sc = g.uniform(0.5, 1.0, size=(30, 8)).astype(np.float32)
    res = run_both(pool, table, ids, sc, 0.6, 2, 200)
    assert res["moved_chunks"] > 0


def test_colocate_pool_too_small_changes_nothing(dev):
    say("case: relocation without room")
    g = np.random.default_rng(9)
    table = g.permutation(100).astype(np.int32).reshape(50, 2)
    pool = g.integers(0, 256, size=(104, 32), dtype=np.uint8)
    ids = np.stack([g.choice(50, 6, replace=False) for _ in range(20)]).astype(np.int32)
    sc = np.ones((20, 6), np.float32)
    gp, gt = up(pool), up(table)
    with pytest.raises(pm.MemError):
        pm.mem_colocate(gp, gt, up(ids), up(sc), 0.7, 2, 100)
    torch.cuda.synchronize()
    assert np.array_equal(gt.cpu().numpy(), table) and np.array_equal(gp.cpu().numpy(), pool)


def test_colocate_benchmark_geometry_device_pool(dev):
    """The benchmark's geometry: 262,144 two-page chunks of 64 KiB (32 GiB),
    1,024 keys x top-32 (seeded ids, scores uniform in [0.4, 1]), tau 0.7.
    Directory, counts and frontier against the oracle on a pool of 16-byte
    pages; sampled relocated chunks read back their own payload through the
    gather, against the oracle's generator."""
    say("case: relocation 262,144 chunks x 2 pages of 64 KiB, 1,024 groups, device-filled pool")
    n, ppc, page, m, k = 262144, 2, 65536, 1024, 32
    g = np.random.default_rng(21)
    ids = np.stack([g.choice(n, k, replace=False) for _ in range(m)]).astype(np.int32)
    sc = g.uniform(0.4, 1.0, size=(m, k)).astype(np.float32)
    table = inputs.identity_layout(n, ppc)
    nf = n * ppc
    n_pages = nf + m * k * ppc
    ref = oracle.colocate(np.zeros((n_pages, 16), np.uint8), table, ids, sc, 0.7, 2, nf)
    key = inputs.payload_key(21, TAG_COLOC)
    pool = torch.empty((n_pages, page), dtype=torch.uint8, device="cuda")
    gt = up(table)
    inputs.fill_payload_device(pool, gt, key)
    res = pm.mem_colocate(pool, gt, up(ids), up(sc), 0.7, 2, nf)
    torch.cuda.synchronize()
    assert np.array_equal(gt.cpu().numpy(), ref["table"])
    assert res["moved_chunks"] == ref["moved"] > 0 and res["groups"] == ref["groups"]
    assert res["next_free_page"] == ref["next_free"]
    moved = np.nonzero((ref["table"] != table).any(axis=1))[0]
    sample = np.unique(np.concatenate([g.choice(moved, 24, replace=False), g.choice(n, 8, replace=False)]))
    out = pm.mem_gather_chunks(pool, gt, up(sample.astype(np.int32)))
    torch.cuda.synchronize()
    exp = oracle.expected_blocks(key, sample.astype(np.int32), oracle.ORDER_RANK, 1, ppc, page)
    assert np.array_equal(out.cpu().numpy().view(np.uint64).reshape(exp.shape), exp)
