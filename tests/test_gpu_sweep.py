"""A seeded sweep of shapes against the oracle: query counts across the
three workgroup shapes, ragged bank sizes (with and without a threshold
sample and the two-launch plan), dimensions, k, scales and cluster
structure, on the matrix-core (bf16) and VALU (fp32) paths, for retrieval
and relation builds.  Every case checks up to 96 of its rows under the
oracle's parity rules; calls go through the C ABI."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_05708_amd as pm
from paper_2607_05708_amd import inputs
from parity import check_topk

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


def case(i):
    """Shape of sweep case i (seeded; the same on every run)."""
    r = np.random.default_rng(1000 + i)
    relation = i % 4 == 3
    dtype = "f32" if i % 6 == 5 else "bf16"
    m = int(r.choice([1, 7, 33, 64, 65, 100, 128, 129, 257, 600, 1100]))
    n = int(r.choice([300, 4097, 20000, 70001, 140000, 300000]))
    if relation:
        n = int(r.choice([900, 5000, 33000, 40001]))
        m = n
    d = int(r.choice([32, 96, 128, 256] if dtype == "bf16" else [20, 64, 100]))
    kmax = 32 if dtype == "bf16" else 64
    k = int(min(r.integers(1, kmax + 1), n - 1))
    scale = float(r.choice([1.0, 8.0, 30.0]))
    clusters = int(r.choice([0, 16, 256]))
    return dict(relation=relation, dtype=dtype, m=m, n=n, d=d, k=k, scale=scale, clusters=clusters, seed=2000 + i)


@pytest.mark.parametrize("i", range(48))
def test_sweep(dev, i):
    c = case(i)
    # bound the oracle's work: at most ~2.5e9 pair-dims over the checked rows
    if c["n"] * c["d"] > 40_000_000:
        c["d"] = 32 if c["dtype"] == "bf16" else 20
    say(f"case: sweep {i}: {c}")
    n, d, m, k = c["n"], c["d"], c["m"], c["k"]
    if c["clusters"]:
        cb = inputs.clustered_bank(c["seed"], 95, n, d, c["clusters"], 0.3, c["dtype"],
                                   m_queries=0 if c["relation"] else m)
        b = cb.emb
        q = b if c["relation"] else cb.queries
    else:
        b = inputs.iid_unit(c["seed"], 95, 0, n, d, c["dtype"])
        q = b if c["relation"] else inputs.iid_unit(c["seed"], 95, 1, m, d, c["dtype"])
    bt = up(b)
    if c["relation"]:
        idx, score, prob, lse = pm.mem_build_relations(bt, k, c["scale"], True)
    else:
        idx, score, prob, lse = pm.mem_retrieve_topk(bt, up(q), k, c["scale"])
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
         "lse": lse.cpu().numpy()}
    rr = np.random.default_rng(c["seed"])
    rows = np.arange(m) if m <= 96 else np.unique(np.concatenate([[0, m - 1], rr.choice(m, 94, replace=False)]))
    sub = {key: v[rows] for key, v in g.items()}
    r = check_topk(f"sweep-{i}", q, b, rows, sub, k, c["scale"],
                   self_idx=np.arange(n) if c["relation"] else None)
    say(f"  rows {r['rows']}, bit-exact sets {r['exact_rows']}, max |lse - lse_ref| {r['lse_err_max']:.3g}")


# ------------------------------------------------------------------ scoped selections

def scoped_case(i):
    r = np.random.default_rng(3000 + i)
    kind = ("scoped", "grouped", "relation")[i % 3]
    dtype = "f32" if (kind == "scoped" and i % 6 == 3) else "bf16"
    n = int(r.choice([500, 6000, 30001, 70001]))
    if kind == "relation":
        n = int(r.choice([500, 3000, 9000]))
    m = n if kind == "relation" else int(r.choice([5, 64, 130, 400]))
    n_ns = int(r.choice([1, 3, 12, 100, 400]))
    dead = float(r.choice([0.0, 0.1, 0.5]))
    run = int(r.choice([1, 8, 64]))
    d = int(r.choice([32, 128]) if dtype == "bf16" else r.choice([24, 64]))
    if kind == "grouped":
        d = int(r.choice([96, 128]))  # the grouped call's stated minimum is 96
    k = int(r.integers(1, (32 if dtype == "bf16" else 64) + 1))
    scale = float(r.choice([1.0, 4.0, 20.0]))
    return dict(kind=kind, dtype=dtype, n=n, m=m, n_ns=n_ns, dead=dead, run=run, d=d, k=k, scale=scale,
                seed=4000 + i)


@pytest.mark.parametrize("i", range(24))
def test_sweep_scoped(dev, i):
    from parity import check_topk_scoped
    c = scoped_case(i)
    say(f"case: scoped sweep {i}: {c}")
    n, m, k, d = c["n"], c["m"], c["k"], c["d"]
    cb = inputs.clustered_bank(c["seed"], 96, n, d, 16, 0.3, c["dtype"], m_queries=0 if c["kind"] == "relation" else m)
    b = cb.emb
    rns, live, kns = inputs.namespaces(c["seed"], 96, n, c["n_ns"], c["dead"], run=c["run"],
                                       query_src=None if c["kind"] == "relation" else cb.query_src)
    abi = inputs.scoped_row_ns(rns, live)
    bt = up(b)
    if c["kind"] == "relation":
        q, key_ns, self_idx = b, abi, np.arange(n)
        out = pm.mem_build_relations_scoped(bt, up(abi), k, c["scale"], True)
    else:
        q, key_ns, self_idx = cb.queries, kns, None
        if c["kind"] == "scoped":
            out = pm.mem_retrieve_topk_scoped(bt, up(abi), up(q), up(kns.astype(np.int32)), k, c["scale"])
        else:
            offsets, chunks = inputs.chunk_tables(abi)
            out = pm.mem_retrieve_topk_grouped(bt, up(offsets), up(chunks), up(q), up(kns.astype(np.int32)), k,
                                               c["scale"])
    torch.cuda.synchronize()
    idx, score, prob, lse = out
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
         "lse": lse.cpu().numpy()}
    rr = np.random.default_rng(c["seed"])
    rows = np.arange(m) if m <= 96 else np.unique(np.concatenate([[0, m - 1], rr.choice(m, 94, replace=False)]))
    sub = {key: v[rows] for key, v in g.items()}
    r = check_topk_scoped(f"scoped-sweep-{i}", q, b, rows, sub, k, c["scale"], rns, live, key_ns,
                          self_idx=self_idx)
    say(f"  rows {r['rows']}, bit-exact sets {r['exact_rows']}")


# ------------------------------------------------------------------ clustered-order relation builds

# Relation builds large enough to take a threshold sample run their full pass
# in clustered key order with the band bound (from 4,096 keys for k > 8, from
# 32,768 for k <= 8), with one to 64 tiles per split.  Each case is one such build:
# (m, d, k, clusters (0: i.i.d.), exclude_self, scale, dup), where dup
# repeats every row of the first half once more (exact ties at every rank).
ORDER_CASES = [
    (32768, 32, 32, 16, True, 1.0, False),     # large clusters: the band is all one cluster
    (33001, 64, 17, 4096, True, 8.0, False),   # about 8 rows per cluster, fewer than k
    (46000, 128, 8, 256, True, 1.0, False),    # lists of 8
    (50000, 96, 1, 1024, True, 30.0, False),   # k = 1
    (65536, 32, 3, 0, False, 1.0, False),      # i.i.d. rows, the row itself kept
    (40000, 768, 32, 256, True, 1.0, False),   # the relation-build dimension
    (36000, 64, 24, 64, True, 8.0, True),      # every row twice
    (33023, 256, 32, 256, False, 1.0, False),  # ragged tail, the row itself kept
    (4096, 768, 32, 256, True, 1.0, False),    # the smallest such build: one tile per split
    (5000, 128, 12, 64, True, 8.0, False),     # two tiles per split, every other split sampled
    (8192, 96, 20, 0, True, 1.0, False),       # i.i.d. rows
    (12289, 64, 32, 4096, False, 1.0, False),  # tiny clusters, ragged, the row itself kept
    (20000, 256, 16, 256, True, 30.0, True),   # lists of 16, every row twice
    (24576, 32, 9, 1024, True, 1.0, False),    # two launches per split
]


@pytest.mark.parametrize("i", range(len(ORDER_CASES)))
def test_sweep_clustered_order(dev, i):
    m, d, k, clusters, excl, scale, dup = ORDER_CASES[i]
    seed = 5000 + i
    say(f"case: clustered-order sweep {i}: m={m} d={d} k={k} clusters={clusters} exclude_self={excl} "
        f"scale={scale} dup={dup}")
    if clusters:
        b = inputs.clustered_bank(seed, 97, m, d, clusters, 0.3, "bf16").emb
    else:
        b = inputs.iid_unit(seed, 97, 0, m, d, "bf16")
    if dup:
        b = np.ascontiguousarray(np.concatenate([b[: m // 2], b[: m - m // 2]]))
    idx, score, prob, lse = pm.mem_build_relations(up(b), k, scale, excl)
    torch.cuda.synchronize()
    g = {"idx": idx.cpu().numpy(), "score": score.cpu().numpy(), "prob": prob.cpu().numpy(),
         "lse": lse.cpu().numpy()}
    # the first and last key of every 64th 256-key tile, the last key, and 64 more
    ends = np.concatenate([np.arange(0, m, 256 * 64), np.arange(255, m, 256 * 64), [m - 1]])
    rows = np.unique(np.concatenate([ends, np.random.default_rng(seed).choice(m, 64, replace=False)]))
    sub = {key: v[rows] for key, v in g.items()}
    r = check_topk(f"order-sweep-{i}", b, b, rows, sub, k, scale, self_idx=np.arange(m) if excl else None)
    say(f"  rows {r['rows']}, bit-exact sets {r['exact_rows']}, max |lse - lse_ref| {r['lse_err_max']:.3g}")
