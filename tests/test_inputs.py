"""Seeded input generators: conversions, layouts and payload (no method arithmetic)."""
import json
import os

import numpy as np
import torch

import oracle
from paper_2607_05708_amd import inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32),
                        # exact halfway cases between two bf16 neighbours
                        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8)], np.float32)])
    ours = inputs.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(inputs.bf16_bits_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_page_layout_is_bijection_with_runs():
    rng = np.random.default_rng(1)
    cl = rng.integers(0, 16, size=3000)
    table = inputs.page_layout(0, 99, cl, 2)
    assert table.shape == (3000, 2)
    assert np.array_equal(np.sort(table.ravel()), np.arange(6000))
    # each cluster has at least floor(0.8 * size) chunks whose two pages are adjacent
    # and that sit in one contiguous run in ascending id order
    for c in range(16):
        members = np.nonzero(cl == c)[0]
        adjacent = members[table[members, 1] == table[members, 0] + 1]
        assert adjacent.shape[0] >= int(np.floor(0.8 * members.shape[0]))
    # deterministic
    assert np.array_equal(table, inputs.page_layout(0, 99, cl, 2))


def test_clustered_rows_are_unit_and_reproducible():
    b1 = inputs.clustered_bank(0, 77, 5000, 64, 8, 0.3, "bf16", m_queries=10)
    b2 = inputs.clustered_bank(0, 77, 5000, 64, 8, 0.3, "bf16", m_queries=10, threads=1)
    assert np.array_equal(b1.emb, b2.emb) and np.array_equal(b1.queries, b2.queries)
    norms = np.linalg.norm(inputs.bf16_bits_to_f32(b1.emb).astype(np.float64), axis=1)
    assert np.all(np.abs(norms - 1) < 4e-3)
    # a perturbed query is closest to members of its source row's cluster
    s = inputs.bf16_bits_to_f32(b1.queries).astype(np.float64) @ inputs.bf16_bits_to_f32(b1.emb).astype(np.float64).T
    assert np.mean(b1.cluster[np.argmax(s, axis=1)] == b1.cluster[b1.query_src]) >= 0.9


def test_host_pool_holds_payload_at_table_pages():
    table = inputs.page_layout(3, 98, np.arange(20) % 3, 2)
    key = inputs.payload_key(3, 98)
    pool = inputs.host_pool(key, table, 512)
    for c in (0, 7, 19):
        for p in (0, 1):
            assert np.array_equal(pool[table[c, p]].view(np.uint64), oracle.payload_page(key, c, p, 2, 512))


def test_golden_tiny_retrieval_reproduces():
    """Regression: the oracle's answer on the tiny fp32 workload is unchanged."""
    with open(os.path.join(GOLDEN, "tiny_retrieval_seed0.json")) as f:
        g = json.load(f)
    bank = inputs.iid_unit(0, inputs.TAG_TINY, 2, 1024, 256, "f32")
    q = inputs.iid_unit(0, inputs.TAG_TINY, 4, 16, 256, "f32")
    r = oracle.retrieve(q, bank, k=8)
    assert r["idx"].tolist() == g["idx"]
    assert [[float.hex(float(x)) for x in row] for row in r["score"]] == g["score"]
    assert [float.hex(float(x)) for x in r["lse"]] == g["lse"]
