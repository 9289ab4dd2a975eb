"""The allocation-free retrieval (mem_retrieve_topk_noalloc) against the
workspace call it varies, through the C ABI: the same kernels on the
library's fixed scratch array must give the same results, call after call,
whatever an earlier call left in that array."""
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


def garbage_out(m, k):
    # outputs start as garbage so that every value compared was written by the call
    return (torch.full((m, k), 12345, dtype=torch.int32, device="cuda"),
            torch.full((m, k), 7.0, device="cuda"), torch.full((m, k), 7.0, device="cuda"),
            torch.full((m,), 7.0, device="cuda"))


def host(out):
    torch.cuda.synchronize()
    return {n: t.cpu().numpy() for n, t in zip(("idx", "score", "prob", "lse"), out)}


def compare(name, bank_np, q_np, k, scale, full=False):
    bank, q = up(bank_np), up(q_np)
    m, n = q_np.shape[0], bank_np.shape[0]
    say(f"case: {name}: {m} queries x {n} rows, d {q_np.shape[1]}, k {k}, "
        f"{'fp32 + full probabilities' if full else 'bf16'}")
    fp_a = torch.full((m, n), 7.0, device="cuda") if full else None
    fp_b = torch.full((m, n), 7.0, device="cuda") if full else None
    a = host(pm.mem_retrieve_topk_noalloc(bank, q, k, scale, out=garbage_out(m, k), full_prob=fp_a))
    b = host(pm.mem_retrieve_topk(bank, q, k, scale, out=garbage_out(m, k), full_prob=fp_b))
    # the same kernels on the same inputs: identical results
    for key in ("idx", "score", "prob", "lse"):
        assert np.array_equal(a[key], b[key]), f"{name}: {key} differs from the workspace call"
    if full:
        assert torch.equal(fp_a, fp_b), f"{name}: full probabilities differ"
    # and both meet the oracle's parity rules
    rows = np.unique(np.concatenate([np.random.default_rng(m).choice(m, min(m, 24), replace=False), [0, m - 1]]))
    check_topk(name, q_np, bank_np, rows, {key: v[rows] for key, v in a.items()}, k, scale)


def test_noalloc_matches_the_workspace_call_on_successive_calls(dev):
    assert pm.mem_scratch_bytes() == 128 << 20
    # 1: 1,024 queries (four 256-query tiles, threshold sample): about 97 MiB
    #    of the 128 MiB scratch
    c1 = inputs.clustered_bank(11, 97, 65536, 256, 64, 0.3, "bf16", m_queries=1024)
    assert pm.mem_workspace_bytes(1024, 65536, 256, 32, pm.MEM_BF16) > 90 << 20
    compare("noalloc-1024x65536", c1.emb, c1.queries, 32, 1.0)
    # 2: a smaller call right after it (narrow 64-query shape, lists of 8,
    #    ragged bank tail) on the array the first call left behind
    c2 = inputs.clustered_bank(12, 97, 5001, 256, 16, 0.3, "bf16", m_queries=40)
    compare("noalloc-40x5001", c2.emb, c2.queries, 8, 2.0)
    # 3: smaller again, the fp32 path with full probabilities
    b3 = inputs.iid_unit(13, 97, 0, 1024, 128, "f32")
    q3 = inputs.iid_unit(13, 97, 4, 16, 128, "f32")
    compare("noalloc-16x1024-fp32", b3, q3, 8, 1.0, full=True)


def test_noalloc_refuses_a_call_beyond_the_scratch(dev):
    # 4,096 queries against 1,310,720 rows need about 161 MiB of workspace:
    # refused on the host, nothing launched, outputs untouched
    n, d, m, k = 1310720, 1024, 4096, 32
    bank = torch.zeros((n, d), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((m, d), dtype=torch.bfloat16, device="cuda")
    out = garbage_out(m, k)
    with pytest.raises(pm.MemError, match="allocation-free"):
        pm.mem_retrieve_topk_noalloc(bank, q, k, 1.0, out=out)
    torch.cuda.synchronize()
    assert int(out[0][0, 0]) == 12345
