#!/usr/bin/env python3
"""Throughput of dense MemAttention retrieval + chunk gather on one MI355X.

One step = one pass of the hot path over one batch: score 1,024 query
embeddings against a resident bank of 1,048,576 chunk embeddings (d = 1024,
bf16, fp32 accumulation), softmax normaliser and top-32 per query
(mem_retrieve_topk), then gather the 32,768 selected chunks' 128 KiB token
blocks in time order through the page table (mem_gather_chunks).  Inputs are
seeded synthetic data already resident in HBM when timing starts.

Prints one JSON line.  Secondary phases (relation build over 32,768 chunks,
batched retrieval over 262,144 chunks, 64 streaming-append rounds, the tiny
fp32 retrieval, small-batch streaming of the 1M bank, namespace-scoped retrieval over the
1M bank, budget-aware gathers of the main selection, and background block
compaction of a 16 GiB page region, association-aware relocation with the
locality it buys, and the request path as the paper runs it: top-5 within
each request's chunk table, then a time-ordered prompt prefix within a
1,536-token budget) are reported under
"phases" with their own roofline figures; `--only` restricts the run.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15      # dense bf16 MFMA, FLOP/s (MI355X datasheet)
PEAK_HBM = 8.0e12       # HBM3E, B/s
PAGE = 65536
PPC = 2


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_sources_hash() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(os.path.join(ROOT, "paper_2607_05708_amd", "csrc"))):
        with open(os.path.join(ROOT, "paper_2607_05708_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(kernel: str):
    """HBM bytes per launch measured by rocprofv3 counters, if taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    e = t.get(kernel)
    if not e or e.get("sources") != kernel_sources_hash():
        return None
    return e.get("hbm_bytes_per_launch")


class Timer:
    """HIP events on the current stream around repeated calls."""

    def __init__(self, torch):
        self.torch = torch
        self.pairs = []

    def __enter__(self):
        self.a = self.torch.cuda.Event(enable_timing=True)
        self.b = self.torch.cuda.Event(enable_timing=True)
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()
        self.pairs.append((self.a, self.b))

    def mean_ms(self):
        self.torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in self.pairs]))

    def median_min_ms(self):
        self.torch.cuda.synchronize()
        t = [a.elapsed_time(b) for a, b in self.pairs]
        return float(np.median(t)), float(np.min(t))


def up(torch, a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            return next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
    except OSError:
        return ""


def oracle_baseline(q, b, k, rows_full: int, what: str, self_idx=None, scale_rows: float = 1.0) -> dict:
    """The fp64 oracle as it stands, timed on the host cores on a sample of a
    workload's keys: pair-scores/s over the sample, and the whole workload's
    time extrapolated from the per-key time (rows_full keys, each costing
    scale_rows times a sampled key)."""
    import oracle
    threads = min(16, os.cpu_count() or 1)
    oracle.build(force=False)
    t = time.perf_counter()
    oracle.retrieve(q, b, k, threads=threads, self_idx=self_idx)
    el = time.perf_counter() - t
    cand = b.shape[0] - (0 if self_idx is None else 1)
    full_s = el / q.shape[0] * rows_full * scale_rows
    return {"value": q.shape[0] * cand / el, "unit": "pair-scores/s", "cores": threads, "kind": "oracle",
            "sample": f"{q.shape[0]} of {rows_full} keys, {what}; {el:.2f} s",
            "sample_s": el, "full_workload_s": full_s,
            "full_workload_s_kind": "measured" if q.shape[0] == rows_full and scale_rows == 1.0 else "extrapolated",
            "host": {"cpu_model": cpu_model(), "nproc": os.cpu_count()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--only", default="all",
                    help="comma list of: main,relation,batched,stream,tiny,diag,scoped,budget,compact,colocate,request "
                         "(the main "
                         "workload's "
                         "bank is always built; it is timed only when 'main' is listed)")
    ap.add_argument("--stream-rounds", type=int, default=64)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-queries", type=int, default=256)
    ap.add_argument("--calib-copy", action="store_true",
                    help="fewer probe repetitions (the 4 GiB copy probe calibrates counters under rocprofv3)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    phases_on = (set(["main", "relation", "batched", "stream", "tiny", "diag", "scoped", "budget", "compact",
                      "colocate", "request"])
                 if args.only == "all"
                 else set(args.only.split(",")))

    import torch

    import paper_2607_05708_amd as pm
    from paper_2607_05708_amd import inputs

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    pm.lib()  # fails loudly if the library is missing
    dev = torch.device("cuda:0")
    S = args.seed
    phases = {}
    # the probes run once before the phases (cool GPU) and once after them;
    # each rate is the better of the two
    peaks_start = inputs.measured_peaks(torch, reps=3 if args.calib_copy else 5)

    # ------------------------------------------------------------ main workload
    n, d, m, k = 1 << 20, 1024, 1024, 32
    stream_rounds = args.stream_rounds if "stream" in phases_on else 0
    cap = n + 4096 * stream_rounds
    t = time.time()
    cb = inputs.clustered_bank(S, inputs.TAG_GATHER, n, d, 1024, 0.3, "bf16", m_queries=m)
    table_np = inputs.page_layout(S, inputs.TAG_GATHER, cb.cluster, PPC)
    key = inputs.payload_key(S, inputs.TAG_GATHER)
    log(f"generated 1M bank + layout in {time.time() - t:.1f}s")
    emb = torch.empty((cap, d), dtype=torch.bfloat16, device=dev)
    emb[:n] = up(torch, cb.emb)
    bank = emb[:n]
    queries = up(torch, cb.queries)
    table = torch.full((cap, PPC), -1, dtype=torch.int32, device=dev)
    table[:n] = up(torch, table_np)
    n_pages_cap = (n + 4096 * stream_rounds) * PPC
    pool = torch.empty((n * PPC, PAGE), dtype=torch.uint8, device=dev)
    inputs.fill_payload_device(pool, table[:n].contiguous(), key)
    out_blocks = torch.empty((m * k, PPC, PAGE), dtype=torch.uint8, device=dev)
    ws = torch.empty(pm.mem_workspace_bytes(m, n, d, k, pm.MEM_BF16), dtype=torch.uint8, device=dev)
    ids = torch.empty((m, k), dtype=torch.int32, device=dev)
    score = torch.empty((m, k), dtype=torch.float32, device=dev)
    prob = torch.empty((m, k), dtype=torch.float32, device=dev)
    lse = torch.empty((m,), dtype=torch.float32, device=dev)
    tbl_live = table[:n]
    torch.cuda.synchronize()

    t_ret, t_gat = Timer(torch), Timer(torch)

    def step(timed):
        if timed:
            with t_ret:
                pm.mem_retrieve_topk(bank, queries, k, 1.0, out=(ids, score, prob, lse), workspace=ws)
            with t_gat:
                pm.mem_gather_chunks(pool, tbl_live, ids, pm.MEM_ORDER_TIME, k, out=out_blocks)
        else:
            pm.mem_retrieve_topk(bank, queries, k, 1.0, out=(ids, score, prob, lse), workspace=ws)
            pm.mem_gather_chunks(pool, tbl_live, ids, pm.MEM_ORDER_TIME, k, out=out_blocks)

    ms_step = ms_ret = ms_gat = ret_tflops = None
    if "main" in phases_on:
        for _ in range(args.warmup):
            step(False)
        torch.cuda.synchronize()
        log("main: timing")
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step(True)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms_step = wall * 1e3 / args.steps
        ms_ret, ms_gat = t_ret.mean_ms(), t_gat.mean_ms()
        flops = 2.0 * m * n * d
        gather_bytes = 2.0 * m * k * PPC * PAGE
        ret_tflops = flops / (ms_ret * 1e-3) / 1e12
        gat_gbs = gather_bytes / (ms_gat * 1e-3) / 1e9
        # locality statistic |P(R)|: distinct pages and contiguous page runs per query's retrieved set
        ids_np = ids.cpu().numpy()
        pages = table_np[ids_np]                          # [m, k, PPC]
        pr = [np.unique(p.ravel()) for p in pages]
        distinct = float(np.mean([p.shape[0] for p in pr]))
        runs = float(np.mean([1 + int(np.sum(np.diff(p) != 1)) for p in pr]))
        phases["retrieval_gather_1M"] = {
            "retrieve_ms": ms_ret, "gather_ms": ms_gat,
            "retrieve_ms_median_min": t_ret.median_min_ms(), "gather_ms_median_min": t_gat.median_min_ms(),
            "retrieve_tflops": ret_tflops, "retrieve_mfma_frac": ret_tflops * 1e12 / PEAK_BF16,
            "retrieve_bank_hbm_frac": (n * d * 2) / (ms_ret * 1e-3) / PEAK_HBM,
            "gather_GBps": gat_gbs, "gather_hbm_frac": gat_gbs * 1e9 / PEAK_HBM,
            "pages_per_query": distinct, "page_runs_per_query": runs, "blocks_per_query": k,
        }
        log(f"main: step {ms_step:.3f} ms (retrieve {ms_ret:.3f} ms = {ret_tflops:.0f} TFLOP/s, "
            f"gather {ms_gat:.3f} ms = {gat_gbs:.0f} GB/s)")

    def time_call(fn, reps=10, warm=2):
        for _ in range(warm):
            fn()
        tm = Timer(torch)
        for _ in range(reps):
            with tm:
                fn()
        return tm.mean_ms()

    # ------------------------------------------------------------ secondary phases
    if "budget" in phases_on:
        # the prompt prefix: the main selection's chunks within a token budget,
        # time-ordered, as 256-byte token rows (memories of 128..512 tokens)
        if ms_ret is None:
            pm.mem_retrieve_topk(bank, queries, k, 1.0, out=(ids, score, prob, lse), workspace=ws)
        tok = up(torch, inputs.token_lengths(S, inputs.TAG_GATHER, n, 128, 512))
        for budget in (512, 1536, 3072):
            rows = torch.empty((m, budget, 256), dtype=torch.uint8, device=dev)
            btok = torch.empty((m,), dtype=torch.int32, device=dev)
            bkept = torch.empty((m, k), dtype=torch.int32, device=dev)
            ms = time_call(lambda: pm.mem_gather_budget(pool, tbl_live, tok, ids, budget, 256,
                                                        out=(rows, btok, bkept)))
            moved = float(btok.sum().item()) * 256 + m * budget * 256.0   # rows read + rows written
            phases[f"budget_gather_{budget}"] = {"ms": ms, "GBps": moved / (ms * 1e-3) / 1e9,
                                                 "hbm_frac": moved / (ms * 1e-3) / PEAK_HBM,
                                                 "tokens_per_key": float(btok.float().mean().item())}
            del rows
        del tok
    if "compact" in phases_on:
        # 4,096 written blocks of 64 pages of 64 KiB (16 GiB), uniform live
        # shares per block, 20 % of chunks relocated earlier, 256 namespaces
        # (runs of 64 chunks), 10 % of chunks deleted
        P_c, nb_c = 64, 4096
        ctab, cnf = inputs.compaction_layout(S, 83, nb_c, P_c, PPC)
        crns, clive, _ = inputs.namespaces(S, 83, ctab.shape[0], 256, 0.1, run=64)
        coffs, cchunks = inputs.chunk_tables(inputs.scoped_row_ns(crns, clive))
        cpool = torch.empty((cnf + cnf * 3 // 4, PAGE), dtype=torch.uint8, device=dev)
        ctab0, ctab_w = up(torch, ctab), up(torch, ctab)
        coffs_t, cch_t = up(torch, coffs), up(torch, cchunks)
        cws = torch.empty(pm.mem_compact_workspace_bytes(cnf, P_c, cchunks.shape[0], PPC, coffs.shape[0] - 1),
                          dtype=torch.uint8, device=dev)
        for theta in (0.75, 0.3):
            tms, res = [], None
            for rep in range(6):
                ctab_w.copy_(ctab0)
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                res, _, _ = pm.mem_compact_blocks(cpool, ctab_w, coffs_t, cch_t, P_c, theta, cnf, workspace=cws)
                b.record()
                torch.cuda.synchronize()
                if rep >= 1:
                    tms.append(a.elapsed_time(b))
            ms = float(np.mean(tms))
            moved_bytes = 2.0 * res["moved_pages"] * PAGE
            phases[f"compact_16GiB_theta{theta}"] = {
                "ms": ms, "moved_pages": res["moved_pages"], "released_blocks": res["released_blocks"],
                "GBps": moved_bytes / (ms * 1e-3) / 1e9, "hbm_frac": moved_bytes / (ms * 1e-3) / PEAK_HBM}
        del cpool, cws
    if "colocate" in phases_on:
        # 262,144 clustered chunks in append order (chunk c at pages 2c, 2c+1),
        # 1,024 queries, top-32; each query's chunks scoring >= tau are
        # rewritten together; the same trace is replayed to count the 4 MiB
        # blocks and page runs each request touches before and after
        n_l, m_l, k_l, P_l = 262144, 1024, 32, 64
        cl = inputs.clustered_bank(S, 85, n_l, d, 1024, 0.3, "bf16", m_queries=m_l)
        bank_l, q_l = up(torch, cl.emb), up(torch, cl.queries)
        tab0 = up(torch, inputs.identity_layout(n_l, PPC))
        tab_w = tab0.clone()
        pool_l = torch.empty((n_l * PPC + m_l * k_l * PPC, PAGE), dtype=torch.uint8, device=dev)
        ids_l, sc_l, _, _ = pm.mem_retrieve_topk(bank_l, q_l, k_l, 1.0)
        wsl = torch.empty(pm.mem_colocate_workspace_bytes(m_l, k_l, n_l), dtype=torch.uint8, device=dev)

        def locality(tab):
            pages = np.sort(tab.cpu().numpy()[ids_l.cpu().numpy()].reshape(m_l, -1), axis=1)
            blocks = np.mean([np.unique(p // P_l).size for p in pages])
            runs = np.mean([1 + int(np.sum(np.diff(p) != 1)) for p in pages])
            return float(blocks), float(runs)

        b0, r0 = locality(tab0)
        for tau in (0.7, 0.9):
            tms, res = [], None
            for rep in range(6):
                tab_w.copy_(tab0)
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                res = pm.mem_colocate(pool_l, tab_w, ids_l, sc_l, tau, 2, n_l * PPC, workspace=wsl)
                b.record()
                torch.cuda.synchronize()
                if rep >= 1:
                    tms.append(a.elapsed_time(b))
            ms = float(np.mean(tms))
            moved_bytes = 2.0 * res["moved_chunks"] * PPC * PAGE
            b1, r1 = locality(tab_w)
            phases[f"colocate_262k_tau{tau}"] = {
                "ms": ms, "moved_chunks": res["moved_chunks"], "groups": res["groups"],
                "GBps": moved_bytes / (ms * 1e-3) / 1e9, "hbm_frac": moved_bytes / (ms * 1e-3) / PEAK_HBM,
                "blocks_per_request_before": b0, "blocks_per_request_after": b1,
                "page_runs_per_request_before": r0, "page_runs_per_request_after": r1}
        del bank_l, q_l, pool_l, wsl
    if "request" in phases_on:
        # Algorithm 1's retrieval branch for 1,024 concurrent requests: top-5
        # (the paper's default p) of the request's own (user, session) chunk
        # table, then FetchByID + SortByTime + Concat within 1,536 tokens
        rns, live, kns = inputs.namespaces(S, inputs.TAG_GATHER, n, 256, 0.1, run=64, query_src=cb.query_src)
        offs, chs = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
        offs_t, chs_t, qns = up(torch, offs), up(torch, chs), up(torch, kns)
        kp, budget = 5, 1536
        wsr = torch.empty(pm.mem_workspace_bytes_grouped(m, offs.shape[0] - 1, chs.shape[0], d, kp),
                          dtype=torch.uint8, device=dev)
        outr = (torch.empty((m, kp), dtype=torch.int32, device=dev), torch.empty((m, kp), device=dev),
                torch.empty((m, kp), device=dev), torch.empty(m, device=dev))
        tok = up(torch, inputs.token_lengths(S, inputs.TAG_GATHER, n, 128, 512))
        rows = torch.empty((m, budget, 256), dtype=torch.uint8, device=dev)
        rtok = torch.empty((m,), dtype=torch.int32, device=dev)
        rkept = torch.empty((m, kp), dtype=torch.int32, device=dev)
        t_sel, t_pre = Timer(torch), Timer(torch)

        def request_batch():
            with t_sel:
                pm.mem_retrieve_topk_grouped(bank, offs_t, chs_t, queries, qns, kp, 1.0, out=outr, workspace=wsr)
            with t_pre:
                pm.mem_gather_budget(pool, tbl_live, tok, outr[0], budget, 256, out=(rows, rtok, rkept))
        for _ in range(2):
            request_batch()
        t_sel.pairs.clear()
        t_pre.pairs.clear()
        torch.cuda.synchronize()
        t0r = time.perf_counter()
        for _ in range(10):
            request_batch()
        torch.cuda.synchronize()
        ms_b = (time.perf_counter() - t0r) * 1e3 / 10
        phases["request_path_1M"] = {
            "requests": m, "top_p": kp, "budget_tokens": budget, "batch_ms": ms_b,
            "requests_per_s": m / (ms_b * 1e-3), "select_ms": t_sel.mean_ms(), "prefix_ms": t_pre.mean_ms(),
            "prefix_tokens_per_request": float(rtok.float().mean().item()),
            "chunks_per_request": float((rkept >= 0).sum().item()) / m}
        del wsr, rows, tok
    if "scoped" in phases_on:
        # the main workload's bank and queries, split into 256 (user, session)
        # namespaces with 10% of rows tombstoned; each query searches its
        # source row's namespace.  "runs": sessions append in bursts (mean 64
        # rows); "mixed": every row draws its own namespace.
        qns = None
        for label, run in (("runs", 64), ("mixed", 1)):
            rns, live, kns = inputs.namespaces(S, inputs.TAG_GATHER, n, 256, 0.1, run=run, query_src=cb.query_src)
            rn_t = up(torch, inputs.scoped_row_ns(rns, live))
            qns = up(torch, kns)
            ms = time_call(lambda: pm.mem_retrieve_topk_scoped(bank, rn_t, queries, qns, k, 1.0,
                                                               out=(ids, score, prob, lse), workspace=ws))
            fl = 2.0 * m * n * d
            phases[f"scoped_retrieval_1M_{label}"] = {
                "ms": ms, "tflops": fl / (ms * 1e-3) / 1e12, "mfma_frac": fl / (ms * 1e-3) / PEAK_BF16,
                "namespaces": 256, "mean_run_rows": run, "tombstoned_frac": 0.1,
                "vs_unscoped": (ms_ret / ms) if ms_ret else None}
            # the same selection over per-namespace chunk tables
            offs, chs = inputs.chunk_tables(inputs.scoped_row_ns(rns, live))
            offs_t, chs_t = up(torch, offs), up(torch, chs)
            wsg = torch.empty(pm.mem_workspace_bytes_grouped(m, offs.shape[0] - 1, chs.shape[0], d, k),
                              dtype=torch.uint8, device=dev)
            msg = time_call(lambda: pm.mem_retrieve_topk_grouped(bank, offs_t, chs_t, queries, qns, k, 1.0,
                                                                  out=(ids, score, prob, lse), workspace=wsg))
            # work done: each query against its own table
            cnt = np.bincount(kns, minlength=offs.shape[0] - 1)
            pairs = float(np.sum(cnt * np.diff(offs)))
            phases[f"grouped_retrieval_1M_{label}"] = {
                "ms": msg, "scored_pairs": pairs, "pair_scores_per_s": pairs / (msg * 1e-3),
                "bank_GBps_once": float(chs.shape[0]) * d * 2 / (msg * 1e-3) / 1e9,
                "vs_scoped_dense": ms / msg}
            del rn_t, offs_t, chs_t, wsg
    if "diag" in phases_on:
        for mm in (16, 64, 128):
            qd = queries[:mm]
            wsd = torch.empty(pm.mem_workspace_bytes(mm, n, d, k, pm.MEM_BF16), dtype=torch.uint8, device=dev)
            ms = time_call(lambda: pm.mem_retrieve_topk(bank, qd, k, 1.0, workspace=wsd))
            phases[f"stream_bank_m{mm}"] = {"ms": ms, "bank_GBps": n * d * 2 / (ms * 1e-3) / 1e9,
                                           "hbm_frac": n * d * 2 / (ms * 1e-3) / PEAK_HBM}
    if "relation" in phases_on:
        cr = inputs.clustered_bank(S, inputs.TAG_RELATION, 32768, 768, 256, 0.3, "bf16")
        rb = up(torch, cr.emb)
        wsr = torch.empty(pm.mem_workspace_bytes(32768, 32768, 768, 32, pm.MEM_BF16), dtype=torch.uint8, device=dev)
        ms = time_call(lambda: pm.mem_build_relations(rb, 32, 1.0, True, workspace=wsr))
        fl = 2.0 * 32768 * 32768 * 768
        phases["relation_build_32k"] = {"ms": ms, "pair_scores_per_s": 32768 * 32767 / (ms * 1e-3),
                                        "tflops": fl / (ms * 1e-3) / 1e12, "mfma_frac": fl / (ms * 1e-3) / PEAK_BF16}
        del rb, wsr
        if not args.no_cpu:
            nk = 512
            phases["relation_build_32k"]["cpu_baseline"] = oracle_baseline(
                cr.emb[:nk], cr.emb, 32, 32768, "each against the whole 32,768-chunk bank, self excluded (fp64 "
                "scores, softmax, top-32)", self_idx=np.arange(nk))
            log(f"relation: oracle {phases['relation_build_32k']['cpu_baseline']['sample']}")
    if "batched" in phases_on:
        c3 = inputs.clustered_bank(S, inputs.TAG_BATCHED, 262144, 1024, 1024, 0.3, "bf16", m_queries=512)
        b3, q3 = up(torch, c3.emb), up(torch, c3.queries)
        ws3 = torch.empty(pm.mem_workspace_bytes(512, 262144, 1024, 16, pm.MEM_BF16), dtype=torch.uint8, device=dev)
        ms = time_call(lambda: pm.mem_retrieve_topk(b3, q3, 16, 1.0, workspace=ws3))
        fl = 2.0 * 512 * 262144 * 1024
        phases["batched_retrieval_262k"] = {"ms": ms, "pair_scores_per_s": 512 * 262144 / (ms * 1e-3),
                                            "retrievals_per_s": 512 / (ms * 1e-3), "tflops": fl / (ms * 1e-3) / 1e12,
                                            "mfma_frac": fl / (ms * 1e-3) / PEAK_BF16,
                                            "bank_hbm_frac": 262144 * 1024 * 2 / (ms * 1e-3) / PEAK_HBM}
        del b3, q3, ws3
        if not args.no_cpu:
            phases["batched_retrieval_262k"]["cpu_baseline"] = oracle_baseline(
                c3.queries[:64], c3.emb, 16, 512, "each against the whole 262,144-chunk bank (fp64 scores, softmax, "
                "top-16)")
            log(f"batched: oracle {phases['batched_retrieval_262k']['cpu_baseline']['sample']}")
    if "tiny" in phases_on:
        bt = up(torch, inputs.iid_unit(S, inputs.TAG_TINY, 2, 1024, 256, "f32"))
        qt = up(torch, inputs.iid_unit(S, inputs.TAG_TINY, 4, 16, 256, "f32"))
        wst = torch.empty(pm.mem_workspace_bytes(16, 1024, 256, 8, pm.MEM_F32), dtype=torch.uint8, device=dev)
        fp = torch.empty((16, 1024), dtype=torch.float32, device=dev)
        outt = (torch.empty((16, 8), dtype=torch.int32, device=dev), torch.empty((16, 8), device=dev),
                torch.empty((16, 8), device=dev), torch.empty(16, device=dev))
        call = lambda: pm.mem_retrieve_topk(bt, qt, 8, 1.0, out=outt, full_prob=fp, workspace=wst)  # noqa: E731
        ms = time_call(call, reps=50)
        # the same call captured once in a HIP graph and replayed: its
        # kernels are launched without host round trips
        graph = torch.cuda.CUDAGraph()
        call()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            call()
        ms_g = time_call(graph.replay, reps=50)
        phases["tiny_retrieval_fp32"] = {"latency_us": ms * 1e3, "pair_scores_per_s": 16384 / (ms * 1e-3),
                                         "graph_replay_latency_us": ms_g * 1e3}
        if not args.no_cpu:
            qt_h = inputs.iid_unit(S, inputs.TAG_TINY, 4, 16, 256, "f32")
            bt_h = inputs.iid_unit(S, inputs.TAG_TINY, 2, 1024, 256, "f32")
            oracle_baseline(qt_h, bt_h, 8, 16, "warm-up")
            runs = [oracle_baseline(qt_h, bt_h, 8, 16, "all 16 queries against the 1,024-row fp32 bank (fp64 "
                                    "scores, softmax, top-8)") for _ in range(5)]
            phases["tiny_retrieval_fp32"]["cpu_baseline"] = min(runs, key=lambda r: r["sample_s"])
    if stream_rounds:
        st = pm.BankState(emb, n, table, n * PPC, n_pages_cap)
        ms_rounds, total_fl = [], 0.0
        new_all = [up(torch, inputs.appended_chunks(S, inputs.TAG_STREAM, r, 4096, cb.centroids, 0.3))
                   for r in range(stream_rounds)]
        wss = torch.empty(pm.mem_workspace_bytes(4096, cap, d, 32, pm.MEM_BF16), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        tm_ret, tm_app = Timer(torch), Timer(torch)
        t0 = time.perf_counter()
        for r in range(stream_rounds):
            nr = st.n
            with tm_ret:
                pm.mem_retrieve_topk(st.live, new_all[r], 32, 1.0, workspace=wss)
            with tm_app:
                pm.mem_append_chunks(st, new_all[r])
            total_fl += 2.0 * 4096 * nr * d
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t0
        ms_r = tm_ret.mean_ms()
        phases["streaming_append_64x4096"] = {
            "rounds": stream_rounds, "total_ms": wall_s * 1e3, "rounds_per_s": stream_rounds / wall_s,
            "retrieve_ms_mean": ms_r, "append_ms_mean": tm_app.mean_ms(),
            "tflops": total_fl / wall_s / 1e12, "mfma_frac": total_fl / wall_s / PEAK_BF16,
            "pair_scores_per_s": total_fl / (2 * d) / wall_s}
        del new_all, wss
        if not args.no_cpu:
            # round 0's first 32 new chunks against the 1,048,576-row bank;
            # the 64 rounds' time extrapolated from the per-key time, scaled
            # by each round's bank size (n + 4,096 r rows)
            new0 = inputs.appended_chunks(S, inputs.TAG_STREAM, 0, 32, cb.centroids, 0.3)
            grow = sum(n + 4096 * r for r in range(stream_rounds)) / (n * stream_rounds)
            phases["streaming_append_64x4096"]["cpu_baseline"] = oracle_baseline(
                new0, cb.emb, 32, 4096 * stream_rounds, f"round 0's first 32 new chunks against the 1,048,576-chunk "
                f"bank (fp64 scores, softmax, top-32); the {stream_rounds} rounds extrapolated per key and bank size",
                scale_rows=grow)
            log(f"stream: oracle {phases['streaming_append_64x4096']['cpu_baseline']['sample']}")

    # rates this GPU sustains on plain probe kernels (context for the fractions;
    # the copy probe is also the known-size kernel that calibrates the
    # rocprofv3 byte counters)
    peaks_end = inputs.measured_peaks(torch, reps=3 if args.calib_copy else 5)
    peaks = dict(peaks_end)
    for key in ("hbm_copy_GBps", "mfma_bf16_TFLOPs"):
        peaks[key] = max(peaks_start[key], peaks_end[key])
        peaks[key + "_before_after"] = [peaks_start[key], peaks_end[key]]
    if "retrieval_gather_1M" in phases:
        ph = phases["retrieval_gather_1M"]
        ph["retrieve_frac_of_mfma_probe"] = ph["retrieve_tflops"] / peaks["mfma_bf16_TFLOPs"]
        ph["gather_frac_of_copy_probe"] = ph["gather_GBps"] / peaks["hbm_copy_GBps"]
    for name, ph in phases.items():
        if name.startswith(("budget_gather_", "compact_", "colocate_")):
            ph["frac_of_copy_probe"] = ph["GBps"] / peaks["hbm_copy_GBps"]
    log(f"probes: copy {peaks['hbm_copy_GBps']:.0f} GB/s, mfma {peaks['mfma_bf16_TFLOPs']:.0f} TFLOP/s")

    if ms_step is None:  # profiling runs of single phases
        print(json.dumps({"metric": "bank pair-scores/s + top-k retrievals/s; % MFMA peak and % HBM peak on 1 MI355X",
                          "value": None, "note": "main workload not run (--only)", "phases": phases,
                          "measured_peaks": peaks}), flush=True)
        return

    # ------------------------------------------------------------ CPU oracle baseline
    cpu = None
    if not args.no_cpu:
        nq = args.cpu_queries
        cpu = oracle_baseline(cb.queries[:nq], cb.emb, k, m, "each against the full 1,048,576-chunk bank (fp64 "
                              "scores, softmax, top-32)")
        phases["retrieval_gather_1M"]["cpu_baseline"] = cpu
        log(f"cpu oracle: {cpu['sample']} on {cpu['cores']} threads")

    pair_scores_per_s = m * n / (ms_step * 1e-3)
    traffic = traffic_from_profile("mem_retrieve_topk")
    result = {
        "metric": "bank pair-scores/s + top-k retrievals/s; % MFMA peak and % HBM peak on 1 MI355X",
        "value": pair_scores_per_s,
        "unit": "pair-scores/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "retrievals_per_s": m / (ms_step * 1e-3),
        "config": {"workload": "retrieval + gather: bank 1,048,576 x 1024 bf16 (1,024-cluster mixture), "
                               "1,024 queries, top-32, gather 32,768 blocks of 128 KiB through 64 KiB pages "
                               "in time order", "bank_rows": n, "dim": d, "queries": m, "k": k,
                   "page_bytes": PAGE, "pages_per_chunk": PPC},
        "roofline": {"kernel": "mem_retrieve_topk: threshold sample pass + k-th search + matrix-core full pass "
                               "(two launches with the k-th-best bound search between them) + merge (one call, "
                               "HIP events on its stream)", "bound": "mfma",
                     "achieved": ret_tflops, "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                     "frac": ret_tflops * 1e12 / PEAK_BF16, "traffic": traffic},
        "cpu_baseline": cpu,
        "measured_peaks": peaks,
        "phases": phases,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
