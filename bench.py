#!/usr/bin/env python3
"""Benchmark of the SRT tree-speculative verification step on one MI355X.

A step is one pass of the whole hot path over one batch: srt_draft (draft
trees from the per-prompt caches) -> srt_tree_attn (tree-masked attention of
every node over its paged context) -> srt_accept (acceptance walk with T=1
Gumbel sampling) -> srt_trie_insert (emitted tokens appended to each
sequence's stream) -> srt_commit (accepted nodes' K/V moved into place,
contexts and draft tails advanced), so consecutive steps form a real decode
loop.  Inputs are resident in HBM before timing starts.

Default workload: the Qwen2.5-7B-shaped layer (256 sequences, 28 query / 4
KV heads, head_dim 128, log-normal contexts with median 4k and max 32k,
64-node draft trees of depth <= 12, vocab 152064), synthetic.

Prints one JSON line: tree tokens verified per second over the step, the
roofline position of the dominant kernel (tree attention; events on its
stream over the timed region) and the CPU oracle timed on a bounded sample.
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

METRIC = "verified draft-tree tokens/sec + tree-attn HBM GB/s (% peak) at 1 GPU"
HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
def counters_path(config_name):
    """Committed rocprofv3 HBM-counter summary of srt_tree_attn on one workload."""
    return os.path.join(ROOT, "profiles", f"tree_attn_{config_name.replace('.', 'p')}_counters.json")
ATTN_SRC = os.path.join(ROOT, "paper_2601_09083_amd", "csrc", "tree_attn.hip")


def attn_work(cfg, ctx_len, n_nodes, tree_depth):
    """Algorithmic bytes and FLOPs of one tree-attention launch: every K/V
    position of every sequence read once (context + tree), Q read once, O
    written once; 4*d FLOPs per (query row, visible key)."""
    n = n_nodes.astype(np.int64)
    L = ctx_len.astype(np.int64)
    d, hq, hkv = cfg.head_dim, cfg.hq, cfg.hkv
    kv_bytes = int(((L + n) * hkv * d * 2 * 2).sum())
    qo_bytes = int((n * hq * d * 2 * 2).sum())
    valid = np.arange(tree_depth.shape[1])[None, :] < n[:, None]
    vis = int((n * L).sum()) + int(np.where(valid, tree_depth.astype(np.int64) + 1, 0).sum())
    flops = 4 * d * hq * vis
    return kv_bytes + qo_bytes, flops


def source_sha(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def counter_traffic(config_name):
    """HBM bytes per launch from committed rocprofv3 counters, if they were
    taken on the current kernel source."""
    path = counters_path(config_name)
    if not os.path.exists(path):
        return None
    try:
        c = json.load(open(path))
        if c.get("source_sha256") != source_sha(ATTN_SRC):
            return None
        return c.get("hbm_bytes_per_launch")
    except Exception:
        return None


ATTN_KERNELS = ("tree_attn_plan_kernel", "tree_attn_kernel<128>", "tree_attn_combine_kernel<128>")


def _short_name(name):
    n = name.replace("(anonymous namespace)::", "").replace("void ", "")
    return n.split("(")[0]


def write_counter_file(d, config_name):
    """HBM traffic per srt_tree_attn launch from four rocprofv3 --pmc runs in
    directory d: pmc_FETCH_SIZE / pmc_WRITE_SIZE of `bench.py --no-cpu-baseline
    --steps 5 --warmup 1` and pmc_copy_* of `bench.py --copy-calibration`.
    Each counter is scaled by what it reads for a 1 GiB device copy.  Only
    the launches of the timed steps are used; their algorithmic bytes come
    from the bench line the same run printed."""
    import csv

    def per_dispatch(sub):
        out = {}
        for r in csv.DictReader(open(os.path.join(d, sub, "run_counter_collection.csv"))):
            out.setdefault(_short_name(r["Kernel_Name"]), []).append(
                (int(r["Dispatch_Id"]), float(r["Counter_Value"])))
        return {k: [v for _, v in sorted(x)] for k, x in out.items()}

    res = {"source_sha256": source_sha(ATTN_SRC),
           "kernel": "srt_tree_attn = " + " + ".join(ATTN_KERNELS) + f" ({config_name} workload)",
           "calibration": {}, "per_kernel_bytes": {}}
    per_launch = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        cp = per_dispatch(f"pmc_copy_{c}").get("__amd_rocclr_copyBuffer", [])
        big = sorted(cp)[-5:]  # the five 1 GiB copies
        kib = float(np.median(big))
        factor = (1 << 30) / 1024.0 / kib
        res["calibration"][c] = {"copy_kib_per_GiB": kib, "factor": factor}
        run = per_dispatch(f"pmc_{c}")
        for k in ATTN_KERNELS:
            vals = run.get(k, [])[-5:]  # launches of the 5 timed steps
            b = float(np.mean(vals)) * 1024.0 * factor if vals else 0.0
            res["per_kernel_bytes"][k] = res["per_kernel_bytes"].get(k, 0.0) + b
            per_launch[c] = per_launch.get(c, 0.0) + b
    res["fetch_bytes_per_launch"] = per_launch["FETCH_SIZE"]
    res["write_bytes_per_launch"] = per_launch["WRITE_SIZE"]
    res["hbm_bytes_per_launch"] = per_launch["FETCH_SIZE"] + per_launch["WRITE_SIZE"]
    line = [l for l in open(os.path.join(d, "pmc_FETCH_SIZE.log")) if l.startswith("{")][-1]
    alg = json.loads(line)["roofline"]["algorithmic_bytes"]
    res["algorithmic_bytes_per_launch"] = alg
    res["traffic_over_algorithmic"] = res["hbm_bytes_per_launch"] / alg
    json.dump(res, open(counters_path(config_name), "w"), indent=1)
    print(json.dumps(res, indent=1))


def host_cores():
    """(CPUs this process may run on, the pool size used): the pool is
    capped at 16, the host-CPU share of one GPU on the measurement boxes."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return n, max(1, min(16, n))


def cpu_baseline(st, tree_np, budget_s: float):
    """The oracle, as it stands, on a bounded sample of the same workload:
    per sequence the draft (from the prompt's stream index), fp64 tree
    attention, the acceptance walk, the online insert and the commit of the
    accepted path.  Timed twice: one thread over sequences in a seeded
    order until ``budget_s`` is spent, then the same work for every
    sequence of the batch on a pool of threads (one sequence per task, the
    fp64 products release the interpreter lock; BLAS kept to one thread per
    task).  ``value`` is the pool's rate; the one-thread rate is kept."""
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    from oracle import accept as AC
    from oracle import attention as AT
    from oracle import commit as CM
    from oracle import draft as DR
    from oracle import trie as TR

    cfg, tw = st.cfg, st.tokens
    tails, ts = tw.ctx_tail(), tw.draft_len()
    order = [int(b) for b in np.random.default_rng(7).permutation(tw.batch)]
    tries = {}
    N = cfg.n_nodes

    def stage(b):
        """Inputs of sequence b in host memory (outside the timed regions)."""
        p = int(tw.seq_prompt[b])
        if p not in tries:
            tries[p] = TR.StreamTrie(tw.streams_of_prompt(p), cfg.trie_depth)
        L = int(tw.ctx_len[b])
        npg = (L + N + cfg.page - 1) // cfg.page
        pages = st.block_table[b, :npg].long()
        return (b, p, L, npg, st.q[b].float().cpu().numpy(), st.k_cache[pages].float().cpu().numpy(),
                st.v_cache[pages].float().cpu().numpy(), st.logits[b].cpu().numpy(),
                st.gumbel[b].cpu().numpy() if st.gumbel is not None else None)

    def one(x):
        b, p, L, npg, q, kc, vc, logits, noise = x
        tok, par, dep, n, qm = DR.draft(tries[p], tails[b], int(ts[b]), cfg.max_match, N, cfg.max_depth)
        AT.tree_attention_seq(q, kc, vc, np.arange(npg), L, par, n, st.scale, cfg.page)
        k, out, nodes = AC.accept(lambda u: logits[u], (lambda s: noise[s]) if noise is not None else None,
                                  1.0, tok, par, n, cfg.max_depth)
        TR.insert_counts({}, tw.seqs[b][-cfg.trie_depth:], out, cfg.trie_depth)
        for cache in (kc, vc):
            CM.commit_kv(AT.gather_positions(cache, np.arange(npg), L + n, cfg.page), L, k, nodes)
        CM.commit_tail(tails[b], int(ts[b]), out)
        return n

    t1, tok1, seqs1 = 0.0, 0, 0
    with threadpool_limits(limits=1):
        for b in order:
            x = stage(b)
            t0 = time.perf_counter()
            tok1 += one(x)
            t1 += time.perf_counter() - t0
            seqs1 += 1
            if t1 >= budget_s:
                break
        nproc, threads = host_cores()
        staged = [stage(b) for b in order]
        t0 = time.perf_counter()
        with ThreadPoolExecutor(threads) as ex:
            tokp = sum(ex.map(one, staged))
        tp = time.perf_counter() - t0
    return {"value": tokp / tp, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"all {tw.batch} sequences of the {cfg.name} workload, one step each (draft + fp64 tree "
                      f"attention + acceptance + insert + commit) on a pool of {threads} threads "
                      f"({nproc} CPUs visible): {tp:.1f} s",
            "host_cpus": nproc,
            "one_thread": {"value": tok1 / t1, "unit": "tokens/s", "cores": 1,
                           "sample": f"{seqs1} of {tw.batch} sequences, {t1:.1f} s on 1 thread"}}


def bulk_build(cfg, tw, reps: int = 2):
    """Set-up bulk build of the per-prompt caches: every prior rollout and
    running sequence inserted into fresh caches by srt_trie_insert, the
    packed token matrices already in device memory.  Timed with events
    around the insert calls; the best of ``reps`` builds."""
    import torch

    from paper_2601_09083_amd import srt
    from paper_2601_09083_amd import workload as W
    from paper_2601_09083_amd.pipeline import Caches, node_capacity_for

    streams, sp = [], []
    for p in range(cfg.n_prompts):
        streams += list(tw.prior[p])
        sp += [p] * len(tw.prior[p])
    streams += list(tw.seqs)
    sp += [int(x) for x in tw.seq_prompt]
    total = int(sum(len(x) for x in streams))
    chunks, i = [], 0
    while i < len(streams):  # the same chunking of the staging matrices as Caches.insert
        j, width = i, 0
        while j < len(streams):
            w = max(width, max(1, len(streams[j])))
            if (j - i + 1) * w > (1 << 26) and j > i:
                break
            width, j = w, j + 1
        mat, lens = W.pack_streams(streams[i:j])
        dev = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device="cuda")
        chunks.append((dev(sp[i:j]), dev(np.arange(i, j)), dev(mat), dev(lens)))
        i = j
    best = None
    for _ in range(reps):
        c = Caches.create(cfg.n_prompts, len(streams) + 1, cfg.trie_depth,
                          node_capacity_for(total, cfg.trie_depth), "cuda")
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for pr, ids, mat, lens in chunks:
            srt.srt_trie_insert(c.ws, pr, ids, mat, lens)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        assert c.status()["flags"] == 0
        best = ms if best is None else min(best, ms)
        del c
    torch.cuda.empty_cache()
    return {"tokens": total, "streams": len(streams), "ms": best, "tokens_per_s": total / (best / 1e3),
            "depth": cfg.trie_depth, "node_updates_per_s": total * cfg.trie_depth / (best / 1e3)}


def full_tree_attention(st, cfg, n, calls: int = 10):
    """srt_tree_attn with every tree forced to n nodes (random parents
    among the 5 preceding nodes, so depths grow like drafted trees) on the
    workload's own contexts and KV cache, timed with events around each of
    ``calls`` launches after one warm-up.  Reported against both rooflines:
    algorithmic bytes (context + tree K/V once, Q, O) and FLOPs (4 d per
    (query row, visible key))."""
    import torch

    from paper_2601_09083_amd import srt

    B, d, hq, hkv = st.tokens.batch, cfg.head_dim, cfg.hq, cfg.hkv
    L = st.tokens.ctx_len.astype(np.int64)
    cap = st.block_table.shape[1] * cfg.page
    if int(L.max()) + n > cap:
        return {"n": n, "skipped": "KV cache has no room for the tree"}
    rng = np.random.default_rng(n)
    par = np.full((B, n), -1, dtype=np.int32)
    depth = np.zeros((B, n), dtype=np.int64)
    for i in range(1, n):
        par[:, i] = rng.integers(np.maximum(0, i - 5), i, size=B) if i > 0 else 0
        depth[:, i] = depth[np.arange(B), par[:, i]] + 1
    dev = st.q.device
    q = torch.randn((B, n, hq, d), device=dev).to(torch.bfloat16)
    out = torch.empty_like(q)
    ctx = torch.as_tensor(st.tokens.ctx_len, device=dev)
    tp = torch.as_tensor(par, device=dev)
    nn = torch.full((B,), n, dtype=torch.int32, device=dev)
    need = srt.srt_tree_attn_scratch_bytes(B, n, hq, hkv, d, cfg.page, st.block_table.shape[1])
    scratch = torch.empty(need, dtype=torch.uint8, device=dev)
    call = lambda: srt.srt_tree_attn(q, st.k_cache, st.v_cache, st.block_table, ctx, tp, nn, st.scale, out=out,
                                     scratch=scratch)
    call()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(calls)]
    for e0, e1 in ev:
        e0.record(stream)
        call()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    nbytes = float(((L + n) * hkv * d * 4).sum() + B * n * hq * d * 4)
    flops = float(4 * d * hq * (n * L.sum() + (depth + 1).sum()))
    tf = flops / (ms / 1e3) / 1e12
    gbps = nbytes / (ms / 1e3) / 1e9
    del q, out, scratch
    torch.cuda.empty_cache()
    bound = "mfma" if flops / (BF16_PEAK_TFLOPS * 1e12) >= nbytes / (HBM_PEAK_GBPS * 1e9) else "hbm"
    return {"n": n, "ms": ms, "TFLOP/s": tf, "mfma_frac": tf / BF16_PEAK_TFLOPS, "GB/s": gbps,
            "hbm_frac": gbps / HBM_PEAK_GBPS, "bound": bound, "flop_per_byte": flops / nbytes,
            "algorithmic_bytes": nbytes, "algorithmic_flops": flops}


FINISH_ROWS = 128  # srt_accept_lmhead finishes the walks in one pass at or below this many subtree nodes


def head_passes(tree, out_nodes, emitted, Dmax):
    """Rows of each product pass srt_accept_lmhead made: level l multiplies
    the current nodes of the sequences still walking, unless the subtrees of
    those nodes (down to depth Dmax) hold at most FINISH_ROWS nodes, in which
    case that one pass covers them all and the walks end there.  Rebuilt
    from the trees and the returned walks (host bookkeeping)."""
    tp, nn = tree["tree_parent"], tree["n_nodes"]
    B, N = tp.shape
    depth = np.full((B, N), -1, dtype=np.int64)
    depth[:, 0] = 0
    for c in range(1, N):
        p = tp[:, c]
        ok = (p >= 0) & (p < c) & (c < nn)
        depth[ok, c] = depth[ok, p[ok]] + 1

    def subtree(b, u):
        n, cnt = int(nn[b]), 0
        for c in range(u, n):
            x = c
            while x > u:
                x = int(tp[b, x])
            cnt += int(x == u and 0 <= depth[b, c] <= Dmax)
        return cnt

    passes = []
    for l in range(int(emitted.max())):
        seqs = np.nonzero(emitted > l)[0]
        cur = [0 if l == 0 else int(out_nodes[b, l - 1]) for b in seqs]
        total = sum(subtree(int(b), u) for b, u in zip(seqs, cur))
        if total <= FINISH_ROWS:
            passes.append(total)
            break
        passes.append(len(seqs))
    return passes


def fused_head(st, cfg, calls: int, unfused: bool):
    """The acceptance walk with the LM head fused in (srt_accept_lmhead) on
    the current trees: synthetic bf16 head [V, d_model] and hidden states
    [B, N, d_model] (d_model = Hq * head_dim, the model width of the
    Qwen2.5 shapes), a node's hidden state planted with its first child's
    head row at the workload's boost rate; the same Gumbel noise.  Timed
    with events around each call; the roofline counts, per product pass,
    the head once plus each row's hidden row and noise row.  With ``unfused`` the LM head over every node (hipBLASLt bf16 GEMM
    to fp32 logits) followed by srt_accept is timed too, for comparison."""
    import torch

    from paper_2601_09083_amd import srt
    from paper_2601_09083_amd import workload as W

    B, N, V, dm = st.tokens.batch, cfg.n_nodes, cfg.vocab, cfg.hq * cfg.head_dim
    tree = {k: v.cpu().numpy() for k, v in st.tree.items()}
    hidden, w = W.make_head(B, N, dm, V, device="cuda", seed=4242, kind="normal", tree_tokens=tree["tree_tokens"],
                            tree_parent=tree["tree_parent"], n_nodes=tree["n_nodes"], plant_p=cfg.boost_p)
    scratch = torch.empty(srt.srt_accept_lmhead_scratch_bytes(B, N, V), dtype=torch.uint8, device="cuda")
    args = (hidden, w, st.gumbel, 1.0, st.tree["tree_tokens"], st.tree["tree_parent"], st.tree["n_nodes"],
            cfg.max_depth)
    out = srt.srt_accept_lmhead(*args, scratch=scratch)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(calls)]
    stream = torch.cuda.current_stream()
    for e0, e1 in ev:
        e0.record(stream)
        srt.srt_accept_lmhead(*args, out=out, scratch=scratch)
        e1.record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    emitted = out["n_emitted"].cpu().numpy().astype(np.int64)
    levels = int(emitted.max())
    walkers = [int((emitted > l).sum()) for l in range(levels)]  # sequences walking at level l
    passes = head_passes(tree, out["out_nodes"].cpu().numpy(), emitted, cfg.max_depth)
    row_bytes = dm * 2 + (V * 4 if st.gumbel is not None else 0)  # hidden row + noise row
    nbytes = sum(V * dm * 2 + rows * row_bytes for rows in passes)  # the head once per pass
    flops = sum(2.0 * rows * dm * V for rows in passes)
    res = {"ms": ms, "d_model": dm, "levels": levels, "walkers_per_level": walkers, "rows_per_pass": passes,
           "mean_emitted": float(emitted.mean()),
           "roofline": {"bound": "hbm", "achieved": nbytes / (ms / 1e3) / 1e9, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                        "frac": nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBPS, "algorithmic_bytes": float(nbytes),
                        "algorithmic_flops": flops, "mfma_tflops": flops / (ms / 1e3) / 1e12}}
    if unfused:
        # the unfused path: LM head over all B*N nodes, then the logits walk
        x = hidden.reshape(B * N, dm)
        wt = w.t().contiguous()
        logits = torch.empty((B, N, V), dtype=torch.float32, device="cuda")
        acc = None
        t = []
        kind = "torch.mm bf16 -> fp32 logits over all B*N nodes + srt_accept"
        try:
            torch.mm(x[:64], wt, out_dtype=torch.float32, out=logits.view(B * N, V)[:64])
            head = lambda: torch.mm(x, wt, out_dtype=torch.float32, out=logits.view(B * N, V))
        except (NotImplementedError, RuntimeError, TypeError):
            kind = "torch.mm bf16 logits over all B*N nodes, converted to fp32, + srt_accept"
            head = lambda: logits.view(B * N, V).copy_(torch.mm(x, wt))
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            head()
            acc = srt.srt_accept(logits, st.gumbel, 1.0, st.tree["tree_tokens"], st.tree["tree_parent"],
                                 st.tree["n_nodes"], cfg.max_depth, out=acc, scratch=st.accept_scratch)
            e1.record(stream)
            t.append((e0, e1))
        torch.cuda.synchronize()
        res["unfused_ms"] = float(np.mean([a.elapsed_time(b) for a, b in t[1:]]))
        res["unfused_kind"] = kind
        same = bool(torch.equal(acc["n_accepted"], out["n_accepted"]))
        res["unfused_same_n_accepted"] = same
        del logits, wt
    del hidden, w, scratch
    torch.cuda.empty_cache()
    return res


def runahead_inserts(cfg, st, sim, n_steps: int):
    """Per-step run-ahead continuations for configurations that insert them
    (the long-tail regime): step k inserts cfg.runahead_streams new streams
    of cfg.runahead_len tokens, stream j a fresh mutation of the next window
    of its sequence's base (sequence j mod B), as run-ahead rollouts that
    generate past the current position would be.  Returns a function that
    performs step k's insertion on the device, or None."""
    import torch

    from paper_2601_09083_amd import srt
    from paper_2601_09083_amd import workload as W

    R, Lr = cfg.runahead_streams, cfg.runahead_len
    if R <= 0 or Lr <= 0:
        return None
    tw = sim.tokens
    B = tw.batch
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(5150 + cfg.index)))
    toks = np.zeros((n_steps, R, Lr), dtype=np.int32)
    lens = np.zeros((n_steps, R), dtype=np.int32)
    prompts = np.array([int(tw.seq_prompt[j % B]) for j in range(R)], dtype=np.int32)
    for k in range(n_steps):
        for j in range(R):
            base = tw.bases[int(prompts[j])]
            start = (int(tw.ctx_len[j % B]) + k * Lr) % max(1, base.shape[0] - Lr)
            r = W.mutate(rng, base[start:start + Lr], vocab=cfg.vocab, p_sub=cfg.p_sub, p_del=cfg.p_del,
                         p_ins=cfg.p_ins)[:Lr]
            toks[k, j, :r.shape[0]] = r
            lens[k, j] = r.shape[0]
    ids = st.caches.new_streams(n_steps * R).reshape(n_steps, R)
    dev = st.attn_len.device
    t_toks = torch.as_tensor(toks, device=dev)
    t_lens = torch.as_tensor(lens, device=dev)
    t_ids = torch.as_tensor(ids, device=dev)
    t_prompts = torch.as_tensor(prompts, device=dev)

    def insert(k):
        srt.srt_trie_insert(st.caches.ws, t_prompts, t_ids[k], t_toks[k], t_lens[k])
    return insert


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="qwen7b")
    ap.add_argument("--greedy", action="store_true", help="greedy acceptance instead of T=1 sampling")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--head-calls", type=int, default=10,
                    help="timed calls of the fused LM-head walk (0: skip it)")
    ap.add_argument("--no-unfused", action="store_true", help="skip timing the unfused LM head + walk")
    ap.add_argument("--no-bulk", action="store_true", help="skip timing the set-up bulk cache build")
    ap.add_argument("--kv-pools", type=int, default=0,
                    help="copies of the KV cache the steps rotate through (0: 3 when the cache fits in the "
                         "256 MB Infinity Cache, else 1)")
    ap.add_argument("--full-tree", default="64,256",
                    help="tree sizes for the full-tree attention pass (every tree forced to that size), "
                         "comma separated; empty to skip")
    ap.add_argument("--part-steps", type=int, default=20,
                    help="steps of the separate pass that times every part with its own events")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (HBM counter calibration)")
    ap.add_argument("--counters-from", metavar="DIR",
                    help="write the attention HBM-traffic file from rocprofv3 --pmc runs in DIR and exit")
    args = ap.parse_args()
    if args.counters_from:
        write_counter_file(args.counters_from, args.config)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this build "
              f"(the path shards per prompt, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2601_09083_amd import simulate as SIM
    from paper_2601_09083_amd import workload as W
    from paper_2601_09083_amd.pipeline import VerifyState

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        n = 1 << 28  # 1 GiB of fp32 read and 1 GiB written per copy
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "copies": 5}), flush=True)
        return
    cfg = W.CONFIGS[args.config]
    t_setup = time.perf_counter()
    n_steps = args.steps + args.warmup + args.part_steps + 4
    # running sequences follow their true continuations (mutated rollouts of
    # their prompt, like every cached rollout); the target logits agree with
    # those continuations, so each step drafts from where the last one left
    sim = SIM.make_sim_tokens(cfg, future_len=(n_steps + 2) * (cfg.max_depth + 1))
    st = VerifyState.build(cfg, tokens=sim.tokens, steps_headroom=n_steps, kv_headroom=n_steps * (cfg.max_depth + 1))
    target = SIM.ContinuationTarget(st, sim.future, sampled=not args.greedy)
    kv_bytes = 2 * st.k_cache.numel() * st.k_cache.element_size()
    n_pools = args.kv_pools if args.kv_pools > 0 else (3 if kv_bytes < 256e6 else 1)
    # rotating copies of the KV cache (same block table and page ids), so a
    # cache smaller than the 256 MB Infinity Cache is not served from it on
    # every step; each step attends to and commits into its own pool
    pools = [(st.k_cache, st.v_cache)] + [(st.k_cache.clone(), st.v_cache.clone()) for _ in range(n_pools - 1)]
    pool_no = [0]

    def next_pool():
        st.k_cache, st.v_cache = pools[pool_no[0] % n_pools]
        pool_no[0] += 1
    torch.cuda.synchronize()
    t_setup = time.perf_counter() - t_setup
    print(f"# setup {t_setup:.1f}s: {cfg.name}, B={st.tokens.batch}", file=sys.stderr, flush=True)
    step_no = [0]

    def draft():
        next_pool()
        st.draft()
        target.apply(st, step_no[0])
        step_no[0] += 1

    def accept():
        st.accept()
        target.advance(st)

    ra_insert = runahead_inserts(cfg, st, sim, n_steps)
    ins_no = [0]

    def insert():
        st.insert()
        if ra_insert is not None:  # run-ahead continuations of this step
            ra_insert(ins_no[0])
            ins_no[0] += 1

    calls = {"draft": draft, "attention": st.attention, "accept": accept, "insert": insert, "commit": st.commit}
    for _ in range(args.warmup):
        for p in ("draft", "attention", "accept", "insert", "commit"):
            calls[p]()
    torch.cuda.synchronize()

    parts = ("draft", "attention", "accept", "insert", "commit")
    stream = torch.cuda.current_stream()
    B = st.tokens.batch
    # per-step record of what each attention launch saw (context lengths
    # and tree sizes / depths), copied on the device after the launch
    rec_len = torch.empty((args.steps, 2, B), dtype=torch.int32, device=st.attn_len.device)
    rec_depth = torch.empty((args.steps, B, cfg.n_nodes), dtype=torch.int32, device=st.attn_len.device)
    rec_emit = torch.empty((args.steps, B), dtype=torch.int32, device=st.attn_len.device)
    # HIP events around every attention launch of the timed region, created
    # beforehand so that the loop only records them (creating events per
    # launch costs more host time than the step's GPU work on a slow host)
    attn_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        draft()
        attn_ev[k][0].record(stream)
        st.attention()
        attn_ev[k][1].record(stream)
        rec_len[k, 0].copy_(st.attn_len)
        rec_len[k, 1].copy_(st.tree["n_nodes"])
        rec_depth[k].copy_(st.tree["tree_depth"])
        accept()
        rec_emit[k].copy_(st.acc["n_emitted"])
        insert()
        st.commit()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    attn_ms = float(np.mean([a.elapsed_time(b) for a, b in attn_ev]))

    # per-part times from a separate, untimed pass with events around every
    # call (the decode loop simply continues)
    part_ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in parts]
               for _ in range(args.part_steps)]
    for k in range(args.part_steps):
        next_pool()
        for j, p in enumerate(parts):
            part_ev[k][j][0].record(stream)
            (insert if p == "insert" else getattr(st, p))()
            part_ev[k][j][1].record(stream)
            if p == "draft":
                target.apply(st, step_no[0])
                step_no[0] += 1
            elif p == "accept":
                target.advance(st)
    torch.cuda.synchronize()
    part_ms = {p: float(np.mean([part_ev[k][j][0].elapsed_time(part_ev[k][j][1]) for k in range(args.part_steps)]))
               for j, p in enumerate(parts)} if args.part_steps > 0 else {}

    rl, rd, re_ = rec_len.cpu().numpy(), rec_depth.cpu().numpy(), rec_emit.cpu().numpy()
    tree_np = {k: v.cpu().numpy() for k, v in st.tree.items()}
    n_tree = int(rl[:, 1].sum())
    n_emit = int(re_.sum())
    ms_step = wall * 1e3 / args.steps
    value = n_tree / args.steps / (ms_step / 1e3)

    work = [attn_work(cfg, rl[k, 0], rl[k, 1], rd[k]) for k in range(args.steps)]
    nbytes = float(np.mean([w[0] for w in work]))
    flops = float(np.mean([w[1] for w in work]))
    t_attn = attn_ms / 1e3
    t_hbm, t_mfma = nbytes / (HBM_PEAK_GBPS * 1e9), flops / (BF16_PEAK_TFLOPS * 1e12)
    if t_mfma >= t_hbm:
        roof = {"bound": "mfma", "achieved": flops / t_attn / 1e12, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": nbytes / t_attn / 1e9, "peak": HBM_PEAK_GBPS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = counter_traffic(cfg.name)
    roof["kernel"] = "srt_tree_attn (tree_attn_plan_kernel + tree_attn_kernel + tree_attn_combine_kernel)"
    roof["algorithmic_bytes"] = nbytes
    roof["algorithmic_flops"] = flops
    roof["launch_ms"] = attn_ms
    attn_hbm = nbytes / t_attn / 1e9

    res = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name}: {st.tokens.batch} sequences, Hq {cfg.hq}/Hkv {cfg.hkv}/d {cfg.head_dim}, "
                         f"contexts {cfg.ctx_len.kind}({cfg.ctx_len.a},{cfg.ctx_len.b}), draft trees N={cfg.n_nodes} "
                         f"Dmax={cfg.max_depth}, vocab {cfg.vocab}, "
                         f"{'greedy' if args.greedy else 'T=1 Gumbel'} acceptance against a target that follows each "
                         f"sequence's continuation, caches of "
                         f"{cfg.rollouts_per_prompt} prior rollouts/prompt"
                         + (f", {cfg.runahead_streams} run-ahead continuations of {cfg.runahead_len} tokens "
                            f"inserted per step" if ra_insert is not None else "")),
            "global_batch": st.tokens.batch,
            "seq_len": int(st.tokens.ctx_len.max()),
            "mean_ctx": float(st.tokens.ctx_len.mean()),
            "parallelism": "none (1 GPU)",
            "kv_pools": n_pools,
        },
        "tree_attn_hbm": {"achieved_GBps": attn_hbm, "peak_GBps": HBM_PEAK_GBPS, "frac": attn_hbm / HBM_PEAK_GBPS},
        "parts_ms": part_ms,
        "parts_steps": args.part_steps,
        "accepted_tokens_per_s": n_emit / args.steps / (ms_step / 1e3),
        "mean_tree_nodes": n_tree / args.steps / B,
        "mean_emitted": n_emit / args.steps / B,
        # sequences still walking at each step of the acceptance walk (mean over timed steps)
        "accept_walkers_per_level": [round(float(np.mean((re_ > lv).sum(axis=1))), 1)
                                     for lv in range(cfg.max_depth + 1)],
        "roofline": roof,
    }
    if args.full_tree:
        res["full_tree"] = [full_tree_attention(st, cfg, int(n)) for n in args.full_tree.split(",") if n]
    if args.head_calls > 0:
        res["fused_head"] = fused_head(st, cfg, args.head_calls, not args.no_unfused)
    if not args.no_bulk:
        bb = bulk_build(cfg, st.tokens)
        res["bulk_insert_tokens_per_s"] = bb["tokens_per_s"]
        res["bulk_build"] = bb
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(st, tree_np, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
