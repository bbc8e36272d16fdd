"""Helpers for the GPU parity tests: oracle evaluations on the same inputs the
HIP path receives, and the comparison rules (bit-exact for cache contents,
trees and acceptance; |gpu - ref| <= 1e-2 + 2e-2 |ref| for attention)."""
from __future__ import annotations

import json
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

from oracle import accept as AC
from oracle import attention as AT
from oracle import draft as DR
from oracle import trie as TR

ATOL, RTOL = 1e-2, 2e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_trie(streams, D, big=False):
    return TR.StreamTrie(streams, D) if big else TR.DictTrie(TR.substring_counts(streams, D), D)


def oracle_draft_rows(state, tries, seqs, alpha=0.0):
    """Oracle draft for the sequences ``seqs`` of a VerifyState."""
    c = state.cfg
    tails = state.tokens.ctx_tail()
    ts = state.tokens.draft_len()
    out = {}
    for b in seqs:
        p = int(state.tokens.seq_prompt[b])
        out[b] = DR.draft(tries[p], tails[b], int(ts[b]), c.max_match, c.n_nodes, c.max_depth, alpha)
    return out


def tree_rows(tree, b):
    n = int(tree["n_nodes"][b])
    tt = tree["tree_tokens"][b].tolist()
    return (tt[:n], tree["tree_parent"][b].tolist()[:n], tree["tree_depth"][b].tolist()[:n], n,
            int(tree["match_len"][b])), tt[n:], tree["tree_parent"][b].tolist()[n:]


def assert_tree_equal(gpu_tree_np, b, want):
    got, pad_t, pad_p = tree_rows(gpu_tree_np, b)
    assert got == tuple(want), f"seq {b}: gpu {got} != oracle {want}"
    assert all(x == -1 for x in pad_t) and all(x == -1 for x in pad_p)


def tree_to_np(tree):
    return {k: v.cpu().numpy() for k, v in tree.items()}


def oracle_attention_seq(state, b, tree_parent_row, n):
    """fp64 oracle output [n, Hq, d] for sequence b (pages gathered from the
    same device buffers the kernel reads)."""
    c = state.cfg
    L = int(state.tokens.ctx_len[b])
    npg = (L + n + c.page - 1) // c.page
    pages = state.block_table[b, :npg].long()
    kc = state.k_cache[pages].float().cpu().numpy()
    vc = state.v_cache[pages].float().cpu().numpy()
    q = state.q[b, :n].float().cpu().numpy()
    return AT.tree_attention_seq(q, kc, vc, np.arange(npg), L, tree_parent_row, n, state.scale, c.page)


def assert_attn_close(gpu, ref, what=""):
    """Element-wise |gpu - ref| <= ATOL + RTOL |ref|.  Returns (max abs
    error, max relative error over elements with |ref| >= 1e-3, largest
    fraction of the tolerance used)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - ref)
    bound = ATOL + RTOL * np.abs(ref)
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance; "
                           f"max abs err {err.max():.3e}, worst excess {(err - bound).max():.3e}")
    if err.size == 0:
        return 0.0, 0.0, 0.0
    big = np.abs(ref) >= 1e-3
    rel = float((err[big] / np.abs(ref[big])).max()) if big.any() else 0.0
    return float(err.max()), rel, float((err / bound).max())


class ErrorLog:
    """Largest attention errors of one test case, printed when the case
    ends and appended as one JSON line to $SRT_ATTN_ERRLOG if that is set."""

    def __init__(self, label):
        self.label, self.abs, self.rel, self.frac, self.rows = label, 0.0, 0.0, 0.0, 0

    def add(self, gpu, ref, what=""):
        a, r, f = assert_attn_close(gpu, ref, f"{self.label} {what}")
        self.abs, self.rel, self.frac = max(self.abs, a), max(self.rel, r), max(self.frac, f)
        self.rows += int(np.asarray(ref).shape[0])
        return a

    def done(self):
        rec = {"case": self.label, "rows": self.rows, "max_abs": self.abs, "max_rel": self.rel,
               "max_frac_of_tol": self.frac}
        say(f"attn error {self.label}: rows {self.rows}, max abs {self.abs:.3e}, max rel (|ref|>=1e-3) "
            f"{self.rel:.3e}, max fraction of tolerance {self.frac:.3f}")
        path = os.environ.get("SRT_ATTN_ERRLOG")
        if path:
            with open(path, "a") as f:
                f.write(json.dumps(rec) + "\n")
        return rec


def oracle_attention_many(state, seqs, parents, n_nodes, threads=None):
    """{b: fp64 oracle output [n_b, Hq, d]} for many sequences, evaluated
    in a thread pool (the fp64 products release the GIL).  Inputs are
    gathered from the device buffers one sequence at a time."""
    threads = threads or min(16, os.cpu_count() or 1)
    jobs = []
    for b in seqs:
        n = int(n_nodes[b])
        c = state.cfg
        L = int(state.tokens.ctx_len[b])
        npg = (L + n + c.page - 1) // c.page
        pages = state.block_table[b, :npg].long()
        jobs.append((b, state.q[b, :n].float().cpu().numpy(), state.k_cache[pages].float().cpu().numpy(),
                     state.v_cache[pages].float().cpu().numpy(), L, np.asarray(parents[b]), n, npg))
        if len(jobs) % 256 == 0:
            say(f"  gathered inputs of {len(jobs)} sequences")

    import time

    from threadpoolctl import threadpool_limits

    def run(job):
        b, q, kc, vc, L, par, n, npg = job
        return b, AT.tree_attention_seq(q, kc, vc, np.arange(npg), L, par, n, state.scale, state.cfg.page)

    out, t0, last = {}, time.time(), time.time()
    with threadpool_limits(limits=1), ThreadPoolExecutor(threads) as ex:  # one BLAS thread per task
        for b, r in ex.map(run, jobs):
            out[b] = r
            if time.time() - last > 10:
                last = time.time()
                say(f"  oracle attention: {len(out)} of {len(jobs)} sequences ({last - t0:.0f} s)")
    return out


def oracle_accept_rows(logits, gumbel, inv_t, tree_np, seqs, Dmax):
    return AC.accept_batch(logits, gumbel, inv_t, tree_np["tree_tokens"], tree_np["tree_parent"],
                           tree_np["n_nodes"], Dmax, seqs=seqs)


def assert_accept_equal(acc_gpu_np, b, want, Dmax):
    k, toks, nodes = want
    assert int(acc_gpu_np["n_accepted"][b]) == k, f"seq {b}: n_accepted {acc_gpu_np['n_accepted'][b]} != {k}"
    assert acc_gpu_np["out_tokens"][b, :k + 1].tolist() == toks, f"seq {b}"
    assert acc_gpu_np["out_nodes"][b, :k].tolist() == nodes, f"seq {b}"
    assert acc_gpu_np["out_nodes"][b, k] == -1
    assert (acc_gpu_np["out_tokens"][b, k + 1:] == -1).all() and (acc_gpu_np["out_nodes"][b, k + 1:] == -1).all()
    if "n_emitted" in acc_gpu_np:
        assert int(acc_gpu_np["n_emitted"][b]) == k + 1


def dict_from_tree(tree_np, b):
    """Oracle-format (tokens, parents, depths, n, q) tuple of a tree row."""
    return tree_rows(tree_np, b)[0]
