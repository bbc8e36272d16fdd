"""Helpers for the GPU parity tests: oracle evaluations on the same inputs the
HIP path receives, and the comparison rules (bit-exact for cache contents,
trees and acceptance; |gpu - ref| <= 1e-2 + 2e-2 |ref| for attention)."""
from __future__ import annotations

import sys

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
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - ref)
    bound = ATOL + RTOL * np.abs(ref)
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance; "
                           f"max abs err {err.max():.3e}, worst excess {(err - bound).max():.3e}")
    return float(err.max()), float((err / np.maximum(np.abs(ref), 1e-30)).max())


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
