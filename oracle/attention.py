"""Oracle for tree-masked attention (test infrastructure only).

Section 3: after drafting, one decode pass of the policy scores every drafted
token in parallel ("classic speculative decoding"); Appendix C: verification
reads the KV cache once for all candidates.  For a draft tree this is
standard scaled-dot-product attention in which tree node i sees the whole
committed context and exactly its own ancestors-or-self in the tree.

Reading of the layout: the K/V of context position j of sequence b sit in
page block_table[b, j // page], slot j % page; tree node i is stored at
position ctx_len[b] + i.  Query head h uses KV head h // (Hq / Hkv).
Everything is computed in fp64 from the bf16 inputs (bf16 -> fp64 is exact).
"""
from __future__ import annotations

import numpy as np


def ancestors(tree_parent, n: int) -> np.ndarray:
    """A[i, j] = True iff tree node j is i or an ancestor of i."""
    A = np.zeros((n, n), dtype=bool)
    for i in range(n):
        j = i
        while j >= 0:
            A[i, j] = True
            j = int(tree_parent[j])
    return A


def gather_positions(cache: np.ndarray, block_table_row, n_pos: int, page: int) -> np.ndarray:
    """[n_pos, Hkv, d] values of positions 0..n_pos-1 of one sequence."""
    idx = np.arange(n_pos)
    pages = np.asarray(block_table_row)[idx // page]
    return cache[pages, :, idx % page, :]


def tree_attention_seq(q, k_cache, v_cache, block_table_row, ctx_len: int, tree_parent,
                       n: int, scale: float, page: int) -> np.ndarray:
    """Outputs [n, Hq, d] (fp64) for one sequence.

    q: [>=n, Hq, d]; caches: [P, Hkv, page, d] (any float dtype)."""
    q = np.asarray(q, dtype=np.float64)
    Hq, d = q.shape[1], q.shape[2]
    Hkv = k_cache.shape[1]
    G = Hq // Hkv
    L = int(ctx_len)
    K = gather_positions(k_cache, block_table_row, L + n, page).astype(np.float64)
    V = gather_positions(v_cache, block_table_row, L + n, page).astype(np.float64)
    visible = np.ones((n, L + n), dtype=bool)
    visible[:, L:] = ancestors(tree_parent, n)
    out = np.zeros((n, Hq, d), dtype=np.float64)
    for h in range(Hq):
        g = h // G
        s = (q[:n, h, :] @ K[:, g, :].T) * scale
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ V[:, g, :]
    return out


def tree_attention(q, k_cache, v_cache, block_table, ctx_len, tree_parent, n_nodes,
                   scale: float, page: int, seqs=None) -> dict:
    """{b: [n_b, Hq, d] fp64} for the sequences in ``seqs`` (default: all)."""
    seqs = range(len(ctx_len)) if seqs is None else seqs
    return {int(b): tree_attention_seq(q[b], k_cache, v_cache, block_table[b], int(ctx_len[b]),
                                       tree_parent[b], int(n_nodes[b]), scale, page)
            for b in seqs}
