"""Oracle for the acceptance walk (test infrastructure only).

Section 1 and Section 3: the current policy verifies the drafted tokens and
accepts them up to the first mismatch, which keeps the on-policy distribution
exactly ("classic speculative decoding procedure").  With a deterministic
tree draft this is a walk from the root: at node u the policy's own next
token is chosen (greedy: arg-max of the logits; sampled at temperature T:
Gumbel-max, arg-max of logits / T + g with g ~ Gumbel(0, 1)); if a child of u
carries that token the walk descends, otherwise that token is the bonus token
and the walk stops.  Rollouts use T = 1.0 (Appendix A, Table 2).

Readings: the noise is indexed by the step of the walk (= depth of u), one
row [V] per depth, so the walk equals sequential Gumbel-max sampling with
that row at that step; x = fl(fl(logit * invT) + g) in fp32 without fused
multiply-add; ties go to the lowest token id; inputs must be finite.
"""
from __future__ import annotations

import numpy as np


def accept(row, noise, inv_temperature: float, tree_tokens, tree_parent, n: int, max_depth: int):
    """Walk one tree.

    row(u) -> fp32 [V] logits of tree node u; noise(k) -> fp32 [V] Gumbel row
    for step k, or ``noise`` is None for greedy.  Returns (n_accepted,
    out_tokens, out_nodes): the accepted drafted tokens followed by the bonus
    token, and the tree indices of the accepted nodes."""
    u, k = 0, 0
    out_tokens, out_nodes = [], []
    while True:
        x = np.asarray(row(u), dtype=np.float32)
        if noise is not None:
            x = (x * np.float32(inv_temperature)).astype(np.float32)
            x = (x + np.asarray(noise(k), dtype=np.float32)).astype(np.float32)
        assert np.all(np.isfinite(x)), "acceptance inputs must be finite"
        tok = int(np.argmax(x))  # first index of the maximum
        child = -1
        for c in range(u + 1, n):
            if int(tree_parent[c]) == u and int(tree_tokens[c]) == tok:
                child = c
                break
        out_tokens.append(tok)
        if child < 0 or k >= max_depth:
            return k, out_tokens, out_nodes
        out_nodes.append(child)
        u, k = child, k + 1


def accept_batch(logits, gumbel, inv_temperature, tree_tokens, tree_parent, n_nodes, max_depth,
                 seqs=None):
    """``accept`` for the given sequences; logits [B,N,V] / gumbel [B,Dmax+1,V]
    may be numpy arrays or torch tensors (rows are fetched one at a time).
    Returns {b: (n_accepted, out_tokens, out_nodes)}."""
    def as_np(t):
        return t.cpu().numpy() if hasattr(t, "cpu") else np.asarray(t)

    seqs = range(len(n_nodes)) if seqs is None else seqs
    out = {}
    for b in seqs:
        b = int(b)
        row = lambda u, b=b: as_np(logits[b, u])
        noise = None if gumbel is None else (lambda k, b=b: as_np(gumbel[b, k]))
        out[b] = accept(row, noise, inv_temperature, tree_tokens[b], tree_parent[b],
                        int(n_nodes[b]), max_depth)
    return out
