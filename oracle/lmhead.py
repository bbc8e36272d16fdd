"""Oracle for the acceptance walk with the LM head applied on demand (test
infrastructure only).

Section 3 verifies a drafted tree in one pass of the policy and Sections 1
and 3 accept its tokens up to the first mismatch (``oracle.accept``).  The
policy's next-token logits at a tree node are its LM head applied to the
node's final hidden state: for node u and vocabulary entry j,

    logit_j(u) = sum_k hidden[u, k] * w_head[j, k].

The walk reads the logits of the nodes it visits only, one row per step, so
a fused implementation never forms the logits of the other nodes.  This
oracle is that definition followed by ``oracle.accept.accept``.

Readings (the paper gives no numeric format for the head):
* hidden states and head weights are bf16 values (given here as float
  arrays holding bf16-representable numbers); each product is exact in fp64,
  the oracle sums the products in fp64 and rounds the sum once to fp32;
* an implementation that sums in fp32 in another order may differ from this
  by at most ``logit_error_bound`` (a standard forward error bound of
  recursive / blocked fp32 summation, see its docstring).  When every
  partial sum is an integer of magnitude below 2^24 (small integer inputs)
  every order gives the same exact fp32 value, and the walk's decisions are
  then identical bit for bit;
* everything else (Gumbel noise row per step, fp32 x = fl(fl(logit * invT) +
  g), lowest index on ties, child search, Dmax) is ``oracle.accept``'s.
"""
from __future__ import annotations

import numpy as np

from . import accept as _accept

U32 = 2.0 ** -24  # unit roundoff of fp32


def head_logits(hidden_rows, w_head) -> np.ndarray:
    """fp32 logits: fp64 dot products rounded once to fp32.

    hidden_rows [d] (one node -> [V]) or [n, d] (n nodes -> [n, V]) and
    w_head [V, d] hold bf16-representable values."""
    h = np.asarray(hidden_rows, dtype=np.float64)
    h2 = h[None, :] if h.ndim == 1 else h
    W = np.asarray(w_head)
    out = np.empty((W.shape[0], h2.shape[0]), dtype=np.float64)
    step = 8192  # head rows per block, only to bound the fp64 temporary
    for j0 in range(0, W.shape[0], step):
        out[j0:j0 + step] = W[j0:j0 + step].astype(np.float64) @ h2.T
    out = out.T.astype(np.float32)
    return out[0] if h.ndim == 1 else out


def logit_error_bound(hidden_row, w_head) -> np.ndarray:
    """Per-entry bound on |fp32 sum in any order - head_logits|.

    Products of bf16 values are exact in fp32 (8 + 8 significant bits), so
    only the d - 1 additions round: |error of any fp32 summation order| <=
    (d - 1) u sum_k |h_k w_jk| / (1 - (d - 1) u) (Higham, Accuracy and
    Stability of Numerical Algorithms, eq. 4.4 and the remark on arbitrary
    orders), plus the final rounding of the oracle's fp64 sum (<= u |logit|)
    and the fp64 summation error (negligible, covered by the factor 2)."""
    h = np.abs(np.asarray(hidden_row, dtype=np.float64))
    W = np.asarray(w_head)
    d = h.shape[0]
    gam = (d - 1) * U32 / (1.0 - (d - 1) * U32)
    mag = np.empty(W.shape[0], dtype=np.float64)
    step = 8192
    for j0 in range(0, W.shape[0], step):
        mag[j0:j0 + step] = np.abs(W[j0:j0 + step].astype(np.float64)) @ h
    return 2.0 * gam * mag + U32 * mag


def accept_lmhead(hidden, w_head, noise, inv_temperature: float, tree_tokens, tree_parent, n: int,
                  max_depth: int):
    """Walk one tree whose node u has final hidden state hidden[u] ([N, d]).

    ``noise(k)`` -> fp32 [V] Gumbel row for step k, or None for greedy.
    Returns (n_accepted, out_tokens, out_nodes) as ``oracle.accept.accept``."""
    return _accept.accept(lambda u: head_logits(hidden[u], w_head), noise, inv_temperature, tree_tokens,
                          tree_parent, n, max_depth)


def accept_lmhead_batch(hidden, w_head, gumbel, inv_temperature, tree_tokens, tree_parent, n_nodes, max_depth,
                        seqs=None):
    """``accept_lmhead`` for the given sequences.  hidden [B, N, d],
    w_head [V, d] (float arrays of bf16 values), gumbel [B, Dmax+1, V] fp32 or
    None.  Returns {b: (n_accepted, out_tokens, out_nodes)}."""
    seqs = range(len(n_nodes)) if seqs is None else seqs
    out = {}
    for b in seqs:
        b = int(b)
        noise = None if gumbel is None else (lambda k, b=b: np.asarray(gumbel[b, k], dtype=np.float32))
        n = min(max(int(n_nodes[b]), 1), len(tree_tokens[b]))
        out[b] = accept_lmhead(hidden[b], w_head, noise, inv_temperature, tree_tokens[b], tree_parent[b], n,
                               max_depth)
    return out
