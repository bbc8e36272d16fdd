"""Oracle for committing an accepted path (test infrastructure only).

Section 3 verifies a whole draft tree in one decode pass and keeps the
accepted tokens as in classic speculative decoding; Appendix C describes the
same loop with the KV cache read once per pass.  After the pass, the key and
value vectors the pass computed for the accepted tree nodes become the
cached vectors of the positions those tokens now occupy, and the sequence
grows by the accepted tokens plus the bonus token.

Layout reading (the paper leaves the engine's bookkeeping open): the context
holds positions 0 .. L-1, the tree root (the last committed token) sits at
position L and tree node i at position L + i.  With accepted nodes
c_1 < c_2 < ... < c_k (tree indices along the accepted path) and bonus
token x:

* position L + j receives the vectors of position L + c_j (j = 1..k);
  positions <= L and > L + k keep their values;
* the cached length becomes L + k + 1 (root and accepted nodes are now
  context; the bonus token's vectors come from the next pass, whose root it
  is);
* the committed token sequence grows by the k accepted tokens and x, so the
  draft tail is the last Qmax tokens of (old tail, emitted tokens) and the
  committed count t grows by k + 1.
"""
from __future__ import annotations

import numpy as np


def commit_kv(kv_seq, L: int, n_accepted: int, out_nodes):
    """kv_seq: array [positions, ...] of one sequence's cached vectors in
    logical position order (context, then tree slots).  Returns a new array
    with the accepted nodes moved into place, and the new cached length."""
    out = np.array(kv_seq, copy=True)
    for j in range(1, n_accepted + 1):
        out[L + j] = kv_seq[L + int(out_nodes[j - 1])]
    return out, L + n_accepted + 1


def commit_tail(tail, t: int, emitted):
    """tail: the last min(t, Qmax) committed tokens right-aligned in a row of
    Qmax entries (-1 padded); emitted: accepted tokens then the bonus token.
    Returns (new tail row, new t)."""
    q = len(tail)
    have = [int(x) for x in tail[q - min(t, q):]]
    seq = have + [int(x) for x in emitted]
    new = np.full(q, -1, dtype=np.int32)
    keep = seq[-q:] if len(seq) >= q else seq
    new[q - len(keep):] = keep
    return new, t + len(emitted)
