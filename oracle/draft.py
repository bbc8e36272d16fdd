"""Oracle for draft extraction (test infrastructure only).

Section 3 ("Speculative Rollout with Tree-Structured Cache"): given the
partial continuation y_1..y_t, find the longest suffix y_{t-q+1..t} that the
cache holds by walking from the root; if none, fall back to one ordinary
decode step.  From the matched node u_q add descendants greedily, ranking an
edge to child v by C(v) = count(v) / sum of count(w) over the children w of
parent(v) (the displayed equation of Section 3), scoring a node by the
product of C along its path from u_q, until a budget B(q) is reached.

Readings (the paper leaves these open):
* the match must have at least one continuation in the cache (a suffix whose
  only occurrences end a stream cannot be drafted from); the longest such q
  with q <= Qmax and q <= t is used, q = 0 means fall back;
* candidates are all descendants of u_q up to relative depth
  min(Dmax, D - q); C and the path product are IEEE fp64, one division and
  one multiplication per edge, score(u_q) = 1;
* ties are broken by relative depth (shallower first), then by the token path
  from u_q compared lexicographically by token id, which makes the order
  total; because fl(x * C) <= x for C <= 1, a parent always ranks before its
  children, so the first B candidates form a connected subtree and greedy
  best-first expansion picks the same nodes in the same order;
* the budget is B = N - 1 drafted nodes (N counts the root row), or
  min(N - 1, floor(alpha * q)) when alpha > 0;
* the tree is emitted in selection order: node 0 is the last committed token
  (parent -1, depth 0), then the selected nodes, each with the index of its
  parent in this list and its depth relative to u_q.

Drafting variants (Section 3 leaves the form of the budget B(q) open; the
example of Fig. 2 drafts the single highest-scoring path):
* score threshold: with min_score > 0 only candidates whose path-product
  score is >= min_score are drafted (still at most B of them); since the
  order is score-descending these are a prefix of it;
* chain: with chain=True every node contributes only its best child (largest
  C(v), i.e. largest count, then smallest token id), so the candidates, and
  the draft, form one path.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple


def longest_match(trie, tail: Sequence[int], t: int, qmax: int) -> int:
    """q* = max q in [1, min(t, Qmax)] whose suffix node exists and has a child."""
    best = 0
    for q in range(1, min(t, qmax) + 1):
        s = tuple(int(x) for x in tail[len(tail) - q:])
        if trie.count(s) >= 1 and len(trie.children(s)) >= 1:
            best = max(best, q)
    return best


def candidates(trie, s: Tuple[int, ...], depth_limit: int, chain: bool = False):
    """Every descendant of node s within ``depth_limit`` edges (only the best
    child of each node when ``chain``), with its fp64 path-product score:
    list of (score, path) where path is the token tuple from s."""
    out = []

    def visit(node: Tuple[int, ...], path: Tuple[int, ...], score: float):
        if len(path) == depth_limit:
            return
        kids = trie.children(node)
        total = float(sum(kids.values()))
        items = list(kids.items())
        if chain and items:
            items = [min(items, key=lambda xc: (-xc[1], xc[0]))]  # largest count, then smallest token
        for x, c in items:
            cv = float(c) / total           # C(v), one fp64 division (denominator over all children)
            sv = score * cv                 # path product, one fp64 multiplication
            out.append((sv, path + (x,)))
            visit(node + (x,), path + (x,), sv)

    visit(s, (), 1.0)
    return out


def draft(trie, tail: Sequence[int], t: int, qmax: int, n_nodes: int, max_depth: int,
          budget_alpha: float = 0.0, min_score: float = 0.0, chain: bool = False):
    """Draft tree for one sequence.

    ``tail`` holds the last min(t, Qmax) committed tokens (right-aligned; any
    earlier entries are ignored).  Returns (tokens, parents, depths, n, q*)
    as Python lists of length n."""
    tail = [int(x) for x in tail]
    root_tok = tail[-1] if t >= 1 else -1
    q = longest_match(trie, tail, t, qmax)
    tokens, parents, depths = [root_tok], [-1], [0]
    if q == 0:
        return tokens, parents, depths, 1, 0
    s = tuple(tail[len(tail) - q:])
    limit = min(max_depth, trie.D - q)
    cands = candidates(trie, s, limit, chain)
    cands.sort(key=lambda c: (-c[0], len(c[1]), c[1]))
    if min_score > 0:
        cands = [c for c in cands if c[0] >= min_score]
    budget = n_nodes - 1
    if budget_alpha > 0:
        budget = min(budget, int(math.floor(budget_alpha * q)))
    index = {(): 0}
    for score, path in cands[:max(0, budget)]:
        parent = index[path[:-1]]  # KeyError here would mean a disconnected selection
        index[path] = len(tokens)
        tokens.append(path[-1])
        parents.append(parent)
        depths.append(len(path))
    return tokens, parents, depths, len(tokens), q


def draft_batch(tries: List, prompt_ids, tails, ts, qmax, n_nodes, max_depth, budget_alpha=0.0, min_score=0.0,
                chain=False):
    """``draft`` for every sequence; outputs padded to N with -1 like the GPU."""
    import numpy as np
    B = len(ts)
    tt = np.full((B, n_nodes), -1, dtype=np.int32)
    tp = np.full((B, n_nodes), -1, dtype=np.int32)
    td = np.full((B, n_nodes), -1, dtype=np.int32)
    nn = np.zeros(B, dtype=np.int32)
    ml = np.zeros(B, dtype=np.int32)
    for b in range(B):
        tok, par, dep, n, q = draft(tries[int(prompt_ids[b])], tails[b], int(ts[b]), qmax,
                                    n_nodes, max_depth, budget_alpha, min_score, chain)
        tt[b, :n], tp[b, :n], td[b, :n] = tok, par, dep
        nn[b], ml[b] = n, q
    return tt, tp, td, nn, ml
