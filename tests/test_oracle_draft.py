"""Pins for the draft oracle (oracle/draft.py) against Section 3 ("Speculative
Rollout with Tree-Structured Cache"): hand-worked trees, an independent
greedy best-first expansion (the paper's procedure) on random tiny caches,
structural invariants, the fallback, the budget rule, and planted mistakes
that the pins must catch."""
import heapq
import json
import math
import os
import random

import pytest

from oracle import draft as DR
from oracle import trie as T


def load_cases(golden_dir):
    return json.load(open(os.path.join(golden_dir, "draft_small.json")))["cases"]


def run_case(impl, c):
    trie = T.DictTrie(T.substring_counts(c["streams"], c["D"]), c["D"])
    return impl(trie, c["tail"], c["t"], c["qmax"], c["N"], c["Dmax"])


def golden_ok(impl, golden_dir):
    for c in load_cases(golden_dir):
        tok, par, dep, n, q = run_case(impl, c)
        if (tok, par, dep, q) != (c["tokens"], c["parents"], c["depths"], c["match_len"]):
            return False
    return True


def test_golden(golden_dir):
    for c in load_cases(golden_dir):
        tok, par, dep, n, q = run_case(DR.draft, c)
        assert (tok, par, dep, n, q) == (c["tokens"], c["parents"], c["depths"], len(c["tokens"]),
                                         c["match_len"]), c


def best_first(trie, tail, t, qmax, N, Dmax, alpha=0.0, min_score=0.0, chain=False):
    """Greedy expansion with a priority queue: pop the best frontier node, add
    its children (only the one with the largest count, then smallest token,
    for chain drafts) and stop at the budget or, with a threshold, at the
    first popped score below it; the match scans q downward and stops at the
    first suffix that has a continuation."""
    tail = list(tail)
    root = tail[-1] if t >= 1 else -1
    q = 0
    for cand in range(min(t, qmax), 0, -1):
        s = tuple(tail[-cand:])
        if trie.children(s):
            q = cand
            break
    if q == 0:
        return [root], [-1], [0], 1, 0
    s = tuple(tail[-q:])
    limit = min(Dmax, trie.D - q)
    budget = N - 1 if alpha <= 0 else min(N - 1, math.floor(alpha * q))
    heap = []

    def push(node_path, idx, score):
        if len(node_path) >= limit:
            return
        kids = trie.children(s + node_path)
        tot = float(sum(kids.values()))
        items = sorted(kids.items(), key=lambda xc: (-xc[1], xc[0]))
        for x, c in (items[:1] if chain else items):
            sc = score * (float(c) / tot)
            heapq.heappush(heap, (-sc, len(node_path) + 1, node_path + (x,), idx))

    tok, par, dep = [root], [-1], [0]
    push((), 0, 1.0)
    while heap and len(tok) - 1 < budget:
        negs, d, path, pidx = heapq.heappop(heap)
        if min_score > 0 and -negs < min_score:
            break
        tok.append(path[-1]); par.append(pidx); dep.append(d)
        push(path, len(tok) - 1, -negs)
    return tok, par, dep, len(tok), q


def rand_case(rng):
    vocab = rng.choice([2, 3, 4])
    D = rng.randrange(3, 9)
    streams = [[rng.randrange(vocab) for _ in range(rng.randrange(1, 25))] for _ in range(rng.randrange(1, 7))]
    trie = T.DictTrie(T.substring_counts(streams, D), D)
    qmax = rng.randrange(1, 5)
    t = rng.randrange(0, 10)
    tail = [rng.randrange(vocab) for _ in range(qmax)]
    N = rng.randrange(1, 20)
    Dmax = rng.randrange(0, 7)
    return trie, tail, t, qmax, N, Dmax


@pytest.mark.parametrize("seed", range(300))
def test_best_first_equals_sort_all(seed):
    rng = random.Random(seed)
    trie, tail, t, qmax, N, Dmax = rand_case(rng)
    assert DR.draft(trie, tail, t, qmax, N, Dmax) == best_first(trie, tail, t, qmax, N, Dmax)


@pytest.mark.parametrize("seed", range(200))
def test_best_first_equals_sort_all_variants(seed):
    rng = random.Random(5000 + seed)
    trie, tail, t, qmax, N, Dmax = rand_case(rng)
    chain = seed % 2 == 1
    tau = [0.0, 0.05, 0.2, 1.0 / 3.0, 0.5][seed % 5]
    assert DR.draft(trie, tail, t, qmax, N, Dmax, min_score=tau, chain=chain) == \
        best_first(trie, tail, t, qmax, N, Dmax, min_score=tau, chain=chain)


def chain_walk(trie, tail, t, qmax, N, Dmax, min_score=0.0):
    """Chain draft by hand: from the match, repeatedly take the child with the
    largest count (smallest token on ties) while the running product of
    C = count / sum of sibling counts stays >= min_score."""
    q = DR.longest_match(trie, tail, t, qmax)
    tok = [tail[-1] if t >= 1 else -1]
    if q == 0:
        return tok, q
    node = tuple(tail[-q:])
    score = 1.0
    for _ in range(min(N - 1, min(Dmax, trie.D - q))):
        kids = trie.children(node)
        if not kids:
            break
        x = max(kids, key=lambda k: (kids[k], -k))
        score = score * (kids[x] / sum(kids.values()))
        if min_score > 0 and score < min_score:
            break
        tok.append(x)
        node = node + (x,)
    return tok, q


@pytest.mark.parametrize("seed", range(150))
def test_chain_equals_walk(seed):
    rng = random.Random(9000 + seed)
    trie, tail, t, qmax, N, Dmax = rand_case(rng)
    tau = [0.0, 0.1, 0.4][seed % 3]
    tok, par, dep, n, q = DR.draft(trie, tail, t, qmax, N, Dmax, min_score=tau, chain=True)
    assert (tok, q) == chain_walk(trie, tail, t, qmax, N, Dmax, tau)
    assert par == list(range(-1, n - 1)) and dep == list(range(n))


def test_chain_hand_case():
    # after "1": 2 follows three times, 7 once; after "1 2": 3 twice, 6 once
    streams = [[1, 2, 3, 4, 5], [1, 2, 3, 4, 5], [1, 2, 6], [1, 7]]
    trie = T.DictTrie(T.substring_counts(streams, 8), 8)
    tok, par, dep, n, q = DR.draft(trie, [1], 1, 1, 10, 6, chain=True)
    assert q == 1 and tok == [1, 2, 3, 4, 5] and par == [-1, 0, 1, 2, 3]
    tok, *_ = DR.draft(trie, [1], 1, 1, 10, 6, min_score=0.5, chain=True)
    assert tok == [1, 2, 3, 4, 5]          # 3/4, then 3/4 * 2/3 = 1/2 exactly, kept (>=)
    tok, *_ = DR.draft(trie, [1], 1, 1, 10, 6, min_score=0.5 + 1e-12, chain=True)
    assert tok == [1, 2]


def test_threshold_is_a_prefix_of_the_order():
    streams = [[1, 2, 3, 4, 5], [1, 2, 3, 4, 5], [1, 6, 7], [1, 6, 8], [1, 6, 9], [1, 6, 10]]
    trie = T.DictTrie(T.substring_counts(streams, 8), 8)
    full = DR.draft(trie, [1], 1, 1, 7, 5)
    assert full[0] == [1, 6, 2, 3, 4, 5, 7]  # scores 2/3, 1/3, 1/3, 1/3, 1/3, 1/6
    tok, *_ = DR.draft(trie, [1], 1, 1, 7, 5, min_score=1.0 / 3.0)
    assert tok == [1, 6, 2, 3, 4, 5]
    tok, *_ = DR.draft(trie, [1], 1, 1, 7, 5, min_score=0.5)
    assert tok == [1, 6]


@pytest.mark.parametrize("seed", range(100))
def test_structure(seed):
    rng = random.Random(1000 + seed)
    trie, tail, t, qmax, N, Dmax = rand_case(rng)
    tok, par, dep, n, q = DR.draft(trie, tail, t, qmax, N, Dmax)
    assert n == len(tok) <= max(1, N)
    assert par[0] == -1 and dep[0] == 0
    s = tuple(tail[len(tail) - q:]) if q else ()
    paths = {0: ()}
    for i in range(1, n):
        assert 0 <= par[i] < i and dep[i] == dep[par[i]] + 1 <= min(Dmax, trie.D - q)
        paths[i] = paths[par[i]] + (tok[i],)
        assert trie.count(s + paths[i]) >= 1
    for i in range(n):  # siblings carry distinct tokens
        kids = [tok[c] for c in range(n) if par[c] == i]
        assert len(kids) == len(set(kids))
    if q == 0:
        assert n == 1
    else:
        # every longer admissible suffix has no continuation
        for q2 in range(q + 1, min(t, qmax) + 1):
            assert not trie.children(tuple(tail[-q2:]))
        # a full budget is used whenever enough candidates exist
        cands = DR.candidates(trie, s, min(Dmax, trie.D - q))
        assert n - 1 == min(N - 1, len(cands))


def test_fallback_on_unseen_token():
    trie = T.DictTrie(T.substring_counts([[1, 2, 3]], 4), 4)
    assert DR.draft(trie, [9], 5, 1, 8, 3) == ([9], [-1], [0], 1, 0)
    assert DR.draft(trie, [3], 5, 1, 8, 3) == ([3], [-1], [0], 1, 0)  # only ends a stream
    assert DR.draft(trie, [], 0, 1, 8, 3) == ([-1], [-1], [0], 1, 0)  # nothing committed


def test_single_chain():
    trie = T.DictTrie(T.substring_counts([[4, 5, 6, 7, 8, 9]], 8), 8)
    tok, par, dep, n, q = DR.draft(trie, [3, 4, 5], 10, 3, 10, 6)
    assert q == 2 and tok == [5, 6, 7, 8, 9] and par == [-1, 0, 1, 2, 3]


def test_budget_alpha():
    trie = T.DictTrie(T.substring_counts([[4, 5, 6, 7, 8, 9]], 10), 10)
    tok, par, dep, n, q = DR.draft(trie, [4, 5], 2, 2, 10, 6, budget_alpha=1.5)
    assert q == 2 and n == 1 + math.floor(1.5 * 2)


def test_bushy_node_versus_long_chain():
    # a unary chain keeps score 1/2 down its length while the bushy side
    # splits into quarters; the chain's depth-3 node still ranks above them
    streams = [[1, 2, 3, 4, 5], [1, 2, 3, 4, 5], [1, 6, 7], [1, 6, 8], [1, 6, 9], [1, 6, 10]]
    trie = T.DictTrie(T.substring_counts(streams, 8), 8)
    tok, par, dep, n, q = DR.draft(trie, [1], 1, 1, 7, 5)
    # (2)=1/3 and (6)=2/3 at depth 1; (6,x)=1/6 each; (2,3),(2,3,4),(2,3,4,5)=1/3
    assert tok == [1, 6, 2, 3, 4, 5, 7]


# --- planted mistakes: each must fail at least one pin -----------------------

def _divide_by_parent_count(trie, tail, t, qmax, N, Dmax, alpha=0.0):
    class Wrapped:
        D = trie.D
        def count(self, s): return trie.count(s)
        def children(self, s):
            kids = trie.children(s)
            if not kids:
                return kids
            # scale so that the children sum to count(parent): divide-by-parent reading
            extra = (trie.count(s) if s else sum(kids.values())) - sum(kids.values())
            if extra:
                kids = dict(kids); kids[10 ** 6] = extra  # phantom sibling absorbs stream ends
            return kids
    res = DR.draft(Wrapped(), tail, t, qmax, N, Dmax, alpha)
    tok, par, dep, n, q = res
    keep = [i for i in range(n) if tok[i] != 10 ** 6]
    remap = {old: new for new, old in enumerate(keep)}
    return ([tok[i] for i in keep], [remap.get(par[i], -1) for i in keep],
            [dep[i] for i in keep], len(keep), q)


def _token_only_ties(trie, tail, t, qmax, N, Dmax, alpha=0.0):
    orig = DR.candidates
    def cands(tr, s, lim):
        return [(sc, p) for sc, p in orig(tr, s, lim)]
    tok, par, dep, n, q = DR.draft(trie, tail, t, qmax, N, Dmax, alpha)
    if q == 0:
        return tok, par, dep, n, q
    s = tuple(tail[-q:])
    cs = cands(trie, s, min(Dmax, trie.D - q))
    cs.sort(key=lambda c: (-c[0], len(c[1]), c[1][-1]))
    idx = {(): 0}; tok2, par2, dep2 = [tok[0]], [-1], [0]
    for sc, p in cs[:N - 1]:
        if p[:-1] not in idx:
            return None
        idx[p] = len(tok2); tok2.append(p[-1]); par2.append(idx[p[:-1]]); dep2.append(len(p))
    return tok2, par2, dep2, len(tok2), q


def _no_child_requirement(trie, tail, t, qmax, N, Dmax, alpha=0.0):
    class Wrapped:
        D = trie.D
        def count(self, s): return trie.count(s)
        def children(self, s): return trie.children(s) if trie.children(s) else ({-5: 1} if trie.count(s) else {})
    tok, par, dep, n, q = DR.draft(Wrapped(), tail, t, qmax, N, Dmax, alpha)
    keep = [i for i in range(n) if tok[i] != -5 or i == 0]
    return [tok[i] for i in keep], [par[i] for i in keep], [dep[i] for i in keep], len(keep), q


def _strict_threshold(trie, tail, t, qmax, N, Dmax, min_score=0.0, chain=False):
    tok, par, dep, n, q = DR.draft(trie, tail, t, qmax, N, Dmax, chain=chain)
    s = tuple(tail[-q:]) if q else ()
    keep = 1
    scores = {(): 1.0}
    paths = {0: ()}
    for i in range(1, n):
        paths[i] = paths[par[i]] + (tok[i],)
        kids = trie.children(s + paths[par[i]])
        sc = scores[paths[par[i]]] * (kids[tok[i]] / sum(kids.values()))
        scores[paths[i]] = sc
        if min_score > 0 and not sc > min_score:
            break
        keep += 1
    return tok[:keep], par[:keep], dep[:keep], keep, q


def _chain_by_token(trie, tail, t, qmax, N, Dmax, min_score=0.0):
    q = DR.longest_match(trie, tail, t, qmax)
    tok = [tail[-1] if t >= 1 else -1]
    if q == 0:
        return tok, q
    node = tuple(tail[-q:])
    for _ in range(min(N - 1, min(Dmax, trie.D - q))):
        kids = trie.children(node)
        if not kids:
            break
        x = min(kids)  # smallest token instead of largest count
        tok.append(x)
        node = node + (x,)
    return tok, q


def test_variant_pins_catch_planted_mistakes():
    streams = [[1, 2, 3, 4, 5], [1, 2, 3, 4, 5], [1, 2, 6], [1, 7]]
    trie = T.DictTrie(T.substring_counts(streams, 8), 8)
    assert _strict_threshold(trie, [1], 1, 1, 10, 6, 0.5, True)[0] != [1, 2, 3, 4, 5]
    streams = [[1, 9, 3], [1, 9, 3], [1, 2, 3]]
    trie = T.DictTrie(T.substring_counts(streams, 8), 8)
    assert _chain_by_token(trie, [1], 1, 1, 10, 6)[0] != DR.draft(trie, [1], 1, 1, 10, 6, chain=True)[0]


def test_pins_catch_planted_mistakes(golden_dir):
    assert golden_ok(DR.draft, golden_dir)
    for bad in (_divide_by_parent_count, _token_only_ties, _no_child_requirement):
        ok = True
        try:
            ok = golden_ok(bad, golden_dir)
        except Exception:
            ok = False
        assert not ok, bad.__name__
