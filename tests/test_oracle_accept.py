"""Pins for the acceptance oracle (oracle/accept.py) against the lossless
claim of Sections 1 and 3: greedy acceptance emits exactly what sequential
greedy decoding would, Gumbel acceptance what sequential Gumbel-max sampling
would; the accepted path is the longest path on which every token is its
parent's choice; the first emitted token is distributed as softmax(logits/T);
plus hand-worked cases and planted mistakes."""
import json
import os
import random

import numpy as np
import pytest

from oracle import accept as AC


def toy_logits(ctx, V, k=3):
    """Deterministic toy policy: logits seeded by the last k tokens."""
    seed = 0
    for x in ctx[-k:]:
        seed = (seed * 1000003 + int(x) + 7) % (1 << 32)
    return np.random.default_rng(seed).standard_normal(V).astype(np.float32)


def golden(golden_dir):
    return json.load(open(os.path.join(golden_dir, "accept_small.json")))


def test_golden(golden_dir):
    g = golden(golden_dir)
    L = np.array(g["logits"], dtype=np.float32)
    n = len(g["tree_tokens"])
    k, toks, nodes = AC.accept(lambda u: L[u], None, 1.0, g["tree_tokens"], g["tree_parent"], n, g["Dmax"])
    assert (k, toks, nodes) == (g["greedy"]["n_accepted"], g["greedy"]["out_tokens"], g["greedy"]["out_nodes"])
    Gm = np.array(g["gumbel"], dtype=np.float32)
    k, toks, nodes = AC.accept(lambda u: L[u], lambda s: Gm[s], 1.0, g["tree_tokens"], g["tree_parent"], n, g["Dmax"])
    assert (k, toks, nodes) == (g["sampled"]["n_accepted"], g["sampled"]["out_tokens"], g["sampled"]["out_nodes"])


def build_tree(rng, ctx, V, N, Dmax, choose, p_follow=0.7):
    """Random tree that often contains the policy's own choice ``choose``."""
    tokens, parents, depth, paths = [ctx[-1]], [-1], [0], [()]
    frontier = [0]
    while frontier and len(tokens) < N:
        u = frontier.pop(0)
        if depth[u] >= Dmax:
            continue
        used = set()
        if rng.random() < p_follow:
            used.add(choose(list(ctx) + list(paths[u]), depth[u]))
        for _ in range(rng.randrange(0, 3)):
            used.add(rng.randrange(V))
        for x in sorted(used, key=lambda _: rng.random()):
            if len(tokens) >= N:
                break
            tokens.append(x); parents.append(u); depth.append(depth[u] + 1); paths.append(paths[u] + (x,))
            frontier.append(len(tokens) - 1)
    return tokens, parents, depth, paths


@pytest.mark.parametrize("seed", range(40))
def test_greedy_equals_sequential_decoding(seed):
    rng = random.Random(seed)
    V, N, Dmax = rng.choice([5, 17, 64]), rng.randrange(1, 30), rng.randrange(0, 6)
    ctx = [rng.randrange(V) for _ in range(5)]
    greedy = lambda c, d: int(np.argmax(toy_logits(c, V)))
    tokens, parents, depth, paths = build_tree(rng, ctx, V, N, Dmax, greedy)
    n = len(tokens)
    k, out, nodes = AC.accept(lambda u: toy_logits(ctx + list(paths[u]), V), None, 1.0, tokens, parents, n, Dmax)
    seq = []
    for _ in range(k + 1):
        seq.append(greedy(ctx + seq, None))
    assert out == seq
    assert [tokens[u] for u in nodes] == out[:k]


@pytest.mark.parametrize("seed", range(40))
def test_gumbel_equals_sequential_sampling(seed):
    rng = random.Random(100 + seed); nrng = np.random.default_rng(seed)
    V, N, Dmax = rng.choice([5, 17, 64]), rng.randrange(1, 30), rng.randrange(0, 6)
    invT = rng.choice([1.0, 0.5, 1.7])
    ctx = [rng.randrange(V) for _ in range(5)]
    noise = (-np.log(-np.log(nrng.uniform(1e-12, 1 - 1e-12, size=(Dmax + 1, V))))).astype(np.float32)
    def sample(c, step):
        x = (toy_logits(c, V) * np.float32(invT)).astype(np.float32) + noise[step]
        return int(np.argmax(x))
    tokens, parents, depth, paths = build_tree(rng, ctx, V, N, Dmax, sample)
    n = len(tokens)
    k, out, nodes = AC.accept(lambda u: toy_logits(ctx + list(paths[u]), V), lambda s: noise[s], invT,
                              tokens, parents, n, Dmax)
    seq = []
    for step in range(k + 1):
        seq.append(sample(ctx + seq, step))
    assert out == seq


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_longest_path(seed):
    rng = random.Random(200 + seed)
    V, N, Dmax = rng.choice([3, 6]), rng.randrange(1, 25), rng.randrange(0, 5)
    ctx = [rng.randrange(V) for _ in range(4)]
    greedy = lambda c, d: int(np.argmax(toy_logits(c, V)))
    tokens, parents, depth, paths = build_tree(rng, ctx, V, N, Dmax, greedy, p_follow=0.8)
    n = len(tokens)
    row = lambda u: toy_logits(ctx + list(paths[u]), V)
    k, out, nodes = AC.accept(row, None, 1.0, tokens, parents, n, Dmax)
    # the unique longest root path on which each token is its parent's arg-max
    best = 0
    for v in range(n):
        ok, u = True, v
        while u > 0:
            ok &= int(np.argmax(row(parents[u]))) == tokens[u]; u = parents[u]
        if ok:
            best = max(best, depth[v])
    assert k == best


def test_first_token_distribution_chi_square():
    # Gumbel-max with the depth-0 noise row draws the first token ~ softmax(l / T)
    V, invT, S = 8, 0.8, 20000
    logits = np.random.default_rng(1).standard_normal(V).astype(np.float32)
    nrng = np.random.default_rng(2)
    counts = np.zeros(V)
    for _ in range(S):
        g = (-np.log(-np.log(nrng.uniform(1e-12, 1 - 1e-12, size=(1, V))))).astype(np.float32)
        k, out, _ = AC.accept(lambda u: logits, lambda s: g[s], invT, [0], [-1], 1, 0)
        counts[out[0]] += 1
    p = np.exp(logits.astype(np.float64) * invT); p /= p.sum()
    chi2 = ((counts - S * p) ** 2 / (S * p)).sum()
    assert chi2 < 24.3  # 99.9% quantile of chi-square with 7 degrees of freedom


def test_chain_tree():
    V = 10
    L = np.zeros((5, V), dtype=np.float32)
    chain = [0, 3, 1, 4, 1]
    for u in range(4):
        L[u, chain[u + 1]] = 1.0
    L[4, 9] = 1.0
    k, out, nodes = AC.accept(lambda u: L[u], None, 1.0, chain, [-1, 0, 1, 2, 3], 5, 4)
    assert (k, out, nodes) == (4, [3, 1, 4, 1, 9], [1, 2, 3, 4])
    L[2, 1] = 0.0; L[2, 7] = 2.0  # mismatch at depth 2
    k, out, nodes = AC.accept(lambda u: L[u], None, 1.0, chain, [-1, 0, 1, 2, 3], 5, 4)
    assert (k, out, nodes) == (2, [3, 1, 7], [1, 2])


def test_pins_catch_planted_mistakes(golden_dir, monkeypatch):
    g = golden(golden_dir)
    L = np.array(g["logits"], dtype=np.float32); Gm = np.array(g["gumbel"], dtype=np.float32)
    n = len(g["tree_tokens"])
    # (a) highest index wins ties
    monkeypatch.setattr(AC.np, "argmax", lambda x: int(len(x) - 1 - np.flip(np.asarray(x)).argmax()))
    k, toks, _ = AC.accept(lambda u: L[u], None, 1.0, g["tree_tokens"], g["tree_parent"], n, g["Dmax"])
    assert toks != g["greedy"]["out_tokens"]
    monkeypatch.undo()
    # (b) noise indexed by node instead of by step
    k, toks, _ = AC.accept(lambda u: L[u], lambda s: Gm[min(2 * s, 2)], 1.0, g["tree_tokens"], g["tree_parent"], n, g["Dmax"])
    assert toks != g["sampled"]["out_tokens"]
