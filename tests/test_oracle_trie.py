"""Pins for the cache oracle (oracle/trie.py) against the definition in
Section 3 ("Per-prompt rollout cache"): hand-worked counts, per-level
occurrence totals, distinct n-gram counts from numpy, two independent
implementations, order independence and the Fig. 2 caption's relation
between a node and its children."""
import json
import os
import random

import numpy as np
import pytest

from oracle import trie as T


def rand_streams(rng, n_streams, max_len, vocab):
    return [[rng.randrange(vocab) for _ in range(rng.randrange(0, max_len + 1))]
            for _ in range(n_streams)]


def test_golden_counts(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "trie_small.json")))
    got = T.substring_counts(g["streams"], g["D"])
    want = {tuple(s): c for s, c in g["counts"]}
    assert got == want


@pytest.mark.parametrize("seed", range(6))
def test_level_totals(seed):
    # sum over |s| = l of count(s) equals the number of length-l windows
    rng = random.Random(seed)
    streams = rand_streams(rng, 5, 30, 3)
    D = 6
    c = T.substring_counts(streams, D)
    for ell in range(1, D + 1):
        tot = sum(v for s, v in c.items() if len(s) == ell)
        assert tot == sum(max(0, len(st) - ell + 1) for st in streams)


@pytest.mark.parametrize("seed", range(6))
def test_distinct_ngrams_match_numpy(seed):
    rng = random.Random(100 + seed)
    streams = rand_streams(rng, 4, 40, 4)
    D = 5
    c = T.substring_counts(streams, D)
    for ell in range(1, D + 1):
        wins = [np.lib.stride_tricks.sliding_window_view(np.array(st), ell)
                for st in streams if len(st) >= ell]
        n_distinct = np.unique(np.concatenate(wins), axis=0).shape[0] if wins else 0
        assert sum(1 for s in c if len(s) == ell) == n_distinct
        # the count of each n-gram is its multiplicity among the windows
        if wins:
            u, mult = np.unique(np.concatenate(wins), axis=0, return_counts=True)
            for row, m in zip(u, mult):
                assert c[tuple(int(x) for x in row)] == m


@pytest.mark.parametrize("seed", range(4))
def test_stream_trie_agrees_with_dict(seed):
    rng = random.Random(200 + seed)
    streams = rand_streams(rng, 6, 25, 3)
    D = 5
    d = T.DictTrie(T.substring_counts(streams, D), D)
    s = T.StreamTrie(streams, D)
    probes = list(d.counts) + [tuple(rng.randrange(4) for _ in range(rng.randrange(1, D + 2)))
                               for _ in range(200)]
    for p in probes:
        assert s.count(p) == d.count(p), p
        if len(p) <= D:
            assert s.children(p) == d.children(p), p
    assert s.children(()) == d.children(())


def test_order_independence():
    rng = random.Random(7)
    streams = rand_streams(rng, 8, 20, 3)
    a = T.substring_counts(streams, 4)
    rng.shuffle(streams)
    assert T.substring_counts(streams, 4) == a


@pytest.mark.parametrize("seed", range(4))
def test_node_minus_children_counts_stream_ends(seed):
    # count(s) - sum_x count(s x) = number of streams that end with s (|s| < D)
    rng = random.Random(300 + seed)
    streams = rand_streams(rng, 6, 20, 3)
    D = 5
    d = T.DictTrie(T.substring_counts(streams, D), D)
    for s, c in d.counts.items():
        if len(s) < D:
            ends = sum(1 for st in streams if len(st) >= len(s) and tuple(st[len(st) - len(s):]) == s)
            assert c - sum(d.children(s).values()) == ends


def _pins_pass(impl, golden_dir):
    """True iff ``impl`` (a substring_counts replacement) passes the golden
    counts and the per-level totals."""
    g = json.load(open(os.path.join(golden_dir, "trie_small.json")))
    if impl(g["streams"], g["D"]) != {tuple(s): c for s, c in g["counts"]}:
        return False
    rng = random.Random(11)
    streams = rand_streams(rng, 5, 30, 3)
    c = impl(streams, 6)
    for ell in range(1, 7):
        if sum(v for s, v in c.items() if len(s) == ell) != sum(max(0, len(st) - ell + 1) for st in streams):
            return False
    return True


def _drop_last_level(streams, D):
    out = {}
    for st in streams:
        for i in range(len(st)):
            for ell in range(1, min(D - 1, len(st) - i) + 1):
                k = tuple(st[i:i + ell])
                out[k] = out.get(k, 0) + 1
    return out


def _joined_streams(streams, D):
    # forgets the stream boundary: occurrences may span two streams
    flat = [x for st in streams for x in st]
    return T.substring_counts([flat], D)


def _set_semantics(streams, D):
    # counts distinct streams containing s instead of occurrences
    out = {}
    for st in streams:
        for k in set(T.substring_counts([st], D)):
            out[k] = out.get(k, 0) + 1
    return out


def test_pins_catch_planted_mistakes(golden_dir):
    assert _pins_pass(T.substring_counts, golden_dir)
    for bad in (_drop_last_level, _joined_streams, _set_semantics):
        assert not _pins_pass(bad, golden_dir), bad.__name__


@pytest.mark.parametrize("seed", range(5))
def test_online_insert_equals_definition(seed):
    # appending chunk by chunk, streams interleaved, gives the batch map
    rng = random.Random(500 + seed)
    streams = rand_streams(rng, 4, 30, 3)
    D = rng.randrange(1, 7)
    counts, pos = {}, [0] * len(streams)
    while any(p < len(s) for p, s in zip(pos, streams)):
        i = rng.randrange(len(streams))
        k = rng.randrange(0, 5)
        T.insert_counts(counts, streams[i][:pos[i]], streams[i][pos[i]:pos[i] + k], D)
        pos[i] += k
    assert counts == T.substring_counts(streams, D)
