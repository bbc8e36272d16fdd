"""GPU parity of srt_draft against the oracle draft, bit-exact: the tiny
configuration, random small-vocabulary caches full of score ties, budget and
depth variants, score thresholds and chain drafts, fallbacks, a candidate pool
pruned while more than a quarter full, a 1500-child list that takes the pool
past 1024 entries (the wide-pool selection and pruning), 1500 children tied
in score that keep it there up to the final pruning, and a 3000-child list
that overflows the 2048-entry pool (the one-at-a-time path then runs, its
frontier evicting; also with chain drafts)."""
import random

import numpy as np
import pytest
import torch

from oracle import draft as DR
from oracle import trie as TR
from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from paper_2601_09083_amd.pipeline import Caches, VerifyState
from tests.gpu_util import assert_tree_equal, oracle_draft_rows, oracle_trie, say, tree_to_np

pytestmark = pytest.mark.gpu


def run_draft(c, prompt_ids, tails, ts, Q, N, Dmax, alpha=0.0, min_score=0.0, chain=False):
    dev = "cuda"
    t = lambda a: torch.as_tensor(np.asarray(a, dtype=np.int32), device=dev)
    out = srt.srt_draft(c.ws, t(prompt_ids), t(tails), t(ts), Q, N, Dmax, alpha, min_score=min_score, chain=chain)
    return tree_to_np(out)


def test_tiny_config_exact():
    cfg = W.CONFIGS["tiny"]
    say("draft: tiny config")
    st = VerifyState.build(cfg)
    tree = tree_to_np(st.draft())
    tries = [oracle_trie(st.tokens.streams_of_prompt(p), cfg.trie_depth) for p in range(cfg.n_prompts)]
    want = oracle_draft_rows(st, tries, range(st.tokens.batch))
    for b, w in want.items():
        assert_tree_equal(tree, b, w)
    assert (tree["n_nodes"] > 1).any()


@pytest.mark.parametrize("seed", range(6))
def test_random_small_vocab_ties(seed):
    rng = random.Random(seed)
    P, B = 40, 120
    D = rng.choice([4, 8, 12, 20])
    vocab = rng.choice([2, 3, 5])
    streams = [[np.array([rng.randrange(vocab) for _ in range(rng.randrange(1, 60))]) for _ in range(rng.randrange(1, 6))]
               for _ in range(P)]
    c = Caches.create(P, sum(len(s) for s in streams) + 1, D, 200000)
    ids = c.new_streams(sum(len(s) for s in streams))
    c.insert([p for p in range(P) for _ in streams[p]], ids, [x for s in streams for x in s])
    tries = [TR.DictTrie(TR.substring_counts(streams[p], D), D) for p in range(P)]
    Q = rng.randrange(1, min(D, 9))
    variants = [(rng.randrange(1, 40), rng.randrange(0, 10), 0.0, 0.0, False), (256, 63, 0.0, 0.0, False),
                (64, 12, 1.7, 0.0, False), (64, 12, 0.0, 0.1, False), (256, 63, 0.0, 1.0 / 3.0, False),
                (64, 12, 0.0, 0.0, True), (64, 12, 0.0, 0.05, True), (32, 4, 2.5, 0.0, True)]
    for N, Dmax, alpha, tau, chain in variants:
        say(f"draft: seed={seed} D={D} vocab={vocab} Q={Q} N={N} Dmax={Dmax} alpha={alpha} tau={tau} chain={chain}")
        pids = [rng.randrange(P) for _ in range(B)]
        tails = [[rng.randrange(vocab) for _ in range(Q)] for _ in range(B)]
        ts = [rng.choice([0, 1, 2, Q, 100]) for _ in range(B)]
        tree = run_draft(c, pids, tails, ts, Q, N, Dmax, alpha, tau, chain)
        for b in range(B):
            want = DR.draft(tries[pids[b]], tails[b][Q - min(ts[b], Q):] if ts[b] else [], ts[b], Q, N, Dmax, alpha,
                            tau, chain)
            assert_tree_equal(tree, b, want)


@pytest.mark.parametrize("n_children", [1500, 3000])
def test_frontier_overflow_and_long_child_lists(n_children):
    # node (7) has up to n_children children of unequal counts.  1500 fit the
    # 2048-entry pool, which then holds more than 1024 entries (the wide-pool
    # selection and pruning); 3000 overflow it, and the one-at-a-time path's
    # frontier (512) must evict without losing any of the best 255 candidates
    rng = np.random.default_rng(0)
    D = 6
    n_str = 8000 if n_children > 2000 else 4000
    streams = [[np.array([7, int(x), int(y)]) for x, y in zip(rng.integers(0, n_children, size=n_str),
                                                               rng.integers(0, 3, size=n_str))]]
    c = Caches.create(1, n_str + 1, D, 200000)
    c.insert([0] * n_str, c.new_streams(n_str), streams[0])
    trie = TR.DictTrie(TR.substring_counts(streams[0], D), D)
    for N, Dmax in [(256, 2), (256, 1), (100, 2)]:
        say(f"draft: {n_children} children N={N} Dmax={Dmax}")
        tree = run_draft(c, [0], [[7]], [5], 1, N, Dmax)
        assert_tree_equal(tree, 0, DR.draft(trie, [7], 5, 1, N, Dmax))
    for tau, chain in [(0.0, True), (1e-4, False), (1e-3, True)]:
        say(f"draft: {n_children} children tau={tau} chain={chain}")
        tree = run_draft(c, [0], [[7]], [5], 1, 256, 2, 0.0, tau, chain)
        assert_tree_equal(tree, 0, DR.draft(trie, [7], 5, 1, 256, 2, 0.0, tau, chain))


def test_wide_pool_ties_to_the_final_pruning():
    # node (7) has 1500 children with 2 occurrences each: every child scores
    # 1/1500, so all of them tie at the budget-th score and are kept; the pool
    # keeps 1501 entries through the final pruning (whose counts then run
    # over two register passes), and the tie order (token ascending) decides
    # which 255 are drafted.  With Dmax = 2 their children (one each, tied
    # with them one level deeper) could never be selected, so they are not
    # walked.
    D = 6
    streams = [np.array([7, 1000 + x, 5000 + x]) for x in range(1500) for _ in range(2)]
    c = Caches.create(1, len(streams) + 1, D, 200000)
    c.insert([0] * len(streams), c.new_streams(len(streams)), streams)
    trie = TR.DictTrie(TR.substring_counts(streams, D), D)
    for N, Dmax in [(256, 1), (256, 2), (64, 2)]:
        say(f"draft: 1500 tied children N={N} Dmax={Dmax}")
        tree = run_draft(c, [0], [[7]], [5], 1, N, Dmax)
        assert_tree_equal(tree, 0, DR.draft(trie, [7], 5, 1, N, Dmax))
        assert int(tree["n_nodes"][0]) == N


def test_pool_over_half_full():
    # u = (7) has 8 children with 70 children each (560 grandchildren whose
    # counts repeat with period 13, so scores tie in groups); each grandchild
    # has up to 3 children.  Drafting 63 nodes first discovers all 560
    # grandchildren, so the candidate pool passes 512 entries and is pruned to
    # what can still be selected (at the budget-th score) before the next
    # level is walked.
    rng = np.random.default_rng(5)
    streams = []
    for a in range(8):
        for b in range(70):
            for _ in range(1 + (a * 70 + b) % 13):
                streams.append(np.array([7, 100 + a, 200 + b, 300 + int(rng.integers(0, 3))]))
    D = 6
    c = Caches.create(1, len(streams) + 1, D, 200000)
    c.insert([0] * len(streams), c.new_streams(len(streams)), streams)
    trie = TR.DictTrie(TR.substring_counts(streams, D), D)
    for N, Dmax, alpha, tau in [(64, 3, 0.0, 0.0), (64, 2, 0.0, 0.0), (256, 3, 0.0, 0.0), (64, 3, 0.0, 1e-3),
                                (200, 3, 0.0, 0.0)]:
        say(f"draft: pool over half full N={N} Dmax={Dmax} tau={tau}")
        tree = run_draft(c, [0], [[7]], [5], 1, N, Dmax, alpha, tau)
        assert_tree_equal(tree, 0, DR.draft(trie, [7], 5, 1, N, Dmax, alpha, tau))
        assert int(tree["n_nodes"][0]) > 1


@pytest.mark.parametrize("tau,chain", [(0.0, True), (0.02, False)])
def test_qwen1p5b_variants_full_batch(tau, chain):
    cfg = W.CONFIGS["qwen1.5b"]
    say(f"draft: qwen1.5b tau={tau} chain={chain}")
    st = VerifyState.build(cfg)
    tree = tree_to_np(st.draft(min_score=tau, chain=chain))
    tw = st.tokens
    tails, ts = tw.ctx_tail(), tw.draft_len()
    tries = {}
    for b in range(tw.batch):  # every sequence of the batch
        p = int(tw.seq_prompt[b])
        if p not in tries:
            tries[p] = oracle_trie(tw.streams_of_prompt(p), cfg.trie_depth, big=True)
        want = DR.draft(tries[p], tails[b], int(ts[b]), cfg.max_match, cfg.n_nodes, cfg.max_depth, 0.0, tau, chain)
        assert_tree_equal(tree, b, want)
    if chain:
        n = tree["n_nodes"]
        par = tree["tree_parent"]
        for b in range(tw.batch):
            assert (par[b, 1:n[b]] == np.arange(n[b] - 1)).all()


def test_deterministic_across_runs():
    cfg = W.CONFIGS["tiny"].scaled(n_nodes=64, max_depth=12)
    st = VerifyState.build(cfg)
    say("draft: repeat determinism")
    a = tree_to_np(st.draft())
    for _ in range(3):
        b = tree_to_np(st.draft())
        for k in a:
            assert np.array_equal(a[k], b[k])
