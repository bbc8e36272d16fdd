"""GPU parity of srt_accept against the oracle walk, bit-exact: greedy and
Gumbel sampling, temperatures, ties, vocabularies with and without 16-byte
alignment, depth caps, long accepted paths; large vocabularies split over
up to 32 cooperating workgroups per sequence, with ties across slices."""
import random

import numpy as np
import pytest
import torch

from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from tests.gpu_util import assert_accept_equal, oracle_accept_rows, say

pytestmark = pytest.mark.gpu


def random_trees(rng, B, N, Dmax, V):
    tt = np.full((B, N), -1, np.int32)
    tp = np.full((B, N), -1, np.int32)
    td = np.full((B, N), -1, np.int32)
    nn = np.zeros(B, np.int32)
    for b in range(B):
        n = rng.randrange(1, N + 1)
        tt[b, 0], td[b, 0] = rng.randrange(V), 0
        used = {}
        k = 1
        while k < n:
            p = rng.randrange(k)
            if td[b, p] >= Dmax:
                if all(td[b, j] >= Dmax for j in range(k)):
                    break
                continue
            x = rng.randrange(V)
            if (p, x) in used:
                continue
            used[(p, x)] = 1
            tt[b, k], tp[b, k], td[b, k] = x, p, td[b, p] + 1
            k += 1
        nn[b] = k
    return {"tree_tokens": tt, "tree_parent": tp, "tree_depth": td, "n_nodes": nn}


def run(tree, logits, gumbel, inv_t, Dmax):
    t = lambda a: torch.as_tensor(a, device="cuda")
    acc = srt.srt_accept(logits, gumbel, inv_t, t(tree["tree_tokens"]), t(tree["tree_parent"]),
                         t(tree["n_nodes"]), Dmax)
    return {k: v.cpu().numpy() for k, v in acc.items()}


@pytest.mark.parametrize("V,sampled,inv_t,boost", [
    (1024, False, 1.0, "top"), (1024, True, 1.0, "top"), (1023, True, 0.7, "top"), (1021, False, 1.0, "top"),
    (151936, True, 1.0, "literal"), (152064, False, 1.0, "top"), (152064, True, 1.3, "top"), (6, False, 1.0, "none"),
    (151937, True, 1.0, "top"), (50001, False, 1.0, "none")])
def test_walk_exact(V, sampled, inv_t, boost):
    rng = random.Random(V * 7 + int(sampled))
    B, N, Dmax = 24, 32, 8
    say(f"accept: V={V} sampled={sampled} invT={inv_t} boost={boost}")
    tree = random_trees(rng, B, N, Dmax, V)
    cfg = W.Config("acc", 0, n_prompts=B, seqs_per_prompt=1, vocab=V, rollouts_per_prompt=0,
                   rollout_len=W.Dist("fixed", 1), ctx_len=W.Dist("fixed", 1), n_nodes=N, max_depth=Dmax,
                   hq=1, hkv=1, head_dim=64, boost_p=0.9)
    logits = W.make_logits(cfg, tree["tree_tokens"], tree["tree_parent"], tree["n_nodes"], device="cuda",
                           seed=V, boost=boost, sigma=2.0)
    if boost == "none":  # heavy ties: integer logits (row maxima repeat, also across the slices of a row)
        logits = torch.round(logits)
    gumbel = W.make_gumbel(cfg, B, device="cuda", seed=V + 1) if sampled else None
    got = run(tree, logits, gumbel, inv_t, Dmax)
    want = oracle_accept_rows(logits, gumbel, inv_t, tree, range(B), Dmax)
    for b in range(B):
        assert_accept_equal(got, b, want[b], Dmax)
    if boost == "top" and not sampled:
        assert got["n_accepted"].max() >= 2


def test_depth_cap_and_chain():
    V, Dmax = 64, 3
    N = 10
    tt = np.array([[5, 1, 2, 3, 4, 6, 7, 8, 9, 10]], np.int32)
    tp = np.array([[-1, 0, 1, 2, 3, 4, 5, 6, 7, 8]], np.int32)  # deeper than Dmax on purpose
    tree = {"tree_tokens": tt, "tree_parent": tp, "n_nodes": np.array([N], np.int32)}
    logits = torch.zeros((1, N, V), device="cuda")
    for u in range(N - 1):
        logits[0, u, tt[0, u + 1]] = 1.0
    say("accept: depth cap")
    got = run(tree, logits, None, 1.0, Dmax)
    want = oracle_accept_rows(logits, None, 1.0, tree, [0], Dmax)
    assert_accept_equal(got, 0, want[0], Dmax)
    assert int(got["n_accepted"][0]) == Dmax
