"""GPU parity of srt_accept against the oracle walk, bit-exact: greedy and
Gumbel sampling, temperatures, ties, vocabularies with and without 16-byte
alignment, depth caps, long accepted paths; large vocabularies split over
up to 32 workgroups per row (chunks), with ties across chunks;
batches of 70-600 sequences with deep walks, and 4000 sequences that all
walk at least three steps deep."""
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


@pytest.mark.parametrize("V,off_l,off_g", [(8192, 1, 3), (152064, 0, 1), (4096, 2, 0)])
def test_walk_exact_misaligned_rows(V, off_l, off_g):
    # V a multiple of 4 but logits / noise passed as views 1-3 floats into a
    # larger buffer: the rows are not 16-byte aligned, so the 4-byte path runs
    rng = random.Random(V + off_l)
    B, N, Dmax = 40, 32, 8
    say(f"accept: misaligned rows V={V} logits +{off_l} noise +{off_g} floats")
    tree = random_trees(rng, B, N, Dmax, V)
    cfg = W.Config("acc", 0, n_prompts=B, seqs_per_prompt=1, vocab=V, rollouts_per_prompt=0,
                   rollout_len=W.Dist("fixed", 1), ctx_len=W.Dist("fixed", 1), n_nodes=N, max_depth=Dmax,
                   hq=1, hkv=1, head_dim=64, boost_p=0.9, boost_add=40.0)
    lg = W.make_logits(cfg, tree["tree_tokens"], tree["tree_parent"], tree["n_nodes"], device="cuda", seed=V,
                       boost="top", sigma=2.0)
    gm = W.make_gumbel(cfg, B, device="cuda", seed=V + 1)
    lbuf = torch.empty(lg.numel() + 4, dtype=torch.float32, device="cuda")
    gbuf = torch.empty(gm.numel() + 4, dtype=torch.float32, device="cuda")
    logits = lbuf[off_l:off_l + lg.numel()].view(lg.shape)
    gumbel = gbuf[off_g:off_g + gm.numel()].view(gm.shape)
    logits.copy_(lg)
    gumbel.copy_(gm)
    got = run(tree, logits, gumbel, 1.0, Dmax)
    want = oracle_accept_rows(lg, gm, 1.0, tree, range(B), Dmax)
    for b in range(B):
        assert_accept_equal(got, b, want[b], Dmax)
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


def deep_trees(rng, B, N, Dmax, V):
    """Trees that mostly extend their newest node (paths of depth up to Dmax)."""
    tt = np.full((B, N), -1, np.int32)
    tp = np.full((B, N), -1, np.int32)
    td = np.full((B, N), -1, np.int32)
    nn = np.zeros(B, np.int32)
    for b in range(B):
        n = rng.randrange(1, N + 1)
        tt[b, 0], td[b, 0] = rng.randrange(V), 0
        used = set()
        k = 1
        while k < n:
            p = k - 1 if rng.random() < 0.75 else rng.randrange(k)
            if td[b, p] >= Dmax:
                p = rng.randrange(k)
                if td[b, p] >= Dmax:
                    continue
            x = rng.randrange(V)
            if (p, x) in used:
                continue
            used.add((p, x))
            tt[b, k], tp[b, k], td[b, k] = x, p, td[b, p] + 1
            k += 1
        nn[b] = k
    return {"tree_tokens": tt, "tree_parent": tp, "tree_depth": td, "n_nodes": nn}


@pytest.mark.parametrize("B,V,sampled,ties,N", [(100, 152064, True, False, 32), (100, 152064, False, True, 32),
                                                (300, 1024, True, False, 32), (70, 50001, False, False, 32),
                                                (600, 152064, True, False, 16)])
def test_walk_exact_large_batch(B, V, sampled, ties, N):
    # a node's last child gets +30 with p = 0.9, so most walks go deep and the
    # late levels run with few walkers left
    rng = random.Random(B * 13 + V)
    Dmax = 12
    say(f"accept: B={B} V={V} sampled={sampled} ties={ties}")
    tree = deep_trees(rng, B, N, Dmax, V)
    g = torch.Generator(device="cuda")
    g.manual_seed(B + V)
    logits = torch.randn((B, N, V), generator=g, device="cuda") * 2.0
    if ties:  # integer logits: row maxima repeat, also across the slices of a row
        logits = torch.round(logits)
    bi, ui, ti = [], [], []
    for b in range(B):
        for c in range(1, int(tree["n_nodes"][b])):
            if rng.random() < 0.9:  # later children overwrite: the node's last child wins
                bi.append(b), ui.append(int(tree["tree_parent"][b, c])), ti.append(int(tree["tree_tokens"][b, c]))
    logits[torch.tensor(bi), torch.tensor(ui), torch.tensor(ti)] = 30.0
    gumbel = None
    if sampled:
        gumbel = -torch.log(-torch.log(torch.rand((B, Dmax + 1, V), generator=g, device="cuda")
                                       .clamp_(1e-20, 1.0 - 1e-7)))
    got = run(tree, logits, gumbel, 1.0, Dmax)
    want = oracle_accept_rows(logits, gumbel, 1.0, tree, range(B), Dmax)
    for b in range(B):
        assert_accept_equal(got, b, want[b], Dmax)
    assert (got["n_accepted"] >= 4).sum() >= 5  # deep walks


def test_many_deep_walks():
    # 4000 chains of 6 nodes whose logits lead down each chain: all 4000 walks
    # reach the fourth step (the level lists hold every sequence)
    B, N, V, Dmax = 4000, 6, 16, 5
    tt = np.tile(np.array([3, 5, 7, 9, 11, 13], np.int32), (B, 1))
    tp = np.tile(np.arange(-1, N - 1, dtype=np.int32), (B, 1))
    nn = np.full(B, N, np.int32)
    rng = np.random.default_rng(3)
    logits = rng.normal(0.0, 1.0, (B, N, V)).astype(np.float32)
    stop = rng.integers(3, N, B)  # the walk of b leaves its chain at node stop[b]
    for b in range(B):
        for u in range(N - 1):
            if u != stop[b]:
                logits[b, u, tt[b, u + 1]] = 10.0
    tree = {"tree_tokens": tt, "tree_parent": tp, "n_nodes": nn}
    logits = torch.from_numpy(logits).cuda()
    gumbel = torch.from_numpy(rng.gumbel(size=(B, Dmax + 1, V)).astype(np.float32) * 0.1).cuda()
    for g in (None, gumbel):
        say(f"accept: {B} walks past the third step, sampled={g is not None}")
        got = run(tree, logits, g, 1.0, Dmax)
        want = oracle_accept_rows(logits, g, 1.0, tree, range(B), Dmax)
        for b in range(B):
            assert_accept_equal(got, b, want[b], Dmax)
        assert (got["n_accepted"] >= 3).all()


@pytest.mark.parametrize("Dmax,sampled", [(63, False), (63, True), (62, True)])
def test_deepest_walk(Dmax, sampled):
    # a 64-node chain whose logits lead down it: the walk takes every level up
    # to the depth cap (all 64 levels when Dmax = 63), the level buffers
    # alternating between their two halves throughout
    B, N, V = 3, 64, 4096
    tt = np.zeros((B, N), np.int32)
    for b in range(B):
        tt[b] = (np.arange(N) * 37 + 11 * b) % V
    tp = np.tile(np.arange(-1, N - 1, dtype=np.int32), (B, 1))
    g = torch.Generator(device="cuda")
    g.manual_seed(Dmax)
    logits = torch.randn((B, N, V), generator=g, device="cuda")
    for b in range(B):
        for u in range(N - 1):
            logits[b, u, int(tt[b, u + 1])] = 50.0
    gumbel = torch.rand((B, Dmax + 1, V), generator=g, device="cuda") if sampled else None
    tree = {"tree_tokens": tt, "tree_parent": tp, "n_nodes": np.full(B, N, np.int32)}
    say(f"accept: deepest walk Dmax={Dmax} sampled={sampled}")
    got = run(tree, logits, gumbel, 1.0, Dmax)
    want = oracle_accept_rows(logits, gumbel, 1.0, tree, range(B), Dmax)
    for b in range(B):
        assert_accept_equal(got, b, want[b], Dmax)
    assert (got["n_accepted"] == min(Dmax, N - 1)).all()
