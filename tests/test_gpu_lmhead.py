"""GPU parity of srt_accept_lmhead (the LM head applied at the visited nodes,
fused with the acceptance walk) against the oracle.

* Integer-valued bf16 inputs make every partial sum of the head exact in
  fp32, so the GPU walk must equal the oracle's bit for bit: ragged
  vocabularies (V = 1, 129, 4099, 50001), d_model of one to several 64-wide
  chunks, more than 256 sequences (two sequence blocks), ties (sparse hidden
  states), greedy and Gumbel at several temperatures, depth caps, root-only
  trees and node counts outside [1, N].  It must also equal srt_accept on
  the materialised logits.
* Real-valued bf16 inputs: every step of the GPU walk must be valid against
  the oracle's fp64 scores within the fp32 summation bound, and nearly all
  walks must equal the oracle's.
* The 7B-shaped head (V = 152064, d_model = 3584, 256 sequences, N = 64,
  Dmax = 12): all sequences against srt_accept on the materialised logits,
  sampled sequences against the oracle.
* Scratch reuse across calls of different sizes."""
import random

import numpy as np
import pytest
import torch

from oracle import accept as AC
from oracle import lmhead as LH
from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from tests.gpu_util import assert_accept_equal, say
from tests.test_gpu_accept import random_trees

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def chain_trees(B, N, Dmax, token=0):
    """Every tree a chain of `token` (the only tree shape a one-token
    vocabulary allows), of length 1 .. min(N, Dmax + 1)."""
    tt = np.full((B, N), -1, np.int32)
    tp = np.full((B, N), -1, np.int32)
    nn = np.zeros(B, np.int32)
    for b in range(B):
        n = 1 + b % min(N, Dmax + 1)
        tt[b, :n] = token
        tp[b, 1:n] = np.arange(n - 1)
        nn[b] = n
    return {"tree_tokens": tt, "tree_parent": tp, "n_nodes": nn}


def tree_tensors(tree):
    t = lambda a: torch.as_tensor(a, device="cuda")
    return t(tree["tree_tokens"]), t(tree["tree_parent"]), t(tree["n_nodes"])


def run_fused(hidden, w, gumbel, inv_t, tree, Dmax, scratch=None):
    tt, tp, nn = tree_tensors(tree)
    acc = srt.srt_accept_lmhead(hidden, w, gumbel, inv_t, tt, tp, nn, Dmax, scratch=scratch)
    return {k: v.cpu().numpy() for k, v in acc.items()}


def run_materialised(hidden, w, gumbel, inv_t, tree, Dmax):
    """srt_accept on logits formed by a plain fp32 product (exact for the
    integer inputs these comparisons use)."""
    B, N, d = hidden.shape
    logits = (hidden.float().reshape(B * N, d) @ w.float().t().contiguous()).reshape(B, N, -1).contiguous()
    tt, tp, nn = tree_tensors(tree)
    acc = srt.srt_accept(logits, gumbel, inv_t, tt, tp, nn, Dmax)
    del logits
    return {k: v.cpu().numpy() for k, v in acc.items()}


def oracle_rows(hidden, w, gumbel, inv_t, tree, seqs, Dmax):
    h = hidden.float().cpu().numpy()
    wn = w.float().cpu().numpy()
    g = None if gumbel is None else gumbel.cpu().numpy()
    return LH.accept_lmhead_batch(h, wn, g, inv_t, tree["tree_tokens"], tree["tree_parent"], tree["n_nodes"],
                                  Dmax, seqs=seqs)


def assert_same(a, b, B):
    for k in ("n_accepted", "out_tokens", "out_nodes", "n_emitted"):
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("V,d,B,sampled,inv_t,plant,density", [
    (1000, 128, 24, False, 1.0, 0.8, 1.0),
    (1000, 128, 24, True, 1.0, 0.8, 1.0),
    (129, 64, 5, True, 0.7, 0.8, 1.0),       # one full tile and a 1-row tail
    (1, 64, 3, False, 1.0, 0.0, 1.0),        # a single token
    (4099, 256, 300, True, 1.0, 0.8, 1.0),   # two sequence blocks, ragged tail
    (2000, 192, 40, False, 1.0, 0.5, 0.02),  # sparse hidden states: many tied scores
    (2000, 192, 40, True, 1.0, 0.5, 0.02),
    (50001, 512, 64, True, 1.3, 0.9, 1.0),
])
def test_exact_integer_inputs(V, d, B, sampled, inv_t, plant, density):
    rng = random.Random(V * 31 + d + B)
    N, Dmax = 32, 8
    say(f"lmhead exact: V={V} d={d} B={B} sampled={sampled} invT={inv_t} plant={plant} density={density}")
    tree = random_trees(rng, B, N, Dmax, V) if V > 1 else chain_trees(B, N, Dmax)
    hidden, w = W.make_head(B, N, d, V, device="cuda", seed=V + d, kind="int", tree_tokens=tree["tree_tokens"],
                            tree_parent=tree["tree_parent"], n_nodes=tree["n_nodes"], plant_p=plant,
                            density=density)
    cfg = W.Config("lmh", 0, n_prompts=B, seqs_per_prompt=1, vocab=V, rollouts_per_prompt=0,
                   rollout_len=W.Dist("fixed", 1), ctx_len=W.Dist("fixed", 1), n_nodes=N, max_depth=Dmax,
                   hq=1, hkv=1, head_dim=64)
    gumbel = W.make_gumbel(cfg, B, device="cuda", seed=V + 5) if sampled else None
    got = run_fused(hidden, w, gumbel, inv_t, tree, Dmax)
    want = oracle_rows(hidden, w, gumbel, inv_t, tree, range(B), Dmax)
    for b in range(B):
        assert_accept_equal(got, b, want[b], Dmax)
    assert_same(got, run_materialised(hidden, w, gumbel, inv_t, tree, Dmax), B)
    if plant >= 0.8 or V == 1:
        assert got["n_accepted"].max() >= 2  # the walks do go deep


def test_depth_cap_root_only_and_clamped_counts():
    rng = random.Random(5)
    B, N, V, d, Dmax = 6, 10, 300, 64, 3
    tree = random_trees(rng, B, N, 9, V)  # deeper than Dmax on purpose
    tree["n_nodes"] = tree["n_nodes"].copy()
    tree["n_nodes"][0] = 1      # root only
    tree["n_nodes"][1] = 0      # clamped to 1
    tree["n_nodes"][2] = 999    # clamped to N
    hidden, w = W.make_head(B, N, d, V, device="cuda", seed=9, kind="int", tree_tokens=tree["tree_tokens"],
                            tree_parent=tree["tree_parent"], n_nodes=np.minimum(np.maximum(tree["n_nodes"], 1), N),
                            plant_p=1.0)
    for Dm in (0, Dmax):
        got = run_fused(hidden, w, None, 1.0, tree, Dm)
        want = oracle_rows(hidden, w, None, 1.0, tree, range(B), Dm)
        for b in range(B):
            assert_accept_equal(got, b, want[b], Dm)
        assert got["n_accepted"].max() <= Dm
    assert got["n_accepted"][0] == 0 and got["n_accepted"][1] == 0


def test_scratch_reuse_across_sizes():
    rng = random.Random(11)
    scratch = torch.empty(srt.srt_accept_lmhead_scratch_bytes(300, 16, 3000), dtype=torch.uint8, device="cuda")
    for B, V, d, seed in ((300, 3000, 128, 1), (17, 700, 64, 2), (300, 3000, 128, 1)):
        N, Dmax = 16, 6
        tree = random_trees(random.Random(seed), B, N, Dmax, V)
        hidden, w = W.make_head(B, N, d, V, device="cuda", seed=seed, kind="int",
                                tree_tokens=tree["tree_tokens"], tree_parent=tree["tree_parent"],
                                n_nodes=tree["n_nodes"], plant_p=0.9)
        got = run_fused(hidden, w, None, 1.0, tree, Dmax, scratch=scratch)
        assert_same(got, run_fused(hidden, w, None, 1.0, tree, Dmax), B)
        want = oracle_rows(hidden, w, None, 1.0, tree, range(B), Dmax)
        for b in range(B):
            assert_accept_equal(got, b, want[b], Dmax)


def check_valid_walk(got, b, h, wn, g, inv_t, tree, Dmax):
    """Every step of the GPU walk of sequence b is a valid choice: its token
    scores within the fp32 summation bound of the best score, it descends
    exactly when a child carries the token, and it stops at Dmax."""
    tt, tp = tree["tree_tokens"][b], tree["tree_parent"][b]
    n = min(max(int(tree["n_nodes"][b]), 1), tt.shape[0])
    k = int(got["n_accepted"][b])
    toks = got["out_tokens"][b]
    nodes = got["out_nodes"][b]
    u = 0
    for s in range(k + 1):
        exact = wn.astype(np.float64) @ h[u].astype(np.float64)
        err = LH.logit_error_bound(h[u], wn)
        x = exact * inv_t if g is not None else exact
        tol = err * (inv_t if g is not None else 1.0)
        if g is not None:
            x = x + g[b, s].astype(np.float64)
        tol = tol + 4 * U32 * np.abs(x) + 1e-30  # roundings of the product and the sum
        t = int(toks[s])
        j = int(np.argmax(x))
        assert 0 <= t < wn.shape[0], (b, s, t)
        assert x[t] >= x[j] - (tol[t] + tol[j]), (b, s, t, j, x[t], x[j])
        child = [c for c in range(u + 1, n) if tp[c] == u and tt[c] == t]
        if s < k:
            assert child and int(nodes[s]) == child[0], (b, s)
            u = child[0]
        else:
            assert not child or s == Dmax, (b, s)
    assert int(got["n_emitted"][b]) == k + 1


@pytest.mark.parametrize("V,d,sampled", [(5000, 256, False), (5000, 256, True), (32000, 1024, True)])
def test_real_valued_walks_valid(V, d, sampled):
    rng = random.Random(V + d)
    B, N, Dmax = 48, 32, 8
    say(f"lmhead real-valued: V={V} d={d} sampled={sampled}")
    tree = random_trees(rng, B, N, Dmax, V)
    hidden, w = W.make_head(B, N, d, V, device="cuda", seed=V * 3 + d, kind="normal",
                            tree_tokens=tree["tree_tokens"], tree_parent=tree["tree_parent"],
                            n_nodes=tree["n_nodes"], plant_p=0.8)
    cfg = W.Config("lmh", 0, n_prompts=B, seqs_per_prompt=1, vocab=V, rollouts_per_prompt=0,
                   rollout_len=W.Dist("fixed", 1), ctx_len=W.Dist("fixed", 1), n_nodes=N, max_depth=Dmax,
                   hq=1, hkv=1, head_dim=64)
    gumbel = W.make_gumbel(cfg, B, device="cuda", seed=V + 7) if sampled else None
    got = run_fused(hidden, w, gumbel, 1.0, tree, Dmax)
    h = hidden.float().cpu().numpy()
    wn = w.float().cpu().numpy()
    g = None if gumbel is None else gumbel.cpu().numpy()
    for b in range(B):
        check_valid_walk(got, b, h[b], wn, g, 1.0, tree, Dmax)
    want = oracle_rows(hidden, w, gumbel, 1.0, tree, range(B), Dmax)
    same = sum(int(got["n_accepted"][b]) == want[b][0] and got["out_tokens"][b, :want[b][0] + 1].tolist() == want[b][1]
               for b in range(B))
    assert same >= B - 2, same
    assert got["n_accepted"].max() >= 2


def test_qwen7b_head_sampled():
    """The 7B-shaped head and batch: V = 152064, d_model = 3584, B = 256,
    N = 64, Dmax = 12, T = 1 Gumbel; integer inputs so that every sequence
    can be compared bit for bit."""
    V, d, B, N, Dmax = 152064, 3584, 256, 64, 12
    rng = random.Random(7)
    say("lmhead qwen7b-shaped: building inputs")
    tree = random_trees(rng, B, N, Dmax, V)
    hidden, w = W.make_head(B, N, d, V, device="cuda", seed=77, kind="int", tree_tokens=tree["tree_tokens"],
                            tree_parent=tree["tree_parent"], n_nodes=tree["n_nodes"], plant_p=0.9)
    cfg = W.Config("lmh7b", 0, n_prompts=B, seqs_per_prompt=1, vocab=V, rollouts_per_prompt=0,
                   rollout_len=W.Dist("fixed", 1), ctx_len=W.Dist("fixed", 1), n_nodes=N, max_depth=Dmax,
                   hq=1, hkv=1, head_dim=64)
    gumbel = W.make_gumbel(cfg, B, device="cuda", seed=78)
    say("lmhead qwen7b-shaped: fused walk")
    got = run_fused(hidden, w, gumbel, 1.0, tree, Dmax)
    say("lmhead qwen7b-shaped: materialised logits + srt_accept")
    assert_same(got, run_materialised(hidden, w, gumbel, 1.0, tree, Dmax), B)
    deep = int(np.argmax(got["n_accepted"]))
    seqs = sorted({deep, 0, B - 1, 131})
    say(f"lmhead qwen7b-shaped: oracle on {seqs} (deepest walk {got['n_accepted'][deep]})")
    wn = w.float().cpu().numpy()
    for b in seqs:
        n = int(tree["n_nodes"][b])
        rows = LH.head_logits(hidden[b, :n].float().cpu().numpy(), wn)  # every node of the tree, fp64 -> fp32
        g = gumbel[b].cpu().numpy()
        want = AC.accept(lambda u: rows[u], lambda k: g[k], 1.0, tree["tree_tokens"][b], tree["tree_parent"][b],
                         n, Dmax)
        assert_accept_equal(got, b, want, Dmax)
    assert got["n_accepted"].max() >= 4
