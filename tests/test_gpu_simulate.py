"""The acceptance simulation harness (paper_2601_09083_amd/simulate.py,
Section 4's comparison of cache maintenance strategies, Fig. 4) on a small
GRPO-shaped group, through libsrt and through the oracle.

Every strategy (history-only, on-the-fly, on-the-fly + run-ahead) and
drafting variant (chain, score threshold, alpha budget) runs the loop on the
GPU (srt_draft -> srt_accept -> srt_trie_insert -> srt_commit) and, with the
same toy greedy target, step by step on the CPU: the cache as the occurrence
counts of the streams inserted so far (oracle/trie), the draft
(oracle/draft), the acceptance walk (oracle/accept) and the growth of each
sequence's stream by its emitted tokens (the online insertion and commit).
Per step and per sequence, the accepted counts and the tree sizes must be
identical; inside run() every committed token must be the sequence's true
continuation."""
import numpy as np
import pytest

from oracle import accept as AC
from oracle import draft as DR
from oracle import trie as TR
from paper_2601_09083_amd import simulate as SIM
from paper_2601_09083_amd import workload as W
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

CFG = W.Config("sim_small", 8, n_prompts=4, seqs_per_prompt=4, vocab=4096, rollouts_per_prompt=8,
               rollout_len=W.Dist("uniform", 400, 1200), ctx_len=W.Dist("uniform", 200, 800), n_nodes=32,
               max_depth=8, hq=4, hkv=1, head_dim=64)


def oracle_replay(cfg, sim, steps, strategy, alpha=0.0, min_score=0.0, chain=False, n_nodes=None):
    """The simulation loop on the oracle: per step, [B] accepted counts and
    tree sizes."""
    N = cfg.n_nodes if n_nodes is None else n_nodes
    tw = sim.tokens
    B, Q, D = tw.batch, cfg.max_match, cfg.trie_depth
    seqs = [np.array(y) for y in tw.seqs]
    used = np.zeros(B, dtype=np.int64)
    acc_rec, node_rec = [], []
    for _ in range(steps):
        tries = {}
        for p in range(cfg.n_prompts):
            streams = list(tw.prior[p])
            if strategy != "history":  # the running rollouts are in the cache and grow online
                streams += [seqs[b] for b in range(B) if tw.seq_prompt[b] == p]
            if strategy == "runahead":
                streams += list(sim.runahead[p])
            tries[p] = TR.StreamTrie(streams, D)
        acc_k, node_k = [], []
        for b in range(B):
            y = seqs[b]
            tail = y[-Q:]
            tok, par, dep, n, q = DR.draft(tries[int(tw.seq_prompt[b])], tail, len(y), Q, N, cfg.max_depth,
                                           alpha, min_score, chain)
            fut = sim.future[b]
            target = [int(fut[min(used[b] + d, fut.shape[0] - 1)]) for d in dep]

            def row(u):
                r = np.zeros(cfg.vocab, dtype=np.float32)
                r[target[u]] = 1.0
                return r
            k, out, nodes = AC.accept(row, None, 1.0, tok, par, n, cfg.max_depth)
            seqs[b] = np.concatenate([y, np.array(out, dtype=y.dtype)])
            used[b] += len(out)
            acc_k.append(k)
            node_k.append(n)
        acc_rec.append(acc_k)
        node_rec.append(node_k)
    return np.array(acc_rec), np.array(node_rec)


@pytest.mark.parametrize("strategy,variant", [("history", {}), ("onthefly", {}), ("runahead", {}),
                                              ("onthefly", {"chain": True, "n_nodes": 9}),
                                              ("onthefly", {"min_score": 0.1}), ("onthefly", {"alpha": 2.0})])
def test_simulation_matches_oracle(strategy, variant):
    steps = 12
    say(f"simulate: {strategy} {variant}")
    sim = SIM.make_sim_tokens(CFG, future_len=(steps + 2) * (CFG.max_depth + 1), runahead_per_prompt=2)
    r = SIM.run(CFG, sim, steps, strategy, record=True, **variant)
    assert 0.0 <= r["mean_accepted_per_step"] <= r["mean_tree_nodes"] - 1.0 + 1e-9
    assert r["mean_emitted_per_step"] == pytest.approx(r["mean_accepted_per_step"] + 1.0)
    assert r["mean_accepted_per_step"] > 0.2, "drafts from mutated rollouts should often be accepted"
    want_acc, want_nodes = oracle_replay(CFG, sim, steps, strategy, **variant)
    got_acc, got_nodes = np.array(r["per_step_accepted"]), np.array(r["per_step_nodes"])
    assert np.array_equal(got_nodes, want_nodes), "tree sizes differ from the oracle's"
    assert np.array_equal(got_acc, want_acc), "accepted counts differ from the oracle's"
    say(f"  equal over {steps} steps x {CFG.batch} sequences: accepted/step {want_acc.mean():.3f}, "
        f"tree nodes {want_nodes.mean():.2f}")

