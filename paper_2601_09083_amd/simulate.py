"""Acceptance simulations on the GPU path: cache maintenance strategies and
drafting variants.

Section 4 ("Effect of On-the-Fly Updates and Run-Ahead Generation") compares
a history-only cache (completed responses of earlier epochs only) with
SRT's online insertion of the running rollouts' tokens and with run-ahead
rollouts inserted during idle time, by the mean number of accepted tokens
per decoding step.  Section 3 leaves the form of the budget B(q) open.  This
module runs the verification loop (srt_draft -> srt_accept -> srt_trie_insert
-> srt_commit, all through libsrt) on synthetic GRPO-shaped rollouts with a
toy greedy target and reports, per strategy or drafting variant, the mean
accepted drafted tokens per step, the emitted tokens per step and the tree
size.

Toy target.  Every running sequence is a prefix of one longer rollout of its
prompt (a mutation of the prompt's base sequence, like every other rollout);
the rest of that rollout is the sequence's true continuation.  The target's
greedy token at a tree node of depth d is the continuation's token d
positions ahead, so the acceptance walk accepts exactly the longest drafted
path that agrees with the true continuation and emits its next token as the
bonus token.  Logits are one-hot rows built on the device from that rule; the
attention pass is left out (it does not change what is accepted).

    python -m paper_2601_09083_amd.simulate [--steps 48] [--which all|strategies|variants]
"""
from __future__ import annotations

import argparse
import json
import time
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np
import torch

from . import workload as W
from .pipeline import VerifyState

# GRPO-shaped group (Section 4.1's DAPO/GRPO settings: several responses per
# prompt in flight at once), with a reduced vocabulary so that the one-hot
# target rows stay small; token ids are uniform over it as in every config.
SIM_CONFIG = W.Config("sim_grpo", 7, n_prompts=32, seqs_per_prompt=8, vocab=32768, rollouts_per_prompt=16,
                      rollout_len=W.Dist("lognormal", 2048, 16384), ctx_len=W.Dist("lognormal", 2048, 16384),
                      n_nodes=64, max_depth=12, hq=12, hkv=2, head_dim=128)


@dataclass
class SimTokens:
    tokens: W.TokenWorkload
    future: np.ndarray             # [B, F] true continuation of every running sequence
    runahead: List[List[np.ndarray]]  # per prompt: run-ahead rollouts


def make_sim_tokens(cfg: W.Config, future_len: int, runahead_per_prompt: int = 4, seed: int = 77) -> SimTokens:
    """Prior rollouts as in the benchmark workloads; each running sequence is
    the first ctx + 1 tokens of a fresh mutation of its prompt's base, and
    its next ``future_len`` tokens are kept as the true continuation."""
    tw = W.make_tokens(cfg)
    ss = np.random.SeedSequence(seed)
    s_seq, s_run = ss.spawn(2)
    mut = dict(vocab=cfg.vocab, p_sub=cfg.p_sub, p_del=cfg.p_del, p_ins=cfg.p_ins)
    B = tw.batch
    future = np.zeros((B, future_len), dtype=np.int32)
    seqs = []
    for b, sd in enumerate(s_seq.spawn(B)):
        rng = np.random.Generator(np.random.PCG64(sd))
        need = int(tw.ctx_len[b]) + 1 + future_len
        base = tw.bases[int(tw.seq_prompt[b])]
        if base.shape[0] < int(need * 1.1) + 64:  # extend the base with fresh tokens if needed
            extra = rng.integers(0, cfg.vocab, size=int(need * 1.1) + 64 - base.shape[0])
            base = np.concatenate([base, extra])
            tw.bases[int(tw.seq_prompt[b])] = base
        r = W.mutate(rng, base[: int(need * 1.1) + 64], **mut)
        while r.shape[0] < need:
            r = np.concatenate([r, rng.integers(0, cfg.vocab, size=need - r.shape[0])])
        seqs.append(r[: need - future_len].copy())
        future[b] = r[need - future_len: need]
    tw.seqs = seqs
    runahead = []
    for p, sd in enumerate(s_run.spawn(cfg.n_prompts)):
        rngs = [np.random.Generator(np.random.PCG64(x)) for x in sd.spawn(runahead_per_prompt)]
        runahead.append([W.mutate(rg, tw.bases[p], **mut) for rg in rngs])
    return SimTokens(tw, future, runahead)


class ContinuationTarget:
    """Per-step logits and Gumbel noise for a decode loop in which every
    running sequence follows its true continuation (``SimTokens.future``).

    The logits are fixed random N(0, sigma) rows [B, N, V] plus ``boost`` at
    each node's continuation token -- the token depth(u) positions past what
    the sequence has committed -- written in place each step and restored to
    the saved values the next, so the walk accepts exactly the drafted path
    that agrees with the continuation and the bonus token continues it.  The
    noise is read at a step-dependent offset of a buffer one sequence larger
    than [B, Dmax+1, V], so consecutive steps see different noise without new
    draws.  All of it is a stand-in for the policy (no part of the method)."""

    def __init__(self, st, future: np.ndarray, boost: float = 100.0, sampled: bool = True, seed: int = 4321):
        cfg, B, dev = st.cfg, st.tokens.batch, st.device
        N, V, D1 = cfg.n_nodes, cfg.vocab, cfg.max_depth + 1
        none = np.full((B, N), -1, dtype=np.int32)
        self.logits = W.make_logits(cfg, none, none, np.ones(B, dtype=np.int32), device=dev, seed=seed,
                                    boost="none")
        self.noise = W.make_gumbel(cfg, B + 1, device=dev, seed=seed + 1) if sampled else None
        self.future = torch.as_tensor(future, device=dev).long()
        self.used = torch.zeros(B, dtype=torch.int64, device=dev)
        self.rowbase = (torch.arange(B * N, device=dev, dtype=torch.int64) * V).view(B, N)
        self.flat = None
        self.saved = None
        self.boost = float(boost)
        self.shape = (B, D1, V)

    def apply(self, st, step: int):
        """Logits and noise for the trees just drafted (call after draft)."""
        flat_l = self.logits.view(-1)
        if self.flat is not None:
            flat_l[self.flat] = self.saved
        depth = st.tree["tree_depth"].long().clamp(min=0)
        pos = (self.used[:, None] + depth).clamp(max=self.future.shape[1] - 1)
        tok = torch.gather(self.future, 1, pos)
        self.flat = (self.rowbase + tok).view(-1)
        self.saved = flat_l[self.flat]
        flat_l[self.flat] = self.saved + self.boost
        st.logits = self.logits
        if self.noise is not None:
            B, D1, V = self.shape
            off = (step * 104729) % (D1 * V) // 4 * 4  # 16-byte aligned, as a caller's tensor is
            st.gumbel = self.noise.view(-1)[off: off + B * D1 * V].view(B, D1, V)
        else:
            st.gumbel = None

    def advance(self, st):
        """Account the tokens the step emitted (call after accept)."""
        self.used += st.acc["n_emitted"].long()


def run(cfg: W.Config, sim: SimTokens, steps: int, strategy: str = "onthefly", alpha: float = 0.0,
        min_score: float = 0.0, chain: bool = False, n_nodes: Optional[int] = None, device: str = "cuda",
        record: bool = False) -> Dict:
    """One simulation: ``strategy`` is "history" (prior rollouts only, no
    online insertion), "onthefly" (running rollouts inserted as they grow)
    or "runahead" (on-the-fly plus the run-ahead rollouts inserted first).
    With ``record`` the result also holds every step's per-sequence accepted
    counts and tree sizes ("per_step_accepted", "per_step_nodes", [steps, B]
    int lists)."""
    if strategy not in ("history", "onthefly", "runahead"):
        raise ValueError(strategy)
    if n_nodes is not None:
        cfg = cfg.scaled(n_nodes=n_nodes)
    tw = W.TokenWorkload(cfg, sim.tokens.bases, sim.tokens.prior, sim.tokens.seq_prompt,
                         [np.array(y) for y in sim.tokens.seqs], sim.tokens.ctx_len.copy())
    st = VerifyState.build(cfg, device=device, tokens=tw, steps_headroom=steps + 4,
                           with_seqs=strategy != "history", kv_headroom=(steps + 4) * (cfg.max_depth + 1))
    if strategy == "runahead":
        ids = st.caches.new_streams(sum(len(r) for r in sim.runahead))
        st.caches.insert([p for p, rs in enumerate(sim.runahead) for _ in rs], ids,
                         [x for rs in sim.runahead for x in rs])
    B, N, V = tw.batch, cfg.n_nodes, cfg.vocab
    future = torch.as_tensor(sim.future, device=device)
    used = torch.zeros(B, dtype=torch.int64, device=device)  # continuation tokens committed so far
    logits = torch.empty((B, N, V), dtype=torch.float32, device=device)
    st.gumbel = None
    acc_sum = torch.zeros(B, dtype=torch.int64, device=device)
    emit_sum = torch.zeros(B, dtype=torch.int64, device=device)
    node_sum = torch.zeros(B, dtype=torch.int64, device=device)
    rec_acc = torch.zeros((steps, B), dtype=torch.int32, device=device)
    rec_nodes = torch.zeros((steps, B), dtype=torch.int32, device=device)
    t0 = time.perf_counter()
    for k in range(steps):
        tree = st.draft(alpha=alpha, min_score=min_score, chain=chain)
        depth = tree["tree_depth"].long().clamp(min=0)
        pos = (used[:, None] + depth).clamp(max=sim.future.shape[1] - 1)
        target = torch.gather(future, 1, pos)  # [B, N] the target's token at each node
        logits.zero_()
        logits.scatter_(2, target[:, :, None].long(), 1.0)
        st.logits = logits
        acc = st.accept()
        if strategy != "history":
            st.insert()
        st.commit()
        used += acc["n_emitted"].long()
        acc_sum += acc["n_accepted"].long()
        emit_sum += acc["n_emitted"].long()
        node_sum += tree["n_nodes"].long()
        if record:
            rec_acc[k].copy_(acc["n_accepted"])
            rec_nodes[k].copy_(tree["n_nodes"])
    torch.cuda.synchronize()
    secs = time.perf_counter() - t0
    # the committed tokens must be the true continuation: check every
    # sequence's draft tail against its rollout
    used_np = used.cpu().numpy()
    tails = st.ctx_tail.cpu().numpy()
    Q = cfg.max_match
    for b in range(B):
        grown = np.concatenate([tw.seqs[b], sim.future[b, : used_np[b]]])
        assert (tails[b] == grown[-Q:]).all(), f"sequence {b} left its true continuation"
    assert int(used_np.max()) <= sim.future.shape[1], "continuation too short for this many steps"
    res = {
        "strategy": strategy, "alpha": alpha, "min_score": min_score, "chain": chain, "n_nodes": N,
        "steps": steps, "sequences": B,
        "mean_accepted_per_step": float(acc_sum.sum()) / (B * steps),
        "mean_emitted_per_step": float(emit_sum.sum()) / (B * steps),
        "mean_tree_nodes": float(node_sum.sum()) / (B * steps),
        "seconds": secs,
    }
    res["accepted_per_drafted"] = res["mean_accepted_per_step"] / max(res["mean_tree_nodes"] - 1.0, 1e-9)
    if record:
        res["per_step_accepted"] = rec_acc.cpu().numpy().tolist()
        res["per_step_nodes"] = rec_nodes.cpu().numpy().tolist()
    del st
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=48)
    ap.add_argument("--which", default="all", choices=["all", "strategies", "variants"])
    args = ap.parse_args()
    cfg = SIM_CONFIG
    sim = make_sim_tokens(cfg, future_len=(args.steps + 2) * (cfg.max_depth + 1))
    runs = []
    if args.which in ("all", "strategies"):
        for strategy in ("history", "onthefly", "runahead"):
            runs.append(run(cfg, sim, args.steps, strategy))
            print(json.dumps(runs[-1]), flush=True)
    if args.which in ("all", "variants"):
        variants = [dict(n_nodes=n) for n in (2, 4, 8, 16, 32, 64, 128)]
        variants += [dict(chain=True, n_nodes=13), dict(alpha=1.0), dict(alpha=2.0), dict(alpha=4.0)]
        variants += [dict(min_score=t) for t in (0.02, 0.05, 0.1, 0.2, 0.4)]
        for v in variants:
            runs.append(run(cfg, sim, args.steps, "onthefly", **v))
            print(json.dumps(runs[-1]), flush=True)
    return runs


if __name__ == "__main__":
    main()
