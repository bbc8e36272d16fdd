"""End-to-end parity of the verification step (draft -> tree attention ->
acceptance -> online insertion) against the oracle.

* tiny configuration: every sequence, two consecutive steps (the second
  drafts from the cache updated by the first);
* the four large configurations at full size, in the launch configuration
  the benchmark times: the whole batch runs on the GPU and EVERY sequence is
  recomputed by the oracle -- draft trees, acceptance walks and the commit
  bit for bit, attention element-wise against fp64 (largest errors printed);
  cache contents are checked exactly for the prompt of the longest context
  (or, for the long-tail prompt, on sampled strings plus per-depth
  occurrence totals)."""
import gc

import numpy as np
import pytest
import torch

from oracle import trie as TR
from paper_2601_09083_amd import workload as W
from paper_2601_09083_amd.pipeline import VerifyState
from tests.gpu_util import (ErrorLog, assert_accept_equal, assert_attn_close, assert_tree_equal,
                            oracle_accept_rows, oracle_attention_many, oracle_attention_seq, oracle_draft_rows,
                            oracle_trie, say, tree_to_np)

pytestmark = pytest.mark.gpu


def overlay(tree_np, oracle_rows, N):
    """Tree arrays with the oracle's rows written over the sampled sequences."""
    t = {k: v.copy() for k, v in tree_np.items()}
    for b, (tok, par, dep, n, q) in oracle_rows.items():
        t["tree_tokens"][b] = -1; t["tree_parent"][b] = -1; t["tree_depth"][b] = -1
        t["tree_tokens"][b, :n], t["tree_parent"][b, :n], t["tree_depth"][b, :n] = tok, par, dep
        t["n_nodes"][b], t["match_len"][b] = n, q
    return t


def oracle_tree_arrays(rows, B, N):
    t = {k: np.full((B, N), -1, np.int32) for k in ("tree_tokens", "tree_parent", "tree_depth")}
    t["n_nodes"] = np.zeros(B, np.int32); t["match_len"] = np.zeros(B, np.int32)
    return overlay(t, rows, N)


@pytest.mark.parametrize("sampled", [False, True])
def test_tiny_two_steps(sampled):
    cfg = W.CONFIGS["tiny"]
    st = VerifyState.build(cfg)
    tw = st.tokens
    B = tw.batch
    streams = [list(tw.prior[p]) for p in range(cfg.n_prompts)]
    seqs = [np.array(y) for y in tw.seqs]
    for step in range(2):
        say(f"step: tiny sampled={sampled} step={step}")
        tries = [oracle_trie(streams[p] + [seqs[b] for b in range(B) if tw.seq_prompt[b] == p], cfg.trie_depth)
                 for p in range(cfg.n_prompts)]
        rows = oracle_draft_rows(st, tries, range(B))
        tree = tree_to_np(st.draft())
        for b in range(B):
            assert_tree_equal(tree, b, rows[b])
        ot = oracle_tree_arrays(rows, B, cfg.n_nodes)
        st.logits = W.make_logits(cfg, ot["tree_tokens"], ot["tree_parent"], ot["n_nodes"], device="cuda",
                                  boost="top", seed=100 + step)
        st.gumbel = W.make_gumbel(cfg, B, device="cuda", seed=200 + step) if sampled else None
        out = st.attention().float().cpu().numpy()
        for b in range(B):
            n = int(ot["n_nodes"][b])
            assert_attn_close(out[b, :n], oracle_attention_seq(st, b, ot["tree_parent"][b], n), f"seq {b}")
        acc = {k: v.cpu().numpy() for k, v in st.accept().items()}
        want = oracle_accept_rows(st.logits, st.gumbel, 1.0, ot, range(B), cfg.max_depth)
        for b in range(B):
            assert_accept_equal(acc, b, want[b], cfg.max_depth)
        st.insert()
        for b in range(B):
            seqs[b] = np.concatenate([seqs[b], np.array(want[b][1])])
        for p in range(cfg.n_prompts):
            allp = streams[p] + [seqs[b] for b in range(B) if tw.seq_prompt[b] == p]
            assert st.caches.export(p) == TR.substring_counts(allp, cfg.trie_depth)
    assert st.caches.status()["flags"] == 0


FULL = ("qwen1.5b", "grpo", "qwen7b", "longtail")


def seq_rows(cache, bt_row, positions, page):
    """[len(positions), Hkv, d] int16 bits of one sequence's logical positions."""
    pos = torch.as_tensor(positions, dtype=torch.long, device=cache.device)
    pages = bt_row.long()[pos // page]
    return cache[pages, :, pos % page, :].view(torch.int16).cpu().numpy()


def check_commit(st, acc, sample):
    """srt_commit over the whole batch; the sampled sequences' tree window,
    lengths and draft tails are compared with the oracle's commit."""
    from oracle import commit as CM
    c = st.cfg
    L = st.attn_len.cpu().numpy().astype(np.int64)
    t = st.draft_len.cpu().numpy().astype(np.int64)
    tails = st.ctx_tail.cpu().numpy()
    before = {b: (seq_rows(st.k_cache, st.block_table[b], np.arange(L[b], L[b] + c.n_nodes), c.page),
                  seq_rows(st.v_cache, st.block_table[b], np.arange(L[b], L[b] + c.n_nodes), c.page)) for b in sample}
    st.commit()
    torch.cuda.synchronize()
    k_acc = acc["n_accepted"]
    assert st.attn_len.cpu().numpy().tolist() == (L + k_acc + 1).tolist()
    assert st.draft_len.cpu().numpy().tolist() == (t + k_acc + 1).tolist()
    new_tails = st.ctx_tail.cpu().numpy()
    for b in sample:
        win = np.arange(L[b], L[b] + c.n_nodes)
        for cache, old in zip((st.k_cache, st.v_cache), before[b]):
            want, _ = CM.commit_kv(old, 0, int(k_acc[b]), acc["out_nodes"][b])
            assert np.array_equal(seq_rows(cache, st.block_table[b], win, c.page), want), f"seq {b}"
        row, _ = CM.commit_tail(tails[b], int(t[b]), acc["out_tokens"][b, :k_acc[b] + 1])
        assert new_tails[b].tolist() == row.tolist(), f"seq {b}"


@pytest.mark.parametrize("name", FULL)
def test_full_size_every_sequence(name):
    import time
    cfg = W.CONFIGS[name]
    say(f"full-size {name}: building caches, KV and queries")
    st = VerifyState.build(cfg)
    tw = st.tokens
    B = tw.batch
    every = list(range(B))
    p_long = int(tw.seq_prompt[int(np.argmax(tw.ctx_len))])
    prompts = sorted(set(int(p) for p in tw.seq_prompt))
    t0 = time.time()
    tries = {p: oracle_trie(tw.streams_of_prompt(p), cfg.trie_depth, big=True) for p in prompts}
    say(f"full-size {name}: draft, all {B} sequences")
    tree = tree_to_np(st.draft())
    rows = oracle_draft_rows(st, tries, every)
    for b in every:
        assert_tree_equal(tree, b, rows[b])
    assert tree["n_nodes"].mean() > 2, "drafts should mostly succeed on this workload"
    say(f"full-size {name}: drafts equal ({time.time() - t0:.1f} s); attention")
    out = st.attention()
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    t0 = time.time()
    refs = oracle_attention_many(st, every, {b: rows[b][1] for b in every}, {b: rows[b][3] for b in every})
    log = ErrorLog(f"full-size {name}")
    for b in every:
        log.add(o[b, :rows[b][3]], refs.pop(b), f"seq {b}")
    log.done()
    say(f"full-size {name}: attention within tolerance ({time.time() - t0:.1f} s); "
        f"acceptance (logits {B}x{cfg.n_nodes}x{cfg.vocab})")
    del o, out
    t_in = overlay(tree, rows, cfg.n_nodes)
    # "top" boost (each node's first-child token set to the row maximum + 40
    # with p = 0.7, enough to beat the Gumbel maximum over the vocabulary) so
    # that walks go deep and every level of the walk is checked
    st.logits = W.make_logits(cfg.scaled(boost_add=40.0), t_in["tree_tokens"], t_in["tree_parent"],
                              t_in["n_nodes"], device="cuda", boost="top")
    st.gumbel = W.make_gumbel(cfg, B, device="cuda")
    acc = {k: v.cpu().numpy() for k, v in st.accept().items()}
    say(f"full-size {name}: emitted per sequence {acc['n_emitted'].mean():.2f}, deepest {acc['n_emitted'].max()}")
    want = oracle_accept_rows(st.logits, st.gumbel, 1.0, t_in, every, cfg.max_depth)
    for b in every:
        assert_accept_equal(acc, b, want[b], cfg.max_depth)
    st.logits = st.gumbel = None
    torch.cuda.empty_cache()
    say(f"full-size {name}: insertion")
    st.insert()
    say(f"full-size {name}: commit, all {B} sequences")
    check_commit(st, acc, every)
    if cfg.runahead_streams:
        ids = st.caches.new_streams(B)
        st.caches.insert(tw.seq_prompt, ids, tw.runahead)
    assert st.caches.status()["flags"] == 0
    p = p_long
    rng = np.random.default_rng(cfg.index)
    streams = list(tw.prior[p]) + [np.concatenate([tw.seqs[b], acc["out_tokens"][b, :acc["n_accepted"][b] + 1]])
                                   for b in range(B) if tw.seq_prompt[b] == p]
    if cfg.runahead_streams:
        streams += [tw.runahead[b] for b in range(B) if tw.seq_prompt[b] == p]
    say(f"full-size {name}: cache contents of prompt {p}")
    got = st.caches.export(p)
    D = cfg.trie_depth
    if sum(len(s) for s in streams) * D < 3_000_000:
        assert got == TR.substring_counts(streams, D)
    else:
        for ell in range(1, D + 1):  # per-depth occurrence totals
            assert sum(c for s, c in got.items() if len(s) == ell) == sum(max(0, len(s) - ell + 1) for s in streams)
        big = TR.StreamTrie(streams, D)
        keys = list(got)
        for i in rng.choice(len(keys), 300, replace=False):
            assert got[keys[i]] == big.count(keys[i])
    del st
    gc.collect()
    torch.cuda.empty_cache()
