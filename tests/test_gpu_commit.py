"""GPU parity of srt_commit (accepted path's K/V moved into place, context and
draft tail advanced) against oracle/commit.py, bit-exact.

* random caches with paths that overlap their own destinations (node c_i = j
  for i < j), identity paths, empty paths, paths of Dmax nodes, short and
  empty draft tails, d = 64 / 128, one to four KV heads, pages of 1, 16, 32
  and 64 tokens; the whole cache
  (including pages of other sequences and unused pages) is compared;
* the tiny configuration run as a real decode loop for three steps: each
  step's draft is checked against the oracle drafting from the grown
  sequences, attention against the fp64 oracle on the committed cache,
  acceptance, and the commit itself."""
import numpy as np
import pytest
import torch

from oracle import commit as CM
from oracle import trie as TR
from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from paper_2601_09083_amd.pipeline import VerifyState
from tests.gpu_util import (assert_accept_equal, assert_attn_close, assert_tree_equal, oracle_accept_rows,
                            oracle_draft_rows, oracle_trie, say, tree_to_np)

pytestmark = pytest.mark.gpu


def logical(cache_np, bt_row, n_pos, page):
    idx = np.arange(n_pos)
    return cache_np[bt_row[idx // page], :, idx % page, :]


def expected_cache(cache_np, bt, L, k_acc, nodes, n_pos, page):
    """The oracle's commit applied to every sequence of a host cache copy."""
    out = cache_np.copy()
    for b in range(bt.shape[0]):
        seq = logical(cache_np, bt[b], n_pos[b], page)
        new, _ = CM.commit_kv(seq, int(L[b]), int(k_acc[b]), nodes[b])
        idx = np.arange(n_pos[b])
        out[bt[b][idx // page], :, idx % page, :] = new
    return out


def bits(t):
    return t.view(torch.int16).cpu().numpy()


@pytest.mark.parametrize("d,Hkv,page", [(64, 1, 16), (128, 4, 16), (128, 2, 16), (128, 2, 32), (64, 3, 64), (128, 1, 1)])
def test_commit_random(d, Hkv, page):
    say(f"commit random d={d} Hkv={Hkv} page={page}")
    rng = np.random.default_rng(100 * d + Hkv + 7 * page)
    B, N, Dmax, Qmax = 9, 24, 6, 5
    L = rng.integers(0, 120, B).astype(np.int32)
    L[0] = 0
    pages_per = (L + N + page - 1) // page
    P = int(pages_per.sum()) + 5  # a few pages no sequence uses
    perm = rng.permutation(P).astype(np.int32)
    bt = np.full((B, int(pages_per.max())), -1, np.int32)
    off = 0
    for b in range(B):
        bt[b, :pages_per[b]] = perm[off: off + pages_per[b]]
        off += pages_per[b]
    paths = [[], [1, 2, 3], [2, 3, 4], [3, 5, 9, 12], [1, 4, 6, 7, 20, 23], [2], [5, 6], [1, 2, 3, 4, 5, 6],
             [7, 8, 9, 10, 11, 12]]
    k_acc = np.array([len(p) for p in paths], np.int32)
    nodes = np.full((B, Dmax + 1), -1, np.int32)
    toks = np.full((B, Dmax + 1), -1, np.int32)
    for b, p in enumerate(paths):
        nodes[b, :len(p)] = p
        toks[b, :len(p) + 1] = rng.integers(0, 1000, len(p) + 1)
    t = np.array([0, 1, 3, 5, 9, 40, 2, 100, 4], np.int32)
    tail = np.full((B, Qmax), -1, np.int32)
    for b in range(B):
        m = min(int(t[b]), Qmax)
        if m:
            tail[b, Qmax - m:] = rng.integers(0, 1000, m)
    dev = "cuda"
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    kc = torch.randn((P, Hkv, page, d), generator=g, device=dev).to(torch.bfloat16)
    vc = torch.randn((P, Hkv, page, d), generator=g, device=dev).to(torch.bfloat16)
    k0, v0 = bits(kc), bits(vc)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    ctx_len, tail_d, t_d = T(L), T(tail), T(t)
    srt.srt_commit(kc, vc, T(bt), ctx_len, T(k_acc), T(toks), T(nodes), N, ctx_tail=tail_d, draft_len=t_d)
    torch.cuda.synchronize()
    n_pos = L + N
    assert np.array_equal(bits(kc), expected_cache(k0, bt, L, k_acc, nodes, n_pos, page))
    assert np.array_equal(bits(vc), expected_cache(v0, bt, L, k_acc, nodes, n_pos, page))
    assert ctx_len.cpu().numpy().tolist() == (L + k_acc + 1).tolist()
    for b in range(B):
        row, tt = CM.commit_tail(tail[b], int(t[b]), toks[b, :k_acc[b] + 1])
        assert tail_d[b].cpu().numpy().tolist() == row.tolist(), f"tail of seq {b}"
        assert int(t_d[b]) == tt


def test_commit_without_tail_and_empty_batch():
    dev = "cuda"
    kc = torch.zeros((4, 1, 16, 64), dtype=torch.bfloat16, device=dev)
    vc = torch.zeros_like(kc)
    bt = torch.arange(4, dtype=torch.int32, device=dev).view(1, 4)
    ctx = torch.tensor([10], dtype=torch.int32, device=dev)
    kc.view(-1, 64)[12] = 3.0  # node 2 of the tree at position 10 + 2
    srt.srt_commit(kc, vc, bt, ctx, torch.tensor([1], dtype=torch.int32, device=dev),
                   torch.tensor([[5, 6, -1]], dtype=torch.int32, device=dev),
                   torch.tensor([[2, -1, -1]], dtype=torch.int32, device=dev), 8)
    torch.cuda.synchronize()
    assert int(ctx[0]) == 12 and float(kc.view(-1, 64)[11, 0]) == 3.0
    e = torch.empty(0, dtype=torch.int32, device=dev)
    srt.srt_commit(kc, vc, bt[:0], e, e, e.view(0, 3), e.view(0, 3), 8)


@pytest.mark.parametrize("sampled", [False, True])
def test_tiny_decode_loop(sampled):
    cfg = W.CONFIGS["tiny"]
    steps = 3
    st = VerifyState.build(cfg, kv_headroom=steps * (cfg.max_depth + 1))
    tw = st.tokens
    B, page = tw.batch, cfg.page
    streams = [list(tw.prior[p]) for p in range(cfg.n_prompts)]
    seqs = [np.array(y) for y in tw.seqs]
    L = tw.ctx_len.astype(np.int64).copy()
    bt = st.block_table.cpu().numpy()
    grown = False
    for step in range(steps):
        say(f"tiny decode loop sampled={sampled} step={step}")
        tries = [oracle_trie(streams[p] + [seqs[b] for b in range(B) if tw.seq_prompt[b] == p], cfg.trie_depth)
                 for p in range(cfg.n_prompts)]
        tw.seqs = seqs  # the oracle drafts from the grown sequences
        rows = oracle_draft_rows(st, tries, range(B))
        tree = tree_to_np(st.draft())
        for b in range(B):
            assert_tree_equal(tree, b, rows[b])
        st.logits = W.make_logits(cfg, tree["tree_tokens"], tree["tree_parent"], tree["n_nodes"], device="cuda",
                                  boost="top", seed=300 + step)
        st.gumbel = W.make_gumbel(cfg, B, device="cuda", seed=400 + step) if sampled else None
        out = st.attention().float().cpu().numpy()
        from oracle import attention as AT
        for b in range(B):
            n = int(tree["n_nodes"][b])
            npg = (int(L[b]) + n + page - 1) // page
            pages = st.block_table[b, :npg].long()
            ref = AT.tree_attention_seq(st.q[b].float().cpu().numpy(), st.k_cache[pages].float().cpu().numpy(),
                                        st.v_cache[pages].float().cpu().numpy(), np.arange(npg), int(L[b]),
                                        tree["tree_parent"][b], n, st.scale, page)
            assert_attn_close(out[b, :n], ref, f"step {step} seq {b}")
        acc = {k: v.cpu().numpy() for k, v in st.accept().items()}
        want = oracle_accept_rows(st.logits, st.gumbel, 1.0, tree, range(B), cfg.max_depth)
        for b in range(B):
            assert_accept_equal(acc, b, want[b], cfg.max_depth)
        k0, v0 = bits(st.k_cache), bits(st.v_cache)
        st.insert()
        st.commit()
        n_pos = L + cfg.n_nodes
        k_acc = acc["n_accepted"]
        assert np.array_equal(bits(st.k_cache), expected_cache(k0, bt, L, k_acc, acc["out_nodes"], n_pos, page))
        assert np.array_equal(bits(st.v_cache), expected_cache(v0, bt, L, k_acc, acc["out_nodes"], n_pos, page))
        L = L + k_acc + 1
        assert st.attn_len.cpu().numpy().tolist() == L.tolist()
        for b in range(B):
            seqs[b] = np.concatenate([seqs[b], np.array(want[b][1])])
            grown |= want[b][0] > 0
        assert st.draft_len.cpu().numpy().tolist() == [len(y) for y in seqs]
        assert st.ctx_tail.cpu().numpy().tolist() == W.TokenWorkload.ctx_tail(tw).tolist()
    assert grown, "the loop should accept drafted tokens with top-boosted logits"
    for p in range(cfg.n_prompts):
        allp = streams[p] + [seqs[b] for b in range(B) if tw.seq_prompt[b] == p]
        assert st.caches.export(p) == TR.substring_counts(allp, cfg.trie_depth)
