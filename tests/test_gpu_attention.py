"""GPU parity of srt_tree_attn against the fp64 oracle: elementwise
|gpu - ref| <= 1e-2 + 2e-2 |ref| over every output row, for the tiny
configuration and for shapes that span several key tiles, ragged tails,
split contexts (with the combine pass), both head sizes, GQA ratios 1-7,
256-node trees, one-node trees, empty contexts and pages of 16-256 tokens."""
import math
import random

import numpy as np
import pytest
import torch

from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from tests.gpu_util import assert_attn_close, oracle_attention_seq, say

pytestmark = pytest.mark.gpu


class Case:
    """Random attention inputs with explicit trees (no cache needed)."""

    def __init__(self, seed, B, N, hq, hkv, d, ctx, n_nodes=None, page=16):
        rng = random.Random(seed)
        self.cfg = W.Config("attn", 0, n_prompts=B, seqs_per_prompt=1, vocab=8, rollouts_per_prompt=0,
                            rollout_len=W.Dist("fixed", 1), ctx_len=W.Dist("fixed", 1), n_nodes=N,
                            max_depth=63, hq=hq, hkv=hkv, head_dim=d, page=page)
        ctx = np.asarray(ctx, dtype=np.int32)
        self.q, self.k_cache, self.v_cache, bt, self.num_pages = W.make_kv(self.cfg, ctx, device="cuda", seed=seed)
        self.block_table = bt.to(torch.int32)
        self.scale = 1.0 / math.sqrt(d)
        nn = [rng.randrange(1, N + 1) for _ in range(B)] if n_nodes is None else list(n_nodes)
        par = np.full((B, N), -1, dtype=np.int32)
        for b in range(B):
            for i in range(1, nn[b]):
                par[b, i] = rng.randrange(max(0, i - 6), i) if rng.random() < 0.8 else rng.randrange(i)
        self.parent = par
        self.n_nodes = np.asarray(nn, dtype=np.int32)
        self.ctx = ctx

        class Tok:
            pass
        self.tokens = Tok()
        self.tokens.ctx_len = ctx

    def run(self):
        t = lambda a: torch.as_tensor(a, device="cuda")
        return srt.srt_tree_attn(self.q, self.k_cache, self.v_cache, self.block_table, t(self.ctx),
                                 t(self.parent), t(self.n_nodes), self.scale)

    def check(self, out, seqs=None):
        o = out.float().cpu().numpy()
        seqs = range(len(self.ctx)) if seqs is None else seqs
        worst = 0.0
        for b in seqs:
            n = int(self.n_nodes[b])
            ref = oracle_attention_seq(self, b, self.parent[b], n)
            e, _ = assert_attn_close(o[b, :n], ref, f"seq {b} (ctx {self.ctx[b]}, n {n})")
            worst = max(worst, e)
        return worst


def test_tiny_config_shape():
    say("attn: tiny config shape (Hq 4, Hkv 1, d 64, N 8)")
    rng = np.random.default_rng(0)
    c = Case(1, 4, 8, 4, 1, 64, rng.integers(128, 513, size=4))
    c.check(c.run())


@pytest.mark.parametrize("d,hq,hkv", [(128, 12, 2), (128, 28, 4), (64, 4, 1), (128, 8, 8), (64, 14, 2)])
def test_shapes_ragged(d, hq, hkv):
    say(f"attn: d={d} hq={hq} hkv={hkv}")
    ctx = [0, 1, 15, 16, 63, 64, 65, 200, 1000, 3001]
    c = Case(7, len(ctx), 32, hq, hkv, d, ctx)
    c.check(c.run())


def test_split_contexts_and_combine():
    # contexts longer than one split exercise the partial + combine path; a
    # batch this small gets 1024-key splits, and the lengths sit on and
    # around split (1024 and 8192) and tile boundaries
    say("attn: split contexts")
    ctx = [4088, 8192 - 64 - 7, 8192 - 64, 8192, 9000, 12345, 16384 - 30, 25000, 100]
    c = Case(11, len(ctx), 64, 28, 4, 128, ctx)
    c.check(c.run())


def test_split_contexts_8192_key_splits():
    # B * Hkv = 256 with 16k-key capacity keeps the largest (8192-key) splits
    say("attn: 8192-key splits")
    base = [8192 - 64 - 7, 8192, 9000, 12345, 16354, 100, 5000, 8193]
    ctx = [base[i % len(base)] for i in range(32)]
    c = Case(31, len(ctx), 4, 8, 8, 128, ctx)
    c.check(c.run(), seqs=[0, 1, 2, 3, 4, 5, 6, 7, 12, 20])


@pytest.mark.parametrize("B,split", [(16, 4096), (8, 2048)])
def test_split_contexts_mid_size_splits(B, split):
    # B * Hkv = 128 / 64 with 16k-key capacity: the call picks 4096- / 2048-key
    # splits; lengths on and around those boundaries
    say(f"attn: {split}-key splits")
    base = [split - 1, split, split + 1, 2 * split - 64, 3 * split + 5, 16000, 100, 7]
    ctx = [base[i % len(base)] for i in range(B)]
    c = Case(37 + B, B, 8, 8, 8, 128, ctx)
    c.check(c.run(), seqs=list(range(len(base))))


@pytest.mark.parametrize("page,d", [(32, 128), (64, 128), (64, 64), (128, 128), (256, 64)])
def test_larger_pages(page, d):
    # pages of 32 to 256 tokens: a 64-key tile spans two pages or lies inside
    # one, ragged tails and split contexts included
    say(f"attn: page {page}, d={d}")
    ctx = [0, 31, 32, 33, 63, 64, 65, 1000, 9000, 4097]
    c = Case(43 + page, len(ctx), 16, 8, 2, d, ctx, page=page)
    c.check(c.run())


def test_split_contexts_d64():
    say("attn: split contexts, d=64")
    ctx = [8200, 17000, 3]
    c = Case(29, len(ctx), 32, 14, 2, 64, ctx)
    c.check(c.run())


def test_wide_tree_256_nodes():
    say("attn: 256-node trees")
    ctx = [300, 5000, 17]
    c = Case(13, 3, 256, 28, 4, 128, ctx, n_nodes=[256, 200, 256])
    c.check(c.run())


def test_one_node_and_chain():
    say("attn: one-node trees (decode) and chains")
    ctx = [5, 700, 4200]
    c = Case(17, 3, 16, 12, 2, 128, ctx, n_nodes=[1, 1, 16])
    c.parent[2] = np.arange(-1, 15)
    c.check(c.run())


def test_qwen1p5b_shape_full_batch():
    cfg = W.CONFIGS["qwen1.5b"]
    tw = W.make_tokens(cfg)
    say("attn: 1.5B-shaped layer, 64 sequences, 1k-4k contexts, full batch")
    c = Case(19, cfg.batch, cfg.n_nodes, cfg.hq, cfg.hkv, cfg.head_dim, tw.ctx_len)
    c.check(c.run())


def test_deterministic():
    ctx = [100, 5000, 9000]
    c = Case(23, 3, 64, 28, 4, 128, ctx)
    say("attn: determinism")
    a = c.run().clone()
    for _ in range(3):
        o = c.run()
        for b in range(3):  # rows >= n_nodes are not written
            n = int(c.n_nodes[b])
            assert torch.equal(a[b, :n], o[b, :n])
