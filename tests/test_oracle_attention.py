"""Pins for the tree-attention oracle (oracle/attention.py): hand-worked
closed forms, a pure-Python loop version, torch's fp64 scaled-dot-product
attention with an explicit boolean mask, causal attention for a chain tree,
decode attention for a one-node tree, and invariance under page
permutation."""
import json
import math
import os
import random

import numpy as np
import pytest
import torch

from oracle import attention as A


def paged(kpos, vpos, page, hkv=1, rng=None):
    """Scatter [n_pos, Hkv, d] position arrays into a shuffled page pool."""
    kpos, vpos = np.asarray(kpos, float), np.asarray(vpos, float)
    if kpos.ndim == 2:
        kpos, vpos = kpos[:, None, :], vpos[:, None, :]
    n, hkv, d = kpos.shape
    npg = (n + page - 1) // page
    perm = np.arange(npg) if rng is None else rng.permutation(npg)
    kc = np.zeros((npg, hkv, page, d)); vc = np.zeros_like(kc)
    for j in range(n):
        kc[perm[j // page], :, j % page] = kpos[j]
        vc[perm[j // page], :, j % page] = vpos[j]
    return kc, vc, perm


def test_golden(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "attention_small.json")))
    kc, vc, bt = paged(g["k_positions"], g["v_positions"], g["page"])
    n = len(g["tree_parent"])
    q = np.zeros((n, 1, 2))
    out = A.tree_attention_seq(q, kc, vc, bt, g["ctx_len"], g["tree_parent"], n, g["scale"], g["page"])
    np.testing.assert_allclose(out[:, 0, :], g["q_zero"]["out"], rtol=0, atol=1e-15)
    q[0, 0] = g["q_node0"]
    out = A.tree_attention_seq(q, kc, vc, bt, g["ctx_len"], g["tree_parent"], n, g["scale"], g["page"])
    np.testing.assert_allclose(out[0, 0], g["q_node0_out"], rtol=1e-14)


def random_tree(rng, n):
    return [-1] + [rng.randrange(i) for i in range(1, n)]


def loop_attention(q, kpos, vpos, L, parent, scale):
    """Textbook per-row loops with math.exp, no numpy."""
    n, Hq, d = len(q), len(q[0]), len(q[0][0])
    Hkv = len(kpos[0]); G = Hq // Hkv
    out = [[[0.0] * d for _ in range(Hq)] for _ in range(n)]
    for i in range(n):
        anc = set(); j = i
        while j >= 0:
            anc.add(j); j = parent[j]
        keys = list(range(L)) + [L + j for j in sorted(anc)]
        for h in range(Hq):
            g = h // G
            s = [sum(q[i][h][c] * kpos[p][g][c] for c in range(d)) * scale for p in keys]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            z = sum(w)
            for c in range(d):
                out[i][h][c] = sum(w[t] * vpos[keys[t]][g][c] for t in range(len(keys))) / z
    return out


@pytest.mark.parametrize("seed", range(8))
def test_matches_python_loops(seed):
    rng = random.Random(seed); nrng = np.random.default_rng(seed)
    n, L, Hkv, G, d, page = rng.randrange(1, 7), rng.randrange(0, 9), rng.choice([1, 2]), rng.choice([1, 3]), 4, rng.choice([1, 2, 4])
    Hq = Hkv * G
    parent = random_tree(rng, n)
    kpos = nrng.standard_normal((L + n, Hkv, d)); vpos = nrng.standard_normal((L + n, Hkv, d))
    q = nrng.standard_normal((n, Hq, d))
    kc, vc, bt = paged(kpos, vpos, page, rng=nrng)
    got = A.tree_attention_seq(q, kc, vc, bt, L, parent, n, 0.5, page)
    want = loop_attention(q.tolist(), kpos.tolist(), vpos.tolist(), L, parent, 0.5)
    np.testing.assert_allclose(got, np.array(want), rtol=1e-12, atol=1e-12)


def sdpa(q, k, v, mask, scale):
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=None if mask is None else torch.from_numpy(mask), scale=scale).numpy()


@pytest.mark.parametrize("seed", range(6))
def test_matches_torch_sdpa_with_mask(seed):
    rng = random.Random(50 + seed); nrng = np.random.default_rng(50 + seed)
    n, L, Hkv, G, d, page = rng.randrange(1, 20), rng.randrange(1, 60), 2, 3, 16, 16
    Hq = Hkv * G
    parent = random_tree(rng, n)
    kpos = nrng.standard_normal((L + n, Hkv, d)); vpos = nrng.standard_normal((L + n, Hkv, d))
    q = nrng.standard_normal((n, Hq, d))
    kc, vc, bt = paged(kpos, vpos, page, rng=nrng)
    got = A.tree_attention_seq(q, kc, vc, bt, L, parent, n, 1 / math.sqrt(d), page)
    vis = np.ones((n, L + n), dtype=bool)
    for i in range(n):
        j = i
        while j >= 0:
            vis[i, L + j] = True; j = parent[j]
        for j in range(n):
            anc = False; a = i
            while a >= 0:
                anc |= a == j; a = parent[a]
            vis[i, L + j] = anc
    kh = np.repeat(kpos.transpose(1, 0, 2), G, axis=0)  # [Hq, L+n, d]
    vh = np.repeat(vpos.transpose(1, 0, 2), G, axis=0)
    want = sdpa(q.transpose(1, 0, 2).copy(), kh.copy(), vh.copy(), vis, 1 / math.sqrt(d))
    np.testing.assert_allclose(got, want.transpose(1, 0, 2), rtol=1e-10, atol=1e-12)


def test_chain_tree_is_causal_attention():
    nrng = np.random.default_rng(3)
    n, L, d, page = 9, 13, 8, 4
    parent = [-1] + list(range(n - 1))
    kpos = nrng.standard_normal((L + n, 1, d)); vpos = nrng.standard_normal((L + n, 1, d))
    q = nrng.standard_normal((n, 1, d))
    kc, vc, bt = paged(kpos, vpos, page, rng=nrng)
    got = A.tree_attention_seq(q, kc, vc, bt, L, parent, n, 0.3, page)
    # queries sit at positions L..L+n-1 of a causal sequence of length L+n
    qf = np.zeros((1, L + n, d)); qf[0, L:] = q[:, 0]
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(qf), torch.from_numpy(kpos[:, 0][None].copy()), torch.from_numpy(vpos[:, 0][None].copy()),
        is_causal=True, scale=0.3).numpy()[0, L:]
    np.testing.assert_allclose(got[:, 0], want, rtol=1e-10, atol=1e-12)


def test_single_node_is_decode_attention():
    nrng = np.random.default_rng(4)
    L, d, page = 37, 8, 16
    kpos = nrng.standard_normal((L + 1, 2, d)); vpos = nrng.standard_normal((L + 1, 2, d))
    q = nrng.standard_normal((1, 4, d))
    kc, vc, bt = paged(kpos, vpos, page, rng=nrng)
    got = A.tree_attention_seq(q, kc, vc, bt, L, [-1], 1, 0.25, page)
    kh = np.repeat(kpos.transpose(1, 0, 2), 2, axis=0); vh = np.repeat(vpos.transpose(1, 0, 2), 2, axis=0)
    want = sdpa(q.transpose(1, 0, 2).copy(), kh.copy(), vh.copy(), None, 0.25)
    np.testing.assert_allclose(got, want.transpose(1, 0, 2), rtol=1e-10, atol=1e-12)


def test_page_permutation_invariance():
    nrng = np.random.default_rng(5); rng = random.Random(5)
    n, L, d, page = 12, 50, 8, 4
    parent = random_tree(rng, n)
    kpos = nrng.standard_normal((L + n, 1, d)); vpos = nrng.standard_normal((L + n, 1, d))
    q = nrng.standard_normal((n, 2, d))
    outs = []
    for s in range(3):
        kc, vc, bt = paged(kpos, vpos, page, rng=np.random.default_rng(s))
        outs.append(A.tree_attention_seq(q, kc, vc, bt, L, parent, n, 0.4, page))
    np.testing.assert_array_equal(outs[0], outs[1]); np.testing.assert_array_equal(outs[0], outs[2])


def test_planted_mask_mistake_is_caught(golden_dir, monkeypatch):
    # a mask that lets every node see all tree nodes fails the golden closed form
    g = json.load(open(os.path.join(golden_dir, "attention_small.json")))
    monkeypatch.setattr(A, "ancestors", lambda parent, n: np.ones((n, n), dtype=bool))
    kc, vc, bt = paged(g["k_positions"], g["v_positions"], g["page"])
    out = A.tree_attention_seq(np.zeros((3, 1, 2)), kc, vc, bt, g["ctx_len"], g["tree_parent"], 3, 1.0, 2)
    assert not np.allclose(out[:, 0, :], g["q_zero"]["out"])
