"""Pins for the on-demand LM-head acceptance oracle (oracle/lmhead.py): the
head's logits against exact rational sums (brute force), a one-hot head that
reduces the walk to the pinned logits walk, designed hidden states whose
walks are known by construction, the summation error bound against other
fp32 orders, and planted mistakes (a transposed head, a dropped noise term,
a wrong noise row)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import accept as AC
from oracle import lmhead as LH


def bf16_round(x):
    """Nearest bf16 value (round to nearest even) of fp32 values, as fp32."""
    a = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    a = (a + 0x7FFF + ((a >> 16) & 1)) & 0xFFFF0000
    return a.astype(np.uint32).view(np.float32)


def test_bf16_round_helper():
    # bf16 keeps 8 significant bits: 1 + 2^-8 rounds to 1 (tie to even), 1 + 3*2^-8 to 1 + 2^-6.
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 3.0e-3], dtype=np.float32)
    r = bf16_round(x)
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == np.float32(1 + 2 ** -6) and r[3] == -2.5
    assert abs(float(r[4]) - 3.0e-3) <= 3.0e-3 * 2 ** -8


def test_head_logits_brute_force_rationals():
    rng = np.random.default_rng(3)
    V, d = 9, 7
    W = bf16_round(rng.standard_normal((V, d)).astype(np.float32))
    h = bf16_round(rng.standard_normal(d).astype(np.float32))
    got = LH.head_logits(h, W)
    for j in range(V):
        exact = sum(Fraction(float(W[j, k])) * Fraction(float(h[k])) for k in range(d))
        assert got[j] == np.float32(float(exact)), j  # one rounding of the exact sum


def test_head_logits_integer_inputs_exact():
    rng = np.random.default_rng(4)
    V, d = 50, 600
    W = rng.integers(-3, 4, size=(V, d)).astype(np.float32)
    h = rng.integers(-3, 4, size=d).astype(np.float32)
    want = [int(sum(int(W[j, k]) * int(h[k]) for k in range(d))) for j in range(V)]
    assert LH.head_logits(h, W).tolist() == [float(x) for x in want]


def test_one_hot_head_reduces_to_logits_walk():
    """w_head[j] = e_{pi(j)} makes logit_j(u) = hidden[u, pi(j)]: the walk must
    be the pinned logits walk over those rows, greedy and with noise."""
    rng = np.random.default_rng(5)
    V = d = 40
    pi = rng.permutation(d)
    W = np.zeros((V, d), dtype=np.float32)
    W[np.arange(V), pi] = 1.0
    N, Dmax = 12, 5
    hidden = bf16_round(rng.standard_normal((N, d)).astype(np.float32))
    tokens = [int(x) for x in rng.integers(0, V, size=N)]
    parents = [-1] + [int(rng.integers(0, i)) for i in range(1, N)]
    G = rng.gumbel(size=(Dmax + 1, V)).astype(np.float32)
    rows = lambda u: hidden[u][pi]
    for noise in (None, lambda k: G[k]):
        for inv_t in (1.0, 0.5):
            got = LH.accept_lmhead(hidden, W, noise, inv_t, tokens, parents, N, Dmax)
            assert got == AC.accept(rows, noise, inv_t, tokens, parents, N, Dmax)


def test_designed_walk_follows_planted_path():
    """Hidden state of node u points at a chosen token t(u) (W = identity,
    V = d): the greedy walk must follow the path on which every node's child
    carries t(parent) and stop with the first t(u) no child carries."""
    V = d = 16
    W = np.eye(V, dtype=np.float32)
    # chain 0 -> 1 -> 2 -> 3 plus decoys; t(u) is the token each node picks
    tokens = [5, 7, 9, 11, 3, 2]
    parents = [-1, 0, 1, 2, 0, 1]
    pick = {0: 7, 1: 9, 2: 11, 3: 13, 4: 0, 5: 0}
    hidden = np.zeros((6, d), dtype=np.float32)
    for u, t in pick.items():
        hidden[u, t] = 1.0
    k, toks, nodes = LH.accept_lmhead(hidden, W, None, 1.0, tokens, parents, 6, 8)
    assert (k, toks, nodes) == (3, [7, 9, 11, 13], [1, 2, 3])
    k, toks, nodes = LH.accept_lmhead(hidden, W, None, 1.0, tokens, parents, 6, 2)  # depth cap
    assert (k, toks, nodes) == (2, [7, 9, 11], [1, 2])


def test_error_bound_covers_other_orders():
    """Any fp32 summation order (sequential, reversed, pairwise, blocked by
    16) stays within logit_error_bound of the oracle's logits."""
    rng = np.random.default_rng(6)
    V, d = 64, 1024
    W = bf16_round((0.05 * rng.standard_normal((V, d))).astype(np.float32))
    h = bf16_round(rng.standard_normal(d).astype(np.float32))
    ref = LH.head_logits(h, W).astype(np.float64)
    bound = LH.logit_error_bound(h, W)
    prods = (W * h[None, :]).astype(np.float32)  # exact: bf16 x bf16 fits fp32

    def seq(p):
        s = np.float32(0)
        for x in p:
            s = np.float32(s + x)
        return s

    def pairwise(p):
        p = list(p)
        while len(p) > 1:
            p = [np.float32(p[i] + p[i + 1]) if i + 1 < len(p) else p[i] for i in range(0, len(p), 2)]
        return p[0]

    def blocked(p):
        acc = np.float32(0)
        for i in range(0, len(p), 16):
            acc = np.float32(acc + seq(p[i:i + 16]))
        return acc

    worst = 0.0
    for j in range(V):
        for f in (seq, lambda p: seq(p[::-1]), pairwise, blocked):
            err = abs(float(f(prods[j])) - ref[j])
            assert err <= bound[j], (j, err, bound[j])
            worst = max(worst, err / bound[j])
    assert worst > 0.0  # the orders do differ from the oracle somewhere


def _seq32(p):
    s = np.float32(0)
    for x in p:
        s = np.float32(s + x)
    return s


@pytest.mark.parametrize("d", [64, 1024, 3584])
def test_error_bound_is_tight_on_a_worst_case_order(d):
    """Closed-form worst case: products 1, t, t, ..., t with t = 255 2^-32,
    just below half an ulp of 1 (2^-24).  Sequential fp32 summation rounds
    every addition down, so it returns exactly 1; the exact sum is
    1 + (d - 1) t and the oracle rounds that once.  The observed error is
    therefore known, and the bound must cover it while staying within its
    own safety factor of 2 (plus the one rounding term): a bound inflated by
    a few percent, or one that ignored the (d - 1) additions, fails here."""
    h = np.full(d, np.float32(255 * 2.0 ** -20), dtype=np.float32)  # 255/256 * 2^-12: bf16
    h[0] = 1.0
    W = np.full((1, d), np.float32(2.0 ** -12), dtype=np.float32)
    W[0, 0] = 1.0
    assert np.array_equal(bf16_round(h), h) and np.array_equal(bf16_round(W), W)
    prods = (W[0] * h).astype(np.float32)
    t = np.float32(255 * 2.0 ** -32)
    assert prods[0] == 1.0 and (prods[1:] == t).all() and t < 2.0 ** -24
    assert _seq32(prods) == np.float32(1.0)  # every addition rounds down
    exact = Fraction(1) + (d - 1) * Fraction(255, 2 ** 32)
    ref = LH.head_logits(h, W)[0]
    assert ref == np.float32(float(exact))  # one rounding of the exact sum
    err = float(ref) - 1.0
    assert err > 0.0
    bound = float(LH.logit_error_bound(h, W)[0])
    assert err <= bound <= 2.05 * err, (d, err, bound, bound / err)


def test_planted_mistakes_fail():
    rng = np.random.default_rng(7)
    V, d, N, Dmax = 24, 24, 10, 4
    W = bf16_round(rng.standard_normal((V, d)).astype(np.float32))
    hidden = bf16_round(rng.standard_normal((N, d)).astype(np.float32))
    G = (4.0 * rng.gumbel(size=(Dmax + 1, V))).astype(np.float32)
    parents = [-1] + [int(rng.integers(0, i)) for i in range(1, N)]
    # tree tokens: every node's first child carries the parent's noisy choice
    pickn = lambda u, depth, Wm, noise_k: int(np.argmax(
        (LH.head_logits(hidden[u], Wm) + (G[noise_k] if noise_k is not None else 0)).astype(np.float32)))
    depth = [0] * N
    for c in range(1, N):
        depth[c] = depth[parents[c]] + 1
    tokens = [0] * N
    seen = set()
    for c in range(1, N):
        p = parents[c]
        tokens[c] = pickn(p, depth[p], W, depth[p]) if p not in seen else int(rng.integers(0, V))
        seen.add(p)
    noise = lambda k: G[k]
    good = LH.accept_lmhead(hidden, W, noise, 1.0, tokens, parents, N, Dmax)
    assert good[0] >= 1
    # transposed head, dropped noise, noise row of the wrong step: each changes the walk
    assert LH.accept_lmhead(hidden, W.T.copy(), noise, 1.0, tokens, parents, N, Dmax) != good
    assert LH.accept_lmhead(hidden, W, None, 1.0, tokens, parents, N, Dmax) != good
    assert LH.accept_lmhead(hidden, W, lambda k: G[min(k + 1, Dmax)], 1.0, tokens, parents, N, Dmax) != good


def test_batch_clamps_node_counts():
    rng = np.random.default_rng(8)
    B, N, V, d, Dmax = 3, 5, 11, 8, 3
    W = rng.integers(-2, 3, size=(V, d)).astype(np.float32)
    hidden = rng.integers(-2, 3, size=(B, N, d)).astype(np.float32)
    tt = rng.integers(0, V, size=(B, N))
    tp = np.tile(np.array([-1, 0, 1, 2, 3]), (B, 1))
    res = LH.accept_lmhead_batch(hidden, W, None, 1.0, tt, tp, [0, 5, 99], Dmax)
    for b, n in ((0, 1), (1, 5), (2, 5)):
        assert res[b] == LH.accept_lmhead(hidden[b], W, None, 1.0, tt[b], tp[b], n, Dmax)
    assert res[0][0] == 0 and len(res[0][1]) == 1  # a root-only tree emits just the bonus


def test_head_logits_rows_match_single():
    rng = np.random.default_rng(9)
    W = bf16_round(rng.standard_normal((300, 64)).astype(np.float32))
    H = bf16_round(rng.standard_normal((5, 64)).astype(np.float32))
    many = LH.head_logits(H, W)
    assert many.shape == (5, 300)
    for i in range(5):
        assert np.array_equal(many[i], LH.head_logits(H[i], W))
