"""Sanity of the seeded input generator (shared by both sides)."""
import numpy as np

from paper_2601_09083_amd import workload as W


def test_mutation_rates():
    rng = np.random.default_rng(0)
    base = rng.integers(0, 1000, size=200000)
    same = W.mutate(np.random.default_rng(1), base, 1000, 0.0, 0.0, 0.0)
    assert np.array_equal(same, base)
    sub = W.mutate(np.random.default_rng(2), base, 1000, 0.1, 0.0, 0.0)
    assert sub.shape == base.shape and abs((sub != base).mean() - 0.1) < 0.01
    indel = W.mutate(np.random.default_rng(3), base, 1000, 0.0, 0.02, 0.02)
    assert abs(indel.shape[0] / base.shape[0] - 1.0) < 0.01


def test_deterministic_and_shaped():
    cfg = W.CONFIGS["tiny"]
    a, b = W.make_tokens(cfg), W.make_tokens(cfg)
    assert all(np.array_equal(x, y) for x, y in zip(a.seqs, b.seqs))
    assert a.batch == 4 and len(a.prior) == 4 and all(len(p) == 8 for p in a.prior)
    assert all(len(s) == 256 for p in a.prior for s in p)
    assert np.all((a.ctx_len >= 128) & (a.ctx_len <= 512))
    assert all(len(y) == L + 1 for y, L in zip(a.seqs, a.ctx_len))
    tail = a.ctx_tail()
    assert tail.shape == (4, cfg.max_match) and np.array_equal(tail[0], a.seqs[0][-cfg.max_match:])


def test_lognormal_lengths():
    d = W.Dist("lognormal", 4096, 32768)
    v = d.sample(np.random.default_rng(0), 100000)
    assert v.min() >= 16 and v.max() <= 32768 and abs(np.median(v) - 4096) < 100


def test_dense_inputs_cpu():
    cfg = W.CONFIGS["tiny"]
    tw = W.make_tokens(cfg)
    q, k, v, bt, P = W.make_kv(cfg, tw.ctx_len)
    assert q.shape == (4, 8, 4, 64) and k.shape == (P, 1, 16, 64)
    used = bt[bt >= 0].numpy()
    assert np.array_equal(np.sort(used), np.arange(P))
    g = W.make_gumbel(cfg, 4)
    assert g.shape == (4, cfg.max_depth + 1, cfg.vocab) and bool(g.isfinite().all())
