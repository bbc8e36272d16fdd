"""GPU parity of the cache (srt_trie_insert / srt_trie_export) against the
oracle's substring counts, bit-exact: full inserts, chunked online inserts,
order independence, depths 1, 2 and 64, segments longer than a workgroup,
and the sticky error flags."""
import random

import numpy as np
import pytest
import torch

from oracle import trie as TR
from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from paper_2601_09083_amd.pipeline import Caches
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def build(streams_by_prompt, D, chunks=None, rng=None, capacity=None):
    """Insert every stream (optionally split into random chunks over several
    calls, in random order) and return the Caches."""
    P = len(streams_by_prompt)
    n_streams = sum(len(s) for s in streams_by_prompt)
    total = sum(len(x) for s in streams_by_prompt for x in s)
    cap = capacity if capacity is not None else total * D + 64
    c = Caches.create(P, n_streams + 4, D, cap)
    items = [(p, st) for p in range(P) for st in streams_by_prompt[p]]
    ids = c.new_streams(len(items))
    if chunks is None:
        c.insert([p for p, _ in items], ids, [st for _, st in items])
    else:
        pos = [0] * len(items)
        while any(pos[i] < len(items[i][1]) for i in range(len(items))):
            sel = [i for i in range(len(items)) if pos[i] < len(items[i][1]) or rng.random() < 0.1]
            rng.shuffle(sel)
            segs = []
            for i in sel:
                k = rng.randrange(0, chunks + 1)
                segs.append(items[i][1][pos[i]:pos[i] + k])
                pos[i] += k
            c.insert([items[i][0] for i in sel], ids[sel], segs)
    return c


def check_prompt(c, p, streams, D):
    got = c.export(p)
    want = TR.substring_counts(streams, D)
    assert got == want, f"prompt {p}: {len(got)} vs {len(want)} strings"


def test_tiny_config_cache_exact():
    cfg = W.CONFIGS["tiny"]
    tw = W.make_tokens(cfg)
    say("cache: tiny config, full insert")
    streams = [tw.streams_of_prompt(p) for p in range(cfg.n_prompts)]
    c = build(streams, cfg.trie_depth)
    assert c.status()["flags"] == 0
    for p in range(cfg.n_prompts):
        check_prompt(c, p, streams[p], cfg.trie_depth)


@pytest.mark.parametrize("seed", range(3))
def test_chunked_online_insert_equals_full(seed):
    rng = random.Random(seed)
    D = rng.choice([3, 6, 12])
    streams = [[np.array([rng.randrange(4) for _ in range(rng.randrange(0, 120))]) for _ in range(5)]
               for _ in range(3)]
    say(f"cache: chunked inserts seed={seed} D={D}")
    c = build(streams, D, chunks=7, rng=rng)
    assert c.status()["flags"] == 0
    for p in range(3):
        check_prompt(c, p, streams[p], D)


def test_long_streams_small_vocab():
    rng = np.random.default_rng(5)
    D = 20
    streams = [[rng.integers(0, 3, size=3000) for _ in range(4)], [rng.integers(0, 50, size=2000)]]
    say("cache: long streams, vocab 3")
    c = build(streams, D)
    for p in range(2):
        check_prompt(c, p, streams[p], D)


def test_flags_and_stream_reset():
    D = 4
    c = Caches.create(2, 8, D, 1000)
    say("cache: flags")
    c.insert([0], np.array([0], np.int32), [np.array([1, 2, 3])])
    c.insert([1], np.array([0], np.int32), [np.array([4, 5])])          # stream 0 belongs to prompt 0
    st = c.status()
    assert st["flags"] & srt.SRT_FLAG_STREAM and not st["flags"] & srt.SRT_FLAG_CAPACITY
    assert c.export(1) == {}
    c.insert([2], np.array([1], np.int32), [np.array([4])])             # prompt out of range
    assert c.status()["flags"] & srt.SRT_FLAG_PROMPT
    c.insert([0], np.array([99], np.int32), [np.array([4])])            # stream out of range
    srt.srt_trie_reset_streams(c.ws, torch.tensor([0], dtype=torch.int32, device="cuda"))
    c.insert([1], np.array([0], np.int32), [np.array([4, 5])])          # rebinding after reset works
    assert c.export(1) == TR.substring_counts([[4, 5]], D)
    assert c.export(0) == TR.substring_counts([[1, 2, 3]], D)
    c.insert([0], np.array([2], np.int32), [np.array([], dtype=np.int64)])  # empty segment
    assert c.export(0) == TR.substring_counts([[1, 2, 3]], D)
    c.insert([0], np.array([3], np.int32), [np.array([1, -2, 3])])      # negative token: entry rejected
    assert c.export(0) == TR.substring_counts([[1, 2, 3]], D)


def test_capacity_overflow_is_sticky():
    D = 8
    c = Caches.create(1, 4, D, 50)
    say("cache: capacity overflow")
    c.insert([0], np.array([0], np.int32), [np.arange(100) % 37])
    st = c.status()
    assert st["status"] == srt.SRT_ERR_CAPACITY and st["flags"] & srt.SRT_FLAG_CAPACITY
    before = st["nodes"]
    c.insert([0], np.array([1], np.int32), [np.arange(40)])
    assert c.status()["nodes"] == before  # later inserts are dropped


def test_export_truncation_reports_capacity():
    D = 3
    c = Caches.create(1, 2, D, 1000)
    c.insert([0], np.array([0], np.int32), [np.array([1, 2, 3, 4, 5])])
    with pytest.raises(srt.SrtError) as e:
        srt.srt_trie_export(c.ws, 0, 4)
    assert e.value.status == srt.SRT_ERR_CAPACITY


@pytest.mark.parametrize("D,chunks", [(64, 9), (64, None), (1, 5), (2, None)])
def test_depth_extremes(D, chunks):
    # D = 64: every stream keeps 63 active nodes between chunks; D = 1 and 2:
    # none or one
    rng = random.Random(D * 7 + (chunks or 0))
    streams = [[np.array([rng.randrange(3) for _ in range(rng.randrange(0, 150))]) for _ in range(4)]
               for _ in range(2)]
    say(f"cache: depth extremes D={D} chunks={chunks}")
    c = build(streams, D, chunks=chunks, rng=rng)
    assert c.status()["flags"] == 0
    for p in range(2):
        check_prompt(c, p, streams[p], D)


def test_segments_longer_than_a_workgroup():
    # one call appends 3000 tokens to a stream (more substring starts than
    # threads in the workgroup) and 1100 tokens to another that already has
    # active nodes
    rng = random.Random(99)
    D = 6
    s0 = np.array([rng.randrange(5) for _ in range(3000)])
    s1 = np.array([rng.randrange(5) for _ in range(1300)])
    c = Caches.create(1, 4, D, (len(s0) + len(s1)) * D + 64)
    ids = c.new_streams(2)
    say("cache: 3000- and 1100-token segments")
    c.insert([0], ids[1:], [s1[:200]])
    c.insert([0, 0], ids, [s0, s1[200:]])
    assert c.status()["flags"] == 0
    check_prompt(c, 0, [s0, s1], D)
