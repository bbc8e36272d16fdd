"""srt_accept_noalloc (the acceptance walk on the library's fixed per-device
scratch array, for callers that cannot allocate) against srt_accept (caller
scratch) through the C ABI: identical outputs, bit for bit, on consecutive
calls of decreasing size -- the largest batch the array holds, then smaller
ones with other tree sizes, vocabularies (one not a multiple of 4) and depth
caps, sampled and greedy -- so that the array's contents from an earlier,
larger call cannot leak into a later one; and the same walk captured in a
HIP graph, replayed three times with other no-alloc calls in between (each
overwriting the shared array), every replay equal to the eager result."""
import numpy as np
import pytest
import torch

from paper_2601_09083_amd import srt
from paper_2601_09083_amd import workload as W
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def problem(seed, B, N, V, Dmax, sampled):
    """Random trees (siblings carry distinct tokens) with logits that make
    the walks go deep: each node's first child's token is set 40 above the
    row maximum with probability 0.7."""
    rng = np.random.default_rng(seed)
    nn = rng.integers(1, N + 1, size=B).astype(np.int32)
    par = np.full((B, N), -1, np.int32)
    tok = np.full((B, N), -1, np.int32)
    for b in range(B):
        tok[b, 0] = int(rng.integers(0, V))
        for i in range(1, int(nn[b])):
            par[b, i] = int(rng.integers(max(0, i - 4), i))
            tok[b, i] = (i * 7919 + b) % V  # distinct for distinct i (V > N, 7919 prime)
    cfg = W.CONFIGS["tiny"].scaled(vocab=V, max_depth=Dmax, n_nodes=N, boost_add=40.0)
    logits = W.make_logits(cfg, tok, par, nn, device="cuda", seed=seed, boost="top")
    gumbel = W.make_gumbel(cfg, B, device="cuda", seed=seed + 1) if sampled else None
    dev = lambda a: torch.as_tensor(a, device="cuda")
    return logits, gumbel, dev(tok), dev(par), dev(nn)


def outputs(B, Dmax):
    return {"n_accepted": torch.full((B,), -7, dtype=torch.int32, device="cuda"),
            "out_tokens": torch.full((B, Dmax + 1), -7, dtype=torch.int32, device="cuda"),
            "out_nodes": torch.full((B, Dmax + 1), -7, dtype=torch.int32, device="cuda"),
            "n_emitted": torch.full((B,), -7, dtype=torch.int32, device="cuda")}


def test_noalloc_matches_scratch_entry_point():
    cases = [  # (seed, B, N, V, Dmax, sampled, inv_T)
        (1, srt.SRT_ACCEPT_NOALLOC_MAX_BATCH, 8, 1024, 4, True, 1.0),
        (2, 1500, 64, 6000, 10, True, 0.8),
        (3, 200, 16, 3001, 5, False, 1.0),
        (4, 37, 256, 2048, 63, True, 1.3),
    ]
    for seed, B, N, V, Dmax, sampled, inv_t in cases:
        say(f"no-alloc accept: B={B} N={N} V={V} Dmax={Dmax} sampled={sampled}")
        logits, gumbel, tt, tp, nn = problem(seed, B, N, V, Dmax, sampled)
        want = srt.srt_accept(logits, gumbel, inv_t, tt, tp, nn, Dmax)
        got = srt.srt_accept_noalloc(logits, gumbel, inv_t, tt, tp, nn, Dmax, out=outputs(B, Dmax))
        torch.cuda.synchronize()
        for k in want:
            assert torch.equal(got[k], want[k]), f"{k} differs (B={B}, seed {seed})"
        emitted = got["n_emitted"].cpu().numpy()
        assert emitted.min() >= 1 and emitted.max() >= min(3, Dmax + 1), "walks should go deep"
        say(f"  equal; emitted per sequence {emitted.mean():.2f}, deepest {emitted.max()}")


def test_noalloc_under_graph_capture():
    B, N, V, Dmax = 300, 32, 4096, 8
    logits, gumbel, tt, tp, nn = problem(11, B, N, V, Dmax, True)
    want = srt.srt_accept(logits, gumbel, 1.0, tt, tp, nn, Dmax)
    out = outputs(B, Dmax)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # first call (and the array's address lookup) outside the capture
        srt.srt_accept_noalloc(logits, gumbel, 1.0, tt, tp, nn, Dmax, out=out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say(f"no-alloc accept under graph capture: B={B} N={N} V={V} Dmax={Dmax}")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        srt.srt_accept_noalloc(logits, gumbel, 1.0, tt, tp, nn, Dmax, out=out)
    torch.cuda.synchronize()
    o_l, o_g, o_tt, o_tp, o_nn = problem(12, 64, 16, 2000, 5, False)
    for r in range(3):
        for v in out.values():
            v.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in want:
            assert torch.equal(out[k], want[k]), f"replay {r}: {k} differs"
        # eager work between replays: another walk through the same array
        srt.srt_accept_noalloc(o_l, o_g, 1.0, o_tt, o_tp, o_nn, 5, out=outputs(64, 5))
        torch.cuda.synchronize()
    say("  three replays equal the eager walk")
