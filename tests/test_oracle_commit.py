"""Pins for the commit oracle (oracle/commit.py).

The defining property: a speculative loop (draft tree -> one verification
pass that writes every node's vectors at its tree slot -> acceptance ->
commit) leaves exactly the KV cache that sequential decoding of the same
tokens would leave, position by position, and the draft tail / committed
count of the grown sequence.  A toy "model" makes the vectors of a position
a hash of the whole prefix ending there, so any misplaced, stale or shifted
vector shows.  Plus hand-worked cases and planted mistakes."""
import random

import numpy as np
import pytest

from oracle import accept as AC
from oracle import commit as CM


def prefix_vec(prefix, width=4):
    """Toy key/value vector of the position holding the last token of
    ``prefix``: a deterministic function of the whole prefix."""
    h = 1469598103934665603
    for x in prefix:
        h = ((h ^ (int(x) + 1)) * 1099511628211) % (1 << 64)
    return np.random.default_rng(h).standard_normal(width)


def toy_logits(prefix, V):
    h = 7
    for x in prefix[-3:]:
        h = (h * 1000003 + int(x) + 11) % (1 << 32)
    return np.random.default_rng(h).standard_normal(V).astype(np.float32)


def random_tree(rng, y, V, N, Dmax, p_follow=0.75):
    """A tree rooted at the last token of y whose nodes often carry the toy
    policy's own greedy choice."""
    tokens, parents, paths, depth = [int(y[-1])], [-1], [()], [0]
    frontier = [0]
    while frontier and len(tokens) < N:
        u = frontier.pop(0)
        if depth[u] >= Dmax:
            continue
        used = []
        if rng.random() < p_follow:
            used.append(int(np.argmax(toy_logits(list(y) + list(paths[u]), V))))
        for _ in range(rng.randrange(0, 3)):
            x = rng.randrange(V)
            if x not in used:
                used.append(x)
        rng.shuffle(used)
        for x in used:
            if len(tokens) >= N:
                break
            tokens.append(x); parents.append(u); paths.append(paths[u] + (x,)); depth.append(depth[u] + 1)
            frontier.append(len(tokens) - 1)
    return tokens, parents, paths


def run_loop(seed, steps=12, V=6, N=10, Dmax=4, Qmax=5, commit_kv=CM.commit_kv, commit_tail=CM.commit_tail,
             t0=7):
    rng = random.Random(seed)
    y = [rng.randrange(V) for _ in range(t0)]
    L = len(y) - 1
    cap = L + steps * (N + Dmax + 2) + N
    kv = np.zeros((cap, 4))
    for p in range(L):
        kv[p] = prefix_vec(y[: p + 1])
    tail = np.full(Qmax, -1, dtype=np.int32)
    k0 = min(len(y), Qmax)
    tail[Qmax - k0:] = y[len(y) - k0:]
    t = len(y)
    for _ in range(steps):
        tokens, parents, paths = random_tree(rng, y, V, N, Dmax)
        n = len(tokens)
        for i in range(n):  # the verification pass writes each node's vectors at its slot
            kv[L + i] = prefix_vec(list(y) + list(paths[i]))
        k, emitted, nodes = AC.accept(lambda u: toy_logits(list(y) + list(paths[u]), V), None, 1.0, tokens,
                                      parents, n, Dmax)
        kv, L = commit_kv(kv, L, k, nodes)
        tail, t = commit_tail(tail, t, emitted)
        y = y + list(emitted)
    return y, kv, L, tail, t


@pytest.mark.parametrize("seed", range(40))
def test_loop_equals_sequential_decoding(seed):
    Qmax = 5
    y, kv, L, tail, t = run_loop(seed, Qmax=Qmax)
    assert L == len(y) - 1 and t == len(y)
    for p in range(L):
        assert np.array_equal(kv[p], prefix_vec(y[: p + 1])), f"position {p}"
    assert tail.tolist() == y[-Qmax:]


def test_loop_accepts_something():
    # the pins above are only meaningful if paths of several nodes get accepted
    total = 0
    for seed in range(40):
        y, *_ = run_loop(seed)
        total += len(y) - 7
    assert total > 40 * 12 * 1.5


def test_hand_case():
    kv = np.arange(20).reshape(20, 1) * 10
    out, L2 = CM.commit_kv(kv, 5, 2, [2, 5])
    want = kv.copy()
    want[6], want[7] = kv[7], kv[10]
    assert np.array_equal(out, want) and L2 == 8
    out, L2 = CM.commit_kv(kv, 5, 0, [])
    assert np.array_equal(out, kv) and L2 == 6


def test_path_reads_a_slot_an_earlier_copy_writes():
    # accepted nodes 2, 3: position L+2 is both the source of j=1 and the
    # destination of j=2; the committed vectors are those of nodes 2 and 3
    kv = np.arange(12).reshape(12, 1)
    out, L2 = CM.commit_kv(kv, 4, 2, [2, 3])
    assert out[5, 0] == 6 and out[6, 0] == 7 and L2 == 7


def test_tail():
    row, t = CM.commit_tail(np.array([-1, -1, 3, 4], np.int32), 2, [7, 8, 9])
    assert row.tolist() == [4, 7, 8, 9] and t == 5
    row, t = CM.commit_tail(np.array([-1, -1, -1, 4], np.int32), 1, [7])
    assert row.tolist() == [-1, -1, 4, 7] and t == 2
    row, t = CM.commit_tail(np.array([1, 2, 3], np.int32), 10, [4, 5, 6, 7, 8])
    assert row.tolist() == [6, 7, 8] and t == 15
    row, t = CM.commit_tail(np.array([-1, -1], np.int32), 0, [5])
    assert row.tolist() == [-1, 5] and t == 1


# ---- planted mistakes: each must fail the loop pin --------------------------

def _identity_copy(kv, L, k, nodes):
    return np.array(kv, copy=True), L + k + 1


def _length_without_root(kv, L, k, nodes):
    out, _ = CM.commit_kv(kv, L, k, nodes)
    return out, L + k


def _in_place_descending(kv, L, k, nodes):
    out = np.array(kv, copy=True)
    for j in range(k, 0, -1):
        out[L + j] = out[L + int(nodes[j - 1])]
    return out, L + k + 1


def _tail_drops_bonus(tail, t, emitted):
    return CM.commit_tail(tail, t, list(emitted)[:-1])


@pytest.mark.parametrize("mistake", ["identity", "no_root", "descending", "tail"])
def test_planted_mistakes_fail(mistake):
    kw = {"identity": dict(commit_kv=_identity_copy), "no_root": dict(commit_kv=_length_without_root),
          "descending": dict(commit_kv=_in_place_descending), "tail": dict(commit_tail=_tail_drops_bonus)}[mistake]
    failed = 0
    for seed in range(40):
        y, kv, L, tail, t = run_loop(seed, **kw)
        ok = L == len(y) - 1 and t == len(y) and tail.tolist() == y[-5:] and all(
            np.array_equal(kv[p], prefix_vec(y[: p + 1])) for p in range(min(L, len(y) - 1)))
        failed += not ok
    assert failed > 0
