"""Oracle for the per-prompt tree-structured cache (test infrastructure only).

Section 3 ("Per-prompt rollout cache using tree-structured cache"): for each
prompt the cache indexes every token substring that occurred in earlier
rollouts; a node is a substring, its outgoing edges are the next tokens, and
count(u) records how often u occurred.  Section 3 ("Cache update strategy"):
tokens of running rollouts and of run-ahead continuations are inserted as
they are produced.

Reading used here (the paper fixes no depth limit or exact count semantics):
the cache of prompt p is the map s -> count(s) over all strings s with
1 <= |s| <= D, where count(s) is the number of (stream, start) positions at
which s occurs in the streams inserted for p.  Streams are kept apart: no
occurrence spans two streams.  Appending tokens to a stream therefore means
the map of the extended streams.  The Fig. 2 caption's "non-leaf = sum of
children" differs from occurrence counts only by occurrences that end a
stream; the edge score C(v) divides by the sum over siblings, so drafts are
identical under both readings.
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Sequence, Tuple

import numpy as np


def substring_counts(streams: Iterable[Sequence[int]], D: int) -> Dict[Tuple[int, ...], int]:
    """count(s) for every substring s, 1 <= |s| <= D, of the given streams.

    Direct statement of the definition: every start position of every stream
    contributes one occurrence to each of its first D prefixes."""
    counts: Dict[Tuple[int, ...], int] = {}
    for st in streams:
        st = [int(x) for x in st]
        n = len(st)
        for i in range(n):
            for ell in range(1, min(D, n - i) + 1):
                key = tuple(st[i:i + ell])
                counts[key] = counts.get(key, 0) + 1
    return counts


class DictTrie:
    """Read access to a substring-count map: counts and child enumeration."""

    def __init__(self, counts: Dict[Tuple[int, ...], int], D: int):
        self.D = D
        self.counts = counts
        self._children: Dict[Tuple[int, ...], List[int]] = {}
        for s in counts:
            self._children.setdefault(s[:-1], []).append(s[-1])

    def count(self, s: Sequence[int]) -> int:
        return self.counts.get(tuple(int(x) for x in s), 0)

    def children(self, s: Sequence[int]) -> Dict[int, int]:
        """{x: count(s + x)} over the children of node s."""
        s = tuple(int(x) for x in s)
        return {x: self.counts[s + (x,)] for x in self._children.get(s, [])}


class StreamTrie:
    """The same map, answered by scanning the streams for each query.

    Memory-light stand-in for ``DictTrie`` on large inputs: count(s) is found
    by locating every occurrence of s in the concatenated streams."""

    def __init__(self, streams: Iterable[Sequence[int]], D: int):
        self.D = D
        parts = []
        for st in streams:
            parts.append(np.asarray(st, dtype=np.int64))
            parts.append(np.array([-1], dtype=np.int64))  # stream separator
        self.a = np.concatenate(parts) if parts else np.array([-1], dtype=np.int64)

    def _occurrences(self, s: Sequence[int]) -> np.ndarray:
        """Start positions of every occurrence of s (separators never match)."""
        a = self.a
        q = len(s)
        if q == 0:
            return np.nonzero(a >= 0)[0]  # every token starts a non-empty occurrence
        pos = np.nonzero(a == int(s[0]))[0]
        for j in range(1, q):
            pos = pos[pos + j < a.shape[0]]
            pos = pos[a[pos + j] == int(s[j])]
        return pos

    def count(self, s: Sequence[int]) -> int:
        if not 1 <= len(s) <= self.D:
            return 0
        return int(self._occurrences(s).shape[0])

    def children(self, s: Sequence[int]) -> Dict[int, int]:
        if len(s) + 1 > self.D:
            return {}
        pos = self._occurrences(s) + len(s)
        nxt = self.a[pos[pos < self.a.shape[0]]]
        nxt = nxt[nxt >= 0]
        xs, cs = np.unique(nxt, return_counts=True)
        return {int(x): int(c) for x, c in zip(xs, cs)}


def insert_counts(counts: Dict[Tuple[int, ...], int], stream_before: Sequence[int], appended: Sequence[int],
                  D: int) -> None:
    """Online insertion (Section 3, "Cache update strategy"): appending token
    x at index j of a stream adds one occurrence to every suffix of the
    stream ending at j, of length 1..min(D, j+1).  Updates ``counts`` in
    place; ``stream_before`` is the stream's content so far."""
    st = [int(x) for x in stream_before]
    for x in appended:
        st.append(int(x))
        j = len(st) - 1
        for ell in range(1, min(D, j + 1) + 1):
            key = tuple(st[j - ell + 1:j + 1])
            counts[key] = counts.get(key, 0) + 1
