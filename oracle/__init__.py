"""CPU oracle for the SRT tree-speculative verification step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
path (``paper_2601_09083_amd``); both receive identical inputs from the
seeded generator module ``paper_2601_09083_amd.workload``, which holds none of
the method's arithmetic.

Each function is a plain, slow, obviously correct statement of what the
method computes, written from the paper (SRT, arXiv 2601.09083):

* ``trie``      -- the per-prompt tree-structured cache as a map from token
                   substring to occurrence count (Section 3, "Per-prompt
                   rollout cache"; Section 3, "Cache update strategy").
* ``draft``     -- longest-suffix match, edge score C(v) (the displayed
                   equation of Section 3), path-product node score and greedy
                   expansion under a node budget (Section 3, "Speculative
                   Rollout with Tree-Structured Cache").
* ``attention`` -- tree-masked softmax attention in fp64 for verifying every
                   drafted node in one decode pass (Section 3; Appendix C,
                   "Speculative Decoding").
* ``accept``    -- lossless acceptance up to the first mismatch, plus the
                   target's own token at the mismatch (Section 1; Section 3).
* ``commit``    -- the accepted path's key/value vectors moved into the
                   committed positions and the context advanced (Section 3,
                   classic speculative decoding; Appendix C).
* ``lmhead``    -- the acceptance walk with the policy's logits at each
                   visited node formed by its LM head on that node's hidden
                   state (Section 3's single verification pass), in fp64
                   rounded once to fp32, with the bound for other fp32
                   summation orders.

Pins (tests marked ``not gpu``) tie each function to closed forms, brute
force, library routines and invariants; see ``tests/test_oracle_*.py``.
"""
from . import accept, attention, commit, draft, lmhead, trie  # noqa: F401
