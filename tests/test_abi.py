"""The C-ABI library loads, exports every entry point include/srt.h declares,
and rejects invalid arguments on the host before any HIP call (these tests
run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2601_09083_amd import srt as S

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "srt.h")



@pytest.fixture(scope="module", autouse=True)
def built_library():
    """The library these host-side checks load: built here (hipcc
    cross-compiles for gfx950 without a GPU) when it is not there yet; a
    failed build fails the tests instead of skipping them."""
    if not os.path.exists(S.LIB_PATH):
        from paper_2601_09083_amd import build as B
        B.build()
    assert os.path.exists(S.LIB_PATH)


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(srt_[a-z_]+)\s*\(", text)))


def test_header_declares_binding_exports():
    assert declared() == sorted(S.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(S.LIB_PATH)
    for name in declared():
        assert hasattr(L, name), name
    assert S.srt_version().startswith("libsrt")


def test_workspace_bytes_host_only():
    assert S.srt_trie_workspace_bytes(4, 8, 12, 1000) > 0
    assert S.srt_trie_workspace_bytes(0, 8, 12, 1000) == 0      # no prompts
    assert S.srt_trie_workspace_bytes(4, 8, 65, 1000) == 0      # D > 64
    assert S.srt_trie_workspace_bytes(4, 8, 12, 0) == 0         # no capacity
    assert S.srt_trie_workspace_bytes(4, 8, 12, 1 << 40) == 0   # beyond 2^31 slots
    a = S.srt_trie_workspace_bytes(4, 8, 12, 10_000)
    b = S.srt_trie_workspace_bytes(4, 8, 12, 1_000_000)
    assert b > a


def test_scratch_bytes():
    # one split: only the work list (header + 2 int32 per item), 256-byte rounded
    one = S.srt_tree_attn_scratch_bytes(4, 8, 4, 1, 64, 16, 40)
    assert one >= (64 + 2 * 4) * 4 and one % 256 == 0 and one < 4096
    n = S.srt_tree_attn_scratch_bytes(256, 64, 28, 4, 128, 16, 2052)
    assert n > one and n % 4 == 0
    assert S.srt_tree_attn_scratch_bytes(4, 8, 5, 2, 64, 16, 40) == 0  # Hq % Hkv != 0


def _expected_attn_scratch(B, N, Hq, Hkv, d, page, max_pages):
    """The scratch size srt_tree_attn documents: its work list (a 64-int
    header, two int32 per (sequence, KV head, split, row block) item and per
    8-row combine unit), plus fp32 partial rows and (max, sum) pairs when a
    context can span several splits.  A split is the largest power of two in
    [1024, 8192] keys that keeps B * Hkv * row blocks * splits >= 512."""
    G = Hq // Hkv
    rb = -(-(N * G) // 256)
    cap = page * max_pages
    chunk = 8192
    while chunk > 1024 and B * Hkv * rb * (-(-cap // chunk)) < 512:
        chunk //= 2
    S = -(-cap // chunk)
    items = B * Hkv * S * rb
    units = B * Hkv * (-(-(N * G) // 8))
    plan = -(-((64 + 2 * items + 2 * units) * 4) // 256) * 256
    return plan if S <= 1 else plan + B * Hkv * S * rb * 256 * (d + 2) * 4, chunk


@pytest.mark.parametrize("shape,chunk", [
    ((64, 32, 12, 2, 128, 16, 288), 1024),    # 1.5B-shaped batch: small, short contexts
    ((16, 8, 8, 8, 128, 16, 1001), 4096),
    ((8, 8, 8, 8, 128, 16, 1001), 2048),
    ((256, 64, 28, 4, 128, 16, 2052), 8192),  # 7B-shaped batch
    ((8, 256, 28, 4, 128, 16, 2100), 8192),   # long-tail: seven row blocks keep large splits
])
def test_scratch_bytes_follow_the_split_rule(shape, chunk):
    want, got_chunk = _expected_attn_scratch(*shape)
    assert got_chunk == chunk
    assert S.srt_tree_attn_scratch_bytes(*shape) == want


def test_host_validation_before_any_hip_call():
    L = S.lib()
    cfg = S.TrieConfig(4, 8, 12, 0, 100)
    assert L.srt_trie_init(None, 1 << 20, ctypes.byref(cfg), None) == S.SRT_ERR_INVALID
    bad = S.TrieConfig(4, 8, 12, 1, 100)  # reserved != 0
    assert L.srt_trie_init(ctypes.c_void_p(256), 1 << 20, ctypes.byref(bad), None) == S.SRT_ERR_INVALID
    assert L.srt_trie_init(ctypes.c_void_p(255), 1 << 20, ctypes.byref(cfg), None) == S.SRT_ERR_INVALID  # alignment
    assert L.srt_trie_init(ctypes.c_void_p(256), 64, ctypes.byref(cfg), None) == S.SRT_ERR_CAPACITY
    assert L.srt_trie_insert(None, 1, None, None, None, None, 4, None) == S.SRT_ERR_INVALID
    assert L.srt_trie_insert(ctypes.c_void_p(256), -1, None, None, None, None, 4, None) == S.SRT_ERR_INVALID
    assert L.srt_trie_insert(ctypes.c_void_p(256), 0, None, None, None, None, 4, None) == S.SRT_OK  # no-op
    assert L.srt_trie_reset_streams(ctypes.c_void_p(256), 0, None, None) == S.SRT_OK
    assert L.srt_trie_status(None, None, None) == S.SRT_ERR_INVALID
    p = S.DraftParams(8, 257, 4, 0, 0.0)   # N > 256
    assert L.srt_draft(ctypes.c_void_p(256), 1, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_ERR_INVALID
    p = S.DraftParams(0, 8, 4, 0, 0.0)     # Qmax < 1
    assert L.srt_draft(ctypes.c_void_p(256), 1, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_ERR_INVALID
    p = S.DraftParams(8, 8, 64, 0, 0.0)    # Dmax > 63
    assert L.srt_draft(ctypes.c_void_p(256), 1, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_ERR_INVALID
    p = S.DraftParams(8, 8, 4, 2, 0.0)    # chain must be 0 or 1
    assert L.srt_draft(ctypes.c_void_p(256), 1, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_ERR_INVALID
    p = S.DraftParams(8, 8, 4, 0, 0.0, float("nan"))  # min_score NaN
    assert L.srt_draft(ctypes.c_void_p(256), 1, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_ERR_INVALID
    p = S.DraftParams(8, 8, 4, 0, 0.0)
    assert L.srt_draft(ctypes.c_void_p(256), 0, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_OK  # B = 0
    assert L.srt_draft(ctypes.c_void_p(256), 2, *[None] * 3, ctypes.byref(p), *[None] * 6) == S.SRT_ERR_INVALID
    args = [4, 8, 4, 1, 96, 16, 40, 100] + [ctypes.c_void_p(256)] * 7 + [0.125, ctypes.c_void_p(256), None, 0, None]
    assert L.srt_tree_attn(*args) == S.SRT_ERR_UNSUPPORTED           # d = 96
    for bad_page in (8, 24, 48):
        a2 = list(args); a2[4] = 64; a2[5] = bad_page
        assert L.srt_tree_attn(*a2) == S.SRT_ERR_UNSUPPORTED         # page not a power of two >= 16
    args[4] = 64; args[2] = 5; args[3] = 2
    assert L.srt_tree_attn(*args) == S.SRT_ERR_INVALID               # Hq % Hkv
    args[2] = 4; args[3] = 1; args[1] = 300
    assert L.srt_tree_attn(*args) == S.SRT_ERR_INVALID               # N > 256
    args[1] = 8; args[6] = 2052
    assert L.srt_tree_attn(*args) == S.SRT_ERR_CAPACITY              # scratch needed, none given
    acc = [4, 0, 16, 4, None, None, 1.0] + [None] * 7 + [None, 0, None]
    assert L.srt_accept(*acc) == S.SRT_ERR_INVALID                   # N = 0
    acc[1] = 8; acc[3] = 64
    assert L.srt_accept(*acc) == S.SRT_ERR_INVALID                   # Dmax > 63
    acc[3] = 4
    assert L.srt_accept(*acc) == S.SRT_ERR_INVALID                   # null pointers
    acc[4:14] = [ctypes.c_void_p(256)] * 2 + [1.0] + [ctypes.c_void_p(256)] * 7
    assert L.srt_accept(*acc) == S.SRT_ERR_CAPACITY                  # scratch needed, none given
    acc[14], acc[15] = ctypes.c_void_p(256 + 16), S.srt_accept_scratch_bytes(4)
    assert L.srt_accept(*acc) == S.SRT_ERR_INVALID                   # scratch not 256-byte aligned
    acc[0] = 0
    assert L.srt_accept(*acc) == S.SRT_OK                            # B = 0
    assert S.srt_accept_scratch_bytes(4) >= 4 * 256 and S.srt_accept_scratch_bytes(-1) == 0
    P = ctypes.c_void_p(256)
    lmh = [4, 8, 128, 1000, 4, P, P, None, 1.0] + [P] * 6 + [None, P, S.srt_accept_lmhead_scratch_bytes(4, 8, 1000), None]
    bad = list(lmh); bad[1] = 0
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # N = 0
    bad = list(lmh); bad[4] = 64
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # Dmax > 63
    bad = list(lmh); bad[3] = 0
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # V = 0
    bad = list(lmh); bad[2] = 96
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_UNSUPPORTED        # d_model not a multiple of 64
    bad = list(lmh); bad[7] = P; bad[8] = float("inf")
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # sampled with a non-finite 1/T
    bad = list(lmh); bad[6] = ctypes.c_void_p(256 + 8)
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # w_head not 16-byte aligned
    bad = list(lmh); bad[11] = None
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # null n_nodes
    bad = list(lmh); bad[16] = ctypes.c_void_p(256 + 64)
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_INVALID            # scratch not 256-byte aligned
    bad = list(lmh); bad[17] -= 1
    assert L.srt_accept_lmhead(*bad) == S.SRT_ERR_CAPACITY           # scratch too small
    bad = list(lmh); bad[0] = 0
    assert L.srt_accept_lmhead(*bad) == S.SRT_OK                     # B = 0
    # candidates: 8 bytes per row per 128 vocabulary entries, a row table, lists
    assert S.srt_accept_lmhead_scratch_bytes(256, 64, 152064) >= 256 * 1188 * 8 + 256 * 64 * 4
    assert S.srt_accept_lmhead_scratch_bytes(4, 8, 1000) >= 128 * 8 * 8  # at least 128 rows
    assert S.srt_accept_lmhead_scratch_bytes(4, 8, 0) == 0 and S.srt_accept_lmhead_scratch_bytes(-1, 8, 10) == 0
    assert S.srt_accept_lmhead_scratch_bytes(4, 0, 10) == 0
    com = [4, 8, 1, 64, 16, 40, 100] + [None] * 4 + [4] + [None] * 3 + [8, None, None, None]
    assert L.srt_commit(*com) == S.SRT_ERR_INVALID                   # null pointers
    com[3] = 12
    assert L.srt_commit(*com) == S.SRT_ERR_UNSUPPORTED               # d not a multiple of 8
    com[3] = 64; com[16] = ctypes.c_void_p(256)
    assert L.srt_commit(*com) == S.SRT_ERR_INVALID                   # ctx_tail without draft_len
    com[0] = 0; com[16] = None
    assert L.srt_commit(*com) == S.SRT_OK                            # B = 0


def test_accept_noalloc_rejects_batches_beyond_its_array():
    """Host checks of srt_accept_noalloc, before any device memory is
    touched: a batch above SRT_ACCEPT_NOALLOC_MAX_BATCH is SRT_ERR_CAPACITY,
    B = 0 is a no-op, invalid sizes are SRT_ERR_INVALID.  (The pointers are
    never dereferenced on these paths.)"""
    L = S.lib()
    fake = ctypes.c_void_p(0x1000)
    args = lambda B, N=8, V=100, Dmax=4: (B, N, V, Dmax, fake, None, 1.0, fake, fake, fake, fake, fake, fake, None,
                                          None)
    assert S.SRT_ACCEPT_NOALLOC_MAX_BATCH == 4096
    hdr = open(HEADER).read()
    assert re.search(r"#define SRT_ACCEPT_NOALLOC_MAX_BATCH 4096\b", hdr)
    assert L.srt_accept_noalloc(*args(4097)) == S.SRT_ERR_CAPACITY
    assert L.srt_accept_noalloc(*args(1 << 30)) == S.SRT_ERR_CAPACITY
    assert L.srt_accept_noalloc(*args(0)) == S.SRT_OK
    assert L.srt_accept_noalloc(*args(4, N=0)) == S.SRT_ERR_INVALID
    assert L.srt_accept_noalloc(*args(4, Dmax=64)) == S.SRT_ERR_INVALID
