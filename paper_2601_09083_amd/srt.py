"""Python binding of libsrt (include/srt.h): argument marshalling only.

Every function here has the name of the C entry point it calls, takes torch
tensors that already live on the GPU, passes their device pointers and the
current HIP stream, and raises ``SrtError`` on a non-zero status.  All work
is done by the HIP kernels in libsrt.so; there is no fallback: if the
library is missing, every call raises.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsrt.so")

SRT_OK, SRT_ERR_INVALID, SRT_ERR_CAPACITY, SRT_ERR_HIP, SRT_ERR_UNSUPPORTED = 0, -1, -2, -3, -4
SRT_FLAG_CAPACITY, SRT_FLAG_STREAM, SRT_FLAG_PROMPT = 1, 2, 4
_NAMES = {SRT_ERR_INVALID: "SRT_ERR_INVALID", SRT_ERR_CAPACITY: "SRT_ERR_CAPACITY",
          SRT_ERR_HIP: "SRT_ERR_HIP", SRT_ERR_UNSUPPORTED: "SRT_ERR_UNSUPPORTED"}

# Every symbol include/srt.h declares.
EXPORTS = ("srt_trie_workspace_bytes", "srt_trie_init", "srt_trie_insert", "srt_trie_reset_streams",
           "srt_trie_status", "srt_trie_export", "srt_draft", "srt_tree_attn_scratch_bytes",
           "srt_tree_attn", "srt_accept_scratch_bytes", "srt_accept", "srt_accept_lmhead_scratch_bytes",
           "srt_accept_lmhead", "srt_commit", "srt_version", "srt_accept_noalloc")
SRT_ACCEPT_NOALLOC_MAX_BATCH = 4096  # include/srt.h


class SrtError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {_NAMES.get(status, status)}")
        self.status = status


class TrieConfig(ctypes.Structure):
    _fields_ = [("n_prompts", ctypes.c_int32), ("max_streams", ctypes.c_int32),
                ("max_depth", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("node_capacity", ctypes.c_int64)]


class DraftParams(ctypes.Structure):
    _fields_ = [("max_match", ctypes.c_int32), ("max_nodes", ctypes.c_int32),
                ("max_depth", ctypes.c_int32), ("chain", ctypes.c_int32),
                ("budget_alpha", ctypes.c_double), ("min_score", ctypes.c_double)]


_lib = None
_P, _I32, _I64, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """The loaded libsrt.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "srt_trie_workspace_bytes": (_SZ, [ctypes.POINTER(TrieConfig)]),
            "srt_trie_init": (ctypes.c_int, [_P, _SZ, ctypes.POINTER(TrieConfig), _P]),
            "srt_trie_insert": (ctypes.c_int, [_P, _I32, _P, _P, _P, _P, _I32, _P]),
            "srt_trie_reset_streams": (ctypes.c_int, [_P, _I32, _P, _P]),
            "srt_trie_status": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int64), _P]),
            "srt_trie_export": (ctypes.c_int, [_P, _I32, _I64, _P, _P, _P, ctypes.POINTER(ctypes.c_int64), _P]),
            "srt_draft": (ctypes.c_int, [_P, _I32, _P, _P, _P, ctypes.POINTER(DraftParams), _P, _P, _P, _P, _P, _P]),
            "srt_tree_attn_scratch_bytes": (_SZ, [_I32] * 7),
            "srt_tree_attn": (ctypes.c_int, [_I32] * 7 + [_I64] + [_P] * 7 + [ctypes.c_float, _P, _P, _SZ, _P]),
            "srt_accept_scratch_bytes": (_SZ, [_I32]),
            "srt_accept": (ctypes.c_int, [_I32] * 4 + [_P, _P, ctypes.c_float] + [_P] * 7 + [_P, _SZ, _P]),
            "srt_accept_noalloc": (ctypes.c_int, [_I32] * 4 + [_P, _P, ctypes.c_float] + [_P] * 7 + [_P]),
            "srt_accept_lmhead_scratch_bytes": (_SZ, [_I32, _I32, _I32]),
            "srt_accept_lmhead": (ctypes.c_int, [_I32] * 5 + [_P, _P, _P, ctypes.c_float] + [_P] * 7 + [_P, _SZ, _P]),
            "srt_commit": (ctypes.c_int, [_I32] * 6 + [_I64] + [_P] * 4 + [_I32] + [_P] * 3 + [_I32, _P, _P, _P]),
            "srt_version": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _check(fn: str, st: int):
    if st != SRT_OK:
        raise SrtError(fn, st)


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _on(stream):
    """Context in which buffers the binding allocates for a call belong to
    the stream the call is enqueued on: torch's caching allocator then never
    hands them out again while that stream may still use them."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


# --------------------------------------------------------------------------- cache

def srt_trie_workspace_bytes(n_prompts: int, max_streams: int, max_depth: int, node_capacity: int) -> int:
    cfg = TrieConfig(n_prompts, max_streams, max_depth, 0, node_capacity)
    return int(lib().srt_trie_workspace_bytes(ctypes.byref(cfg)))


def srt_trie_init(ws: torch.Tensor, n_prompts: int, max_streams: int, max_depth: int, node_capacity: int,
                  stream=None):
    cfg = TrieConfig(n_prompts, max_streams, max_depth, 0, node_capacity)
    _check("srt_trie_init", lib().srt_trie_init(_ptr(ws, torch.uint8, "ws"), ws.numel(), ctypes.byref(cfg),
                                               _stream(stream)))


def srt_trie_insert(ws: torch.Tensor, prompt_ids, stream_ids, tokens, lengths, stream=None):
    n = int(prompt_ids.numel())
    stride = int(tokens.shape[1]) if tokens.dim() == 2 else max(1, int(tokens.numel()))
    _check("srt_trie_insert", lib().srt_trie_insert(
        _ptr(ws, torch.uint8, "ws"), n, _ptr(prompt_ids, torch.int32, "prompt_ids"),
        _ptr(stream_ids, torch.int32, "stream_ids"), _ptr(tokens, torch.int32, "tokens"),
        _ptr(lengths, torch.int32, "lengths"), stride, _stream(stream)))


def srt_trie_reset_streams(ws: torch.Tensor, stream_ids, stream=None):
    _check("srt_trie_reset_streams", lib().srt_trie_reset_streams(
        _ptr(ws, torch.uint8, "ws"), int(stream_ids.numel()), _ptr(stream_ids, torch.int32, "stream_ids"),
        _stream(stream)))


def srt_trie_status(ws: torch.Tensor, stream=None) -> dict:
    info = (ctypes.c_int64 * 4)()
    st = lib().srt_trie_status(_ptr(ws, torch.uint8, "ws"), info, _stream(stream))
    if st not in (SRT_OK, SRT_ERR_CAPACITY):
        raise SrtError("srt_trie_status", st)
    return {"flags": int(info[0]), "nodes": int(info[1]), "node_capacity": int(info[2]),
            "slots": int(info[3]), "status": st}


def srt_trie_export(ws: torch.Tensor, prompt_id: int, max_nodes: int, stream=None):
    """(parent, token, count) int64 numpy arrays of the prompt's cache, BFS order."""
    dev = ws.device
    parent = torch.empty(max(1, max_nodes), dtype=torch.int32, device=dev)
    token = torch.empty_like(parent)
    count = torch.empty_like(parent)
    n = ctypes.c_int64(0)
    st = lib().srt_trie_export(_ptr(ws, torch.uint8, "ws"), prompt_id, max_nodes, _ptr(parent), _ptr(token),
                               _ptr(count), ctypes.byref(n), _stream(stream))
    _check("srt_trie_export", st)
    k = n.value
    return (parent[:k].cpu().numpy().astype("int64"), token[:k].cpu().numpy().astype("int64"),
            count[:k].cpu().numpy().view("uint32").astype("int64"))


# --------------------------------------------------------------------------- draft

def srt_draft(ws: torch.Tensor, prompt_ids, ctx_tail, ctx_len, max_match: int, max_nodes: int, max_depth: int,
              budget_alpha: float = 0.0, out=None, stream=None, min_score: float = 0.0, chain: bool = False) -> dict:
    B = int(prompt_ids.numel())
    if ctx_tail.shape != (B, max_match):
        raise ValueError("ctx_tail must be [B, max_match]")
    dev = prompt_ids.device
    if out is None:
        with _on(stream):
            out = {k: torch.empty((B, max_nodes), dtype=torch.int32, device=dev)
                   for k in ("tree_tokens", "tree_parent", "tree_depth")}
            out["n_nodes"] = torch.empty(B, dtype=torch.int32, device=dev)
            out["match_len"] = torch.empty(B, dtype=torch.int32, device=dev)
    prm = DraftParams(max_match, max_nodes, max_depth, int(bool(chain)), float(budget_alpha), float(min_score))
    _check("srt_draft", lib().srt_draft(
        _ptr(ws, torch.uint8, "ws"), B, _ptr(prompt_ids, torch.int32, "prompt_ids"),
        _ptr(ctx_tail, torch.int32, "ctx_tail"), _ptr(ctx_len, torch.int32, "ctx_len"), ctypes.byref(prm),
        _ptr(out["tree_tokens"], torch.int32), _ptr(out["tree_parent"], torch.int32),
        _ptr(out["tree_depth"], torch.int32), _ptr(out["n_nodes"], torch.int32),
        _ptr(out["match_len"], torch.int32), _stream(stream)))
    return out


# --------------------------------------------------------------------------- attention

def srt_tree_attn_scratch_bytes(B: int, N: int, Hq: int, Hkv: int, d: int, page: int, max_pages: int) -> int:
    return int(lib().srt_tree_attn_scratch_bytes(B, N, Hq, Hkv, d, page, max_pages))


def srt_tree_attn(q, k_cache, v_cache, block_table, ctx_len, tree_parent, n_nodes, scale: float,
                  out=None, scratch=None, stream=None):
    """q [B,N,Hq,d] bf16; caches [P,Hkv,page,d] bf16; block_table [B,max_pages] int32."""
    B, N, Hq, d = q.shape
    P, Hkv, page, d2 = k_cache.shape
    if d2 != d or v_cache.shape != k_cache.shape:
        raise ValueError("cache shape mismatch")
    max_pages = int(block_table.shape[1])
    need = srt_tree_attn_scratch_bytes(B, N, Hq, Hkv, d, page, max_pages)
    with _on(stream):
        if out is None:
            out = torch.empty_like(q)
        if need and (scratch is None or scratch.numel() < need):
            scratch = torch.empty(need, dtype=torch.uint8, device=q.device)
    _check("srt_tree_attn", lib().srt_tree_attn(
        B, N, Hq, Hkv, d, page, max_pages, P, _ptr(q, torch.bfloat16, "q"), _ptr(k_cache, torch.bfloat16, "k_cache"),
        _ptr(v_cache, torch.bfloat16, "v_cache"), _ptr(block_table, torch.int32, "block_table"),
        _ptr(ctx_len, torch.int32, "ctx_len"), _ptr(tree_parent, torch.int32, "tree_parent"),
        _ptr(n_nodes, torch.int32, "n_nodes"), float(scale), _ptr(out, torch.bfloat16, "out"),
        _ptr(scratch) if need else None, need, _stream(stream)))
    return out


# --------------------------------------------------------------------------- acceptance

def _walk_outputs(B: int, max_depth: int, dev) -> dict:
    return {"n_accepted": torch.empty(B, dtype=torch.int32, device=dev),
            "out_tokens": torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev),
            "out_nodes": torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev),
            "n_emitted": torch.empty(B, dtype=torch.int32, device=dev)}


def srt_accept_scratch_bytes(B: int) -> int:
    return int(lib().srt_accept_scratch_bytes(B))


def srt_accept(logits, gumbel, inv_temperature: float, tree_tokens, tree_parent, n_nodes, max_depth: int,
               out=None, scratch=None, stream=None) -> dict:
    """logits [B,N,V] fp32; gumbel [B,max_depth+1,V] fp32 or None (greedy)."""
    B, N, V = logits.shape
    if gumbel is not None and tuple(gumbel.shape) != (B, max_depth + 1, V):
        raise ValueError("gumbel must be [B, max_depth+1, V]")
    dev = logits.device
    need = srt_accept_scratch_bytes(B)
    with _on(stream):
        if out is None:
            out = _walk_outputs(B, max_depth, dev)
        if scratch is None or scratch.numel() < need:
            scratch = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("srt_accept", lib().srt_accept(
        B, N, V, max_depth, _ptr(logits, torch.float32, "logits"), _ptr(gumbel, torch.float32, "gumbel"),
        float(inv_temperature), _ptr(tree_tokens, torch.int32, "tree_tokens"),
        _ptr(tree_parent, torch.int32, "tree_parent"), _ptr(n_nodes, torch.int32, "n_nodes"),
        _ptr(out["n_accepted"], torch.int32), _ptr(out["out_tokens"], torch.int32),
        _ptr(out["out_nodes"], torch.int32), _ptr(out.get("n_emitted"), torch.int32), _ptr(scratch, name="scratch"),
        scratch.numel(), _stream(stream)))
    return out


def srt_accept_noalloc(logits, gumbel, inv_temperature: float, tree_tokens, tree_parent, n_nodes, max_depth: int,
                       out, stream=None) -> dict:
    """srt_accept with the library's fixed per-device scratch array: the
    caller passes preallocated outputs (``out`` as srt_accept returns it) and
    nothing is allocated, here or in the library.  B <= 4096."""
    B, N, V = logits.shape
    if gumbel is not None and tuple(gumbel.shape) != (B, max_depth + 1, V):
        raise ValueError("gumbel must be [B, max_depth+1, V]")
    _check("srt_accept_noalloc", lib().srt_accept_noalloc(
        B, N, V, max_depth, _ptr(logits, torch.float32, "logits"), _ptr(gumbel, torch.float32, "gumbel"),
        float(inv_temperature), _ptr(tree_tokens, torch.int32, "tree_tokens"),
        _ptr(tree_parent, torch.int32, "tree_parent"), _ptr(n_nodes, torch.int32, "n_nodes"),
        _ptr(out["n_accepted"], torch.int32), _ptr(out["out_tokens"], torch.int32),
        _ptr(out["out_nodes"], torch.int32), _ptr(out.get("n_emitted"), torch.int32), _stream(stream)))
    return out


def srt_accept_lmhead_scratch_bytes(B: int, N: int, V: int) -> int:
    return int(lib().srt_accept_lmhead_scratch_bytes(B, N, V))


def srt_accept_lmhead(hidden, w_head, gumbel, inv_temperature: float, tree_tokens, tree_parent, n_nodes,
                      max_depth: int, out=None, scratch=None, stream=None) -> dict:
    """hidden [B,N,d_model] bf16; w_head [V,d_model] bf16; gumbel [B,max_depth+1,V]
    fp32 or None (greedy).  Outputs as srt_accept."""
    B, N, dm = hidden.shape
    V, dm2 = w_head.shape
    if dm2 != dm:
        raise ValueError("w_head must be [V, d_model]")
    if gumbel is not None and tuple(gumbel.shape) != (B, max_depth + 1, V):
        raise ValueError("gumbel must be [B, max_depth+1, V]")
    if tuple(tree_tokens.shape) != (B, N) or tuple(tree_parent.shape) != (B, N):
        raise ValueError("tree arrays must be [B, N]")
    dev = hidden.device
    need = srt_accept_lmhead_scratch_bytes(B, N, V)
    with _on(stream):
        if out is None:
            out = _walk_outputs(B, max_depth, dev)
        if scratch is None or scratch.numel() < need:
            scratch = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("srt_accept_lmhead", lib().srt_accept_lmhead(
        B, N, dm, V, max_depth, _ptr(hidden, torch.bfloat16, "hidden"), _ptr(w_head, torch.bfloat16, "w_head"),
        _ptr(gumbel, torch.float32, "gumbel"), float(inv_temperature),
        _ptr(tree_tokens, torch.int32, "tree_tokens"), _ptr(tree_parent, torch.int32, "tree_parent"),
        _ptr(n_nodes, torch.int32, "n_nodes"), _ptr(out["n_accepted"], torch.int32),
        _ptr(out["out_tokens"], torch.int32), _ptr(out["out_nodes"], torch.int32),
        _ptr(out.get("n_emitted"), torch.int32), _ptr(scratch, name="scratch"), scratch.numel(),
        _stream(stream)))
    return out


# --------------------------------------------------------------------------- commit

def srt_commit(k_cache, v_cache, block_table, ctx_len, n_accepted, out_tokens, out_nodes, n_nodes_max: int,
               ctx_tail=None, draft_len=None, stream=None):
    """Moves the accepted nodes' K/V into place and advances ctx_len (and, if
    given, ctx_tail [B, Qmax] / draft_len [B]) in place."""
    B = int(ctx_len.numel())
    P, Hkv, page, d = k_cache.shape
    if v_cache.shape != k_cache.shape:
        raise ValueError("cache shape mismatch")
    dmax = int(out_tokens.shape[1]) - 1
    qmax = int(ctx_tail.shape[1]) if ctx_tail is not None else 0
    _check("srt_commit", lib().srt_commit(
        B, int(n_nodes_max), Hkv, d, page, int(block_table.shape[1]), P,
        _ptr(k_cache, torch.bfloat16, "k_cache"), _ptr(v_cache, torch.bfloat16, "v_cache"),
        _ptr(block_table, torch.int32, "block_table"), _ptr(ctx_len, torch.int32, "ctx_len"), dmax,
        _ptr(n_accepted, torch.int32, "n_accepted"), _ptr(out_tokens, torch.int32, "out_tokens"),
        _ptr(out_nodes, torch.int32, "out_nodes"), qmax, _ptr(ctx_tail, torch.int32, "ctx_tail"),
        _ptr(draft_len, torch.int32, "draft_len"), _stream(stream)))


def srt_version() -> str:
    return lib().srt_version().decode()
