"""One SRT verification step on the GPU, assembled from the libsrt calls.

``VerifyState`` owns the device buffers of one workload (per-prompt caches,
paged KV cache, queries, logits, noise) and runs the calls of a step:
``srt_draft`` -> ``srt_tree_attn`` -> ``srt_accept`` -> ``srt_trie_insert``
-> ``srt_commit`` (the accepted path becomes context, so the next step drafts
and attends from the grown sequence).
Only buffer management and argument passing happen here; every step of the
path runs in the HIP kernels of libsrt.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

from . import srt
from . import workload as W


def _dev(a, device, dtype=torch.int32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


@dataclass
class Caches:
    """Per-prompt caches in one workspace, with stream bookkeeping."""

    ws: torch.Tensor
    n_prompts: int
    max_streams: int
    depth: int
    node_capacity: int
    next_stream: int = 0

    @classmethod
    def create(cls, n_prompts: int, max_streams: int, depth: int, node_capacity: int, device="cuda"):
        nbytes = srt.srt_trie_workspace_bytes(n_prompts, max_streams, depth, node_capacity)
        if nbytes == 0:
            raise ValueError("invalid cache configuration")
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        srt.srt_trie_init(ws, n_prompts, max_streams, depth, node_capacity)
        return cls(ws, n_prompts, max_streams, depth, node_capacity)

    def new_streams(self, k: int) -> np.ndarray:
        ids = np.arange(self.next_stream, self.next_stream + k, dtype=np.int32)
        self.next_stream += k
        if self.next_stream > self.max_streams:
            raise ValueError("out of stream ids")
        return ids

    def insert(self, prompt_ids, stream_ids, streams: List[np.ndarray], max_elems: int = 1 << 26):
        """Appends host token arrays to streams (chunked to bound the staging
        buffer)."""
        device = self.ws.device
        order = list(range(len(streams)))
        i = 0
        while i < len(order):
            j, width = i, 0
            while j < len(order):
                w = max(width, max(1, len(streams[order[j]])))
                if (j - i + 1) * w > max_elems and j > i:
                    break
                width = w
                j += 1
            sel = order[i:j]
            mat, lens = W.pack_streams([streams[k] for k in sel])
            srt.srt_trie_insert(self.ws, _dev(np.asarray(prompt_ids)[sel], device),
                                _dev(np.asarray(stream_ids)[sel], device), _dev(mat, device),
                                _dev(lens, device))
            i = j

    def status(self) -> dict:
        return srt.srt_trie_status(self.ws)

    def export(self, prompt_id: int, max_nodes: Optional[int] = None) -> Dict[tuple, int]:
        """Cache of one prompt as {token path: count}."""
        if max_nodes is None:
            max_nodes = self.status()["nodes"] + 1
        parent, token, count = srt.srt_trie_export(self.ws, prompt_id, max_nodes)
        paths: List[tuple] = [()] * len(parent)
        out = {}
        for r in range(len(parent)):
            p = int(parent[r])
            paths[r] = (paths[p] if p >= 0 else ()) + (int(token[r]),)
            out[paths[r]] = int(count[r])
        return out


def node_capacity_for(total_tokens: int, depth: int, headroom_tokens: int = 0) -> int:
    """An upper bound on distinct strings: every inserted token ends at most
    ``depth`` new strings."""
    return int((total_tokens + headroom_tokens) * depth) + 1024


@dataclass
class VerifyState:
    cfg: W.Config
    tokens: W.TokenWorkload
    caches: Caches
    seq_stream: np.ndarray
    device: str
    prompt_ids: torch.Tensor
    ctx_tail: torch.Tensor
    draft_len: torch.Tensor
    attn_len: torch.Tensor
    q: torch.Tensor
    k_cache: torch.Tensor
    v_cache: torch.Tensor
    block_table: torch.Tensor
    num_pages: int
    scale: float
    tree: dict = field(default_factory=dict)
    attn_out: Optional[torch.Tensor] = None
    scratch: Optional[torch.Tensor] = None
    logits: Optional[torch.Tensor] = None
    gumbel: Optional[torch.Tensor] = None
    acc: dict = field(default_factory=dict)
    accept_scratch: Optional[torch.Tensor] = None
    extra_streams: int = 0

    # ---- set-up ---------------------------------------------------------
    @classmethod
    def build(cls, cfg: W.Config, device="cuda", tokens: Optional[W.TokenWorkload] = None,
              steps_headroom: int = 64, with_seqs: bool = True, kv_headroom: int = 0):
        tw = W.make_tokens(cfg) if tokens is None else tokens
        B = tw.batch
        streams, sp = [], []
        for p in range(cfg.n_prompts):
            for s in tw.prior[p]:
                streams.append(s)
                sp.append(p)
        n_prior = len(streams)
        if with_seqs:
            streams += list(tw.seqs)
            sp += [int(x) for x in tw.seq_prompt]
        total = sum(len(s) for s in streams)
        run = cfg.runahead_streams * cfg.runahead_len
        head = steps_headroom * (B * (cfg.max_depth + 1) + run)
        max_streams = len(streams) + B + steps_headroom * cfg.runahead_streams + 16
        caches = Caches.create(cfg.n_prompts, max_streams, cfg.trie_depth,
                               node_capacity_for(total, cfg.trie_depth, head), device)
        ids = caches.new_streams(len(streams))
        caches.insert(sp, ids, streams)
        seq_stream = ids[n_prior:] if with_seqs else caches.new_streams(B)
        q, k, v, bt, P = W.make_kv(cfg, tw.ctx_len, device=device, headroom=kv_headroom)
        st = cls(cfg=cfg, tokens=tw, caches=caches, seq_stream=seq_stream.astype(np.int32), device=device,
                 prompt_ids=_dev(tw.seq_prompt, device), ctx_tail=_dev(tw.ctx_tail(), device),
                 draft_len=_dev(tw.draft_len(), device), attn_len=_dev(tw.ctx_len, device), q=q, k_cache=k,
                 v_cache=v, block_table=bt.to(torch.int32), num_pages=P,
                 scale=1.0 / math.sqrt(cfg.head_dim))
        st.seq_stream_dev = _dev(st.seq_stream, device)
        st.attn_out = torch.empty_like(q)
        need = srt.srt_tree_attn_scratch_bytes(B, cfg.n_nodes, cfg.hq, cfg.hkv, cfg.head_dim, cfg.page,
                                               int(bt.shape[1]))
        st.scratch = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
        return st

    def make_logits(self, boost: Optional[str] = None, sampled: bool = True, sigma: Optional[float] = None):
        """Per-node logits (boosting each node's first drafted child) and
        per-depth Gumbel noise, from the current tree."""
        tt = self.tree["tree_tokens"].cpu().numpy()
        tp = self.tree["tree_parent"].cpu().numpy()
        nn = self.tree["n_nodes"].cpu().numpy()
        self.logits = W.make_logits(self.cfg, tt, tp, nn, device=self.device, boost=boost, sigma=sigma)
        self.gumbel = W.make_gumbel(self.cfg, self.tokens.batch, device=self.device) if sampled else None

    # ---- the four calls of one step ---------------------------------------
    def draft(self, alpha: float = 0.0, min_score: float = 0.0, chain: bool = False):
        c = self.cfg
        self.tree = srt.srt_draft(self.caches.ws, self.prompt_ids, self.ctx_tail, self.draft_len, c.max_match,
                                  c.n_nodes, c.max_depth, alpha, out=self.tree or None, min_score=min_score,
                                  chain=chain)
        return self.tree

    def attention(self):
        return srt.srt_tree_attn(self.q, self.k_cache, self.v_cache, self.block_table, self.attn_len,
                                 self.tree["tree_parent"], self.tree["n_nodes"], self.scale, out=self.attn_out,
                                 scratch=self.scratch)

    def accept(self, inv_temperature: float = 1.0):
        if self.accept_scratch is None:
            self.accept_scratch = torch.empty(max(srt.srt_accept_scratch_bytes(self.tokens.batch), 1),
                                              dtype=torch.uint8, device=self.device)
        self.acc = srt.srt_accept(self.logits, self.gumbel, inv_temperature, self.tree["tree_tokens"],
                                  self.tree["tree_parent"], self.tree["n_nodes"], self.cfg.max_depth,
                                  out=self.acc or None, scratch=self.accept_scratch)
        return self.acc

    def insert(self):
        srt.srt_trie_insert(self.caches.ws, self.prompt_ids, self.seq_stream_dev, self.acc["out_tokens"],
                            self.acc["n_emitted"])

    def commit(self):
        srt.srt_commit(self.k_cache, self.v_cache, self.block_table, self.attn_len, self.acc["n_accepted"],
                       self.acc["out_tokens"], self.acc["out_nodes"], self.cfg.n_nodes, ctx_tail=self.ctx_tail,
                       draft_len=self.draft_len)

    def step(self, inv_temperature: float = 1.0):
        self.draft()
        self.attention()
        self.accept(inv_temperature)
        self.insert()
        self.commit()
