"""Seeded synthetic inputs for the SRT verification step.

This module is the only code shared by the HIP path's harness and the CPU
oracle.  It draws random inputs and nothing else: it holds none of the
method's arithmetic (no substring counting, no scoring, no attention, no
acceptance).  Every array it returns is handed byte-identically to both sides.

Workload shapes follow the five configurations the build is measured on
(see ``CONFIGS``).  They stand in for the paper's RL rollouts (PPO/GRPO on
MATH, DAPO/ReTool on DAPO-Math-17k, Section 4.1), which are not available:

* One uniform-random base sequence per prompt; every rollout of that prompt
  is an independent mutation of it (per base token: deleted with p_del;
  otherwise substituted by a uniformly different token with p_sub, then
  followed by an inserted uniform token with p_ins).  This models the
  cross-step similarity of rollouts of one prompt (Section 2, Fig. 1c).
* Context lengths are uniform or log-normal (median m, max M, sigma =
  ln(M/m)/3, clipped to [16, M]) to model the long-tailed response lengths
  of Section 2 (Fig. 1b) and the length limits of Appendix A, Table 2.
* Q/K/V are N(0,1) rounded to bf16; the KV page pool is a random
  permutation.  Logits are N(0, sigma) per tree node, optionally with the
  token of the node's first drafted child boosted; Gumbel noise is
  -log(-log U) with U uniform on the open interval (0, 1).
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

# ---------------------------------------------------------------------------
# configurations
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class Dist:
    """A length distribution: ("fixed", n), ("uniform", lo, hi) or
    ("lognormal", median, max)."""

    kind: str
    a: int
    b: int = 0

    def sample(self, rng: np.random.Generator, n: int) -> np.ndarray:
        if self.kind == "fixed":
            return np.full(n, self.a, dtype=np.int64)
        if self.kind == "uniform":
            return rng.integers(self.a, self.b + 1, size=n, dtype=np.int64)
        if self.kind == "lognormal":
            sigma = math.log(self.b / self.a) / 3.0
            z = rng.standard_normal(n)
            v = np.round(self.a * np.exp(sigma * z)).astype(np.int64)
            return np.clip(v, 16, self.b)
        raise ValueError(self.kind)

    @property
    def max(self) -> int:
        return self.a if self.kind == "fixed" else self.b


@dataclass(frozen=True)
class Config:
    name: str
    index: int                 # seed base: 1000 + index
    n_prompts: int
    seqs_per_prompt: int
    vocab: int
    rollouts_per_prompt: int
    rollout_len: Dist
    ctx_len: Dist
    n_nodes: int               # draft tree size N, root included
    max_depth: int             # Dmax, relative to the root
    hq: int
    hkv: int
    head_dim: int
    page: int = 16
    max_match: int = 8         # Qmax
    logit_sigma: float = 2.0
    boost: str = "literal"     # "none" | "literal" | "top"
    boost_add: float = 4.0
    boost_p: float = 0.7
    runahead_streams: int = 0  # run-ahead continuations inserted per step
    runahead_len: int = 0
    p_sub: float = 0.1
    p_del: float = 0.02
    p_ins: float = 0.02

    @property
    def batch(self) -> int:
        return self.n_prompts * self.seqs_per_prompt

    @property
    def trie_depth(self) -> int:
        """Depth cap D of the per-prompt tries: Qmax + Dmax."""
        return self.max_match + self.max_depth

    def scaled(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    # 4 prompts x 1 sequence, tries of 8 rollouts x 256 tokens, vocab 1024.
    "tiny": Config("tiny", 0, n_prompts=4, seqs_per_prompt=1, vocab=1024,
                   rollouts_per_prompt=8, rollout_len=Dist("fixed", 256),
                   ctx_len=Dist("uniform", 128, 512), n_nodes=8, max_depth=4,
                   hq=4, hkv=1, head_dim=64, logit_sigma=1.0, boost="none"),
    # Qwen2.5-1.5B-shaped attention layer, 64 sequences, contexts 1k-4k.
    "qwen1.5b": Config("qwen1.5b", 1, n_prompts=64, seqs_per_prompt=1, vocab=151936,
                       rollouts_per_prompt=16, rollout_len=Dist("uniform", 1024, 4096),
                       ctx_len=Dist("uniform", 1024, 4096), n_nodes=32, max_depth=8,
                       hq=12, hkv=2, head_dim=128),
    # GRPO group: 128 prompts x 8 responses, log-normal contexts (median 2k, max 16k).
    "grpo": Config("grpo", 2, n_prompts=128, seqs_per_prompt=8, vocab=151936,
                   rollouts_per_prompt=16, rollout_len=Dist("lognormal", 2048, 16384),
                   ctx_len=Dist("lognormal", 2048, 16384), n_nodes=64, max_depth=12,
                   hq=12, hkv=2, head_dim=128),
    # Qwen2.5-7B-shaped attention layer, 256 sequences, log-normal contexts
    # (median 4k, max 32k); prior rollouts are log-normal like the contexts,
    # so the caches cover the positions being drafted.
    "qwen7b": Config("qwen7b", 3, n_prompts=256, seqs_per_prompt=1, vocab=152064,
                     rollouts_per_prompt=16, rollout_len=Dist("lognormal", 4096, 32768),
                     ctx_len=Dist("lognormal", 4096, 32768), n_nodes=64, max_depth=12,
                     hq=28, hkv=4, head_dim=128),
    # Long-tail run-ahead regime: 8 sequences of 16k-32k, 256-node trees,
    # tries of 64 rollouts, 8 run-ahead continuations of 512 tokens per step.
    "longtail": Config("longtail", 4, n_prompts=8, seqs_per_prompt=1, vocab=152064,
                       rollouts_per_prompt=64, rollout_len=Dist("uniform", 16384, 32768),
                       ctx_len=Dist("uniform", 16384, 32768), n_nodes=256, max_depth=16,
                       hq=28, hkv=4, head_dim=128,
                       runahead_streams=8, runahead_len=512),
}


# ---------------------------------------------------------------------------
# token-level data: rollouts, running sequences, run-ahead continuations
# ---------------------------------------------------------------------------


def mutate(rng: np.random.Generator, base: np.ndarray, vocab: int, p_sub: float,
           p_del: float, p_ins: float) -> np.ndarray:
    """One mutated copy of ``base`` (see the module docstring)."""
    n = base.shape[0]
    deleted = rng.random(n) < p_del
    subst = rng.random(n) < p_sub
    offset = rng.integers(1, vocab, size=n)
    inserted = rng.random(n) < p_ins
    ins_tok = rng.integers(0, vocab, size=n)
    kept_tok = np.where(subst, (base + offset) % vocab, base)
    keep = ~deleted
    ins = keep & inserted
    per = keep.astype(np.int64) + ins.astype(np.int64)
    out = np.empty(int(per.sum()), dtype=np.int64)
    start = np.cumsum(per) - per
    out[start[keep]] = kept_tok[keep]
    out[start[ins] + 1] = ins_tok[ins]
    return out


@dataclass
class TokenWorkload:
    cfg: Config
    bases: List[np.ndarray]                 # per prompt
    prior: List[List[np.ndarray]]           # per prompt: prior rollouts
    seq_prompt: np.ndarray                  # [B] prompt of each running sequence
    seqs: List[np.ndarray]                  # [B] running sequence y (ctx_len + 1 tokens)
    ctx_len: np.ndarray                     # [B] tokens whose K/V are cached (L_b)
    runahead: List[np.ndarray] = field(default_factory=list)  # per sequence (may be empty)

    @property
    def batch(self) -> int:
        return int(self.seq_prompt.shape[0])

    def streams_of_prompt(self, p: int, with_seqs: bool = True) -> List[np.ndarray]:
        """Every stream inserted into prompt ``p``'s trie at set-up."""
        out = list(self.prior[p])
        if with_seqs:
            out += [self.seqs[b] for b in range(self.batch) if self.seq_prompt[b] == p]
        return out

    def ctx_tail(self) -> np.ndarray:
        """[B, Qmax] last Qmax committed tokens, right-aligned, -1 padded."""
        q = self.cfg.max_match
        out = np.full((self.batch, q), -1, dtype=np.int32)
        for b, y in enumerate(self.seqs):
            t = min(q, y.shape[0])
            out[b, q - t:] = y[y.shape[0] - t:]
        return out

    def draft_len(self) -> np.ndarray:
        """[B] committed tokens per sequence (t in the method section)."""
        return np.array([y.shape[0] for y in self.seqs], dtype=np.int32)


def make_tokens(cfg: Config, seed: Optional[int] = None) -> TokenWorkload:
    """Rollouts, running sequences and run-ahead continuations for ``cfg``."""
    ss = np.random.SeedSequence(1000 + cfg.index if seed is None else seed)
    s_len, s_base, s_roll, s_seq, s_run = ss.spawn(5)
    rng_len = np.random.Generator(np.random.PCG64(s_len))
    B = cfg.batch
    ctx = cfg.ctx_len.sample(rng_len, B)
    roll_len = cfg.rollout_len.sample(rng_len, cfg.n_prompts * cfg.rollouts_per_prompt)
    roll_len = roll_len.reshape(cfg.n_prompts, cfg.rollouts_per_prompt)
    seq_prompt = np.repeat(np.arange(cfg.n_prompts, dtype=np.int32), cfg.seqs_per_prompt)

    need = max(int(roll_len.max(initial=0)), int(ctx.max()) + 1 + cfg.runahead_len)
    base_len = int(need * 1.1) + 256
    base_seeds = s_base.spawn(cfg.n_prompts)
    bases = [np.random.Generator(np.random.PCG64(s)).integers(0, cfg.vocab, size=base_len)
             for s in base_seeds]

    mut = dict(vocab=cfg.vocab, p_sub=cfg.p_sub, p_del=cfg.p_del, p_ins=cfg.p_ins)
    prior: List[List[np.ndarray]] = []
    roll_seeds = s_roll.spawn(cfg.n_prompts)
    for p in range(cfg.n_prompts):
        rs = roll_seeds[p].spawn(cfg.rollouts_per_prompt)
        lst = []
        for r in range(cfg.rollouts_per_prompt):
            rng = np.random.Generator(np.random.PCG64(rs[r]))
            n = int(roll_len[p, r])
            lst.append(mutate(rng, bases[p][: int(n * 1.08) + 32], **mut)[:n].copy())
        prior.append(lst)

    seqs = []
    seq_seeds = s_seq.spawn(B)
    for b in range(B):
        rng = np.random.Generator(np.random.PCG64(seq_seeds[b]))
        n = int(ctx[b]) + 1
        y = mutate(rng, bases[seq_prompt[b]][: int(n * 1.08) + 32], **mut)[:n]
        if y.shape[0] < n:  # pad with fresh tokens in the unlikely short case
            y = np.concatenate([y, rng.integers(0, cfg.vocab, size=n - y.shape[0])])
        seqs.append(y.copy())

    runahead = []
    if cfg.runahead_streams:
        run_seeds = s_run.spawn(B)
        for b in range(B):
            rng = np.random.Generator(np.random.PCG64(run_seeds[b]))
            t = int(ctx[b]) + 1
            seg = bases[seq_prompt[b]][t: t + cfg.runahead_len + 64]
            runahead.append(mutate(rng, seg, **mut)[: cfg.runahead_len].copy())

    return TokenWorkload(cfg, bases, prior, seq_prompt, seqs, ctx.astype(np.int32), runahead)


def pack_streams(streams: Sequence[np.ndarray]):
    """Pack token streams into a padded [n, stride] int32 matrix + lengths."""
    n = len(streams)
    lens = np.array([s.shape[0] for s in streams], dtype=np.int32)
    stride = max(1, int(lens.max(initial=1)))
    mat = np.zeros((n, stride), dtype=np.int32)
    for i, s in enumerate(streams):
        mat[i, : s.shape[0]] = s
    return mat, lens


# ---------------------------------------------------------------------------
# dense tensors (torch, on any device)
# ---------------------------------------------------------------------------


def _gen(device, seed: int):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def make_kv(cfg: Config, ctx_len: np.ndarray, device="cpu", seed: Optional[int] = None,
            n_nodes: Optional[int] = None, headroom: int = 0):
    """Paged bf16 KV cache with room for ``n_nodes`` tree tokens per sequence,
    plus ``headroom`` positions for contexts that grow.

    Returns (q [B,N,Hq,d] bf16, k_cache, v_cache [P,Hkv,page,d] bf16,
    block_table [B,max_pages] int32 (-1 padded), num_pages)."""
    import torch
    seed = (1000 + cfg.index) * 7 + 1 if seed is None else seed
    N = cfg.n_nodes if n_nodes is None else n_nodes
    B = int(ctx_len.shape[0])
    pages_per = (ctx_len.astype(np.int64) + N + headroom + cfg.page - 1) // cfg.page
    P = int(pages_per.sum())
    max_pages = int(pages_per.max())
    rng = np.random.Generator(np.random.PCG64(seed))
    perm = rng.permutation(P).astype(np.int32)
    bt = np.full((B, max_pages), -1, dtype=np.int32)
    off = 0
    for b in range(B):
        k = int(pages_per[b])
        bt[b, :k] = perm[off: off + k]
        off += k
    g = _gen(device, seed)
    shape_kv = (P, cfg.hkv, cfg.page, cfg.head_dim)
    q = torch.randn((B, N, cfg.hq, cfg.head_dim), generator=g, device=device).to(torch.bfloat16)
    k = torch.randn(shape_kv, generator=g, device=device).to(torch.bfloat16)
    v = torch.randn(shape_kv, generator=g, device=device).to(torch.bfloat16)
    return q, k, v, torch.from_numpy(bt).to(device), P


def boost_tokens(tree_tokens: np.ndarray, tree_parent: np.ndarray, n_nodes: np.ndarray):
    """For every tree node, the token of its first child in tree order, or -1.

    Pure bookkeeping on the given tree (no part of the method)."""
    B, N = tree_tokens.shape
    out = np.full((B, N), -1, dtype=np.int64)
    for b in range(B):
        for c in range(int(n_nodes[b]) - 1, 0, -1):
            p = int(tree_parent[b, c])
            if 0 <= p < N:
                out[b, p] = tree_tokens[b, c]
    return out


def make_logits(cfg: Config, tree_tokens: np.ndarray, tree_parent: np.ndarray,
                n_nodes: np.ndarray, device="cpu", seed: Optional[int] = None,
                boost: Optional[str] = None, sigma: Optional[float] = None):
    """fp32 logits [B, N, V]: N(0, sigma), and with probability boost_p the
    token of each node's first child is boosted: "literal" adds boost_add,
    "top" sets it to the row maximum + boost_add."""
    import torch
    seed = (1000 + cfg.index) * 7 + 2 if seed is None else seed
    boost = cfg.boost if boost is None else boost
    sigma = cfg.logit_sigma if sigma is None else sigma
    B, N = tree_tokens.shape
    g = _gen(device, seed)
    logits = torch.randn((B, N, cfg.vocab), generator=g, device=device)
    logits.mul_(sigma)
    if boost != "none":
        bt = boost_tokens(tree_tokens, tree_parent, n_nodes)
        rng = np.random.Generator(np.random.PCG64(seed + 1))
        hit = (bt >= 0) & (rng.random(bt.shape) < cfg.boost_p)
        bi, ni = np.nonzero(hit)
        if bi.size:
            ti = torch.from_numpy(bt[bi, ni]).to(device)
            bi_t = torch.from_numpy(bi).to(device)
            ni_t = torch.from_numpy(ni).to(device)
            if boost == "literal":
                logits[bi_t, ni_t, ti] += cfg.boost_add
            elif boost == "top":
                rowmax = logits[bi_t, ni_t].amax(dim=-1)
                logits[bi_t, ni_t, ti] = rowmax + cfg.boost_add
            else:
                raise ValueError(boost)
    return logits


def make_gumbel(cfg: Config, batch: int, device="cpu", seed: Optional[int] = None):
    """fp32 Gumbel noise [B, Dmax+1, V], one row per tree depth."""
    import torch
    seed = (1000 + cfg.index) * 7 + 3 if seed is None else seed
    g = _gen(device, seed)
    shape = (batch, cfg.max_depth + 1, cfg.vocab)
    k = torch.randint(1, 1 << 24, shape, generator=g, device=device, dtype=torch.int32)
    u = k.to(torch.float64) * (1.0 / (1 << 24))
    return (-torch.log(-torch.log(u))).to(torch.float32)


def make_head(batch: int, n_nodes_max: int, d_model: int, vocab: int, device="cpu", seed: int = 0,
              kind: str = "normal", tree_tokens: Optional[np.ndarray] = None,
              tree_parent: Optional[np.ndarray] = None, n_nodes: Optional[np.ndarray] = None,
              plant_p: float = 0.0, density: float = 1.0):
    """Final hidden states [B, N, d_model] and LM-head weights [V, d_model],
    bf16 (synthetic: no trained head).

    kind "normal": N(0, 1) entries rounded to bf16.  kind "int": integers,
    uniform in [-3, 3] for the head and in [-1, 1] for the hidden states
    (zero with probability 1 - density), so every dot product and partial
    sum is an integer far below 2^24.  With probability plant_p a node's
    hidden state is replaced by the head row of its first drafted child's
    token (bookkeeping on the given tree, like the logit boost), which makes
    that token's score large for the walk to follow."""
    import torch
    g = _gen(device, seed)
    if kind == "normal":
        w = torch.randn((vocab, d_model), generator=g, device=device).to(torch.bfloat16)
        h = torch.randn((batch, n_nodes_max, d_model), generator=g, device=device).to(torch.bfloat16)
    elif kind == "int":
        w = torch.randint(-3, 4, (vocab, d_model), generator=g, device=device).to(torch.bfloat16)
        h = torch.randint(-1, 2, (batch, n_nodes_max, d_model), generator=g, device=device)
        if density < 1.0:
            keep = torch.rand((batch, n_nodes_max, d_model), generator=g, device=device) < density
            h = h * keep
        h = h.to(torch.bfloat16)
    else:
        raise ValueError(kind)
    if plant_p > 0.0:
        bt = boost_tokens(tree_tokens, tree_parent, n_nodes)
        rng = np.random.Generator(np.random.PCG64(seed + 1))
        hit = (bt >= 0) & (rng.random(bt.shape) < plant_p)
        bi, ni = np.nonzero(hit)
        if bi.size:
            ti = torch.from_numpy(bt[bi, ni]).to(device)
            h[torch.from_numpy(bi).to(device), torch.from_numpy(ni).to(device)] = w[ti]
    return h, w
