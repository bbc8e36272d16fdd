// Draft extraction: longest-suffix match and best-first expansion.
//
// Method: Section 3 of the paper ("Speculative Rollout with Tree-Structured
// Cache").  The longest suffix of the committed tokens that the prompt's
// cache holds (with at least one continuation) selects node u; descendants
// of u are ranked by the product of edge scores C(v) = count(v) / sum of the
// counts of v's siblings (the displayed equation of Section 3) and drafted
// greedily up to the budget.
//
// Drafting variants: with min_score > 0 selection stops at the first
// candidate whose path-product score is below it (candidates leave the
// frontier in score order), and chain drafts push only the best child of
// each selected node, found while the child list is summed.
//
// GPU design: one wavefront per sequence.  Lane q-1 walks the suffix of
// length q from the root (all q in parallel) and a ballot picks the longest
// one that has a child.  Expansion keeps the candidate frontier in LDS; each
// selection is a wave-wide arg-max over a packed 128-bit key (fp64 score
// bits, depth, lexicographic rank of the parent, token), so the order is the
// exact total order: score descending, depth ascending, token path from u
// ascending.  The lexicographic order of token paths is represented by
// per-depth ranks of the selected nodes: two same-depth candidates compare
// by their parents' ranks, then by token; ranks of existing nodes keep their
// relative order when a node is added.  A frontier bounded at twice the node
// budget is exact: when it overflows, the worst of more than `budget`
// candidates is dropped, and it could never be selected.
#include <cmath>

#include "common.h"

using namespace srt;

namespace {

constexpr int kMaxN = 256;      // tree rows (root included)
constexpr int kFrontier = 512;  // frontier capacity, >= 2 * kMaxN
constexpr int kChildBuf = 64;   // children gathered per list segment

struct DraftArgs {
  int32_t Q, N, Dmax, chain;
  double alpha, min_score;
};

struct Smem {
  double sel_score[kMaxN];
  uint32_t sel_first[kMaxN];  // head of the node's child list
  int32_t sel_tok[kMaxN];
  int16_t sel_par[kMaxN];
  uint16_t sel_rank[kMaxN];
  uint8_t sel_depth[kMaxN];
  double f_score[kFrontier];
  uint32_t f_first[kFrontier];
  int32_t f_tok[kFrontier];
  uint16_t f_par[kFrontier];
  // one list segment: count, token and child-list head of each child
  uint32_t c_count[kChildBuf];
  int32_t c_tok[kChildBuf];
  uint32_t c_first[kChildBuf];
  uint32_t cursor;
  int nbuf;
};

struct Key {
  uint64_t hi, lo;  // larger is better; lo bit 63 marks a valid entry
};

__device__ inline bool better(const Key& a, const Key& b) { return a.hi > b.hi || (a.hi == b.hi && a.lo > b.lo); }

__device__ inline Key make_key(double score, int depth, int prank, int32_t tok, int idx) {
  Key k;
  k.hi = static_cast<uint64_t>(__double_as_longlong(score));  // scores are >= 0
  k.lo = (1ull << 63) | (static_cast<uint64_t>(63 - depth) << 50) | (static_cast<uint64_t>(255 - prank) << 42) |
         (static_cast<uint64_t>(0x7FFFFFFF - tok) << 11) | static_cast<uint64_t>(idx);
  return k;
}

__device__ inline Key wave_max(Key k) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    Key o{shfl_xor_u64(k.hi, off), shfl_xor_u64(k.lo, off)};
    if (better(o, k)) k = o;
  }
  return k;
}

__device__ inline Key wave_min(Key k) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    Key o{shfl_xor_u64(k.hi, off), shfl_xor_u64(k.lo, off)};
    if (better(k, o)) k = o;
  }
  return k;
}

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += shfl_xor_u64(v, off);
  return v;
}

__device__ inline int wave_sum_i(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, SRT_WAVE);
  return v;
}

__device__ inline Key frontier_key(const Smem& sm, int e) {
  const int par = sm.f_par[e];
  return make_key(sm.f_score[e], sm.sel_depth[par] + 1, sm.sel_rank[par], sm.f_tok[e], e);
}

// Lane 0 walks up to kChildBuf list entries starting at sm.cursor.  For
// each child the next pointer, count, token and the child's own list head
// are loaded together, so a list of k children costs k dependent loads and
// nothing more (a selected node's list head was fetched when it became a
// candidate).
__device__ inline int gather_children(const TrieView& t, Smem& sm, int lane) {
  if (lane == 0) {
    uint32_t c = sm.cursor;
    int k = 0;
    while (c != kNone && k < kChildBuf) {
      const uint32_t nx = t.next[c];
      sm.c_count[k] = t.count[c];
      sm.c_tok[k] = static_cast<int32_t>(t.keys[c] & 0xFFFFFFFFull);
      sm.c_first[k] = t.first[c];
      ++k;
      c = nx;
    }
    sm.cursor = c;
    sm.nbuf = k;
  }
  __syncthreads();
  return sm.nbuf;
}

// Pushes the children of selected node `i` onto the frontier (only the best
// one -- largest count, then smallest token -- for chain drafts).
__device__ void expand(const TrieView& t, Smem& sm, int i, int lane, int& fsize, bool chain) {
  const double ps = sm.sel_score[i];
  const int cdepth = sm.sel_depth[i] + 1;
  const int prank = sm.sel_rank[i];

  // Pass 1: the sum of the children's counts (the denominator of C); a list
  // that fits one segment stays in LDS for pass 2.
  if (lane == 0) sm.cursor = sm.sel_first[i];
  __syncthreads();
  uint64_t total = 0;
  int segments = 0, k;
  // best child so far: key (count << 32 | 0x7FFFFFFF - token), its list head
  uint64_t best_key = 0;
  uint32_t best_first = kNone;
  do {
    k = gather_children(t, sm, lane);
    const uint64_t c = lane < k ? sm.c_count[lane] : 0u;
    total += wave_sum_u64(c);
    if (chain) {
      const uint64_t key = lane < k ? (c << 32) | static_cast<uint32_t>(0x7FFFFFFF - sm.c_tok[lane]) : 0ull;
      uint64_t mx = key;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const uint64_t o = shfl_xor_u64(mx, off);
        mx = o > mx ? o : mx;
      }
      const uint64_t hit = __ballot(lane < k && key == mx);  // sibling tokens are distinct
      if (mx > best_key) {
        best_key = mx;
        best_first = __shfl(lane < k ? sm.c_first[lane] : kNone, __ffsll(static_cast<long long>(hit)) - 1, SRT_WAVE);
      }
    }
    ++segments;
    if (sm.cursor != kNone) __syncthreads();
  } while (sm.cursor != kNone);
  if (chain) {
    if (best_key != 0 && fsize < kFrontier) {
      if (lane == 0) {
        const double cv = static_cast<double>(static_cast<uint32_t>(best_key >> 32)) / static_cast<double>(total);
        sm.f_score[fsize] = ps * cv;  // C(v), then the path product
        sm.f_first[fsize] = best_first;
        sm.f_tok[fsize] = static_cast<int32_t>(0x7FFFFFFF - static_cast<uint32_t>(best_key & 0xFFFFFFFFull));
        sm.f_par[fsize] = static_cast<uint16_t>(i);
      }
      ++fsize;
    }
    __syncthreads();
    return;
  }
  if (segments > 1) {  // long list: walk it again
    __syncthreads();
    if (lane == 0) sm.cursor = sm.sel_first[i];
    __syncthreads();
  }
  const double dtotal = static_cast<double>(total);

  // Pass 2: scores, then insertion.
  for (int seg = 0; seg < segments; ++seg) {
    if (segments > 1) k = gather_children(t, sm, lane);
    double sc = 0.0;
    int32_t tok = 0;
    uint32_t cs = kNone;
    if (lane < k) {
      cs = sm.c_first[lane];
      const double cv = static_cast<double>(sm.c_count[lane]) / dtotal;  // C(v)
      sc = ps * cv;                                                       // path product
      tok = sm.c_tok[lane];
    }
    if (fsize + k <= kFrontier) {
      if (lane < k) {
        const int e = fsize + lane;
        sm.f_score[e] = sc;
        sm.f_first[e] = cs;
        sm.f_tok[e] = tok;
        sm.f_par[e] = static_cast<uint16_t>(i);
      }
      fsize += k;
      __syncthreads();
    } else {
      for (int j = 0; j < k; ++j) {
        const double jsc = __shfl(sc, j, SRT_WAVE);
        const int32_t jtok = __shfl(tok, j, SRT_WAVE);
        const uint32_t jslot = __shfl(cs, j, SRT_WAVE);
        if (fsize < kFrontier) {
          if (lane == 0) {
            sm.f_score[fsize] = jsc;
            sm.f_first[fsize] = jslot;
            sm.f_tok[fsize] = jtok;
            sm.f_par[fsize] = static_cast<uint16_t>(i);
          }
          ++fsize;
          __syncthreads();
          continue;
        }
        Key worst{~0ull, ~0ull};
        for (int e = lane; e < fsize; e += SRT_WAVE) {
          const Key ke = frontier_key(sm, e);
          if (better(worst, ke)) worst = ke;
        }
        worst = wave_min(worst);
        const Key kj = make_key(jsc, cdepth, prank, jtok, 0);
        // keys never tie across distinct entries, so compare without the index
        const bool replace = (kj.hi > worst.hi) || (kj.hi == worst.hi && (kj.lo >> 11) > (worst.lo >> 11));
        if (replace && lane == 0) {
          const int e = static_cast<int>(worst.lo & 0x7FF);
          sm.f_score[e] = jsc;
          sm.f_first[e] = jslot;
          sm.f_tok[e] = jtok;
          sm.f_par[e] = static_cast<uint16_t>(i);
        }
        __syncthreads();
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(64) void draft_kernel(const void* ws, const int32_t* __restrict__ prompt_ids,
                                                   const int32_t* __restrict__ ctx_tail,
                                                   const int32_t* __restrict__ ctx_len, DraftArgs a,
                                                   int32_t* __restrict__ tree_tokens, int32_t* __restrict__ tree_parent,
                                                   int32_t* __restrict__ tree_depth, int32_t* __restrict__ n_nodes,
                                                   int32_t* __restrict__ match_len) {
  __shared__ Smem sm;
  const TrieView t = trie_view_dev(ws);
  const int D = t.depth;
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int Q = a.Q, N = a.N;
  const int32_t* tail = ctx_tail + static_cast<int64_t>(b) * Q;
  const int tlen = max(ctx_len[b], 0);
  const int p = prompt_ids[b];
  const bool pvalid = p >= 0 && p < t.hdr->n_prompts;
  const int32_t root_tok = tlen >= 1 ? tail[Q - 1] : -1;

  // Longest suffix with a continuation: lane q-1 tries length q.
  const int qlim = pvalid ? min(min(tlen, Q), D - 1) : 0;
  const int q = lane + 1;
  uint32_t node = kNone, head = kNone;
  if (q <= qlim) {
    node = t.roots[p];
    for (int i = 0; i < q && node != kNone; ++i) {
      const int32_t x = tail[Q - q + i];
      node = x < 0 ? kNone : trie_lookup(t, node, static_cast<uint32_t>(x));
    }
    if (node != kNone) head = t.first[node];
  }
  const uint64_t ballot = __ballot(head != kNone);
  const int qstar = ballot ? 64 - __clzll(static_cast<long long>(ballot)) : 0;
  const uint32_t u_head = __shfl(head, qstar > 0 ? qstar - 1 : 0, SRT_WAVE);  // child list of u

  int budget = N - 1;
  if (a.alpha > 0.0 && qstar > 0) {
    const double f = floor(a.alpha * static_cast<double>(qstar));
    if (f < static_cast<double>(budget)) budget = static_cast<int>(f);
  }
  const int limit = qstar > 0 ? min(a.Dmax, D - qstar) : 0;

  if (lane == 0) {
    sm.sel_first[0] = qstar > 0 ? u_head : kNone;
    sm.sel_tok[0] = root_tok;
    sm.sel_par[0] = -1;
    sm.sel_depth[0] = 0;
    sm.sel_rank[0] = 0;
    sm.sel_score[0] = 1.0;
  }
  __syncthreads();
  int nsel = 1, fsize = 0;
  const bool chain = a.chain != 0;
  if (qstar > 0 && budget > 0 && limit > 0) expand(t, sm, 0, lane, fsize, chain);

  while (nsel - 1 < budget && fsize > 0) {
    Key best{0ull, 0ull};
    for (int e = lane; e < fsize; e += SRT_WAVE) {
      const Key ke = frontier_key(sm, e);
      if (better(ke, best)) best = ke;
    }
    best = wave_max(best);
    const int e = static_cast<int>(best.lo & 0x7FF);
    const double sc = sm.f_score[e];
    if (a.min_score > 0.0 && sc < a.min_score) break;  // every remaining candidate scores lower
    const uint32_t cs = sm.f_first[e];
    const int32_t tok = sm.f_tok[e];
    const int par = sm.f_par[e];
    const int depth = sm.sel_depth[par] + 1;
    const int prank = sm.sel_rank[par];
    __syncthreads();
    if (lane == 0 && e != fsize - 1) {  // remove entry e
      sm.f_score[e] = sm.f_score[fsize - 1];
      sm.f_first[e] = sm.f_first[fsize - 1];
      sm.f_tok[e] = sm.f_tok[fsize - 1];
      sm.f_par[e] = sm.f_par[fsize - 1];
    }
    --fsize;
    // Rank of the new node among the selected nodes of its depth.
    int before = 0;
    for (int m = lane; m < nsel; m += SRT_WAVE) {
      if (sm.sel_depth[m] == depth) {
        const int mp = sm.sel_par[m];
        const bool lt = sm.sel_rank[mp] < prank || (mp == par && sm.sel_tok[m] < tok);
        before += lt;
        if (!lt) sm.sel_rank[m] = sm.sel_rank[m] + 1;
      }
    }
    before = wave_sum_i(before);
    if (lane == 0) {
      sm.sel_first[nsel] = cs;
      sm.sel_tok[nsel] = tok;
      sm.sel_par[nsel] = static_cast<int16_t>(par);
      sm.sel_depth[nsel] = static_cast<uint8_t>(depth);
      sm.sel_rank[nsel] = static_cast<uint16_t>(before);
      sm.sel_score[nsel] = sc;
    }
    __syncthreads();
    ++nsel;
    if (depth < limit) expand(t, sm, nsel - 1, lane, fsize, chain);
  }

  const int64_t row = static_cast<int64_t>(b) * N;
  for (int i = lane; i < N; i += SRT_WAVE) {
    const bool in = i < nsel;
    tree_tokens[row + i] = in ? sm.sel_tok[i] : -1;
    tree_parent[row + i] = in ? sm.sel_par[i] : -1;
    tree_depth[row + i] = in ? sm.sel_depth[i] : -1;
  }
  if (lane == 0) {
    n_nodes[b] = nsel;
    match_len[b] = qstar;
  }
}

}  // namespace

extern "C" int srt_draft(const void* ws, int32_t B, const int32_t* prompt_ids, const int32_t* ctx_tail,
                         const int32_t* ctx_len, const srt_draft_params* params, int32_t* tree_tokens,
                         int32_t* tree_parent, int32_t* tree_depth, int32_t* n_nodes, int32_t* match_len,
                         void* stream) {
  if (!ws || !params || B < 0) return SRT_ERR_INVALID;
  const srt_draft_params& p = *params;
  if (p.max_match < 1 || p.max_match > 64 || p.max_nodes < 1 || p.max_nodes > kMaxN || p.max_depth < 0 ||
      p.max_depth > 63 || (p.chain != 0 && p.chain != 1) || !(p.budget_alpha == p.budget_alpha) ||
      !(p.min_score == p.min_score))
    return SRT_ERR_INVALID;
  if (B == 0) return SRT_OK;
  if (!prompt_ids || !ctx_tail || !ctx_len || !tree_tokens || !tree_parent || !tree_depth || !n_nodes ||
      !match_len)
    return SRT_ERR_INVALID;
  DraftArgs a{p.max_match, p.max_nodes, p.max_depth, p.chain, p.budget_alpha, p.min_score};
  draft_kernel<<<B, 64, 0, as_stream(stream)>>>(ws, prompt_ids, ctx_tail, ctx_len, a, tree_tokens, tree_parent,
                                               tree_depth, n_nodes, match_len);
  return launch_status();
}
