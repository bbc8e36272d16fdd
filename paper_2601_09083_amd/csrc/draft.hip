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
//
// Tree drafts take a faster route first: a level-synchronous expansion that
// walks the child lists of many candidates at once (one list per lane) and
// orders the result once at the end (see draft_levels).  It gives the same
// tree; a sequence whose candidates overflow its LDS pool falls back to the
// one-at-a-time selection above, which also serves chain drafts.
#include <cmath>
#include <cstdint>
#include <type_traits>

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

// ---------------------------------------------------------------------------
// Level-synchronous expansion (tree drafts).
//
// The selected nodes are the `budget` best candidates under the total order,
// and no node ranks above its parent (its score is at most the parent's, its
// depth larger).  So the candidates can be discovered a level at a time: keep
// a pool of discovered candidates and, in each round, expand every pool entry
// not yet expanded that ranks, by (score, depth), behind fewer than `budget`
// entries, and whose children could too (see Cut).  When a round finds no
// such entry the pool holds the best `budget` candidates: an undiscovered
// candidate v has a discovered ancestor a that was never expanded, so at
// least `budget` candidates rank strictly above a by (score, depth), or above
// any child of a, and therefore strictly above v (which scores at most as
// much as a, deeper).  Each round adds the next level of the
// final tree, so the rounds follow the tree depth rather than the node count.
// The order itself (lexicographic token paths break ties) is computed once at
// the end.  Entries that cannot be selected are dropped as they are found; a
// round whose children do not fit the pool reports failure.
// ---------------------------------------------------------------------------
constexpr int kPool = 2048;     // candidate pool entries (entry 0 is u)
constexpr int kCompactAt = 512; // pool size above which a round starts with a compaction
constexpr uint8_t kOpen = 0;    // discovered, children not yet walked
constexpr uint8_t kDone = 1;    // children walked, or a leaf, or at the depth limit
constexpr uint8_t kDropped = 2; // cannot be selected
constexpr int64_t kNoKey = INT64_MAX;

struct Pool {
  double score[kPool];            // path product; -1 below the score threshold
  unsigned long long num[kPool];  // own count until scored, then the children's count sum; scratch at the end
  uint32_t first[kPool];          // child-list head
  int32_t tok[kPool];
  uint16_t par[kPool];
  uint16_t aux[kPool];            // compaction map, rank of the token path among its depth, position
  uint16_t pos[kPool];            // entries scoring strictly higher (set by compaction)
  uint16_t list[kPool];           // entries to expand; then all entries, by depth
  uint8_t depth[kPool];
  uint8_t state[kPool];
  uint32_t dcount[64];            // entries per depth (then per depth slot)
  uint32_t tcount[64];            // candidates tied at the cut's score, per depth
  uint32_t dstart[64];            // first list slot of each depth
  uint32_t m;                     // entries in use; appends reserve slots here
};

__device__ inline int rank_below(uint64_t bal) {
  return static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(bal >> 32),
                                                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bal), 0u)));
}

// Scores as signed integers: ordered like the (non-negative) scores, with the
// -1 of an entry below the score threshold under all of them.
__device__ inline int64_t score_key(double s) { return __double_as_longlong(s); }

// Runs f with a compile-time number of 64-entry chunks per lane covering n
// entries (n <= kWide).  Larger pools go through the out-of-line *_wide
// functions below, so that their register arrays do not weigh on the rest
// of the kernel.
constexpr int kWide = 16 * SRT_WAVE;

template <typename F>
__device__ inline auto by_chunks(int n, F f) {
  if (n <= SRT_WAVE) return f(std::integral_constant<int, 1>{});
  if (n <= 2 * SRT_WAVE) return f(std::integral_constant<int, 2>{});
  if (n <= 4 * SRT_WAVE) return f(std::integral_constant<int, 4>{});
  if (n <= 8 * SRT_WAVE) return f(std::integral_constant<int, 8>{});
  return f(std::integral_constant<int, kWide / SRT_WAVE>{});
}

// c[r] += the number of entries w in 1 .. M-1 scoring strictly above key r.
// Each entry is read from LDS once and compared with all R keys held here.
template <int R>
__device__ inline void count_above(const Pool& P, int M, const int64_t (&ks)[R], int (&c)[R]) {
#pragma unroll 4
  for (int w = 1; w < M; ++w) {
    const int64_t sw = score_key(P.score[w]);
#pragma unroll
    for (int r = 0; r < R; ++r) c[r] += static_cast<int>(sw > ks[r]);
  }
}

// The `budget`-th largest score key among entries 1 .. M-1 (0 if fewer than
// `budget` entries score above 0; entries below the score threshold never
// count), found bit by bit from the top with wave ballots.  An entry has fewer
// than `budget` entries of strictly larger score exactly when its key is at
// least this value.
template <int R>
__device__ int64_t kth_score_key(const Pool& P, int lane, int M, int budget) {
  int64_t k[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = lane + SRT_WAVE * r;
    k[r] = i >= 1 && i < M ? score_key(P.score[i]) : -1;
  }
  int64_t t = 0;
  for (int bit = 62; bit >= 0; --bit) {
    const int64_t c = t | (int64_t{1} << bit);
    int n = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) n += __popcll(__ballot(k[r] >= c));
    if (n >= budget) t = c;
  }
  return t;
}

// Which candidates can still be selected.  An entry has fewer than `budget`
// entries of strictly larger score exactly when its key is at least t, the
// `budget`-th largest key (kth_score_key).  Entries of equal score rank by
// depth first, so an entry scoring exactly t at depth d has, strictly ahead
// of it, every entry scoring above t and every entry scoring t at a smaller
// depth; it stays selectable while those number fewer than `budget`, i.e.
// while d <= dmax.  Adding entries only moves entries back, so whatever is
// not selectable never becomes so; and a selectable entry's parent is
// selectable too (it scores at least as much, at a smaller depth).
struct Cut {
  int64_t t;
  int dmax;
};

constexpr Cut kNoCut{INT64_MIN, 63};  // every entry (fewer entries than the budget)

__device__ inline bool selectable(int64_t key, int depth, const Cut& c) {
  return key > c.t || (key == c.t && depth <= c.dmax);
}

__device__ inline int64_t kth_key(const Pool& P, int lane, int M, int budget);

// The cut for entries 1 .. M-1 (M - 1 > budget): t, then one pass that
// counts the entries scoring above t and, per depth, those scoring t (the
// same entries kth_score_key counts, whatever their state: an entry dropped
// earlier either scores below t now or lies deeper than any depth it
// could change).
__device__ Cut cut_of(Pool& P, int lane, int M, int budget) {
  Cut c{kth_key(P, lane, M, budget), 63};
  P.tcount[lane] = 0;
  __syncthreads();
  int above = 0;
  for (int i0 = 0; i0 < M; i0 += SRT_WAVE) {
    const int i = i0 + lane;
    const int64_t k = i >= 1 && i < M ? score_key(P.score[i]) : INT64_MIN;
    above += __popcll(__ballot(k > c.t));
    if (k == c.t) atomicAdd(&P.tcount[P.depth[i]], 1u);
  }
  __syncthreads();
  const int cnt = static_cast<int>(P.tcount[lane]);  // lane = depth
  int incl = cnt;
#pragma unroll
  for (int off = 1; off < SRT_WAVE; off <<= 1) {
    const int o = __shfl_up(incl, off, SRT_WAVE);
    if (lane >= off) incl += o;
  }
  // tied entries shallower than depth `lane`, plus those above t
  const uint64_t ok = __ballot(above + incl - cnt < budget);
  c.dmax = 63 - __clzll(static_cast<long long>(ok));
  return c;
}

// Drops the n listed open entries that cannot be selected any more (see
// Cut), closes those that can but whose children cannot (scoring exactly t
// at depth dmax or deeper: a child scores at most as much, one level
// deeper), and compacts the list in place to the entries still to expand;
// returns its new length.
__device__ int drop_below(Pool& P, int lane, int n, const Cut& cut) {
  int kept = 0;
  for (int base = 0; base < n; base += SRT_WAVE) {
    const int j = base + lane;
    const int i = j < n ? P.list[j] : -1;
    const int64_t k = i >= 0 ? score_key(P.score[i]) : 0;
    const int d = i >= 0 ? P.depth[i] : 0;
    const bool sel = i >= 0 && selectable(k, d, cut);
    const bool keep = sel && !(k == cut.t && d >= cut.dmax);
    const uint64_t bal = __ballot(keep);  // every lane has read its entry
    if (keep) P.list[kept + rank_below(bal)] = static_cast<uint16_t>(i);
    else if (i >= 0) P.state[i] = sel ? kDone : kDropped;
    kept += __popcll(bal);
  }
  return kept;
}

// Marks for keeping entry 0 and every entry that can still be selected (not
// dropped, selectable under the cut), drops the rest, writes each kept
// entry's new index to aux and its count of entries scoring strictly higher
// to pos; returns the number kept.  Every entry scoring above a kept one is
// kept too, so the count holds after compaction.
template <int R>
__device__ int keep_marks(Pool& P, int lane, int M, const Cut& cut) {
  int c[R];
  int64_t ks[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = lane + SRT_WAVE * r;
    const bool live = i >= 1 && i < M && P.state[i] != kDropped;
    ks[r] = live ? score_key(P.score[i]) : kNoKey;
    c[r] = 0;
  }
  count_above<R>(P, M, ks, c);
  int kept = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = lane + SRT_WAVE * r;
    const bool keep = i == 0 || (i < M && ks[r] != kNoKey && selectable(ks[r], P.depth[i], cut));
    if (i < M && !keep) P.state[i] = kDropped;
    const uint64_t bal = __ballot(keep);
    if (keep) {
      P.aux[i] = static_cast<uint16_t>(kept + rank_below(bal));
      P.pos[i] = static_cast<uint16_t>(c[r]);
    }
    kept += __popcll(bal);
  }
  return kept;
}

// keep_marks without the counts (a round's compaction, where only the kept
// set matters); pos is left as it was.
template <int R>
__device__ int keep_marks_at(Pool& P, int lane, int M, const Cut& cut) {
  int kept = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = lane + SRT_WAVE * r;
    const bool live = i >= 1 && i < M && P.state[i] != kDropped;
    const bool keep = i == 0 || (live && selectable(score_key(P.score[i]), P.depth[i], cut));
    if (i < M && !keep) P.state[i] = kDropped;
    const uint64_t bal = __ballot(keep);
    if (keep) P.aux[i] = static_cast<uint16_t>(kept + rank_below(bal));
    kept += __popcll(bal);
  }
  return kept;
}

// Pools of more than kWide entries (a round that found many children, or
// many candidates tied at the budget-th score): the same results as the
// register-held versions, with at most kWide / SRT_WAVE chunks in registers.
constexpr int kWideR = kWide / SRT_WAVE;

// kth_score_key: the first kWide entries' keys held here, the rest read
// from LDS at every bit.
__device__ int64_t kth_score_key_wide(const Pool& P, int lane, int M, int budget) {
  int64_t k[kWideR];
#pragma unroll
  for (int r = 0; r < kWideR; ++r) {
    const int i = lane + SRT_WAVE * r;
    k[r] = i >= 1 && i < M ? score_key(P.score[i]) : -1;
  }
  int64_t t = 0;
  for (int bit = 62; bit >= 0; --bit) {
    const int64_t c = t | (int64_t{1} << bit);
    int n = 0;
#pragma unroll
    for (int r = 0; r < kWideR; ++r) n += __popcll(__ballot(k[r] >= c));
    for (int i0 = kWide; i0 < M; i0 += SRT_WAVE) {
      const int i = i0 + lane;
      n += __popcll(__ballot(i < M && score_key(P.score[i]) >= c));
    }
    if (n >= budget) t = c;
  }
  return t;
}

// keep_marks, kWide entries at a time.
__device__ int keep_marks_wide(Pool& P, int lane, int M, const Cut& cut) {
  int kept = 0;
  for (int base = 0; base < M; base += kWide) {
    int c[kWideR];
    int64_t ks[kWideR];
#pragma unroll
    for (int r = 0; r < kWideR; ++r) {
      const int i = base + lane + SRT_WAVE * r;
      const bool live = i >= 1 && i < M && P.state[i] != kDropped;
      ks[r] = live ? score_key(P.score[i]) : kNoKey;
      c[r] = 0;
    }
    count_above<kWideR>(P, M, ks, c);
#pragma unroll
    for (int r = 0; r < kWideR; ++r) {
      const int i = base + lane + SRT_WAVE * r;
      const bool keep = i == 0 || (i < M && ks[r] != kNoKey && selectable(ks[r], P.depth[i], cut));
      if (i < M && !keep) P.state[i] = kDropped;
      const uint64_t bal = __ballot(keep);
      if (keep) {
        P.aux[i] = static_cast<uint16_t>(kept + rank_below(bal));
        P.pos[i] = static_cast<uint16_t>(c[r]);
      }
      kept += __popcll(bal);
    }
  }
  return kept;
}

// keep_marks_at over any number of chunks.
__device__ int keep_marks_at_wide(Pool& P, int lane, int M, const Cut& cut) {
  int kept = 0;
  for (int i0 = 0; i0 < M; i0 += SRT_WAVE) {
    const int i = i0 + lane;
    const bool live = i >= 1 && i < M && P.state[i] != kDropped;
    const bool keep = i == 0 || (live && selectable(score_key(P.score[i]), P.depth[i], cut));
    if (i < M && !keep) P.state[i] = kDropped;
    const uint64_t bal = __ballot(keep);
    if (keep) P.aux[i] = static_cast<uint16_t>(kept + rank_below(bal));
    kept += __popcll(bal);
  }
  return kept;
}

// The budget-th largest score key among entries 1 .. M-1 (kth_score_key).
__device__ inline int64_t kth_key(const Pool& P, int lane, int M, int budget) {
  if (M > kWide) return kth_score_key_wide(P, lane, M, budget);
  return by_chunks(M, [&](auto rc) { return kth_score_key<decltype(rc)::value>(P, lane, M, budget); });
}

// Keeps entry 0 and every entry that can still be selected (see Cut), moved
// down in index order.  A kept entry's parent is kept too, and stays ahead
// of it.  With `counts`, each kept entry's count of entries scoring strictly
// higher goes to pos (the final compaction); without, only the kept set is
// made (a round's compaction).  Returns the new entry count.
__device__ __forceinline__ int compact(Pool& P, int lane, int M, int budget, bool counts) {
  const Cut cut = M - 1 > budget ? cut_of(P, lane, M, budget) : kNoCut;
  int kept;
  if (M > kWide) {
    kept = counts ? keep_marks_wide(P, lane, M, cut) : keep_marks_at_wide(P, lane, M, cut);
  } else {
    kept = by_chunks(M, [&](auto rc) {
      constexpr int R = decltype(rc)::value;
      if (counts) return keep_marks<R>(P, lane, M, cut);
      return keep_marks_at<R>(P, lane, M, cut);
    });
  }
  __syncthreads();
  if (kept < M) {
    // chunk by chunk: a chunk's new indices lie below its own range and above
    // every index already written
    for (int base = 0; base < M; base += SRT_WAVE) {
      const int i = base + lane;
      const bool keep = i < M && P.state[i] != kDropped;
      double sc = 0.0;
      unsigned long long nu = 0;
      uint32_t fi = 0;
      int32_t tk = 0;
      int ni = 0, np = 0xFFFF, dp = 0, stt = 0, above = 0;
      if (keep) {
        above = P.pos[i];
        sc = P.score[i];
        nu = P.num[i];
        fi = P.first[i];
        tk = P.tok[i];
        dp = P.depth[i];
        stt = P.state[i];
        ni = P.aux[i];
        if (i > 0) np = P.aux[P.par[i]];
      }
      __syncthreads();
      if (keep) {
        P.score[ni] = sc;
        P.num[ni] = nu;
        P.first[ni] = fi;
        P.tok[ni] = tk;
        P.par[ni] = static_cast<uint16_t>(np);
        P.depth[ni] = static_cast<uint8_t>(dp);
        P.state[ni] = static_cast<uint8_t>(stt);
        P.pos[ni] = static_cast<uint16_t>(above);
      }
      __syncthreads();
    }
  }
  if (lane == 0) P.m = static_cast<uint32_t>(kept);
  __syncthreads();
  return kept;
}

// Drafts the tree below u (child-list head u_head) and writes rows 1 .. n-1 of
// it; returns n, or 0 if the candidates overflowed the pool (nothing written).
__device__ int draft_levels(const TrieView& t, Pool& P, int lane, uint32_t u_head, int budget, int limit,
                            double min_score, int32_t* __restrict__ tree_tokens, int32_t* __restrict__ tree_parent,
                            int32_t* __restrict__ tree_depth) {
  if (lane == 0) {
    P.score[0] = 1.0;
    P.first[0] = u_head;
    P.par[0] = 0xFFFF;
    P.depth[0] = 0;
    P.state[0] = kOpen;
    P.m = 1;
  }
  __syncthreads();
  int M = 1;
  for (;;) {
    if (M > kCompactAt) M = compact(P, lane, M, budget, false);
    // List the open entries, then drop those that can no longer be selected.
    int n_open = 0;
    for (int base = 0; base < M; base += SRT_WAVE) {
      const int i = base + lane;
      const bool open = i < M && P.state[i] == kOpen;
      const uint64_t bal = __ballot(open);
      if (open) P.list[n_open + rank_below(bal)] = static_cast<uint16_t>(i);
      n_open += __popcll(bal);
    }
    if (n_open > 0 && M - 1 > budget) {
      __syncthreads();
      n_open = drop_below(P, lane, n_open, cut_of(P, lane, M, budget));
    }
    if (n_open == 0) break;
    __syncthreads();
    // Walk their child lists, one list per lane: each step loads the next
    // pointer, count, token and list head of a child together.
    for (int j = lane; j < n_open; j += SRT_WAVE) {
      const int i = P.list[j];
      const int cd = P.depth[i] + 1;
      const uint8_t cstate = cd >= limit ? kDone : kOpen;
      uint32_t c = P.first[i];
      unsigned long long total = 0;
      while (c != kNone) {
        const uint32_t nx = t.next[c];
        const uint32_t cn = t.count[c];
        const int32_t tk = static_cast<int32_t>(t.keys[c] & 0xFFFFFFFFull);
        const uint32_t f = t.first[c];
        const uint32_t slot = atomicAdd(&P.m, 1u);
        if (slot >= static_cast<uint32_t>(kPool)) break;
        P.num[slot] = cn;
        P.tok[slot] = tk;
        P.first[slot] = f;
        P.par[slot] = static_cast<uint16_t>(i);
        P.depth[slot] = static_cast<uint8_t>(cd);
        P.state[slot] = f == kNone ? kDone : cstate;
        total += cn;
        c = nx;
      }
      P.num[i] = total;
      P.state[i] = kDone;
    }
    __syncthreads();
    const uint32_t m1 = P.m;
    if (m1 > static_cast<uint32_t>(kPool)) return 0;
    // Scores of the new entries: C(v), then the path product.
    for (int i = M + lane; i < static_cast<int>(m1); i += SRT_WAVE) {
      const int pa = P.par[i];
      const double cv = static_cast<double>(static_cast<uint32_t>(P.num[i])) / static_cast<double>(P.num[pa]);
      double sc = P.score[pa] * cv;
      if (min_score > 0.0 && sc < min_score) {  // never selected, nor any descendant
        sc = -1.0;
        P.state[i] = kDropped;
      }
      P.score[i] = sc;
    }
    __syncthreads();
    M = static_cast<int>(m1);
  }

  __syncthreads();
  M = compact(P, lane, M, budget, true);

  // Entries 1 .. M-1 listed by depth (counting sort).
  P.dcount[lane] = 0;
  __syncthreads();
  for (int i = 1 + lane; i < M; i += SRT_WAVE) P.aux[i] = static_cast<uint16_t>(atomicAdd(&P.dcount[P.depth[i]], 1u));
  __syncthreads();
  const int cnt = static_cast<int>(P.dcount[lane]);  // lane = depth
  int start = cnt;
#pragma unroll
  for (int off = 1; off < SRT_WAVE; off <<= 1) {
    const int o = __shfl_up(start, off, SRT_WAVE);
    if (lane >= off) start += o;
  }
  start -= cnt;
  P.dstart[lane] = static_cast<uint32_t>(start);
  __syncthreads();
  for (int i = 1 + lane; i < M; i += SRT_WAVE) P.list[P.dstart[P.depth[i]] + P.aux[i]] = static_cast<uint16_t>(i);
  const uint64_t used = __ballot(cnt > 0);
  const int maxd = used ? 63 - __clzll(static_cast<long long>(used)) : 0;
  __syncthreads();
  if (lane == 0) P.aux[0] = 0;
  __syncthreads();

  // Rank of each token path among the paths of its depth, a depth at a time:
  // it orders (parent's rank, token).  num holds the keys of one depth.
  for (int d = 1; d <= maxd; ++d) {
    const int n = __shfl(cnt, d, SRT_WAVE);
    const int s0 = __shfl(start, d, SRT_WAVE);
    for (int j = lane; j < n; j += SRT_WAVE) {
      const int i = P.list[s0 + j];
      P.num[s0 + j] = (static_cast<unsigned long long>(P.aux[P.par[i]]) << 32) | static_cast<uint32_t>(P.tok[i]);
    }
    __syncthreads();
    for (int j = lane; j < n; j += SRT_WAVE) {
      const unsigned long long k = P.num[s0 + j];
      int r = 0;
#pragma unroll 4
      for (int w = 0; w < n; ++w) r += static_cast<int>(P.num[s0 + w] < k);
      P.aux[P.list[s0 + j]] = static_cast<uint16_t>(r);
    }
    __syncthreads();
  }

  // Position in the total order (score descending, depth ascending, token
  // path ascending).  Entries of equal score share their count of entries
  // scoring higher, which is where their group starts; within a group they
  // rank by the tie key (depth and path rank packed, larger first).  The keys
  // are gathered in group order by a counting sort on that start (into num;
  // the walks and their counts are done with it).
  for (int i = lane; i < M; i += SRT_WAVE) P.first[i] = 0;  // group sizes
  __syncthreads();
  for (int i = 1 + lane; i < M; i += SRT_WAVE) {
    const int g0 = P.pos[i];
    P.num[g0 + atomicAdd(&P.first[g0], 1u)] =
        (static_cast<unsigned long long>(63 - P.depth[i]) << 16) | static_cast<uint32_t>(0xFFFF - P.aux[i]);
  }
  __syncthreads();
  for (int i = 1 + lane; i < M; i += SRT_WAVE) {
    const int g0 = P.pos[i];
    const int g = static_cast<int>(P.first[g0]);
    const unsigned long long k =
        (static_cast<unsigned long long>(63 - P.depth[i]) << 16) | static_cast<uint32_t>(0xFFFF - P.aux[i]);
    int r = 0;
    for (int j = 0; j < g; ++j) r += static_cast<int>(P.num[g0 + j] > k);
    P.aux[i] = static_cast<uint16_t>(g0 + r);
  }
  __syncthreads();
  for (int i = 1 + lane; i < M; i += SRT_WAVE) {
    const int ps = P.aux[i];
    if (ps < budget) {
      const int pa = P.par[i];
      tree_tokens[ps + 1] = P.tok[i];
      tree_parent[ps + 1] = pa == 0 ? 0 : P.aux[pa] + 1;
      tree_depth[ps + 1] = P.depth[i];
    }
  }
  return 1 + min(budget, M - 1);
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
  __shared__ union {
    Smem seq;
    Pool pool;
  } shared;
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
  const bool chain = a.chain != 0;
  const int64_t row = static_cast<int64_t>(b) * N;

  if (!chain && qstar > 0 && budget > 0 && limit > 0) {
    const int n = draft_levels(t, shared.pool, lane, u_head, budget, limit, a.min_score, tree_tokens + row,
                               tree_parent + row, tree_depth + row);
    if (n > 0) {
      for (int i = n + lane; i < N; i += SRT_WAVE) {
        tree_tokens[row + i] = -1;
        tree_parent[row + i] = -1;
        tree_depth[row + i] = -1;
      }
      if (lane == 0) {
        tree_tokens[row] = root_tok;
        tree_parent[row] = -1;
        tree_depth[row] = 0;
        n_nodes[b] = n;
        match_len[b] = qstar;
      }
      return;
    }
    __syncthreads();  // the pool and the one-at-a-time state share memory
  }

  // One node at a time (chain drafts, and tree drafts that overflowed the pool).
  Smem& sm = shared.seq;
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
