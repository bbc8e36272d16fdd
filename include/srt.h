/*
 * srt.h -- C ABI of libsrt: the tree-speculative verification step of SRT
 * (Speculative Rollout with Tree-Structured Cache, arXiv 2601.09083) on AMD
 * Instinct MI355X (gfx950).
 *
 * One verification step is
 *   srt_draft      -> tree of drafted tokens from the per-prompt cache
 *   (caller)       -> writes the tree's K/V into the paged cache, RoPE, ...
 *   srt_tree_attn  -> attention of every tree node over context + ancestors
 *   (caller)       -> LM head: per-node logits
 *   srt_accept     -> accepted path + bonus token
 *   (or srt_accept_lmhead: the LM head and the walk fused, on the visited
 *    nodes only)
 *   srt_trie_insert-> emitted tokens appended to the sequence's stream
 *   srt_commit     -> accepted nodes' K/V moved into place, context advanced
 *
 * Conventions shared by every entry point
 *   - Pointers are device pointers unless the comment says "host".  All
 *     device memory is owned by the caller and the library allocates
 *     nothing.  The only state kept between calls is a per-device cache of
 *     the compute-unit count (read once per device, used to size the
 *     persistent attention grid) and, for srt_accept_noalloc only, a fixed
 *     per-device scratch array and its address; no call's results depend on
 *     an earlier call except through the buffers the caller passes.
 *   - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *     Every call only enqueues work on it and returns, except those marked
 *     "synchronises".  Calls sharing a workspace must be ordered on one
 *     stream (or by the caller).
 *   - Return value: SRT_OK, or a negative srt_status.  Argument errors are
 *     found on the host before anything is enqueued (SRT_ERR_INVALID /
 *     SRT_ERR_UNSUPPORTED); launch failures give SRT_ERR_HIP.  Conditions
 *     only the device can see (cache full, a stream bound to another prompt,
 *     out-of-range ids) set sticky flags in the workspace, read with
 *     srt_trie_status; the kernels never access memory outside the
 *     documented extents, whatever the device-side values are.
 *   - bf16 values travel as uint16_t bit patterns.
 */
#ifndef SRT_H_
#define SRT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SRT_OK = 0,
  SRT_ERR_INVALID = -1,      /* bad argument (host check) */
  SRT_ERR_CAPACITY = -2,     /* workspace / output too small */
  SRT_ERR_HIP = -3,          /* HIP runtime or launch error */
  SRT_ERR_UNSUPPORTED = -4   /* valid but not implemented (e.g. head_dim) */
} srt_status;

/* Sticky device-side flags reported by srt_trie_status (bit mask). */
#define SRT_FLAG_CAPACITY  1u  /* node table full: later inserts are dropped */
#define SRT_FLAG_STREAM    2u  /* a stream id was out of range or bound to another prompt */
#define SRT_FLAG_PROMPT    4u  /* a prompt id was out of range */

/* ------------------------------------------------------------------------
 * Per-prompt cache (Section 3, "Per-prompt rollout cache using
 * tree-structured cache" and "Cache update strategy").
 *
 * The cache of prompt p holds count(s) for every token string s with
 * 1 <= |s| <= max_depth that occurs in the streams inserted for p, where
 * count(s) is the number of occurrences (stream, start position); no
 * occurrence spans two streams.  A stream is one rollout (prior, running, or
 * run-ahead) and is identified by a caller-chosen id < max_streams; it is
 * bound to the prompt of its first insert.
 * ---------------------------------------------------------------------- */
typedef struct {
  int32_t n_prompts;      /* number of per-prompt caches, >= 1 */
  int32_t max_streams;    /* stream ids are 0..max_streams-1, >= 1 */
  int32_t max_depth;      /* D: longest indexed substring, 1..64 */
  int32_t reserved;       /* must be 0 */
  int64_t node_capacity;  /* most nodes (strings) over all prompts, >= 1 */
} srt_trie_config;

/* Bytes of device memory the workspace needs for `cfg` (host only, no HIP
 * call).  Returns 0 if `cfg` is invalid. */
size_t srt_trie_workspace_bytes(const srt_trie_config* cfg);

/* Formats `ws` (device, ws_bytes >= srt_trie_workspace_bytes(cfg), 256-byte
 * aligned) as empty caches for every prompt and unbound streams. */
int srt_trie_init(void* ws, size_t ws_bytes, const srt_trie_config* cfg, void* stream);

/* Appends tokens to streams and updates the counts (online insertion).
 * Entry i appends tokens[i*stride + 0 .. lengths[i]-1] to stream
 * stream_ids[i] of prompt prompt_ids[i]: for each appended token at stream
 * index j, every suffix of the stream ending at j of length <= D gains one
 * occurrence.  Arrays: prompt_ids, stream_ids, lengths [n] int32; tokens
 * [n, stride] int32 (tokens >= 0).  Stream ids must be distinct within one
 * call.  n == 0 is a no-op.  Entries with an out-of-range prompt or stream,
 * or a stream bound to another prompt, are skipped and flagged. */
int srt_trie_insert(void* ws, int32_t n, const int32_t* prompt_ids, const int32_t* stream_ids,
                    const int32_t* tokens, const int32_t* lengths, int32_t stride, void* stream);

/* Unbinds streams so their ids can start new rollouts (of any prompt).  The
 * counts they contributed stay in the cache.  stream_ids [n] int32. */
int srt_trie_reset_streams(void* ws, int32_t n, const int32_t* stream_ids, void* stream);

/* Synchronises.  info (host, [4] int64): flags (SRT_FLAG_*), nodes in use,
 * node_capacity, hash-table slots.  Returns SRT_ERR_CAPACITY if the
 * capacity flag is set, else SRT_OK. */
int srt_trie_status(const void* ws, int64_t* info, void* stream);

/* Synchronises.  Dumps the cache of `prompt_id` breadth-first: row r is one
 * string s (depth 1 first), with parent[r] the row of s minus its last token
 * (-1 at depth 1), token[r] its last token and count[r] = count(s).  The
 * order of rows within a depth is unspecified.  Arrays (device) hold
 * max_nodes rows.  *n_out (host) receives the number of strings; if it
 * exceeds max_nodes only max_nodes rows are written and SRT_ERR_CAPACITY is
 * returned.  Test and checkpoint hook, not on the hot path. */
int srt_trie_export(const void* ws, int32_t prompt_id, int64_t max_nodes, int32_t* parent,
                    int32_t* token, uint32_t* count, int64_t* n_out, void* stream);

/* ------------------------------------------------------------------------
 * Draft extraction (Section 3, "Speculative Rollout with Tree-Structured
 * Cache"; the edge score is the displayed equation there).
 *
 * For sequence b with t = ctx_len[b] committed tokens, the last
 * min(t, max_match) of them right-aligned in ctx_tail[b, 0..max_match-1]:
 *   q* = the longest q <= min(t, max_match) such that the last q tokens form
 *        a string of the prompt's cache with at least one continuation;
 *   u  = that string; q* = 0 means fall back to a one-node tree.
 *   Candidates are the descendants v of u up to relative depth
 *   min(max_depth, D - q*), with C(v) = count(v) / sum over the children w
 *   of parent(v) of count(w) (one IEEE fp64 division) and
 *   score(v) = score(parent(v)) * C(v) (one fp64 multiplication),
 *   score(u) = 1.  They are ranked by score (descending), then relative
 *   depth (ascending), then token path from u (lexicographic by token id),
 *   and the first B are drafted, B = max_nodes - 1, or
 *   min(max_nodes - 1, floor(budget_alpha * q*)) when budget_alpha > 0;
 *   with min_score > 0 only those of score >= min_score; chain drafts keep
 *   only each node's best child among the candidates.
 * Output tree (row-major [B, max_nodes] int32, rows >= n_nodes[b] set to -1):
 *   node 0 = last committed token (ctx_tail[b, max_match-1], -1 if t == 0),
 *   parent -1, depth 0; nodes 1.. = drafted nodes in rank order, each with
 *   the index of its parent (< its own index) and its depth relative to u.
 * n_nodes[b] = 1 + drafted, match_len[b] = q*.  Results are bit-identical
 * across runs and launch shapes.
 * ---------------------------------------------------------------------- */
typedef struct {
  int32_t max_match;     /* Qmax: 1..64, columns of ctx_tail */
  int32_t max_nodes;     /* N: tree rows including the root, 1..256 */
  int32_t max_depth;     /* Dmax: 0..63 */
  int32_t chain;         /* 0: tree draft; 1: chain draft -- every node
                            contributes only its best child (largest count,
                            then smallest token), so the draft is one path */
  double budget_alpha;   /* <= 0: budget N-1 */
  double min_score;      /* <= 0: off; else only candidates whose score is
                            >= min_score are drafted (at most B of them) */
} srt_draft_params;

int srt_draft(const void* ws, int32_t B, const int32_t* prompt_ids, const int32_t* ctx_tail,
              const int32_t* ctx_len, const srt_draft_params* params, int32_t* tree_tokens,
              int32_t* tree_parent, int32_t* tree_depth, int32_t* n_nodes, int32_t* match_len,
              void* stream);

/* ------------------------------------------------------------------------
 * Tree-masked attention over a paged KV cache (Section 3: one decode pass
 * verifies every drafted token; Appendix C: the KV cache is read once).
 *
 * For sequence b, query head h (KV head g = h / (Hq / Hkv)) and tree node
 * i < n_nodes[b]:
 *   keys = positions [0, L) and L + j for every ancestor-or-self j of i,
 *   L = ctx_len[b]; position p lives in page block_table[b, p / page],
 *   slot p % page;  out[b,i,h,:] = softmax(scale * q.K^T) V, with q and K
 *   used exactly as given (fp32 dot products, the scale applied to them).
 *   scale must be finite (else SRT_ERR_INVALID).
 * Layouts (bf16 bits): q, out [B, N, Hq, d]; k_cache, v_cache
 *   [num_pages, Hkv, page, d]; block_table [B, max_pages] int32;
 *   ctx_len, n_nodes [B] int32; tree_parent [B, N] int32 as from srt_draft.
 * Requirements: 1 <= n_nodes[b] <= N <= 256, parent[i] < i,
 *   L + n_nodes[b] <= max_pages * page, block_table entries < num_pages for
 *   the pages those positions use; page a power of two >= 16 (else
 *   SRT_ERR_UNSUPPORTED).  Values outside these ranges are clamped
 *   or read as zero (never out of bounds); rows i >= n_nodes[b] of out are
 *   not written.  d must be 64 or 128; Hq % Hkv == 0.
 * scratch: device buffer, 256-byte aligned, of at least
 * srt_tree_attn_scratch_bytes(...) bytes (always > 0): the work list the
 * call builds for its own kernels, plus split-context partial results when
 * a context can exceed one split.  A split is 8192 keys, or a smaller power
 * of two (down to 1024) when B * Hkv is small, chosen from B, Hkv, page and
 * max_pages alone (the results do not depend on it beyond fp32 rounding).
 * Owned by the caller; contents are overwritten; calls that share a
 * scratch buffer must not overlap.
 * Unsupported (SRT_ERR_UNSUPPORTED): B > 65535, Hkv > 255, max_pages *
 * page beyond 4095 splits, or N * Hq / Hkv / 256 > 2046.
 * ---------------------------------------------------------------------- */
size_t srt_tree_attn_scratch_bytes(int32_t B, int32_t N, int32_t Hq, int32_t Hkv, int32_t d,
                                   int32_t page, int32_t max_pages);

int srt_tree_attn(int32_t B, int32_t N, int32_t Hq, int32_t Hkv, int32_t d, int32_t page,
                  int32_t max_pages, int64_t num_pages, const uint16_t* q,
                  const uint16_t* k_cache, const uint16_t* v_cache, const int32_t* block_table,
                  const int32_t* ctx_len, const int32_t* tree_parent, const int32_t* n_nodes,
                  float scale, uint16_t* out, void* scratch, size_t scratch_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Acceptance walk (Sections 1 and 3: accept drafted tokens up to the first
 * mismatch, which keeps the policy's distribution exactly).
 *
 * From u = root, step k = 0, 1, ...:
 *   x_j = logits[b,u,j]                                   (gumbel == NULL)
 *   x_j = fl(fl(logits[b,u,j] * inv_temperature) + gumbel[b,k,j])  (fp32)
 *   tok = arg-max_j x_j, lowest j on ties;
 *   if a child c of u (tree_parent[b,c] == u, c > u) has tree_tokens[b,c]
 *   == tok and k < Dmax: accept it (out_tokens[b,k] = tok,
 *   out_nodes[b,k] = c), u = c, next step; else out_tokens[b,k] = tok is
 *   the bonus token, n_accepted[b] = k, stop.
 * Layouts: logits [B, N, V] fp32; gumbel [B, Dmax+1, V] fp32 or NULL
 * (greedy); tree_tokens, tree_parent [B, N] int32; n_nodes [B] int32;
 * outputs n_accepted [B], out_tokens, out_nodes [B, Dmax+1] int32 (unused
 * entries -1) and, if not NULL, n_emitted [B] = n_accepted + 1, the number
 * of tokens the sequence appends (ready as `lengths` for srt_trie_insert
 * with tokens = out_tokens, stride Dmax+1).  Inputs must be finite (results
 * are unspecified otherwise).
 * The batch walks one step per kernel (Dmax + 1 level kernels, the first
 * of which also resets the walk's state, and a last step kernel are always
 * enqueued; a level with no walking sequence exits at once).
 * scratch: device buffer, 256-byte aligned, of at least
 * srt_accept_scratch_bytes(B) bytes (else SRT_ERR_CAPACITY): per-step
 * lists of the walking sequences, their current nodes and per-chunk arg-max
 * candidates, two levels' worth (about 530 bytes per sequence).  Owned by the caller; contents are overwritten;
 * calls sharing a scratch buffer must not overlap.
 * ---------------------------------------------------------------------- */
size_t srt_accept_scratch_bytes(int32_t B);

int srt_accept(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits,
               const float* gumbel, float inv_temperature, const int32_t* tree_tokens,
               const int32_t* tree_parent, const int32_t* n_nodes, int32_t* n_accepted,
               int32_t* out_tokens, int32_t* out_nodes, int32_t* n_emitted, void* scratch,
               size_t scratch_bytes, void* stream);

/* ------------------------------------------------------------------------
 * srt_accept for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc).
 *
 * The same walk, arguments, outputs and results as srt_accept, bit for bit,
 * without the scratch argument: the per-level walker lists, current nodes
 * and candidates live in one fixed device array inside the library (about
 * 2.1 MB, sized for SRT_ACCEPT_NOALLOC_MAX_BATCH sequences), which every GPU
 * the library runs on holds until the process ends.  Its address is looked
 * up once per device on the first call made with that device current; the
 * call allocates nothing and calls no allocating routine.  B larger than
 * SRT_ACCEPT_NOALLOC_MAX_BATCH returns SRT_ERR_CAPACITY before anything is
 * enqueued; a failed address lookup returns SRT_ERR_HIP.  The array keeps
 * the last call's contents (every call resets the counters it needs itself).
 * All calls on one GPU share the array: calls that may overlap on one GPU
 * (different streams without ordering between them) race and must not be
 * issued.
 * ---------------------------------------------------------------------- */
#define SRT_ACCEPT_NOALLOC_MAX_BATCH 4096

int srt_accept_noalloc(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits,
                       const float* gumbel, float inv_temperature, const int32_t* tree_tokens,
                       const int32_t* tree_parent, const int32_t* n_nodes, int32_t* n_accepted,
                       int32_t* out_tokens, int32_t* out_nodes, int32_t* n_emitted, void* stream);

/* ------------------------------------------------------------------------
 * Acceptance walk with the LM head applied at the visited nodes only
 * (Sections 1 and 3: the single verification pass supplies the policy's
 * next-token distribution at every drafted node; the walk needs it only at
 * the nodes it visits).
 *
 * Same walk, outputs and conventions as srt_accept, with
 *   logits[b,u,j] = sum_k hidden[b,u,k] * w_head[j,k]
 * formed on demand for the visited nodes (fp32 sums of the exact bf16
 * products; the summation order is the kernel's, so a logit may differ from
 * the correctly rounded dot product by the fp32 rounding of its additions,
 * and with it an arg-max whose top two scores are that close; with inputs
 * whose partial sums are exact in fp32 the result equals srt_accept on the
 * materialised logits bit for bit).  No [B, N, V] logits tensor is formed.
 * The walk advances one depth level per kernel pair for the whole batch
 * (Dmax + 1 pairs are always enqueued; a level with no walking sequence
 * exits at once); each level reads the head once.  Once the subtrees of
 * the walking sequences' current nodes hold few enough nodes, one pass
 * computes the arg-max of all of them and every walk is completed from
 * those (same results: a node's dot product does not depend on the pass).
 * Layouts: hidden [B, N, d_model] bf16 bits (the final hidden state of each
 * tree node), w_head [V, d_model] bf16 bits, both 16-byte aligned; gumbel
 * [B, Dmax+1, V] fp32 or NULL (greedy; inv_temperature then unused, else it
 * must be finite); tree arrays and outputs as srt_accept (unused entries
 * of out_tokens / out_nodes are -1).  d_model must be a multiple of 64
 * (else SRT_ERR_UNSUPPORTED); 0 <= Dmax <= 63.
 * scratch: device buffer, 256-byte aligned, of at least
 * srt_accept_lmhead_scratch_bytes(B, N, V) bytes (else SRT_ERR_CAPACITY):
 * per-level lists of walking sequences and of their subtrees' nodes, a
 * node-to-row table (4 bytes per tree node) and per-tile arg-max
 * candidates (8 bytes per row per 128 vocabulary entries, for max(B, 128)
 * rows).  Owned by
 * the caller; contents are overwritten; calls sharing a scratch buffer must
 * not overlap.
 * ---------------------------------------------------------------------- */
size_t srt_accept_lmhead_scratch_bytes(int32_t B, int32_t N, int32_t V);

int srt_accept_lmhead(int32_t B, int32_t N, int32_t d_model, int32_t V, int32_t Dmax,
                      const uint16_t* hidden, const uint16_t* w_head, const float* gumbel,
                      float inv_temperature, const int32_t* tree_tokens, const int32_t* tree_parent,
                      const int32_t* n_nodes, int32_t* n_accepted, int32_t* out_tokens,
                      int32_t* out_nodes, int32_t* n_emitted, void* scratch, size_t scratch_bytes,
                      void* stream);

/* ------------------------------------------------------------------------
 * Commit of the accepted path (Section 3: the verification pass keeps the
 * accepted tokens as classic speculative decoding does; Appendix C).
 *
 * The verification pass computed the key/value vectors of every tree node i
 * at position L + i (L = ctx_len[b], the root at L).  With
 * k = n_accepted[b] and accepted nodes c_j = out_nodes[b, j-1], j = 1..k, as
 * returned by srt_accept (increasing tree indices, 1 <= c_j < N):
 *   K/V at position L + j  <-  K/V at position L + c_j, every KV head;
 *   positions <= L and > L + k are not written;
 *   ctx_len[b] += k + 1   (root and accepted nodes become context);
 * and, if ctx_tail is not NULL, the draft inputs advance by the k + 1
 * emitted tokens out_tokens[b, 0..k] (accepted tokens, then the bonus
 * token): ctx_tail[b] (right-aligned last max_match committed tokens, -1
 * padded, as srt_draft reads it) becomes the last max_match tokens of the
 * grown sequence and draft_len[b] += k + 1.  The bonus token is the next
 * pass's root; its vectors are the caller's to write at the new L.
 * Layouts: k_cache, v_cache [num_pages, Hkv, page, d] bf16 bits, 16-byte
 * aligned, updated in place; block_table [B, max_pages] int32; ctx_len,
 * n_accepted, draft_len [B] int32; out_tokens, out_nodes [B, Dmax+1]
 * int32; ctx_tail [B, max_match] int32.  ctx_tail and draft_len are both
 * NULL or both set.  k is clamped to [0, min(Dmax, N-1)]; a copy whose node
 * index is outside [1, N) or whose page is outside the block table or the
 * pool is skipped.  d must be a multiple of 8 up to 1024
 * (else SRT_ERR_UNSUPPORTED).
 * ---------------------------------------------------------------------- */
int srt_commit(int32_t B, int32_t N, int32_t Hkv, int32_t d, int32_t page, int32_t max_pages,
               int64_t num_pages, uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
               int32_t* ctx_len, int32_t Dmax, const int32_t* n_accepted, const int32_t* out_tokens,
               const int32_t* out_nodes, int32_t max_match, int32_t* ctx_tail, int32_t* draft_len,
               void* stream);

/* Library version string (host only). */
const char* srt_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SRT_H_ */
