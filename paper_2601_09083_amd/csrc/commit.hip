// Commit of the accepted path: key/value move and context advance.
//
// Method: Section 3 of the paper verifies the whole draft tree in one decode
// pass and keeps the accepted tokens as classic speculative decoding does
// (Appendix C: one pass, the KV cache read once).  The pass has computed the
// key and value vectors of every tree node at its tree slot; the accepted
// ones become the cached vectors of the positions their tokens now occupy:
// with the root at position L, tree node i at L + i and accepted nodes
// c_1 < ... < c_k, position L + j receives the vectors of L + c_j, the
// cached length becomes L + k + 1 and the bonus token (whose vectors the
// next pass computes, as its root) ends the committed sequence.  The draft
// tail and committed count advance by the k + 1 emitted tokens.
//
// GPU design: one workgroup per sequence.  The rows to move (accepted node
// j's K and V vectors of every KV head, d * 2 bytes each) are split into
// 16-byte pieces ordered by j; a chunk of up to kChunkPieces pieces is read
// into registers, the workgroup synchronises, and the chunk is written.  A
// chunk never reads a position an earlier chunk wrote (its sources are
// L + c_j' with c_j' >= j' > every earlier destination's j), and within a
// chunk every read precedes every write, so a path whose node c_i = j is
// both a source and a later destination is moved correctly.
#include "common.h"

using namespace srt;

namespace {

constexpr int kThreads = 256;
constexpr int kPer = 4;                          // pieces per thread per chunk
constexpr int kChunkPieces = kThreads * kPer;
constexpr int kMaxN = 256;

struct CommitArgs {
  uint16_t* k;
  uint16_t* v;
  const int32_t* bt;
  int32_t* ctx_len;
  const int32_t* n_accepted;
  const int32_t* out_tokens;
  const int32_t* out_nodes;
  int32_t* ctx_tail;
  int32_t* draft_len;
  int64_t num_pages;
  int32_t N, Hkv, d, page, max_pages, Dmax, Qmax;
};

// Element offset of (position, KV head) in a cache, or -1 if the position's
// page is outside the block table or the pool.
__device__ inline int64_t row_offset(const CommitArgs& a, int b, int64_t pos, int head) {
  if (pos < 0 || pos >= static_cast<int64_t>(a.max_pages) * a.page) return -1;
  const int pg = a.bt[static_cast<int64_t>(b) * a.max_pages + pos / a.page];
  if (pg < 0 || pg >= a.num_pages) return -1;
  return ((static_cast<int64_t>(pg) * a.Hkv + head) * a.page + pos % a.page) * a.d;
}

__global__ __launch_bounds__(kThreads) void commit_kernel(CommitArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t L = a.ctx_len[b];
  const int kmax = min(a.Dmax, a.N - 1);
  const int k = min(max(a.n_accepted[b], 0), kmax);
  const int32_t* nodes = a.out_nodes + static_cast<int64_t>(b) * (a.Dmax + 1);
  const int cpr = a.d / 8;  // 16-byte pieces per row
  const int64_t pieces = static_cast<int64_t>(k) * 2 * a.Hkv * cpr;

  for (int64_t c0 = 0; c0 < pieces; c0 += kChunkPieces) {
    uint4 val[kPer];
    int64_t dst[kPer];
    uint16_t* base[kPer];
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      dst[r] = -1;
      base[r] = nullptr;
      const int64_t it = c0 + r * kThreads + tid;
      if (it >= pieces) continue;
      const int c = static_cast<int>(it % cpr);
      const int64_t rowi = it / cpr;                 // ((j-1) * 2 + tensor) * Hkv + head
      const int head = static_cast<int>(rowi % a.Hkv);
      const int tensor = static_cast<int>((rowi / a.Hkv) % 2);
      const int j = static_cast<int>(rowi / (2 * a.Hkv)) + 1;
      const int src_node = nodes[j - 1];
      if (src_node < 1 || src_node >= a.N) continue;
      const int64_t so = row_offset(a, b, L + src_node, head);
      const int64_t dof = row_offset(a, b, L + j, head);
      if (so < 0 || dof < 0) continue;
      uint16_t* t = tensor ? a.v : a.k;
      val[r] = *reinterpret_cast<const uint4*>(t + so + 8 * c);
      dst[r] = dof + 8 * c;
      base[r] = t;
    }
    // Every read of the chunk has returned before any wave writes: the loads
    // are waited for explicitly (a workgroup fence alone does not order a
    // load of one wave before a store of another to the same address).
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPer; ++r)
      if (dst[r] >= 0) *reinterpret_cast<uint4*>(base[r] + dst[r]) = val[r];
    __syncthreads();
  }

  // Draft tail: shift left by the k + 1 emitted tokens and append them.
  const int e = k + 1;
  if (a.ctx_tail) {
    const int64_t t = a.draft_len[b];
    int32_t* row = a.ctx_tail + static_cast<int64_t>(b) * a.Qmax;
    const int32_t* emitted = a.out_tokens + static_cast<int64_t>(b) * (a.Dmax + 1);
    int32_t nv = -1;
    const int i = tid;
    if (i < a.Qmax) {
      const int src = i + e;  // in the frame old tail [0, Qmax) ++ emitted [Qmax, Qmax + e)
      const int64_t valid_from = a.Qmax - min<int64_t>(max<int64_t>(t, 0), a.Qmax);
      if (src >= a.Qmax) nv = emitted[src - a.Qmax];
      else if (src >= valid_from) nv = row[src];
    }
    __syncthreads();
    if (i < a.Qmax) row[i] = nv;
    if (tid == 0) a.draft_len[b] = static_cast<int32_t>(t + e);
  }
  __syncthreads();  // every thread has read ctx_len[b]
  if (tid == 0) a.ctx_len[b] = static_cast<int32_t>(L + e);
}

}  // namespace

extern "C" int srt_commit(int32_t B, int32_t N, int32_t Hkv, int32_t d, int32_t page, int32_t max_pages,
                          int64_t num_pages, uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                          int32_t* ctx_len, int32_t Dmax, const int32_t* n_accepted, const int32_t* out_tokens,
                          const int32_t* out_nodes, int32_t max_match, int32_t* ctx_tail, int32_t* draft_len,
                          void* stream) {
  if (B < 0 || N < 1 || N > kMaxN || Hkv < 1 || page < 1 || max_pages < 1 || num_pages < 1 || Dmax < 0 || Dmax > 63)
    return SRT_ERR_INVALID;
  if (d < 8 || d > 1024 || d % 8) return SRT_ERR_UNSUPPORTED;
  if ((ctx_tail == nullptr) != (draft_len == nullptr)) return SRT_ERR_INVALID;
  if (ctx_tail && (max_match < 1 || max_match > 64)) return SRT_ERR_INVALID;
  if (B == 0) return SRT_OK;
  if (!k_cache || !v_cache || !block_table || !ctx_len || !n_accepted || !out_tokens || !out_nodes)
    return SRT_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(k_cache) | reinterpret_cast<uintptr_t>(v_cache)) % 16) return SRT_ERR_INVALID;
  CommitArgs a;
  a.k = k_cache;
  a.v = v_cache;
  a.bt = block_table;
  a.ctx_len = ctx_len;
  a.n_accepted = n_accepted;
  a.out_tokens = out_tokens;
  a.out_nodes = out_nodes;
  a.ctx_tail = ctx_tail;
  a.draft_len = draft_len;
  a.num_pages = num_pages;
  a.N = N;
  a.Hkv = Hkv;
  a.d = d;
  a.page = page;
  a.max_pages = max_pages;
  a.Dmax = Dmax;
  a.Qmax = ctx_tail ? max_match : 0;
  commit_kernel<<<B, kThreads, 0, as_stream(stream)>>>(a);
  return launch_status();
}
