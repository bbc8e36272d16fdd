// Per-prompt token cache on the GPU: initialisation, online insertion,
// stream reset, status and export.
//
// Method: Section 3 of the paper ("Per-prompt rollout cache using
// tree-structured cache"; "Cache update strategy").  Every substring of at
// most D tokens of the inserted streams is a node whose count is its number
// of occurrences.  Appending token x at index j of a stream adds one
// occurrence to each suffix ending at j.
//
// GPU design: one workgroup per inserted segment; its threads walk
// independent chains, one per start position k of a substring that ends in
// the new segment.  A stream remembers its active nodes -- the nodes of its
// suffixes of length 1 .. D-1 -- so a chain that starts j tokens before the
// segment starts at the active node of length j instead of walking from the
// root; a chain that starts inside the segment starts at the prompt's root.
// Chain k descends along the segment's tokens creating nodes on demand (hash
// CAS) and adds one to the count of each node it reaches (every such
// substring ends in the new segment).  A segment of n tokens exposes
// n + D - 1 parallel chains of at most min(n, D) steps, so appending a few
// tokens costs a few dependent probes; count updates commute, so the
// resulting map does not depend on scheduling.  The chains that reach the
// end of the segment with fewer than D tokens are the new active nodes.
#include <algorithm>
#include <cstring>

#include "common.h"

using namespace srt;

namespace {

struct Layout {
  uint64_t slots;
  int32_t stream_stride;
  uint64_t off_roots, off_streams, off_keys, off_count, off_first, off_next, total;
};

uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

bool config_ok(const srt_trie_config* c) {
  return c && c->n_prompts >= 1 && c->max_streams >= 1 && c->max_depth >= 1 && c->max_depth <= 64 &&
         c->reserved == 0 && c->node_capacity >= 1;
}

bool make_layout(const srt_trie_config& c, Layout* L) {
  const double want = (static_cast<double>(c.node_capacity) + c.n_prompts) * 1.25 + 64.0;
  uint64_t slots = 64;
  while (static_cast<double>(slots) < want) {
    slots <<= 1;
    if (slots > (uint64_t(1) << kMaxSlotsLog2)) return false;
  }
  L->slots = slots;
  L->stream_stride = kStreamHead + c.max_depth;  // active nodes of lengths 1..D-1 (+1 spare)
  uint64_t off = align256(sizeof(WsHeader));
  L->off_roots = off;
  off = align256(off + sizeof(uint32_t) * static_cast<uint64_t>(c.n_prompts));
  L->off_streams = off;
  off = align256(off + sizeof(int32_t) * static_cast<uint64_t>(c.max_streams) * L->stream_stride);
  L->off_keys = off;
  off = align256(off + sizeof(uint64_t) * slots);
  L->off_count = off;
  off = align256(off + sizeof(uint32_t) * slots);
  L->off_first = off;
  off = align256(off + sizeof(uint32_t) * slots);
  L->off_next = off;
  off = align256(off + sizeof(uint32_t) * slots);
  L->total = off;
  return true;
}

unsigned grid_for(uint64_t n, unsigned block) {
  uint64_t g = (n + block - 1) / block;
  return static_cast<unsigned>(std::min<uint64_t>(std::max<uint64_t>(g, 1), 65536));
}

__global__ void fill_u32_kernel(uint32_t* p, uint64_t n, uint32_t v) {
  for (uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x; i < n; i += uint64_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

__global__ void fill_u64_kernel(unsigned long long* p, uint64_t n, unsigned long long v) {
  for (uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x; i < n; i += uint64_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

__global__ void write_header_kernel(WsHeader* dst, WsHeader h) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *dst = h;
}

__global__ void create_roots_kernel(void* ws, int32_t n_prompts) {
  const TrieView t = trie_view_dev(ws);
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < n_prompts) t.roots[p] = trie_get_or_create(t, kRootParent, static_cast<uint32_t>(p));
}

__global__ __launch_bounds__(1024) void insert_kernel(void* ws, const int32_t* __restrict__ prompt_ids,
                                                     const int32_t* __restrict__ stream_ids,
                                                     const int32_t* __restrict__ tokens,
                                                     const int32_t* __restrict__ lengths, int32_t stride) {
  const TrieView t = trie_view_dev(ws);
  const int D = t.depth;
  const int entry = blockIdx.x;
  __shared__ int s_ok, s_m;
  __shared__ uint32_t s_act[64];
  __shared__ uint32_t s_created;
  __shared__ int32_t* s_rec;

  const int p = prompt_ids[entry];
  const int sid = stream_ids[entry];
  const int len = lengths[entry];
  const int32_t* tok = tokens + static_cast<int64_t>(entry) * stride;

  if (threadIdx.x == 0) {
    int ok = 1, m = 0;
    int32_t* rec = nullptr;
    if (t.hdr->flags & SRT_FLAG_CAPACITY) {
      ok = 0;
    } else if (p < 0 || p >= t.hdr->n_prompts) {
      set_flag(t, SRT_FLAG_PROMPT);
      ok = 0;
    } else if (sid < 0 || sid >= t.hdr->max_streams || len < 0 || len > stride) {
      set_flag(t, SRT_FLAG_STREAM);
      ok = 0;
    } else {
      rec = t.streams + static_cast<int64_t>(sid) * t.hdr->stream_stride;
      if (rec[0] == -1) {
        rec[0] = p;
        rec[1] = 0;
      } else if (rec[0] != p) {
        set_flag(t, SRT_FLAG_STREAM);
        ok = 0;
      }
      if (ok) m = min(rec[1], D - 1);
    }
    s_ok = ok;
    s_m = m;
    s_rec = rec;
    s_created = 0;
  }
  __syncthreads();
  if (!s_ok) return;

  // Reject the entry whole if any token is negative.
  int bad = 0;
  for (int j = threadIdx.x; j < len; j += blockDim.x) bad |= tok[j] < 0;
  if (__syncthreads_or(bad)) {
    if (threadIdx.x == 0) set_flag(t, SRT_FLAG_STREAM);
    return;
  }

  // Active nodes before the segment: s_act[j-1] = node of the suffix of
  // length j (j = 1..m).
  const int m = s_m;
  int32_t* rec = s_rec;
  if (static_cast<int>(threadIdx.x) < m) s_act[threadIdx.x] = static_cast<uint32_t>(rec[kStreamHead + threadIdx.x]);
  __syncthreads();

  const uint32_t root = t.roots[p];
  const int chains = m + len;
  for (int c = threadIdx.x; c < chains; c += blockDim.x) {
    const int k = c - m;  // start of the substring, relative to the segment
    uint32_t node = k < 0 ? s_act[-k - 1] : root;
    int depth = k < 0 ? -k : 0;
    int j = k < 0 ? 0 : k;
    // Each step is one round trip: the probe is the CAS itself (a failed
    // CAS returns the slot's key), and the child-list push of a node created
    // in the previous step is issued together with this step's probe.
    uint32_t link = kNone, link_parent = 0;
    for (; j < len && depth < D && node != kNone; ++j, ++depth) {
      const uint64_t key = node_key(node, static_cast<uint32_t>(tok[j]));
      uint64_t h = mix64(key) & t.mask;
      uint32_t prev = kNone;
      if (link != kNone) prev = atomicExch(&t.first[link_parent], link);
      unsigned long long old = atomicCAS(&t.keys[h], kEmptyKey, (unsigned long long)key);
      if (link != kNone) t.next[link] = prev;
      uint64_t probes = 1;
      while (old != kEmptyKey && old != key && probes <= t.mask) {
        h = (h + 1) & t.mask;
        old = atomicCAS(&t.keys[h], kEmptyKey, (unsigned long long)key);
        ++probes;
      }
      if (old != kEmptyKey && old != key) {  // every slot taken
        set_flag(t, SRT_FLAG_CAPACITY);
        node = kNone;
        link = kNone;
        break;
      }
      if (old == kEmptyKey) {
        link = static_cast<uint32_t>(h);
        link_parent = node;
        atomicAdd(&s_created, 1u);
      } else {
        link = kNone;
      }
      node = static_cast<uint32_t>(h);
      atomicAdd(&t.count[node], 1u);
    }
    if (link != kNone) t.next[link] = atomicExch(&t.first[link_parent], link);
    // A chain that consumed the whole segment with fewer than D tokens ends
    // at the new active node of its length.
    if (j == len && depth < D && depth >= 1) rec[kStreamHead + depth - 1] = static_cast<int32_t>(node);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    rec[1] = rec[1] + len;
    // Nodes created by this segment are counted against the capacity once.
    const unsigned long long n = atomicAdd(&t.hdr->used, static_cast<unsigned long long>(s_created));
    if (n + s_created > t.hdr->node_limit) set_flag(t, SRT_FLAG_CAPACITY);
  }
}

__global__ void reset_streams_kernel(void* ws, int32_t n, const int32_t* __restrict__ ids) {
  const TrieView t = trie_view_dev(ws);
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int sid = ids[i];
  if (sid < 0 || sid >= t.hdr->max_streams) {
    set_flag(t, SRT_FLAG_STREAM);
    return;
  }
  int32_t* rec = t.streams + static_cast<int64_t>(sid) * t.hdr->stream_stride;
  rec[0] = -1;
  rec[1] = 0;
}

__global__ void export_reset_kernel(void* ws) {
  if (threadIdx.x == 0 && blockIdx.x == 0) static_cast<WsHeader*>(ws)->export_n = 0;
}

// Depth-1 strings of the prompt: every slot whose parent is the root.
__global__ void export_level1_kernel(const void* ws, uint32_t root, int64_t max_nodes, int32_t* parent,
                                     int32_t* token, uint32_t* count) {
  const TrieView t = trie_view_dev(ws);
  const uint64_t slots = t.mask + 1;
  for (uint64_t h = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x; h < slots;
       h += uint64_t(gridDim.x) * blockDim.x) {
    const unsigned long long key = t.keys[h];
    if (key != kEmptyKey && static_cast<uint32_t>(key >> 32) == root) {
      const unsigned long long idx = atomicAdd(&t.hdr->export_n, 1ull);
      if (static_cast<int64_t>(idx) < max_nodes) {
        parent[idx] = -1;
        token[idx] = static_cast<int32_t>(key & 0xFFFFFFFFull);
        count[idx] = static_cast<uint32_t>(h);  // slot id until its level is expanded
      }
    }
  }
}

// Breadth-first expansion of the remaining levels by one workgroup.  While a
// row's children are being appended, count[row] holds the row's slot id; it
// is replaced by the real count once its level is done.
__global__ __launch_bounds__(1024) void export_bfs_kernel(const void* ws, int64_t max_nodes, int32_t* parent,
                                                          int32_t* token, uint32_t* count) {
  const TrieView t = trie_view_dev(ws);
  __shared__ long long s_hi;
  if (threadIdx.x == 0) s_hi = static_cast<long long>(min<unsigned long long>(
                            atomicAdd(&t.hdr->export_n, 0ull), static_cast<unsigned long long>(max_nodes)));
  __syncthreads();
  long long lo = 0, hi = s_hi;
  while (lo < hi) {
    for (long long r = lo + threadIdx.x; r < hi; r += blockDim.x) {
      const uint32_t slot = count[r];
      for (uint32_t c = t.first[slot]; c != kNone; c = t.next[c]) {
        const unsigned long long idx = atomicAdd(&t.hdr->export_n, 1ull);
        if (static_cast<int64_t>(idx) < max_nodes) {
          parent[idx] = static_cast<int32_t>(r);
          token[idx] = static_cast<int32_t>(t.keys[c] & 0xFFFFFFFFull);
          count[idx] = c;
        }
      }
    }
    __syncthreads();
    for (long long r = lo + threadIdx.x; r < hi; r += blockDim.x) count[r] = t.count[count[r]];
    __syncthreads();
    if (threadIdx.x == 0) s_hi = static_cast<long long>(min<unsigned long long>(
                              atomicAdd(&t.hdr->export_n, 0ull), static_cast<unsigned long long>(max_nodes)));
    __syncthreads();
    lo = hi;
    hi = s_hi;
  }
}

int read_header(const void* ws, WsHeader* h, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(h, ws, sizeof(WsHeader), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return SRT_ERR_HIP;
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return SRT_ERR_HIP;
  return h->magic == kMagic ? SRT_OK : SRT_ERR_INVALID;
}

}  // namespace

extern "C" {

size_t srt_trie_workspace_bytes(const srt_trie_config* cfg) {
  if (!config_ok(cfg)) return 0;
  Layout L;
  if (!make_layout(*cfg, &L)) return 0;
  return static_cast<size_t>(L.total);
}

int srt_trie_init(void* ws, size_t ws_bytes, const srt_trie_config* cfg, void* stream) {
  if (!config_ok(cfg) || !ws || (reinterpret_cast<uintptr_t>(ws) & 255)) return SRT_ERR_INVALID;
  Layout L;
  if (!make_layout(*cfg, &L)) return SRT_ERR_INVALID;
  if (ws_bytes < L.total) return SRT_ERR_CAPACITY;
  hipStream_t s = as_stream(stream);

  WsHeader h;
  std::memset(&h, 0, sizeof(h));
  h.magic = kMagic;
  h.n_prompts = cfg->n_prompts;
  h.max_streams = cfg->max_streams;
  h.max_depth = cfg->max_depth;
  h.stream_stride = L.stream_stride;
  h.slots = L.slots;
  h.node_limit = static_cast<uint64_t>(cfg->node_capacity) + cfg->n_prompts;
  h.off_roots = L.off_roots;
  h.off_streams = L.off_streams;
  h.off_keys = L.off_keys;
  h.off_count = L.off_count;
  h.off_first = L.off_first;
  h.off_next = L.off_next;
  h.total_bytes = L.total;
  h.node_capacity = cfg->node_capacity;

  char* base = static_cast<char*>(ws);
  write_header_kernel<<<1, 1, 0, s>>>(reinterpret_cast<WsHeader*>(base), h);
  const uint64_t n_stream_words = static_cast<uint64_t>(cfg->max_streams) * L.stream_stride;
  fill_u32_kernel<<<grid_for(cfg->n_prompts, 256), 256, 0, s>>>(
      reinterpret_cast<uint32_t*>(base + L.off_roots), cfg->n_prompts, kNone);
  fill_u32_kernel<<<grid_for(n_stream_words, 256), 256, 0, s>>>(
      reinterpret_cast<uint32_t*>(base + L.off_streams), n_stream_words, 0xFFFFFFFFu);
  fill_u64_kernel<<<grid_for(L.slots, 256), 256, 0, s>>>(
      reinterpret_cast<unsigned long long*>(base + L.off_keys), L.slots, kEmptyKey);
  fill_u32_kernel<<<grid_for(L.slots, 256), 256, 0, s>>>(reinterpret_cast<uint32_t*>(base + L.off_count),
                                                          L.slots, 0u);
  fill_u32_kernel<<<grid_for(L.slots, 256), 256, 0, s>>>(reinterpret_cast<uint32_t*>(base + L.off_first),
                                                          L.slots, kNone);
  fill_u32_kernel<<<grid_for(L.slots, 256), 256, 0, s>>>(reinterpret_cast<uint32_t*>(base + L.off_next),
                                                          L.slots, kNone);
  create_roots_kernel<<<grid_for(cfg->n_prompts, 256), 256, 0, s>>>(ws, cfg->n_prompts);
  return launch_status();
}

int srt_trie_insert(void* ws, int32_t n, const int32_t* prompt_ids, const int32_t* stream_ids,
                    const int32_t* tokens, const int32_t* lengths, int32_t stride, void* stream) {
  if (!ws || n < 0 || stride < 1) return SRT_ERR_INVALID;
  if (n == 0) return SRT_OK;
  if (!prompt_ids || !stream_ids || !tokens || !lengths) return SRT_ERR_INVALID;
  // one thread per substring start (up to 63 starts before the segment plus
  // one per token), so a segment of up to ~960 tokens walks its chains in
  // a single round of at most D dependent steps
  const int64_t starts = static_cast<int64_t>(stride) + 63;
  const unsigned threads = static_cast<unsigned>(std::min<int64_t>(1024, (starts + 63) / 64 * 64));
  insert_kernel<<<n, threads, 0, as_stream(stream)>>>(ws, prompt_ids, stream_ids, tokens, lengths, stride);
  return launch_status();
}

int srt_trie_reset_streams(void* ws, int32_t n, const int32_t* stream_ids, void* stream) {
  if (!ws || n < 0) return SRT_ERR_INVALID;
  if (n == 0) return SRT_OK;
  if (!stream_ids) return SRT_ERR_INVALID;
  reset_streams_kernel<<<(n + 255) / 256, 256, 0, as_stream(stream)>>>(ws, n, stream_ids);
  return launch_status();
}

int srt_trie_status(const void* ws, int64_t* info, void* stream) {
  if (!ws || !info) return SRT_ERR_INVALID;
  WsHeader h;
  const int st = read_header(ws, &h, as_stream(stream));
  if (st != SRT_OK) return st;
  info[0] = h.flags;
  info[1] = static_cast<int64_t>(h.used);
  info[2] = h.node_capacity;
  info[3] = static_cast<int64_t>(h.slots);
  return (h.flags & SRT_FLAG_CAPACITY) ? SRT_ERR_CAPACITY : SRT_OK;
}

int srt_trie_export(const void* ws, int32_t prompt_id, int64_t max_nodes, int32_t* parent, int32_t* token,
                    uint32_t* count, int64_t* n_out, void* stream) {
  if (!ws || !n_out || max_nodes < 0 || (max_nodes > 0 && (!parent || !token || !count)))
    return SRT_ERR_INVALID;
  hipStream_t s = as_stream(stream);
  WsHeader h;
  int st = read_header(ws, &h, s);
  if (st != SRT_OK) return st;
  if (prompt_id < 0 || prompt_id >= h.n_prompts) return SRT_ERR_INVALID;
  uint32_t root;
  const char* base = static_cast<const char*>(ws);
  if (hipMemcpyAsync(&root, base + h.off_roots + sizeof(uint32_t) * prompt_id, sizeof(root),
                     hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return SRT_ERR_HIP;
  if (root == kNone) return SRT_ERR_INVALID;
  void* wsm = const_cast<void*>(ws);
  export_reset_kernel<<<1, 1, 0, s>>>(wsm);
  export_level1_kernel<<<grid_for(h.slots, 256), 256, 0, s>>>(ws, root, max_nodes, parent, token, count);
  export_bfs_kernel<<<1, 1024, 0, s>>>(ws, max_nodes, parent, token, count);
  if ((st = launch_status()) != SRT_OK) return st;
  if ((st = read_header(ws, &h, s)) != SRT_OK) return st;
  const int64_t total = static_cast<int64_t>(h.export_n);
  *n_out = std::min<int64_t>(total, max_nodes);
  return total > max_nodes ? SRT_ERR_CAPACITY : SRT_OK;
}

const char* srt_version(void) { return "libsrt 0.1 (gfx950)"; }

}  // extern "C"
