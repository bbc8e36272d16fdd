// Internal helpers shared by the libsrt HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "srt.h"

#define SRT_WAVE 64

namespace srt {

// ---------------------------------------------------------------------------
// Host-side helpers
// ---------------------------------------------------------------------------
inline int hip_status(hipError_t e) { return e == hipSuccess ? SRT_OK : SRT_ERR_HIP; }

inline int launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? SRT_OK : SRT_ERR_HIP;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ---------------------------------------------------------------------------
// Per-prompt cache workspace layout (device memory, caller-owned).
//
// Nodes live in an open-addressing hash table whose slot index is the node
// id: key = (parent_id << 32) | token, roots use parent = kRootParent and
// token = prompt id.  Per slot: key (u64), count (u32), first child (u32),
// next sibling (u32).  Children of a node form a singly linked list pushed at
// creation time.
// ---------------------------------------------------------------------------
constexpr uint32_t kMagic = 0x53525431u;  // "SRT1"
constexpr uint64_t kEmptyKey = ~0ull;
constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr uint32_t kRootParent = 0xFFFFFFFFu;
constexpr uint32_t kMaxSlotsLog2 = 31;  // node ids stay below kRootParent

struct alignas(256) WsHeader {
  uint32_t magic;
  uint32_t flags;               // sticky SRT_FLAG_* bits
  int32_t n_prompts;
  int32_t max_streams;
  int32_t max_depth;            // D
  int32_t stream_stride;        // int32 words per stream record
  uint64_t slots;               // power of two
  uint64_t node_limit;          // node_capacity + n_prompts
  unsigned long long used;      // nodes created, roots included
  unsigned long long export_n;  // scratch counter of srt_trie_export
  uint64_t off_roots, off_streams, off_keys, off_count, off_first, off_next;
  uint64_t total_bytes;
  int64_t node_capacity;
};

// Stream record: [0] prompt (-1 = unbound), [1] tokens appended so far,
// [2 + j - 1] the node of the stream's suffix of length j, j = 1 ..
// min(appended, D-1) (its active nodes; kNone if the table was full).
constexpr int kStreamHead = 2;

struct TrieView {
  WsHeader* hdr;
  uint32_t* roots;
  int32_t* streams;
  unsigned long long* keys;
  uint32_t* count;
  uint32_t* first;
  uint32_t* next;
  uint64_t mask;
  int32_t depth;
};

__host__ __device__ inline TrieView trie_view(void* ws, const WsHeader& h) {
  char* base = static_cast<char*>(ws);
  TrieView v;
  v.hdr = reinterpret_cast<WsHeader*>(base);
  v.roots = reinterpret_cast<uint32_t*>(base + h.off_roots);
  v.streams = reinterpret_cast<int32_t*>(base + h.off_streams);
  v.keys = reinterpret_cast<unsigned long long*>(base + h.off_keys);
  v.count = reinterpret_cast<uint32_t*>(base + h.off_count);
  v.first = reinterpret_cast<uint32_t*>(base + h.off_first);
  v.next = reinterpret_cast<uint32_t*>(base + h.off_next);
  v.mask = h.slots - 1;
  v.depth = h.max_depth;
  return v;
}

__device__ inline TrieView trie_view_dev(const void* ws) {
  const WsHeader* h = static_cast<const WsHeader*>(ws);
  return trie_view(const_cast<void*>(ws), *h);
}

__host__ __device__ inline uint64_t node_key(uint32_t parent, uint32_t token) {
  return (static_cast<uint64_t>(parent) << 32) | static_cast<uint64_t>(token);
}

// 64-bit finaliser (MurmurHash3 fmix64).
__host__ __device__ inline uint64_t mix64(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

__device__ inline void set_flag(const TrieView& t, uint32_t f) { atomicOr(&t.hdr->flags, f); }

// Slot of (parent, token), or kNone.  Read-only probe.
__device__ inline uint32_t trie_lookup(const TrieView& t, uint32_t parent, uint32_t token) {
  const uint64_t key = node_key(parent, token);
  uint64_t h = mix64(key) & t.mask;
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    const unsigned long long k = t.keys[h];
    if (k == key) return static_cast<uint32_t>(h);
    if (k == kEmptyKey) return kNone;
    h = (h + 1) & t.mask;
  }
  return kNone;
}

// Slot of (parent, token), creating the node (count 0) if absent.  A newly
// created child is pushed onto its parent's child list.  Returns kNone and
// raises the capacity flag if the table is full.
__device__ inline uint32_t trie_get_or_create(const TrieView& t, uint32_t parent, uint32_t token) {
  const uint64_t key = node_key(parent, token);
  uint64_t h = mix64(key) & t.mask;
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    unsigned long long k = t.keys[h];
    if (k == key) return static_cast<uint32_t>(h);
    if (k == kEmptyKey) {
      const unsigned long long old = atomicCAS(&t.keys[h], kEmptyKey, (unsigned long long)key);
      if (old == kEmptyKey) {
        const unsigned long long n = atomicAdd(&t.hdr->used, 1ull);
        if (n + 1 > t.hdr->node_limit) set_flag(t, SRT_FLAG_CAPACITY);
        if (parent != kRootParent) t.next[h] = atomicExch(&t.first[parent], static_cast<uint32_t>(h));
        return static_cast<uint32_t>(h);
      }
      if (old == key) return static_cast<uint32_t>(h);
    }
    h = (h + 1) & t.mask;
  }
  set_flag(t, SRT_FLAG_CAPACITY);
  return kNone;
}

// ---------------------------------------------------------------------------
// Wave helpers
// ---------------------------------------------------------------------------
__device__ inline int lane_id() { return __lane_id(); }

template <typename T>
__device__ inline T shfl_xor(T v, int m) {
  return __shfl_xor(v, m, SRT_WAVE);
}

__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, SRT_WAVE);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, SRT_WAVE);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ inline uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl(static_cast<uint32_t>(v), src, SRT_WAVE);
  const uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), src, SRT_WAVE);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

}  // namespace srt
