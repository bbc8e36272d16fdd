// Acceptance walk over the draft tree.
//
// Method: Sections 1 and 3 of the paper -- the policy verifies the drafted
// tokens and accepts them up to the first mismatch, emitting its own token
// there, which keeps its sampling distribution exactly.  At each step the
// policy's choice is the arg-max of the node's logits (greedy) or of
// logits * inv_T + Gumbel noise (sampling by the Gumbel-max trick, one noise
// row per step); if a child of the current node carries that token the walk
// descends.
//
// GPU design: the batch walks one step (= tree depth) at a time, and each
// step is spread over the whole GPU.
//   * A level kernel splits the visited row of every sequence still walking
//     (and its noise row) into up to 32 chunks, one workgroup per chunk, so
//     that late steps, when few long walks remain, still read their rows
//     with many compute units.  Each workgroup streams its chunk with
//     16-byte loads, keeps a per-thread running arg-max in ascending index
//     order, merges lanes with wave shuffles and waves through LDS, and
//     stores one packed 64-bit (score, token) candidate: order-preserving
//     score bits above the complement of the token, so the largest key is
//     the arg-max with the lowest index (+0 and -0 compare equal, as fp32
//     comparisons do).  Blocks map onto the rows that exist at the level,
//     working blocks first in dispatch order.
//   * The step's decision is folded into the next level's kernel: every
//     block of a walker first takes the largest candidate of the walker's
//     previous row, looks for the child that carries the token (all blocks
//     of the walker reach the same answer; the node count and the tree
//     row load together with the candidates), and one of them writes the
//     step's output and, if it descends, appends the sequence to the next
//     level's list; then each block reads its chunk of the child's row.  A
//     last walk kernel decides the final level, and the level-0 kernel
//     resets the walk's state (no separate launch).  Candidates and current
//     nodes alternate between two buffers by level parity, so no launch
//     reads a buffer it writes.
// x = fl(fl(l * inv_T) + g) is evaluated with explicitly rounded multiply
// and add (no FMA), matching the fp32 reference bit for bit.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <mutex>

#include "common.h"

using namespace srt;

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kMaxN = 256;
constexpr int kMaxLevels = 64;   // Dmax + 1 <= 64
constexpr int kMaxChunks = 32;   // chunks per visited row, at most
constexpr int kMinChunk = 4096;  // vocabulary entries per chunk, at least
constexpr int kWalkWaves = 4;

struct AcceptArgs {
  const float* logits;
  const float* gumbel;
  const int32_t* tree_tokens;
  const int32_t* tree_parent;
  const int32_t* n_nodes;
  int32_t* n_accepted;
  int32_t* out_tokens;
  int32_t* out_nodes;
  int32_t* n_emitted;
  int32_t* n_act;            // [kMaxLevels + 1] sequences walking at each level
  int32_t* act;              // [2, B] those sequences, by level parity
  int32_t* cur;              // [2, B] node each sequence stands on, by level parity
  unsigned long long* cand;  // [2, B, kMaxChunks] packed candidates of a level, by parity
  int B, N, V, Dmax, chunk, n_chunks;
  int vec;                   // rows can be read as float4
  float invT;
};

// Scratch layout: level counters, two walker lists, current nodes, candidates.
struct ScratchLayout {
  size_t off_act, off_cur, off_cand, total;
};

constexpr size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

constexpr ScratchLayout scratch_layout(int64_t B) {
  ScratchLayout s{};
  s.off_act = round256(sizeof(int32_t) * (kMaxLevels + 1));
  s.off_cur = s.off_act + round256(sizeof(int32_t) * 2 * static_cast<size_t>(B));
  s.off_cand = s.off_cur + round256(sizeof(int32_t) * 2 * static_cast<size_t>(B));
  s.total = s.off_cand + round256(sizeof(unsigned long long) * 2 * static_cast<size_t>(B) * kMaxChunks);
  return s;
}

__device__ inline unsigned long long pack_key(float x, int tok) {
  uint32_t u = __float_as_uint(x == 0.f ? 0.f : x);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<unsigned long long>(u) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(tok));
}

__device__ inline int key_token(unsigned long long k) {
  return static_cast<int>(~static_cast<uint32_t>(k & 0xFFFFFFFFull));
}

struct Best {
  float v;
  int i;
};

__device__ inline void take(Best& b, float v, int i) {
  if (v > b.v || (v == b.v && i < b.i)) {
    b.v = v;
    b.i = i;
  }
}

__device__ inline float score(float l, float g, float invT, bool noisy) {
  return noisy ? __fadd_rn(__fmul_rn(l, invT), g) : l;
}

// Arg-max of x_j over j in [lo, hi) of one row, in every thread.
template <bool kNoise>
__device__ inline Best chunk_argmax(const AcceptArgs& a, const float* __restrict__ row,
                                    const float* __restrict__ noise, int lo, int hi) {
  Best b{-INFINITY, 0x7FFFFFFF};
  const int tid = threadIdx.x;
  if (a.vec) {  // lo, hi multiples of 4 and rows 16-byte aligned
    const f32x4* r4 = reinterpret_cast<const f32x4*>(row);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(noise);
    const int e4 = hi / 4;
    int i = lo / 4 + tid;
    for (; i + 3 * kThreads < e4; i += 4 * kThreads) {
      f32x4 x[4], g[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = __builtin_nontemporal_load(&r4[i + u * kThreads]);
      if (kNoise) {
#pragma unroll
        for (int u = 0; u < 4; ++u) g[u] = __builtin_nontemporal_load(&g4[i + u * kThreads]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = 4 * (i + u * kThreads);
        take(b, score(x[u].x, kNoise ? g[u].x : 0.f, a.invT, kNoise), j);
        take(b, score(x[u].y, kNoise ? g[u].y : 0.f, a.invT, kNoise), j + 1);
        take(b, score(x[u].z, kNoise ? g[u].z : 0.f, a.invT, kNoise), j + 2);
        take(b, score(x[u].w, kNoise ? g[u].w : 0.f, a.invT, kNoise), j + 3);
      }
    }
    for (; i < e4; i += kThreads) {
      const f32x4 x = r4[i];
      f32x4 g = {0.f, 0.f, 0.f, 0.f};
      if (kNoise) g = g4[i];
      take(b, score(x.x, g.x, a.invT, kNoise), 4 * i);
      take(b, score(x.y, g.y, a.invT, kNoise), 4 * i + 1);
      take(b, score(x.z, g.z, a.invT, kNoise), 4 * i + 2);
      take(b, score(x.w, g.w, a.invT, kNoise), 4 * i + 3);
    }
  } else {
    int j = lo + tid;
    for (; j + 7 * kThreads < hi; j += 8 * kThreads) {
      float x[8], g[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = __builtin_nontemporal_load(&row[j + u * kThreads]);
      if (kNoise) {
#pragma unroll
        for (int u = 0; u < 8; ++u) g[u] = __builtin_nontemporal_load(&noise[j + u * kThreads]);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) take(b, score(x[u], kNoise ? g[u] : 0.f, a.invT, kNoise), j + u * kThreads);
    }
    for (; j < hi; j += kThreads) take(b, score(row[j], kNoise ? noise[j] : 0.f, a.invT, kNoise), j);
  }
  // lanes, then waves through LDS
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(b.v, off, SRT_WAVE);
    const int oi = __shfl_xor(b.i, off, SRT_WAVE);
    take(b, ov, oi);
  }
  __shared__ float s_v[kThreads / SRT_WAVE];
  __shared__ int s_i[kThreads / SRT_WAVE];
  if (tid % SRT_WAVE == 0) {
    s_v[tid / SRT_WAVE] = b.v;
    s_i[tid / SRT_WAVE] = b.i;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kThreads / SRT_WAVE; ++w) take(b, s_v[w], s_i[w]);
  return b;
}

// The decision of step `level` for sequence b standing on node u, from the
// candidates of its row, in one wave: the token, and the child that carries
// it (-1 if none or if the walk is at its depth cap).
struct Step {
  int tok, child;
};

__device__ inline Step decide(const AcceptArgs& a, int b, int u, int level, int lane) {
  const unsigned long long* cand = a.cand + (static_cast<int64_t>(level & 1) * a.B + b) * kMaxChunks;
  const int64_t tr = static_cast<int64_t>(b) * a.N;
  // the node count and the tree row's first 64 nodes load together with the
  // candidates (their addresses do not depend on the step's token)
  const int n = min(max(a.n_nodes[b], 1), a.N);
  const int32_t par0 = lane < a.N ? a.tree_parent[tr + lane] : -1;
  const int32_t tok0 = lane < a.N ? a.tree_tokens[tr + lane] : -1;
  unsigned long long best = lane < a.n_chunks ? cand[lane] : 0ull;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const unsigned long long o = shfl_xor_u64(best, off);
    best = o > best ? o : best;
  }
  Step st{key_token(best), -1};
  if (level < a.Dmax) {  // children of u have larger indices
    unsigned long long m = __ballot(lane > u && lane < n && par0 == u && tok0 == st.tok);
    if (m) st.child = __ffsll(static_cast<long long>(m)) - 1;
    for (int c0 = SRT_WAVE; c0 < n && st.child < 0; c0 += SRT_WAVE) {
      const int cc = c0 + lane;
      const bool hit = cc > u && cc < n && a.tree_parent[tr + cc] == u && a.tree_tokens[tr + cc] == st.tok;
      m = __ballot(hit);
      if (m) st.child = c0 + __ffsll(static_cast<long long>(m)) - 1;
    }
  }
  return st;
}

// Records step `level` of sequence b (one thread): the token, then descend
// (next node, next level's list) or stop.
__device__ inline void record(const AcceptArgs& a, int b, int level, const Step& st) {
  const int64_t orow = static_cast<int64_t>(b) * (a.Dmax + 1);
  a.out_tokens[orow + level] = st.tok;
  if (st.child >= 0) {
    a.out_nodes[orow + level] = st.child;
    a.cur[((level + 1) & 1) * a.B + b] = st.child;
    const int pos = atomicAdd(&a.n_act[level + 1], 1);
    a.act[((level + 1) & 1) * a.B + pos] = b;
  } else {
    a.n_accepted[b] = level;
    if (a.n_emitted) a.n_emitted[b] = level + 1;
  }
}

// One chunk of the visited row of one walker at this level.  For level > 0
// the walker is one of those of the previous level, and the block first
// takes that level's step (block 0 of the walker records it).
template <bool kNoise>
__global__ __launch_bounds__(kThreads) void accept_level_kernel(AcceptArgs a, int level) {
  const int g = blockIdx.x;
  const int slot = g / a.n_chunks, c = g - slot * a.n_chunks;
  const int lv = level > 0 ? level - 1 : 0;  // the list the walker comes from
  int b, u;
  if (level == 0) {  // every sequence; the walk's state is reset here
    if (slot >= a.B) return;
    b = slot;
    u = 0;
    if (g == 0 && threadIdx.x <= kMaxLevels) a.n_act[threadIdx.x] = threadIdx.x == 0 ? a.B : 0;
    if (c == 0) {
      const int64_t orow = static_cast<int64_t>(b) * (a.Dmax + 1);
      for (int k = threadIdx.x; k <= a.Dmax; k += kThreads) {
        a.out_tokens[orow + k] = -1;
        a.out_nodes[orow + k] = -1;
      }
      if (threadIdx.x == 0) {
        a.act[b] = b;  // level 0, parity 0
        a.cur[b] = 0;
      }
    }
  } else {
    if (slot >= a.n_act[lv]) return;
    b = min(max(a.act[(lv & 1) * a.B + slot], 0), a.B - 1);
    __shared__ int s_child;
    if (threadIdx.x < SRT_WAVE) {
      const int prev = min(max(a.cur[(lv & 1) * a.B + b], 0), a.N - 1);
      const Step st = decide(a, b, prev, lv, threadIdx.x);
      if (threadIdx.x == 0) {
        if (c == 0) record(a, b, lv, st);
        s_child = st.child;
      }
    }
    __syncthreads();
    u = s_child;
    if (u < 0) return;
  }
  const float* row = a.logits + (static_cast<int64_t>(b) * a.N + u) * a.V;
  const float* noise = kNoise ? a.gumbel + (static_cast<int64_t>(b) * (a.Dmax + 1) + level) * a.V : nullptr;
  const int lo = c * a.chunk, hi = min(a.V, lo + a.chunk);
  const Best best = chunk_argmax<kNoise>(a, row, noise, lo, hi);
  if (threadIdx.x == 0)
    a.cand[(static_cast<int64_t>(level & 1) * a.B + b) * kMaxChunks + c] = pack_key(best.v, best.i);
}

// The step of the last level (Dmax), one wave per walker.
__global__ __launch_bounds__(kWalkWaves * SRT_WAVE) void accept_walk_kernel(AcceptArgs a, int level) {
  const int lane = threadIdx.x % SRT_WAVE;
  const int slot = blockIdx.x * kWalkWaves + threadIdx.x / SRT_WAVE;
  if (slot >= a.n_act[level]) return;
  const int b = min(max(a.act[(level & 1) * a.B + slot], 0), a.B - 1);
  const int u = min(max(a.cur[(level & 1) * a.B + b], 0), a.N - 1);
  const Step st = decide(a, b, u, level, lane);
  if (lane == 0) record(a, b, level, st);
}

// Host checks shared by both entry points (before any scratch is touched).
int check_args(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits, float inv_temperature,
               const int32_t* tree_tokens, const int32_t* tree_parent, const int32_t* n_nodes,
               const int32_t* n_accepted, const int32_t* out_tokens, const int32_t* out_nodes) {
  if (B < 0 || N < 1 || N > kMaxN || V < 1 || Dmax < 0 || Dmax >= kMaxLevels) return SRT_ERR_INVALID;
  if (!(inv_temperature == inv_temperature)) return SRT_ERR_INVALID;
  if (B == 0) return SRT_OK;
  if (!logits || !tree_tokens || !tree_parent || !n_nodes || !n_accepted || !out_tokens || !out_nodes)
    return SRT_ERR_INVALID;
  return SRT_OK;
}

// The walk itself on scratch memory `base` (device, 256-byte aligned, at
// least scratch_layout(B).total bytes); the level-0 kernel resets the level
// counters, so the scratch contents on entry do not matter.
int launch_accept(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits, const float* gumbel,
                  float inv_temperature, const int32_t* tree_tokens, const int32_t* tree_parent,
                  const int32_t* n_nodes, int32_t* n_accepted, int32_t* out_tokens, int32_t* out_nodes,
                  int32_t* n_emitted, char* base, void* stream) {
  const ScratchLayout L = scratch_layout(B);
  AcceptArgs a;
  a.logits = logits;
  a.gumbel = gumbel;
  a.tree_tokens = tree_tokens;
  a.tree_parent = tree_parent;
  a.n_nodes = n_nodes;
  a.n_accepted = n_accepted;
  a.out_tokens = out_tokens;
  a.out_nodes = out_nodes;
  a.n_emitted = n_emitted;
  a.n_act = reinterpret_cast<int32_t*>(base);
  a.act = reinterpret_cast<int32_t*>(base + L.off_act);
  a.cur = reinterpret_cast<int32_t*>(base + L.off_cur);
  a.cand = reinterpret_cast<unsigned long long*>(base + L.off_cand);
  a.B = B;
  a.N = N;
  a.V = V;
  a.Dmax = Dmax;
  // chunk: a multiple of 4 of at least kMinChunk entries, at most kMaxChunks per row
  const int64_t per = (static_cast<int64_t>(V) + kMaxChunks - 1) / kMaxChunks;
  a.chunk = static_cast<int>(std::max<int64_t>(kMinChunk, (per + 3) / 4 * 4));
  a.n_chunks = static_cast<int>((static_cast<int64_t>(V) + a.chunk - 1) / a.chunk);
  a.vec = V % 4 == 0 && (reinterpret_cast<uintptr_t>(logits) & 15) == 0 &&
          (!gumbel || (reinterpret_cast<uintptr_t>(gumbel) & 15) == 0);
  a.invT = inv_temperature;
  const int64_t grid = static_cast<int64_t>(B) * a.n_chunks;
  if (grid > 0x7FFFFFFF) return SRT_ERR_UNSUPPORTED;

  hipStream_t s = as_stream(stream);
  int st = SRT_OK;
  const unsigned walk_grid = static_cast<unsigned>((B + kWalkWaves - 1) / kWalkWaves);
  for (int level = 0; level <= Dmax && st == SRT_OK; ++level) {
    if (gumbel)
      accept_level_kernel<true><<<static_cast<unsigned>(grid), kThreads, 0, s>>>(a, level);
    else
      accept_level_kernel<false><<<static_cast<unsigned>(grid), kThreads, 0, s>>>(a, level);
    st = launch_status();
  }
  if (st == SRT_OK) {
    accept_walk_kernel<<<walk_grid, kWalkWaves * SRT_WAVE, 0, s>>>(a, Dmax);
    st = launch_status();
  }
  return st;
}

// Scratch of srt_accept_noalloc: one fixed array per device, sized for
// kNoAllocMaxB sequences, whose device address is looked up once per device
// (hipGetSymbolAddress) and kept; host code never uses the array's name as
// an address.
constexpr int32_t kNoAllocMaxB = SRT_ACCEPT_NOALLOC_MAX_BATCH;
constexpr int kMaxDevices = 64;
std::mutex g_noalloc_mu;
char* g_noalloc_ptr[kMaxDevices] = {};

constexpr size_t kNoAllocBytes = scratch_layout(kNoAllocMaxB).total;  // 2,163,200 bytes

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace {

// Device address of this device's fixed scratch array (nullptr on error).
char* noalloc_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (!g_noalloc_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_noalloc_ptr[dev] = static_cast<char*>(ptr);
  }
  return g_noalloc_ptr[dev];
}

}  // namespace

extern "C" size_t srt_accept_scratch_bytes(int32_t B) {
  if (B < 0) return 0;
  return scratch_layout(std::max(B, 1)).total;
}

extern "C" int srt_accept(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits, const float* gumbel,
                          float inv_temperature, const int32_t* tree_tokens, const int32_t* tree_parent,
                          const int32_t* n_nodes, int32_t* n_accepted, int32_t* out_tokens, int32_t* out_nodes,
                          int32_t* n_emitted, void* scratch_buf, size_t scratch_bytes, void* stream) {
  int st = check_args(B, N, V, Dmax, logits, inv_temperature, tree_tokens, tree_parent, n_nodes, n_accepted,
                      out_tokens, out_nodes);
  if (st != SRT_OK || B == 0) return st;
  if (!scratch_buf || scratch_bytes < srt_accept_scratch_bytes(B)) return SRT_ERR_CAPACITY;
  if (reinterpret_cast<uintptr_t>(scratch_buf) % 256) return SRT_ERR_INVALID;
  return launch_accept(B, N, V, Dmax, logits, gumbel, inv_temperature, tree_tokens, tree_parent, n_nodes,
                       n_accepted, out_tokens, out_nodes, n_emitted, static_cast<char*>(scratch_buf), stream);
}

extern "C" int srt_accept_noalloc(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits,
                                  const float* gumbel, float inv_temperature, const int32_t* tree_tokens,
                                  const int32_t* tree_parent, const int32_t* n_nodes, int32_t* n_accepted,
                                  int32_t* out_tokens, int32_t* out_nodes, int32_t* n_emitted, void* stream) {
  int st = check_args(B, N, V, Dmax, logits, inv_temperature, tree_tokens, tree_parent, n_nodes, n_accepted,
                      out_tokens, out_nodes);
  if (st != SRT_OK || B == 0) return st;
  if (B > kNoAllocMaxB) return SRT_ERR_CAPACITY;
  char* base = noalloc_scratch();
  if (!base) return SRT_ERR_HIP;
  return launch_accept(B, N, V, Dmax, logits, gumbel, inv_temperature, tree_tokens, tree_parent, n_nodes,
                       n_accepted, out_tokens, out_nodes, n_emitted, base, stream);
}
