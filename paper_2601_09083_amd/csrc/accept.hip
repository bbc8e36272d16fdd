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
// GPU design: W cooperating workgroups per sequence.  At each step every
// member streams its contiguous slice of the visited row (and of the noise
// row) with 16-byte loads, four in flight per thread, keeps a per-thread
// running arg-max in ascending index order and merges lanes with wave
// shuffles and waves through LDS using (value desc, index asc).  It then
// publishes the slice's (value, index) in the sequence's slot of the
// caller's scratch as one tagged 64-bit word; once the words of all W
// members carry the step's tag, each member reduces them in the same order,
// so all take the same decision, find the child in the tree (kept in LDS)
// and move on together.  The words are the only shared data and are read
// and written whole by relaxed device-scope atomics, so the step barrier
// costs no cache flushes.  The walk is a serial chain of rows, so spreading each
// row over W compute units shortens it W-fold when few sequences are still
// walking.  W is chosen from the device's occupancy so that all B * W
// workgroups are resident at once and the launch is cooperative, which
// guarantees it; with W = 1 no member waits for another.  Every wait is
// bounded.  x = fl(fl(l * inv_T) + g) is evaluated with explicitly rounded
// multiply and add (no FMA), matching the fp32 reference bit for bit.
#include <algorithm>
#include <cfloat>

#include "common.h"

using namespace srt;

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kMaxN = 256;
constexpr int kMaxW = 32;                   // workgroups per sequence
constexpr int kMinSlice = 4096;             // vocabulary entries per member, at least
constexpr unsigned kSpinLimit = 1u << 22;   // bounded wait at a step barrier
constexpr int kMaxIndex = (1 << 25) - 1;    // vocabulary indices in a slot word

// Per-sequence slots in the scratch buffer: member m's result of step k is
// one 64-bit word in slot[k % 2][m] = (value bits << 32) | (index << 7) |
// tag, tag = k + 1 (1..64; 0 = empty).  A reader accepts a word only with
// the tag of the step it waits for, so the words need no fences: each is
// written and read whole by relaxed device-scope atomics, and a member
// cannot reach step k + 2 (reusing the slot) before every member has
// published step k + 1, which it does after reading step k.
struct alignas(256) SeqSync {
  unsigned long long slot[2][kMaxW];
};

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
  SeqSync* sync;
  int N, V, Dmax, W;
  float invT;
};

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

// Arg-max of x_j over j in [lo, hi) of one row.
template <bool kNoise>
__device__ inline Best slice_argmax(const float* __restrict__ row, const float* __restrict__ noise, int lo, int hi,
                                    float invT) {
  Best b{-INFINITY, 0x7FFFFFFF};
  const int tid = threadIdx.x;
  const bool vec = (lo % 4 == 0) && (hi % 4 == 0) && ((reinterpret_cast<uintptr_t>(row) & 15) == 0) &&
                   (!kNoise || (reinterpret_cast<uintptr_t>(noise) & 15) == 0);
  if (vec) {
    const f32x4* r4 = reinterpret_cast<const f32x4*>(row);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(noise);
    const int e4 = hi / 4;
    int i = lo / 4 + tid;
    for (; i + 3 * kThreads < e4; i += 4 * kThreads) {
      f32x4 a[4], g[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] = __builtin_nontemporal_load(&r4[i + u * kThreads]);
      if (kNoise) {
#pragma unroll
        for (int u = 0; u < 4; ++u) g[u] = __builtin_nontemporal_load(&g4[i + u * kThreads]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = 4 * (i + u * kThreads);
        take(b, score(a[u].x, kNoise ? g[u].x : 0.f, invT, kNoise), j);
        take(b, score(a[u].y, kNoise ? g[u].y : 0.f, invT, kNoise), j + 1);
        take(b, score(a[u].z, kNoise ? g[u].z : 0.f, invT, kNoise), j + 2);
        take(b, score(a[u].w, kNoise ? g[u].w : 0.f, invT, kNoise), j + 3);
      }
    }
    for (; i < e4; i += kThreads) {
      const f32x4 a = r4[i];
      f32x4 g = {0.f, 0.f, 0.f, 0.f};
      if (kNoise) g = g4[i];
      take(b, score(a.x, g.x, invT, kNoise), 4 * i);
      take(b, score(a.y, g.y, invT, kNoise), 4 * i + 1);
      take(b, score(a.z, g.z, invT, kNoise), 4 * i + 2);
      take(b, score(a.w, g.w, invT, kNoise), 4 * i + 3);
    }
  } else {
    for (int j = lo + tid; j < hi; j += kThreads) take(b, score(row[j], kNoise ? noise[j] : 0.f, invT, kNoise), j);
  }
  return b;
}

__device__ inline Best block_argmax(Best b, float* s_v, int* s_i) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(b.v, off, SRT_WAVE);
    const int oi = __shfl_xor(b.i, off, SRT_WAVE);
    take(b, ov, oi);
  }
  const int w = threadIdx.x / SRT_WAVE;
  if ((threadIdx.x & (SRT_WAVE - 1)) == 0) {
    s_v[w] = b.v;
    s_i[w] = b.i;
  }
  __syncthreads();
  Best r{s_v[0], s_i[0]};
  for (int k = 1; k < kThreads / SRT_WAVE; ++k) take(r, s_v[k], s_i[k]);
  __syncthreads();
  return r;
}

// Empties every slot (tag 0) before a call.
__global__ void accept_reset_kernel(SeqSync* sync, int B) {
  static_assert(sizeof(SeqSync) == 2 * kMaxW * sizeof(unsigned long long), "slots only");
  const int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (i < static_cast<int64_t>(B) * 2 * kMaxW) reinterpret_cast<unsigned long long*>(sync)[i] = 0ull;
}

__global__ __launch_bounds__(kThreads) void accept_kernel(AcceptArgs a) {
  __shared__ int32_t s_tok[kMaxN], s_par[kMaxN];
  __shared__ float s_v[kThreads / SRT_WAVE];
  __shared__ int s_i[kThreads / SRT_WAVE];
  __shared__ int s_child, s_tokc, s_failed;
  const int W = a.W;
  const int b = blockIdx.x / W;
  const int wi = blockIdx.x % W;
  const int N = a.N, V = a.V, Dmax = a.Dmax;
  const int n = min(max(a.n_nodes[b], 1), N);
  for (int i = threadIdx.x; i < n; i += kThreads) {
    s_tok[i] = a.tree_tokens[static_cast<int64_t>(b) * N + i];
    s_par[i] = a.tree_parent[static_cast<int64_t>(b) * N + i];
  }
  if (threadIdx.x == 0) s_failed = 0;
  __syncthreads();
  int32_t* otok = a.out_tokens + static_cast<int64_t>(b) * (Dmax + 1);
  int32_t* onode = a.out_nodes + static_cast<int64_t>(b) * (Dmax + 1);
  SeqSync* sy = a.sync + b;
  // this member's slice of the vocabulary (a multiple of 4 entries)
  const int chunk = ((V + W - 1) / W + 3) / 4 * 4;
  const int lo = min(V, wi * chunk), hi = min(V, lo + chunk);

  int u = 0, k = 0;
  while (true) {
    const float* row = a.logits + (static_cast<int64_t>(b) * N + u) * V;
    Best best;
    if (a.gumbel) {
      const float* noise = a.gumbel + (static_cast<int64_t>(b) * (Dmax + 1) + k) * V;
      best = slice_argmax<true>(row, noise, lo, hi, a.invT);
    } else {
      best = slice_argmax<false>(row, nullptr, lo, hi, a.invT);
    }
    best = block_argmax(best, s_v, s_i);
    if (W == 1) {
      if (threadIdx.x == 0) s_tokc = best.i;
    } else if (threadIdx.x < SRT_WAVE) {
      // publish this slice's result, then wave 0 polls the W words of the
      // step (one lane per member) until all carry the step's tag
      const int par = k & 1;
      const unsigned long long tag = static_cast<unsigned long long>(k + 1);
      if (threadIdx.x == 0) {
        const unsigned long long word = (static_cast<unsigned long long>(__float_as_uint(best.v)) << 32) |
                                        (static_cast<unsigned long long>(min(best.i, kMaxIndex)) << 7) | tag;
        __hip_atomic_store(&sy->slot[par][wi], word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      const int lane = threadIdx.x;
      unsigned long long w = 0;
      bool ready = lane >= W;
      for (unsigned spins = 0;; ++spins) {
        if (!ready) {
          w = __hip_atomic_load(&sy->slot[par][lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ready = (w & 127ull) == tag;
        }
        if (__all(ready)) break;
        if (spins >= kSpinLimit) {
          if (lane == 0) s_failed = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      Best r{-INFINITY, 0x7FFFFFFF};
      if (lane < W) r = Best{__uint_as_float(static_cast<unsigned>(w >> 32)), static_cast<int>((w & 0xFFFFFFFFull) >> 7)};
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const float ov = __shfl_xor(r.v, off, SRT_WAVE);
        const int oi = __shfl_xor(r.i, off, SRT_WAVE);
        take(r, ov, oi);
      }
      if (lane == 0) s_tokc = r.i;
    }
    if (threadIdx.x == 0) s_child = 0x7FFFFFFF;
    __syncthreads();
    const int tok = s_tokc;
    if (s_failed) {  // a member never arrived (cannot happen with all members resident)
      if (wi == 0 && threadIdx.x == 0) {
        a.n_accepted[b] = -1;
        if (a.n_emitted) a.n_emitted[b] = 0;
      }
      break;
    }
    for (int c = u + 1 + threadIdx.x; c < n; c += kThreads)
      if (s_par[c] == u && s_tok[c] == tok) atomicMin(&s_child, c);
    __syncthreads();
    const int child = s_child;
    if (child != 0x7FFFFFFF && k < Dmax) {
      if (wi == 0 && threadIdx.x == 0) {
        otok[k] = tok;
        onode[k] = child;
      }
      u = child;
      ++k;
      __syncthreads();
      continue;
    }
    if (wi == 0) {
      if (threadIdx.x == 0) {
        otok[k] = tok;
        onode[k] = -1;
        a.n_accepted[b] = k;
        if (a.n_emitted) a.n_emitted[b] = k + 1;
      }
      for (int r = k + 1 + threadIdx.x; r <= Dmax; r += kThreads) {
        otok[r] = -1;
        onode[r] = -1;
      }
    }
    break;
  }
}

int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  if (dev < 64 && cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
  if (dev < 64) cached[dev] = n;
  return n;
}

// Workgroups the device holds at once for accept_kernel.
int64_t resident_groups() {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(accept_kernel), kThreads,
                                                   0) != hipSuccess)
    return 0;
  return static_cast<int64_t>(per_cu) * cu_count();
}

}  // namespace

extern "C" size_t srt_accept_scratch_bytes(int32_t B) {
  if (B < 0) return 0;
  return static_cast<size_t>(std::max(B, 1)) * sizeof(SeqSync);
}

extern "C" int srt_accept(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits, const float* gumbel,
                          float inv_temperature, const int32_t* tree_tokens, const int32_t* tree_parent,
                          const int32_t* n_nodes, int32_t* n_accepted, int32_t* out_tokens, int32_t* out_nodes,
                          int32_t* n_emitted, void* scratch, size_t scratch_bytes, void* stream) {
  if (B < 0 || N < 1 || N > kMaxN || V < 1 || Dmax < 0 || Dmax > 63) return SRT_ERR_INVALID;
  if (!(inv_temperature == inv_temperature)) return SRT_ERR_INVALID;
  if (B == 0) return SRT_OK;
  if (!logits || !tree_tokens || !tree_parent || !n_nodes || !n_accepted || !out_tokens || !out_nodes)
    return SRT_ERR_INVALID;
  if (!scratch || scratch_bytes < srt_accept_scratch_bytes(B)) return SRT_ERR_CAPACITY;
  if (reinterpret_cast<uintptr_t>(scratch) % 256) return SRT_ERR_INVALID;
  const int64_t resident = resident_groups();
  if (resident <= 0) return SRT_ERR_HIP;
  int W = static_cast<int>(std::min<int64_t>({resident / B, static_cast<int64_t>(kMaxW),
                                               static_cast<int64_t>((V + kMinSlice - 1) / kMinSlice)}));
  if (W < 1 || V > kMaxIndex) W = 1;
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
  a.sync = static_cast<SeqSync*>(scratch);
  a.N = N;
  a.V = V;
  a.Dmax = Dmax;
  a.W = W;
  a.invT = inv_temperature;
  hipStream_t s = as_stream(stream);
  if (W == 1) {  // no member waits for another: an ordinary launch
    accept_kernel<<<B, kThreads, 0, s>>>(a);
    return launch_status();
  }
  accept_reset_kernel<<<static_cast<unsigned>((static_cast<int64_t>(B) * 2 * kMaxW + 255) / 256), 256, 0, s>>>(a.sync, B);
  if (launch_status() != SRT_OK) return SRT_ERR_HIP;
  void* params[] = {&a};
  // all B * W members must be resident at once: a cooperative launch
  // guarantees it (and fails instead of launching otherwise)
  const hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(accept_kernel),
                                                  dim3(static_cast<unsigned>(B) * W), dim3(kThreads), params, 0, s);
  return e == hipSuccess ? SRT_OK : SRT_ERR_HIP;
}
