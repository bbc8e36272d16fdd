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
// GPU design: one workgroup per sequence streams each visited row once with
// 16-byte loads (four in flight per thread), keeps a per-thread running
// arg-max in ascending index order, and merges lanes with wave shuffles and
// waves through LDS using (value desc, index asc).  x = fl(fl(l * inv_T) + g)
// is evaluated with explicitly rounded multiply and add (no FMA), matching
// the fp32 reference bit for bit.
#include <cfloat>

#include "common.h"

using namespace srt;

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;
constexpr int kMaxN = 256;

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

__device__ inline float score(float l, const float* g, int j, float invT) {
  return g ? __fadd_rn(__fmul_rn(l, invT), g[j]) : l;
}

template <bool kNoise>
__device__ inline Best row_argmax(const float* __restrict__ row, const float* __restrict__ noise, int V, float invT) {
  Best b{-INFINITY, 0x7FFFFFFF};
  const int tid = threadIdx.x;
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(row) & 15) == 0) &&
                   (!kNoise || (reinterpret_cast<uintptr_t>(noise) & 15) == 0);
  if (vec) {
    const f32x4* r4 = reinterpret_cast<const f32x4*>(row);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(noise);
    const int n4 = V / 4;
    int i = tid;
    for (; i + 3 * kThreads < n4; i += 4 * kThreads) {
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
        float x0 = a[u].x, x1 = a[u].y, x2 = a[u].z, x3 = a[u].w;
        if (kNoise) {
          x0 = __fadd_rn(__fmul_rn(x0, invT), g[u].x);
          x1 = __fadd_rn(__fmul_rn(x1, invT), g[u].y);
          x2 = __fadd_rn(__fmul_rn(x2, invT), g[u].z);
          x3 = __fadd_rn(__fmul_rn(x3, invT), g[u].w);
        }
        take(b, x0, j);
        take(b, x1, j + 1);
        take(b, x2, j + 2);
        take(b, x3, j + 3);
      }
    }
    for (; i < n4; i += kThreads) {
      const f32x4 a = r4[i];
      float x0 = a.x, x1 = a.y, x2 = a.z, x3 = a.w;
      if (kNoise) {
        const f32x4 g = g4[i];
        x0 = __fadd_rn(__fmul_rn(x0, invT), g.x);
        x1 = __fadd_rn(__fmul_rn(x1, invT), g.y);
        x2 = __fadd_rn(__fmul_rn(x2, invT), g.z);
        x3 = __fadd_rn(__fmul_rn(x3, invT), g.w);
      }
      take(b, x0, 4 * i);
      take(b, x1, 4 * i + 1);
      take(b, x2, 4 * i + 2);
      take(b, x3, 4 * i + 3);
    }
  } else {
    for (int j = tid; j < V; j += kThreads) take(b, score(row[j], kNoise ? noise : nullptr, j, invT), j);
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

__global__ __launch_bounds__(kThreads) void accept_kernel(int N, int V, int Dmax, const float* __restrict__ logits,
                                                          const float* __restrict__ gumbel, float invT,
                                                          const int32_t* __restrict__ tree_tokens,
                                                          const int32_t* __restrict__ tree_parent,
                                                          const int32_t* __restrict__ n_nodes,
                                                          int32_t* __restrict__ n_accepted,
                                                          int32_t* __restrict__ out_tokens,
                                                          int32_t* __restrict__ out_nodes,
                                                          int32_t* __restrict__ n_emitted) {
  __shared__ int32_t s_tok[kMaxN], s_par[kMaxN];
  __shared__ float s_v[kThreads / SRT_WAVE];
  __shared__ int s_i[kThreads / SRT_WAVE];
  __shared__ int s_child;
  const int b = blockIdx.x;
  const int n = min(max(n_nodes[b], 1), N);
  for (int i = threadIdx.x; i < n; i += kThreads) {
    s_tok[i] = tree_tokens[static_cast<int64_t>(b) * N + i];
    s_par[i] = tree_parent[static_cast<int64_t>(b) * N + i];
  }
  __syncthreads();
  int32_t* otok = out_tokens + static_cast<int64_t>(b) * (Dmax + 1);
  int32_t* onode = out_nodes + static_cast<int64_t>(b) * (Dmax + 1);

  int u = 0, k = 0;
  while (true) {
    const float* row = logits + (static_cast<int64_t>(b) * N + u) * V;
    Best best;
    if (gumbel) {
      const float* noise = gumbel + (static_cast<int64_t>(b) * (Dmax + 1) + k) * V;
      best = row_argmax<true>(row, noise, V, invT);
    } else {
      best = row_argmax<false>(row, nullptr, V, invT);
    }
    best = block_argmax(best, s_v, s_i);
    const int tok = best.i;
    if (threadIdx.x == 0) s_child = 0x7FFFFFFF;
    __syncthreads();
    for (int c = u + 1 + threadIdx.x; c < n; c += kThreads)
      if (s_par[c] == u && s_tok[c] == tok) atomicMin(&s_child, c);
    __syncthreads();
    const int child = s_child;
    if (child != 0x7FFFFFFF && k < Dmax) {
      if (threadIdx.x == 0) {
        otok[k] = tok;
        onode[k] = child;
      }
      u = child;
      ++k;
      __syncthreads();
      continue;
    }
    if (threadIdx.x == 0) {
      otok[k] = tok;
      onode[k] = -1;
      n_accepted[b] = k;
      if (n_emitted) n_emitted[b] = k + 1;
    }
    for (int r = k + 1 + threadIdx.x; r <= Dmax; r += kThreads) {
      otok[r] = -1;
      onode[r] = -1;
    }
    break;
  }
}

}  // namespace

extern "C" int srt_accept(int32_t B, int32_t N, int32_t V, int32_t Dmax, const float* logits, const float* gumbel,
                          float inv_temperature, const int32_t* tree_tokens, const int32_t* tree_parent,
                          const int32_t* n_nodes, int32_t* n_accepted, int32_t* out_tokens, int32_t* out_nodes,
                          int32_t* n_emitted, void* stream) {
  if (B < 0 || N < 1 || N > kMaxN || V < 1 || Dmax < 0 || Dmax > 63) return SRT_ERR_INVALID;
  if (!(inv_temperature == inv_temperature)) return SRT_ERR_INVALID;
  if (B == 0) return SRT_OK;
  if (!logits || !tree_tokens || !tree_parent || !n_nodes || !n_accepted || !out_tokens || !out_nodes)
    return SRT_ERR_INVALID;
  accept_kernel<<<B, kThreads, 0, as_stream(stream)>>>(N, V, Dmax, logits, gumbel, inv_temperature, tree_tokens,
                                                       tree_parent, n_nodes, n_accepted, out_tokens, out_nodes, n_emitted);
  return launch_status();
}
