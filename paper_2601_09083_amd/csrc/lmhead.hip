// Acceptance walk with the LM head applied at the visited nodes only
// (MFMA, gfx950).
//
// Method: the lossless acceptance walk of Sections 1 and 3 (descend while
// the policy's own next token -- greedy arg-max, or Gumbel-max for sampling
// at temperature T -- is a child's token, then emit it as the bonus token),
// where the policy's logits at tree node u are its LM head applied to the
// node's final hidden state, logit_j = <hidden[b,u], w_head[j]>.  The walk
// needs the arg-max at the nodes it visits and nothing else, so the
// [B, N, V] logits tensor and the head's products for unvisited nodes are
// never formed.
//
// GPU design.  The walk advances one depth level at a time for the whole
// batch; at level l every sequence still walking sits at one node of depth
// l.  Per level:
//   * a GEMM kernel multiplies the walking sequences' hidden rows (gathered
//     by node index) with the whole head, C^T = W H^T on
//     v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  A workgroup of 4
//     waves owns 128 head rows (32 per wave) and a block of 64 walking
//     sequences.  Each head row is used by one wave only, so the head is
//     read from HBM straight into the MFMA operand registers, four 64-wide
//     chunks of d_model ahead of the MFMAs (16 KB in flight per wave); the
//     hidden rows are shared by the 4 waves and staged through
//     double-buffered, padded LDS.  A sequence lives in one lane column, so
//     its scores (plus the level's Gumbel row) reduce to a (value, token)
//     candidate inside the lane, then across the two lane halves and the
//     four waves; one packed 64-bit candidate per (sequence, tile) goes to
//     scratch with a plain store.  Blocks whose sequence block has no
//     walkers exit at once;
//   * a walk kernel (one workgroup per walking sequence) takes the maximum
//     candidate over the tiles, looks for the child carrying that token,
//     writes the step's outputs and, if it descends, appends the sequence to
//     the next level's list.
// A level is bound by streaming the head (V x d_model bf16) from HBM; the
// blocks of one head tile and different sequence blocks are placed on one
// XCD back to back, so the head rows they share come from its L2.
#include <algorithm>
#include <cmath>

#include "common.h"


using namespace srt;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kTV = 32 * kWaves;         // vocabulary rows per workgroup (32 per wave)
constexpr int kKC = 64;                  // d_model elements per chunk
constexpr int kInFlight = 4;             // head chunks each wave keeps in flight
constexpr int kRowBytes = kKC * 2 + 16;  // padded LDS row (conflict-free fragment reads)
constexpr int kThreads = kWaves * SRT_WAVE;
constexpr int kMaxLevels = 64;           // Dmax + 1 <= 64
constexpr int kXcds = 8;
constexpr int kWalkThreads = 256;
#ifndef SRT_HEAD_FINISH_ROWS
#define SRT_HEAD_FINISH_ROWS 128
#endif
constexpr int kFinishRows = SRT_HEAD_FINISH_ROWS;  // rows of a finishing pass

struct HeadArgs {
  const uint16_t* hidden;   // [B, N, dm]
  const uint16_t* w_head;   // [V, dm]
  const float* gumbel;      // [B, Dmax+1, V] or null
  const int32_t* tree_tokens;
  const int32_t* tree_parent;
  const int32_t* n_nodes;
  int32_t* n_accepted;
  int32_t* out_tokens;
  int32_t* out_nodes;
  int32_t* n_emitted;
  int32_t* n_act;           // [kMaxLevels + 1] walking sequences per level
  int32_t* fin_n;           // [kMaxLevels + 1] nodes in the walkers' subtrees per level
  int32_t* act;             // [2, B] walking sequences, by level parity
  int32_t* fin;             // [2, 3, kFinishRows] (sequence, node, depth) of those nodes
  int32_t* cur;             // [B] current node of each sequence
  int32_t* rowtab;          // [B, N] row of a node in its level's subtree list
  unsigned long long* cand; // [max(B, kFinishRows), n_vt] packed candidates of the level
  int B, N, dm, V, Dmax, n_vt;
  int vec_noise;            // gumbel rows can be read as float4
  float invT;
};

// Scratch layout: counters, lists, current nodes, node rows, candidates.
struct ScratchLayout {
  size_t off_fin_n, off_act, off_fin, off_cur, off_rowtab, off_cand, total;
};

inline ScratchLayout scratch_layout(int64_t B, int64_t N, int64_t V) {
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  ScratchLayout s;
  const int64_t n_vt = (V + kTV - 1) / kTV;
  const int64_t rows = std::max<int64_t>(B, kFinishRows);
  s.off_fin_n = up(sizeof(int32_t) * (kMaxLevels + 1));
  s.off_act = s.off_fin_n + up(sizeof(int32_t) * (kMaxLevels + 1));
  s.off_fin = s.off_act + up(sizeof(int32_t) * 2 * static_cast<size_t>(B));
  s.off_cur = s.off_fin + up(sizeof(int32_t) * 2 * 3 * kFinishRows);
  s.off_rowtab = s.off_cur + up(sizeof(int32_t) * static_cast<size_t>(B));
  s.off_cand = s.off_rowtab + up(sizeof(int32_t) * static_cast<size_t>(B) * static_cast<size_t>(N));
  s.total = s.off_cand + up(sizeof(unsigned long long) * static_cast<size_t>(rows) * static_cast<size_t>(n_vt));
  return s;
}

// Total order key of a (score, token) candidate: larger score first, then
// the lower token.  +0 and -0 compare equal, as fp32 comparisons do.
__device__ inline unsigned long long pack_key(float x, int tok) {
  uint32_t u = __float_as_uint(x == 0.f ? 0.f : x);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<unsigned long long>(u) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(tok));
}

__device__ inline int key_token(unsigned long long k) {
  return static_cast<int>(~static_cast<uint32_t>(k & 0xFFFFFFFFull));
}

__device__ inline void take(float& bv, int& bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

// A level runs as a finishing pass when the subtrees of its walkers' current
// nodes (down to depth Dmax) hold at most kFinishRows nodes: one product pass
// then gives the arg-max of every node the remaining walks can visit, and
// the walk kernel completes every walk.
__device__ inline bool finishing(const HeadArgs& a, int level) {
  const int nf = a.fin_n[level];
  return nf > 0 && nf <= kFinishRows;
}

// Row `slot` of a level: its sequence, tree node and depth (= walk step).
__device__ inline void level_row(const HeadArgs& a, int level, bool fin, int slot, int& b, int& u, int& d) {
  if (fin) {
    const int32_t* f = a.fin + (level & 1) * 3 * kFinishRows;
    b = min(max(f[slot], 0), a.B - 1);
    u = min(max(f[kFinishRows + slot], 0), a.N - 1);
    d = min(max(f[2 * kFinishRows + slot], 0), a.Dmax);
  } else {
    b = min(max(a.act[(level & 1) * a.B + slot], 0), a.B - 1);
    u = min(max(a.cur[b], 0), a.N - 1);
    d = level;
  }
}

// One wave lists node u of sequence b (depth du) and its descendants of
// depth <= Dmax in the subtree list of `level`.  Descendants have larger
// indices; a node's ancestry is followed up through parents with smaller
// indices only, so malformed parent links end the search.
__device__ inline void list_subtree(const HeadArgs& a, int level, int b, int u, int du, int n) {
  const int lane = threadIdx.x % SRT_WAVE;
  const int64_t tr = static_cast<int64_t>(b) * a.N;
  int32_t* f = a.fin + (level & 1) * 3 * kFinishRows;
  for (int c0 = u; c0 < n; c0 += SRT_WAVE) {
    const int c = c0 + lane;
    int depth = -1;
    if (c < n) {
      int x = c, steps = 0;
      while (x > u && steps <= a.Dmax - du) {
        const int p = a.tree_parent[tr + x];
        if (p < 0 || p >= x) break;
        x = p;
        ++steps;
      }
      if (x == u && du + steps <= a.Dmax) depth = du + steps;
    }
    const unsigned long long m = __ballot(depth >= 0);
    if (!m) continue;
    int base = 0;
    if (lane == 0) base = atomicAdd(&a.fin_n[level], __popcll(m));
    base = __shfl(base, 0, SRT_WAVE);
    if (depth >= 0) {
      const int r = base + __popcll(m & ((1ull << lane) - 1));
      if (r < kFinishRows) {
        f[r] = b;
        f[kFinishRows + r] = c;
        f[2 * kFinishRows + r] = depth;
        a.rowtab[tr + c] = r;
      }
    }
  }
}

// Level counters: n_act[0] = B, the rest 0.
__global__ __launch_bounds__(128) void head_reset_kernel(HeadArgs a) {
  for (int i = threadIdx.x; i <= kMaxLevels; i += blockDim.x) {
    a.n_act[i] = i == 0 ? a.B : 0;
    a.fin_n[i] = 0;
  }
}

// One wave per sequence: outputs to -1, walking at level 0 from the root,
// whole tree listed for a level-0 finishing pass.
__global__ __launch_bounds__(SRT_WAVE) void head_init_kernel(HeadArgs a) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t row = static_cast<int64_t>(b) * (a.Dmax + 1);
  for (int k = lane; k <= a.Dmax; k += SRT_WAVE) {
    a.out_tokens[row + k] = -1;
    a.out_nodes[row + k] = -1;
  }
  if (lane == 0) {
    a.act[b] = b;
    a.cur[b] = 0;
  }
  list_subtree(a, 0, b, 0, 0, min(max(a.n_nodes[b], 1), a.N));
}

// Wave layouts of a level pass: the 4 waves of a workgroup split its 128
// head rows into WV groups of 32 VT rows and its TM = 32 WS ST sequences
// into WS groups of 32 ST; a wave multiplies its head rows with its
// sequences (VT x ST MFMA tiles).  Narrow (4 x 1 waves, 64 sequences) for
// levels with at most 64 rows; wide (2 x 2 waves, 128 sequences) above,
// which stages each sequence block's rows once per 128 sequences and
// reads a quarter less LDS per product.
struct Narrow {
  static constexpr int WV = 4, VT = 1, WS = 1, ST = 2, TM = 64;
};
struct Wide {
  static constexpr int WV = 2, VT = 2, WS = 2, ST = 2, TM = 128;
};
static_assert(Narrow::WV * Narrow::WS * SRT_WAVE == kThreads && Wide::WV * Wide::WS * SRT_WAVE == kThreads,
              "the WV x WS waves of either layout fill the workgroup");
static_assert(Narrow::TM == 32 * Narrow::WS * Narrow::ST && Wide::TM == 32 * Wide::WS * Wide::ST,
              "TM = 32 WS ST sequences");
constexpr int kMaxTM = 128;
constexpr int kWideAbove = 64;  // rows of a level above which it runs wide

template <bool kNoise, typename Lay>
__device__ inline void level_pass(const HeadArgs& a, int level, bool fin, int n_rows, uint8_t (*s_w)[kTV * kRowBytes],
                                  uint8_t (*s_h)[kMaxTM * kRowBytes], unsigned long long* s_key) {
  constexpr int TM = Lay::TM, HJ = TM / 32;
  // block -> (head tile, sequence block) over the sequence blocks that have
  // rows at this level, so the working blocks come first in dispatch order
  // (blocks that exit at once, interleaved with working ones, leave CUs
  // idle); consecutive blocks on one XCD take the sequence blocks of one
  // tile, so the head rows they share come from its L2.
  const int n_mb = (n_rows + TM - 1) / TM;
  const int n_vt_pad = (a.n_vt + kXcds - 1) / kXcds * kXcds;
  const int g = blockIdx.x;
  if (g >= n_vt_pad * n_mb) return;
  const int i = g / kXcds;
  const int mb = i % n_mb;
  const int vt = (i / n_mb) * kXcds + g % kXcds;
  const int m0 = mb * TM;
  if (vt >= a.n_vt) return;
  const int v0 = vt * kTV;

  const int tid = threadIdx.x;
  const int lane = tid % SRT_WAVE;
  const int wave = __builtin_amdgcn_readfirstlane(tid / SRT_WAVE);
  const int l32 = lane % 32, hf = lane / 32;
  const int wv = wave % Lay::WV, ws = wave / Lay::WV;

  // Global loads stage 16-byte column `col` of rows r0 + 32 j: eight
  // consecutive threads read one row's 128-byte chunk, so every load
  // instruction reads whole cache lines.  Head rows past V read row V - 1
  // and sequence slots past the rows read the first sequence's root row
  // (their products are never used), so every load is unconditional.
  const int col = tid % 8, r0 = tid / 8;
  const uint16_t* wp[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    wp[j] = a.w_head + static_cast<int64_t>(min(v0 + r0 + 32 * j, a.V - 1)) * a.dm + col * 8;
  const uint16_t* hp[HJ];
#pragma unroll
  for (int j = 0; j < HJ; ++j) {
    const int slot = m0 + r0 + 32 * j;
    int64_t off = 0;
    if (slot < n_rows) {
      int b, u, d;
      level_row(a, level, fin, slot, b, u, d);
      off = (static_cast<int64_t>(b) * a.N + u) * a.dm;
    }
    hp[j] = a.hidden + off + col * 8;
  }

  const int n_chunks = a.dm / kKC;
  // Chunk j of the head rows is loaded into wr[j % kInFlight] and chunk j of
  // the hidden rows into hr[j % kInFlight], kInFlight steps before use, and
  // copied to s_w / s_h[j % 2] one step before use.  Vector-memory loads
  // retire in order, so every wait below is for loads issued kInFlight
  // steps earlier and the loads of the steps since stay in flight.
  // (Native vectors: HIP's uint4 class is kept in private memory here.)
  u32x4 wr[kInFlight][4];
  u32x4 hr[kInFlight][HJ];
  auto wload = [&](int s, int c) __attribute__((always_inline)) {
    c = min(c, n_chunks - 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) wr[s][j] = *reinterpret_cast<const u32x4*>(wp[j] + c * kKC);
  };
  auto hload = [&](int s, int c) __attribute__((always_inline)) {
    c = min(c, n_chunks - 1);
#pragma unroll
    for (int j = 0; j < HJ; ++j) hr[s][j] = *reinterpret_cast<const u32x4*>(hp[j] + c * kKC);
  };
  auto stage = [&](int s, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) *reinterpret_cast<u32x4*>(&s_w[buf][(r0 + 32 * j) * kRowBytes + col * 16]) = wr[s][j];
#pragma unroll
    for (int j = 0; j < HJ; ++j)
      *reinterpret_cast<u32x4*>(&s_h[buf][(r0 + 32 * j) * kRowBytes + col * 16]) = hr[s][j];
  };

  f32x16 acc[Lay::VT][Lay::ST];
#pragma unroll
  for (int x = 0; x < Lay::VT; ++x)
#pragma unroll
    for (int y = 0; y < Lay::ST; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.f;
  // A operand (head): rows 32 VT wv + 32 x + l32; B operand (hidden): rows
  // 32 ST ws + 32 y + l32; elements 16 ks + 8 hf .. +7 of each step ks.
  const int a_rd = (32 * Lay::VT * wv + l32) * kRowBytes + 16 * hf;
  const int b_rd = (32 * Lay::ST * ws + l32) * kRowBytes + 16 * hf;

  // Step c (s = c % kInFlight): load head chunk c + kInFlight, multiply
  // chunk c, stage chunk c + 1, load hidden chunk c + 1 + kInFlight.
  // (always_inline: a lambda left out of line would take the register
  // arrays it captures through private memory)
  auto step = [&](int s, int c) __attribute__((always_inline)) {
    wload(s, c + kInFlight);
    bf16x8 af[4][Lay::VT], bfr[4][Lay::ST];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int x = 0; x < Lay::VT; ++x)
        af[ks][x] = *reinterpret_cast<const bf16x8*>(&s_w[s & 1][a_rd + 32 * x * kRowBytes + ks * 32]);
#pragma unroll
      for (int y = 0; y < Lay::ST; ++y)
        bfr[ks][y] = *reinterpret_cast<const bf16x8*>(&s_h[s & 1][b_rd + 32 * y * kRowBytes + ks * 32]);
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int x = 0; x < Lay::VT; ++x)
#pragma unroll
        for (int y = 0; y < Lay::ST; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks][x], bfr[ks][y], acc[x][y], 0, 0, 0);
    const int s1 = (s + 1) % kInFlight;
    stage(s1, (s & 1) ^ 1);
    hload(s1, c + 1 + kInFlight);
    __syncthreads();
  };

  // Prologue in the steady state's load order (as if steps -kInFlight ..
  // -1 had run), so that the waits inside the loop count the same loads on
  // entry as after a full iteration.
  hload(0, 0);
#pragma unroll
  for (int s = 0; s < kInFlight; ++s) {
    wload(s, s);
    if (s == kInFlight - 1) stage(0, 0);
    hload((s + 1) % kInFlight, s + 1);
  }
  __syncthreads();
  const int groups = n_chunks / kInFlight;
  for (int grp = 0; grp < groups; ++grp) {
#pragma unroll
    for (int s = 0; s < kInFlight; ++s) step(s, grp * kInFlight + s);
  }
#pragma unroll
  for (int s = 0; s < kInFlight - 1; ++s)  // the last n_chunks % kInFlight chunks
    if (s < n_chunks - groups * kInFlight) step(s, groups * kInFlight + s);

  // Epilogue: lane column l32 of tile y is sequence slot m0 + 32 ST ws +
  // 32 y + l32; element r of tile x is head row v0 + 32 VT wv + 32 x +
  // 8 (r / 4) + 4 hf + r % 4.
#pragma unroll
  for (int y = 0; y < Lay::ST; ++y) {
    const int sl = 32 * Lay::ST * ws + 32 * y + l32;
    const int slot = m0 + sl;
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
    if (slot < n_rows) {
      const float* gr = nullptr;
      if (kNoise) {
        int b, u, d;
        level_row(a, level, fin, slot, b, u, d);
        gr = a.gumbel + (static_cast<int64_t>(b) * (a.Dmax + 1) + d) * a.V;
      }
#pragma unroll
      for (int x = 0; x < Lay::VT; ++x)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int vb = v0 + 32 * Lay::VT * wv + 32 * x + 8 * q + 4 * hf;
          float gv[4] = {0.f, 0.f, 0.f, 0.f};
          if (kNoise) {
            if (a.vec_noise && vb < a.V) {
              const float4 g4 = *reinterpret_cast<const float4*>(gr + vb);
              gv[0] = g4.x; gv[1] = g4.y; gv[2] = g4.z; gv[3] = g4.w;
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) gv[e] = vb + e < a.V ? gr[vb + e] : 0.f;
            }
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int v = vb + e;
            if (v < a.V) {
              float sc = acc[x][y][4 * q + e];
              if (kNoise) sc = __fadd_rn(__fmul_rn(sc, a.invT), gv[e]);
              take(bv, bi, sc, v);
            }
          }
        }
    }
    const float ov = __shfl_xor(bv, 32, SRT_WAVE);
    const int oi = __shfl_xor(bi, 32, SRT_WAVE);
    take(bv, bi, ov, oi);
    if (hf == 0) s_key[wv * TM + sl] = pack_key(bv, bi);
  }
  __syncthreads();
  if (tid < TM && m0 + tid < n_rows) {
    unsigned long long k = s_key[tid];
#pragma unroll
    for (int w = 1; w < Lay::WV; ++w) k = s_key[w * TM + tid] > k ? s_key[w * TM + tid] : k;
    a.cand[static_cast<int64_t>(m0 + tid) * a.n_vt + vt] = k;
  }
}

// One level's products and per-tile arg-max candidates.
template <bool kNoise>
__global__ __launch_bounds__(kThreads) void head_level_kernel(HeadArgs a, int level) {
  __shared__ __attribute__((aligned(16))) uint8_t s_w[2][kTV * kRowBytes];
  __shared__ __attribute__((aligned(16))) uint8_t s_h[2][kMaxTM * kRowBytes];
  __shared__ unsigned long long s_key[4 * 64];
  const bool fin = finishing(a, level);
  const int n_rows = fin ? a.fin_n[level] : a.n_act[level];
  if (n_rows > kWideAbove)
    level_pass<kNoise, Wide>(a, level, fin, n_rows, s_w, s_h, s_key);
  else
    level_pass<kNoise, Narrow>(a, level, fin, n_rows, s_w, s_h, s_key);
}

// Best candidate of one row over the tiles: every thread of the workgroup
// takes a few, then a block reduction; the result is in every thread.
__device__ inline unsigned long long row_best(const HeadArgs& a, int r, unsigned long long* s_best) {
  const int tid = threadIdx.x, lane = tid % SRT_WAVE, wave = tid / SRT_WAVE;
  const unsigned long long* c = a.cand + static_cast<int64_t>(r) * a.n_vt;
  unsigned long long best = 0;
  for (int t = tid; t < a.n_vt; t += kWalkThreads) best = c[t] > best ? c[t] : best;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const unsigned long long o = shfl_xor_u64(best, off);
    best = o > best ? o : best;
  }
  __syncthreads();  // s_best is free (previous readers done)
  if (lane == 0) s_best[wave] = best;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kWalkThreads / SRT_WAVE; ++w) best = s_best[w] > best ? s_best[w] : best;
  return best;
}

// Child of u carrying tok (wave-wide search), or -1.
__device__ inline int find_child(const HeadArgs& a, int64_t tr, int u, int n, int tok) {
  const int lane = threadIdx.x % SRT_WAVE;
  int child = -1;
  for (int c0 = u + 1; c0 < n && child < 0; c0 += SRT_WAVE) {
    const int cc = c0 + lane;
    const bool hit = cc < n && a.tree_parent[tr + cc] == u && a.tree_tokens[tr + cc] == tok;
    const unsigned long long m = __ballot(hit);
    if (m) child = c0 + __ffsll(static_cast<long long>(m)) - 1;
  }
  return child;
}

// One workgroup per walking sequence.  Ordinary level: one step of the walk
// from the row's candidates; a sequence that descends joins the next level
// with its new node's subtree listed.  Finishing pass: the walk runs to its
// end, every visited node's candidates found through the node-row table.
__global__ __launch_bounds__(kWalkThreads) void head_walk_kernel(HeadArgs a, int level) {
  __shared__ unsigned long long s_best[kWalkThreads / SRT_WAVE];
  __shared__ int s_next;
  const int slot = blockIdx.x;
  if (slot >= a.n_act[level]) return;
  const bool fin = finishing(a, level);
  const int tid = threadIdx.x, lane = tid % SRT_WAVE, wave = tid / SRT_WAVE;
  const int b = min(max(a.act[(level & 1) * a.B + slot], 0), a.B - 1);
  const int n = min(max(a.n_nodes[b], 1), a.N);
  const int64_t tr = static_cast<int64_t>(b) * a.N;
  const int64_t orow = static_cast<int64_t>(b) * (a.Dmax + 1);
  int u = a.cur[b];
  for (int k = level; k <= a.Dmax; ++k) {
    const int r = fin ? min(max(a.rowtab[tr + u], 0), kFinishRows - 1) : slot;
    const int tok = key_token(row_best(a, r, s_best));
    if (wave == 0) {
      const int child = k < a.Dmax ? find_child(a, tr, u, n, tok) : -1;
      if (lane == 0) {
        a.out_tokens[orow + k] = tok;
        if (child >= 0) {
          a.out_nodes[orow + k] = child;
          a.cur[b] = child;
        } else {
          a.n_accepted[b] = k;
          if (a.n_emitted) a.n_emitted[b] = k + 1;
        }
        s_next = child;
      }
      if (!fin && child >= 0) {
        if (lane == 0) {
          const int pos = atomicAdd(&a.n_act[level + 1], 1);
          a.act[((level + 1) & 1) * a.B + pos] = b;
        }
        list_subtree(a, level + 1, b, child, k + 1, n);
      }
    }
    __syncthreads();
    const int next = s_next;
    if (!fin || next < 0) break;
    u = next;
  }
}

}  // namespace

extern "C" size_t srt_accept_lmhead_scratch_bytes(int32_t B, int32_t N, int32_t V) {
  if (B < 0 || N < 1 || V < 1) return 0;
  return scratch_layout(std::max(B, 1), N, V).total;
}

extern "C" int srt_accept_lmhead(int32_t B, int32_t N, int32_t d_model, int32_t V, int32_t Dmax,
                                 const uint16_t* hidden, const uint16_t* w_head, const float* gumbel,
                                 float inv_temperature, const int32_t* tree_tokens, const int32_t* tree_parent,
                                 const int32_t* n_nodes, int32_t* n_accepted, int32_t* out_tokens,
                                 int32_t* out_nodes, int32_t* n_emitted, void* scratch, size_t scratch_bytes,
                                 void* stream) {
  if (B < 0 || N < 1 || V < 1 || d_model < 1 || Dmax < 0 || Dmax >= kMaxLevels) return SRT_ERR_INVALID;
  if (gumbel && !std::isfinite(inv_temperature)) return SRT_ERR_INVALID;
  if (d_model % kKC != 0) return SRT_ERR_UNSUPPORTED;
  if (B == 0) return SRT_OK;
  if (!hidden || !w_head || !tree_tokens || !tree_parent || !n_nodes || !n_accepted || !out_tokens || !out_nodes ||
      !scratch)
    return SRT_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(hidden) | reinterpret_cast<uintptr_t>(w_head)) & 15) return SRT_ERR_INVALID;
  if (reinterpret_cast<uintptr_t>(scratch) & 255) return SRT_ERR_INVALID;
  const ScratchLayout L = scratch_layout(B, N, V);
  if (scratch_bytes < L.total) return SRT_ERR_CAPACITY;
  const int64_t n_vt = (static_cast<int64_t>(V) + kTV - 1) / kTV;
  const int64_t n_mb = (std::max<int64_t>(B, kFinishRows) + Narrow::TM - 1) / Narrow::TM;
  const int64_t n_vt_pad = (n_vt + kXcds - 1) / kXcds * kXcds;
  if (n_vt_pad * n_mb > 0x7FFFFFFF) return SRT_ERR_UNSUPPORTED;

  char* base = static_cast<char*>(scratch);
  HeadArgs a;
  a.hidden = hidden;
  a.w_head = w_head;
  a.gumbel = gumbel;
  a.tree_tokens = tree_tokens;
  a.tree_parent = tree_parent;
  a.n_nodes = n_nodes;
  a.n_accepted = n_accepted;
  a.out_tokens = out_tokens;
  a.out_nodes = out_nodes;
  a.n_emitted = n_emitted;
  a.n_act = reinterpret_cast<int32_t*>(base);
  a.fin_n = reinterpret_cast<int32_t*>(base + L.off_fin_n);
  a.act = reinterpret_cast<int32_t*>(base + L.off_act);
  a.fin = reinterpret_cast<int32_t*>(base + L.off_fin);
  a.cur = reinterpret_cast<int32_t*>(base + L.off_cur);
  a.rowtab = reinterpret_cast<int32_t*>(base + L.off_rowtab);
  a.cand = reinterpret_cast<unsigned long long*>(base + L.off_cand);
  a.B = B;
  a.N = N;
  a.dm = d_model;
  a.V = V;
  a.Dmax = Dmax;
  a.n_vt = static_cast<int>(n_vt);
  a.invT = inv_temperature;
  a.vec_noise = gumbel && V % 4 == 0 && (reinterpret_cast<uintptr_t>(gumbel) & 15) == 0;

  hipStream_t s = as_stream(stream);
  head_reset_kernel<<<1, 128, 0, s>>>(a);
  int st = launch_status();
  if (st == SRT_OK) {
    head_init_kernel<<<B, SRT_WAVE, 0, s>>>(a);
    st = launch_status();
  }
  const unsigned grid = static_cast<unsigned>(n_vt_pad * n_mb);
  const unsigned walk_grid = static_cast<unsigned>(B);
  for (int level = 0; level <= Dmax && st == SRT_OK; ++level) {
    if (gumbel)
      head_level_kernel<true><<<grid, kThreads, 0, s>>>(a, level);
    else
      head_level_kernel<false><<<grid, kThreads, 0, s>>>(a, level);
    st = launch_status();
    if (st != SRT_OK) break;
    head_walk_kernel<<<walk_grid, kWalkThreads, 0, s>>>(a, level);
    st = launch_status();
  }
  return st;
}
