// Tree-masked attention over a paged bf16 KV cache (MFMA, gfx950).
//
// Method: Section 3 of the paper -- one decode pass of the policy verifies
// every drafted token -- and Appendix C (verification reads the KV cache
// once for all candidates).  Tree node i of sequence b attends to the whole
// committed context [0, L) and to the tree positions L + j of its
// ancestors-or-self j; query head h uses KV head h / (Hq / Hkv).
//
// GPU design.  For one (sequence, KV head) all n * G query rows (G query
// heads per KV head) share every K/V tile, so they are processed together:
// a workgroup of 4 waves owns 128 rows (32 per wave, two 16-row MFMA tiles)
// and streams one split of the key range in 64-key tiles.
//   * K and V tiles are read from HBM with 16-byte coalesced loads,
//     prefetched into registers one tile ahead, and staged in LDS (V is
//     transposed on the way in).
//   * S^T = K Q^T and O^T = V^T P^T run on v_mfma_f32_16x16x32_bf16 with
//     fp32 accumulation.  In this orientation a query row lives in one lane
//     column of both accumulators, so the online-softmax statistics and the
//     rescale of O are lane-local, and the probabilities P feed the second
//     MFMA straight from registers: the contraction index of P^T is
//     permuted to match the S^T output layout and V^T is read with the same
//     permutation.
//   * Softmax uses exp2 with scale*log2(e) folded in; row max and sum need
//     two cross-lane shuffles.  The ancestor mask is a bitset per tree node
//     in LDS and is applied only on tiles that reach the tree positions or
//     the end of the range.
//   * Long contexts are split into fixed chunks of keys so the grid has
//     enough independent work; each split writes unnormalised partial
//     output plus (max, sum) and a small combine kernel merges them.  A
//     sequence that fits in one chunk writes bf16 output directly.
//   * Block ids are remapped so that the row blocks and splits of one
//     (sequence, KV head) run on the same XCD and share its L2.
#include <cmath>
#include <type_traits>

#include "common.h"

using namespace srt;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * SRT_WAVE;
constexpr int kRowsPerBlock = kWaves * 32;
constexpr int kTile = 64;      // keys per tile
constexpr int kMaxN = 256;     // tree rows
constexpr int kChunk = 4096;   // keys per split
constexpr int kXcds = 8;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* bt;
  const int32_t* ctx_len;
  const int32_t* parent;
  const int32_t* n_nodes;
  uint16_t* out;
  float* part_o;
  float* part_ml;
  int32_t B, N, Hq, Hkv, G, page, page_shift, max_pages;
  int64_t num_pages;
  float scale_log2;
  int32_t S, RB, total;
};

template <int D>
struct Shape {
  static constexpr int KD = D / 32;      // MFMA steps over the head dimension
  static constexpr int DT = D / 16;      // 16-wide blocks of the head dimension
};

__device__ inline uint16_t to_bf16_bits(float x) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x)); }

struct SeqInfo {
  int n, L, total;
};

__device__ inline SeqInfo seq_info(const AttnArgs& a, int b) {
  SeqInfo s;
  const int cap = a.max_pages * a.page;
  s.n = min(max(a.n_nodes[b], 1), min(a.N, cap));
  s.L = min(max(a.ctx_len[b], 0), cap - s.n);
  s.total = s.L + s.n;
  return s;
}

// Loads kLoads x 1 KB from `base` (nbytes valid, the rest reads as zero)
// straight into LDS: load j writes lds + j*stride_elems, lane l's 16 bytes
// (from byte offset voff[j]) at offset 16*l.
template <int kLoads>
__device__ inline void buffer_to_lds(const uint16_t* base, int nbytes, uint16_t* lds, int stride_elems,
                                     const int (&voff)[kLoads]) {
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, nbytes, 0x00020000);
#pragma unroll
  for (int j = 0; j < kLoads; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(lds + j * stride_elems),
                                             16, voff[j], 0, 0, 0);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void tree_attn_kernel(AttnArgs a) {
  using Sh = Shape<D>;
  constexpr int CPR = D / 8;                 // 16-byte chunks per K/V row
  constexpr int kTileElems = kTile * D;      // unpadded, chunk-swizzled rows
  // K is consumed one tile before V (pipelining below), so each has its own
  // pair of LDS buffers.
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2 * kTileElems];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2 * kTileElems];
  __shared__ uint64_t anc[kMaxN][4];
  __shared__ int32_t spar[kMaxN];

  const int nb = gridDim.x;
  const int item = (blockIdx.x % kXcds) * (nb / kXcds) + blockIdx.x / kXcds;
  if (item >= a.total) return;
  int rest = item;
  const int rb = rest % a.RB;
  rest /= a.RB;
  const int s = rest % a.S;
  rest /= a.S;
  const int g = rest % a.Hkv;
  const int b = rest / a.Hkv;

  const SeqInfo si = seq_info(a, b);
  const int rows = si.n * a.G;
  if (rb * kRowsPerBlock >= rows) return;
  const int k_begin = s * kChunk;
  if (k_begin >= si.total) return;
  const int k_end = min(k_begin + kChunk, si.total);
  const int nsplit = (si.total + kChunk - 1) / kChunk;

  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / SRT_WAVE);  // wave-uniform, in an SGPR
  const int lane = tid % SRT_WAVE;
  const int l16 = lane % 16;
  const int lg = lane / 16;
  const int row0 = rb * kRowsPerBlock + w * 32;
  const bool wave_active = row0 < rows;  // wave-uniform

  // Ancestor-or-self bitsets, needed only when this split reaches the tree.
  if (k_end > si.L) {
    for (int i = tid; i < si.n; i += kThreads) spar[i] = a.parent[static_cast<int64_t>(b) * a.N + i];
    __syncthreads();
    for (int i = tid; i < si.n; i += kThreads) {
      uint64_t bits[4] = {0, 0, 0, 0};
      int j = i;
      while (j >= 0) {
        bits[j >> 6] |= 1ull << (j & 63);
        const int pj = spar[j];
        if (pj >= j) break;  // malformed parent: stop (parents precede children)
        j = pj;
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) anc[i][x] = bits[x];
    }
  }

  // Query fragments: B operand of S^T = K Q^T (lane: row l16, head dims 8*lg..+7).
  bf16x8 qf[2][Sh::KD];
  int node_of[2];
  bool row_ok[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int r = row0 + nt * 16 + l16;
    row_ok[nt] = r < rows;
    const int node = row_ok[nt] ? r / a.G : 0;
    const int h = g * a.G + (row_ok[nt] ? r % a.G : 0);
    node_of[nt] = node;
    const bf16x8* qp = reinterpret_cast<const bf16x8*>(
        a.q + ((static_cast<int64_t>(b) * a.N + node) * a.Hq + h) * D + 8 * lg);
#pragma unroll
    for (int kd = 0; kd < Sh::KD; ++kd) qf[nt][kd] = row_ok[nt] ? qp[4 * kd] : bf16x8{};
  }

  f32x4 o[2][Sh::DT];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int dt = 0; dt < Sh::DT; ++dt) o[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Reference maximum (log2 units) and lane-partial sums per row tile.  The
  // reference is raised only when a row's maximum exceeds it by more than
  // kLazy, so most tiles need no rescale of O.
  constexpr float kLazy = 8.f;
  float m[2] = {-INFINITY, -INFINITY};
  float l[2] = {0.f, 0.f};
  const float c = a.scale_log2;

  // ---- staging ----------------------------------------------------------
  // K and V tiles go straight from HBM to LDS (buffer loads with the LDS
  // destination; no staging registers).  Wave w moves the w-th 16-key
  // sub-block of a tile, which lies inside one page (pages are powers of two
  // >= 16): one buffer descriptor covers exactly its valid keys, so keys past
  // the split end or on an invalid page read as zero.  Row r's 16-byte chunk
  // c is stored at chunk position c ^ (r % CPR) (conflict-free operand reads);
  // a load instruction writes 1 KB contiguous, lane l at offset 16*l, so lane
  // l fetches the chunk that belongs at its position.
  const int pshift = a.page_shift;
  const int pmask = (1 << pshift) - 1;
  const int64_t bt_row = static_cast<int64_t>(b) * a.max_pages;
  const int32_t __attribute__((address_space(4)))* btc =
      (const int32_t __attribute__((address_space(4)))*)(a.bt) + bt_row;
  const int64_t head_stride = static_cast<int64_t>(a.page) * D;  // elements per (page, head)
  constexpr int kRowsPerLoad = 1024 / (2 * D);                    // 4 (d=128) or 8 (d=64)
  constexpr int kLoadsPerWave = 16 / kRowsPerLoad;                // per tile, per tensor
  // Per-lane byte offset inside the sub-block and LDS placement of each load.
  int lane_voff[kLoadsPerWave];
#pragma unroll
  for (int j = 0; j < kLoadsPerWave; ++j) {
    const int r = kRowsPerLoad * j + lane / CPR;     // row within the sub-block (0..15)
    const int pos = lane % CPR;                      // chunk position written by this lane
    const int row = 16 * w + r;                      // row within the tile
    const int chunk = pos ^ (row & (CPR - 1));
    lane_voff[j] = (r * D + chunk * 8) * 2;
  }

  // Page id of this wave's sub-block of the tile at t0 (-1 if none).
  auto sub_page = [&](int t0) {
    const int p0 = t0 + 16 * w;
    return p0 < k_end ? btc[p0 >> pshift] : -1;
  };
  auto issue_tile = [&](const uint16_t* src, uint16_t* dst, int t0, int pg) {
    const int p0 = t0 + 16 * w;
    const bool ok = pg >= 0 && pg < a.num_pages && p0 < k_end;
    const int nkeys = ok ? min(16, k_end - p0) : 0;
    const uint16_t* base = ok ? src + (static_cast<int64_t>(pg) * a.Hkv + g) * head_stride + (p0 & pmask) * D : src;
    buffer_to_lds<kLoadsPerWave>(base, nkeys * D * 2, dst + 16 * w * D, kRowsPerLoad * D, lane_voff);
  };

  // ---- MFMA phases -------------------------------------------------------
  // Lane offsets (elements) of the swizzled operand reads.  For K the XOR
  // term depends only on the lane's row within a 16-row group, so row groups
  // (mt) add a constant; for V it depends on the row within 16 as well, so
  // ks and the +16-row half add constants.  Only the head-dim index varies
  // non-linearly and gets its own register.
  int koff[Sh::KD];
#pragma unroll
  for (int kd = 0; kd < Sh::KD; ++kd) koff[kd] = (l16 * CPR + ((4 * kd + lg) ^ (l16 & (CPR - 1)))) * 8;
  int voff[Sh::DT];
  {
    const int r0 = 4 * lg + l16 / 4;  // row within the 32-row group, < 16
#pragma unroll
    for (int dt = 0; dt < Sh::DT; ++dt)
      voff[dt] = (r0 * CPR + ((2 * dt + ((l16 & 3) >> 1)) ^ (r0 & (CPR - 1)))) * 8 + (l16 & 1) * 4;
  }

  // S^T[key][row] of one tile: 4 key groups x 2 row tiles.
  auto qk = [&](const uint16_t* Kb, f32x4 (&sacc)[2][4]) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) sacc[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kd = 0; kd < Sh::KD; ++kd) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(Kb + 16 * mt * D + koff[kd]);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
          sacc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[nt][kd], sacc[nt][mt], 0, 0, 0);
      }
    }
  };

  // Mask, online softmax with lazy rescale; returns P in bf16.
  auto softmax = [&](int t0, f32x4 (&sacc)[2][4], bf16x8 (&pb)[2][2]) {
    const bool need_mask = (t0 + kTile > si.L) || (t0 + kTile > k_end);
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      if (need_mask) {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          f32x4 t = sacc[nt][mt];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int pos = t0 + 16 * mt + 4 * lg + r;
            bool vis = pos < k_end;
            if (vis && pos >= si.L) {
              const int j = pos - si.L;
              vis = (anc[node_of[nt]][j >> 6] >> (j & 63)) & 1ull;
            }
            t[r] = vis ? t[r] : -INFINITY;
          }
          sacc[nt][mt] = t;
        }
      }
      float mloc = fmaxf(fmaxf(sacc[nt][0][0], sacc[nt][0][1]), fmaxf(sacc[nt][0][2], sacc[nt][0][3]));
#pragma unroll
      for (int mt = 1; mt < 4; ++mt)
        mloc = fmaxf(mloc, fmaxf(fmaxf(sacc[nt][mt][0], sacc[nt][mt][1]), fmaxf(sacc[nt][mt][2], sacc[nt][mt][3])));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16, SRT_WAVE));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, SRT_WAVE));
      const float ms = mloc * c;  // row max in log2 units (c > 0)
      const bool raise = ms > m[nt] + kLazy;
      if (__ballot(raise)) {
        const float mnew = raise ? ms : m[nt];
        const float alpha = m[nt] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[nt] - mnew);
        l[nt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < Sh::DT; ++dt) o[nt][dt] *= alpha;
        m[nt] = mnew;
      }
      const float mref = m[nt] == -INFINITY ? 0.f : m[nt];
      float psum = 0.f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[nt][mt][r], c, -mref));
          sacc[nt][mt][r] = p;
          psum += p;
        }
      }
      l[nt] += psum;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pb[nt][ks][r] = static_cast<__bf16>(sacc[nt][2 * ks][r]);
          pb[nt][ks][4 + r] = static_cast<__bf16>(sacc[nt][2 * ks + 1][r]);
        }
      }
    }
  };

  // O^T[d][row] += V^T P^T.  Contraction index (8*lg + e) <-> key
  // 32*ks + 16*(e/4) + 4*lg + e%4, matching the S^T layout; the V^T operand
  // comes from transposing LDS reads: lane (lg, l16) addresses row
  // 32*ks + 4*lg + l16/4 (+16), head dims 16*dt + 4*(l16%4) .. +3.
  auto pv = [&](const uint16_t* Vb, const bf16x8 (&pb)[2][2]) {
    typedef short i16x4 __attribute__((ext_vector_type(4)));
    typedef short i16x8 __attribute__((ext_vector_type(8)));
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int dt = 0; dt < Sh::DT; ++dt) {
        const uint16_t* p0 = Vb + 32 * ks * D + voff[dt];
        const uint16_t* p1 = p0 + 16 * D;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p0));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p1));
        const i16x8 both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        const bf16x8 va = __builtin_bit_cast(bf16x8, both);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
          o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[nt][ks], o[nt][dt], 0, 0, 0);
      }
    }
  };

  // ---- software pipeline -------------------------------------------------
  // Iteration t: global loads of K(t+2) and V(t+1) are issued; S(t+1) = K Q^T
  // of the next tile runs on the MFMA pipe while softmax(t) runs on the VALU;
  // then O += V(t)^T P(t); finally K(t+2) and V(t+1) go to the buffers that
  // K(t) and V(t-1) have left.  One barrier per tile.
  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  int pgA = sub_page(k_begin), pgB = sub_page(k_begin + kTile), pgC = sub_page(k_begin + 2 * kTile);
  issue_tile(a.k, Ks, k_begin, pgA);
  issue_tile(a.v, Vs, k_begin, pgA);
  if (ntiles > 1) issue_tile(a.k, Ks + kTileElems, k_begin + kTile, pgB);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  f32x4 scur[2][4];
  if (wave_active) qk(Ks, scur);
  __syncthreads();  // every wave has read K(0) before iteration 0 refills its buffer

  // One pipeline step for tile `it` (buffer parity CUR = it & 1, a
  // compile-time constant so LDS buffer bases fold into immediates).
  auto step = [&](int it, auto cur_c) {
    constexpr int cur = decltype(cur_c)::value;
    const int t0 = k_begin + it * kTile;
    // page ids: pgA <- tile t+1, pgB <- t+2, pgC <- t+3
    pgA = pgB;
    pgB = pgC;
    pgC = sub_page(t0 + 3 * kTile);
    // K(t+2) into the buffer K(t) left, V(t+1) into the one V(t-1) left.
    if (it + 2 < ntiles) issue_tile(a.k, Ks + cur * kTileElems, t0 + 2 * kTile, pgB);
    if (it + 1 < ntiles) issue_tile(a.v, Vs + (cur ^ 1) * kTileElems, t0 + kTile, pgA);
    if (wave_active) {
      f32x4 snext[2][4];
      if (it + 1 < ntiles) qk(Ks + (cur ^ 1) * kTileElems, snext);
      bf16x8 pb[2][2];
      softmax(t0, scur, pb);
      pv(Vs + cur * kTileElems, pb);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) scur[nt][mt] = snext[nt][mt];
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(it, std::integral_constant<int, 0>());
    if (it + 1 < ntiles) step(it + 1, std::integral_constant<int, 1>());
  }

  // Epilogue: lane holds row l16 and head dims 16*dt + 4*lg + 0..3.
  const int RBR = a.RB * kRowsPerBlock;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    float lt = l[nt];
    lt += __shfl_xor(lt, 16, SRT_WAVE);
    lt += __shfl_xor(lt, 32, SRT_WAVE);
    if (!row_ok[nt]) continue;
    const int r = row0 + nt * 16 + l16;
    if (nsplit == 1) {
      const int h = g * a.G + r % a.G;
      uint16_t* op = a.out + ((static_cast<int64_t>(b) * a.N + r / a.G) * a.Hq + h) * D + 4 * lg;
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
      for (int dt = 0; dt < Sh::DT; ++dt) {
        const uint32_t x0 = to_bf16_bits(o[nt][dt][0] * inv) | (uint32_t(to_bf16_bits(o[nt][dt][1] * inv)) << 16);
        const uint32_t x1 = to_bf16_bits(o[nt][dt][2] * inv) | (uint32_t(to_bf16_bits(o[nt][dt][3] * inv)) << 16);
        *reinterpret_cast<uint2*>(op + 16 * dt) = make_uint2(x0, x1);
      }
    } else {
      const int64_t prow = ((static_cast<int64_t>(b) * a.Hkv + g) * a.S + s) * RBR + r;
      float* po = a.part_o + prow * D + 4 * lg;
#pragma unroll
      for (int dt = 0; dt < Sh::DT; ++dt) *reinterpret_cast<f32x4*>(po + 16 * dt) = o[nt][dt];
      if (lg == 0) {
        a.part_ml[2 * prow] = m[nt];
        a.part_ml[2 * prow + 1] = lt;
      }
    }
  }
}

// Merges the split partials of sequences that needed more than one split.
// One wave per output row (b, node, head).
template <int D>
__global__ __launch_bounds__(256) void tree_attn_combine_kernel(AttnArgs a) {
  const int wave = blockIdx.x * 4 + threadIdx.x / SRT_WAVE;
  const int lane = threadIdx.x % SRT_WAVE;
  const int per_seq = a.N * a.Hq;
  if (wave >= a.B * per_seq) return;
  const int b = wave / per_seq;
  const int node = (wave % per_seq) / a.Hq;
  const int h = wave % a.Hq;
  const SeqInfo si = seq_info(a, b);
  if (node >= si.n) return;
  const int nsplit = (si.total + kChunk - 1) / kChunk;
  if (nsplit <= 1) return;
  const int g = h / a.G;
  const int r = node * a.G + h % a.G;
  const int RBR = a.RB * kRowsPerBlock;
  const int64_t base = (static_cast<int64_t>(b) * a.Hkv + g) * a.S * RBR + r;
  float M = -INFINITY;
  for (int s = 0; s < nsplit; ++s) M = fmaxf(M, a.part_ml[2 * (base + static_cast<int64_t>(s) * RBR)]);
  constexpr int PER = D / SRT_WAVE;
  float num[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) num[i] = 0.f;
  float den = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const int64_t prow = base + static_cast<int64_t>(s) * RBR;
    const float ms = a.part_ml[2 * prow];
    const float wgt = ms == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ms - M);
    den += wgt * a.part_ml[2 * prow + 1];
#pragma unroll
    for (int i = 0; i < PER; ++i) num[i] += wgt * a.part_o[prow * D + lane + SRT_WAVE * i];
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  uint16_t* op = a.out + ((static_cast<int64_t>(b) * a.N + node) * a.Hq + h) * D;
#pragma unroll
  for (int i = 0; i < PER; ++i) op[lane + SRT_WAVE * i] = to_bf16_bits(num[i] * inv);
}

int splits_for(int32_t page, int32_t max_pages) {
  const int64_t cap = static_cast<int64_t>(page) * max_pages;
  return static_cast<int>((cap + kChunk - 1) / kChunk);
}

}  // namespace

extern "C" size_t srt_tree_attn_scratch_bytes(int32_t B, int32_t N, int32_t Hq, int32_t Hkv, int32_t d, int32_t page,
                                              int32_t max_pages) {
  if (B < 0 || N < 1 || N > kMaxN || Hq < 1 || Hkv < 1 || Hq % Hkv || page < 1 || max_pages < 1) return 0;
  const int S = splits_for(page, max_pages);
  if (S <= 1) return 0;
  const int G = Hq / Hkv;
  const int64_t RBR = static_cast<int64_t>((N * G + kRowsPerBlock - 1) / kRowsPerBlock) * kRowsPerBlock;
  return static_cast<size_t>(B) * Hkv * S * RBR * (d + 2) * sizeof(float);
}

extern "C" int srt_tree_attn(int32_t B, int32_t N, int32_t Hq, int32_t Hkv, int32_t d, int32_t page,
                             int32_t max_pages, int64_t num_pages, const uint16_t* q, const uint16_t* k_cache,
                             const uint16_t* v_cache, const int32_t* block_table, const int32_t* ctx_len,
                             const int32_t* tree_parent, const int32_t* n_nodes, float scale, uint16_t* out,
                             void* scratch, size_t scratch_bytes, void* stream) {
  if (B < 0 || N < 1 || N > kMaxN || Hq < 1 || Hkv < 1 || Hq % Hkv || page < 1 || max_pages < 1 || num_pages < 1)
    return SRT_ERR_INVALID;
  if (!(scale == scale)) return SRT_ERR_INVALID;
  if (d != 64 && d != 128) return SRT_ERR_UNSUPPORTED;
  if (page < 16 || (page & (page - 1))) return SRT_ERR_UNSUPPORTED;
  if (B == 0) return SRT_OK;
  if (!q || !k_cache || !v_cache || !block_table || !ctx_len || !tree_parent || !n_nodes || !out)
    return SRT_ERR_INVALID;
  const size_t need = srt_tree_attn_scratch_bytes(B, N, Hq, Hkv, d, page, max_pages);
  if (need > 0 && (!scratch || scratch_bytes < need)) return SRT_ERR_CAPACITY;

  AttnArgs a;
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.bt = block_table;
  a.ctx_len = ctx_len;
  a.parent = tree_parent;
  a.n_nodes = n_nodes;
  a.out = out;
  a.B = B;
  a.N = N;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = Hq / Hkv;
  a.page = page;
  a.page_shift = __builtin_ctz(static_cast<unsigned>(page));
  a.max_pages = max_pages;
  a.num_pages = num_pages;
  a.scale_log2 = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
  a.S = splits_for(page, max_pages);
  a.RB = (N * a.G + kRowsPerBlock - 1) / kRowsPerBlock;
  const int64_t total = static_cast<int64_t>(B) * Hkv * a.S * a.RB;
  if (total > (int64_t(1) << 30)) return SRT_ERR_INVALID;
  a.total = static_cast<int32_t>(total);
  const int64_t RBR = static_cast<int64_t>(a.RB) * kRowsPerBlock;
  a.part_o = static_cast<float*>(scratch);
  a.part_ml = need ? static_cast<float*>(scratch) + static_cast<int64_t>(B) * Hkv * a.S * RBR * d : nullptr;

  const unsigned grid = static_cast<unsigned>((total + kXcds - 1) / kXcds * kXcds);
  hipStream_t s = as_stream(stream);
  if (d == 128) {
    tree_attn_kernel<128><<<grid, kThreads, 0, s>>>(a);
  } else {
    tree_attn_kernel<64><<<grid, kThreads, 0, s>>>(a);
  }
  if (a.S > 1) {
    const int64_t rows = static_cast<int64_t>(B) * N * Hq;
    const unsigned cgrid = static_cast<unsigned>((rows + 3) / 4);
    if (d == 128) {
      tree_attn_combine_kernel<128><<<cgrid, 256, 0, s>>>(a);
    } else {
      tree_attn_combine_kernel<64><<<cgrid, 256, 0, s>>>(a);
    }
  }
  return launch_status();
}
