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
// a workgroup of 8 waves owns 256 rows (32 per wave) and streams one split
// of the key range in 64-key tiles; one workgroup per CU.
//   * Products run on v_mfma_f32_32x32x16_bf16 (the full-rate bf16 shape on
//     gfx950) with fp32 accumulation: S^T = K Q^T (32 keys x 32 rows per
//     MFMA) and O^T = V^T P^T (32 head dims x 32 rows).  In this orientation
//     a query row lives in one lane column of both accumulators, so the
//     online-softmax statistics and the rescale of O are lane-local (the
//     two lane halves are merged with one permlane32 swap) and P feeds the
//     second MFMA straight from registers: the contraction index of P^T is
//     permuted to match the S^T output layout, and V^T is read with the same
//     permutation by ds_read_b64_tr_b16 transposing reads.  The head-dim
//     order inside each 32-row block of O^T is permuted too (lane halves of
//     a transposing read take head dims D/2 apart), which the epilogue undoes.
//   * K and V tiles are read from HBM with 16-byte buffer loads (one scalar
//     descriptor per 8-key sub-block of a page, so tails read as zero),
//     prefetched into registers one tile ahead and stored to double-buffered
//     LDS.  LDS rows are padded (K by 16 bytes, V by 32) so that the operand
//     reads of every MFMA are bank-conflict free and their addresses are one
//     base register plus immediate offsets.
//   * Softmax uses exp2 of fma(q.k, scale*log2(e), -reference) (Q is never
//     rescaled or re-rounded) and a lazily raised reference maximum; a tile
//     whose probabilities all stay below 2^8 of the reference (checked on
//     their sum) needs no row maximum at all.  The ancestor mask is a bitset per tree node in LDS;
//     on tiles that reach the tree positions or the end of the range each
//     row takes a 64-bit visibility window of it (two LDS words) and masks
//     its scores bit by bit.
//   * Long contexts are split into chunks of keys so the grid has enough
//     independent work (8192 keys, or a smaller power of two down to 1024
//     when the batch has few sequences and KV heads); each split writes
//     unnormalised partial output plus (max, sum) and a small combine
//     kernel merges them.  A sequence that fits in one split writes bf16
//     output directly.
//   * Work is scheduled by a small plan kernel that lists the (sequence, KV
//     head, split, row block) items that have work, longest first; one
//     persistent workgroup per CU takes items from an atomic counter, so no
//     CU idles on empty grid slots and long items do not form a tail.
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.h"

using namespace srt;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * SRT_WAVE;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerBlock = kWaves * kRowsPerWave;
constexpr int kTile = 64;                  // keys per tile
constexpr int kSubRows = kTile / kWaves;   // keys of each tile one wave stages
constexpr int kMaxN = 256;                 // tree rows
constexpr int kChunk = 8192;               // keys per split, at most (the split size is chosen per call)
constexpr int kMinChunk = 1024;            // keys per split, at least

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
  int32_t* plan;  // work lists built by the plan kernel
  int64_t combine_at;  // offset (int32 elements) of the combine list in plan
  int32_t max_units;   // capacity of the combine list
  int32_t B, N, Hq, Hkv, G, page, page_shift, max_pages;
  int64_t num_pages;
  float scale_log2;
  int32_t S, RB, total;
  int32_t chunk;  // keys per split: a power of two in [kMinChunk, kChunk]
};

// Work list: plan[0] = number of items, plan[1] = next item to hand out,
// then item i at plan[kPlanHeader + 2 i] = sequence, [.. + 1] = KV head |
// split << 8 | row block << 20.  Items are ordered by decreasing cost
// (tiles, then active waves) so that the longest ones start first.
// plan[2] = number of combine units; unit u (8 rows of one sequence and KV
// head whose context spans several splits) at plan[a.combine_at + u] =
// sequence | KV head << 16 (the host rejects B > 65535) and the 8-row group
// at plan[a.combine_at + a.max_units + u].
constexpr int kPlanHeader = 64;
constexpr int kPlanKeys = (kChunk / kTile) * kWaves;  // (tiles, waves) classes

__device__ inline int plan_key(int tiles, int waves) {  // 0 = most expensive
  return kPlanKeys - 1 - ((tiles - 1) * kWaves + (waves - 1));
}

template <int D>
struct Shape {
  static constexpr int KS = D / 16;            // k-steps of S^T = K Q^T
  static constexpr int DB = D / 32;            // 32-dim blocks of O^T
  static constexpr int CPR = D / 8;            // 16-byte chunks per K/V row
  static constexpr int KSTRIDE = 2 * D + 16;   // LDS bytes per K row
  static constexpr int VSTRIDE = 2 * D + 32;   // LDS bytes per V row
  static constexpr int KTILE = kTile * KSTRIDE;
  static constexpr int VTILE = kTile * VSTRIDE;
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

// Buffer descriptor over `nbytes` bytes at `base` (loads past nbytes read 0).
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const uint16_t* base, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, nbytes, 0x00020000);
}

// kLoads 16-byte loads through one descriptor: lane byte offset voff plus
// j * step for load j.
template <int kLoads, int kStep>
__device__ inline void buffer_load16(const uint16_t* base, int nbytes, int voff, uint4 (&r)[kLoads]) {
  const __amdgpu_buffer_rsrc_t rsrc = make_rsrc(base, nbytes);
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    typedef int i32x4 __attribute__((ext_vector_type(4)));
    const i32x4 x = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff + j * kStep, 0, 0);
    r[j] = __builtin_bit_cast(uint4, x);
  }
}

// The two 32-lane halves of x exchanged by v_permlane32_swap: returns
// {x, x of lane ^ 32} in some order.  (Each result element is copied to a
// scalar before the bit cast: a bit cast of a vector element reads
// element 0 with this compiler.)
__device__ inline void swap_halves(float x, float& u, float& v) {
  const unsigned a = __builtin_bit_cast(unsigned, x);
  const auto s = __builtin_amdgcn_permlane32_swap(a, a, false, false);
  const unsigned s0 = s[0], s1 = s[1];
  u = __builtin_bit_cast(float, s0);
  v = __builtin_bit_cast(float, s1);
}

// Maximum / sum over the two 32-lane halves, result in every lane.
__device__ inline float max_halves(float x) {
  float u, v;
  swap_halves(x, u, v);
  return __builtin_elementwise_maximum(u, v);
}

__device__ inline float sum_halves(float x) {
  float u, v;
  swap_halves(x, u, v);
  return u + v;
}

template <int D>
__global__ __launch_bounds__(kThreads, 1) void tree_attn_kernel(AttnArgs a) {
  using Sh = Shape<D>;
  constexpr int CPR = Sh::CPR;
  __shared__ __attribute__((aligned(16))) uint8_t Ks[2 * Sh::KTILE];
  __shared__ __attribute__((aligned(16))) uint8_t Vs[2 * Sh::VTILE];
  __shared__ uint64_t anc[kMaxN][4];
  __shared__ int32_t spar[kMaxN];

  __shared__ int32_t s_item;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid / SRT_WAVE);  // wave-uniform, in an SGPR
  const int lane = tid % SRT_WAVE;
  const int l32 = lane % 32;  // query row of this lane inside the wave's 32
  const int h = lane / 32;    // lane half
  const int n_items = a.plan[0];

  // Persistent workgroups: each takes the next item of the work list until
  // the list is exhausted.
  auto run_item = [&](const int b, const int g, const int s, const int rb) {
  const SeqInfo si = seq_info(a, b);
  const int rows = si.n * a.G;
  if (rb * kRowsPerBlock >= rows) return;
  const int k_begin = s * a.chunk;
  if (k_begin >= si.total) return;
  const int k_end = min(k_begin + a.chunk, si.total);
  const int nsplit = (si.total + a.chunk - 1) / a.chunk;
  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  const int row0 = rb * kRowsPerBlock + w * kRowsPerWave;
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

  // Query fragment: B operand of S^T = K Q^T; lane holds row l32 and head
  // dims 16 ks + 8 h .. +7 for k-step ks.
  const int row = row0 + l32;
  const bool row_ok = row < rows;
  const int node = row_ok ? row / a.G : 0;
  bf16x8 qf[Sh::KS];
  {
    const int hq = g * a.G + (row_ok ? row % a.G : 0);
    const bf16x8* qp =
        reinterpret_cast<const bf16x8*>(a.q + ((static_cast<int64_t>(b) * a.N + node) * a.Hq + hq) * D + 8 * h);
#pragma unroll
    for (int ks = 0; ks < Sh::KS; ++ks) qf[ks] = row_ok ? qp[2 * ks] : bf16x8{};
    // Q is used exactly as given: the scale is applied to the fp32 scores
    // (rounding a scaled Q back to bf16 would perturb every score by up to
    // 2^-9 of its magnitude).
  }
  const float c_log2 = a.scale_log2;  // scale * log2(e)

  f32x16 o[Sh::DB];
#pragma unroll
  for (int db = 0; db < Sh::DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  // Reference maximum (log2 units) and lane-partial sum of the row.  The
  // reference is raised only when the row maximum exceeds it by more than
  // kLazy, so most tiles need no rescale of O.
  constexpr float kLazy = 8.f;
  float m = -INFINITY;
  float l = 0.f;

  // ---- staging ----------------------------------------------------------
  // Wave w moves keys 8w .. 8w+7 of every K and V tile; they lie inside one
  // page (pages are powers of two >= 16), so one scalar buffer descriptor
  // covers exactly the valid keys and keys past the split end or on an
  // invalid page read as zero.  Loads go to registers one tile ahead and are
  // stored to LDS after the tile's compute.
  const int pshift = a.page_shift;
  const int pmask = (1 << pshift) - 1;
  const int64_t bt_row = static_cast<int64_t>(b) * a.max_pages;
  const int64_t head_stride = static_cast<int64_t>(a.page) * D;  // elements per (page, head)
  constexpr int kRowsPerLoad = SRT_WAVE / CPR;                    // 4 (d=128) or 8 (d=64)
  constexpr int kLoadsPerWave = kSubRows / kRowsPerLoad;          // per tile, per tensor
  static_assert(kLoadsPerWave >= 1 && kSubRows % kRowsPerLoad == 0, "staging shape");
  const int st_row = kSubRows * w + lane / CPR;  // tile row of this lane's first chunk
  const int gl_off = ((lane / CPR) * D + (lane % CPR) * 8) * 2;
  const int k_st = st_row * Sh::KSTRIDE + (lane % CPR) * 16;
  const int v_st = st_row * Sh::VSTRIDE + (lane % CPR) * 16;

  // Page ids of this wave's sub-block of every tile of the split, one tile
  // per lane and register (a split has 128 tiles), fetched once; the loop
  // reads them with v_readlane and touches no block-table memory.
  static_assert(kChunk / kTile == 2 * SRT_WAVE, "two registers of page ids per split (of at most kChunk keys)");
  int pg_lane[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int p0 = k_begin + kTile * (SRT_WAVE * j + lane) + kSubRows * w;
    pg_lane[j] = p0 < k_end ? a.bt[bt_row + (p0 >> pshift)] : -1;
  }
  auto page_of = [&](int it) {
    if (it >= ntiles) return -1;
    return it < SRT_WAVE ? __builtin_amdgcn_readlane(pg_lane[0], it)
                         : __builtin_amdgcn_readlane(pg_lane[1], it - SRT_WAVE);
  };
  uint4 kreg[kLoadsPerWave], vreg[kLoadsPerWave];
  auto load_sub = [&](const uint16_t* base, int t0, int pg, uint4 (&r)[kLoadsPerWave]) {
    const int p0 = t0 + kSubRows * w;
    const bool ok = pg >= 0 && pg < a.num_pages && p0 < k_end;
    const int nbytes = ok ? min(kSubRows, k_end - p0) * D * 2 : 0;
    const int64_t off = ok ? (static_cast<int64_t>(pg) * a.Hkv + g) * head_stride + (p0 & pmask) * D : 0;
    buffer_load16<kLoadsPerWave, kRowsPerLoad * D * 2>(base + off, nbytes, gl_off, r);
  };
  auto store_k = [&](uint8_t* Kb) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) *reinterpret_cast<uint4*>(Kb + k_st + j * kRowsPerLoad * Sh::KSTRIDE) = kreg[j];
  };
  auto store_v = [&](uint8_t* Vb) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) *reinterpret_cast<uint4*>(Vb + v_st + j * kRowsPerLoad * Sh::VSTRIDE) = vreg[j];
  };

  // ---- MFMA phases -------------------------------------------------------
  // K operand (A of S^T): lane reads key l32 (+32 kb), head dims
  // 16 ks + 8 h .. +7.
  const int k_rd = l32 * Sh::KSTRIDE + 16 * h;
  // V^T operand (A of O^T) by transposing reads: in each 16-lane group G,
  // lane x addresses key 16 ks + 4 h + x/4 (+8 for the second half of the
  // contraction) and head dims (D/2)(G%2) + 16 db + 4 (x%4) .. +3.
  const int xg = lane % 16;
  const int k_vd = (4 * h + xg / 4) * Sh::VSTRIDE + ((CPR / 2) * ((lane / 16) & 1) + (xg % 4) / 2) * 16 + 8 * (xg & 1);

  // S^T[key][row] = q . k of one tile (raw fp32 dot products): two 32-key
  // blocks.
  auto qk = [&](const uint8_t* Kb, f32x16 (&sacc)[2]) {
    // All fragment reads are issued before the first MFMA so that one LDS
    // latency, not one per k-step, is exposed.
    bf16x8 kf[Sh::KS][2];
#pragma unroll
    for (int ks = 0; ks < Sh::KS; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        kf[ks][kb] = *reinterpret_cast<const bf16x8*>(Kb + k_rd + kb * 32 * Sh::KSTRIDE + ks * 32);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < Sh::KS; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks][kb], qf[ks], sacc[kb], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * Sh::KS, 0);  // DS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * Sh::KS, 0);  // then MFMAs
  };

  // Mask, online softmax with lazy rescale; returns P in bf16.  Lane holds
  // keys 32 kb + 8 (r/4) + 4 h + r%4 of its row in sacc[kb][r].
  auto softmax = [&](int t0, f32x16 (&sacc)[2], bf16x8 (&pb)[4], float mref0) {
    // Scores in log2 units relative to the reference: q.k * scale * log2(e)
    // - mref0, one fp32 fused multiply-add per score (masked scores are set
    // to -inf afterwards, so any finite scale is safe).
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = __builtin_fmaf(sacc[kb][r], c_log2, -mref0);
    const bool need_mask = (t0 + kTile > si.L) || (t0 + kTile > k_end);
    if (need_mask) {
      // Visibility of keys t0 .. t0+63 for this lane's row as one 64-bit
      // window: bit x is set iff key t0 + x < k_end and it is a context key
      // or the tree position of an ancestor-or-self of the row's node.  (If
      // the split ends before the tree, bits of tree positions are cleared
      // by the k_end limit, so stale bitsets are never used.)
      const int lim = k_end - t0;
      uint64_t vis = lim >= 64 ? ~0ull : (lim <= 0 ? 0ull : (~0ull >> (64 - lim)));
      const int j0 = t0 - si.L;  // tree index of key t0
      if (j0 > -kTile) {
        uint64_t win;
        if (j0 >= 0) {
          const int wd = j0 >> 6, sh = j0 & 63;
          const uint64_t lo = wd < 4 ? anc[node][wd] : 0ull;
          const uint64_t hi = wd + 1 < 4 ? anc[node][wd + 1] : 0ull;
          win = sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
        } else {
          const int sh = -j0;  // 1..63 context keys lead the window
          win = (anc[node][0] << sh) | (~0ull >> (64 - sh));
        }
        vis &= win;
      }
      // lane half h holds keys 32 kb + 8 (r/4) + 4 h + r%4
      const uint64_t vh = vis >> (4 * h);
      const uint32_t v0 = static_cast<uint32_t>(vh), v1 = static_cast<uint32_t>(vh >> 32);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const uint32_t vw = kb ? v1 : v0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int x = 8 * (r / 4) + r % 4;
          sacc[kb][r] = ((vw >> x) & 1u) ? sacc[kb][r] : -INFINITY;
        }
      }
    }
    // Probabilities exp2(score - mref0 - dm), rounded to bf16 for the second
    // product (sacc holds score - mref0); returns this lane's sum of them
    // (its 32 keys of the row, two bf16 pairs per dot2, two accumulators).
    // Contraction index 8 h + e of k-step ks <-> key 16 ks + 8 (e/4) + 4 h + e%4.
    auto probs = [&](auto dm_c, float dm) {
      typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
      const bf16x2 one2 = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
      float ps[2] = {0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pb[ks][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(
              decltype(dm_c)::value ? sacc[ks / 2][8 * (ks % 2) + e] - dm : sacc[ks / 2][8 * (ks % 2) + e]));
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2 pr = {pb[ks][e], pb[ks][e + 1]};
          ps[ks & 1] = __builtin_amdgcn_fdot2_f32_bf16(pr, one2, ps[ks & 1], false);
        }
      }
      return ps[0] + ps[1];
    };
    // Fast path: exponentiate against the current reference without first
    // taking the row maximum.  If every rounded probability of the row is
    // below 2^kLazy (their sum is), no score exceeds the reference by kLazy,
    // so the reference would not be raised and these are the final values.
    // Otherwise (or while the reference is still -inf) the wave takes the
    // row maximum, raises the reference as needed and exponentiates again.
    float psum = probs(std::false_type(), 0.f);
    const bool fast = m != -INFINITY && psum < 256.f;  // 256 = 2^kLazy
    if (__ballot(!fast)) {
      // (maximum, not fmaxf: no NaN-quieting of every operand; scores are
      // finite or -inf)
      float mloc = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; r += 2)
          mloc = __builtin_elementwise_maximum(mloc, __builtin_elementwise_maximum(sacc[kb][r], sacc[kb][r + 1]));
      mloc = max_halves(mloc);
      const float ms = mloc + mref0;  // row max in log2 units
      const bool raise = ms > m + kLazy;
      if (__ballot(raise)) {
        const float mnew = raise ? ms : m;
        const float alpha = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mnew);
        l *= alpha;
#pragma unroll
        for (int db = 0; db < Sh::DB; ++db) o[db] *= alpha;
        m = mnew;
      }
      psum = probs(std::true_type(), (m == -INFINITY ? 0.f : m) - mref0);
    }
    l += psum;
  };

  // O^T[d][row] += V^T P^T.
  // V^T fragments of k-steps ks0, ks0+1 (two transposing reads per MFMA).
  typedef short i16x4v __attribute__((ext_vector_type(4)));
  auto v_read = [&](const uint8_t* Vb, int ks0, i16x4v (&vf)[2][Sh::DB][2]) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int db = 0; db < Sh::DB; ++db)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          vf[k2][db][hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) i16x4v*)(Vb + k_vd + (ks0 + k2) * 16 * Sh::VSTRIDE +
                                                          hh * 8 * Sh::VSTRIDE + db * 32));
  };
  auto pv = [&](const i16x4v (&vf)[2][Sh::DB][2], int ks0, const bf16x8 (&pb)[4]) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int db = 0; db < Sh::DB; ++db) {
        const bf16x8 va =
            __builtin_bit_cast(bf16x8, __builtin_shufflevector(vf[k2][db][0], vf[k2][db][1], 0, 1, 2, 3, 4, 5, 6, 7));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[ks0 + k2], o[db], 0, 0, 0);
      }
  };

  // ---- tile loop ---------------------------------------------------------
  // Iteration t: global loads of tile t+1 are issued to registers; the K
  // fragments of tile t are read from LDS and S = K Q^T runs; the V^T
  // fragments are read while softmax runs on the VALU; O += V^T P^T; then
  // tile t+1 is stored into the buffers tile t-1 left.  One barrier per tile.
  {
    const int pg0 = page_of(0);
    load_sub(a.k, k_begin, pg0, kreg);
    load_sub(a.v, k_begin, pg0, vreg);
    store_k(Ks);
    store_v(Vs);
  }
  __syncthreads();

  auto step = [&](int it, auto cur_c) {
    constexpr int cur = decltype(cur_c)::value;
    const int t0 = k_begin + it * kTile;
    const bool next = it + 1 < ntiles;
    if (next) {
      const int pg = page_of(it + 1);
      load_sub(a.k, t0 + kTile, pg, kreg);
      load_sub(a.v, t0 + kTile, pg, vreg);
    }
    if (wave_active) {
      f32x16 sacc[2];
      const float mref0 = m == -INFINITY ? 0.f : m;
      qk(Ks + cur * Sh::KTILE, sacc);
      // First half of the V^T fragments is read while softmax runs, the
      // second half while the first half's MFMAs run.
      i16x4v vf0[2][Sh::DB][2], vf1[2][Sh::DB][2];
      v_read(Vs + cur * Sh::VTILE, 0, vf0);
      bf16x8 pb[4];
      softmax(t0, sacc, pb, mref0);
      v_read(Vs + cur * Sh::VTILE, 2, vf1);
      pv(vf0, 0, pb);
      pv(vf1, 2, pb);
    }
    if (next) {
      store_k(Ks + (cur ^ 1) * Sh::KTILE);
      store_v(Vs + (cur ^ 1) * Sh::VTILE);
    }
    __syncthreads();
  };
  for (int it = 0; it < ntiles; it += 2) {
    step(it, std::integral_constant<int, 0>());
    if (it + 1 < ntiles) step(it + 1, std::integral_constant<int, 1>());
  }

  // Epilogue: lane holds row l32 and, for block db and quad q = r/4, head
  // dims (D/2)(q/2) + 16 db + 8 (q%2) + 4 h + 0..3.
  const float lt = sum_halves(l);
  if (!row_ok) return;
  const int RBR = a.RB * kRowsPerBlock;
  if (nsplit == 1) {
    const int hq = g * a.G + row % a.G;
    uint16_t* op = a.out + ((static_cast<int64_t>(b) * a.N + node) * a.Hq + hq) * D + 4 * h;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
    for (int db = 0; db < Sh::DB; ++db) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int d0 = (D / 2) * (q / 2) + 16 * db + 8 * (q % 2);
        const uint32_t x0 =
            to_bf16_bits(o[db][4 * q] * inv) | (uint32_t(to_bf16_bits(o[db][4 * q + 1] * inv)) << 16);
        const uint32_t x1 =
            to_bf16_bits(o[db][4 * q + 2] * inv) | (uint32_t(to_bf16_bits(o[db][4 * q + 3] * inv)) << 16);
        *reinterpret_cast<uint2*>(op + d0) = make_uint2(x0, x1);
      }
    }
  } else {
    const int64_t prow = ((static_cast<int64_t>(b) * a.Hkv + g) * a.S + s) * RBR + row;
    float* po = a.part_o + prow * D + 4 * h;
#pragma unroll
    for (int db = 0; db < Sh::DB; ++db) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int d0 = (D / 2) * (q / 2) + 16 * db + 8 * (q % 2);
        *reinterpret_cast<f32x4*>(po + d0) = f32x4{o[db][4 * q], o[db][4 * q + 1], o[db][4 * q + 2], o[db][4 * q + 3]};
      }
    }
    if (h == 0) {
      a.part_ml[2 * prow] = m;
      a.part_ml[2 * prow + 1] = lt;
    }
  }
  };

  for (;;) {
    if (tid == 0) s_item = atomicAdd(a.plan + 1, 1);
    __syncthreads();
    const int idx = s_item;
    if (idx >= n_items) break;
    const int b = a.plan[kPlanHeader + 2 * idx];
    const int packed = a.plan[kPlanHeader + 2 * idx + 1];
    run_item(b, packed & 0xff, (packed >> 8) & 0xfff, packed >> 20);
    __syncthreads();  // LDS and s_item are reused by the next item
  }
}

// Builds the work list: one item per (sequence, KV head, split, row block)
// that has work, counting-sorted by decreasing (tiles, active waves of the
// first row block).  The row blocks of one (sequence, KV head, split) are
// listed next to each other, so workgroups that take them start at about
// the same time and the second stream of the same K/V tiles is served by
// the caches.  One workgroup; also resets the hand-out counter.
__global__ __launch_bounds__(1024) void tree_attn_plan_kernel(AttnArgs a) {
  __shared__ int32_t cnt[kPlanKeys], off[kPlanKeys], fill[kPlanKeys];
  __shared__ int32_t wsum[1024 / SRT_WAVE];
  const int tid = threadIdx.x;
  for (int k = tid; k < kPlanKeys; k += 1024) {
    cnt[k] = 0;
    fill[k] = 0;
  }
  __syncthreads();
  // Visits the item classes of sequence b: f(key, first split, splits,
  // row blocks).
  auto classes = [&](int b, auto&& f) {
    const SeqInfo si = seq_info(a, b);
    const int rows = si.n * a.G;
    const int rbs = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
    const int full = si.total / a.chunk;
    const int tail = si.total - full * a.chunk;
    const int waves = min(kWaves, (rows + kRowsPerWave - 1) / kRowsPerWave);
    if (full > 0) f(plan_key(a.chunk / kTile, waves), 0, full, rbs);
    if (tail > 0) f(plan_key((tail + kTile - 1) / kTile, waves), full, 1, rbs);
  };
  for (int b = tid; b < a.B; b += 1024)
    classes(b, [&](int key, int, int ns, int rbs) { atomicAdd(&cnt[key], ns * a.Hkv * rbs); });
  __syncthreads();
  // Exclusive prefix sum of the class counts (one class per thread).
  static_assert(kPlanKeys <= 1024, "one class per thread");
  const int lane = tid % SRT_WAVE, wv = tid / SRT_WAVE;
  const int mine = tid < kPlanKeys ? cnt[tid] : 0;
  int incl = mine;
#pragma unroll
  for (int d = 1; d < SRT_WAVE; d <<= 1) {
    const int y = __shfl_up(incl, d, SRT_WAVE);
    if (lane >= d) incl += y;
  }
  if (lane == SRT_WAVE - 1) wsum[wv] = incl;
  __syncthreads();
  int before = 0;
  for (int j = 0; j < wv; ++j) before += wsum[j];
  if (tid < kPlanKeys) off[tid] = before + incl - mine;
  __shared__ int32_t ncomb;
  if (tid == 1023) {
    a.plan[0] = before + incl;  // all classes
    a.plan[1] = 0;
    ncomb = 0;
  }
  __syncthreads();
  // combine units: 8-row groups of every (sequence, KV head) with several splits
  for (int b = tid; b < a.B; b += 1024) {
    const SeqInfo si = seq_info(a, b);
    if (si.total <= a.chunk) continue;
    const int groups = (si.n * a.G + 7) / 8;
    int u = atomicAdd(&ncomb, groups * a.Hkv);
    for (int g = 0; g < a.Hkv; ++g)
      for (int r8 = 0; r8 < groups; ++r8, ++u) {
        a.plan[a.combine_at + u] = b | (g << 16);
        a.plan[a.combine_at + a.max_units + u] = r8;
      }
  }
  __syncthreads();
  if (tid == 0) a.plan[2] = ncomb;
  for (int b = tid; b < a.B; b += 1024)
    classes(b, [&](int key, int s0, int ns, int rbs) {
      int pos = off[key] + atomicAdd(&fill[key], ns * a.Hkv * rbs);
      for (int s = s0; s < s0 + ns; ++s)
        for (int g = 0; g < a.Hkv; ++g)
          for (int rb = 0; rb < rbs; ++rb, ++pos) {
            a.plan[kPlanHeader + 2 * pos] = b;
            a.plan[kPlanHeader + 2 * pos + 1] = g | (s << 8) | (rb << 20);
          }
    });
}

// Merges the split partials of sequences that needed more than one split:
// out = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s with M = max_s m_s (m
// in log2 units).  Persistent workgroups stride over the combine units of
// the plan; a unit is 8 rows, one thread per row and four head dims, so
// partial reads are 16-byte coalesced.  The splits are folded with a
// running maximum, so the loads of different splits are independent.
template <int D>
__global__ __launch_bounds__(256) void tree_attn_combine_kernel(AttnArgs a) {
  constexpr int Q = D / 4;
  constexpr int kRowsPerUnit = 256 / Q;
  static_assert(kRowsPerUnit * Q == 256 && kRowsPerUnit >= 8, "unit shape");
  const int n_units = a.plan[2];
  const int RBR = a.RB * kRowsPerBlock;
  for (int u = blockIdx.x; u < n_units; u += gridDim.x) {
    const int bg = a.plan[a.combine_at + u];
    const int b = bg & 0xffff, g = bg >> 16;
    const SeqInfo si = seq_info(a, b);
    const int nsplit = (si.total + a.chunk - 1) / a.chunk;
    const int rows = si.n * a.G;
    for (int sub = threadIdx.x; sub < 8 * Q; sub += 256) {
      const int r = a.plan[a.combine_at + a.max_units + u] * 8 + sub / Q, q = sub % Q;
      if (r >= rows) continue;
      const int64_t base = (static_cast<int64_t>(b) * a.Hkv + g) * a.S * RBR + r;
      float M = -INFINITY, den = 0.f;
      f32x4 num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
      for (int s = 0; s < nsplit; ++s) {
        const int64_t prow = base + static_cast<int64_t>(s) * RBR;
        const float ms = a.part_ml[2 * prow];
        const float ls = a.part_ml[2 * prow + 1];
        const f32x4 os = *reinterpret_cast<const f32x4*>(a.part_o + prow * D + 4 * q);
        if (ms == -INFINITY) continue;
        const float mn = fmaxf(M, ms);
        const float c_old = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - mn);
        const float c_new = __builtin_amdgcn_exp2f(ms - mn);
        den = den * c_old + ls * c_new;
        num = num * c_old + os * c_new;
        M = mn;
      }
      const float inv = den > 0.f ? 1.f / den : 0.f;
      const int node = r / a.G, h = g * a.G + r % a.G;
      uint16_t* op = a.out + ((static_cast<int64_t>(b) * a.N + node) * a.Hq + h) * D + 4 * q;
      const uint32_t x0 = to_bf16_bits(num[0] * inv) | (uint32_t(to_bf16_bits(num[1] * inv)) << 16);
      const uint32_t x1 = to_bf16_bits(num[2] * inv) | (uint32_t(to_bf16_bits(num[3] * inv)) << 16);
      *reinterpret_cast<uint2*>(op) = make_uint2(x0, x1);
    }
  }
}

// Keys per split: the largest power of two in [kMinChunk, kChunk] that still
// gives B * Hkv * RB * (capacity / chunk) >= 512 work items (two per CU of
// the 256; RB row blocks per sequence and KV head), so that small batches
// of long contexts are split over enough workgroups; large batches and wide
// trees keep 8192-key splits (fewer partial results).
int chunk_for(int32_t B, int32_t Hkv, int64_t RB, int32_t page, int32_t max_pages) {
  const int64_t cap = static_cast<int64_t>(page) * max_pages;
  int chunk = kChunk;
  while (chunk > kMinChunk && static_cast<int64_t>(B) * Hkv * RB * ((cap + chunk - 1) / chunk) < 512) chunk /= 2;
  return chunk;
}

int splits_for(int32_t page, int32_t max_pages, int chunk) {
  const int64_t cap = static_cast<int64_t>(page) * max_pages;
  return static_cast<int>((cap + chunk - 1) / chunk);
}

// Combine units (8-row groups) needed at most.
int64_t max_combine_units(int32_t B, int32_t N, int32_t G, int32_t Hkv) {
  return static_cast<int64_t>(B) * Hkv * ((static_cast<int64_t>(N) * G + 7) / 8);
}

// Bytes of the work lists for at most `items` items and `units` combine
// units, rounded to 256.
size_t plan_bytes(int64_t items, int64_t units) {
  return ((kPlanHeader + 2 * items + 2 * units) * sizeof(int32_t) + 255) / 256 * 256;
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

}  // namespace

extern "C" size_t srt_tree_attn_scratch_bytes(int32_t B, int32_t N, int32_t Hq, int32_t Hkv, int32_t d, int32_t page,
                                              int32_t max_pages) {
  if (B < 0 || N < 1 || N > kMaxN || Hq < 1 || Hkv < 1 || Hq % Hkv || page < 1 || max_pages < 1) return 0;
  const int G = Hq / Hkv;
  const int64_t RB = (N * G + kRowsPerBlock - 1) / kRowsPerBlock;
  const int S = splits_for(page, max_pages, chunk_for(B, Hkv, RB, page, max_pages));
  const size_t plan = plan_bytes(static_cast<int64_t>(B) * Hkv * S * RB, max_combine_units(B, N, G, Hkv));
  if (S <= 1) return plan;
  return plan + static_cast<size_t>(B) * Hkv * S * RB * kRowsPerBlock * (d + 2) * sizeof(float);
}

extern "C" int srt_tree_attn(int32_t B, int32_t N, int32_t Hq, int32_t Hkv, int32_t d, int32_t page,
                             int32_t max_pages, int64_t num_pages, const uint16_t* q, const uint16_t* k_cache,
                             const uint16_t* v_cache, const int32_t* block_table, const int32_t* ctx_len,
                             const int32_t* tree_parent, const int32_t* n_nodes, float scale, uint16_t* out,
                             void* scratch, size_t scratch_bytes, void* stream) {
  if (B < 0 || N < 1 || N > kMaxN || Hq < 1 || Hkv < 1 || Hq % Hkv || page < 1 || max_pages < 1 || num_pages < 1)
    return SRT_ERR_INVALID;
  if (!std::isfinite(scale)) return SRT_ERR_INVALID;
  if (d != 64 && d != 128) return SRT_ERR_UNSUPPORTED;
  if (page < 16 || (page & (page - 1))) return SRT_ERR_UNSUPPORTED;
  // work-list packing: sequence < 65536, KV head < 256, split < 4096,
  // row block < 2048, combine units < 2^31
  const int chunk = chunk_for(B, Hkv, (N * (Hq / Hkv) + kRowsPerBlock - 1) / kRowsPerBlock, page, max_pages);
  if (B > 65535 || Hkv > 255 || splits_for(page, max_pages, chunk) > 4095 || (N * (Hq / Hkv)) / kRowsPerBlock > 2046 ||
      max_combine_units(B, N, Hq / Hkv, Hkv) > (int64_t(1) << 30))
    return SRT_ERR_UNSUPPORTED;
  if (B == 0) return SRT_OK;
  if (!q || !k_cache || !v_cache || !block_table || !ctx_len || !tree_parent || !n_nodes || !out)
    return SRT_ERR_INVALID;
  const size_t need = srt_tree_attn_scratch_bytes(B, N, Hq, Hkv, d, page, max_pages);
  if (!scratch || scratch_bytes < need) return SRT_ERR_CAPACITY;
  if (reinterpret_cast<uintptr_t>(scratch) % 256) return SRT_ERR_INVALID;

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
  a.chunk = chunk;
  a.S = splits_for(page, max_pages, chunk);
  a.RB = (N * a.G + kRowsPerBlock - 1) / kRowsPerBlock;
  const int64_t total = static_cast<int64_t>(B) * Hkv * a.S * a.RB;
  if (total > (int64_t(1) << 30)) return SRT_ERR_INVALID;
  a.total = static_cast<int32_t>(total);
  const int64_t RBR = static_cast<int64_t>(a.RB) * kRowsPerBlock;
  const int64_t units = max_combine_units(B, N, a.G, Hkv);
  const size_t pbytes = plan_bytes(total, units);
  a.plan = static_cast<int32_t*>(scratch);
  a.combine_at = kPlanHeader + 2 * total;
  a.max_units = static_cast<int32_t>(units);
  a.part_o = a.S > 1 ? reinterpret_cast<float*>(static_cast<uint8_t*>(scratch) + pbytes) : nullptr;
  a.part_ml = a.S > 1 ? a.part_o + static_cast<int64_t>(B) * Hkv * a.S * RBR * d : nullptr;

  const int cus = cu_count();
  if (cus <= 0) return SRT_ERR_HIP;
  const unsigned grid = static_cast<unsigned>(std::min<int64_t>(total, cus));
  hipStream_t s = as_stream(stream);
  tree_attn_plan_kernel<<<1, 1024, 0, s>>>(a);
  if (d == 128) {
    tree_attn_kernel<128><<<grid, kThreads, 0, s>>>(a);
  } else {
    tree_attn_kernel<64><<<grid, kThreads, 0, s>>>(a);
  }
  if (a.S > 1) {
    const unsigned cgrid = static_cast<unsigned>(std::min<int64_t>(units, 4 * cus));
    if (d == 128) {
      tree_attn_combine_kernel<128><<<cgrid, 256, 0, s>>>(a);
    } else {
      tree_attn_combine_kernel<64><<<cgrid, 256, 0, s>>>(a);
    }
  }
  return launch_status();
}
