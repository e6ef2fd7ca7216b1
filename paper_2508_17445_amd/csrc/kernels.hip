// gfx950 kernels of the segment-tree decode path: KV append (scatter into the
// pools), the VALU node-partial kernel, and the log-sum-exp combine.
//
// Node-partial attention (cascade schedule): for a work item -- a chunk of one
// node run's KV tiles and the query rows of a group of its descendant leaves
// (the nested sub-groups of TreePO Sec. 2.3) -- one 256-thread workgroup
// streams every KV tile once from HBM into LDS with 128-bit global->LDS loads,
// scores all query rows of the group against it, and writes per-row partials
// (O unnormalised, running max, sum) in fp32.  The combine merges, per leaf
// and query head, the partials of its chain (exact log-sum-exp algebra).
//
// Layouts: K pool [Hkv][blocks][64][D] (token rows), V pool
// [Hkv][blocks][2][D][32] (each 32-token half block transposed, so a d-row
// holds 32 consecutive tokens).  The decode kernels stream half blocks
// (32-token tiles), each one contiguous 8 KiB (D = 128) range per pool.
#include "kernels.h"

#include <math.h>

namespace treepo {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                         __builtin_bit_cast(bf16x2, b), c, false);
}

// Sum over the four lanes of a quad (DPP quad permutations xor 1, xor 2).
__device__ __forceinline__ float quad_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, true));
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, true));
  return x;
}

template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

// Reduce-scatter over the 8 lanes j = lane % 8 of a half row: lane j returns
// sum over the 8 lanes of x[j].  Butterfly with DPP: half-row mirror (j <-> 7-j),
// then quad swaps (j <-> j^2, j <-> j^1); each step keeps half of the rows.
__device__ __forceinline__ float reduce_scatter8(const float (&x)[8], int j) {
  const bool h4 = (j & 4) != 0, h2 = (j & 2) != 0, h1 = (j & 1) != 0;
  float k4[4], k2[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float send = h4 ? x[i] : x[4 + i];
    const float own = h4 ? x[4 + i] : x[i];
    k4[i] = own + dppf<0x141>(send);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float send = h2 ? k4[i] : k4[2 + i];
    const float own = h2 ? k4[2 + i] : k4[i];
    k2[i] = own + dppf<0x4E>(send);
  }
  const float send = h1 ? k2[0] : k2[1];
  const float own = h1 ? k2[1] : k2[0];
  return own + dppf<0xB1>(send);
}

__device__ __forceinline__ uint32_t f2bf_bits(float x) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(x)));
}
__device__ __forceinline__ float bf_bits2f(uint32_t b) { return __builtin_bit_cast(float, b << 16); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---- KV tile staging ----------------------------------------------------------
//
// A tile is 32 tokens: one half of a 64-token pool block.  LDS tile = K rows
// [32][D] then V^T rows [D][32], in 16-byte chunks with XOR swizzles that make
// the compute reads conflict free (per 8-lane LDS phase):
//   K: chunk c of token row r sits at position c ^ ((r & 3) | ((r >> 1) & 4));
//      the VALU reader takes 8 chunks of one row, the MFMA reader one chunk of
//      rows {R+0..3, R+8..11} -- both hit 8 distinct bank groups.
//   V: chunk c of d-row d sits at position c ^ ((d >> 1) & 3); both readers
//      take one chunk of 8 consecutive d-rows.
// Each wave moves whole 1 KiB LDS slots; the swizzle is applied on the global
// side (a lane picks which chunk of the same row it fetches), so each slot is
// still read from HBM in whole row segments.  kNBuf tile buffers per
// workgroup keep kDepth tiles in flight while one is consumed.  Depth 3
// (66.5 KB of LDS at D = 128) lets two workgroups share a CU; depth 2
// (50 KB) lets three.
#ifndef TREEPO_PIPE_DEPTH
#define TREEPO_PIPE_DEPTH 3
#endif
constexpr int kSub = 32;                   // tokens per tile
constexpr int kDepth = TREEPO_PIPE_DEPTH;  // tiles in flight while one is consumed
constexpr int kNBuf = kDepth + 1;          // LDS tile buffers per workgroup
constexpr int kWgsPerCu = kDepth == 3 ? 2 : 3;
static_assert(kDepth == 2 || kDepth == 3, "pipeline depth 2 or 3");

constexpr int kMaxItemTiles = 128;  // the planner keeps items at <= 128 tiles
constexpr int kItemInts = 12;       // work-item record size (int32)

template <int D>
struct TileSmem {
  static constexpr int kElems = kSub * D;   // K (or V^T) elements per tile
  uint16_t kv[kNBuf][2 * kElems];
  uint32_t pbuf[kWaves][4][16];  // per wave: token pair x (8 hi, 8 lo) packed P words
  int2 tile_meta[kMaxItemTiles];  // per tile of the item: (2 * block + half, valid tokens)
};

__device__ __forceinline__ int k_swz(int r) { return (r & 3) | ((r >> 1) & 4); }
__device__ __forceinline__ int v_swz(int d) { return (d >> 1) & 3; }

// One 16-byte global->LDS load per lane into the 1 KiB LDS slot at byte
// address `lds` (wave-uniform).  Issued as inline asm so that the compiler does
// not treat the in-flight LDS writes as aliasing every later LDS access (which
// would drain the prefetch); completion is tracked by hand with vmcnt waits
// before the barrier that publishes a tile.
// NT marks the load non-temporal: the line is not kept in the caches, which
// raises the streaming rate when every byte is read once per step.
template <bool NT>
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                 :: "v"(g), "s"(lds) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(g), "s"(lds) : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)p));
}

// Loads per lane per tile.
template <int D>
constexpr int dma_per_tile() { return D / 32; }

// Stages tile (block, half) of KV head g into the LDS buffer at byte address `dst`.
template <int D, bool NT>
__device__ __forceinline__ void dma_tile(const uint16_t* __restrict__ kpool,
                                         const uint16_t* __restrict__ vpool, int64_t num_blocks,
                                         int g, int block, int half, uint32_t dst, int wave, int lane) {
  constexpr int kKChunks = D / 8;   // 16-byte chunks per K row
  constexpr int kPerWave = D / 64;  // 1 KiB slots per wave for each of K and V
  const int64_t blk = static_cast<int64_t>(g) * num_blocks + block;
  const char* kg = reinterpret_cast<const char*>(kpool + (blk * kTile + half * kSub) * D);
  const char* vg = reinterpret_cast<const char*>(vpool + (blk * kTile + half * kSub) * D);
  const uint32_t vd = dst + kSub * D * 2;
#pragma unroll
  for (int j = 0; j < kPerWave; ++j) {
    const int slot = wave * kPerWave + j;
    const int c = slot * 64 + lane;
    const int row = c / kKChunks;
    const int col = (c % kKChunks) ^ k_swz(row);
    dma16<NT>(kg + row * (D * 2) + col * 16, __builtin_amdgcn_readfirstlane(dst + slot * 1024));
  }
#pragma unroll
  for (int j = 0; j < kPerWave; ++j) {
    const int slot = wave * kPerWave + j;
    const int c = slot * 64 + lane;
    const int row = c >> 2;
    const int col = (c & 3) ^ v_swz(row);
    dma16<NT>(vg + row * (kSub * 2) + col * 16, __builtin_amdgcn_readfirstlane(vd + slot * 1024));
  }
}

// Barrier after which this workgroup's global->LDS loads, except the newest N
// per lane, have landed; it also orders each wave's earlier LDS reads before
// any later overwrite (every wave waits for its own LDS reads before it).
template <int N>
__device__ __forceinline__ void barrier_tile_landed() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(N) : "memory");
}

// Waits for tile k (tiles up to k+kDepth may have been issued) and publishes it.
template <int D>
__device__ __forceinline__ void wait_tile(int k, int nt) {
  constexpr int kD = dma_per_tile<D>();
  const int ahead = nt - 1 - k;  // tiles issued after tile k (capped at kDepth - 1)
  if (kDepth == 3 && ahead >= 2)
    barrier_tile_landed<(kDepth - 1) * kD>();
  else if (ahead >= 1)
    barrier_tile_landed<kD>();
  else
    barrier_tile_landed<0>();
}

// Kernel arguments: the pointers are passed as separate __restrict__ kernel
// parameters so that uniform metadata reads become scalar loads.
struct Scalars {
  int64_t num_blocks;
  int32_t hq, hkv, group;
  float scale_log2;
};

#define TREEPO_PARTIAL_PARAMS                                                         \
  const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,            \
      const uint16_t *__restrict__ q, const int32_t *__restrict__ items,             \
      const int32_t *__restrict__ rowsets, const int32_t *__restrict__ tiles,        \
      float *__restrict__ part_o, float *__restrict__ part_ml, Scalars sc
#define TREEPO_PARTIAL_ARGS kpool, vpool, q, items, rowsets, tiles, part_o, part_ml, sc

// Issues the first min(kDepth, nt) tiles of an item (their sources ride in the
// item record, so this needs no further metadata load), then stages the
// item's per-tile (source, valid) pairs into LDS for the loop; the loop reads
// them from LDS instead of waiting on a scalar load every iteration.
template <int D, bool NT>
__device__ __forceinline__ void item_prologue(TREEPO_PARTIAL_PARAMS, const int32_t* it, int g, uint32_t buf0,
                                              TileSmem<D>& sm, int wave, int lane) {
  constexpr uint32_t kBufBytes = 2 * kSub * D * 2;
  const int tb = it[3], te = it[4];
#pragma unroll
  for (int p = 0; p < kDepth; ++p) {
    const int src = it[8 + p];
    if (src >= 0)
      dma_tile<D, NT>(kpool, vpool, sc.num_blocks, g, src >> 1, src & 1, buf0 + p * kBufBytes, wave, lane);
  }
  for (int t = threadIdx.x; t < te - tb; t += kThreads) {
    const int4 rec = reinterpret_cast<const int4*>(tiles)[tb + t];
    sm.tile_meta[t] = make_int2(2 * rec.x + (rec.z & 1), rec.w);
  }
}

// After tile k is published: prefetch tile k+kDepth into the buffer tile k-1
// used (buffer index `nb`, i.e. (k + kDepth) mod kNBuf).
template <int D, bool NT>
__device__ __forceinline__ void dma_ahead(TREEPO_PARTIAL_PARAMS, int nt, int k, int nb, int g, uint32_t buf0,
                                          const TileSmem<D>& sm, int wave, int lane) {
  constexpr uint32_t kBufBytes = 2 * kSub * D * 2;
  if (k + kDepth < nt) {
    const int src = __builtin_amdgcn_readfirstlane(sm.tile_meta[k + kDepth].x);
    dma_tile<D, NT>(kpool, vpool, sc.num_blocks, g, src >> 1, src & 1, buf0 + nb * kBufBytes, wave, lane);
  }
}

// ---- VALU node-partial ----------------------------------------------------------
//
// M query rows (M <= 8) per workgroup.  Wave w takes tokens [8w, 8w+8) of
// every tile and keeps its own online-softmax state; the four states are
// merged at the end.
//   QK: lane (t = lane/8, j = lane%8) owns token 8w+t and the K chunks j, j+8
//       of its row; q rows sit in registers in the same chunk order.  The
//       partial dot products (v_dot2 bf16 -> fp32) of all rows are combined by
//       a DPP reduce-scatter, after which lane j holds row j's score, so the
//       softmax work is done once per (token, row).
//   P : split into two bf16 terms, hi = bf16(p) and lo = bf16(p - hi), so the
//       weights keep about 16 significant bits (a single bf16 P can be off by
//       2^-8 relative, too much for short, peaked chains).  Token pairs are
//       packed into 32-bit words and staged in a per-wave LDS slot.
//   PV: lane i owns d = i (+64); V^T words hold two consecutive tokens of one
//       d, matching the packed P pairs, so each v_dot2 does two tokens (one
//       v_dot2 for hi and one for lo).
template <int D, int M, bool NT>
__device__ __forceinline__ void valu_item(TREEPO_PARTIAL_PARAMS, const int32_t* it, int g,
                                          TileSmem<D>& sm) {
  constexpr int kKC = D / 64;  // K chunks per lane in QK
  constexpr int kKW = 4 * kKC; // K words per lane in QK
  constexpr int kDD = D / 64;  // d values per lane in PV
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = lane >> 3;
  const int j = lane & 7;
  const int rowset = it[1], tb = it[3], te = it[4], pbase = it[5], rows = it[6];
  const int G = sc.group;
  const int nt = te - tb;
  const uint32_t buf0 = lds_addr(sm.kv[0]);
  item_prologue<D, NT>(TREEPO_PARTIAL_ARGS, it, g, buf0, sm, wave, lane);

  uint32_t qr[M][kKW];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int leaf = rowsets[rowset + m / G];
    const int head = g * G + m % G;
    const uint4* qp = reinterpret_cast<const uint4*>(q + (static_cast<int64_t>(leaf) * sc.hq + head) * D);
#pragma unroll
    for (int i = 0; i < kKC; ++i) {
      const uint4 v = qp[j + 8 * i];
      qr[m][4 * i + 0] = v.x;
      qr[m][4 * i + 1] = v.y;
      qr[m][4 * i + 2] = v.z;
      qr[m][4 * i + 3] = v.w;
    }
  }
  // Make the query loads complete here, outside the tile loop: the compiler
  // does not see the asm tile loads, and a wait for q inside the loop would
  // also drain the prefetch.
#pragma unroll
  for (int m = 0; m < M; ++m)
#pragma unroll
    for (int w = 0; w < kKW; ++w) asm volatile("" ::"v"(qr[m][w]));

  // per lane: reference max and weight sum of row j (lanes with equal j agree
  // on the reference; each sums the weights of its own token slot)
  float m_ref = -INFINITY, l_sum = 0.f;
  float acc[M][kDD];
#pragma unroll
  for (int m = 0; m < M; ++m)
#pragma unroll
    for (int dd = 0; dd < kDD; ++dd) acc[m][dd] = 0.f;

  for (int k = 0, cb = 0, nb = kDepth; k < nt; ++k, cb = cb == kNBuf - 1 ? 0 : cb + 1,
                                             nb = nb == kNBuf - 1 ? 0 : nb + 1) {
    wait_tile<D>(k, nt);  // also publishes the tile metadata staged in the prologue
    const int valid = __builtin_amdgcn_readfirstlane(sm.tile_meta[k].y);
    dma_ahead<D, NT>(TREEPO_PARTIAL_ARGS, nt, k, nb, g, buf0, sm, wave, lane);
    const char* kt = reinterpret_cast<const char*>(sm.kv[cb]);
    const char* vt = kt + kSub * D * 2;

    // ---- scores: lane j ends with row j's score of token 8w+t
    const int row = wave * 8 + t;
    uint32_t kr[kKW];
#pragma unroll
    for (int i = 0; i < kKC; ++i) {
      const int c = j + 8 * i;
      const uint4 v = *reinterpret_cast<const uint4*>(kt + row * (D * 2) + ((c ^ k_swz(row)) << 4));
      kr[4 * i + 0] = v.x;
      kr[4 * i + 1] = v.y;
      kr[4 * i + 2] = v.z;
      kr[4 * i + 3] = v.w;
    }
    float part[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      float x = 0.f;
      if (m < M) {
#pragma unroll
        for (int w = 0; w < kKW; ++w) x = dot2(qr[m][w], kr[w], x);
      }
      part[m] = x;
    }
    const float sc_j = reduce_scatter8(part, j);
    const float s = (row < valid && j < M) ? sc_j * sc.scale_log2 : -INFINITY;

    // ---- online softmax.  m_ref is a per-row reference, not necessarily the
    // exact running max: the weights are 2^(s - m_ref) and the result does not
    // depend on the reference.  Only when a score exceeds it by more than 2^8
    // (always on the first tile) are the exact tile maxima reduced across the
    // wave and the state rescaled.
    if (__builtin_amdgcn_ballot_w64(s > m_ref + 8.f) != 0) {
      float mx = s;
      mx = fmaxf(mx, __shfl_xor(mx, 8));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m_ref, mx);
      const float alpha = mn == -INFINITY ? 1.f : fast_exp2(m_ref - mn);
      m_ref = mn;
      l_sum *= alpha;
#pragma unroll
      for (int m = 0; m < M; ++m) {
        // row m's factor from lane m (token slot 0, j = m)
        const float am = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), m));
#pragma unroll
        for (int dd = 0; dd < kDD; ++dd) acc[m][dd] *= am;
      }
    }
    const float p = s == -INFINITY ? 0.f : fast_exp2(s - m_ref);
    const uint32_t pb = f2bf_bits(p);
    const uint32_t pl = f2bf_bits(p - bf_bits2f(pb));
    l_sum += bf_bits2f(pb) + bf_bits2f(pl);
    // token t-1 sits 8 lanes down in the same row of 16 lanes
    const uint32_t both = pb | (pl << 16);
    const uint32_t prev = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(0, static_cast<int>(both), 0x118, 0xF, 0xF, false));
    if ((t & 1) == 1 && j < M) {
      sm.pbuf[wave][t >> 1][j] = (prev & 0xFFFFu) | (both << 16);
      sm.pbuf[wave][t >> 1][8 + j] = (prev >> 16) | (both & 0xFFFF0000u);
    }

    // ---- P V
    uint32_t vw[kDD][4];
#pragma unroll
    for (int dd = 0; dd < kDD; ++dd) {
      const int d = lane + 64 * dd;
      const uint4 v = *reinterpret_cast<const uint4*>(vt + d * (kSub * 2) + ((wave ^ v_swz(d)) << 4));
      vw[dd][0] = v.x;
      vw[dd][1] = v.y;
      vw[dd][2] = v.z;
      vw[dd][3] = v.w;
    }
    if (valid < kSub) {
      // tokens past the node's length may hold anything; P is 0 there, and the
      // V halves are cleared so that 0 * garbage cannot produce NaN
#pragma unroll
      for (int tp = 0; tp < 4; ++tp) {
        const int tk = wave * 8 + 2 * tp;
        const uint32_t msk = tk >= valid ? 0u : (tk + 1 >= valid ? 0xFFFFu : 0xFFFFFFFFu);
#pragma unroll
        for (int dd = 0; dd < kDD; ++dd) vw[dd][tp] &= msk;
      }
    }
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      const uint4 p0 = *reinterpret_cast<const uint4*>(&sm.pbuf[wave][tp][0]);
      const uint4 p1 = *reinterpret_cast<const uint4*>(&sm.pbuf[wave][tp][4]);
      const uint4 p2 = *reinterpret_cast<const uint4*>(&sm.pbuf[wave][tp][8]);
      const uint4 p3 = *reinterpret_cast<const uint4*>(&sm.pbuf[wave][tp][12]);
      const uint32_t pw[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
      const uint32_t pwl[8] = {p2.x, p2.y, p2.z, p2.w, p3.x, p3.y, p3.z, p3.w};
#pragma unroll
      for (int m = 0; m < M; ++m)
#pragma unroll
        for (int dd = 0; dd < kDD; ++dd) acc[m][dd] = dot2(pwl[m], vw[dd][tp], dot2(pw[m], vw[dd][tp], acc[m][dd]));
    }
  }
  __syncthreads();

  // ---- merge the four waves' states and write the partial rows
  float l = l_sum;
  l += __shfl_xor(l, 8);
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  float* oacc = reinterpret_cast<float*>(sm.kv);  // [waves][M][D]
  float* mlb = oacc + kWaves * M * D;             // [waves][M][2]
#pragma unroll
  for (int m = 0; m < M; ++m)
#pragma unroll
    for (int dd = 0; dd < kDD; ++dd) oacc[(wave * M + m) * D + lane + 64 * dd] = acc[m][dd];
  if (t == 0 && j < M) {
    mlb[(wave * M + j) * 2 + 0] = m_ref;
    mlb[(wave * M + j) * 2 + 1] = l;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < M * D; idx += kThreads) {
    const int m = idx / D;
    const int d = idx % D;
    float mstar = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mstar = fmaxf(mstar, mlb[(w * M + m) * 2]);
    float o = 0.f, lt = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = mlb[(w * M + m) * 2];
      if (mw != -INFINITY) {
        const float f = fast_exp2(mw - mstar);
        o += f * oacc[(w * M + m) * D + d];
        lt += f * mlb[(w * M + m) * 2 + 1];
      }
    }
    const int64_t slot = static_cast<int64_t>(pbase) + static_cast<int64_t>(g) * rows + m;
    part_o[slot * D + d] = o;
    if (d == 0) {
      part_ml[slot * 2 + 0] = mstar;
      part_ml[slot * 2 + 1] = lt;
    }
  }
}

// ---- MFMA node-partial ------------------------------------------------------------
//
// For shared nodes whose stacked query rows (descendant leaves x GQA group)
// form dense tiles.  Rows are cut into 16-row blocks; wave w owns blocks
// w, w+4 (NRB per wave) and keeps their online-softmax state; all four waves
// read every KV tile from LDS.  Items hold at most 128 rows (two row blocks
// per wave) so that the K and V operands read from LDS are reused across a
// wave's row blocks without spilling registers.
//   QK: S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (A = 16 K rows, B = Q^T).
//       The K rows of token block b (0, 1) are read in the order
//       tau(b, r) = 8(r/4) + 4b + r%4, so that each lane's four outputs of the
//       two blocks are the eight consecutive tokens 8(lane/16) + 0..7 --
//       exactly the B operand layout of the PV product, so P never leaves
//       registers.
//   P : split into hi = bf16(p) and lo = bf16(p - hi) (about 16 significant
//       bits for the weights).
//   PV: O^T = V^T P_hi^T + V^T P_lo^T (A = 16 d-rows of the transposed V
//       tile, B = P^T).
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

__device__ __forceinline__ int tau(int b, int r) { return 8 * (r >> 2) + 4 * b + (r & 3); }

template <int D, int NRB, bool NT>
__device__ __forceinline__ void mfma_item(TREEPO_PARTIAL_PARAMS, const int32_t* it, int g, TileSmem<D>& sm) {
  constexpr int kKS = D / 32;  // QK k-steps
  constexpr int kDB = D / 16;  // PV output d-blocks
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int a = lane >> 4;      // lane group
  const int r16 = lane & 15;    // row within a 16-row block / output column
  const int rowset = it[1], tb = it[3], te = it[4], pbase = it[5], rows = it[6];
  const int G = sc.group;
  const int nt = te - tb;
  const uint32_t buf0 = lds_addr(sm.kv[0]);
  item_prologue<D, NT>(TREEPO_PARTIAL_ARGS, it, g, buf0, sm, wave, lane);

  // Q^T operands: lane holds row m = 16 rb + r16, d chunk 4 ks + a
  uint4 qb[NRB][kKS];
#pragma unroll
  for (int i = 0; i < NRB; ++i) {
    const int m = 16 * (wave + 4 * i) + r16;
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) qb[i][ks] = make_uint4(0, 0, 0, 0);
    if (m < rows) {
      const int leaf = rowsets[rowset + m / G];
      const int head = g * G + m % G;
      const uint4* qp = reinterpret_cast<const uint4*>(q + (static_cast<int64_t>(leaf) * sc.hq + head) * D);
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) qb[i][ks] = qp[4 * ks + a];
    }
  }
#pragma unroll
  for (int i = 0; i < NRB; ++i)
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) asm volatile("" ::"v"(qb[i][ks].x), "v"(qb[i][ks].y), "v"(qb[i][ks].z), "v"(qb[i][ks].w));

  const int nrb_total = (rows + 15) >> 4;
  const int my_rb = nrb_total > wave ? (nrb_total - wave + 3) >> 2 : 0;  // row blocks of this wave (<= NRB)

  f32x4 acc[NRB][kDB];
  float m_run[NRB], l_run[NRB];
#pragma unroll
  for (int i = 0; i < NRB; ++i) {
    m_run[i] = -INFINITY;
    l_run[i] = 0.f;
#pragma unroll
    for (int db = 0; db < kDB; ++db) acc[i][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int k = 0, cb = 0, nb = kDepth; k < nt; ++k, cb = cb == kNBuf - 1 ? 0 : cb + 1,
                                             nb = nb == kNBuf - 1 ? 0 : nb + 1) {
    wait_tile<D>(k, nt);
    const int valid = __builtin_amdgcn_readfirstlane(sm.tile_meta[k].y);
    dma_ahead<D, NT>(TREEPO_PARTIAL_ARGS, nt, k, nb, g, buf0, sm, wave, lane);
    const char* kt = reinterpret_cast<const char*>(sm.kv[cb]);
    const char* vt = kt + kSub * D * 2;
    if (my_rb > 0) {
      // ---- S^T = K Q^T for the wave's row blocks
      f32x4 S[NRB][2];
#pragma unroll
      for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int b = 0; b < 2; ++b) S[i][b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int tok = tau(b, r16);
          const int c = 4 * ks + a;
          const uint4 ka = *reinterpret_cast<const uint4*>(kt + tok * (D * 2) + ((c ^ k_swz(tok)) << 4));
#pragma unroll
          for (int i = 0; i < NRB; ++i)
            if (i < my_rb) S[i][b] = mfma16(ka, qb[i][ks], S[i][b]);
        }
      }
      // ---- online softmax; lane holds row r16, tokens 8a + 4b + e
      uint4 P[NRB], PL[NRB];
#pragma unroll
      for (int i = 0; i < NRB; ++i) {
        if (i >= my_rb) continue;
        float mx = -INFINITY;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int tok = 8 * a + 4 * b + e;
            const float x = tok < valid ? S[i][b][e] * sc.scale_log2 : -INFINITY;
            S[i][b][e] = x;
            mx = fmaxf(mx, x);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m_run[i], mx);
        const float alpha = mn == -INFINITY ? 1.f : fast_exp2(m_run[i] - mn);
        m_run[i] = mn;
        float ls = 0.f;
        uint32_t pw[4], pwl[4];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int e = 0; e < 4; e += 2) {
            const float x0 = S[i][b][e], x1 = S[i][b][e + 1];
            const float f0 = x0 == -INFINITY ? 0.f : fast_exp2(x0 - mn);
            const float f1 = x1 == -INFINITY ? 0.f : fast_exp2(x1 - mn);
            const uint32_t p0 = f2bf_bits(f0), p1 = f2bf_bits(f1);
            const uint32_t q0 = f2bf_bits(f0 - bf_bits2f(p0)), q1 = f2bf_bits(f1 - bf_bits2f(p1));
            ls += (bf_bits2f(p0) + bf_bits2f(q0)) + (bf_bits2f(p1) + bf_bits2f(q1));
            pw[2 * b + (e >> 1)] = p0 | (p1 << 16);
            pwl[2 * b + (e >> 1)] = q0 | (q1 << 16);
          }
        P[i] = make_uint4(pw[0], pw[1], pw[2], pw[3]);
        PL[i] = make_uint4(pwl[0], pwl[1], pwl[2], pwl[3]);
        l_run[i] = l_run[i] * alpha + ls;
#pragma unroll
        for (int db = 0; db < kDB; ++db) acc[i][db] *= alpha;
      }
      // ---- O^T += V^T P^T
#pragma unroll
      for (int db = 0; db < kDB; ++db) {
        const int d = 16 * db + r16;
        uint4 va = *reinterpret_cast<const uint4*>(vt + d * (kSub * 2) + ((a ^ v_swz(d)) << 4));
        if (valid < kSub) {
          // clear the V halves of tokens past the node's length (P is 0 there)
          uint32_t w[4] = {va.x, va.y, va.z, va.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int tk = 8 * a + 2 * e;
            w[e] &= tk >= valid ? 0u : (tk + 1 >= valid ? 0xFFFFu : 0xFFFFFFFFu);
          }
          va = make_uint4(w[0], w[1], w[2], w[3]);
        }
#pragma unroll
        for (int i = 0; i < NRB; ++i)
          if (i < my_rb) acc[i][db] = mfma16(va, PL[i], mfma16(va, P[i], acc[i][db]));
      }
    }
  }

  // ---- write the partial rows (each wave owns its row blocks)
#pragma unroll
  for (int i = 0; i < NRB; ++i) {
    if (i >= my_rb) continue;
    float l = l_run[i];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int m = 16 * (wave + 4 * i) + r16;
    if (m < rows) {
      const int64_t slot = static_cast<int64_t>(pbase) + static_cast<int64_t>(g) * rows + m;
#pragma unroll
      for (int db = 0; db < kDB; ++db)
        *reinterpret_cast<f32x4*>(part_o + slot * D + 16 * db + 4 * a) = acc[i][db];
      if (a == 0) {
        part_ml[slot * 2 + 0] = m_run[i];
        part_ml[slot * 2 + 1] = l;
      }
    }
  }
}

// ---- MFMA node-partial, token split ----------------------------------------------
//
// Items of at most 32 rows (one or two 16-row blocks: one leaf's GQA group, or
// a few leaves of a shared node).  Splitting rows over waves would leave most
// waves idle, so the tile is split by tokens instead: wave w takes row block
// w/2 and token block b = w%2 of every tile -- the 16 tokens tau(b, 0..15) --
// and keeps its own online-softmax state; the two waves of a row block merge
// at the end.
//   QK: as in mfma_item, for the wave's token block only (four MFMAs per row
//       block); each lane's four scores are the consecutive tokens
//       8(lane/16) + 4b + 0..3.
//   PV: O^T += V^T P^T with v_mfma_f32_16x16x16_bf16: the B operand (four
//       tokens x row) is exactly the lane's four scores, the A operand four
//       consecutive tokens of one V^T row (8 bytes).
//   Max: lazy reference per row: the running sum and O are rescaled only when a
//       score exceeds the reference by more than 2^8, so in steady state a tile
//       costs no cross-lane max and no rescale.
typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16k16(const uint2& a, const uint2& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a), __builtin_bit_cast(s16x4, b), c,
                                                   0, 0, 0);
}

constexpr float kLazyMaxSlack = 8.f;  // log2 units: weights stay <= 2^8 before a rescale

template <int D, bool NT>
__device__ __forceinline__ void mfma_split_item(TREEPO_PARTIAL_PARAMS, const int32_t* it, int g, TileSmem<D>& sm) {
  constexpr int kKS = D / 32;  // QK k-steps
  constexpr int kDB = D / 16;  // PV output d-blocks
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int a = lane >> 4;    // lane group
  const int r16 = lane & 15;  // row within the 16-row block
  const int rb = wave >> 1;   // row block
  const int tb = wave & 1;    // token block
  const int rowset = it[1], tbeg = it[3], tend = it[4], pbase = it[5], rows = it[6];
  const int G = sc.group;
  const int nt = tend - tbeg;
  const uint32_t buf0 = lds_addr(sm.kv[0]);
  item_prologue<D, NT>(TREEPO_PARTIAL_ARGS, it, g, buf0, sm, wave, lane);

  const bool active = 16 * rb < rows;  // wave-uniform
  const int m = 16 * rb + r16;         // this lane's query row
  uint4 qb[kKS];
#pragma unroll
  for (int ks = 0; ks < kKS; ++ks) qb[ks] = make_uint4(0, 0, 0, 0);
  if (m < rows) {
    const int leaf = rowsets[rowset + m / G];
    const int head = g * G + m % G;
    const uint4* qp = reinterpret_cast<const uint4*>(q + (static_cast<int64_t>(leaf) * sc.hq + head) * D);
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) qb[ks] = qp[4 * ks + a];
  }
#pragma unroll
  for (int ks = 0; ks < kKS; ++ks) asm volatile("" ::"v"(qb[ks].x), "v"(qb[ks].y), "v"(qb[ks].z), "v"(qb[ks].w));

  f32x4 acc[kDB];
#pragma unroll
  for (int db = 0; db < kDB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_ref = -INFINITY;  // per row (equal on the row's four lane groups)
  float l_sum = 0.f;        // per lane: this lane's tokens only
  const int tok0 = 8 * a + 4 * tb;  // first of the lane's four tokens

  for (int k = 0, cb = 0, nb = kDepth; k < nt; ++k, cb = cb == kNBuf - 1 ? 0 : cb + 1,
                                             nb = nb == kNBuf - 1 ? 0 : nb + 1) {
    wait_tile<D>(k, nt);
    const int valid = __builtin_amdgcn_readfirstlane(sm.tile_meta[k].y);
    dma_ahead<D, NT>(TREEPO_PARTIAL_ARGS, nt, k, nb, g, buf0, sm, wave, lane);
    if (!active) continue;
    const char* kt = reinterpret_cast<const char*>(sm.kv[cb]);
    const char* vt = kt + kSub * D * 2;
    // ---- S^T = K Q^T for the wave's 16 tokens
    f32x4 S = f32x4{0.f, 0.f, 0.f, 0.f};
    {
      const int tok = tau(tb, r16);
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
        const int c = 4 * ks + a;
        const uint4 ka = *reinterpret_cast<const uint4*>(kt + tok * (D * 2) + ((c ^ k_swz(tok)) << 4));
        S = mfma16(ka, qb[ks], S);
      }
    }
    // ---- scores (log2 units), masked past the node's length
    float x[4];
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = tok0 + e < valid ? S[e] * sc.scale_log2 : -INFINITY;
      mx = fmaxf(mx, x[e]);
    }
    if (__builtin_amdgcn_ballot_w64(mx > m_ref + kLazyMaxSlack) != 0) {
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m_ref, mx);
      const float alpha = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - mn);
      m_ref = mn;
      l_sum *= alpha;
#pragma unroll
      for (int db = 0; db < kDB; ++db) acc[db] *= alpha;
    }
    // ---- P = 2^(x - m_ref) as hi + lo bf16 terms
    uint32_t ph[2], pl[2];
#pragma unroll
    for (int e = 0; e < 4; e += 2) {
      const float f0 = x[e] == -INFINITY ? 0.f : fast_exp2(x[e] - m_ref);
      const float f1 = x[e + 1] == -INFINITY ? 0.f : fast_exp2(x[e + 1] - m_ref);
      const uint32_t h0 = f2bf_bits(f0), h1 = f2bf_bits(f1);
      const uint32_t q0 = f2bf_bits(f0 - bf_bits2f(h0)), q1 = f2bf_bits(f1 - bf_bits2f(h1));
      l_sum += (bf_bits2f(h0) + bf_bits2f(q0)) + (bf_bits2f(h1) + bf_bits2f(q1));
      ph[e >> 1] = h0 | (h1 << 16);
      pl[e >> 1] = q0 | (q1 << 16);
    }
    const uint2 P = make_uint2(ph[0], ph[1]), PL = make_uint2(pl[0], pl[1]);
    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      const int d = 16 * db + r16;
      uint2 va = *reinterpret_cast<const uint2*>(vt + d * (kSub * 2) + ((a ^ v_swz(d)) << 4) + tb * 8);
      if (valid < kSub) {
        // clear the V entries of tokens past the node's length (P is 0 there)
        va.x &= tok0 >= valid ? 0u : (tok0 + 1 >= valid ? 0xFFFFu : 0xFFFFFFFFu);
        va.y &= tok0 + 2 >= valid ? 0u : (tok0 + 3 >= valid ? 0xFFFFu : 0xFFFFFFFFu);
      }
      acc[db] = mfma16k16(va, PL, mfma16k16(va, P, acc[db]));
    }
  }

  // ---- merge the two token blocks of each row block, write the partial rows
  l_sum += __shfl_xor(l_sum, 16);
  l_sum += __shfl_xor(l_sum, 32);
  float* xs = reinterpret_cast<float*>(sm.kv[0]);  // [row block][2 + 4 kDB][64] floats
  constexpr int kFields = 2 + 4 * kDB;
  float* mine = xs + (rb * kFields) * 64 + lane;
  barrier_tile_landed<0>();  // every wave is done with the tile buffers
  if (active && tb == 1) {
    mine[0] = m_ref;
    mine[64] = l_sum;
#pragma unroll
    for (int db = 0; db < kDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) mine[(2 + 4 * db + i) * 64] = acc[db][i];
  }
  barrier_tile_landed<0>();
  if (active && tb == 0 && m < rows) {
    const float m1 = mine[0], l1 = mine[64];
    const float mn = fmaxf(m_ref, m1);
    const float a0 = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - mn);
    const float a1 = m1 == -INFINITY ? 0.f : fast_exp2(m1 - mn);
    const int64_t slot = static_cast<int64_t>(pbase) + static_cast<int64_t>(g) * rows + m;
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      f32x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = a0 * acc[db][i] + a1 * mine[(2 + 4 * db + i) * 64];
      *reinterpret_cast<f32x4*>(part_o + slot * D + 16 * db + 4 * a) = o;
    }
    if (a == 0) {
      part_ml[slot * 2 + 0] = mn;
      part_ml[slot * 2 + 1] = a0 * l_sum + a1 * l1;
    }
  }
}

// ---- the node-partial kernel ----------------------------------------------------
//
// One launch covers every work item of a decode step; each workgroup runs one
// (item, KV head) on the VALU or the MFMA path according to the item's kind.
// kWgsPerCu workgroups fit per CU (register budget 256 / kWgsPerCu per lane).
template <int D, bool NT>
__global__ __launch_bounds__(kThreads, kWgsPerCu) void partial_kernel(TREEPO_PARTIAL_PARAMS, int32_t first_item) {
  __shared__ __attribute__((aligned(1024))) TileSmem<D> sm;
  const int item = first_item + static_cast<int>(blockIdx.x) / sc.hkv;
  const int g = static_cast<int>(blockIdx.x) % sc.hkv;
  const int32_t* it = items + kItemInts * item;
  if (it[0] == 0) {
    switch (it[6]) {
      case 1: valu_item<D, 1, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 2: valu_item<D, 2, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 3: valu_item<D, 3, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 4: valu_item<D, 4, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 5: valu_item<D, 5, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 6: valu_item<D, 6, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 7: valu_item<D, 7, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      case 8: valu_item<D, 8, NT>(TREEPO_PARTIAL_ARGS, it, g, sm); break;
      default: break;
    }
  } else if (it[6] <= 32) {
    mfma_split_item<D, NT>(TREEPO_PARTIAL_ARGS, it, g, sm);
  } else {
    const int nrb = (((it[6] + 15) >> 4) + 3) >> 2;
    if (nrb == 1)
      mfma_item<D, 1, NT>(TREEPO_PARTIAL_ARGS, it, g, sm);
    else if (nrb == 2)
      mfma_item<D, 2, NT>(TREEPO_PARTIAL_ARGS, it, g, sm);
    // the planner keeps MFMA items at <= 128 rows
  }
}

// ---- combine ------------------------------------------------------------------
//
// One wave per (leaf, query head): m* = max m_i, L = sum l_i 2^(m_i - m*),
// out = sum 2^(m_i - m*) O_i / L, lse = (m* + log2 L) ln 2.  Partials of empty
// pieces (m = -inf) contribute nothing.  Entries are taken 64 at a time: the
// lanes load their (m, l) pairs in parallel, then the weights are broadcast
// with readlane while every lane accumulates its d-slice of the O rows (the
// row loads are independent, so they overlap).  The order of the sum is fixed
// (chain order), so results are deterministic.
template <int D>
__global__ __launch_bounds__(kThreads) void combine_kernel(const int32_t* __restrict__ leaf_off,
                                                           const int32_t* __restrict__ entries,
                                                           const float* __restrict__ part_o,
                                                           const float* __restrict__ part_ml,
                                                           float* __restrict__ out, float* __restrict__ lse,
                                                           int32_t n_leaves, int32_t hq, int32_t group) {
  constexpr int kPL = D / 64;
  const int lane = threadIdx.x & 63;
  const int gw = static_cast<int>(blockIdx.x) * kWaves + (threadIdx.x >> 6);
  if (gw >= n_leaves * hq) return;
  const int x = gw / hq;
  const int h = gw % hq;
  const int g = h / group;
  const int hp = h % group;
  const int e0 = leaf_off[x], e1 = leaf_off[x + 1];
  float run_m = -INFINITY, run_l = 0.f;
  float o[kPL];
#pragma unroll
  for (int i = 0; i < kPL; ++i) o[i] = 0.f;
  for (int base = e0; base < e1; base += 64) {
    const int cnt = e1 - base < 64 ? e1 - base : 64;
    const bool mine = lane < cnt;
    const int e = base + (mine ? lane : 0);
    const int slot = entries[2 * e] + g * entries[2 * e + 1] + hp;
    const float mi = mine ? part_ml[2 * static_cast<int64_t>(slot)] : -INFINITY;
    const float li = mine ? part_ml[2 * static_cast<int64_t>(slot) + 1] : 0.f;
    float cm = mi;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) cm = fmaxf(cm, __shfl_xor(cm, sh));
    const float nm = fmaxf(run_m, cm);
    const float keep = run_m == -INFINITY ? 0.f : fast_exp2(run_m - nm);
    const float w = mi == -INFINITY ? 0.f : fast_exp2(mi - nm);
    float wl = w * li;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) wl += __shfl_xor(wl, sh);
    run_l = run_l * keep + wl;
#pragma unroll
    for (int i = 0; i < kPL; ++i) o[i] *= keep;
    run_m = nm;
#pragma unroll 4
    for (int k = 0; k < cnt; ++k) {
      const float wk = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), k));
      const int sk = __builtin_amdgcn_readlane(slot, k);
      const float* po = part_o + static_cast<int64_t>(sk) * D + lane * kPL;
#pragma unroll
      for (int i = 0; i < kPL; ++i) o[i] += wk * po[i];
    }
  }
  const float inv = 1.f / run_l;
  float* op = out + (static_cast<int64_t>(x) * hq + h) * D + lane * kPL;
#pragma unroll
  for (int i = 0; i < kPL; ++i) op[i] = o[i] * inv;
  if (lse != nullptr && lane == 0) lse[static_cast<int64_t>(x) * hq + h] = (run_m + __log2f(run_l)) * kLn2;
}

// ---- KV append --------------------------------------------------------------
//
// One workgroup per (piece, KV head).  K rows are copied with 16-byte moves;
// V rows are transposed through LDS (padded rows, no bank conflicts) and
// written as runs of consecutive tokens of each d-row of the transposed half
// blocks.
constexpr int kMaxPieces = 128;
struct AppendBatch {
  int32_t n;
  int32_t pad;
  AppendPiece p[kMaxPieces];
};

template <int D>
__global__ __launch_bounds__(kThreads) void kv_append_kernel(const uint16_t* __restrict__ ksrc,
                                                             const uint16_t* __restrict__ vsrc,
                                                             uint16_t* __restrict__ kpool,
                                                             uint16_t* __restrict__ vpool,
                                                             int64_t num_blocks, int32_t hkv,
                                                             AppendBatch b) {
  constexpr int kPad = D + 2;
  __shared__ uint16_t vt[kTile * kPad];
  const AppendPiece pc = b.p[blockIdx.x];
  const int g = blockIdx.y;
  const int64_t blk = static_cast<int64_t>(g) * num_blocks + pc.block;
  constexpr int kCh = D / 8;
  for (int idx = threadIdx.x; idx < pc.count * kCh; idx += kThreads) {
    const int i = idx / kCh, c = idx % kCh;
    const int64_t src = (static_cast<int64_t>(pc.src_row + i) * hkv + g) * D + c * 8;
    const uint4 kvv = *reinterpret_cast<const uint4*>(ksrc + src);
    *reinterpret_cast<uint4*>(kpool + (blk * kTile + pc.off + i) * D + c * 8) = kvv;
    const uint4 vv = *reinterpret_cast<const uint4*>(vsrc + src);
    const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vt[i * kPad + c * 8 + 2 * e] = static_cast<uint16_t>(w[e] & 0xFFFFu);
      vt[i * kPad + c * 8 + 2 * e + 1] = static_cast<uint16_t>(w[e] >> 16);
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < D * pc.count; idx += kThreads) {
    const int d = idx / pc.count, i = idx % pc.count;
    const int p = pc.off + i;  // token within the 64-token block
    vpool[(blk * kTile + (p / kSub) * kSub) * D + d * kSub + (p % kSub)] = vt[i * kPad + d];
  }
}

}  // namespace

int32_t partial_workgroups_per_cu() { return kWgsPerCu; }

hipError_t launch_partial(const DecodeArgs& a, int32_t first_item, int32_t n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(n_items) * a.hkv);
  const Scalars sc{a.num_blocks, a.hq, a.hkv, a.group, a.scale_log2};
  auto go = [&](auto kernel) {
    kernel<<<grid, kThreads, 0, s>>>(a.k_pool, a.v_pool, a.q, a.items, a.rowsets, a.tiles, a.part_o, a.part_ml, sc,
                                     first_item);
  };
  if (a.d == 128)
    a.nontemporal ? go(partial_kernel<128, true>) : go(partial_kernel<128, false>);
  else
    a.nontemporal ? go(partial_kernel<64, true>) : go(partial_kernel<64, false>);
  return hipGetLastError();
}

hipError_t launch_combine(const DecodeArgs& a, hipStream_t s) {
  const int64_t waves = static_cast<int64_t>(a.n_leaves) * a.hq;
  const dim3 grid(static_cast<unsigned>((waves + kWaves - 1) / kWaves));
  if (a.d == 128)
    combine_kernel<128><<<grid, kThreads, 0, s>>>(a.leaf_off, a.entries, a.part_o, a.part_ml, a.out, a.lse,
                                                  a.n_leaves, a.hq, a.group);
  else
    combine_kernel<64><<<grid, kThreads, 0, s>>>(a.leaf_off, a.entries, a.part_o, a.part_ml, a.out, a.lse,
                                                 a.n_leaves, a.hq, a.group);
  return hipGetLastError();
}

hipError_t launch_kv_append(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_pool,
                            uint16_t* v_pool, int64_t num_blocks, int32_t hkv, int32_t d,
                            const AppendPiece* pieces, int32_t n_pieces, hipStream_t s) {
  for (int32_t p0 = 0; p0 < n_pieces; p0 += kMaxPieces) {
    AppendBatch b{};
    b.n = n_pieces - p0 < kMaxPieces ? n_pieces - p0 : kMaxPieces;
    for (int32_t i = 0; i < b.n; ++i) b.p[i] = pieces[p0 + i];
    const dim3 grid(static_cast<unsigned>(b.n), static_cast<unsigned>(hkv));
    if (d == 128)
      kv_append_kernel<128><<<grid, kThreads, 0, s>>>(k_src, v_src, k_pool, v_pool, num_blocks, hkv, b);
    else
      kv_append_kernel<64><<<grid, kThreads, 0, s>>>(k_src, v_src, k_pool, v_pool, num_blocks, hkv, b);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace treepo
