// gfx950 kernels of the segment-tree decode path: KV append (scatter into the
// pools), the node-partial kernel, and the log-sum-exp combine; and the
// prefill of appended tokens (causal attention over their chain).
//
// Node-partial attention (cascade schedule): the work is a list of pieces --
// consecutive KV tiles of one node run, scored against the query rows of a
// group of its descendant leaves for one KV head (the nested sub-groups of
// TreePO Sec. 2.3) -- cut into streams of equal cost, one per resident
// workgroup.  A workgroup streams its tiles once from HBM into LDS with 128-bit
// non-temporal global->LDS loads, three tiles ahead, without draining the
// pipeline between pieces, and writes per-row partials (O unnormalised,
// running max, sum) in fp32.  The combine merges, per leaf and query head, the
// partials of its chain (exact log-sum-exp algebra).
//
// Layouts (R = pool rows per KV head = blocks * B): K pool [Hkv][R][D]
// (token rows), V pool [Hkv][R / 16][D][16] (each 16-row group transposed,
// so a d-row of a group holds 16 consecutive tokens).  The kernels stream
// 32-token tiles -- 32 consecutive rows of a node from a 16-row boundary --,
// each one contiguous 8 KiB (D = 128) range per pool.
#include "kernels.h"

#include <hip/hip_ext.h>

#include <math.h>

#include "partial_format.h"
#include "tree_core.h"

namespace treepo {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ uint32_t f2bf_bits(float x) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(x)));
}
__device__ __forceinline__ float bf_bits2f(uint32_t b) { return __builtin_bit_cast(float, b << 16); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)p));
}

// ---- KV tile staging ----------------------------------------------------------
//
// A tile is 32 tokens: two consecutive 16-row groups of the pool.  LDS tile =
// K rows [32][D] then V^T rows [D][32] (chunks 0-1 of a d-row from the first
// group, 2-3 from the second), in 16-byte chunks with XOR swizzles that make
// the compute reads conflict free (per 8-lane LDS phase):
//   K: chunk c of token row r sits at position c ^ ((r & 3) | ((r >> 1) & 4));
//      the MFMA reader takes one chunk of rows {R+0..3, R+8..11} -- 8 distinct
//      bank groups.
//   V: chunk c of d-row d sits at position c ^ ((d >> 1) & 3); the reader takes
//      one chunk of 8 consecutive d-rows.
// Each wave moves whole 1 KiB LDS slots; the swizzle is applied on the global
// side (a lane picks which chunk of the same row it fetches), so each slot is
// still read from HBM in whole row segments.  Four tile buffers per workgroup
// keep three tiles in flight while one is consumed; two workgroups share a CU.
// A query tile -- up to 64 query rows [row][D] of a piece -- travels through
// the same buffers ahead of the piece's KV tiles.
constexpr int kSub = 32;   // tokens per tile
constexpr int kNBuf = 4;   // LDS tile buffers per workgroup
constexpr int kDepth = 3;  // tiles in flight while one is consumed
constexpr int kWgsPerCu = 2;
constexpr int kPrefillWaves = 4;  // waves per prefill workgroup (4 or 8)

template <int D>
struct Smem {
  static constexpr int kElems = kSub * D;  // K (or V^T) elements per tile
  uint16_t kv[kNBuf][2 * kElems];
  int32_t blk[kMaxBlockInts];              // the stream's block (pieces, tiles, segments, live tiles)
  int32_t live_len[kMaxStreamLive];        // current length of each live tile's node
};

// LDS views of the stream block's tables.
struct BlockTables {
  const int2* tiles;        // StreamTile records
  const int32_t* segs;      // query segment offsets
  const int32_t* dests;     // per (piece, leaf): partial row of its h' = 0
  const int32_t* live;      // per live tile: node, base (first token of the tile)
  const int32_t* live_len;  // per live tile: its node's length at this decode
};

// Tokens of a KV tile from its record's valid field: the planned count, or,
// for a live tile, the tokens its node holds now past the tile's first.
__device__ __forceinline__ int tile_tokens(int y, const BlockTables& bt) {
  if (y >= 0) return y;
  const int i = -1 - y;
  const int v = __builtin_amdgcn_readfirstlane(bt.live_len[i]) - __builtin_amdgcn_readfirstlane(bt.live[2 * i + 1]);
  return v < 0 ? 0 : (v > kSub ? kSub : v);
}

__device__ __forceinline__ int k_swz(int r) { return (r & 3) | ((r >> 1) & 4); }
__device__ __forceinline__ int v_swz(int d) { return (d >> 1) & 3; }

// One 16-byte global->LDS load per lane into the 1 KiB LDS slot at byte
// address `lds` (wave-uniform; lane l writes bytes [16 l, 16 l + 16) of it).
// Non-temporal: every byte is read once per call, so it is not kept in the
// caches.  Issued as inline asm so that the compiler does not treat the
// in-flight LDS writes as aliasing every later LDS access (which would drain
// the prefetch); completion is tracked by hand with vmcnt waits before the
// barrier that publishes a tile.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
               :: "v"(g), "s"(lds) : "memory", "m0");
}

// One 4-byte global->LDS load per lane (lane l writes bytes [4 l, 4 l + 4) at
// `lds`).
__device__ __forceinline__ void dma4(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :: "v"(g), "s"(lds) : "memory", "m0");
}

// The same load from a wave-uniform base address (SGPRs) plus a per-lane byte
// offset: no per-lane 64-bit address arithmetic.
__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
               :: "v"(voff), "s"(sbase), "s"(lds) : "memory", "m0");
}

// Loads per lane per tile.
template <int D>
constexpr int dma_per_tile() { return D / 32; }

// Rows of a transposed V group of the pool.
constexpr int kVGroup = 16;

// Global byte offset, within a tile's V^T data, of 16-byte chunk q (tokens
// 8q .. 8q + 7) of d-row d: chunks 0-1 lie in the tile's first 16-row group
// ([D][16], d-rows of 32 bytes), chunks 2-3 in the second.
template <int D>
__device__ __forceinline__ uint32_t v_chunk_off(int d, int q) {
  return (q >> 1) * (D * kVGroup * 2) + d * (kVGroup * 2) + (q & 1) * 16;
}

// The tile pipeline of a workgroup: LDS buffers, this lane's byte offsets in
// a tile's K and V^T ranges for each of its loads (the swizzles of the LDS
// layout applied on the global side), and the record of the next tile to
// issue, read from LDS one step early so that a tile's loads go out right
// after the barrier that frees its buffer.
template <int D>
struct Pipe {
  static constexpr int kPerWave = D / 64;  // 1 KiB slots per wave for each of K and V
  uint32_t buf0;                           // LDS byte address of buffer 0
  int ntot;                                // tiles of the stream
  uint32_t koff[kPerWave], voff[kPerWave];
  int2 next;                               // record of tile k + kDepth while tile k is current
};

template <int D>
__device__ __forceinline__ void pipe_init(Pipe<D>& p, uint32_t buf0, int ntot, int wave, int lane) {
  constexpr int kKChunks = D / 8;  // 16-byte chunks per K row
  p.buf0 = buf0;
  p.ntot = ntot;
  p.next = make_int2(0, 0);
#pragma unroll
  for (int j = 0; j < Pipe<D>::kPerWave; ++j) {
    const int c = (wave * Pipe<D>::kPerWave + j) * 64 + lane;
    const int row = c / kKChunks;
    p.koff[j] = row * (D * 2) + (((c % kKChunks) ^ k_swz(row)) << 4);
    const int vrow = c >> 2;
    p.voff[j] = v_chunk_off<D>(vrow, (c & 3) ^ v_swz(vrow));
  }
}

// Stages the tile whose first row is pool row 16 t16 (KV head included: t16 =
// (g * R + first row of head g's pool) / 16) into the LDS buffer at byte
// address `dst`.
// An empty live tile keeps its place in the load count, but every lane reads
// the tile's first 16 bytes (one request per load instruction).
template <int D>
__device__ __forceinline__ void dma_tile(const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
                                         int t16, bool empty, uint32_t dst, const Pipe<D>& p, int wave) {
  const int64_t off = static_cast<int64_t>(t16) * kVGroup * D;
  const uint16_t* kg = kpool + off;
  const uint16_t* vg = vpool + off;
  const uint32_t vd = dst + kSub * D * 2;
#pragma unroll
  for (int j = 0; j < Pipe<D>::kPerWave; ++j)
    dma16s(kg, empty ? 0u : p.koff[j], __builtin_amdgcn_readfirstlane(dst + (wave * Pipe<D>::kPerWave + j) * 1024));
#pragma unroll
  for (int j = 0; j < Pipe<D>::kPerWave; ++j)
    dma16s(vg, empty ? 0u : p.voff[j], __builtin_amdgcn_readfirstlane(vd + (wave * Pipe<D>::kPerWave + j) * 1024));
}

// Barrier after which this workgroup's global->LDS loads, except the newest N
// per lane, have landed; it also orders each wave's earlier LDS reads before
// any later overwrite (every wave waits for its own LDS reads before it).
// Loads complete in issue order, so vector stores issued in between only make
// the wait stricter.
template <int N>
__device__ __forceinline__ void barrier_tile_landed() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(N) : "memory");
}

// Waits for tile k of the stream (tiles up to k + 2 may have been issued)
// and publishes it.
template <int D>
__device__ __forceinline__ void wait_tile(int k, int ntot) {
  constexpr int kD = dma_per_tile<D>();
  const int ahead = ntot - 1 - k;  // tiles issued after tile k, capped at kDepth - 1
  if (ahead >= 2)
    barrier_tile_landed<2 * kD>();
  else if (ahead == 1)
    barrier_tile_landed<kD>();
  else
    barrier_tile_landed<0>();
}

// Kernel arguments, passed as separate __restrict__ kernel parameters.
struct Scalars {
  int32_t hq, hkv, group;
  float scale_log2;
  int32_t packed;  // partial rows as written-through block floating point (compact plans)
};

#define TREEPO_PARTIAL_PARAMS                                                         \
  const uint16_t *__restrict__ kpool, const uint16_t *__restrict__ vpool,            \
      const uint16_t *__restrict__ q, float *__restrict__ part_o, float *__restrict__ part_ml, Scalars sc
#define TREEPO_PARTIAL_ARGS kpool, vpool, q, part_o, part_ml, sc

// Stages rows [row0, row0 + n) of a piece's queries into the LDS buffer at
// `dst` as [64][D]: row r of the piece is head h' = r % G of its leaf j = r / G,
// whose G rows start at element segs[seg_base + j] of the query tensor.  Every
// lane issues the same loads as for a KV tile (rows past n repeat the last row).
template <int D>
__device__ __forceinline__ void dma_qtile(const uint16_t* __restrict__ q, int seg_base, int row0, int n, int G,
                                          const BlockTables& bt, uint32_t dst, int wave, int lane) {
  constexpr int kCPR = D / 8;       // 16-byte chunks per row
  constexpr int kPerWave = D / 32;  // 1 KiB slots per wave
#pragma unroll
  for (int j = 0; j < kPerWave; ++j) {
    const int slot = wave * kPerWave + j;
    const int c = slot * 64 + lane;
    const int r = c / kCPR;
    const int row = row0 + (r < n ? r : n - 1);
    const int leaf = row / G;
    const int h = row - leaf * G;
    const uint16_t* src = q + bt.segs[seg_base + leaf] + h * D + (c % kCPR) * 8;
    dma16(src, __builtin_amdgcn_readfirstlane(dst + slot * 1024));
  }
}

// Issues tile k of the stream (KV or query; `rec` its record) into buffer
// k mod 4.  `lengths` says whether the live tiles' lengths have landed in LDS;
// before that a live tile is loaded in full (it lies inside the pool: its
// node's reserved rows, or with 16-token blocks up to 16 rows past them) and
// only the compute looks at its length.
template <int D>
__device__ __forceinline__ void dma_stream_tile(TREEPO_PARTIAL_PARAMS, int k, int2 rec, const BlockTables& bt,
                                                const Pipe<D>& p, int wave, int lane, bool lengths) {
  constexpr uint32_t kBufBytes = 2 * kSub * D * 2;
  const int hb = __builtin_amdgcn_readfirstlane(rec.x);
  const uint32_t dst = p.buf0 + (k & (kNBuf - 1)) * kBufBytes;
  if (hb >= 0) {
    const int y = __builtin_amdgcn_readfirstlane(rec.y);
    dma_tile<D>(kpool, vpool, hb, lengths && y < 0 && tile_tokens(y, bt) == 0, dst, p, wave);
  } else {
    const int y = __builtin_amdgcn_readfirstlane(rec.y);
    dma_qtile<D>(q, -1 - hb, y & 0xFFFF, y >> 16, sc.group, bt, dst, wave, lane);
  }
}

// After tile k is published: tile k + 3 into the buffer tile k - 1 used (its
// record is already in registers), then the record of tile k + 4.  The live
// lengths were gathered before tile 0 was issued, so they have landed.
template <int D>
__device__ __forceinline__ void dma_ahead(TREEPO_PARTIAL_PARAMS, int k, const BlockTables& bt, Pipe<D>& p,
                                          int wave, int lane) {
  if (k + kDepth < p.ntot) {
    dma_stream_tile<D>(TREEPO_PARTIAL_ARGS, k + kDepth, p.next, bt, p, wave, lane, true);
    if (k + kDepth + 1 < p.ntot) p.next = bt.tiles[k + kDepth + 1];
  }
}

// A piece's record in the stream block.
struct PieceRec {
  int rows, k0, nk, seg;
};

// Partial row of the piece's query row m (leaf j = m / G, head h' = m % G).
__device__ __forceinline__ int64_t partial_row(const BlockTables& bt, int seg, int m, int G) {
  const int j = m / G;
  return static_cast<int64_t>(bt.dests[seg + j]) + (m - j * G);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Partial O rows.  Strided plans (a few MB of partials, which stay in the L2
// until the combine reads them) keep fp32 rows of D floats, written back.
// Compact plans, whose partial rows far exceed the L2 (45-83 MB in fp32 for
// the 64-prompt batch rollout, the irregular 32-prompt tree and the 16k-token
// long-context tree), store them in a block floating-point format at half
// the bytes and write them through:
//   * A lane's d-group (values at d = 4c .. 4c + 3) is one 64-bit word, 14-bit
//     mantissas under the group's exponent (format in partial_format.h); a
//     row is D / 4 words.  Each value is off by at most 2^-13 of its group's
//     largest magnitude; a merged output, a weighted mean of normalised
//     partials, by at most 2^-13 of the largest |V| value it averages --
//     about 8e-4 for N(0, 1) values at the sizes here, against the 2e-3 bar,
//     and measured far smaller.  Accumulation stays fp32.
//     Partial rows cost far more than their bytes while the KV stream is read
//     (a timing build without them ran the irregular tree 21% faster): at
//     half the bytes its kernel ran 6% faster (0.401 -> 0.377 ms), the batch
//     rollout's 2% (1.178 -> 1.153 ms) and the long-context tree's 0.5%.
//   * Write-through (sc1: device scope): the rows leave the L2 as they are
//     written instead of being written back in bursts while the KV stream
//     fills it: the batch rollout's kernel 1.258 -> 1.179 ms, the irregular
//     tree's 0.408 -> 0.399, the long-context tree's 1.916 -> 1.846; for the
//     16 leaves of 7680 tokens (strided) it was slower (35.6 -> 37.2 us).
// The s_nop in the store covers the store-data hazard the compiler cannot see
// through the asm.

// The d-group's four values are passed by value (a bit cast of a vector
// element itself reads the vector's first element).
__device__ __forceinline__ u32x2 pack_group(const f32x4& v) {
  uint32_t w0, w1;
  pack_group4(v.x, v.y, v.z, v.w, &w0, &w1);
  return u32x2{w0, w1};
}

__device__ __forceinline__ void unpack_group(const u32x2& p, float (&f)[4]) { unpack_group4(p.x, p.y, f); }

// Stores d-group c (values 4c .. 4c + 3) of partial row `slot`.
template <int D>
__device__ __forceinline__ void store_partial(float* part_o, int64_t slot, int c, const f32x4& v, bool packed) {
  if (packed) {
    const u32x2 w = pack_group(v);
    uint32_t* p = reinterpret_cast<uint32_t*>(part_o) + slot * (D / 2) + 2 * c;
    asm volatile("global_store_dwordx2 %0, %1, off sc1\n\ts_nop 1" :: "v"(p), "v"(w) : "memory");
  } else {
    *reinterpret_cast<f32x4*>(part_o + slot * D + 4 * c) = v;
  }
}

__device__ __forceinline__ f32x4 mfma16(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

// QK: S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (A = 16 K rows, B = Q^T).  The
// K rows of token block b (0, 1) are read in the order
// tau(b, r) = 8(r/4) + 4b + r%4, so that each lane's four outputs of block b
// are the consecutive tokens 8(lane/16) + 4b + 0..3 -- the layout of the P
// operand of the PV product, so P never leaves registers.
__device__ __forceinline__ int tau(int b, int r) { return 8 * (r >> 2) + 4 * b + (r & 3); }

// Lazy softmax reference (log2 units): O and the running sum are rescaled only
// when a score exceeds the row's reference by more than 2^8, so the weights
// stay <= 2^8 and in steady state a tile costs no cross-lane max and no
// rescale.
constexpr float kLazyMaxSlack = 8.f;

// P = 2^(x - ref) for the lane's four scores as hi + lo bf16 terms (about 16
// significant bits for the weights; a single bf16 P can be off by 2^-8
// relative, too much for short, peaked chains).  Returns the sum of the four
// represented weights.
__device__ __forceinline__ float softmax_p4(const float (&x)[4], float ref, uint2& P, uint2& PL) {
  uint32_t ph[2], pl[2];
  float ls = 0.f;
#pragma unroll
  for (int e = 0; e < 4; e += 2) {
    const float f0 = x[e] == -INFINITY ? 0.f : fast_exp2(x[e] - ref);
    const float f1 = x[e + 1] == -INFINITY ? 0.f : fast_exp2(x[e + 1] - ref);
    const uint32_t h0 = f2bf_bits(f0), h1 = f2bf_bits(f1);
    const uint32_t q0 = f2bf_bits(f0 - bf_bits2f(h0)), q1 = f2bf_bits(f1 - bf_bits2f(h1));
    ls += (bf_bits2f(h0) + bf_bits2f(q0)) + (bf_bits2f(h1) + bf_bits2f(q1));
    ph[e >> 1] = h0 | (h1 << 16);
    pl[e >> 1] = q0 | (q1 << 16);
  }
  P = make_uint2(ph[0], ph[1]);
  PL = make_uint2(pl[0], pl[1]);
  return ls;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Full tile (every token holds data): P = 2^(s scale - ref) for the lane's
// four raw scores s as hi + lo bf16 pairs.  ref is finite here (a piece's
// first tile always moves it off -inf).  Returns the sum of the four fp32
// weights (the represented hi + lo differ from them by < 2^-17 relative).
__device__ __forceinline__ float weights4(const f32x4& s, float scale_log2, float neg_ref, uint2& P, uint2& PL) {
  float ls = 0.f;
  uint32_t ph[2], pl[2];
#pragma unroll
  for (int e = 0; e < 4; e += 2) {
    const float f0 = fast_exp2(fmaf(s[e], scale_log2, neg_ref));
    const float f1 = fast_exp2(fmaf(s[e + 1], scale_log2, neg_ref));
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){f0, f1}, bf16x2));
    const float h0 = __builtin_bit_cast(float, h << 16), h1 = __builtin_bit_cast(float, h & 0xFFFF0000u);
    pl[e >> 1] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){f0 - h0, f1 - h1}, bf16x2));
    ph[e >> 1] = h;
    ls += f0 + f1;
  }
  P = make_uint2(ph[0], ph[1]);
  PL = make_uint2(pl[0], pl[1]);
  return ls;
}

// Clears the V^T entries of tokens tok0..tok0+3 past the node's length (their
// P is 0, but the pool may hold any bits there).
__device__ __forceinline__ uint2 mask_v4(uint2 v, int tok0, int valid) {
  v.x &= tok0 >= valid ? 0u : (tok0 + 1 >= valid ? 0xFFFFu : 0xFFFFFFFFu);
  v.y &= tok0 + 2 >= valid ? 0u : (tok0 + 3 >= valid ? 0xFFFFu : 0xFFFFFFFFu);
  return v;
}

// ---- column-split piece (at most 32 rows) ------------------------------------------
//
// One or two 16-row blocks: one leaf's GQA group, or a few leaves of a shared
// node.  Splitting rows over waves would leave most waves idle, so the waves
// of a row block split the output columns instead: wave w takes row block
// w / DSPLIT and d columns [D/DSPLIT * (w % DSPLIT), +D/DSPLIT) (DSPLIT = 4 for
// one row block, 2 for two).  Every wave scores all 32 tokens of the tile for
// its rows -- the waves of a row block compute the same scores and softmax
// state bit for bit -- and accumulates its own slice of O, so each query row
// gets one partial with no cross-wave merge.
//   QK: S^T = K Q^T, eight MFMAs (two token blocks x D/32 k-steps).
//   PV: O^T += V^T P^T with v_mfma_f32_16x16x32_bf16 over all 32 tokens for
//       the wave's d-blocks (A = 16 d-rows of V^T, B = P^T: the lane's eight
//       scores, tokens 8(lane/16) + 0..7).
template <int D, int DSPLIT>
__device__ __forceinline__ void dsplit_piece(TREEPO_PARTIAL_PARAMS, const PieceRec& pc, Pipe<D>& pp, Smem<D>& sm,
                                             const BlockTables& bt) {
  constexpr int kKS = D / 32;             // QK k-steps
  constexpr int kDBw = D / 16 / DSPLIT;   // PV output d-blocks of this wave
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int a = lane >> 4;    // lane group
  const int r16 = lane & 15;  // row within the 16-row block
  const int rb = wave / DSPLIT;
  const int db0 = (wave % DSPLIT) * kDBw;
  const int rows = pc.rows, k0 = pc.k0, nk = pc.nk;
  const bool active = 16 * rb < rows;  // wave-uniform
  const int m = 16 * rb + r16;         // this lane's query row

  // ---- the piece's query tile: Q^T operands, lane holds row m, d chunk 4 ks + a
  uint4 qb[kKS];
  wait_tile<D>(k0, pp.ntot);
  dma_ahead<D>(TREEPO_PARTIAL_ARGS, k0, bt, pp, wave, lane);
  {
    const uint4* qt = reinterpret_cast<const uint4*>(sm.kv[k0 & (kNBuf - 1)]) + m * (D / 8);
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) qb[ks] = m < rows ? qt[4 * ks + a] : make_uint4(0, 0, 0, 0);
  }

  f32x4 acc[kDBw];
#pragma unroll
  for (int db = 0; db < kDBw; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_ref = -INFINITY;  // per row (equal on the row's four lane groups)
  float l_sum = 0.f;        // per lane: this lane's tokens only

  for (int k = k0 + 1; k <= k0 + nk; ++k) {
    wait_tile<D>(k, pp.ntot);
    dma_ahead<D>(TREEPO_PARTIAL_ARGS, k, bt, pp, wave, lane);
    const int valid = tile_tokens(__builtin_amdgcn_readfirstlane(bt.tiles[k].y), bt);
    if (!active || valid == 0) continue;
    const char* kt = reinterpret_cast<const char*>(sm.kv[k & (kNBuf - 1)]);
    const char* vt = kt + kSub * D * 2;
    // ---- S^T = K Q^T for the 32 tokens
    f32x4 S[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int tok = tau(b, r16);
        const int c = 4 * ks + a;
        const uint4 ka = *reinterpret_cast<const uint4*>(kt + tok * (D * 2) + ((c ^ k_swz(tok)) << 4));
        S[b] = mfma16(ka, qb[ks], S[b]);
      }
    }
    // ---- scores (log2 units) with a lazy reference: O and the sum are
    // rescaled only when a row's maximum passes it by more than the slack
    if (valid == kSub) {
      // full tile (the common case): no masking; max over the raw scores
      // (the scale is positive)
      float mx = fmaxf(fmaxf(fmaxf(S[0][0], S[0][1]), fmaxf(S[0][2], S[0][3])),
                       fmaxf(fmaxf(S[1][0], S[1][1]), fmaxf(S[1][2], S[1][3]))) * sc.scale_log2;
      if (__builtin_amdgcn_ballot_w64(mx > m_ref + kLazyMaxSlack) != 0) {
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m_ref, mx);
        const float alpha = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - mn);
        m_ref = mn;
        l_sum *= alpha;
#pragma unroll
        for (int db = 0; db < kDBw; ++db) acc[db] *= alpha;
      }
      uint2 p0, pl0, p1, pl1;
      l_sum += weights4(S[0], sc.scale_log2, -m_ref, p0, pl0) + weights4(S[1], sc.scale_log2, -m_ref, p1, pl1);
      const uint4 P = make_uint4(p0.x, p0.y, p1.x, p1.y), PL = make_uint4(pl0.x, pl0.y, pl1.x, pl1.y);
      // ---- O^T += V^T P^T for the wave's d-blocks
#pragma unroll
      for (int db = 0; db < kDBw; ++db) {
        const int d = 16 * (db0 + db) + r16;
        const uint4 va = *reinterpret_cast<const uint4*>(vt + d * (kSub * 2) + ((a ^ v_swz(d)) << 4));
        acc[db] = mfma16(va, PL, mfma16(va, P, acc[db]));
      }
      continue;
    }
    // the node's last tile: tokens past its length are masked
    float x[2][4];
    float mx = -INFINITY;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[b][e] = 8 * a + 4 * b + e < valid ? S[b][e] * sc.scale_log2 : -INFINITY;
        mx = fmaxf(mx, x[b][e]);
      }
    if (__builtin_amdgcn_ballot_w64(mx > m_ref + kLazyMaxSlack) != 0) {
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m_ref, mx);
      const float alpha = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - mn);
      m_ref = mn;
      l_sum *= alpha;
#pragma unroll
      for (int db = 0; db < kDBw; ++db) acc[db] *= alpha;
    }
    uint2 p0, pl0, p1, pl1;
    l_sum += softmax_p4(x[0], m_ref, p0, pl0) + softmax_p4(x[1], m_ref, p1, pl1);
    const uint4 P = make_uint4(p0.x, p0.y, p1.x, p1.y), PL = make_uint4(pl0.x, pl0.y, pl1.x, pl1.y);
#pragma unroll
    for (int db = 0; db < kDBw; ++db) {
      const int d = 16 * (db0 + db) + r16;
      uint4 va = *reinterpret_cast<const uint4*>(vt + d * (kSub * 2) + ((a ^ v_swz(d)) << 4));
      const uint2 lo = mask_v4(make_uint2(va.x, va.y), 8 * a, valid);
      const uint2 hi = mask_v4(make_uint2(va.z, va.w), 8 * a + 4, valid);
      va = make_uint4(lo.x, lo.y, hi.x, hi.y);
      acc[db] = mfma16(va, PL, mfma16(va, P, acc[db]));
    }
  }

  // ---- partial rows: this wave's column slice
  l_sum += __shfl_xor(l_sum, 16);
  l_sum += __shfl_xor(l_sum, 32);
  if (active && m < rows) {
    const int64_t slot = partial_row(bt, pc.seg, m, sc.group);
#pragma unroll
    for (int db = 0; db < kDBw; ++db)
      store_partial<D>(part_o, slot, 4 * (db0 + db) + a, acc[db], sc.packed != 0);
    if (a == 0 && db0 == 0) {
      part_ml[slot * 2 + 0] = m_ref;
      part_ml[slot * 2 + 1] = l_sum;
    }
  }
}

// ---- row-split piece (33 to 128 rows) ---------------------------------------------
//
// Shared nodes whose stacked query rows (descendant leaves x GQA group) form
// dense tiles.  Rows are cut into 16-row blocks; wave w owns blocks w, w+4
// (NRB per wave) and keeps their online-softmax state; all four waves read
// every KV tile from LDS, so K and V operands are reused across a wave's row
// blocks.
//   QK: both token blocks of the tile (eight MFMAs per row block).
//   PV: O^T += V^T P^T with v_mfma_f32_16x16x32_bf16 over all 32 tokens (A =
//       16 d-rows of the transposed V tile, B = P^T: the lane's eight scores).
template <int D, int NRB>
__device__ __forceinline__ void rows_piece(TREEPO_PARTIAL_PARAMS, const PieceRec& pc, Pipe<D>& pp, Smem<D>& sm,
                                           const BlockTables& bt) {
  constexpr int kKS = D / 32;
  constexpr int kDB = D / 16;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int a = lane >> 4;
  const int r16 = lane & 15;
  const int rows = pc.rows, k0 = pc.k0, nk = pc.nk;
  const int nq = (rows + kQTileRows - 1) / kQTileRows;
  const int nrb_total = (rows + 15) >> 4;
  const int my_rb = nrb_total > wave ? (nrb_total - wave + 3) >> 2 : 0;  // row blocks of this wave (<= NRB)

  // ---- the piece's query tiles (64 rows each): row block wave + 4 i sits in
  // tile i; lane holds row m = 16 (wave + 4 i) + r16, d chunk 4 ks + a
  uint4 qb[NRB][kKS];
#pragma unroll
  for (int i = 0; i < NRB; ++i) {
    if (i >= nq) continue;
    wait_tile<D>(k0 + i, pp.ntot);
    dma_ahead<D>(TREEPO_PARTIAL_ARGS, k0 + i, bt, pp, wave, lane);
    const int m = 16 * (wave + 4 * i) + r16;
    const uint4* qt =
        reinterpret_cast<const uint4*>(sm.kv[(k0 + i) & (kNBuf - 1)]) + (m - kQTileRows * i) * (D / 8);
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) qb[i][ks] = m < rows ? qt[4 * ks + a] : make_uint4(0, 0, 0, 0);
  }

  f32x4 acc[NRB][kDB];
  float m_ref[NRB], l_sum[NRB];
#pragma unroll
  for (int i = 0; i < NRB; ++i) {
    m_ref[i] = -INFINITY;
    l_sum[i] = 0.f;
#pragma unroll
    for (int db = 0; db < kDB; ++db) acc[i][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int k = k0 + nq; k < k0 + nq + nk; ++k) {
    wait_tile<D>(k, pp.ntot);
    dma_ahead<D>(TREEPO_PARTIAL_ARGS, k, bt, pp, wave, lane);
    const int valid = tile_tokens(__builtin_amdgcn_readfirstlane(bt.tiles[k].y), bt);
    if (my_rb == 0 || valid == 0) continue;
    const char* kt = reinterpret_cast<const char*>(sm.kv[k & (kNBuf - 1)]);
    const char* vt = kt + kSub * D * 2;
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
      float x[2][4];
      float mx = -INFINITY;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[b][e] = 8 * a + 4 * b + e < valid ? S[i][b][e] * sc.scale_log2 : -INFINITY;
          mx = fmaxf(mx, x[b][e]);
        }
      if (__builtin_amdgcn_ballot_w64(mx > m_ref[i] + kLazyMaxSlack) != 0) {
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m_ref[i], mx);
        const float alpha = m_ref[i] == -INFINITY ? 0.f : fast_exp2(m_ref[i] - mn);
        m_ref[i] = mn;
        l_sum[i] *= alpha;
#pragma unroll
        for (int db = 0; db < kDB; ++db) acc[i][db] *= alpha;
      }
      uint2 p0, pl0, p1, pl1;
      l_sum[i] += softmax_p4(x[0], m_ref[i], p0, pl0) + softmax_p4(x[1], m_ref[i], p1, pl1);
      P[i] = make_uint4(p0.x, p0.y, p1.x, p1.y);
      PL[i] = make_uint4(pl0.x, pl0.y, pl1.x, pl1.y);
    }
    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      const int d = 16 * db + r16;
      uint4 va = *reinterpret_cast<const uint4*>(vt + d * (kSub * 2) + ((a ^ v_swz(d)) << 4));
      if (valid < kSub) {
        const uint2 lo = mask_v4(make_uint2(va.x, va.y), 8 * a, valid);
        const uint2 hi = mask_v4(make_uint2(va.z, va.w), 8 * a + 4, valid);
        va = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
#pragma unroll
      for (int i = 0; i < NRB; ++i)
        if (i < my_rb) acc[i][db] = mfma16(va, PL[i], mfma16(va, P[i], acc[i][db]));
    }
  }

  // ---- write the partial rows (each wave owns its row blocks)
#pragma unroll
  for (int i = 0; i < NRB; ++i) {
    if (i >= my_rb) continue;
    float l = l_sum[i];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int m = 16 * (wave + 4 * i) + r16;
    if (m < rows) {
      const int64_t slot = partial_row(bt, pc.seg, m, sc.group);
#pragma unroll
      for (int db = 0; db < kDB; ++db)
        store_partial<D>(part_o, slot, 4 * db + a, acc[i][db], sc.packed != 0);
      if (a == 0) {
        part_ml[slot * 2 + 0] = m_ref[i];
        part_ml[slot * 2 + 1] = l;
      }
    }
  }
}

// ---- the node-partial kernel ----------------------------------------------------
//
// One workgroup per stream.  Prologue: the stream's block (its piece records,
// tile list and query segment offsets) into LDS with one round of
// global->LDS loads from an address computed from the workgroup index, so
// the first tiles are issued one memory round trip after the start; then the
// first three tiles.  The pieces run in order over one continuous tile
// pipeline: every load is a global->LDS load counted by hand and every piece
// record comes from LDS, so no compiler-inserted wait ever drains it.
template <int D>
__global__ __launch_bounds__(kThreads, kWgsPerCu) void partial_kernel(const int32_t* __restrict__ blocks,
                                                                     int32_t block_ints,
                                                                     const int32_t* __restrict__ node_len,
                                                                     TREEPO_PARTIAL_PARAMS) {
  __shared__ __attribute__((aligned(1024))) Smem<D> sm;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t buf0 = lds_addr(sm.kv[0]);
  {
    // the block: block_ints (a multiple of 4, at most kMaxBlockInts) in 16-byte loads
    const char* src = reinterpret_cast<const char*>(blocks + static_cast<int64_t>(blockIdx.x) * block_ints);
    const uint32_t dst = lds_addr(sm.blk);
    const int nch = block_ints >> 2;
    for (int c0 = wave * 64; c0 < nch; c0 += kThreads)
      if (c0 + lane < nch) dma16(src + 16 * (c0 + lane), dst + 16 * c0);
  }
  barrier_tile_landed<0>();
  const int np = __builtin_amdgcn_readfirstlane(sm.blk[0]);
  const int ntot = __builtin_amdgcn_readfirstlane(sm.blk[1]);
  const int nseg = __builtin_amdgcn_readfirstlane(sm.blk[2]);
  const int n_live = __builtin_amdgcn_readfirstlane(sm.blk[3]);
  const int tile_at = kBlockHeaderInts + kBlockPieceInts * np;
  const int seg_at = tile_at + 2 * ((ntot + 1) & ~1);
  const int live_at = seg_at + 2 * ((nseg + 3) & ~3);
  const BlockTables bt{reinterpret_cast<const int2*>(sm.blk + tile_at), sm.blk + seg_at,
                       sm.blk + seg_at + ((nseg + 3) & ~3), sm.blk + live_at, sm.live_len};
  // live tiles: their nodes' current lengths, gathered into LDS ahead of the
  // first tile loads (older loads, so they have landed when tile 0 has; the
  // first tiles are issued before that and load live tiles in full)
  for (int c0 = wave * 64; c0 < n_live; c0 += kThreads)
    if (c0 + lane < n_live)
      dma4(node_len + bt.live[2 * (c0 + lane)], __builtin_amdgcn_readfirstlane(lds_addr(sm.live_len + c0)));
  Pipe<D> pp;
  pipe_init<D>(pp, buf0, ntot, wave, lane);
#pragma unroll
  for (int t = 0; t < kDepth; ++t)
    if (t < ntot) dma_stream_tile<D>(TREEPO_PARTIAL_ARGS, t, bt.tiles[t], bt, pp, wave, lane, false);
  if (kDepth < ntot) pp.next = bt.tiles[kDepth];
  for (int pi = 0; pi < np; ++pi) {
    const int4 r = *reinterpret_cast<const int4*>(sm.blk + kBlockHeaderInts + kBlockPieceInts * pi);
    const PieceRec pc{__builtin_amdgcn_readfirstlane(r.x), __builtin_amdgcn_readfirstlane(r.y),
                      __builtin_amdgcn_readfirstlane(r.z), __builtin_amdgcn_readfirstlane(r.w)};
    if (pc.rows <= 16) {
      dsplit_piece<D, 4>(TREEPO_PARTIAL_ARGS, pc, pp, sm, bt);
    } else if (pc.rows <= kSplitMaxRows) {
      dsplit_piece<D, 2>(TREEPO_PARTIAL_ARGS, pc, pp, sm, bt);
    } else {
      const int nrb = (((pc.rows + 15) >> 4) + 3) >> 2;
      if (nrb == 1)
        rows_piece<D, 1>(TREEPO_PARTIAL_ARGS, pc, pp, sm, bt);
      else
        rows_piece<D, 2>(TREEPO_PARTIAL_ARGS, pc, pp, sm, bt);  // the planner keeps pieces at <= 128 rows
    }
  }
}

// ---- combine ------------------------------------------------------------------
//
// One wave per (leaf, query head h = g G + h'): over the n partial entries of
// key = (leaf, g), m* = max m_e, L = sum l_e 2^(m_e - m*), out = sum
// 2^(m_e - m*) O_e / L, lse = (m* + log2 L) ln 2.  Partials without tokens
// (m = -inf) contribute nothing.  Entry e of the key sits at partial row
// (base + e) G + h'; comb[key] = {base, n}.  Two layouts:
//   strided (base = key E, E the largest count; fp32 rows, every lane its
//     D / 64 values of each row): the (m, l) pairs of entries
//     0..min(E, 64)-1 (one per lane) and the O rows of entries
//     0..min(E, R0)-1 are loaded in the same round as the count, so a key
//     with up to R0 entries costs one memory round trip; entries past the
//     count (stale values of earlier calls) are masked out by selection.  For
//     plans whose speculative reads are small (the decode is then latency
//     bound).  Later entries follow in batches of 16 independent row loads.
//   compact (base = the prefix sum of the counts; block floating-point rows):
//     {base, n} first, then exactly the n entries' rows -- a second round
//     trip, but no row is read that the key does not hold (plans with many
//     keys, where the combine is bound by the bytes it reads).  A row's D / 4
//     packed d-groups are read by D / 4 lanes, so the wave forms S = 256 / D
//     slots that read S entries side by side (slot s takes entries s, s + S,
//     ...); the slots' sums are added at the end.
// The sums run in a fixed order, so results are deterministic.

// Strided layout: adds sum over entries k in [k0, cnt) of the 64-entry batch
// starting at entry `base` of w_k O_k to o (w_k in lane k of w), 16
// independent row loads at a time.
template <int D>
__device__ __forceinline__ void combine_rows(float (&o)[D / 64], const float* __restrict__ part_o, int64_t row0,
                                             int group, int base, int k0, int cnt, float w, int lane) {
  constexpr int kPL = D / 64;
  constexpr int kGroup = 16;
  for (; k0 < cnt; k0 += kGroup) {
    float v[kGroup][kPL];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int k = k0 + i < cnt ? k0 + i : cnt - 1;
      const float* po = part_o + (row0 + static_cast<int64_t>(base + k) * group) * D + lane * kPL;
#pragma unroll
      for (int j = 0; j < kPL; ++j) v[i][j] = po[j];
    }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const float wk = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), k0 + i));
      if (k0 + i < cnt) {
#pragma unroll
        for (int j = 0; j < kPL; ++j) o[j] += wk * v[i][j];
      }
    }
  }
}

// Compact layout (block floating-point rows): the same sum, lane (slot s, group c) reading
// entries k0 + s + S t, eight rows per lane at a time.
template <int D>
__device__ __forceinline__ void combine_rows_packed(float (&o)[4], const uint32_t* __restrict__ part_o, int64_t row0,
                                                    int group, int base, int k0, int cnt, float w, int lane) {
  constexpr int kNG = D / 4, kS = 64 / kNG, kRow = D / 2, kT = 8;
  const int c = lane % kNG, sl = lane / kNG;
  for (; k0 < cnt; k0 += kT * kS) {
    u32x2 v[kT];
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      if (k0 + kS * t >= cnt) break;  // wave-uniform
      const int k = k0 + sl + kS * t;
      const int kk = k < cnt ? k : cnt - 1;
      v[t] = *reinterpret_cast<const u32x2*>(part_o + (row0 + static_cast<int64_t>(base + kk) * group) * kRow + 2 * c);
    }
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      if (k0 + kS * t >= cnt) break;
      const int k = k0 + sl + kS * t;
      const float wk = __shfl(w, k < cnt ? k : 0);
      float f[4];
      unpack_group(v[t], f);
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = k >= cnt || wk == 0.f ? o[j] : fmaf(wk, f[j], o[j]);
    }
  }
}

template <int D, int R0, bool kCompact>
__global__ __launch_bounds__(kThreads) void combine_kernel(const int2* __restrict__ comb, int32_t emax,
                                                           const float* __restrict__ part_o,
                                                           const float* __restrict__ part_ml,
                                                           float* __restrict__ out, float* __restrict__ lse,
                                                           int32_t n_leaves, int32_t hq, int32_t hkv, int32_t group) {
  constexpr int kPL = D / 64;                    // strided: values per lane of a row
  constexpr int kNG = D / 4, kS = 64 / kNG;      // compact: d-groups per row, slots per wave
  constexpr int kO = kCompact ? 4 : kPL;         // output values per lane
  constexpr int kV = kCompact ? R0 / kS : R0;    // round-0 rows per lane
  const uint32_t* __restrict__ packed = reinterpret_cast<const uint32_t*>(part_o);
  const int lane = threadIdx.x & 63;
  const int c = lane % kNG, sl = lane / kNG;
  const int gw = static_cast<int>(blockIdx.x) * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (gw >= n_leaves * hq) return;
  const int x = gw / hq;
  const int h = gw % hq;
  const int g = h / group;
  const int hp = h % group;
  const int key = x * hkv + g;
  int n, base, lim;
  if (kCompact) {
    const int2 cb = comb[key];
    base = __builtin_amdgcn_readfirstlane(cb.x);
    n = __builtin_amdgcn_readfirstlane(cb.y);
    lim = n;          // rows the key holds
  } else {
    base = key * emax;
    n = comb[key].y;  // lands with the speculative loads below
    lim = emax;       // rows its slots can hold
  }
  const int64_t row0 = static_cast<int64_t>(base) * group + hp;  // entry e: row0 + e * group

  // round 0: (m, l) of entries 0..min(lim, 64)-1 and O rows of entries
  // 0..min(lim, R0)-1
  const int avail = lim < 64 ? lim : 64;
  const int avail_o = lim < R0 ? lim : R0;
  const int64_t my_row = row0 + static_cast<int64_t>(lane < avail ? lane : avail - 1) * group;
  float vf[kCompact ? 1 : kV][kPL];
  u32x2 vp[kCompact ? kV : 1];
#pragma unroll
  for (int i = 0; i < kV; ++i) {
    if constexpr (kCompact) {
      const int e = sl + kS * i;
      vp[i] = e < avail_o ? *reinterpret_cast<const u32x2*>(packed + (row0 + static_cast<int64_t>(e) * group) *
                                                                         (D / 2) + 2 * c)
                          : u32x2{0u, 0u};
    } else {
      if (i < avail_o) {
        const float* po = part_o + (row0 + static_cast<int64_t>(i) * group) * D + lane * kPL;
#pragma unroll
        for (int j = 0; j < kPL; ++j) vf[i][j] = po[j];
      } else {
#pragma unroll
        for (int j = 0; j < kPL; ++j) vf[i][j] = 0.f;
      }
    }
  }
  const float m_ld = part_ml[2 * my_row];
  const float l_ld = part_ml[2 * my_row + 1];
  // keeps every round-0 load ahead of the count-dependent code (otherwise the
  // compiler may sink a load under the weight test, a second round trip)
#pragma unroll
  for (int i = 0; i < kV; ++i) {
    if constexpr (kCompact) {
      asm volatile("" ::"v"(vp[i].x), "v"(vp[i].y));
    } else {
#pragma unroll
      for (int j = 0; j < kPL; ++j) asm volatile("" ::"v"(vf[i][j]));
    }
  }
  asm volatile("" ::"v"(m_ld), "v"(l_ld));

  float o[kO];
#pragma unroll
  for (int j = 0; j < kO; ++j) o[j] = 0.f;
  int cnt = n < 64 ? n : 64;
  float mi = lane < cnt ? m_ld : -INFINITY;
  float li = lane < cnt ? l_ld : 0.f;
  float run_m = mi;
#pragma unroll
  for (int sh = 1; sh < 64; sh <<= 1) run_m = fmaxf(run_m, __shfl_xor(run_m, sh));
  float w = mi == -INFINITY ? 0.f : fast_exp2(mi - run_m);
  float run_l = w * li;
#pragma unroll
  for (int sh = 1; sh < 64; sh <<= 1) run_l += __shfl_xor(run_l, sh);
  // entries past the count have w = 0 and may hold anything: select, not multiply
#pragma unroll
  for (int i = 0; i < kV; ++i) {
    if constexpr (kCompact) {
      if (kS * i >= avail_o) break;  // no slot holds an entry from here on (wave-uniform)
      const float wk = __shfl(w, sl + kS * i);
      float f[4];
      unpack_group(vp[i], f);
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = wk == 0.f ? o[j] : fmaf(wk, f[j], o[j]);
    } else {
      const float wk = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), i));
#pragma unroll
      for (int j = 0; j < kPL; ++j) o[j] = wk == 0.f ? o[j] : fmaf(wk, vf[i][j], o[j]);
    }
  }
  auto rows = [&](int b, int k0) {
    if constexpr (kCompact)
      combine_rows_packed<D>(o, packed, row0, group, b, k0, cnt, w, lane);
    else
      combine_rows<D>(o, part_o, row0, group, b, k0, cnt, w, lane);
  };
  if (n > R0) {
    rows(0, R0);
    for (int b = 64; b < n; b += 64) {
      cnt = n - b < 64 ? n - b : 64;
      const int64_t r = row0 + static_cast<int64_t>(b + (lane < cnt ? lane : 0)) * group;
      mi = lane < cnt ? part_ml[2 * r] : -INFINITY;
      li = lane < cnt ? part_ml[2 * r + 1] : 0.f;
      float cm = mi;
#pragma unroll
      for (int sh = 1; sh < 64; sh <<= 1) cm = fmaxf(cm, __shfl_xor(cm, sh));
      const float nm = fmaxf(run_m, cm);
      const float keep = fast_exp2(run_m - nm);  // run_m is finite: some entry holds tokens
      w = mi == -INFINITY ? 0.f : fast_exp2(mi - nm);
      float wl = w * li;
#pragma unroll
      for (int sh = 1; sh < 64; sh <<= 1) wl += __shfl_xor(wl, sh);
      run_l = run_l * keep + wl;
#pragma unroll
      for (int j = 0; j < kO; ++j) o[j] *= keep;
      run_m = nm;
      rows(b, 0);
    }
  }
  const float inv = 1.f / run_l;
  float* op = out + (static_cast<int64_t>(x) * hq + h) * D;
  if constexpr (kCompact) {
    // the slots' sums, then the lanes of slot 0 write the row
#pragma unroll
    for (int sh = kNG; sh < 64; sh <<= 1)
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] += __shfl_xor(o[j], sh);
    if (sl == 0) *reinterpret_cast<f32x4*>(op + 4 * c) = f32x4{o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv};
  } else {
#pragma unroll
    for (int j = 0; j < kPL; ++j) op[lane * kPL + j] = o[j] * inv;
  }
  if (lse != nullptr && lane == 0) lse[static_cast<int64_t>(x) * hq + h] = (run_m + __log2f(run_l)) * kLn2;
}

// ---- KV append --------------------------------------------------------------
//
// One workgroup per (piece, KV head).  K rows are copied with 16-byte moves;
// V rows are transposed through LDS (padded rows, no bank conflicts) and
// written as runs of consecutive tokens of each d-row of the transposed
// 16-row groups.
constexpr int kMaxPieces = 128;
struct AppendBatch {
  int32_t n;      // pieces
  int32_t n_upd;  // length updates (node, length)
  AppendPiece p[kMaxPieces];
  int2 upd[kMaxPieces];
};

// One piece for KV head blockIdx.y: K rows copied with 16-byte moves, V
// transposed through padded LDS into the pool's [D][16] groups.
template <int D>
__device__ __forceinline__ void append_piece(const uint16_t* __restrict__ ksrc, const uint16_t* __restrict__ vsrc,
                                             uint16_t* __restrict__ kpool, uint16_t* __restrict__ vpool,
                                             int64_t rows, int32_t hkv, const AppendPiece& pc, uint16_t* vt) {
  constexpr int kPad = D + 2;
  const int g = blockIdx.y;
  const int64_t row0 = static_cast<int64_t>(g) * rows + static_cast<int64_t>(pc.block) * kTile + pc.off;
  constexpr int kCh = D / 8;
  for (int idx = threadIdx.x; idx < pc.count * kCh; idx += kThreads) {
    const int i = idx / kCh, c = idx % kCh;
    const int64_t src = (static_cast<int64_t>(pc.src_row + i) * hkv + g) * D + c * 8;
    const uint4 kvv = *reinterpret_cast<const uint4*>(ksrc + src);
    *reinterpret_cast<uint4*>(kpool + (row0 + i) * D + c * 8) = kvv;
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
    const int64_t p = row0 + i;  // pool row (KV head included; g * rows is a multiple of 16)
    vpool[(p / kVGroup) * kVGroup * D + d * kVGroup + p % kVGroup] = vt[i * kPad + d];
  }
}

// Pieces and length updates passed by value (up to kMaxPieces per launch).
template <int D>
__global__ __launch_bounds__(kThreads) void kv_append_kernel(const uint16_t* __restrict__ ksrc,
                                                             const uint16_t* __restrict__ vsrc,
                                                             uint16_t* __restrict__ kpool,
                                                             uint16_t* __restrict__ vpool,
                                                             int64_t rows, int32_t hkv,
                                                             int32_t* __restrict__ node_len, AppendBatch b) {
  __shared__ uint16_t vt[kTile * (D + 2)];
  if (node_len != nullptr && blockIdx.y == 0 && threadIdx.x == 0 && static_cast<int>(blockIdx.x) < b.n_upd)
    node_len[b.upd[blockIdx.x].x] = b.upd[blockIdx.x].y;
  if (static_cast<int>(blockIdx.x) >= b.n) return;
  append_piece<D>(ksrc, vsrc, kpool, vpool, rows, hkv, b.p[blockIdx.x], vt);
}

// The same with the pieces and length updates in device memory: one launch
// for any number of pieces.
template <int D>
__global__ __launch_bounds__(kThreads) void kv_append_dev_kernel(
    const uint16_t* __restrict__ ksrc, const uint16_t* __restrict__ vsrc, uint16_t* __restrict__ kpool,
    uint16_t* __restrict__ vpool, int64_t rows, int32_t hkv, int32_t* __restrict__ node_len,
    const AppendPiece* __restrict__ pieces, int32_t n, const int2* __restrict__ upd, int32_t n_upd) {
  __shared__ uint16_t vt[kTile * (D + 2)];
  if (node_len != nullptr && blockIdx.y == 0 && threadIdx.x == 0 && static_cast<int>(blockIdx.x) < n_upd) {
    const int2 u = upd[blockIdx.x];
    node_len[u.x] = u.y;
  }
  if (static_cast<int>(blockIdx.x) >= n) return;
  const AppendPiece pc = pieces[blockIdx.x];
  append_piece<D>(ksrc, vsrc, kpool, vpool, rows, hkv, pc, vt);
}


// ---- prefill ------------------------------------------------------------------------
//
// Causal attention of tokens just appended to a node, over its chain (a
// query's shared prompt, prefilled once for all of its rollouts).  A
// workgroup takes up to 128 consecutive new tokens of one sequence for one
// query head; with W waves (4 or 8), wave w owns tokens [R w, R w + R),
// R = 128 / W, as R / 16 row blocks that share every K and V operand it reads
// from LDS.  Eight waves of 16 rows keep the registers under 128 per lane,
// so that four waves share each SIMD and hide each other's latencies.  The workgroup streams the
// 32-token tiles of the chain up to its last token through the decode's
// four-buffer global->LDS pipeline.  Tiles that every row of a wave sees in
// full take the unmasked path; the others mask keys past each row's own
// position and, at a node's end, past the tile's tokens.
//
// Work order: a unit is (item, KV head); the host lists each XCD's units,
// longest first, keeping a sequence's units for one KV head on one XCD where
// the balance allows.  Workgroup w runs on XCD x = w % 8; its index s = w / 8
// on that XCD gives slot s / G of the schedule and head h = g G + s % G, so
// the G query heads of a unit run on one XCD at about the same time and the
// chain's K/V tiles are reused through that XCD's L2.
// The prefill's tile loads: a 32-token tile is 2 D / 16 slots of 1 KiB (K
// rows, then V^T rows, swizzled as for the decode); each of the W waves
// issues D / (8 W) of them per tile, one 16-byte global->LDS load per lane
// each, so every wave counts the same number of loads per tile.
template <int D, int W>
struct PfPipe {
  static constexpr int kKSlots = kSub * D * 2 / 1024;
  static constexpr int kSlots = 2 * kKSlots / W;  // per wave
  uint32_t buf0;
  uint32_t off[kSlots];

  __device__ __forceinline__ void init(uint32_t b0, int wave, int lane) {
    constexpr int kKChunks = D / 8;
    buf0 = b0;
#pragma unroll
    for (int j = 0; j < kSlots; ++j) {
      const int sl = wave * kSlots + j;
      if (sl < kKSlots) {
        const int c = sl * 64 + lane;
        const int row = c / kKChunks;
        off[j] = row * (D * 2) + (((c % kKChunks) ^ k_swz(row)) << 4);
      } else {
        const int c = (sl - kKSlots) * 64 + lane;
        const int vrow = c >> 2;
        off[j] = v_chunk_off<D>(vrow, (c & 3) ^ v_swz(vrow));
      }
    }
  }
  // Stages the tile whose first row is pool row 16 t16 into the buffer at
  // LDS byte address dst.
  __device__ __forceinline__ void issue(const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool,
                                        int t16, uint32_t dst, int wave) const {
    const int64_t o = static_cast<int64_t>(t16) * kVGroup * D;
#pragma unroll
    for (int j = 0; j < kSlots; ++j) {
      const int sl = wave * kSlots + j;
      if (sl < kKSlots)
        dma16s(kpool + o, off[j], __builtin_amdgcn_readfirstlane(dst + sl * 1024));
      else
        dma16s(vpool + o, off[j], __builtin_amdgcn_readfirstlane(dst + kSub * D * 2 + (sl - kKSlots) * 1024));
    }
  }
  // Waits for tile k when up to `cap` newer tiles may have been issued, and
  // publishes it.
  __device__ __forceinline__ void wait(int k, int ntot, int cap) const {
    const int ahead = ntot - 1 - k < cap ? ntot - 1 - k : cap;
    if (ahead >= 2)
      barrier_tile_landed<2 * kSlots>();
    else if (ahead == 1)
      barrier_tile_landed<kSlots>();
    else
      barrier_tile_landed<0>();
  }
};

template <int D, int W>
__global__ __launch_bounds__(64 * W, W / 2) void prefill_kernel(
    const uint16_t* __restrict__ kpool, const uint16_t* __restrict__ vpool, const uint16_t* __restrict__ q,
    const PrefillItem* __restrict__ items, const int2* __restrict__ tiles, const int32_t* __restrict__ sched,
    float* __restrict__ out, float* __restrict__ lse, int32_t n_sched, int32_t rows16, int32_t hq, int32_t hkv,
    float scale_log2) {
  constexpr int kKS = D / 32;  // QK k-steps
  constexpr int kDB = D / 16;  // PV output d-blocks
  constexpr int kRB = 8 / W;   // 16-row blocks per wave
  constexpr int kRows = 16 * kRB;
  constexpr uint32_t kBufBytes = 2 * kSub * D * 2;
  __shared__ __attribute__((aligned(16))) uint16_t kv[kNBuf][2 * kSub * D];

  const int G = hq / hkv;
  const int wg = blockIdx.x;
  const int s_x = wg >> 3;
  const int slot = (s_x / G) * 8 + (wg & 7);
  if (slot >= n_sched) return;  // whole workgroup
  const int unit = sched[slot];
  if (unit < 0) return;
  const int item_i = unit / hkv;
  const int g = unit - item_i * hkv;
  const int h = g * G + s_x % G;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int a = lane >> 4;    // lane group
  const int r16 = lane & 15;  // row within a 16-row block
  const PrefillItem it = items[item_i];
  const int nk = it.nk;
  const int2* __restrict__ tl = tiles + it.tile_off;
  const int hb_base = g * rows16;  // KV head g's pool rows start at row 16 hb_base

  // Q^T operands: lane holds row kRows wave + 16 rb + r16, d chunk 4 ks + a
  uint4 qb[kRB][kKS];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    const int m = kRows * wave + 16 * rb + r16;
    if (m < it.n_rows) {
      const uint4* src = reinterpret_cast<const uint4*>(q + (static_cast<int64_t>(it.row0 + m) * hq + h) * D);
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) qb[rb][ks] = src[4 * ks + a];
    } else {
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) qb[rb][ks] = make_uint4(0, 0, 0, 0);
    }
  }
  // The query loads land before the first tile is issued: otherwise the
  // compiler, which does not see the tile loads, would wait for them (and so
  // drain the tile pipeline) at their first use inside the loop.
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) asm volatile("" ::"v"(qb[rb][ks].x));

  PfPipe<D, W> pp;
  pp.init(lds_addr(kv[0]), wave, lane);
  for (int k = 0; k < kDepth && k < nk; ++k) pp.issue(kpool, vpool, hb_base + tl[k].x, pp.buf0 + k * kBufBytes, wave);
  int2 next = kDepth < nk ? tl[kDepth] : make_int2(0, 0);

  const int row_w = kRows * wave;  // the wave's first row
  const bool wave_on = row_w < it.n_rows;
  const int pos_lo = it.pos0 + row_w;
  const int pos_hi = it.pos0 + (row_w + kRows - 1 < it.n_rows - 1 ? row_w + kRows - 1 : it.n_rows - 1);
  int prow[kRB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) prow[rb] = it.pos0 + row_w + 16 * rb + r16;

  f32x4 acc[kRB][kDB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
    for (int db = 0; db < kDB; ++db) acc[rb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_ref[kRB], l_sum[kRB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    m_ref[rb] = -INFINITY;
    l_sum[rb] = 0.f;
  }

  // S^T = K Q^T for the 32 tokens of tile k, both row blocks
  auto qk = [&](int k, f32x4 (&S)[kRB][2]) {
    const char* kt = reinterpret_cast<const char*>(kv[k & (kNBuf - 1)]);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) S[rb][0] = S[rb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int tok = tau(b, r16);
        const int c = 4 * ks + a;
        const uint4 ka = *reinterpret_cast<const uint4*>(kt + tok * (D * 2) + ((c ^ k_swz(tok)) << 4));
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) S[rb][b] = mfma16(ka, qb[rb][ks], S[rb][b]);
      }
    }
  };

  // weights of tile k (lazy reference per row, as in the decode), then
  // O^T += V^T P^T with one V operand per d-block for both row blocks
  auto softmax_pv = [&](int k, const f32x4 (&S)[kRB][2], int first, int cnt) {
    const char* vt = reinterpret_cast<const char*>(kv[k & (kNBuf - 1)]) + kSub * D * 2;
    const bool full = cnt == kSub && first + kSub - 1 <= pos_lo;
    uint4 P[kRB], PL[kRB];
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      float x[2][4];
      float mx = -INFINITY;
      if (full) {
        // every key visible: max over the raw scores (the scale is positive)
        mx = fmaxf(fmaxf(fmaxf(S[rb][0][0], S[rb][0][1]), fmaxf(S[rb][0][2], S[rb][0][3])),
                   fmaxf(fmaxf(S[rb][1][0], S[rb][1][1]), fmaxf(S[rb][1][2], S[rb][1][3]))) * scale_log2;
      } else {
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int t = 8 * a + 4 * b + e;
            x[b][e] = t < cnt && first + t <= prow[rb] ? S[rb][b][e] * scale_log2 : -INFINITY;
            mx = fmaxf(mx, x[b][e]);
          }
      }
      if (__builtin_amdgcn_ballot_w64(mx > m_ref[rb] + kLazyMaxSlack) != 0) {
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m_ref[rb], mx);
        const float alpha = m_ref[rb] == -INFINITY ? 0.f : fast_exp2(m_ref[rb] - mn);
        m_ref[rb] = mn;
        l_sum[rb] *= alpha;
#pragma unroll
        for (int db = 0; db < kDB; ++db) acc[rb][db] *= alpha;
      }
      uint2 p0, pl0, p1, pl1;
      if (full) {
        l_sum[rb] += weights4(S[rb][0], scale_log2, -m_ref[rb], p0, pl0) +
                     weights4(S[rb][1], scale_log2, -m_ref[rb], p1, pl1);
      } else {
        l_sum[rb] += softmax_p4(x[0], m_ref[rb], p0, pl0) + softmax_p4(x[1], m_ref[rb], p1, pl1);
      }
      P[rb] = make_uint4(p0.x, p0.y, p1.x, p1.y);
      PL[rb] = make_uint4(pl0.x, pl0.y, pl1.x, pl1.y);
    }
    // one test per tile (not per d-block), so that the common full tile
    // issues its V reads together and its MFMAs back to back
    uint4 va[kDB];
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      const int d = 16 * db + r16;
      va[db] = *reinterpret_cast<const uint4*>(vt + d * (kSub * 2) + ((a ^ v_swz(d)) << 4));
    }
    if (cnt < kSub) {
#pragma unroll
      for (int db = 0; db < kDB; ++db) {
        const uint2 lo = mask_v4(make_uint2(va[db].x, va[db].y), 8 * a, cnt);
        const uint2 hi = mask_v4(make_uint2(va[db].z, va[db].w), 8 * a + 4, cnt);
        va[db] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
    }
#pragma unroll
    for (int db = 0; db < kDB; ++db)
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) acc[rb][db] = mfma16(va[db], PL[rb], mfma16(va[db], P[rb], acc[rb][db]));
  };

  // Software pipeline: iteration k scores tile k + 1 (its K) while it turns
  // tile k's scores into weights and accumulates tile k's V, so the matrix
  // cores work on QK while the vector ALUs do the softmax.  Tile k + 1 must
  // have landed at the start of iteration k; two tiles stay in flight.
  f32x4 Sc[kRB][2], Sn[kRB][2];
  pp.wait(0, nk, 2);
  int first_c = __builtin_amdgcn_readfirstlane(tl[0].y >> 6);
  int cnt_c = __builtin_amdgcn_readfirstlane(tl[0].y & 63);
  bool vis_c = wave_on && first_c <= pos_hi;
  if (vis_c) qk(0, Sc);
  for (int k = 0; k < nk; ++k) {
    int first_n = 0, cnt_n = 0;
    bool vis_n = false;
    if (k + 1 < nk) {
      pp.wait(k + 1, nk, 1);
      if (k + kDepth < nk) {
        pp.issue(kpool, vpool, hb_base + next.x, pp.buf0 + ((k + kDepth) & (kNBuf - 1)) * kBufBytes, wave);
        if (k + kDepth + 1 < nk) next = tl[k + kDepth + 1];
      }
      const int2 rn = tl[k + 1];
      first_n = __builtin_amdgcn_readfirstlane(rn.y >> 6);
      cnt_n = __builtin_amdgcn_readfirstlane(rn.y & 63);
      vis_n = wave_on && first_n <= pos_hi;
    }
    if (vis_n) qk(k + 1, Sn);
    if (vis_c) softmax_pv(k, Sc, first_c, cnt_c);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      Sc[rb][0] = Sn[rb][0];
      Sc[rb][1] = Sn[rb][1];
    }
    first_c = first_n;
    cnt_c = cnt_n;
    vis_c = vis_n;
  }

  // ---- normalised rows and their log-sum-exp
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    float l = l_sum[rb];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int m = row_w + 16 * rb + r16;
    if (wave_on && m < it.n_rows) {
      const int64_t orow = static_cast<int64_t>(it.row0 + m) * hq + h;
      const float inv = 1.f / l;
#pragma unroll
      for (int db = 0; db < kDB; ++db)
        *reinterpret_cast<f32x4*>(out + orow * D + 16 * db + 4 * a) = acc[rb][db] * inv;
      if (lse != nullptr && a == 0) lse[orow] = (m_ref[rb] + __log2f(l)) * kLn2;
    }
  }
}

}  // namespace

int32_t partial_workgroups_per_cu() { return kWgsPerCu; }

// Launches `kernel` on `s`; with a.ev_start set, the events record the
// kernel's own start and end.
template <typename A, typename... Args, typename F>
void launch_timed_block(const A& a, F kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  if (a.ev_start)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a.ev_start, a.ev_stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

template <typename A, typename... Args, typename F>
void launch_timed(const A& a, F kernel, dim3 grid, hipStream_t s, Args... args) {
  if (a.ev_start)
    hipExtLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, a.ev_start, a.ev_stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, args...);
}

hipError_t launch_partial(const DecodeArgs& a, hipStream_t s) {
  if (a.n_streams <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(a.n_streams));
  const Scalars sc{a.hq, a.hkv, a.group, a.scale_log2, a.compact ? 1 : 0};
  if (a.block_ints <= 0 || a.block_ints > kMaxBlockInts || a.block_ints % 4 != 0) return hipErrorInvalidValue;
  if (a.d == 128)
    launch_timed(a, partial_kernel<128>, grid, s, a.blocks, a.block_ints, a.node_len, a.k_pool, a.v_pool, a.q,
                 a.part_o, a.part_ml, sc);
  else
    launch_timed(a, partial_kernel<64>, grid, s, a.blocks, a.block_ints, a.node_len, a.k_pool, a.v_pool, a.q,
                 a.part_o, a.part_ml, sc);
  return hipGetLastError();
}

template <int D>
void launch_combine_d(const DecodeArgs& a, dim3 grid, hipStream_t s) {
  if (a.compact)
    launch_timed(a, combine_kernel<D, 16, true>, grid, s, a.comb, a.emax, a.part_o, a.part_ml, a.out, a.lse,
                 a.n_leaves, a.hq, a.hkv, a.group);
  else if (a.emax > 16)
    launch_timed(a, combine_kernel<D, 32, false>, grid, s, a.comb, a.emax, a.part_o, a.part_ml, a.out, a.lse,
                 a.n_leaves, a.hq, a.hkv, a.group);
  else
    launch_timed(a, combine_kernel<D, 16, false>, grid, s, a.comb, a.emax, a.part_o, a.part_ml, a.out, a.lse,
                 a.n_leaves, a.hq, a.hkv, a.group);
}

hipError_t launch_combine(const DecodeArgs& a, hipStream_t s) {
  const int64_t waves = static_cast<int64_t>(a.n_leaves) * a.hq;
  const dim3 grid(static_cast<unsigned>((waves + kWaves - 1) / kWaves));
  if (a.d == 128)
    launch_combine_d<128>(a, grid, s);
  else
    launch_combine_d<64>(a, grid, s);
  return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs& a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.hkv <= 0 || a.hq % a.hkv != 0 || (a.d != 64 && a.d != 128)) return hipErrorInvalidValue;
  if (a.n_sched <= 0 || a.n_sched % 8 != 0) return hipErrorInvalidValue;
  const int64_t group = a.hq / a.hkv;
  const int64_t wgs = static_cast<int64_t>(a.n_sched) * group;
  if (wgs > 0x7FFFFFFF || a.pool_rows % kVGroup != 0 || a.hkv * (a.pool_rows / kVGroup) > 0x7FFFFFFF)
    return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(wgs));
  const int32_t nb = static_cast<int32_t>(a.pool_rows / kVGroup);
  const dim3 block(64 * kPrefillWaves);
  if (a.d == 128)
    launch_timed_block(a, prefill_kernel<128, kPrefillWaves>, grid, block, s, a.k_pool, a.v_pool, a.q, a.items,
                       a.tiles, a.sched, a.out, a.lse, a.n_sched, nb, a.hq, a.hkv, a.scale_log2);
  else
    launch_timed_block(a, prefill_kernel<64, kPrefillWaves>, grid, block, s, a.k_pool, a.v_pool, a.q, a.items,
                       a.tiles, a.sched, a.out, a.lse, a.n_sched, nb, a.hq, a.hkv, a.scale_log2);
  return hipGetLastError();
}

hipError_t launch_kv_append_dev(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_pool, uint16_t* v_pool,
                                int64_t rows, int32_t hkv, int32_t d, const AppendPiece* pieces,
                                int32_t n_pieces, const int2* upd, int32_t n_upd, int32_t* node_len,
                                hipStream_t s) {
  if (node_len == nullptr) n_upd = 0;
  const int32_t gx = n_pieces > n_upd ? n_pieces : n_upd;
  if (gx <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(hkv));
  if (d == 128)
    kv_append_dev_kernel<128><<<grid, kThreads, 0, s>>>(k_src, v_src, k_pool, v_pool, rows, hkv, node_len,
                                                       pieces, n_pieces, upd, n_upd);
  else
    kv_append_dev_kernel<64><<<grid, kThreads, 0, s>>>(k_src, v_src, k_pool, v_pool, rows, hkv, node_len,
                                                      pieces, n_pieces, upd, n_upd);
  return hipGetLastError();
}

hipError_t launch_kv_append(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_pool,
                            uint16_t* v_pool, int64_t rows, int32_t hkv, int32_t d,
                            const AppendPiece* pieces, int32_t n_pieces, const int32_t* upd_node,
                            const int32_t* upd_len, int32_t n_upd, int32_t* node_len, hipStream_t s) {
  if (node_len == nullptr) n_upd = 0;
  for (int32_t p0 = 0; p0 < n_pieces || p0 < n_upd; p0 += kMaxPieces) {
    AppendBatch b{};
    b.n = n_pieces - p0 < kMaxPieces ? (n_pieces > p0 ? n_pieces - p0 : 0) : kMaxPieces;
    b.n_upd = n_upd - p0 < kMaxPieces ? (n_upd > p0 ? n_upd - p0 : 0) : kMaxPieces;
    for (int32_t i = 0; i < b.n; ++i) b.p[i] = pieces[p0 + i];
    for (int32_t i = 0; i < b.n_upd; ++i) b.upd[i] = make_int2(upd_node[p0 + i], upd_len[p0 + i]);
    const int32_t gx = b.n > b.n_upd ? b.n : b.n_upd;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(hkv));
    if (d == 128)
      kv_append_kernel<128><<<grid, kThreads, 0, s>>>(k_src, v_src, k_pool, v_pool, rows, hkv, node_len, b);
    else
      kv_append_kernel<64><<<grid, kThreads, 0, s>>>(k_src, v_src, k_pool, v_pool, rows, hkv, node_len, b);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace treepo
