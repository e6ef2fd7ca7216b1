// Launch interface between the C-ABI host code and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace treepo {

constexpr int kTile = 64;  // rows of an append piece at most (a 64-row chunk of the pool)

// Device views of the decode plan and buffers (record layouts in tree_core.h).
struct DecodeArgs {
  const uint16_t* k_pool;  // bf16 [Hkv][R][D], R = pool rows per KV head
  const uint16_t* v_pool;  // bf16 [Hkv][R / 16][D][16] (V^T per 16-row group)
  int64_t pool_rows;       // R
  int32_t hq, hkv, group, d;
  const uint16_t* q;       // bf16 [n_leaves][Hq][D]
  float scale_log2;        // softmax scale * log2(e)
  const int32_t* node_len; // device token count per node (live tiles), or null
  const int32_t* blocks;   // stream blocks, block_ints int32 each (layout in tree_core.h)
  int32_t block_ints;
  int32_t n_streams;
  float* part_o;           // unnormalised rows: fp32 [partial_rows][D], or (compact) [partial_rows][D / 4] 64-bit block-float groups
  float* part_ml;          // fp32 [partial_rows][2]: running max (log2 units), sum
  const int2* comb;           // per key (leaf, KV head): {first entry, entries to merge}
  int32_t emax;               // entries per key at most (partial slot stride of strided plans)
  bool compact;               // entries packed by prefix sums (else key k starts at entry k * emax)
  // Profiling: when set, the launch records these events at the kernel's
  // start and end (hipExtLaunchKernelGGL), so they time the kernel alone.
  hipEvent_t ev_start = nullptr, ev_stop = nullptr;
  int32_t n_leaves;
  float* out;              // fp32 [n_leaves][Hq][D]
  float* lse;              // fp32 [n_leaves][Hq] or null
};

// The decode entry point that allocates nothing keeps a plan image and the
// partial slots in one static device array of this many bytes per device
// (noalloc.hip).  noalloc_scratch gives its address on the current device
// (looked up once per device) and the slot recording which plan image it
// holds (0: none).
constexpr size_t kNoAllocScratchBytes = size_t{64} << 20;
hipError_t noalloc_scratch(void** ptr, uint64_t** holder);

// One workgroup per stream: every piece's node partials.
hipError_t launch_partial(const DecodeArgs& a, hipStream_t s);
hipError_t launch_combine(const DecodeArgs& a, hipStream_t s);
// Node-partial workgroups resident per compute unit (set by the kernel's
// register and LDS budget); the planner makes one stream per resident slot.
int32_t partial_workgroups_per_cu();

// TreePO advantage (advantage.hip): one workgroup over index arrays built on
// the host from the leaves' chains.  Sub-group g = the call positions whose
// chain contains node g (members grp_mem[grp_off[g], grp_off[g+1]));
// position p's strict predecessors are the sub-groups
// pos_grp[pos_off[p], pos_off[p+1]) (root first), its query's group
// pos_root[p].
struct AdvantageArgs {
  const int32_t* grp_off;
  const int32_t* grp_mem;
  int32_t n_groups;
  const int32_t* pos_off;
  const int32_t* pos_grp;
  const int32_t* pos_root;
  int32_t n_pos;
  const float* rewards;    // [n_pos], device
  int32_t size_weighted;   // 0: mean over sub-groups, 1: |G|-weighted mean
  double* gmean;           // [n_groups] scratch
  int32_t* gkeep;          // [n_groups] scratch: rewards of the sub-group not all equal
  double* pooled;          // [n_pos] scratch
  float* adv;              // [n_pos], device
};
hipError_t launch_advantage(const AdvantageArgs& a, hipStream_t s);

// Prefill: causal attention of tokens just appended to a node over its chain.
// A work item is up to kPrefillRows consecutive new tokens of one sequence;
// the kernel runs it for every query head.  Tile records (int2): x = (first
// row of the 32-token tile in KV head 0's pool rows) / 16 (the kernel adds
// KV head g's R / 16), y = (chain position of the tile's first token) << 6 |
// tokens.
constexpr int32_t kPrefillRows = 128;
struct PrefillItem {
  int32_t row0;      // packed row (of q, out, lse) of the item's first token
  int32_t n_rows;    // tokens of the item, 1..kPrefillRows
  int32_t pos0;      // chain position of the item's first token
  int32_t tile_off;  // first tile record of the sequence's chain
  int32_t nk;        // tiles the item streams: those starting at or before its last token
  int32_t pad[3];    // pad[0]: the item's sequence (host scheduling only)
};
struct PrefillArgs {
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  int64_t pool_rows;         // pool rows per KV head (a multiple of 16)
  int32_t hq, hkv, d;
  const uint16_t* q;         // bf16 [rows][Hq][D]
  const PrefillItem* items;  // n_items, longest first
  int32_t n_items;
  const int2* tiles;
  const int32_t* sched;      // [slot * 8 + xcd] -> unit = item * Hkv + KV head, or -1
  int32_t n_sched;           // a multiple of 8
  float scale_log2;
  float* out;                // fp32 [rows][Hq][D]
  float* lse;                // fp32 [rows][Hq] or null
  hipEvent_t ev_start = nullptr, ev_stop = nullptr;
};
hipError_t launch_prefill(const PrefillArgs& a, hipStream_t s);

// One run of appended tokens: source rows [src_row, +count) go to pool rows
// [64 block + off, +count) of every KV head (off + count <= 64).
struct AppendPiece {
  int32_t src_row;
  int32_t block;
  int32_t off;
  int32_t count;
};

// node_len (device lengths table or null) receives len[i] at node[i] for the
// n_upd appended nodes (n_upd <= n_pieces).
hipError_t launch_kv_append(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_pool,
                            uint16_t* v_pool, int64_t pool_rows, int32_t hkv, int32_t d,
                            const AppendPiece* pieces, int32_t n_pieces, const int32_t* upd_node,
                            const int32_t* upd_len, int32_t n_upd, int32_t* node_len, hipStream_t s);
// The same with pieces and updates (x = node, y = length) in device memory,
// in one launch.
hipError_t launch_kv_append_dev(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_pool, uint16_t* v_pool,
                                int64_t pool_rows, int32_t hkv, int32_t d, const AppendPiece* pieces,
                                int32_t n_pieces, const int2* upd, int32_t n_upd, int32_t* node_len,
                                hipStream_t s);

}  // namespace treepo
