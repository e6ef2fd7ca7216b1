// Host core of the segment-tree KV cache: node table, block allocator and the
// decode planner.  Pure C++17 (no HIP), so it builds and tests on any CPU.
//
// Tree rules (TreePO Sec. 2.2 preliminaries and Alg. 1): a root per query at
// depth 0; children are forked from a path before each segment step and
// continue its sequence; each node holds one segment of at most `cap` tokens;
// a node with children is frozen.  Every node reserves ceil(cap/B) contiguous
// blocks at creation, at the running total of all earlier reservations.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace treepo {

enum Status : int32_t {
  kOk = 0,
  kEInval = -1,
  kENoMem = -2,
  kEFull = -3,
  kEFrozen = -4,
  kEEmpty = -5,
  kEWorkspace = -6,
  kEHip = -7,
  kEUnsupported = -8,
};

struct Node {
  int32_t parent;
  int32_t depth;
  int32_t start;  // token position of the node's first row within its sequence
  int32_t len;    // tokens held
  int32_t cap;    // tokens it may hold
  int32_t block_begin;
  int32_t n_blocks;
  int32_t tree_id;
  int32_t n_children;
};

class Tree {
 public:
  Tree(int32_t block_tokens, int64_t num_blocks, int32_t max_nodes)
      : B_(block_tokens), num_blocks_(num_blocks), max_nodes_(max_nodes) {}

  int32_t new_root(int32_t cap, int32_t* node_out, std::string* err);
  int32_t fork(int32_t parent, int32_t n, int32_t cap, int32_t* out, std::string* err);
  // Validates a batched append; on success fills `dest_rows` (if non-null)
  // with the pool token row of every appended token, in call order.
  int32_t check_append(int32_t n, const int32_t* nodes, const int32_t* ntok,
                       std::vector<int64_t>* dest_rows, std::string* err) const;
  void apply_append(int32_t n, const int32_t* nodes, const int32_t* ntok);

  int32_t check_leaves(int32_t n, const int32_t* leaves, std::string* err) const;

  const std::vector<Node>& nodes() const { return nodes_; }
  int32_t block_tokens() const { return B_; }
  // Bumped by every mutation; plans are cached against it.
  uint64_t version() const { return version_; }
  void chain(int32_t x, std::vector<int32_t>* out) const;
  int64_t chain_tokens(int32_t x) const;

 private:
  int32_t reserve_check(int32_t count, int32_t cap, std::string* err) const;
  int32_t make(int32_t parent, int32_t depth, int32_t start, int32_t cap, int32_t tree_id);

  int32_t B_;
  int64_t num_blocks_;
  int32_t max_nodes_;
  int64_t next_block_ = 0;
  int32_t n_roots_ = 0;
  uint64_t version_ = 0;
  std::vector<Node> nodes_;
};

// ---- decode plan -----------------------------------------------------------

enum PlanMode : int32_t { kModeTree = 0, kModeNaive = 1 };

// Tokens per decode tile (half of a 64-token pool block).
constexpr int32_t kPlanTileTokens = 32;
enum ItemKind : int32_t { kKindValu = 0, kKindMfma = 1 };

// One work item: a chunk of consecutive KV tiles of one run (a maximal chain
// segment whose nodes share the same descendant-leaf set), scored against the
// query rows of a group of those leaves.  A workgroup processes one item for
// one KV head.  Rows are (leaf j of the group, head h' of the GQA group):
// row = j * G + h'.
struct Item {
  int32_t kind;
  int32_t rowset_begin;  // index into Plan::rowsets
  int32_t n_leaves;      // leaves in the group
  int32_t tile_begin;    // index into Plan::tiles
  int32_t tile_end;
  int32_t partial_base;  // partial row of (g=0, row 0); (g, r) -> base + g*rows + r
  int32_t rows;          // n_leaves * G
  int32_t run;
  int32_t first_src[3];  // half-block index (2 * block + half) of the first tiles, -1 past the end
  int32_t pad;
};
constexpr int32_t kItemInts = 12;

// A KV tile: up to kPlanTileTokens tokens of one node, tokens
// [32 k, 32 k + 32) of the node for tile_in_node = k, inside pool block
// block_begin + k / 2.
struct Tile {
  int32_t block;
  int32_t node;
  int32_t tile_in_node;
  int32_t valid;  // tokens of the tile holding data (1..32)
};

// Per leaf, the partials to merge: slot(g, h') = a + g * b + h'.
struct Entry {
  int32_t a;
  int32_t b;
};

struct PlanParams {
  int32_t group;            // G = Hq / Hkv
  int32_t num_kv_heads;     // Hkv
  int32_t valu_max_rows;    // rows <= this use the VALU kernel
  int32_t mfma_max_rows;    // rows per MFMA item at most
  int32_t concurrent_wgs;   // workgroups resident at once (chunking target)
  int32_t max_chunk_tiles;  // upper bound on tiles per item
  int32_t mfma_enabled;     // 0: every item is split to the VALU row limit
};

struct Plan {
  PlanMode mode = kModeTree;
  std::vector<Item> items;  // VALU items first, then MFMA items
  int32_t n_valu_items = 0;
  std::vector<int32_t> rowsets;
  std::vector<Tile> tiles;
  std::vector<int32_t> leaf_off;  // n_leaves + 1
  std::vector<Entry> entries;
  int64_t partial_rows = 0;       // total partial rows over items and KV heads
  int32_t chunk_tiles = 0;
  int64_t unique_kv_tokens = 0;   // tokens streamed per KV head (tree: unique)
  int64_t kv_token_visits = 0;    // tiles' tokens x item groups (reads per head)
};

// Builds the decode schedule for `leaves` (validated by the caller).
int32_t build_plan(const Tree& t, int32_t n_leaves, const int32_t* leaves, PlanMode mode,
                   const PlanParams& p, Plan* out, std::string* err);

// Node -> ascending call positions of the leaves whose chain contains it, for
// every node on some chain (ascending id).
void desc_sets(const Tree& t, int32_t n_leaves, const int32_t* leaves,
               std::vector<int32_t>* nodes, std::vector<int32_t>* off,
               std::vector<int32_t>* desc);

}  // namespace treepo
