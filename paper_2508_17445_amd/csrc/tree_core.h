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
  // With 16-token blocks the pool's last block is never reserved: a node's
  // last 32-token tile may reach 16 rows past its blocks, and this keeps
  // such a tile inside the pool.
  Tree(int32_t block_tokens, int64_t num_blocks, int32_t max_nodes)
      : B_(block_tokens),
        num_blocks_(block_tokens < 32 && num_blocks > 0 ? num_blocks - 1 : num_blocks),
        max_nodes_(max_nodes) {}

  int32_t new_root(int32_t cap, int32_t* node_out, std::string* err);
  int32_t fork(int32_t parent, int32_t n, int32_t cap, int32_t* out, std::string* err);
  // Fork n (>= 0) children after the first `offset` tokens of `node`: the
  // node keeps [0, offset), a new tail node (next id) takes [offset, len),
  // the rest of the capacity and blocks and the node's children (their
  // subtree one level deeper); offset == len is a plain fork (tail -1), any
  // other offset must be a multiple of the block size.
  int32_t fork_at(int32_t node, int32_t offset, int32_t n, int32_t cap, int32_t* out, int32_t* tail,
                  std::string* err);
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
  // Bumped by new_root and fork only (appends change lengths, not shape).
  uint64_t shape_version() const { return shape_version_; }
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
  uint64_t shape_version_ = 0;
  std::vector<Node> nodes_;
};

// ---- decode plan -----------------------------------------------------------
//
// Cascade schedule (the nested descendant sub-groups of TreePO Sec. 2.3 as the
// unit of shared attention work): the chain nodes of the decoded leaves are
// cut into runs (maximal chain segments whose nodes have the same descendant
// leaves), every run is streamed once per KV head for the query rows of its
// descendant leaves, and the per-leaf results are merged by log-sum-exp.
//
// Work distribution: every (run, leaf group, KV head) contributes a sequence
// of 32-token KV tiles.  The sequences are concatenated and cut into streams
// of equal estimated cost, one stream per resident workgroup, so every
// workgroup streams the same amount of KV and its load pipeline runs across
// the pieces of its stream without draining.

enum PlanMode : int32_t { kModeTree = 0, kModeNaive = 1 };

// The combine reads the O rows of the first min(emax, 32) entries of every
// key before it knows the key's count when that costs at most this many
// bytes (one memory round trip); larger plans pack the entries and read
// exactly the rows each key holds.
constexpr int64_t kStridedCombineBytes = int64_t{8} << 20;

// Tokens per decode tile (32 consecutive rows of a node from a 16-row line of the pool).
constexpr int32_t kPlanTileTokens = 32;
// Upper bounds on the tiles, query segments and pieces of one stream (sized
// for the kernel's LDS copy of its stream block).  A piece holds at least one
// query tile and one KV tile.
constexpr int32_t kMaxStreamTiles = 256;
constexpr int32_t kMaxStreamSegs = 256;
constexpr int32_t kMaxStreamPieces = kMaxStreamTiles / 2;
// Live tiles (token count read on the device at decode time) of one stream.
constexpr int32_t kMaxStreamLive = kMaxStreamTiles;
// Query rows carried by one query tile (a tile buffer holds 64 rows of D).
constexpr int32_t kQTileRows = 64;
// Query rows of a piece that the column-split kernel path handles (two 16-row
// blocks); larger row groups use the row-split path.
constexpr int32_t kSplitMaxRows = 32;

// A piece: consecutive tiles of one (run, leaf group, KV head) sequence, all
// in one stream.  Rows are (leaf j of the group, head h' of the GQA group):
// row = j * G + h'.  In its stream's tile list a piece is n_qtiles query tiles
// (its query rows, 64 per tile) followed by n_tiles KV tiles.  It writes one
// partial row per query row, at the partial slot of its leaf's key (see
// Plan::dests).
struct Piece {
  int32_t rowset_begin;  // index into Plan::rowsets (the group's call positions)
  int32_t n_leaves;
  int32_t rows;          // n_leaves * G
  int32_t g;             // KV head
  int32_t tile_begin;    // its first query tile, index into the stream's tile list
  int32_t n_tiles;       // KV tiles
  int32_t reserved;      // 0
  int32_t seg_begin;     // its first query segment, index into the stream's segment list
  int32_t run;
  int32_t stream;
  int32_t plan_tile;     // index of its first KV tile in Plan::tiles
  int32_t n_qtiles;
  int32_t pad[4];
};
constexpr int32_t kPieceInts = 16;
static_assert(sizeof(Piece) == kPieceInts * sizeof(int32_t), "piece record size");

// A stream: pieces [piece_begin, piece_end) processed in order by one
// workgroup; its tiles are Plan::stream_tiles[tile_off, tile_off + n_tiles),
// its query segments Plan::segs[seg_off, seg_off + n_segs) and its live tiles
// Plan::live[2 live_off, 2 (live_off + n_live)).  tile_off is even and seg_off
// a multiple of 4; both arrays are padded so that a stream's lists can be
// read in 16-byte pieces.
struct Stream {
  int32_t piece_begin, piece_end;
  int32_t tile_off, n_tiles;
  int32_t seg_off, n_segs;
  int32_t live_off, n_live;
};
constexpr int32_t kStreamInts = 8;
static_assert(sizeof(Stream) == kStreamInts * sizeof(int32_t), "stream record size");

// Device record of a tile.  KV tile: hb = (first pool row of the tile, KV
// head g's g * num_blocks * B rows included) / 16 >= 0 locates its K and V
// data, valid = tokens holding data (1..32), or, for
// a live tile, valid = -1 - i: entry i = {node, base} of the stream's live
// table, and the tile holds min(32, max(0, len(node) - base)) tokens at decode
// time.  Query tile: hb = -1 - (the piece's first segment, stream-local),
// valid = row0 | (n_rows << 16): rows [row0, row0 + n_rows) of the piece.
struct StreamTile {
  int32_t hb;
  int32_t valid;
};

// Device copy of one stream, all a workgroup needs to run it: stream s is the
// block of block_ints int32 at s * block_ints (the same size for every stream
// of a plan, a multiple of 4 ints, so the kernel fetches it with one round of
// 16-byte loads from an address it computes itself):
//   [0, 4)                   n_pieces, n_tiles, n_segs, 0
//   [4, 4 + 4 n_pieces)      per piece: rows, tile_begin, n_tiles, seg_begin
//   then n_tiles StreamTile records (two ints each, padded to an even count)
//   then n_segs query segment offsets (padded to a multiple of 4)
//   then n_segs partial destinations, Plan::dests (padded to a multiple of 4)
//   then n_live live-tile entries {node, base} (header[3] = n_live)
constexpr int32_t kBlockHeaderInts = 4;
constexpr int32_t kBlockPieceInts = 4;
constexpr int32_t kMaxBlockInts = kBlockHeaderInts + kBlockPieceInts * kMaxStreamPieces + 2 * kMaxStreamTiles +
                                  2 * kMaxStreamSegs + 2 * kMaxStreamLive;

// Host record of a KV tile, for inspection: tokens [32 k, 32 k + 32) of node
// `node` (k = tile_in_node) in pool block `block` (= block_begin + k / 2).
struct Tile {
  int32_t block;
  int32_t node;
  int32_t tile_in_node;
  int32_t valid;
};

struct PlanParams {
  int32_t group;            // G = Hq / Hkv
  int32_t num_kv_heads;     // Hkv
  int32_t num_q_heads;      // Hq
  int32_t head_dim;         // D
  int64_t num_blocks;       // pool blocks per KV head
  int32_t max_rows;         // query rows of a piece at most (leaf groups are split to fit)
  int32_t concurrent_wgs;   // workgroups resident at once (streams per round)
  // Relative speed of a first-round stream by its slot on the CU.  The
  // dispatcher fills every CU's first slot before any second one, so stream s
  // runs in slot s / compute_units; streams are sized in proportion to
  // slot_speed[slot] (both 1.0: equal cost per stream).
  int32_t compute_units;
  double slot_speed[2];
  // Relative speed by accelerator die (XCD): workgroups are dealt to the
  // xcds dies round robin, so stream s runs on die s % xcds; stream sizes
  // (every round) are scaled by xcd_speed[s % xcds] (all 1.0: no scaling).
  int32_t xcds;
  double xcd_speed[8];
  // Lengths are read on the device: unfrozen nodes are planned up to their
  // capacity, tiles not yet full become live tiles.
  bool live_lengths;
};

struct Plan {
  PlanMode mode = kModeTree;
  std::vector<Stream> streams;
  std::vector<Piece> pieces;          // stream order
  std::vector<int32_t> rowsets;
  std::vector<StreamTile> stream_tiles;
  std::vector<Tile> tiles;            // host view of the KV tiles, piece order
  // Query segments: element offset in the query tensor of the G rows of one
  // leaf for one KV head (contiguous there), one per (piece, leaf).
  std::vector<int32_t> segs;
  // Live tiles: {node, base} per live tile, stream order.
  std::vector<int32_t> live;
  // The device copy of the streams (layout above kBlockHeaderInts).
  std::vector<int32_t> blocks;
  int32_t block_ints = 0;
  // Partial slots.  Key (leaf x, KV head g) = x * Hkv + g has comb_count[key]
  // entries (one per piece over its chain, in plan order, at most emax); entry
  // e holds the partial rows (comb_base[key] + e) * G + h' for query heads
  // g * G + h', with comb_base[key] = key * emax (strided) or the prefix sum
  // of the counts (compact: plans whose strided combine would read more than
  // kStridedCombineBytes in its speculative first round).  dests (parallel to
  // segs) gives, per (piece, leaf), the row of its entry's h' = 0.
  std::vector<int32_t> comb_count;
  std::vector<int32_t> comb_base;
  int32_t emax = 0;
  bool compact = false;
  std::vector<int32_t> dests;
  int64_t partial_rows = 0;
  int64_t unique_kv_tokens = 0;   // tokens streamed per KV head (tree: unique)
  int64_t kv_token_visits = 0;    // tokens streamed, summed over leaf groups (per KV head)
};

// Branching budget over n active paths (TreePO Sec. 2.2 budget transfer;
// Sec. 4.4 probability-based assignment): every path gets one branch, the
// other max(total - n, 0) are split in proportion to the weights by largest
// remainders (ties to the lower index).  Weights: 1/n (kBudgetEven),
// softmax(scores / T) (kBudgetHighProb) or softmax(-scores / T)
// (kBudgetLowProb), in double with the maximum subtracted.
enum BudgetMode : int32_t { kBudgetEven = 0, kBudgetHighProb = 1, kBudgetLowProb = 2 };
int32_t branch_budget(int32_t n, const float* scores, int32_t total, int32_t mode, double temperature,
                      int32_t* out, std::string* err);

// Builds the decode schedule for `leaves` (validated by the caller).
int32_t build_plan(const Tree& t, int32_t n_leaves, const int32_t* leaves, PlanMode mode,
                   const PlanParams& p, Plan* out, std::string* err);

// Node -> ascending call positions of the leaves whose chain contains it, for
// every node on some chain (ascending id).
void desc_sets(const Tree& t, int32_t n_leaves, const int32_t* leaves,
               std::vector<int32_t>* nodes, std::vector<int32_t>* off,
               std::vector<int32_t>* desc);

}  // namespace treepo
