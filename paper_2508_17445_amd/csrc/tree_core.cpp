// Node table, block allocator and decode planner (host, C++17).
#include "tree_core.h"

#include <cmath>

#include <algorithm>
#include <unordered_map>

namespace treepo {

static int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

int32_t Tree::reserve_check(int32_t count, int32_t cap, std::string* err) const {
  if (cap < 1) {
    if (err) *err = "capacity must be >= 1 token";
    return kEInval;
  }
  if (count < 1) {
    if (err) *err = "child count must be >= 1";
    return kEInval;
  }
  if (static_cast<int64_t>(nodes_.size()) + count > max_nodes_) {
    if (err) *err = "node table full";
    return kENoMem;
  }
  const int64_t need = static_cast<int64_t>(count) * ceil_div64(cap, B_);
  if (next_block_ + need > num_blocks_) {
    if (err) *err = "pool blocks exhausted";
    return kENoMem;
  }
  return kOk;
}

int32_t Tree::make(int32_t parent, int32_t depth, int32_t start, int32_t cap, int32_t tree_id) {
  Node n;
  n.parent = parent;
  n.depth = depth;
  n.start = start;
  n.len = 0;
  n.cap = cap;
  n.block_begin = static_cast<int32_t>(next_block_);
  n.n_blocks = static_cast<int32_t>(ceil_div64(cap, B_));
  n.tree_id = tree_id;
  n.n_children = 0;
  next_block_ += n.n_blocks;
  nodes_.push_back(n);
  return static_cast<int32_t>(nodes_.size() - 1);
}

int32_t Tree::new_root(int32_t cap, int32_t* node_out, std::string* err) {
  if (!node_out) {
    if (err) *err = "null output pointer";
    return kEInval;
  }
  int32_t st = reserve_check(1, cap, err);
  if (st != kOk) return st;
  *node_out = make(-1, 0, 0, cap, n_roots_++);
  ++version_;
  ++shape_version_;
  return kOk;
}

int32_t Tree::fork(int32_t parent, int32_t n, int32_t cap, int32_t* out, std::string* err) {
  if (!out) {
    if (err) *err = "null output pointer";
    return kEInval;
  }
  if (parent < 0 || parent >= static_cast<int32_t>(nodes_.size())) {
    if (err) *err = "fork of an unknown node";
    return kEInval;
  }
  int32_t st = reserve_check(n, cap, err);
  if (st != kOk) return st;
  const Node p = nodes_[parent];
  for (int32_t i = 0; i < n; ++i) out[i] = make(parent, p.depth + 1, p.start + p.len, cap, p.tree_id);
  nodes_[parent].n_children += n;
  ++version_;
  ++shape_version_;
  return kOk;
}

int32_t Tree::fork_at(int32_t node, int32_t offset, int32_t n, int32_t cap, int32_t* out, int32_t* tail,
                      std::string* err) {
  if (!tail || (n > 0 && !out)) {
    if (err) *err = "null output pointer";
    return kEInval;
  }
  if (node < 0 || node >= static_cast<int32_t>(nodes_.size())) {
    if (err) *err = "fork of an unknown node";
    return kEInval;
  }
  const Node x = nodes_[node];
  if (offset < 0 || offset > x.len || n < 0) {
    if (err) *err = "split offset outside the node's tokens or negative child count";
    return kEInval;
  }
  if (offset == x.len) {
    int32_t st = fork(node, n, cap, out, err);
    if (st == kOk) *tail = -1;
    return st;
  }
  if (offset % B_ != 0) {
    if (err) *err = "split offset is not a multiple of the block size";
    return kEInval;
  }
  if (n > 0 && cap < 1) {
    if (err) *err = "capacity must be >= 1 token";
    return kEInval;
  }
  if (static_cast<int64_t>(nodes_.size()) + 1 + n > max_nodes_) {
    if (err) *err = "node table full";
    return kENoMem;
  }
  if (n > 0 && next_block_ + static_cast<int64_t>(n) * ceil_div64(cap, B_) > num_blocks_) {
    if (err) *err = "pool blocks exhausted";
    return kENoMem;
  }
  const int32_t keep = offset / B_;
  Node t;
  t.parent = node;
  t.depth = x.depth + 1;
  t.start = x.start + offset;
  t.len = x.len - offset;
  t.cap = x.cap - offset;
  t.block_begin = x.block_begin + keep;
  t.n_blocks = x.n_blocks - keep;
  t.tree_id = x.tree_id;
  t.n_children = x.n_children;
  nodes_.push_back(t);
  const int32_t tid = static_cast<int32_t>(nodes_.size() - 1);
  // the node's children move under the tail; their subtrees one level down
  std::vector<int32_t> stack;
  for (int32_t c = 0; c < tid; ++c)
    if (nodes_[c].parent == node) {
      nodes_[c].parent = tid;
      stack.push_back(c);
    }
  if (!stack.empty()) {
    std::vector<std::vector<int32_t>> kids(nodes_.size());
    for (int32_t c = 0; c < tid; ++c)
      if (nodes_[c].parent >= 0) kids[nodes_[c].parent].push_back(c);
    while (!stack.empty()) {
      const int32_t c = stack.back();
      stack.pop_back();
      ++nodes_[c].depth;
      for (int32_t d : kids[c]) stack.push_back(d);
    }
  }
  nodes_[node].len = offset;
  nodes_[node].cap = offset;
  nodes_[node].n_blocks = keep;
  nodes_[node].n_children = 1;
  ++version_;
  ++shape_version_;
  *tail = tid;
  if (n > 0) return fork(node, n, cap, out, err);  // checked above: cannot fail
  return kOk;
}

int32_t Tree::check_append(int32_t n, const int32_t* nodes, const int32_t* ntok,
                           std::vector<int64_t>* dest_rows, std::string* err) const {
  if (n < 0 || (n > 0 && (!nodes || !ntok))) {
    if (err) *err = "bad append arrays";
    return kEInval;
  }
  std::unordered_map<int32_t, int32_t> pending;
  if (dest_rows) dest_rows->clear();
  for (int32_t i = 0; i < n; ++i) {
    const int32_t nd = nodes[i];
    if (nd < 0 || nd >= static_cast<int32_t>(nodes_.size()) || ntok[i] < 0) {
      if (err) *err = "append to an unknown node or negative token count";
      return kEInval;
    }
    const Node& node = nodes_[nd];
    if (node.n_children > 0) {
      if (err) *err = "append to a node that has children";
      return kEFrozen;
    }
    auto it = pending.find(nd);
    const int32_t cur = it == pending.end() ? node.len : it->second;
    if (static_cast<int64_t>(cur) + ntok[i] > node.cap) {
      if (err) *err = "append past the node's capacity";
      return kEFull;
    }
    if (dest_rows) {
      const int64_t base = static_cast<int64_t>(node.block_begin) * B_ + cur;
      for (int32_t k = 0; k < ntok[i]; ++k) dest_rows->push_back(base + k);
    }
    pending[nd] = cur + ntok[i];
  }
  return kOk;
}

void Tree::apply_append(int32_t n, const int32_t* nodes, const int32_t* ntok) {
  for (int32_t i = 0; i < n; ++i) nodes_[nodes[i]].len += ntok[i];
  if (n > 0) ++version_;
}

void Tree::chain(int32_t x, std::vector<int32_t>* out) const {
  out->clear();
  for (int32_t y = x; y != -1; y = nodes_[y].parent) out->push_back(y);
  std::reverse(out->begin(), out->end());
}

int64_t Tree::chain_tokens(int32_t x) const {
  int64_t s = 0;
  for (int32_t y = x; y != -1; y = nodes_[y].parent) s += nodes_[y].len;
  return s;
}

int32_t Tree::check_leaves(int32_t n, const int32_t* leaves, std::string* err) const {
  if (n < 1 || !leaves) {
    if (err) *err = "need at least one leaf";
    return kEInval;
  }
  for (int32_t i = 0; i < n; ++i) {
    if (leaves[i] < 0 || leaves[i] >= static_cast<int32_t>(nodes_.size())) {
      if (err) *err = "unknown leaf id";
      return kEInval;
    }
  }
  for (int32_t i = 0; i < n; ++i) {
    if (chain_tokens(leaves[i]) == 0) {
      if (err) *err = "a leaf's chain holds no tokens";
      return kEEmpty;
    }
  }
  return kOk;
}

int32_t branch_budget(int32_t n, const float* scores, int32_t total, int32_t mode, double temperature,
                      int32_t* out, std::string* err) {
  if (n < 1 || !out || total < 0) {
    if (err) *err = "need at least one path, an output array and a non-negative total";
    return kEInval;
  }
  if (mode != kBudgetEven && mode != kBudgetHighProb && mode != kBudgetLowProb) {
    if (err) *err = "bad budget mode";
    return kEInval;
  }
  std::vector<double> w(n);
  if (mode == kBudgetEven) {
    for (double& x : w) x = 1.0 / n;
  } else {
    if (!scores || !(temperature > 0.0) || !std::isfinite(temperature)) {
      if (err) *err = "probability modes need scores and a positive finite temperature";
      return kEInval;
    }
    const double sign = mode == kBudgetHighProb ? 1.0 : -1.0;
    double m = -INFINITY;
    for (int32_t k = 0; k < n; ++k) {
      if (!std::isfinite(scores[k])) {
        if (err) *err = "scores must be finite";
        return kEInval;
      }
      w[k] = sign * static_cast<double>(scores[k]) / temperature;
      m = std::max(m, w[k]);
    }
    double tot = 0.0;
    for (double& x : w) {
      x = std::exp(x - m);
      tot += x;
    }
    for (double& x : w) x /= tot;
  }
  const int32_t rest = std::max(total - n, 0);
  std::vector<double> frac(n);
  int64_t left = rest;
  for (int32_t k = 0; k < n; ++k) {
    const double q = rest * w[k];
    const double f = std::floor(q);
    out[k] = 1 + static_cast<int32_t>(f);
    frac[k] = q - f;
    left -= static_cast<int64_t>(f);
  }
  std::vector<int32_t> order(n);
  for (int32_t k = 0; k < n; ++k) order[k] = k;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return frac[a] > frac[b]; });
  for (int64_t i = 0; i < left && i < n; ++i) ++out[order[i]];
  return kOk;
}

void desc_sets(const Tree& t, int32_t n_leaves, const int32_t* leaves, std::vector<int32_t>* nodes,
               std::vector<int32_t>* off, std::vector<int32_t>* desc) {
  const auto& nd = t.nodes();
  std::vector<int32_t> count(nd.size(), 0);
  nodes->clear();
  for (int32_t x = 0; x < n_leaves; ++x)
    for (int32_t y = leaves[x]; y != -1; y = nd[y].parent)
      if (count[y]++ == 0) nodes->push_back(y);
  std::sort(nodes->begin(), nodes->end());
  std::vector<int32_t> cursor(nd.size(), 0);
  off->assign(nodes->size() + 1, 0);
  for (size_t i = 0; i < nodes->size(); ++i) {
    (*off)[i + 1] = (*off)[i] + count[(*nodes)[i]];
    cursor[(*nodes)[i]] = (*off)[i];
  }
  desc->assign(off->back(), 0);
  for (int32_t x = 0; x < n_leaves; ++x)
    for (int32_t y = leaves[x]; y != -1; y = nd[y].parent) (*desc)[cursor[y]++] = x;
}

namespace {

struct Run {
  std::vector<int32_t> nodes;   // root-first
  std::vector<int32_t> leaves;  // ascending call positions
  std::vector<Tile> tiles;
  std::vector<char> live;       // per tile: token count read at decode time
  double weight = 0.0;          // tiles, an empty live tile counting kLiveEmptyWeight
  int32_t group_leaves = 1;     // leaves per group
};

// A piece's query tile takes a step of the tile pipeline like a KV tile (the
// loads of 64 rows, repeats of the last row for a small piece) but no
// matrix work; with the piece's start and end (partial-row stores, softmax
// state reset) it costs about 1.2 KV tiles: a least-squares fit of
// per-workgroup end times of decodes of a 16-leaf tree (leaves of 7680 tokens,
// 35 launches) to the streams' tile and piece counts gave 1.22 per piece
// with tile costs within 0.1 of tile_cost below.
constexpr double kQTileCost = 1.2;
// Guided stream sizes when the work takes several rounds of workgroups.
constexpr double kGuide = 2.0;
// Snapping of guided streams to sequence boundaries (fractions of the
// stream's size): finish a sequence whose remaining cost is at most
// kSnapFinish, close before a new sequence within kSnapEarly of the size.
// Partial rows written by the decode kernel cost far more than their bytes
// (they reach memory while the KV stream is read: removing them entirely
// made the 64-prompt batch rollout's kernel 16% faster), so fewer cuts pay
// for less even stream sizes.  Measured against no snapping, kernel time of
// the batch rollout, the irregular 32-prompt tree and the 16k-token
// long-context tree: -2.5%, -1.4%, -2.7% at (1.0, 0.5); (0.5, 0.25) gave
// -2.4%, -2.4%, +4%.
constexpr double kSnapFinish = 1.0;
constexpr double kSnapEarly = 0.5;
constexpr double kGuideMinCost = 8.0;
// A live tile empty at planning time costs a few loads and no compute until it
// fills; the plan serves a whole segment, so it is weighted at about its
// average over the segment.
constexpr double kLiveEmptyWeight = 0.5;

// Estimated cost of one KV tile for a piece of `rows` query rows, in units of
// one tile's load time at full load (fitted to per-workgroup timestamps and
// swept on the five workloads): the token-split path hides its compute under
// the loads (1.0 for one 16-row block, 1.1 for two); the row-split path takes
// about 1.4 (one 16-row block per wave) and 2.6 (two per wave) times as long.
double tile_cost(int32_t rows) { return rows <= 16 ? 1.0 : rows <= 32 ? 1.1 : rows <= 64 ? 1.4 : 2.6; }

}  // namespace

int32_t build_plan(const Tree& t, int32_t n_leaves, const int32_t* leaves, PlanMode mode,
                   const PlanParams& p, Plan* out, std::string* err) {
  const auto& nd = t.nodes();
  const int32_t B = t.block_tokens();
  const int32_t G = p.group;
  const int32_t Hkv = p.num_kv_heads;
  if (G < 1 || G > p.max_rows) {
    if (err) *err = "GQA group larger than the kernels' row limit";
    return kEUnsupported;
  }
  if (static_cast<int64_t>(Hkv) * p.num_blocks * B / 16 > INT32_MAX ||
      static_cast<int64_t>(n_leaves) * p.num_q_heads * p.head_dim > INT32_MAX) {
    if (err) *err = "pool or query tensor too large for 32-bit tile and row offsets";
    return kEUnsupported;
  }
  *out = Plan();
  out->mode = mode;

  // ---- runs ------------------------------------------------------------------
  std::vector<Run> runs;
  std::vector<int32_t> run_of(nd.size(), -1);
  if (mode == kModeTree) {
    std::vector<int32_t> nodes, off, desc;
    desc_sets(t, n_leaves, leaves, &nodes, &off, &desc);
    std::vector<int32_t> dcount(nd.size(), 0);
    for (size_t i = 0; i < nodes.size(); ++i) dcount[nodes[i]] = off[i + 1] - off[i];
    for (size_t i = 0; i < nodes.size(); ++i) {
      const int32_t n = nodes[i];
      const int32_t par = nd[n].parent;
      // a node whose parent has the same descendant leaves continues its run
      if (par >= 0 && run_of[par] >= 0 && dcount[par] == dcount[n]) {
        run_of[n] = run_of[par];
        runs[run_of[n]].nodes.push_back(n);
      } else {
        run_of[n] = static_cast<int32_t>(runs.size());
        Run r;
        r.nodes.push_back(n);
        r.leaves.assign(desc.begin() + off[i], desc.begin() + off[i + 1]);
        runs.push_back(std::move(r));
      }
    }
  } else {
    std::vector<int32_t> ch;
    for (int32_t x = 0; x < n_leaves; ++x) {
      t.chain(leaves[x], &ch);
      Run r;
      r.nodes = ch;
      r.leaves.push_back(x);
      runs.push_back(std::move(r));
    }
  }

  // ---- tiles and leaf groups ---------------------------------------------------
  for (Run& r : runs) {
    for (int32_t n : r.nodes) {
      const int32_t ln = nd[n].len;
      constexpr int32_t T = kPlanTileTokens;
      // with device lengths an unfrozen node is planned up to its capacity
      const bool grows = p.live_lengths && nd[n].n_children == 0 && ln < nd[n].cap;
      const int32_t span = grows ? nd[n].cap : ln;
      for (int32_t k = 0; k * T < span; ++k) {
        Tile tl;
        tl.block = nd[n].block_begin + k * T / B;  // the block of the tile's first token
        tl.node = n;
        tl.tile_in_node = k;
        tl.valid = std::max(0, std::min(T, ln - k * T));
        const bool live = grows && (k + 1) * T > ln;
        r.tiles.push_back(tl);
        r.live.push_back(live ? 1 : 0);
        r.weight += live && tl.valid == 0 ? kLiveEmptyWeight : 1.0;
        out->unique_kv_tokens += tl.valid;
      }
    }
    const int32_t nl = static_cast<int32_t>(r.leaves.size());
    // split the leaves evenly into the fewest groups that fit the row limit
    const int32_t lim = std::max(1, p.max_rows / G);
    const int32_t ng = (nl + lim - 1) / lim;
    r.group_leaves = (nl + ng - 1) / ng;
  }

  // ---- sequences: (run, leaf group, KV head) -------------------------------------
  struct Seq {
    int32_t run, rowset_begin, n_leaves, g;
  };
  std::vector<Seq> seqs;
  double total_cost = 0.0;
  int64_t total_tiles = 0;
  for (int32_t ri = 0; ri < static_cast<int32_t>(runs.size()); ++ri) {
    const Run& r = runs[ri];
    if (r.tiles.empty()) continue;
    const int32_t nl = static_cast<int32_t>(r.leaves.size());
    for (int32_t l0 = 0; l0 < nl; l0 += r.group_leaves) {
      const int32_t l1 = std::min(nl, l0 + r.group_leaves);
      const int32_t rs = static_cast<int32_t>(out->rowsets.size());
      for (int32_t l = l0; l < l1; ++l) out->rowsets.push_back(r.leaves[l]);
      int64_t tok = 0;
      for (const Tile& tl : r.tiles) tok += tl.valid;
      out->kv_token_visits += tok;
      for (int32_t g = 0; g < Hkv; ++g) {
        seqs.push_back(Seq{ri, rs, l1 - l0, g});
        total_cost += tile_cost((l1 - l0) * G) * r.weight +
                      kQTileCost * ((l1 - l0) * G + kQTileRows - 1) / kQTileRows;
        total_tiles += static_cast<int64_t>(r.tiles.size());
      }
    }
  }
  if (total_tiles == 0) {
    if (err) *err = "no KV tokens on the leaves' chains";
    return kEEmpty;
  }

  // ---- streams ------------------------------------------------------------------
  // One round (every stream resident at once): the concatenated sequences are
  // cut at equal cumulative cost, each stream's share in proportion to its
  // slot's and its die's speed.  Several rounds: later streams start wherever
  // a slot of their die frees up, so the hardware dispatcher balances them
  // within a die; stream sizes shrink with the work left (each takes 1/kGuide
  // of an even share of the remainder, scaled by its die's speed, between
  // kGuideMinCost and a full LDS table), so the last streams to start are
  // short and the slots drain together.
  const int64_t S0 = std::max(1, p.concurrent_wgs);
  const int32_t nx = p.xcds >= 1 && p.xcds <= 8 ? p.xcds : 1;
  auto xcd_speed = [&](int64_t s) { return nx > 1 ? p.xcd_speed[s % nx] : 1.0; };
  double xcd_mean = 0.0;
  for (int32_t x = 0; x < nx; ++x) xcd_mean += xcd_speed(x);
  xcd_mean /= nx;
  const double full_stream = 3 * kMaxStreamTiles / 4;
  const bool one_round = total_cost <= static_cast<double>(S0) * full_stream;
  const int64_t planned = one_round ? std::min<int64_t>(total_tiles, S0) : INT64_MAX;
  // One round: stream s closes once the running cost passes quota[s], its
  // share of the total cost in proportion to its slot's and die's speed.  The
  // query tiles that a stream starting inside a sequence loads again are left
  // out of the running cost (each stream has about one such start), so the
  // last stream's share stays proportional.
  std::vector<double> quota;
  if (one_round) {
    quota.resize(static_cast<size_t>(planned));
    std::vector<double> w(static_cast<size_t>(planned), 1.0);
    if (p.compute_units > 0)
      for (int64_t s = 0; s < planned; ++s) w[s] = p.slot_speed[s < p.compute_units ? 0 : 1];
    for (int64_t s = 0; s < planned; ++s) w[s] *= xcd_speed(s);
    double wsum = 0.0;
    for (double x : w) wsum += x;
    double cum = 0.0;
    for (int64_t s = 0; s < planned; ++s) {
      cum += w[s];
      quota[s] = total_cost * cum / wsum;
    }
  }
  // Several rounds: the open stream closes once the running cost reaches
  // guided_end; its size follows the KV work not yet assigned (kv_acc counts
  // KV tiles only, as total_kv_cost does).
  double total_kv_cost = 0.0, kv_acc = 0.0, guided_end = 0.0;
  for (const Seq& sq : seqs) total_kv_cost += tile_cost(sq.n_leaves * G) * runs[sq.run].weight;
  auto guided_quota = [&](double acc_now) {
    const double speed = xcd_speed(static_cast<int64_t>(out->streams.size()) - 1) / xcd_mean;  // the open stream
    const double share = speed * (total_kv_cost - kv_acc) / (kGuide * static_cast<double>(S0));
    return acc_now + std::min(full_stream, std::max(kGuideMinCost, share));
  };
  double acc = 0.0;
  double stream_begin = 0.0;  // running cost when the open stream was opened
  auto pad_to = [](auto* v, size_t m, auto fill) {
    while (v->size() % m) v->push_back(fill);
  };
  auto open_stream = [&]() {
    pad_to(&out->stream_tiles, 2, StreamTile{0, 0});
    pad_to(&out->segs, 4, 0);
    Stream st{};
    st.piece_begin = st.piece_end = static_cast<int32_t>(out->pieces.size());
    st.tile_off = static_cast<int32_t>(out->stream_tiles.size());
    st.seg_off = static_cast<int32_t>(out->segs.size());
    st.live_off = static_cast<int32_t>(out->live.size() / 2);
    out->streams.push_back(st);
  };
  open_stream();
  if (!one_round) guided_end = guided_quota(0.0);
  for (int32_t si = 0; si < static_cast<int32_t>(seqs.size()); ++si) {
    const Seq& sq = seqs[si];
    const Run& r = runs[sq.run];
    const int32_t rows = sq.n_leaves * G;
    const int32_t nq = (rows + kQTileRows - 1) / kQTileRows;
    const double c = tile_cost(rows);
    bool new_piece = true;
    for (size_t ti = 0; ti < r.tiles.size(); ++ti) {
      const Tile& tl = r.tiles[ti];
      const bool live = r.live[ti] != 0;
      Stream* st = &out->streams.back();
      const int64_t s = static_cast<int64_t>(out->streams.size()) - 1;
      bool full;
      if (one_round) {
        full = s + 1 < planned && acc >= quota[s];
      } else {
        // Several rounds: a stream that cuts a sequence makes its rows a
        // second partial entry (and query tile), so streams snap to sequence
        // boundaries: one that reaches its size inside a sequence finishes
        // it when little is left, and one close to its size closes before a
        // new sequence.
        const double size = guided_end - stream_begin;
        full = acc >= guided_end;
        if (full && ti > 0 && c * static_cast<double>(r.tiles.size() - ti) <= kSnapFinish * size) full = false;
        if (!full && ti == 0 && acc >= guided_end - kSnapEarly * size) full = true;
      }
      const bool room = st->n_tiles + (new_piece ? nq + 1 : 1) <= kMaxStreamTiles &&
                        st->n_segs + (new_piece ? sq.n_leaves : 0) <= kMaxStreamSegs &&
                        st->piece_end - st->piece_begin + (new_piece ? 1 : 0) <= kMaxStreamPieces &&
                        st->n_live + (live ? 1 : 0) <= kMaxStreamLive;
      if (st->n_tiles > 0 && (full || !room)) {
        open_stream();
        st = &out->streams.back();
        new_piece = true;
        if (!one_round) {
          guided_end = guided_quota(acc);
          stream_begin = acc;
        }
      }
      if (new_piece) {
        Piece pc{};
        pc.rowset_begin = sq.rowset_begin;
        pc.n_leaves = sq.n_leaves;
        pc.rows = rows;
        pc.g = sq.g;
        pc.tile_begin = st->n_tiles;
        pc.n_tiles = 0;
        pc.seg_begin = st->n_segs;
        pc.run = sq.run;
        pc.stream = static_cast<int32_t>(out->streams.size()) - 1;
        pc.plan_tile = static_cast<int32_t>(out->tiles.size());
        pc.n_qtiles = nq;
        for (int32_t j = 0; j < sq.n_leaves; ++j) {
          const int32_t x = out->rowsets[sq.rowset_begin + j];
          out->segs.push_back((x * p.num_q_heads + sq.g * G) * p.head_dim);
        }
        st->n_segs += sq.n_leaves;
        for (int32_t t = 0; t < nq; ++t) {
          const int32_t row0 = t * kQTileRows;
          const int32_t n = std::min(kQTileRows, rows - row0);
          out->stream_tiles.push_back(StreamTile{-1 - pc.seg_begin, row0 | (n << 16)});
        }
        st->n_tiles += nq;
        // the sequence's own query tiles are part of total_cost; those a cut
        // piece loads again are a per-stream overhead left out of the running
        // cost (one-round quotas are fractions of total_cost)
        if (ti == 0) acc += kQTileCost * nq;
        out->pieces.push_back(pc);
        st->piece_end = static_cast<int32_t>(out->pieces.size());
        new_piece = false;
      }
      // first pool row of the tile over 16, KV head g's rows included
      const int64_t row = (static_cast<int64_t>(sq.g) * p.num_blocks + nd[tl.node].block_begin) * B +
                          static_cast<int64_t>(tl.tile_in_node) * kPlanTileTokens;
      int32_t valid = tl.valid;
      if (live) {
        valid = -1 - st->n_live++;
        out->live.push_back(tl.node);
        out->live.push_back(tl.tile_in_node * kPlanTileTokens);
      }
      out->stream_tiles.push_back(
          StreamTile{static_cast<int32_t>(row / 16), valid});
      out->tiles.push_back(tl);
      ++st->n_tiles;
      ++out->pieces.back().n_tiles;
      const double w = live && tl.valid == 0 ? kLiveEmptyWeight : 1.0;
      acc += c * w;
      kv_acc += c * w;
    }
  }
  pad_to(&out->stream_tiles, 2, StreamTile{0, 0});
  pad_to(&out->segs, 4, 0);

  // ---- partial slots: entry e of key (leaf x, KV head g) -------------------------------
  // Every piece adds one entry to each of its leaves' keys, in piece order (the
  // fixed merge order); entry e of key k holds rows (base[k] + e) * G + h'.
  // Strided layout (base[k] = k * emax) when the combine's speculative first
  // round (the O rows of min(emax, 32) entries of every key) reads little;
  // else compact (base = the prefix sum of the counts).
  const int64_t nkeys = static_cast<int64_t>(n_leaves) * Hkv;
  out->comb_count.assign(nkeys, 0);
  for (const Piece& pc : out->pieces)
    for (int32_t j = 0; j < pc.n_leaves; ++j)
      ++out->comb_count[static_cast<int64_t>(out->rowsets[pc.rowset_begin + j]) * Hkv + pc.g];
  out->emax = 1;
  int64_t entries = 0;
  for (int32_t c : out->comb_count) {
    out->emax = std::max(out->emax, c);
    entries += c;
  }
  const int64_t spec_bytes = nkeys * G * std::min(out->emax, 32) * (static_cast<int64_t>(p.head_dim) * 4 + 8);
  out->compact = spec_bytes > kStridedCombineBytes;
  out->comb_base.assign(nkeys, 0);
  int64_t acc_e = 0;
  for (int64_t k = 0; k < nkeys; ++k) {
    out->comb_base[k] = static_cast<int32_t>(out->compact ? acc_e : k * out->emax);
    acc_e += out->comb_count[k];
  }
  out->partial_rows = (out->compact ? entries : nkeys * out->emax) * G;
  if (out->partial_rows > INT32_MAX) {
    if (err) *err = "too many partial rows";
    return kEUnsupported;
  }
  out->dests.assign(out->segs.size(), 0);
  {
    std::vector<int32_t> next(nkeys, 0);
    for (const Piece& pc : out->pieces) {
      const Stream& st = out->streams[pc.stream];
      for (int32_t j = 0; j < pc.n_leaves; ++j) {
        const int64_t key = static_cast<int64_t>(out->rowsets[pc.rowset_begin + j]) * Hkv + pc.g;
        out->dests[st.seg_off + pc.seg_begin + j] = static_cast<int32_t>((out->comb_base[key] + next[key]++) * G);
      }
    }
  }

  // ---- stream blocks ----------------------------------------------------------------
  auto round_up = [](int32_t x, int32_t m) { return (x + m - 1) / m * m; };
  int32_t bi = kBlockHeaderInts;
  for (const Stream& st : out->streams)
    bi = std::max(bi, kBlockHeaderInts + kBlockPieceInts * (st.piece_end - st.piece_begin) +
                          2 * round_up(st.n_tiles, 2) + 2 * round_up(st.n_segs, 4) + 2 * st.n_live);
  out->block_ints = round_up(bi, 4);
  out->blocks.assign(out->streams.size() * static_cast<size_t>(out->block_ints), 0);
  for (size_t si = 0; si < out->streams.size(); ++si) {
    const Stream& st = out->streams[si];
    int32_t* b = &out->blocks[si * out->block_ints];
    const int32_t np = st.piece_end - st.piece_begin;
    b[0] = np;
    b[1] = st.n_tiles;
    b[2] = st.n_segs;
    b[3] = st.n_live;
    int32_t* w = b + kBlockHeaderInts;
    for (int32_t i = st.piece_begin; i < st.piece_end; ++i) {
      const Piece& pc = out->pieces[i];
      *w++ = pc.rows;
      *w++ = pc.tile_begin;
      *w++ = pc.n_tiles;
      *w++ = pc.seg_begin;
    }
    for (int32_t k = 0; k < st.n_tiles; ++k) {
      *w++ = out->stream_tiles[st.tile_off + k].hb;
      *w++ = out->stream_tiles[st.tile_off + k].valid;
    }
    w += 2 * (round_up(st.n_tiles, 2) - st.n_tiles);
    for (int32_t k = 0; k < st.n_segs; ++k) w[k] = out->segs[st.seg_off + k];
    w += round_up(st.n_segs, 4);
    for (int32_t k = 0; k < st.n_segs; ++k) w[k] = out->dests[st.seg_off + k];
    w += round_up(st.n_segs, 4);
    for (int32_t k = 0; k < 2 * st.n_live; ++k) w[k] = out->live[2 * st.live_off + k];
  }

  return kOk;
}

}  // namespace treepo
