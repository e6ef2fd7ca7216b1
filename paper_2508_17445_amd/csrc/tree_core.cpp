// Node table, block allocator and decode planner (host, C++17).
#include "tree_core.h"

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
  std::vector<int32_t> nodes;  // root-first
  std::vector<int32_t> leaves; // ascending call positions
  int32_t tile_begin = 0, tile_end = 0;
  int32_t group_leaves = 1;    // leaves per item group
  std::vector<std::vector<int32_t>> group_items;  // per group: item ids (pre-sort)
};

}  // namespace

int32_t build_plan(const Tree& t, int32_t n_leaves, const int32_t* leaves, PlanMode mode,
                   const PlanParams& p, Plan* out, std::string* err) {
  const auto& nd = t.nodes();
  const int32_t B = t.block_tokens();
  const int32_t G = p.group;
  if (G < 1 || G > (p.mfma_enabled ? p.mfma_max_rows : p.valu_max_rows)) {
    if (err) *err = "GQA group larger than the kernels' row limit";
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

  // ---- tiles -----------------------------------------------------------------
  for (Run& r : runs) {
    r.tile_begin = static_cast<int32_t>(out->tiles.size());
    for (int32_t n : r.nodes) {
      const int32_t ln = nd[n].len;
      constexpr int32_t T = kPlanTileTokens;
      const int32_t per_block = B / T;
      for (int32_t k = 0; k * T < ln; ++k) {
        Tile tl;
        tl.block = nd[n].block_begin + k / per_block;
        tl.node = n;
        tl.tile_in_node = k;
        tl.valid = std::min(T, ln - k * T);
        out->tiles.push_back(tl);
        out->unique_kv_tokens += tl.valid;
      }
    }
    r.tile_end = static_cast<int32_t>(out->tiles.size());
    const int32_t nl = static_cast<int32_t>(r.leaves.size());
    if (nl * G <= p.valu_max_rows) {
      r.group_leaves = nl;
    } else {
      // split the leaves evenly into the fewest groups that fit the row limit
      const int32_t lim = std::max(1, (p.mfma_enabled ? p.mfma_max_rows : p.valu_max_rows) / G);
      const int32_t ng = (nl + lim - 1) / lim;
      r.group_leaves = (nl + ng - 1) / ng;
    }
  }

  // ---- chunk size: minimise rounds x (tiles per item + one tile of overhead) --
  auto groups_of = [](const Run& r) {
    return (static_cast<int32_t>(r.leaves.size()) + r.group_leaves - 1) / r.group_leaves;
  };
  const int64_t S = std::max(1, p.concurrent_wgs);
  int32_t best_c = 1;
  double best_cost = 1e300;
  for (int32_t c = 1; c <= std::max(1, p.max_chunk_tiles); ++c) {
    int64_t w = 0;
    for (const Run& r : runs) {
      const int32_t nt = r.tile_end - r.tile_begin;
      if (nt == 0) continue;
      w += static_cast<int64_t>(groups_of(r)) * ((nt + c - 1) / c);
    }
    w *= p.num_kv_heads;
    const double cost = static_cast<double>((w + S - 1) / S) * (c + 1.0);
    if (cost <= best_cost) {
      best_cost = cost;
      best_c = c;
    }
  }
  out->chunk_tiles = best_c;

  // ---- items -----------------------------------------------------------------
  std::vector<Item> tmp;
  for (int32_t ri = 0; ri < static_cast<int32_t>(runs.size()); ++ri) {
    Run& r = runs[ri];
    const int32_t nt = r.tile_end - r.tile_begin;
    const int32_t ng = groups_of(r);
    r.group_items.assign(ng, {});
    if (nt == 0) continue;
    const int32_t nchunks = (nt + best_c - 1) / best_c;
    for (int32_t gi = 0; gi < ng; ++gi) {
      const int32_t l0 = gi * r.group_leaves;
      const int32_t l1 = std::min<int32_t>(static_cast<int32_t>(r.leaves.size()), l0 + r.group_leaves);
      const int32_t rs = static_cast<int32_t>(out->rowsets.size());
      for (int32_t l = l0; l < l1; ++l) out->rowsets.push_back(r.leaves[l]);
      for (int32_t c = 0; c < nchunks; ++c) {
        Item it;
        it.rowset_begin = rs;
        it.n_leaves = l1 - l0;
        it.rows = it.n_leaves * G;
        it.kind = it.rows <= p.valu_max_rows ? kKindValu : kKindMfma;
        it.tile_begin = r.tile_begin + static_cast<int32_t>(static_cast<int64_t>(nt) * c / nchunks);
        it.tile_end = r.tile_begin + static_cast<int32_t>(static_cast<int64_t>(nt) * (c + 1) / nchunks);
        it.partial_base = 0;
        it.run = ri;
        for (int32_t f = 0; f < 3; ++f) {
          const int32_t ti = it.tile_begin + f;
          it.first_src[f] = ti < it.tile_end ? 2 * out->tiles[ti].block + (out->tiles[ti].tile_in_node & 1) : -1;
        }
        it.pad = 0;
        r.group_items[gi].push_back(static_cast<int32_t>(tmp.size()));
        tmp.push_back(it);
      }
    }
  }
  // VALU items first, stable
  std::vector<int32_t> order(tmp.size()), newid(tmp.size());
  for (size_t i = 0; i < tmp.size(); ++i) order[i] = static_cast<int32_t>(i);
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t a, int32_t b) { return tmp[a].kind < tmp[b].kind; });
  int64_t base = 0;
  for (size_t k = 0; k < order.size(); ++k) {
    Item it = tmp[order[k]];
    if (base > INT32_MAX - static_cast<int64_t>(it.rows) * p.num_kv_heads) {
      if (err) *err = "too many partial rows";
      return kEUnsupported;
    }
    it.partial_base = static_cast<int32_t>(base);
    base += static_cast<int64_t>(it.rows) * p.num_kv_heads;
    newid[order[k]] = static_cast<int32_t>(k);
    if (it.kind == kKindValu) ++out->n_valu_items;
    for (int32_t ti = it.tile_begin; ti < it.tile_end; ++ti) out->kv_token_visits += out->tiles[ti].valid;
    out->items.push_back(it);
  }
  out->partial_rows = base;

  // ---- per-leaf combine entries, chain order -----------------------------------
  out->leaf_off.assign(n_leaves + 1, 0);
  std::vector<int32_t> ch;
  for (int32_t x = 0; x < n_leaves; ++x) {
    std::vector<int32_t> leaf_runs;
    if (mode == kModeTree) {
      t.chain(leaves[x], &ch);
      for (int32_t n : ch)
        if (leaf_runs.empty() || leaf_runs.back() != run_of[n]) leaf_runs.push_back(run_of[n]);
    } else {
      leaf_runs.push_back(x);
    }
    for (int32_t ri : leaf_runs) {
      const Run& r = runs[ri];
      const auto pos = std::lower_bound(r.leaves.begin(), r.leaves.end(), x) - r.leaves.begin();
      const int32_t gi = static_cast<int32_t>(pos) / r.group_leaves;
      const int32_t j = static_cast<int32_t>(pos) - gi * r.group_leaves;
      for (int32_t old : r.group_items[gi]) {
        const Item& it = out->items[newid[old]];
        out->entries.push_back(Entry{it.partial_base + j * G, it.rows});
      }
    }
    out->leaf_off[x + 1] = static_cast<int32_t>(out->entries.size());
  }
  return kOk;
}

}  // namespace treepo
