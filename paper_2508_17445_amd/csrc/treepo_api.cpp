// C-ABI of the segment-tree decode-attention library: argument validation,
// plan caching (each cached plan's device image in memory the context owns,
// uploaded through pinned staging), kernel launches on the caller's stream,
// metadata export and kernel timing.
#include "treepo.h"

#include <algorithm>
#include <array>
#include <atomic>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "kernels.h"
#include "tree_core.h"

using treepo::Plan;
using treepo::PlanMode;
using treepo::PlanParams;

namespace {

constexpr size_t kAlign = 256;
constexpr int kPlanCache = 4;
constexpr int kRing = 4;

// Machine shape when no device is visible (host-only use): MI355X, 256
// compute units in 8 XCDs of 32.
constexpr int32_t kDefaultComputeUnits = 256;
constexpr int32_t kComputeUnitsPerXcd = 32;
// Planner tunables, fitted to per-workgroup timestamps of back-to-back
// decodes of a 16-leaf tree (leaves of 7680 tokens): the second workgroup on a CU
// progressed about 0.80 as fast as the first (the dispatcher fills every CU's
// first slot before any second one), and the odd-numbered XCDs streamed
// 0.93-0.94 as many tiles per microsecond as the even ones on every box
// measured.  Streams are sized in proportion to these speeds.
constexpr double kSecondSlotSpeed = 0.80;
constexpr double kOddXcdSpeed = 0.935;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

std::atomic<uint64_t> g_plan_uid{0};

struct CachedPlan {
  uint64_t uid = 0;  // process-unique id of this plan build
  uint64_t version = 0;
  int32_t mode = 0;
  std::vector<int32_t> leaves;
  Plan plan;
  std::vector<char> blob;  // host image of the plan's device data
  size_t off_blocks = 0;
  size_t off_comb = 0;
  size_t off_part_o = 0, off_part_ml = 0, ws_bytes = 0;  // partials, in the caller's workspace
  uint64_t last_use = 0;
  // Device copy of `blob` in memory the context owns.  Uploaded on the first
  // decode with the plan, on that call's stream; decodes on other streams
  // wait for the upload's event.  No event follows each decode: when the plan
  // leaves the cache its buffer is retired with one event recorded on the
  // stream of its last decode (see RetiredImage).
  void* dev = nullptr;
  size_t dev_cap = 0;
  bool dev_valid = false;
  hipStream_t up_stream = nullptr;
  hipEvent_t up_ev = nullptr;
  hipStream_t last_stream = nullptr;  // stream of the latest decode with this plan
  bool multi_stream = false;          // read on more than one stream
};

// A plan image buffer no longer in the cache: reused for a new plan, or
// freed, once `ev` (recorded after every decode that read it; null if none
// did) has completed.
struct RetiredImage {
  void* dev;
  size_t cap;
  hipEvent_t ev;
};
constexpr size_t kMaxRetired = 8;

struct PinnedSlot {
  void* p = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};

// Index arrays of the advantage kernel for a leaf list, as one int32 image
// (uploaded into the workspace), plus the scratch that follows it.
struct AdvPlan {
  std::vector<int32_t> ints;
  int32_t n_groups = 0;
  size_t off_grp_off = 0, off_grp_mem = 0, off_pos_off = 0, off_pos_grp = 0, off_pos_root = 0;  // in ints
  size_t off_gmean = 0, off_gkeep = 0, off_pooled = 0, ws_bytes = 0;                           // in bytes
  uint64_t shape_version = 0;  // the tree shape it was built for
  std::vector<int32_t> leaves;
};

struct TimedLaunch {
  int kind;
  hipEvent_t start, stop;
};

}  // namespace

struct treepo_ctx {
  treepo_config cfg;
  treepo::Tree tree;
  PlanParams params;
  std::string last_error;
  std::vector<CachedPlan> plans;
  uint64_t clock = 0;
  std::array<PinnedSlot, kRing> ring;
  int ring_next = 0;
  bool profiling = false;
  std::vector<TimedLaunch> timed;
  std::vector<hipEvent_t> spare_events;
  std::vector<RetiredImage> retired;
  AdvPlan adv;  // the last advantage call's index arrays (reused for the same shape and leaves)
  // Device lengths (cfg.node_len): stale after kv_commit, new_root or fork;
  // the next decode uploads the host table on its stream.
  bool live = false;
  bool dev_len_stale = true;
  std::vector<int32_t> len_stage;  // host lengths of the last pageable upload (no-alloc decode)
  double prof_ms[TREEPO_KERNEL_KINDS] = {};
  int64_t prof_n[TREEPO_KERNEL_KINDS] = {};

  treepo_ctx(const treepo_config& c)
      : cfg(c), tree(c.block_tokens, c.num_blocks, c.max_nodes) {}
};

namespace {

// Pool rows per KV head.
int64_t pool_rows(const treepo_ctx* ctx) {
  return static_cast<int64_t>(ctx->cfg.num_blocks) * ctx->cfg.block_tokens;
}

int32_t fail(treepo_ctx* ctx, int32_t code, const std::string& msg) {
  if (ctx) ctx->last_error = msg;
  return code;
}

int32_t hip_fail(treepo_ctx* ctx, hipError_t e, const char* what) {
  return fail(ctx, TREEPO_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

hipError_t get_event(treepo_ctx* ctx, hipEvent_t* ev) {
  if (!ctx->spare_events.empty()) {
    *ev = ctx->spare_events.back();
    ctx->spare_events.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(ev);
}

hipError_t drain_timings(treepo_ctx* ctx) {
  for (const TimedLaunch& t : ctx->timed) {
    hipError_t e = hipEventSynchronize(t.stop);
    if (e != hipSuccess) return e;
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, t.start, t.stop);
    if (e != hipSuccess) return e;
    ctx->prof_ms[t.kind] += ms;
    ctx->prof_n[t.kind] += 1;
    ctx->spare_events.push_back(t.start);
    ctx->spare_events.push_back(t.stop);
  }
  ctx->timed.clear();
  return hipSuccess;
}

// Runs `launch(start, stop)`; with profiling on it gets two timing events
// that the launch attaches to its kernel (recorded at the kernel's own start
// and end), otherwise two null events.
template <class F>
hipError_t timed_launch_attached(treepo_ctx* ctx, int kind, F launch) {
  if (!ctx->profiling) return launch(nullptr, nullptr);
  if (ctx->timed.size() > 8192) {
    hipError_t e = drain_timings(ctx);
    if (e != hipSuccess) return e;
  }
  TimedLaunch t{kind, nullptr, nullptr};
  hipError_t e = get_event(ctx, &t.start);
  if (e == hipSuccess) e = get_event(ctx, &t.stop);
  if (e != hipSuccess) return e;
  e = launch(t.start, t.stop);
  if (e != hipSuccess) return e;
  ctx->timed.push_back(t);
  return hipSuccess;
}

// Runs `launch` bracketed by events when profiling is on.
template <class F>
hipError_t timed_launch(treepo_ctx* ctx, int kind, hipStream_t s, F launch) {
  if (!ctx->profiling) return launch();
  if (ctx->timed.size() > 8192) {
    hipError_t e = drain_timings(ctx);
    if (e != hipSuccess) return e;
  }
  TimedLaunch t{kind, nullptr, nullptr};
  hipError_t e = get_event(ctx, &t.start);
  if (e == hipSuccess) e = get_event(ctx, &t.stop);
  if (e == hipSuccess) e = hipEventRecord(t.start, s);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(t.stop, s);
  if (e != hipSuccess) return e;
  ctx->timed.push_back(t);
  return hipSuccess;
}

// Copies `bytes` of host data to device `dst` on `s` through a pinned slot.
hipError_t upload(treepo_ctx* ctx, void* dst, const void* src, size_t bytes, hipStream_t s) {
  PinnedSlot& sl = ctx->ring[ctx->ring_next];
  ctx->ring_next = (ctx->ring_next + 1) % kRing;
  hipError_t e;
  if (sl.pending) {
    e = hipEventSynchronize(sl.ev);
    if (e != hipSuccess) return e;
    sl.pending = false;
  }
  if (!sl.ev) {
    e = hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming);
    if (e != hipSuccess) return e;
  }
  if (sl.cap < bytes) {
    if (sl.p) {
      e = hipHostFree(sl.p);
      if (e != hipSuccess) return e;
      sl.p = nullptr;
      sl.cap = 0;
    }
    const size_t cap = std::max<size_t>(bytes, 1 << 20);
    e = hipHostMalloc(&sl.p, cap, hipHostMallocDefault);
    if (e != hipSuccess) return e;
    sl.cap = cap;
  }
  std::memcpy(sl.p, src, bytes);
  e = hipMemcpyAsync(dst, sl.p, bytes, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return e;
  e = hipEventRecord(sl.ev, s);
  if (e != hipSuccess) return e;
  sl.pending = true;
  return hipSuccess;
}

template <class T>
void put(std::vector<char>& blob, size_t off, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(blob.data() + off, v.data(), v.size() * sizeof(T));
}

// Frees a retired buffer after its last reader has finished.
hipError_t free_retired(RetiredImage& r) {
  hipError_t e = hipSuccess;
  if (r.ev) {
    e = hipEventSynchronize(r.ev);
    (void)hipEventDestroy(r.ev);
    r.ev = nullptr;
  }
  if (r.dev) {
    const hipError_t f = hipFree(r.dev);
    if (e == hipSuccess) e = f;
    r.dev = nullptr;
  }
  return e;
}

// Moves a cache entry's image buffer to the retired list: one event on the
// stream of its last decode marks when no kernel reads it any more (a device
// synchronisation if it was read on several streams).  Keeps the list short
// by freeing the oldest buffers.
hipError_t retire_image(treepo_ctx* ctx, CachedPlan& cp, bool trim = true) {
  hipError_t e = hipSuccess;
  if (cp.up_ev) {
    (void)hipEventDestroy(cp.up_ev);
    cp.up_ev = nullptr;
  }
  if (cp.dev) {
    RetiredImage r{cp.dev, cp.dev_cap, nullptr};
    if (cp.dev_valid) {
      if (cp.multi_stream) {
        e = hipDeviceSynchronize();
      } else {
        e = hipEventCreateWithFlags(&r.ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventRecord(r.ev, cp.last_stream);
      }
    }
    if (e != hipSuccess) {
      // cannot tell when its readers finish: wait for the whole device
      if (r.ev) (void)hipEventDestroy(r.ev);
      r.ev = nullptr;
      e = hipDeviceSynchronize();
    }
    ctx->retired.push_back(r);
  }
  cp.dev = nullptr;
  cp.dev_cap = 0;
  cp.dev_valid = false;
  cp.multi_stream = false;
  while (trim && ctx->retired.size() > kMaxRetired) {
    const hipError_t f = free_retired(ctx->retired.front());
    ctx->retired.erase(ctx->retired.begin());
    if (e == hipSuccess) e = f;
  }
  return e;
}

// Makes the plan's device image current for a decode on `s`: uploads it on
// the first use (into a retired buffer whose readers have finished, or a new
// one), else orders `s` after the upload.
hipError_t stage_image(treepo_ctx* ctx, CachedPlan& cp, hipStream_t s) {
  hipError_t e;
  if (cp.dev_valid) {
    if (s != cp.up_stream) {
      cp.multi_stream = true;
      e = hipStreamWaitEvent(s, cp.up_ev, 0);
      if (e != hipSuccess) return e;
    }
    cp.last_stream = s;
    return hipSuccess;
  }
  const size_t bytes = std::max<size_t>(cp.blob.size(), kAlign);
  if (!cp.dev) {
    for (size_t i = 0; i < ctx->retired.size(); ++i) {
      RetiredImage& r = ctx->retired[i];
      if (r.cap < bytes) continue;
      if (r.ev) {
        const hipError_t q = hipEventQuery(r.ev);
        if (q == hipErrorNotReady) continue;
        if (q != hipSuccess) return q;
        (void)hipEventDestroy(r.ev);
      }
      cp.dev = r.dev;
      cp.dev_cap = r.cap;
      ctx->retired.erase(ctx->retired.begin() + static_cast<std::ptrdiff_t>(i));
      break;
    }
  }
  if (!cp.dev) {
    e = hipMalloc(&cp.dev, bytes);
    if (e != hipSuccess) return e;
    cp.dev_cap = bytes;
  }
  if (!cp.up_ev) {
    e = hipEventCreateWithFlags(&cp.up_ev, hipEventDisableTiming);
    if (e != hipSuccess) return e;
  }
  e = upload(ctx, cp.dev, cp.blob.data(), cp.blob.size(), s);
  if (e != hipSuccess) return e;
  e = hipEventRecord(cp.up_ev, s);
  if (e != hipSuccess) return e;
  cp.up_stream = s;
  cp.last_stream = s;
  cp.dev_valid = true;
  return hipSuccess;
}

// The cached plan for these leaves and mode, built if needed.  With
// may_free false an evicted plan's image is retired without freeing any
// device memory (the no-alloc entry point).
int32_t get_plan(treepo_ctx* ctx, int32_t n, const int32_t* leaves, int32_t mode, CachedPlan** out,
                 bool may_free = true) {
  ++ctx->clock;
  for (CachedPlan& cp : ctx->plans) {
    // with device lengths a plan outlives appends (it covers unfrozen nodes up
    // to their capacity); otherwise any mutation invalidates it
    const uint64_t v = ctx->live ? ctx->tree.shape_version() : ctx->tree.version();
    if (cp.version == v && cp.mode == mode &&
        cp.leaves.size() == static_cast<size_t>(n) &&
        std::equal(cp.leaves.begin(), cp.leaves.end(), leaves)) {
      cp.last_use = ctx->clock;
      *out = &cp;
      return TREEPO_OK;
    }
  }
  CachedPlan cp;
  std::string err;
  int32_t st = treepo::build_plan(ctx->tree, n, leaves, static_cast<PlanMode>(mode), ctx->params,
                                  &cp.plan, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  const Plan& p = cp.plan;
  size_t off = 0;
  auto place = [&](size_t* at, size_t bytes) {
    *at = off;
    off = align_up(off + bytes);
  };
  place(&cp.off_blocks, p.blocks.size() * sizeof(int32_t));
  std::vector<int32_t> comb(2 * p.comb_count.size());
  for (size_t k = 0; k < p.comb_count.size(); ++k) {
    comb[2 * k] = p.comb_base[k];
    comb[2 * k + 1] = p.comb_count[k];
  }
  place(&cp.off_comb, comb.size() * sizeof(int32_t));
  cp.blob.assign(off, 0);
  put(cp.blob, cp.off_blocks, p.blocks);
  put(cp.blob, cp.off_comb, comb);
  off = 0;
  cp.off_part_o = off;
  // fp32 rows of D floats, or block floating-point rows of D / 2 dwords (compact plans)
  const size_t row_words = p.compact ? static_cast<size_t>(ctx->cfg.head_dim) / 2 : ctx->cfg.head_dim;
  off = align_up(off + static_cast<size_t>(p.partial_rows) * row_words * sizeof(uint32_t));
  cp.off_part_ml = off;
  off = align_up(off + static_cast<size_t>(p.partial_rows) * 2 * sizeof(float));
  cp.ws_bytes = off;
  cp.uid = ++g_plan_uid;
  cp.version = ctx->live ? ctx->tree.shape_version() : ctx->tree.version();
  cp.mode = mode;
  cp.leaves.assign(leaves, leaves + n);
  cp.last_use = ctx->clock;
  if (static_cast<int>(ctx->plans.size()) >= kPlanCache) {
    auto lru = std::min_element(ctx->plans.begin(), ctx->plans.end(),
                                [](const CachedPlan& a, const CachedPlan& b) { return a.last_use < b.last_use; });
    hipError_t e = retire_image(ctx, *lru, may_free);
    if (e != hipSuccess) return hip_fail(ctx, e, "plan cache");
    *lru = std::move(cp);
    *out = &*lru;
  } else {
    ctx->plans.push_back(std::move(cp));
    *out = &ctx->plans.back();
  }
  return TREEPO_OK;
}

int32_t check_decode_args(treepo_ctx* ctx, int32_t n, const int32_t* leaves, const void* q, float scale,
                          float* out) {
  if (!q || !out) return fail(ctx, TREEPO_EINVAL, "null q or out");
  if (reinterpret_cast<uintptr_t>(q) % 16 != 0) return fail(ctx, TREEPO_EINVAL, "q must be 16-byte aligned");
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(ctx, TREEPO_EINVAL, "scale must be positive and finite");
  std::string err;
  const int32_t st = ctx->tree.check_leaves(n, leaves, &err);
  return st == treepo::kOk ? TREEPO_OK : fail(ctx, st, err);
}

// Uploads the host length table to node_len on `s` when it is stale: through
// the pinned ring, or (pinned false) straight from pageable host memory kept
// in the context.
hipError_t stage_lengths(treepo_ctx* ctx, hipStream_t s, bool pinned) {
  if (!ctx->live || !ctx->dev_len_stale) return hipSuccess;
  const auto& nd = ctx->tree.nodes();
  std::vector<int32_t>& lens = ctx->len_stage;
  lens.resize(nd.size());
  for (size_t i = 0; i < nd.size(); ++i) lens[i] = nd[i].len;
  if (!lens.empty()) {
    const hipError_t e = pinned ? upload(ctx, ctx->cfg.node_len, lens.data(), lens.size() * sizeof(int32_t), s)
                                : hipMemcpyAsync(ctx->cfg.node_len, lens.data(), lens.size() * sizeof(int32_t),
                                                 hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return e;
  }
  ctx->dev_len_stale = false;
  return hipSuccess;
}

// Launches the node-partial and combine kernels of a plan whose image is at
// `img` (device) with its partial slots in `wsb` (device).
int32_t launch_decode(treepo_ctx* ctx, const CachedPlan& cp, const char* img, char* wsb, int32_t n, const void* q,
                      float scale, float* out, float* lse, hipStream_t stream) {
  const Plan& p = cp.plan;
  treepo::DecodeArgs a;
  a.k_pool = static_cast<const uint16_t*>(ctx->cfg.k_pool);
  a.v_pool = static_cast<const uint16_t*>(ctx->cfg.v_pool);
  a.pool_rows = pool_rows(ctx);
  a.hq = ctx->cfg.num_q_heads;
  a.hkv = ctx->cfg.num_kv_heads;
  a.group = a.hq / a.hkv;
  a.d = ctx->cfg.head_dim;
  a.q = static_cast<const uint16_t*>(q);
  a.scale_log2 = scale * 1.4426950408889634f;
  a.node_len = static_cast<const int32_t*>(ctx->cfg.node_len);
  a.blocks = reinterpret_cast<const int32_t*>(img + cp.off_blocks);
  a.block_ints = p.block_ints;
  a.n_streams = static_cast<int32_t>(p.streams.size());
  a.part_o = reinterpret_cast<float*>(wsb + cp.off_part_o);
  a.part_ml = reinterpret_cast<float*>(wsb + cp.off_part_ml);
  a.comb = reinterpret_cast<const int2*>(img + cp.off_comb);
  a.emax = p.emax;
  a.compact = p.compact;
  a.n_leaves = n;
  a.out = out;
  a.lse = lse;
  hipError_t e = timed_launch_attached(ctx, TREEPO_KERNEL_PARTIAL, [&](hipEvent_t t0, hipEvent_t t1) {
    a.ev_start = t0;
    a.ev_stop = t1;
    return treepo::launch_partial(a, stream);
  });
  if (e != hipSuccess) return hip_fail(ctx, e, "partial kernel launch");
  e = timed_launch_attached(ctx, TREEPO_KERNEL_COMBINE, [&](hipEvent_t t0, hipEvent_t t1) {
    a.ev_start = t0;
    a.ev_stop = t1;
    return treepo::launch_combine(a, stream);
  });
  if (e != hipSuccess) return hip_fail(ctx, e, "combine kernel launch");
  return TREEPO_OK;
}

int32_t decode(treepo_ctx* ctx, int32_t n, const int32_t* leaves, const void* q, float scale,
               float* out, float* lse, void* ws, size_t ws_bytes, hipStream_t stream, int32_t mode) {
  if (!ctx) return TREEPO_EINVAL;
  int32_t st = check_decode_args(ctx, n, leaves, q, scale, out);
  if (st != TREEPO_OK) return st;
  CachedPlan* cp = nullptr;
  st = get_plan(ctx, n, leaves, mode, &cp);
  if (st != TREEPO_OK) return st;
  if (!ws || ws_bytes < cp->ws_bytes || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return fail(ctx, TREEPO_EWORKSPACE,
                "workspace missing, smaller than treepo_decode_workspace_size or not 256-byte aligned");
  hipError_t e = stage_image(ctx, *cp, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "plan upload");
  e = stage_lengths(ctx, stream, true);
  if (e != hipSuccess) return hip_fail(ctx, e, "length table upload");
  return launch_decode(ctx, *cp, static_cast<const char*>(cp->dev), static_cast<char*>(ws), n, q, scale, out, lse,
                       stream);
}

// The cascade decode with the plan image and partial slots in the library's
// static device scratch (treepo_tree_decode_noalloc).  The scratch records
// which plan image it holds, so a plan is uploaded only when another plan
// (of any context) used the scratch since; uploads go straight from the
// plan's pageable host image, so no pinned staging is allocated.
int32_t decode_noalloc(treepo_ctx* ctx, int32_t n, const int32_t* leaves, const void* q, float scale, float* out,
                       float* lse, hipStream_t stream) {
  if (!ctx) return TREEPO_EINVAL;
  int32_t st = check_decode_args(ctx, n, leaves, q, scale, out);
  if (st != TREEPO_OK) return st;
  CachedPlan* cp = nullptr;
  st = get_plan(ctx, n, leaves, TREEPO_MODE_TREE, &cp, false);
  if (st != TREEPO_OK) return st;
  const size_t img_bytes = align_up(std::max<size_t>(cp->blob.size(), 1));
  if (img_bytes + cp->ws_bytes > treepo::kNoAllocScratchBytes)
    return fail(ctx, TREEPO_EWORKSPACE,
                "decode needs " + std::to_string(img_bytes + cp->ws_bytes) + " bytes of scratch (plan image " +
                    std::to_string(img_bytes) + ", partial slots " + std::to_string(cp->ws_bytes) +
                    "); the no-alloc scratch holds " + std::to_string(treepo::kNoAllocScratchBytes));
  void* base = nullptr;
  uint64_t* holder = nullptr;
  hipError_t e = treepo::noalloc_scratch(&base, &holder);
  if (e != hipSuccess) return hip_fail(ctx, e, "no-alloc scratch");
  char* sb = static_cast<char*>(base);
  if (*holder != cp->uid) {
    *holder = 0;
    e = hipMemcpyAsync(sb, cp->blob.data(), cp->blob.size(), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "plan upload (scratch)");
    *holder = cp->uid;
  }
  e = stage_lengths(ctx, stream, false);
  if (e != hipSuccess) return hip_fail(ctx, e, "length table upload");
  return launch_decode(ctx, *cp, sb, sb + img_bytes, n, q, scale, out, lse, stream);
}

// Splits a validated append into block-aligned pieces (source rows in call order).
void append_pieces(const treepo::Tree& t, int32_t n, const int32_t* nodes, const int32_t* ntok,
                   std::vector<treepo::AppendPiece>* out,
                   std::vector<std::pair<int32_t, int32_t>>* upd = nullptr) {
  const int32_t B = t.block_tokens();
  std::vector<std::pair<int32_t, int32_t>> pending;  // node -> len so far in this call
  out->clear();
  int32_t src = 0;
  for (int32_t i = 0; i < n; ++i) {
    const treepo::Node& nd = t.nodes()[nodes[i]];
    auto it = std::find_if(pending.begin(), pending.end(),
                           [&](const std::pair<int32_t, int32_t>& pr) { return pr.first == nodes[i]; });
    int32_t cur = it == pending.end() ? nd.len : it->second;
    int32_t left = ntok[i];
    while (left > 0) {
      // pieces end at 64-row boundaries of the pool (whatever the block size)
      const int64_t row = static_cast<int64_t>(nd.block_begin) * B + cur;
      const int32_t off = static_cast<int32_t>(row % treepo::kTile);
      const int32_t cnt = std::min(left, treepo::kTile - off);
      out->push_back(treepo::AppendPiece{src, static_cast<int32_t>(row / treepo::kTile), off, cnt});
      src += cnt;
      cur += cnt;
      left -= cnt;
    }
    if (it == pending.end())
      pending.emplace_back(nodes[i], cur);
    else
      it->second = cur;
  }
  // the nodes that received tokens, with their lengths after the whole call
  if (upd)
    for (const auto& pr : pending)
      if (pr.second != t.nodes()[pr.first].len) upd->push_back(pr);
}

}  // namespace

namespace {

// Sub-group g = a node on some leaf's chain, numbered in order of first
// appearance (positions ascending, chains root first); its members are the
// positions whose chain contains it, ascending.
void build_adv_plan(const treepo::Tree& t, int32_t n, const int32_t* leaves, AdvPlan* ap) {
  std::vector<std::vector<int32_t>> chains(n);
  std::vector<int32_t> gid(t.nodes().size(), -1);
  std::vector<std::vector<int32_t>> members;
  for (int32_t p = 0; p < n; ++p) {
    t.chain(leaves[p], &chains[p]);
    for (int32_t x : chains[p]) {
      if (gid[x] < 0) {
        gid[x] = static_cast<int32_t>(members.size());
        members.emplace_back();
      }
      members[gid[x]].push_back(p);
    }
  }
  const int32_t G = static_cast<int32_t>(members.size());
  std::vector<int32_t>& v = ap->ints;
  v.clear();
  ap->n_groups = G;
  ap->off_grp_off = v.size();
  int32_t acc = 0;
  for (int32_t g = 0; g < G; ++g) {
    v.push_back(acc);
    acc += static_cast<int32_t>(members[g].size());
  }
  v.push_back(acc);
  ap->off_grp_mem = v.size();
  for (const auto& m : members) v.insert(v.end(), m.begin(), m.end());
  ap->off_pos_off = v.size();
  acc = 0;
  for (int32_t p = 0; p < n; ++p) {
    v.push_back(acc);
    acc += static_cast<int32_t>(chains[p].size()) - 1;
  }
  v.push_back(acc);
  ap->off_pos_grp = v.size();
  for (int32_t p = 0; p < n; ++p)
    for (size_t j = 0; j + 1 < chains[p].size(); ++j) v.push_back(gid[chains[p][j]]);
  ap->off_pos_root = v.size();
  for (int32_t p = 0; p < n; ++p) v.push_back(gid[chains[p][0]]);
  size_t off = align_up(v.size() * sizeof(int32_t));
  ap->off_gmean = off;
  off = align_up(off + static_cast<size_t>(G) * sizeof(double));
  ap->off_gkeep = off;
  off = align_up(off + static_cast<size_t>(G) * sizeof(int32_t));
  ap->off_pooled = off;
  off = align_up(off + static_cast<size_t>(n) * sizeof(double));
  ap->ws_bytes = off;
}

// The machine the decode planner sizes its streams for: one stream per
// resident workgroup slot (partial_workgroups_per_cu() per compute unit),
// workgroups dealt to the XCDs round robin.
void set_machine(treepo_ctx* ctx, int32_t compute_units, int32_t xcds) {
  PlanParams& p = ctx->params;
  p.compute_units = compute_units;
  p.concurrent_wgs = compute_units * treepo::partial_workgroups_per_cu();
  p.slot_speed[0] = 1.0;
  p.slot_speed[1] = kSecondSlotSpeed;
  p.xcds = xcds;
  for (int x = 0; x < 8; ++x) p.xcd_speed[x] = x % 2 ? kOddXcdSpeed : 1.0;
}

int32_t check_ids(treepo_ctx* ctx, int32_t n, const int32_t* leaves) {
  if (n < 1 || !leaves) return fail(ctx, TREEPO_EINVAL, "need at least one leaf");
  for (int32_t i = 0; i < n; ++i)
    if (leaves[i] < 0 || leaves[i] >= static_cast<int32_t>(ctx->tree.nodes().size()))
      return fail(ctx, TREEPO_EINVAL, "unknown leaf id");
  return TREEPO_OK;
}

}  // namespace

extern "C" {

int32_t treepo_create(const treepo_config* cfg, treepo_ctx** out) {
  if (!cfg || !out) return TREEPO_EINVAL;
  const treepo_config& c = *cfg;
  if (c.num_q_heads < 1 || c.num_kv_heads < 1 || c.num_q_heads % c.num_kv_heads != 0 ||
      c.num_blocks < 0 || c.num_blocks > INT32_MAX || c.max_nodes < 0 || c.reserved != 0 ||
      !c.k_pool || !c.v_pool || reinterpret_cast<uintptr_t>(c.k_pool) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(c.v_pool) % 16 != 0 || reinterpret_cast<uintptr_t>(c.node_len) % 4 != 0)
    return TREEPO_EINVAL;
  if ((c.head_dim != 64 && c.head_dim != 128) ||
      (c.block_tokens != 16 && c.block_tokens != 32 && c.block_tokens != 64) ||
      c.num_q_heads / c.num_kv_heads > 128)
    return TREEPO_EUNSUPPORTED;
  treepo_ctx* ctx = new (std::nothrow) treepo_ctx(c);
  if (!ctx) return TREEPO_ENOMEM;
  ctx->params.group = c.num_q_heads / c.num_kv_heads;
  ctx->params.num_kv_heads = c.num_kv_heads;
  ctx->params.num_q_heads = c.num_q_heads;
  ctx->params.head_dim = c.head_dim;
  ctx->params.num_blocks = c.num_blocks;
  ctx->params.max_rows = 128;
  int32_t cus = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    cus = kDefaultComputeUnits;
  set_machine(ctx, cus, std::max(1, std::min(8, cus / kComputeUnitsPerXcd)));
  ctx->live = c.node_len != nullptr;
  ctx->params.live_lengths = ctx->live;
  *out = ctx;
  return TREEPO_OK;
}

int32_t treepo_destroy(treepo_ctx* ctx) {
  if (!ctx) return TREEPO_OK;
  for (PinnedSlot& s : ctx->ring) {
    if (s.pending) (void)hipEventSynchronize(s.ev);
    if (s.p) (void)hipHostFree(s.p);
    if (s.ev) (void)hipEventDestroy(s.ev);
  }
  for (const TimedLaunch& t : ctx->timed) {
    (void)hipEventSynchronize(t.stop);
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  for (hipEvent_t e : ctx->spare_events) (void)hipEventDestroy(e);
  for (CachedPlan& cp : ctx->plans) (void)retire_image(ctx, cp);
  for (RetiredImage& r : ctx->retired) (void)free_retired(r);
  delete ctx;
  return TREEPO_OK;
}

int32_t treepo_set_device_shape(treepo_ctx* ctx, int32_t compute_units, int32_t xcds) {
  if (!ctx) return TREEPO_EINVAL;
  if (compute_units < 1 || compute_units > 4096 || xcds < 1 || xcds > 8 || compute_units < xcds)
    return fail(ctx, TREEPO_EINVAL, "compute_units must be in [xcds, 4096] and xcds in [1, 8]");
  hipError_t e = hipSuccess;
  for (CachedPlan& cp : ctx->plans) {
    const hipError_t r = retire_image(ctx, cp);
    if (e == hipSuccess) e = r;
  }
  ctx->plans.clear();
  set_machine(ctx, compute_units, xcds);
  return e == hipSuccess ? TREEPO_OK : hip_fail(ctx, e, "plan cache");
}

int32_t treepo_new_root(treepo_ctx* ctx, int32_t cap_tokens, int32_t* node_out) {
  if (!ctx) return TREEPO_EINVAL;
  std::string err;
  const int32_t st = ctx->tree.new_root(cap_tokens, node_out, &err);
  if (st == treepo::kOk) ctx->dev_len_stale = true;
  return st == treepo::kOk ? TREEPO_OK : fail(ctx, st, err);
}

int32_t treepo_fork(treepo_ctx* ctx, int32_t parent, int32_t n_children, int32_t child_cap,
                    int32_t* children_out) {
  if (!ctx) return TREEPO_EINVAL;
  std::string err;
  const int32_t st = ctx->tree.fork(parent, n_children, child_cap, children_out, &err);
  if (st == treepo::kOk) ctx->dev_len_stale = true;
  return st == treepo::kOk ? TREEPO_OK : fail(ctx, st, err);
}

int32_t treepo_fork_at(treepo_ctx* ctx, int32_t node, int32_t offset, int32_t n_children, int32_t child_cap,
                       int32_t* children_out, int32_t* tail_out) {
  if (!ctx) return TREEPO_EINVAL;
  std::string err;
  const int32_t st = ctx->tree.fork_at(node, offset, n_children, child_cap, children_out, tail_out, &err);
  if (st == treepo::kOk) ctx->dev_len_stale = true;
  return st == treepo::kOk ? TREEPO_OK : fail(ctx, st, err);
}

int32_t treepo_kv_slots(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok,
                        int64_t* rows_out) {
  if (!ctx) return TREEPO_EINVAL;
  std::string err;
  std::vector<int64_t> rows;
  const int32_t st = ctx->tree.check_append(n, nodes, ntok, &rows, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  if (!rows.empty()) {
    if (!rows_out) return fail(ctx, TREEPO_EINVAL, "null rows_out");
    std::copy(rows.begin(), rows.end(), rows_out);
  }
  return TREEPO_OK;
}

int32_t treepo_kv_commit(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok) {
  if (!ctx) return TREEPO_EINVAL;
  std::string err;
  const int32_t st = ctx->tree.check_append(n, nodes, ntok, nullptr, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  ctx->tree.apply_append(n, nodes, ntok);
  ctx->dev_len_stale = true;
  return TREEPO_OK;
}

namespace {

// Scatters the rows into the pools and advances the lengths; the call has
// been validated by check_append.
int32_t append_validated(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok, const void* k,
                         const void* v, hipStream_t stream) {
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) total += ntok[i];
  if (total > 0) {
    if (!k || !v) return fail(ctx, TREEPO_EINVAL, "null k or v with tokens to append");
    std::vector<treepo::AppendPiece> pieces;
    std::vector<std::pair<int32_t, int32_t>> upd;
    append_pieces(ctx->tree, n, nodes, ntok, &pieces, &upd);
    std::vector<int32_t> upd_node(upd.size()), upd_len(upd.size());
    for (size_t i = 0; i < upd.size(); ++i) {
      upd_node[i] = upd[i].first;
      upd_len[i] = upd[i].second;
    }
    const hipError_t e = timed_launch(ctx, TREEPO_KERNEL_APPEND, stream, [&] {
      return treepo::launch_kv_append(static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                                      static_cast<uint16_t*>(ctx->cfg.k_pool),
                                      static_cast<uint16_t*>(ctx->cfg.v_pool), pool_rows(ctx),
                                      ctx->cfg.num_kv_heads, ctx->cfg.head_dim, pieces.data(),
                                      static_cast<int32_t>(pieces.size()), upd_node.data(), upd_len.data(),
                                      static_cast<int32_t>(upd.size()), static_cast<int32_t*>(ctx->cfg.node_len),
                                      stream);
    });
    if (e != hipSuccess) return hip_fail(ctx, e, "append kernel launch");
  }
  ctx->tree.apply_append(n, nodes, ntok);
  return TREEPO_OK;
}

// Work of a prefill call: each sequence's chain as 32-token tiles (after the
// append), and items of up to kPrefillRows new tokens, longest first.
struct PrefillPlan {
  std::vector<treepo::PrefillItem> items;
  std::vector<int32_t> tiles;  // int2 records
  std::vector<int32_t> sched;  // [slot * 8 + xcd] -> unit (item * Hkv + KV head), or -1
  std::vector<treepo::AppendPiece> pieces;  // the append, uploaded with the tables
  std::vector<int32_t> upd;                 // int2 (node, new length) per appended node
  size_t tiles_off = 0, sched_off = 0, pieces_off = 0, upd_off = 0, bytes = 0;
};

// Units (item, KV head) onto the 8 XCDs, longest first: a unit goes to the
// XCD that already holds its (sequence, KV head), so that the chain's tiles
// stay in that XCD's L2, unless that XCD would pass an even share of the
// work by more than 5%; then to the least loaded XCD.  Slot p of XCD x runs
// the p-th unit assigned to it.
void schedule_prefill(PrefillPlan* pl, int32_t hkv, int32_t n_seq) {
  constexpr int kX = 8;
  double total = 0;
  for (const auto& it : pl->items) total += static_cast<double>(it.nk) * hkv;
  const double cap = total / kX * 1.05;
  std::vector<double> load(kX, 0.0);
  std::vector<int32_t> home(static_cast<size_t>(n_seq) * hkv, -1);
  std::vector<std::vector<int32_t>> lists(kX);
  for (size_t i = 0; i < pl->items.size(); ++i) {
    const auto& it = pl->items[i];
    for (int32_t g = 0; g < hkv; ++g) {
      int32_t& h = home[static_cast<size_t>(it.pad[0]) * hkv + g];
      int x = h;
      if (x < 0 || load[x] + it.nk > cap)
        x = static_cast<int>(std::min_element(load.begin(), load.end()) - load.begin());
      if (h < 0) h = x;
      load[x] += it.nk;
      lists[x].push_back(static_cast<int32_t>(i) * hkv + g);
    }
  }
  size_t depth = 0;
  for (const auto& l : lists) depth = std::max(depth, l.size());
  pl->sched.assign(depth * kX, -1);
  for (int x = 0; x < kX; ++x)
    for (size_t p = 0; p < lists[x].size(); ++p) pl->sched[p * kX + x] = lists[x][p];
}

int32_t build_prefill_plan(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok,
                           PrefillPlan* pl) {
  const auto& nd = ctx->tree.nodes();
  constexpr int32_t kT = 32;
  const int32_t B = ctx->tree.block_tokens();
  std::vector<int32_t> chain;
  std::vector<int32_t> firsts;
  int64_t row = 0;
  int32_t n_seq = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (ntok[i] == 0) continue;
    ++n_seq;
    const int32_t x = nodes[i];
    ctx->tree.chain(x, &chain);
    const int64_t pos0 = ctx->tree.chain_tokens(x);
    if (pos0 + ntok[i] >= (int64_t{1} << 25)) return fail(ctx, TREEPO_EINVAL, "chain too long for a prefill");
    const int32_t tile_off = static_cast<int32_t>(pl->tiles.size() / 2);
    firsts.clear();
    for (int32_t y : chain) {
      const treepo::Node& b = nd[y];
      const int32_t len = y == x ? b.len + ntok[i] : b.len;
      for (int32_t j = 0; j * kT < len; ++j) {
        const int32_t first = b.start + j * kT;
        const int32_t cnt = std::min(kT, len - j * kT);
        pl->tiles.push_back(static_cast<int32_t>((static_cast<int64_t>(b.block_begin) * B + j * kT) / 16));
        pl->tiles.push_back((first << 6) | cnt);
        firsts.push_back(first);
      }
    }
    for (int32_t t0 = 0; t0 < ntok[i]; t0 += treepo::kPrefillRows) {
      treepo::PrefillItem it{};
      it.row0 = static_cast<int32_t>(row + t0);
      it.n_rows = std::min(treepo::kPrefillRows, ntok[i] - t0);
      it.pos0 = static_cast<int32_t>(pos0 + t0);
      it.tile_off = tile_off;
      const int32_t last = it.pos0 + it.n_rows - 1;
      it.nk = static_cast<int32_t>(std::upper_bound(firsts.begin(), firsts.end(), last) - firsts.begin());
      it.pad[0] = n_seq - 1;  // sequence index, for the XCD schedule
      pl->items.push_back(it);
    }
    row += ntok[i];
  }
  if (row >= (int64_t{1} << 31) / 64) return fail(ctx, TREEPO_EINVAL, "too many prefill rows");
  std::stable_sort(pl->items.begin(), pl->items.end(),
                   [](const treepo::PrefillItem& a, const treepo::PrefillItem& b) { return a.nk > b.nk; });
  schedule_prefill(pl, ctx->cfg.num_kv_heads, n_seq);
  std::vector<std::pair<int32_t, int32_t>> upd;
  append_pieces(ctx->tree, n, nodes, ntok, &pl->pieces, &upd);
  for (const auto& u : upd) {
    pl->upd.push_back(u.first);
    pl->upd.push_back(u.second);
  }
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  pl->tiles_off = up(pl->items.size() * sizeof(treepo::PrefillItem));
  pl->sched_off = up(pl->tiles_off + pl->tiles.size() * sizeof(int32_t));
  pl->pieces_off = up(pl->sched_off + pl->sched.size() * sizeof(int32_t));
  pl->upd_off = up(pl->pieces_off + pl->pieces.size() * sizeof(treepo::AppendPiece));
  pl->bytes = std::max<size_t>(256, pl->upd_off + pl->upd.size() * sizeof(int32_t));
  return TREEPO_OK;
}

int32_t check_prefill(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok) {
  std::string err;
  const int32_t st = ctx->tree.check_append(n, nodes, ntok, nullptr, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  std::vector<int32_t> seen(nodes, nodes + n);
  std::sort(seen.begin(), seen.end());
  if (std::adjacent_find(seen.begin(), seen.end()) != seen.end())
    return fail(ctx, TREEPO_EINVAL, "a node appears twice in one prefill");
  return TREEPO_OK;
}

}  // namespace

int32_t treepo_kv_append(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok,
                         const void* k, const void* v, hipStream_t stream) {
  if (!ctx) return TREEPO_EINVAL;
  std::string err;
  const int32_t st = ctx->tree.check_append(n, nodes, ntok, nullptr, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  return append_validated(ctx, n, nodes, ntok, k, v, stream);
}

int32_t treepo_prefill_workspace_size(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok,
                                      size_t* bytes) {
  if (!ctx) return TREEPO_EINVAL;
  if (!bytes) return fail(ctx, TREEPO_EINVAL, "null bytes");
  int32_t st = check_prefill(ctx, n, nodes, ntok);
  if (st != TREEPO_OK) return st;
  PrefillPlan pl;
  st = build_prefill_plan(ctx, n, nodes, ntok, &pl);
  if (st != TREEPO_OK) return st;
  *bytes = pl.bytes;
  return TREEPO_OK;
}

int32_t treepo_prefill(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok, const void* q,
                       const void* k, const void* v, float scale, float* out, float* lse, void* workspace,
                       size_t ws_bytes, hipStream_t stream) {
  if (!ctx) return TREEPO_EINVAL;
  int32_t st = check_prefill(ctx, n, nodes, ntok);
  if (st != TREEPO_OK) return st;
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) total += ntok[i];
  if (total == 0) return TREEPO_OK;
  if (!q || !k || !v || !out) return fail(ctx, TREEPO_EINVAL, "null q, k, v or out with tokens to prefill");
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(ctx, TREEPO_EINVAL, "scale must be positive and finite");
  PrefillPlan pl;
  st = build_prefill_plan(ctx, n, nodes, ntok, &pl);
  if (st != TREEPO_OK) return st;
  if (!workspace || ws_bytes < pl.bytes || reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(ctx, TREEPO_EWORKSPACE,
                "workspace missing, smaller than treepo_prefill_workspace_size or not 256-byte aligned");
  char* wsb = static_cast<char*>(workspace);
  std::vector<char> blob(pl.bytes, 0);
  std::memcpy(blob.data(), pl.items.data(), pl.items.size() * sizeof(treepo::PrefillItem));
  std::memcpy(blob.data() + pl.tiles_off, pl.tiles.data(), pl.tiles.size() * sizeof(int32_t));
  std::memcpy(blob.data() + pl.sched_off, pl.sched.data(), pl.sched.size() * sizeof(int32_t));
  std::memcpy(blob.data() + pl.pieces_off, pl.pieces.data(), pl.pieces.size() * sizeof(treepo::AppendPiece));
  std::memcpy(blob.data() + pl.upd_off, pl.upd.data(), pl.upd.size() * sizeof(int32_t));
  hipError_t e = upload(ctx, wsb, blob.data(), blob.size(), stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "prefill table upload");
  // the append: every piece in one launch, from the uploaded tables
  e = timed_launch(ctx, TREEPO_KERNEL_APPEND, stream, [&] {
    return treepo::launch_kv_append_dev(
        static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), static_cast<uint16_t*>(ctx->cfg.k_pool),
        static_cast<uint16_t*>(ctx->cfg.v_pool), pool_rows(ctx), ctx->cfg.num_kv_heads, ctx->cfg.head_dim,
        reinterpret_cast<const treepo::AppendPiece*>(wsb + pl.pieces_off), static_cast<int32_t>(pl.pieces.size()),
        reinterpret_cast<const int2*>(wsb + pl.upd_off), static_cast<int32_t>(pl.upd.size() / 2),
        static_cast<int32_t*>(ctx->cfg.node_len), stream);
  });
  if (e != hipSuccess) return hip_fail(ctx, e, "prefill append launch");
  ctx->tree.apply_append(n, nodes, ntok);
  treepo::PrefillArgs a;
  a.k_pool = static_cast<const uint16_t*>(ctx->cfg.k_pool);
  a.v_pool = static_cast<const uint16_t*>(ctx->cfg.v_pool);
  a.pool_rows = pool_rows(ctx);
  a.hq = ctx->cfg.num_q_heads;
  a.hkv = ctx->cfg.num_kv_heads;
  a.d = ctx->cfg.head_dim;
  a.q = static_cast<const uint16_t*>(q);
  a.items = reinterpret_cast<const treepo::PrefillItem*>(wsb);
  a.n_items = static_cast<int32_t>(pl.items.size());
  a.tiles = reinterpret_cast<const int2*>(wsb + pl.tiles_off);
  a.sched = reinterpret_cast<const int32_t*>(wsb + pl.sched_off);
  a.n_sched = static_cast<int32_t>(pl.sched.size());
  a.scale_log2 = scale * 1.44269504088896340736f;
  a.out = out;
  a.lse = lse;
  e = timed_launch_attached(ctx, TREEPO_KERNEL_PREFILL, [&](hipEvent_t s0, hipEvent_t s1) {
    a.ev_start = s0;
    a.ev_stop = s1;
    return treepo::launch_prefill(a, stream);
  });
  if (e != hipSuccess) return hip_fail(ctx, e, "prefill kernel launch");
  return TREEPO_OK;
}

int32_t treepo_branch_budget(int32_t n_paths, const float* scores, int32_t total, int32_t mode,
                             float temperature, int32_t* budget_out) {
  return treepo::branch_budget(n_paths, scores, total, mode, temperature, budget_out, nullptr) == treepo::kOk
             ? TREEPO_OK
             : TREEPO_EINVAL;
}

int32_t treepo_advantage_workspace_size(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                                        size_t* bytes) {
  if (!ctx) return TREEPO_EINVAL;
  if (!bytes) return fail(ctx, TREEPO_EINVAL, "null bytes");
  const int32_t st = check_ids(ctx, n_leaves, leaves);
  if (st != TREEPO_OK) return st;
  AdvPlan ap;
  build_adv_plan(ctx->tree, n_leaves, leaves, &ap);
  *bytes = ap.ws_bytes;
  return TREEPO_OK;
}

int32_t treepo_tree_advantage(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, const float* rewards,
                              int32_t weighting, float* adv, void* workspace, size_t ws_bytes,
                              hipStream_t stream) {
  if (!ctx) return TREEPO_EINVAL;
  int32_t st = check_ids(ctx, n_leaves, leaves);
  if (st != TREEPO_OK) return st;
  if (!rewards || !adv) return fail(ctx, TREEPO_EINVAL, "null rewards or adv");
  if (weighting != TREEPO_ADV_MEAN && weighting != TREEPO_ADV_SIZE_WEIGHTED)
    return fail(ctx, TREEPO_EINVAL, "bad weighting");
  AdvPlan& ap = ctx->adv;
  if (ap.ints.empty() || ap.shape_version != ctx->tree.shape_version() ||
      ap.leaves.size() != static_cast<size_t>(n_leaves) || !std::equal(ap.leaves.begin(), ap.leaves.end(), leaves)) {
    build_adv_plan(ctx->tree, n_leaves, leaves, &ap);
    ap.shape_version = ctx->tree.shape_version();
    ap.leaves.assign(leaves, leaves + n_leaves);
  }
  if (!workspace || ws_bytes < ap.ws_bytes || reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(ctx, TREEPO_EWORKSPACE,
                "workspace missing, smaller than treepo_advantage_workspace_size or not 256-byte aligned");
  char* wsb = static_cast<char*>(workspace);
  hipError_t e = upload(ctx, wsb, ap.ints.data(), ap.ints.size() * sizeof(int32_t), stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "advantage index upload");
  const int32_t* ints = reinterpret_cast<const int32_t*>(wsb);
  treepo::AdvantageArgs a;
  a.grp_off = ints + ap.off_grp_off;
  a.grp_mem = ints + ap.off_grp_mem;
  a.n_groups = ap.n_groups;
  a.pos_off = ints + ap.off_pos_off;
  a.pos_grp = ints + ap.off_pos_grp;
  a.pos_root = ints + ap.off_pos_root;
  a.n_pos = n_leaves;
  a.rewards = rewards;
  a.size_weighted = weighting == TREEPO_ADV_SIZE_WEIGHTED;
  a.gmean = reinterpret_cast<double*>(wsb + ap.off_gmean);
  a.gkeep = reinterpret_cast<int32_t*>(wsb + ap.off_gkeep);
  a.pooled = reinterpret_cast<double*>(wsb + ap.off_pooled);
  a.adv = adv;
  e = timed_launch(ctx, TREEPO_KERNEL_ADVANTAGE, stream, [&] { return treepo::launch_advantage(a, stream); });
  if (e != hipSuccess) return hip_fail(ctx, e, "advantage kernel launch");
  return TREEPO_OK;
}

int32_t treepo_decode_workspace_size(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                                     int32_t mode, size_t* bytes) {
  if (!ctx) return TREEPO_EINVAL;
  if (!bytes || (mode != TREEPO_MODE_TREE && mode != TREEPO_MODE_NAIVE))
    return fail(ctx, TREEPO_EINVAL, "null bytes or bad mode");
  std::string err;
  int32_t st = ctx->tree.check_leaves(n_leaves, leaves, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  CachedPlan* cp = nullptr;
  st = get_plan(ctx, n_leaves, leaves, mode, &cp);
  if (st != TREEPO_OK) return st;
  *bytes = cp->ws_bytes;
  return TREEPO_OK;
}

int32_t treepo_tree_decode(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, const void* q,
                           float scale, float* out, float* lse, void* workspace, size_t ws_bytes,
                           hipStream_t stream) {
  return decode(ctx, n_leaves, leaves, q, scale, out, lse, workspace, ws_bytes, stream, TREEPO_MODE_TREE);
}

int32_t treepo_tree_decode_noalloc(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, const void* q,
                                   float scale, float* out, float* lse, hipStream_t stream) {
  return decode_noalloc(ctx, n_leaves, leaves, q, scale, out, lse, stream);
}

int32_t treepo_paged_decode_naive(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                                  const void* q, float scale, float* out, float* lse, void* workspace,
                                  size_t ws_bytes, hipStream_t stream) {
  return decode(ctx, n_leaves, leaves, q, scale, out, lse, workspace, ws_bytes, stream, TREEPO_MODE_NAIVE);
}

int32_t treepo_num_nodes(treepo_ctx* ctx, int32_t* n_nodes) {
  if (!ctx || !n_nodes) return TREEPO_EINVAL;
  *n_nodes = static_cast<int32_t>(ctx->tree.nodes().size());
  return TREEPO_OK;
}

int32_t treepo_export_nodes(treepo_ctx* ctx, int32_t* records, int32_t capacity, int32_t* n_nodes) {
  if (!ctx || !n_nodes || capacity < 0 || (capacity > 0 && !records)) return TREEPO_EINVAL;
  const auto& nd = ctx->tree.nodes();
  *n_nodes = static_cast<int32_t>(nd.size());
  const int32_t m = std::min<int32_t>(capacity, static_cast<int32_t>(nd.size()));
  for (int32_t i = 0; i < m; ++i) {
    const treepo::Node& x = nd[i];
    const int32_t r[TREEPO_NODE_FIELDS] = {x.parent, x.depth, x.start, x.len,
                                           x.cap, x.block_begin, x.n_blocks, x.tree_id};
    std::copy(r, r + TREEPO_NODE_FIELDS, records + static_cast<size_t>(i) * TREEPO_NODE_FIELDS);
  }
  return TREEPO_OK;
}

int32_t treepo_export_chains(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                             int32_t* chain_off, int32_t* chain_nodes, int32_t* block_off,
                             int32_t* blocks, int32_t* total_chain, int32_t* total_blocks) {
  if (!ctx || n_leaves < 0 || (n_leaves > 0 && !leaves) || !total_chain || !total_blocks)
    return TREEPO_EINVAL;
  const auto& nd = ctx->tree.nodes();
  for (int32_t i = 0; i < n_leaves; ++i)
    if (leaves[i] < 0 || leaves[i] >= static_cast<int32_t>(nd.size()))
      return fail(ctx, TREEPO_EINVAL, "unknown leaf id");
  const int32_t B = ctx->tree.block_tokens();
  std::vector<int32_t> ch;
  int32_t tc = 0, tb = 0;
  const bool fill = chain_off && chain_nodes && block_off && blocks;
  if (fill) {
    chain_off[0] = 0;
    block_off[0] = 0;
  }
  for (int32_t i = 0; i < n_leaves; ++i) {
    ctx->tree.chain(leaves[i], &ch);
    for (int32_t n : ch) {
      if (fill) chain_nodes[tc] = n;
      ++tc;
      const int32_t nb = (nd[n].len + B - 1) / B;
      for (int32_t k = 0; k < nb; ++k) {
        if (fill) blocks[tb] = nd[n].block_begin + k;
        ++tb;
      }
    }
    if (fill) {
      chain_off[i + 1] = tc;
      block_off[i + 1] = tb;
    }
  }
  *total_chain = tc;
  *total_blocks = tb;
  return TREEPO_OK;
}

int32_t treepo_export_desc(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, int32_t* nodes,
                           int32_t* desc_off, int32_t* desc, int32_t* n_nodes, int32_t* total) {
  if (!ctx || n_leaves < 0 || (n_leaves > 0 && !leaves) || !n_nodes || !total) return TREEPO_EINVAL;
  const auto& nd = ctx->tree.nodes();
  for (int32_t i = 0; i < n_leaves; ++i)
    if (leaves[i] < 0 || leaves[i] >= static_cast<int32_t>(nd.size()))
      return fail(ctx, TREEPO_EINVAL, "unknown leaf id");
  std::vector<int32_t> nv, off, dv;
  treepo::desc_sets(ctx->tree, n_leaves, leaves, &nv, &off, &dv);
  *n_nodes = static_cast<int32_t>(nv.size());
  *total = static_cast<int32_t>(dv.size());
  if (nodes && desc_off && desc) {
    std::copy(nv.begin(), nv.end(), nodes);
    std::copy(off.begin(), off.end(), desc_off);
    std::copy(dv.begin(), dv.end(), desc);
  }
  return TREEPO_OK;
}

int32_t treepo_export_plan(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, int32_t mode,
                           int32_t* pieces, int32_t* rowsets, int32_t* tiles, int32_t* n_pieces,
                           int32_t* n_rowsets, int32_t* n_tiles, int32_t* n_streams) {
  if (!ctx) return TREEPO_EINVAL;
  if (!n_pieces || !n_rowsets || !n_tiles || !n_streams || (mode != TREEPO_MODE_TREE && mode != TREEPO_MODE_NAIVE))
    return fail(ctx, TREEPO_EINVAL, "null count pointer or bad mode");
  std::string err;
  int32_t st = ctx->tree.check_leaves(n_leaves, leaves, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  CachedPlan* cp = nullptr;
  st = get_plan(ctx, n_leaves, leaves, mode, &cp);
  if (st != TREEPO_OK) return st;
  const Plan& p = cp->plan;
  *n_pieces = static_cast<int32_t>(p.pieces.size());
  *n_rowsets = static_cast<int32_t>(p.rowsets.size());
  *n_tiles = static_cast<int32_t>(p.tiles.size());
  *n_streams = static_cast<int32_t>(p.streams.size());
  if (pieces && rowsets && tiles) {
    std::memcpy(pieces, p.pieces.data(), p.pieces.size() * sizeof(treepo::Piece));
    std::memcpy(rowsets, p.rowsets.data(), p.rowsets.size() * sizeof(int32_t));
    std::memcpy(tiles, p.tiles.data(), p.tiles.size() * sizeof(treepo::Tile));
  }
  return TREEPO_OK;
}

int32_t treepo_export_blocks(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, int32_t mode,
                             int32_t* blocks, int32_t* block_ints, int32_t* n_streams) {
  if (!ctx) return TREEPO_EINVAL;
  if (!block_ints || !n_streams || (mode != TREEPO_MODE_TREE && mode != TREEPO_MODE_NAIVE))
    return fail(ctx, TREEPO_EINVAL, "null count pointer or bad mode");
  std::string err;
  int32_t st = ctx->tree.check_leaves(n_leaves, leaves, &err);
  if (st != treepo::kOk) return fail(ctx, st, err);
  CachedPlan* cp = nullptr;
  st = get_plan(ctx, n_leaves, leaves, mode, &cp);
  if (st != TREEPO_OK) return st;
  const Plan& p = cp->plan;
  *block_ints = p.block_ints;
  *n_streams = static_cast<int32_t>(p.streams.size());
  if (blocks) std::memcpy(blocks, p.blocks.data(), p.blocks.size() * sizeof(int32_t));
  return TREEPO_OK;
}

int32_t treepo_set_profiling(treepo_ctx* ctx, int32_t enable) {
  if (!ctx) return TREEPO_EINVAL;
  const hipError_t e = drain_timings(ctx);
  ctx->profiling = enable != 0;
  std::fill(ctx->prof_ms, ctx->prof_ms + TREEPO_KERNEL_KINDS, 0.0);
  std::fill(ctx->prof_n, ctx->prof_n + TREEPO_KERNEL_KINDS, 0);
  return e == hipSuccess ? TREEPO_OK : hip_fail(ctx, e, "profiling events");
}

int32_t treepo_profile_read(treepo_ctx* ctx, int32_t kind, double* total_ms, int64_t* launches) {
  if (!ctx || kind < 0 || kind >= TREEPO_KERNEL_KINDS || !total_ms || !launches) return TREEPO_EINVAL;
  const hipError_t e = drain_timings(ctx);
  if (e != hipSuccess) return hip_fail(ctx, e, "profiling events");
  *total_ms = ctx->prof_ms[kind];
  *launches = ctx->prof_n[kind];
  return TREEPO_OK;
}

const char* treepo_strerror(int32_t code) {
  switch (code) {
    case TREEPO_OK: return "ok";
    case TREEPO_EINVAL: return "invalid argument";
    case TREEPO_ENOMEM: return "pool blocks or node slots exhausted";
    case TREEPO_EFULL: return "append past node capacity";
    case TREEPO_EFROZEN: return "append to a node that has children";
    case TREEPO_EEMPTY: return "decode of an empty chain";
    case TREEPO_EWORKSPACE: return "workspace missing or too small";
    case TREEPO_EHIP: return "HIP runtime error";
    case TREEPO_EUNSUPPORTED: return "unsupported shape";
    default: return "unknown status";
  }
}

const char* treepo_last_error(treepo_ctx* ctx) { return ctx ? ctx->last_error.c_str() : ""; }

}  // extern "C"
