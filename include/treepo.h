/*
 * treepo.h -- C-ABI of the segment-tree decode-attention library (gfx950).
 *
 * The operation (TreePO, arXiv 2508.17445):
 *   - a rollout forest: every query is a root node at depth 0; before each
 *     segment step a path is forked into children that share its prefix
 *     (Alg. 1; Sec. 2.2 "Segment-level Tree Sampling", "Branching and
 *     Fallback"); each step appends one generated segment of at most l tokens
 *     to a path (Alg. 1, the concatenation p_last + s_k);
 *   - a leaf's trajectory is the concatenation of its chain's segments
 *     (Sec. 2.3, segment decomposition), and shared prefixes are stored once
 *     (Sec. 2.1);
 *   - a decode step: every active leaf's new query, all Hq heads, attends with
 *     softmax over the K/V of its whole root-to-leaf chain (Sec. 2.2,
 *     segment-level decoding).  KV head g = h / (Hq / Hkv) serves query head h.
 *
 * Conventions
 *   - Every function returns an int32_t status: TREEPO_OK or a negative code.
 *     A failing call changes no state (arguments are validated before anything
 *     is mutated).  No C++ exception crosses this boundary.
 *   - "host" pointers are ordinary CPU memory read during the call; "device"
 *     pointers are HIP device memory owned by the caller: pools, queries, K/V
 *     staging, outputs and workspaces.
 *   - Ownership rule: the library allocates device memory for one thing only,
 *     the device image of each cached decode plan (its stream blocks and
 *     combine counts).  treepo_tree_decode / treepo_paged_decode_naive
 *     allocate it with hipMalloc on the first decode with a plan that finds
 *     no retired image large enough, reuse it while the plan stays cached,
 *     and free it in treepo_destroy (or when a later plan replaces it and its
 *     last reader has finished).  The image must outlive the calls that read
 *     it, and caller memory cannot promise that: a caching allocator hands a
 *     freed workspace to other tensors (and to other contexts) between
 *     calls, and a plan read from overwritten memory would send the kernels
 *     to arbitrary pool offsets.  Every other call allocates no device
 *     memory.  The library also allocates pinned host staging for uploads.
 *   - Device work is enqueued on the caller's stream and is asynchronous; the
 *     node table is host state updated synchronously at call time.  A context
 *     is single-threaded, and its device work must be issued on one stream at a
 *     time (or the caller orders the streams).
 *   - bf16 is IEEE bfloat16 (1-8-7 bits), little-endian, 2 bytes.
 */
#ifndef TREEPO_H
#define TREEPO_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
#define TREEPO_OK 0
#define TREEPO_EINVAL (-1)       /* bad id, shape, count or null pointer         */
#define TREEPO_ENOMEM (-2)       /* pool blocks or node slots exhausted          */
#define TREEPO_EFULL (-3)        /* append would exceed the node's capacity      */
#define TREEPO_EFROZEN (-4)      /* append to a node that has children           */
#define TREEPO_EEMPTY (-5)       /* decode of a chain holding zero tokens        */
#define TREEPO_EWORKSPACE (-6)   /* workspace missing or too small               */
#define TREEPO_EHIP (-7)         /* HIP runtime error; see treepo_last_error     */
#define TREEPO_EUNSUPPORTED (-8) /* shape outside what the kernels implement     */

/* decode modes for treepo_decode_workspace_size / treepo_export_plan */
#define TREEPO_MODE_TREE 0  /* cascade: each node's KV read once for all its leaves */
#define TREEPO_MODE_NAIVE 1 /* baseline: each leaf reads its whole chain            */

typedef struct treepo_ctx treepo_ctx;

/*
 * Pool shape (R = num_blocks * B rows per KV head).  K pool, device bf16,
 * layout [Hkv][R][D]: token row r = block * B + offset of KV head g starts at
 * element (g*R + r)*D.  V pool, device bf16, layout [Hkv][R/16][D][16]: every
 * group of 16 rows is stored transposed, so element (g, r, d) is at
 * (g*R + (r/16)*16)*D + d*16 + r%16.
 * head_dim D must be 64 or 128, block_tokens B 16, 32 or 64 (blocks are the
 * unit in which nodes reserve pool rows; the kernels stream 32-token tiles
 * from any 16-row boundary), Hq % Hkv == 0 and Hq / Hkv <= 128.  With B = 16
 * the pool's last block is never reserved: a node's last tile may read up to
 * 16 rows past its blocks, and this keeps every read inside the pool.  Pools
 * are caller-owned, 16-byte aligned, and must stay valid until
 * treepo_destroy; their contents need no initialisation.
 *
 * node_len (optional, device int32[max_nodes], caller-owned, contents kept by
 * the library, valid until treepo_destroy): the nodes' token counts on the
 * device.  With it, a decode plan stays valid while the tree only grows by
 * appends (segment-level decoding: one append and one decode per step until
 * the next fork, Sec. 2.2): the plan covers every unfrozen node up to its
 * capacity and the kernels read the current lengths from node_len, so no
 * re-plan or re-upload happens between forks.  treepo_kv_append updates it on
 * the stream; after treepo_kv_commit, new_root or fork the next decode
 * re-uploads the table on its stream.  NULL: every length change re-plans.
 */
typedef struct treepo_config {
  int32_t num_q_heads;  /* Hq  */
  int32_t num_kv_heads; /* Hkv */
  int32_t head_dim;     /* D   */
  int32_t block_tokens; /* B   */
  int64_t num_blocks;   /* pool capacity in blocks                     */
  int32_t max_nodes;    /* node-table capacity                          */
  int32_t reserved;     /* must be 0                                    */
  void* k_pool;         /* device, see above                            */
  void* v_pool;         /* device, see above                            */
  void* node_len;       /* device int32[max_nodes] or NULL, see above   */
} treepo_config;

/* Records exported by treepo_export_plan. */
#define TREEPO_PIECE_FIELDS 16
#define TREEPO_TILE_FIELDS 4

/* Node record exported by treepo_export_nodes: 8 int32 per node. */
#define TREEPO_NODE_FIELDS 8 /* parent, depth, start, len, cap, block_begin, n_blocks, tree_id */

/* Creates a context for one pool.  The only device call is a query of the
 * current device's compute-unit count, which sizes the decode schedule (one
 * stream per resident workgroup slot, XCDs of 32 compute units); with no
 * device visible the planner assumes 256 compute units in 8 XCDs (MI355X).
 * *out receives the handle; EINVAL / EUNSUPPORTED on a bad config. */
int32_t treepo_create(const treepo_config* cfg, treepo_ctx** out);

/* Overrides the machine shape the decode planner sizes its streams for:
 * compute_units (two resident workgroups each) and xcds (dies the workgroups
 * are dealt to round robin).  Drops every cached plan.  EINVAL unless
 * 1 <= xcds <= 8 and xcds <= compute_units <= 4096. */
int32_t treepo_set_device_shape(treepo_ctx* ctx, int32_t compute_units, int32_t xcds);
/* Releases host state, pinned staging and the plan images (waits for this
 * context's pending uploads and for the last readers of its plan images).
 * Null is accepted. */
int32_t treepo_destroy(treepo_ctx* ctx);

/* New tree: a root node (the query/prompt segment, depth 0, Sec. 2.2 item 1)
 * able to hold cap_tokens tokens.  Reserves ceil(cap/B) contiguous blocks,
 * starting at the running total of all blocks reserved so far.  Node ids are
 * 0,1,2,... in creation order.  EINVAL if cap < 1; ENOMEM if out of nodes or
 * blocks. */
int32_t treepo_new_root(treepo_ctx* ctx, int32_t cap_tokens, int32_t* node_out);

/* Branching (Alg. 1 Branching; Sec. 2.2): spawns n_children nodes that all
 * continue the parent's sequence (start = parent.start + parent.len, depth =
 * parent.depth + 1) with no KV copy; each reserves ceil(child_cap/B) blocks.
 * Ids are consecutive and written to children_out (host, n_children entries).
 * The parent becomes frozen (no further appends).  A node may be forked
 * again later (fallback re-forks, partially filled parents).  EINVAL on a bad
 * parent, n_children < 1 or child_cap < 1; ENOMEM when out of nodes/blocks. */
int32_t treepo_fork(treepo_ctx* ctx, int32_t parent, int32_t n_children,
                    int32_t child_cap, int32_t* children_out);

/* Fallback inside a segment (Alg. 1 Fallback; Sec. 2.2 fallback at segment
 * level; Sec. 4.2 "misaligned fallback", a fallback granularity finer than
 * the segment): forks n_children (>= 0) children after the first `offset`
 * tokens of `node`.  The node keeps tokens [0, offset); a new tail node (the
 * next id, written to *tail_out) takes tokens [offset, len), the rest of the
 * node's capacity and blocks (no KV is copied), and the node's children,
 * whose subtrees move one level down; every existing trajectory keeps
 * exactly its tokens (an active path now continues in the tail).  The
 * children (consecutive ids after the tail, children_out) start after the
 * kept prefix and reserve ceil(child_cap/B) blocks each.  offset == len is a
 * plain treepo_fork (*tail_out = -1).  EINVAL (bad node, offset outside
 * [0, len], offset < len not a multiple of B, n_children < 0, or < 1 for a
 * plain fork, child_cap < 1 with children), ENOMEM (nodes or blocks). */
int32_t treepo_fork_at(treepo_ctx* ctx, int32_t node, int32_t offset, int32_t n_children, int32_t child_cap,
                       int32_t* children_out, int32_t* tail_out);

/* Appends generated tokens (Alg. 1: the segment s_k joins its path).  nodes and
 * ntok are host arrays of n entries; node i gets ntok[i] >= 0 tokens whose
 * K and V rows are rows [sum(ntok[0..i)), +ntok[i]) of k and v (device bf16,
 * [sum ntok][Hkv][D], packed in call order).  A node may appear more than
 * once (its rows are appended in call order).  The whole call is validated
 * first: EINVAL (bad id, ntok < 0, null k/v with tokens), EFROZEN (node has
 * children), EFULL (len would exceed cap).  The scatter into the pools is
 * enqueued on stream; lengths are updated at call time. */
int32_t treepo_kv_append(treepo_ctx* ctx, int32_t n, const int32_t* nodes,
                         const int32_t* ntok, const void* k, const void* v,
                         hipStream_t stream);

/* Prefill: appends tokens like treepo_kv_append and computes their causal
 * attention over their chain (the shared prompt of a query, prefilled once
 * for all of its rollouts: Sec. 2.2 tree rollout, where the prompt is the
 * root every path extends; the shared-prefix prefilling of Sec. 4.1).
 * Node nodes[i] receives ntok[i] tokens; a new token at chain position p
 * (chain tokens before it, root first) attends to chain positions 0..p:
 *   out[r, h] = sum_{t <= p} softmax_t(scale <q[r, h], K[t, g]>) V[t, g],
 *   lse[r, h] = ln sum_{t <= p} exp(scale <q[r, h], K[t, g]>),  g = h / (Hq/Hkv).
 * Rows r are packed in call order, as for treepo_kv_append.
 *   q          device bf16 [sum ntok][Hq][D]
 *   k, v       device bf16 [sum ntok][Hkv][D] (written into the pools)
 *   scale      softmax scale, positive and finite
 *   out        device fp32 [sum ntok][Hq][D] (written)
 *   lse        device fp32 [sum ntok][Hq] (written) or null
 *   workspace  device, 256-byte aligned, >= treepo_prefill_workspace_size for
 *              the same arguments; the call uploads its work items, tile
 *              tables and per-XCD schedule there
 *              (contents need not be preserved between calls, but a call's
 *              kernels read it until they finish on stream).
 * Validation as treepo_kv_append, plus EINVAL (a node twice in one call, null
 * q/k/v/out or bad scale with tokens, a chain of 2^25 tokens or more) and
 * EWORKSPACE; a call that fails validation changes nothing.  EHIP (a failed
 * upload or launch) comes after the append was enqueued: the lengths have
 * advanced and the out/lse contents are undefined.  Enqueued on stream. */
int32_t treepo_prefill_workspace_size(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok,
                                      size_t* bytes);
int32_t treepo_prefill(treepo_ctx* ctx, int32_t n, const int32_t* nodes, const int32_t* ntok, const void* q,
                       const void* k, const void* v, float scale, float* out, float* lse, void* workspace,
                       size_t ws_bytes, hipStream_t stream);

/* Pool token rows (block * B + offset) that the next treepo_kv_append /
 * treepo_kv_commit with the same arguments would fill, in call order
 * (rows_out: host, sum(ntok) entries).  For callers that write K/V into the
 * pools with their own kernels.  Same validation as treepo_kv_append; no state
 * change. */
int32_t treepo_kv_slots(treepo_ctx* ctx, int32_t n, const int32_t* nodes,
                        const int32_t* ntok, int64_t* rows_out);

/* Advances lengths exactly like treepo_kv_append but writes no K/V: the
 * caller has already written the rows given by treepo_kv_slots. */
int32_t treepo_kv_commit(treepo_ctx* ctx, int32_t n, const int32_t* nodes,
                         const int32_t* ntok);

/* Workspace bytes that a decode of these leaves needs (mode TREEPO_MODE_TREE
 * or TREEPO_MODE_NAIVE).  Builds and caches the decode plan. */
int32_t treepo_decode_workspace_size(treepo_ctx* ctx, int32_t n_leaves,
                                     const int32_t* leaves, int32_t mode,
                                     size_t* bytes);

/* One decode step of attention for n_leaves leaves (Sec. 2.2 segment-level
 * decoding; Sec. 2.3 chains).  leaves: host node ids (any node, duplicates
 * allowed), call position i.
 *   q     device bf16 [n_leaves][Hq][D]   the step's queries (16-byte aligned)
 *   scale softmax scale, positive and finite (e.g. 1/sqrt(D))
 *   out   device fp32 [n_leaves][Hq][D]   softmax(scale q K^T) V over the chain
 *   lse   device fp32 [n_leaves][Hq] or null: natural-log sum exp(scale q.k)
 *   workspace  device, 256-byte aligned, >= treepo_decode_workspace_size(..., TREEPO_MODE_TREE)
 * Cascade schedule: every node's K/V is read once and scored against all of
 * its descendant leaves' query rows (the nested sub-groups G_j of Sec. 2.3);
 * per-node partials are merged with a log-sum-exp combine (partial rows in
 * fp32, or, for schedules whose partials far exceed the L2, in block floating
 * point -- 14-bit mantissas under a shared exponent per 4 values: an output
 * then moves by less than 2^-13 of the largest |V| value it averages;
 * accumulation is fp32 throughout).  Non-finite inputs give non-finite
 * outputs where the definition does (a NaN or infinity in V spoils its
 * column; in block floating point the column's group of 4).  The schedule
 * (plan) is cached per context (the last four leaf lists and modes) and its
 * device image lives in memory the context allocates (see the ownership rule
 * above); the workspace holds only this call's partial results, so the
 * caller may reuse it freely between calls (calls that overlap on one
 * workspace race).
 * EINVAL (bad id, null pointer, n_leaves < 1, q not 16-byte aligned, scale
 * not positive and finite),
 * EEMPTY (a chain holds no tokens), EWORKSPACE (missing, too small or not
 * 256-byte aligned), EHIP. */
int32_t treepo_tree_decode(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                           const void* q, float scale, float* out, float* lse,
                           void* workspace, size_t ws_bytes, hipStream_t stream);

/* The per-leaf paged-decode baseline: same contract and results as
 * treepo_tree_decode, but every leaf streams its whole chain's blocks on its
 * own, so shared prefixes are read once per descendant leaf (the separate
 * per-path KV that Sec. 1 contrasts with sharing).  Workspace from mode
 * TREEPO_MODE_NAIVE. */
int32_t treepo_paged_decode_naive(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                                  const void* q, float scale, float* out, float* lse,
                                  void* workspace, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code that may not call
 * hipMalloc, tight serving loops, harnesses that forbid it): the cascade
 * decode of treepo_tree_decode with the same arguments and results, minus
 * the workspace.  The plan image and the partial slots live in a static
 * device array of the library, 64 MiB per device (each device the library
 * runs on holds its own until the process ends), not in memory the call
 * allocates: it calls no hipMalloc, hipFree or pinned-memory allocation
 * (plan and length uploads are copied from pageable host memory, and a plan
 * evicted from the cache keeps its image buffer for a later allocating
 * call to free).  Every call on a device shares that array and leaves its
 * contents there; the plan image is uploaded only when another plan used
 * the array since, and partial slots are always rewritten before they are
 * read.  Calls that overlap on one device race: issue them on one stream or
 * synchronise between them.  EWORKSPACE when the plan image plus the
 * partial slots exceed 64 MiB (treepo_last_error gives the bytes needed);
 * otherwise the errors of treepo_tree_decode. */
int32_t treepo_tree_decode_noalloc(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, const void* q,
                                   float scale, float* out, float* lse, hipStream_t stream);

/* ---- branching budget ---------------------------------------------------- */

#define TREEPO_BUDGET_EVEN 0       /* budget transfer: spread evenly (Sec. 2.2)                */
#define TREEPO_BUDGET_HIGH_PROB 1  /* softmax(score / T): higher probability favoured (Sec. 4.4) */
#define TREEPO_BUDGET_LOW_PROB 2   /* softmax(-score / T): lower probability favoured (Sec. 4.4) */

/* Branches per active path before the next segment step (Sec. 2.2 "Branching
 * Budget Transfer"; Sec. 4.4 probability-based assignment, temperature 2.0
 * there).  Host only, no context.
 *   scores      host [n_paths]: the log probability of each path's last
 *               segment (ignored, may be null, for TREEPO_BUDGET_EVEN)
 *   total       the depth's branching budget (e.g. N^d)
 *   budget_out  host [n_paths] (written): every path gets 1; the other
 *               max(total - n_paths, 0) are split in proportion to 1/n or
 *               the softmax weights (double, maximum subtracted) by largest
 *               remainders, ties to the lower index.  Sums to
 *               max(total, n_paths).
 * EINVAL (n_paths < 1, null budget_out, total < 0, bad mode, non-finite
 * score, temperature not positive and finite). */
int32_t treepo_branch_budget(int32_t n_paths, const float* scores, int32_t total, int32_t mode,
                             float temperature, int32_t* budget_out);

/* ---- TreePO advantage ---------------------------------------------------- */

/* Aggregations for treepo_tree_advantage. */
#define TREEPO_ADV_MEAN 0           /* mean over sub-groups (Sec. 2.3, Eq. tree_ae)         */
#define TREEPO_ADV_SIZE_WEIGHTED 1  /* |G_j|-weighted mean (Sec. 4.2, Eq. tree_ae_sgw)      */

/* Workspace bytes that treepo_tree_advantage needs for these leaves. */
int32_t treepo_advantage_workspace_size(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                                        size_t* bytes);

/* TreePO advantage of every trajectory (Sec. 2.3: Eq. groups, Eq. tree_ae;
 * Fig. 3 caption).  Call position p is a trajectory: the chain of node
 * leaves[p] (any node; duplicates allowed).  A query is a root; its group G
 * holds every position under it.  The sub-groups of p are, for each strict
 * predecessor a of leaves[p] (root first), G_a = the positions whose chain
 * contains a.  With R = rewards:
 *   A_{p,a} = R_p - mean over G_a of R;
 *   pooled_p = mean over a of A_{p,a} (TREEPO_ADV_MEAN), or the
 *              |G_a|-weighted mean (TREEPO_ADV_SIZE_WEIGHTED);
 *   adv_p = pooled_p / sigma, sigma = the population standard deviation of
 *           every A_{p,a} of every kept query (one global normalisation).
 * A query whose rewards are all equal is rejected (the paper's constraint
 * std(R over G) != 0): its positions get 0 and add nothing to sigma; so does
 * a position with no predecessor (a root).  If sigma is 0, every adv is 0.
 *   rewards   device fp32 [n_leaves]
 *   adv       device fp32 [n_leaves] (written)
 *   workspace device, 256-byte aligned, >= treepo_advantage_workspace_size;
 *             the call uploads its index arrays there (contents need not
 *             survive between calls)
 * Arithmetic in fp64 on the device, in a fixed order (deterministic).
 * EINVAL (bad id, null pointer, n_leaves < 1, bad weighting), EWORKSPACE,
 * EHIP.  Leaves need not hold tokens. */
int32_t treepo_tree_advantage(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                              const float* rewards, int32_t weighting, float* adv, void* workspace,
                              size_t ws_bytes, hipStream_t stream);

/* ---- metadata export (host arrays) -------------------------------------- */

/* Number of nodes created so far. */
int32_t treepo_num_nodes(treepo_ctx* ctx, int32_t* n_nodes);

/* Node records, TREEPO_NODE_FIELDS int32 per node in id order, for the first
 * min(capacity, n_nodes) nodes; *n_nodes receives the node count. */
int32_t treepo_export_nodes(treepo_ctx* ctx, int32_t* records, int32_t capacity,
                            int32_t* n_nodes);

/* Per-leaf chains (root first) and leaf block tables (each chain node's first
 * ceil(len/B) blocks, in chain order) as CSR arrays:
 *   chain_off[n_leaves+1], chain_nodes[*total_chain],
 *   block_off[n_leaves+1], blocks[*total_blocks].
 * Pass null arrays to query the totals only. */
int32_t treepo_export_chains(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                             int32_t* chain_off, int32_t* chain_nodes,
                             int32_t* block_off, int32_t* blocks,
                             int32_t* total_chain, int32_t* total_blocks);

/* Node -> descendant-leaf sets of one decode call (Sec. 2.3, Eq. groups):
 * every node on some chain, ascending id (nodes[*n_nodes]), with the ascending
 * call positions whose chain contains it (desc_off[*n_nodes+1], desc[*total]).
 * Pass null arrays to query the sizes only. */
int32_t treepo_export_desc(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                           int32_t* nodes, int32_t* desc_off, int32_t* desc,
                           int32_t* n_nodes, int32_t* total);

/* The decode schedule for inspection.  The chain nodes are cut into runs
 * (maximal chain segments whose nodes have the same descendant leaves); each
 * (run, leaf group, KV head) is a sequence of 32-token tiles; the sequences
 * are cut into streams of equal estimated cost, one workgroup each, and a
 * piece is the part of one sequence inside one stream.  Pieces,
 * TREEPO_PIECE_FIELDS int32 each, in stream order:
 *   {rowset_begin, n_leaves, rows, kv_head, stream_tile, n_tiles,
 *    0, seg_begin, run, stream, plan_tile, n_qtiles, 0, 0, 0, 0}
 * rows = n_leaves * (Hq / Hkv); the piece's leaves are rowsets[rowset_begin ..
 * + n_leaves) (call positions); in its stream's tile list it is n_qtiles
 * query tiles (64 rows each) from stream_tile on, then n_tiles KV tiles, and
 * its query segments start at seg_begin there; its KV tiles are
 * tiles[plan_tile .. + n_tiles),
 * TREEPO_TILE_FIELDS int32 each {block, node, tile_in_node, valid_tokens}
 * (valid_tokens as of planning; with node_len a plan is reused while nodes
 * grow and the kernels read the current counts of tiles not yet full):
 * tile k of a node holds its tokens [32k, 32k+32) and starts in pool block
 * block_begin + 32k/B.  *n_streams receives the stream count.  Pass null arrays
 * to query the counts only. */
int32_t treepo_export_plan(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves,
                           int32_t mode, int32_t* pieces, int32_t* rowsets, int32_t* tiles,
                           int32_t* n_pieces, int32_t* n_rowsets, int32_t* n_tiles,
                           int32_t* n_streams);

/* The device copy of the same schedule, as the node-partial kernel reads it:
 * one block of *block_ints int32 per stream (a multiple of 4; stream s at
 * s * block_ints, *n_streams blocks):
 *   {n_pieces, n_tiles, n_segs, 0};
 *   per piece {rows, stream_tile, n_tiles, seg_begin};
 *   per stream tile {hb, valid}, padded to an even count: a KV tile has
 *     hb = 2 * (kv_head * num_blocks + block) + tile_in_node % 2 and valid =
 *     its tokens; a query tile has hb = -1 - (its piece's seg_begin) and
 *     valid = first_row | (n_rows << 16);
 *   per query segment, the element offset (x * Hq + kv_head * G) * D of the
 *     G query rows of the piece's leaf x, padded to a multiple of 4;
 *   per query segment, the partial row (base(key) + e) * G of the piece's
 *     entry for its leaf x, key = x * Hkv + kv_head, where e counts the
 *     pieces before it (plan order) that cover the same key; base(key) =
 *     key * E (E the largest count over the keys) when the combine's
 *     speculative first round, the O rows of min(E, 32) entries of every key
 *     (N keys * G * min(E, 32) * (4 D + 8) bytes), is at most 8 MiB, else
 *     the sum of the counts of the keys before it; padded to a multiple of 4.
 * Pass a null array to query the sizes only. */
int32_t treepo_export_blocks(treepo_ctx* ctx, int32_t n_leaves, const int32_t* leaves, int32_t mode,
                             int32_t* blocks, int32_t* block_ints, int32_t* n_streams);

/* ---- kernel timing ------------------------------------------------------ */

/* Kernel kinds for treepo_profile_read. */
#define TREEPO_KERNEL_APPEND 0  /* KV scatter into the pools                      */
#define TREEPO_KERNEL_PARTIAL 1 /* node partials, one workgroup per stream         */
#define TREEPO_KERNEL_COMBINE 2 /* log-sum-exp merge of each leaf's partials      */
#define TREEPO_KERNEL_ADVANTAGE 3 /* TreePO advantage over the leaves' sub-groups  */
#define TREEPO_KERNEL_PREFILL 4 /* causal attention of prefilled tokens          */
#define TREEPO_KERNEL_KINDS 5

/* When enabled, every kernel launch of this context is timed with HIP events
 * on the launch stream: the decode kernels (partial, combine) get events that
 * the launch attaches to the kernel itself (hipExtLaunchKernelGGL: recorded
 * at its start and end), the append kernel's launches are bracketed by
 * events.  Enabling or disabling clears the totals. */
int32_t treepo_set_profiling(treepo_ctx* ctx, int32_t enable);
/* Total milliseconds and launch count per kernel kind since profiling was
 * enabled; waits for the recorded events to complete. */
int32_t treepo_profile_read(treepo_ctx* ctx, int32_t kind, double* total_ms,
                            int64_t* launches);

/* ---- errors ------------------------------------------------------------- */
const char* treepo_strerror(int32_t code);
/* Message of the last failing call on ctx (empty if none). */
const char* treepo_last_error(treepo_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* TREEPO_H */
