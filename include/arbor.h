/*
 * arbor.h -- C ABI of a gfx950 (MI355X) library for structure-aware KV eviction
 * in Tree-of-Thoughts decoding, after ArborKV (arxiv 2605.22106).
 *
 * The library implements the data-parallel hot path of the method:
 *   arbor_score             MSVE block score (Sec. 4): accumulated attention A_i(t)
 *                           of later tokens, block attention a_i, s_i.
 *   arbor_allocate          TAE keep-counts (Eq. 2, Eq. 3) under a global budget
 *                           (KKT view of Sec. 4; Transition/Pressure of Alg. 2).
 *   arbor_select            tail + heavy-hitter retained set per block (Sec. 4
 *                           Execution; Alg. 1 Evict).
 *   arbor_compact           token-extractive, order-preserving compaction of the
 *                           retained K/V inside a paged tree KV pool (Sec. 4).
 *   arbor_select_compact    the two above on the same k, in fewer launches.
 *   arbor_rehydrate         lazy rehydration of Path* blocks (Sec. 4; Alg. 2).
 *   arbor_tree_decode_attn  decode attention of each active leaf over its
 *                           ancestor chain (Sec. 1 and Sec. 3: the next step
 *                           depends only on the chain).
 *   arbor_uncertainty       normalised next-token entropy u_i at block
 *                           boundaries (Sec. 4 MSVE, Eq. 1), the input u_in of
 *                           arbor_score.
 *
 * Conventions
 *  - Every pointer is a DEVICE pointer unless marked (host) or (pinned host).
 *    Struct arguments themselves are host memory, read during the call only.
 *  - Every call enqueues work on `stream` and returns without synchronising.
 *    The C return value reports host-side argument validation and launch
 *    failures.  Outcomes that depend on device data are written to the device
 *    int32 *status (read it after synchronising the stream).
 *  - *status is sticky: a call does nothing on the device when *status < 0 on
 *    entry, writes a negative code on error and ARBOR_OVER_BUDGET (1) as a
 *    warning only over ARBOR_OK.  The caller zeroes it at the start of a
 *    sequence of calls (one policy event).
 *  - On any negative status every piece of pool/tree state (n_kept, page_table,
 *    slot_pos, free_stack, free_top, K/V bytes of retained tokens) is unchanged;
 *    pure outputs (k_out, sel_pos, out, ...) are then unspecified.
 *  - The library allocates no memory.  The caller owns every buffer, including
 *    the scratch `workspace` of `workspace_bytes` bytes (at least
 *    arbor_workspace_size()).  Calls on distinct buffers are independent;
 *    calls that share a workspace must be ordered (same stream).
 *  - Node ids satisfy parent[0] = -1 and 0 <= parent[i] < i (creation order;
 *    BFS order qualifies).  Depth of any node <= ARBOR_MAX_DEPTH.
 *  - Positions are node-local: position p of node i is token a_i + p of the
 *    paper's span x_{a_i:b_i}.  Per-token arrays (A, sel_pos) are indexed by
 *    tok_off[i] + p.
 */
#ifndef ARBOR_H
#define ARBOR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARBOR_MAX_DEPTH 63

typedef enum {
  ARBOR_OK = 0,
  ARBOR_OVER_BUDGET = 1,    /* warning: even the minimum counts exceed the budget  */
  ARBOR_EINVAL = -1,        /* bad argument or malformed tree/selection            */
  ARBOR_ENOPAGES = -2,      /* rehydration needs more pages than are free          */
  ARBOR_EHIP = -3,          /* a HIP launch failed                                 */
  ARBOR_EUNSUPPORTED = -4,  /* shape outside what the kernels implement            */
  ARBOR_ENONFINITE = -5,    /* NaN in A or s; NaN or infinite logit                */
  ARBOR_EWORKSPACE = -6,    /* workspace too small for this tree                   */
  ARBOR_ECORRUPT = -7       /* pool bookkeeping inconsistent (free stack overflow) */
} arbor_status_t;

typedef enum { ARBOR_BF16 = 0, ARBOR_F32 = 1 } arbor_dtype_t;

/* Intra-block retention rules (Sec. 4 Execution; the three rows of Table 7). */
typedef enum {
  ARBOR_SELECT_TAIL_HEAVY = 0,  /* global sinks + block tail + heavy hitters by A        */
  ARBOR_SELECT_TAIL_ONLY = 1,   /* the most recent resident tokens, no sinks             */
  ARBOR_SELECT_SINKS_TAIL = 2   /* global sinks, then the most recent resident tokens    */
} arbor_select_mode_t;

/* Kernels of the path that a caller can time on their own (arbor_timing_t). */
typedef enum {
  ARBOR_KERNEL_SCORE_ATTN = 0,    /* the two-pass score kernel of arbor_score      */
  ARBOR_KERNEL_SELECT = 1,        /* the selection kernel of arbor_select          */
  ARBOR_KERNEL_COMPACT_MOVE = 2,  /* the row-move kernel of arbor_compact          */
  ARBOR_KERNEL_DECODE_ATTN = 3,   /* the attention kernels of arbor_tree_decode_attn */
  ARBOR_KERNEL_DECODE_CREDIT = 4, /* the merge-and-credit kernel of
                                     arbor_tree_decode_attn_scored                 */
  ARBOR_KERNEL_COUNT = 5
} arbor_kernel_t;

/* (host) A timing request that belongs to one call: when a call launches
 * `kernel`, it records `start` on the launch stream right before that launch
 * and `stop` right after it (for ARBOR_KERNEL_DECODE_ATTN around the up to
 * three attention launches of the call, which run back to back), so
 * hipEventElapsedTime(start, stop) after the stream has synchronised is the
 * kernel's own duration.  The caller owns the events (created with timing on
 * the device of the call) and the struct; the library keeps no reference
 * after the call returns.  Calls that do not launch `kernel` record nothing. */
typedef struct {
  int32_t kernel;           /* arbor_kernel_t                                     */
  hipEvent_t start;
  hipEvent_t stop;
} arbor_timing_t;

/* (host) Shape of the KV pool.  head_dim in {64, 128}; page_size a multiple of
 * 16 and at most 256; q_per_kv = G query heads share one KV head (query head h
 * reads KV head h / G).  `timing` is an optional per-call timing request
 * (NULL: none); it is read during the call only. */
typedef struct {
  int32_t num_layers;
  int32_t num_kv_heads;
  int32_t q_per_kv;
  int32_t head_dim;
  int32_t page_size;
  int32_t dtype;            /* arbor_dtype_t of K, V, q_win and decode q */
  int64_t num_pages;
  const arbor_timing_t *timing;   /* (host, nullable) */
} arbor_geom_t;

/* (host struct of device pointers) The thought tree T = (V, E) of Sec. 3. */
typedef struct {
  int32_t num_nodes;         /* V                                                 */
  int64_t num_tokens;        /* N = tok_off[V]                                    */
  const int32_t *parent;     /* [V]  parent[0] = -1                               */
  const int32_t *n_full;     /* [V]  n_i = b_i - a_i + 1                          */
  const int64_t *tok_off;    /* [V+1] prefix sum of n_full                        */
  const int64_t *page_off;   /* [V+1] prefix sum of ceil(n_full / page_size)      */
  int32_t *n_kept;           /* [V]  c_i, resident tokens (in/out)                */
  int32_t *page_table;       /* [page_off[V]] physical page of logical page q of
                                node i at page_off[i] + q; -1 = unused (in/out)   */
} arbor_tree_t;

/* (host struct of device pointers) The paged tree KV pool.  Slot s of node i
 * lives in page page_table[page_off[i] + s / P] at row s % P; the resident
 * slots of a node hold strictly increasing positions. */
typedef struct {
  void *k;                   /* [L][num_pages][Hkv][P][head_dim] dtype            */
  void *v;                   /* same layout                                      */
  int32_t *slot_pos;         /* [num_pages][P] position held by a slot, -1 empty  */
  int32_t *free_stack;       /* [num_pages] free pages in [0, *free_top)          */
  int32_t *free_top;         /* [1] number of free pages; the top is free_top-1   */
} arbor_pool_t;

/* (host) Parameter bundle of Alg. 1 / Alg. 2.  The paper prints no values. */
typedef struct {
  double alpha_max;          /* upper bound of the global scale alpha (Eq. 2); +inf
                                means alpha is set by the budget alone (KKT view)   */
  double gamma;              /* importance exponent (Eq. 2)                         */
  double lambda_d;           /* depth decay (Eq. 2)                                 */
  double lambda_delta;       /* distance-to-active-leaf decay (Eq. 2)               */
  double eta;                /* off-path discount, 0 < eta <= 1 (Eq. 2)             */
  double r_min;              /* ratio floor (Eq. 2)                                 */
  int32_t k_min;             /* per-block minimum K_min (invariant (ii), Eq. 3)     */
  int32_t l_tail;            /* tail window L_tail (Eq. 3, Sec. 4 Execution)        */
  float theta[3];            /* MSVE weights on phi = [v, u, a]                     */
  float softmax_scale;       /* score attention scale; <= 0 means 1/sqrt(head_dim)  */
  int32_t select_mode;       /* arbor_select_mode_t                                 */
  int32_t score_self_window; /* 0: credit proper ancestors only (u > b_i);
                                1: also an observer's own earlier tokens            */
  int32_t lazy_rehydration;  /* 1: Path* blocks are restored to full retention
                                (arbor_rehydrate) and count n_i; 0: evicted tokens
                                stay lost for the episode, Path* blocks keep (and
                                count) their resident c_i                           */
  int32_t n_sinks;           /* |S|: the global sinks are positions [0, n_sinks) of
                                the root block 0, the initial prompt (Sec. 4
                                Execution (i)); 0 = none                            */
  int32_t k_protect;         /* active-path protection (Sec. 3 invariant (i)): 0 =
                                full (Path* blocks keep all n_i tokens); > 0 = a
                                floor: Path* blocks take part in Eq. 2-3 without
                                the eta discount and keep at least k_protect
                                tokens (up to n_i, or c_i without rehydration)      */
} arbor_params_t;

/* (host) Upper bounds used to size the workspace. */
typedef struct {
  int32_t num_nodes;         /* V                                                 */
  int64_t num_tokens;        /* N                                                 */
  int64_t max_context;       /* >= sum of n_full over any root-to-node chain      */
  int32_t max_observers;     /* arbor_score: largest n_obs                        */
  int32_t window;            /* arbor_score: W                                    */
  int32_t n_slice;           /* arbor_score: slice layers per call                */
  int32_t max_leaves;        /* arbor_tree_decode_attn: largest n_leaves          */
  int32_t max_layers;        /* arbor_tree_decode_attn: largest layer_end-begin   */
} arbor_sizes_t;

/* Bytes of workspace that every call of the library needs for these bounds. */
size_t arbor_workspace_size(const arbor_geom_t *geom, const arbor_sizes_t *sizes);

/* Static text for a status code. */
const char *arbor_strerror(int code);

/*
 * arbor_score -- MSVE scoring (Sec. 4 "Multi-Signal Value Estimation": the
 * accumulated attention A_i(t) over a thin slice of layers and heads, the block
 * attention a_i and s_i = clip(sigmoid(theta^T [v_i, u_i, a_i]), 0, 1);
 * Alg. 1 MSVE).
 *
 * For each observer j = observers[o], slice layer slice_layers[s] and query
 * head h, the window query of position u = n_j - w_j + t (t < w_j =
 * min(window, n_j)) is q_win[o][s][h][t][:] (layout [n_obs][n_slice][Hq]
 * [window][head_dim], dtype geom->dtype).  It attends (softmax, scale
 * params->softmax_scale) over every resident token of j's proper ancestors and
 * j's own resident tokens at positions <= u.  Its probability on each token of
 * a proper ancestor of j (also on j's tokens p < u when score_self_window = 1)
 * is added to A[tok_off[i] + p]; rows_seen[i] grows by the number of such rows
 * that credited block i.  Then for every node
 *   a_out[i] = sum_{p < n_i} A[tok_off[i] + p] / rows_seen[i]   (0 if never seen)
 *   s_out[i] = clip(sigmoid(theta[0] v_in[i] + theta[1] u_in[i] + theta[2] a_out[i]), 0, 1).
 * A is fp32 [N] (in/out), rows_seen int64 [V] (in/out), v_in/u_in/a_out/s_out
 * fp32 [V].  slice_layers is a (host) array of n_slice (<= 8) layer ids.
 * Results are bitwise reproducible run to run (no atomics in any sum).  With
 * n_obs = 0 (observers and q_win may be NULL) A and rows_seen are unchanged
 * and only a_out, s_out are computed.  On an error status A, rows_seen, a_out
 * and s_out are left unchanged.
 * Errors: EINVAL (bad ids), EWORKSPACE, EUNSUPPORTED (page_size/head_dim, an
 * observer deeper than ARBOR_MAX_DEPTH).
 */
int arbor_score(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                const int32_t *observers, int32_t n_obs, const void *q_win, int32_t window,
                const int32_t *slice_layers, int32_t n_slice, const float *v_in,
                const float *u_in, float *A, int64_t *rows_seen, float *a_out, float *s_out,
                const arbor_params_t *params, int32_t *status, void *workspace,
                size_t workspace_bytes, hipStream_t stream);

/*
 * arbor_allocate -- tree-aware keep-counts (Eq. 2 and Eq. 3; the KKT view of
 * Sec. 4; the Transition and Pressure branches of Alg. 2).
 *
 * Path* = union of the root-to-leaf chains of active[0 .. n_active) (device
 * int32).  delta_out[i] = tree distance from i to the nearest active leaf,
 * on_path_out[i] = 1 on Path* (uint8).  With full protection
 * (params->k_protect = 0) Path* nodes get k = n_i (invariant (i)), or k = c_i
 * when params->lazy_rehydration = 0 (no restoring).  Every other node i gets
 * Eq. 3 at its Eq. 2 ratio r_i = clip(alpha w_i, r_min, 1),
 * w_i = eta^[i not in Path*] s_i^gamma e^{-lambda_d d_i} e^{-lambda_delta Delta_i},
 * capped at its resident count c_i (off-path blocks are only ever lowered),
 * where alpha is the largest value <= alpha_max whose total fits
 * budget_tokens.  With floor protection (k_protect > 0) Path* nodes are among
 * those "other" nodes, with the floor max(Eq. 3 floor, k_protect) and the cap
 * n_i (c_i when lazy_rehydration = 0).  Token j of block i is kept when
 * alpha >= j / (w_i n_i) (its price, fp64); equal prices enter together.  If
 * the Eq. 3 floors already exceed the budget (Pressure) off-path blocks are
 * lowered towards min(K_min, c_i) in ascending w_i (ties: lower id); if that
 * is not enough *status gets ARBOR_OVER_BUDGET and k_out holds the lowered
 * counts.
 * s is fp32 [V] in [0, 1] (the clipped MSVE score; -0 counts as +0); k_out
 * int32 [V].  fp64 arithmetic, no contraction; s^gamma is correctly rounded
 * for gamma in {1, 2, 3, 4} and the device pow otherwise.
 * Errors: EINVAL (malformed tree, bad leaf ids, n_active < 1, an off-path s
 * outside [0, 1]), ENONFINITE (NaN s off the path).
 */
int arbor_allocate(const arbor_tree_t *tree, const int32_t *active, int32_t n_active,
                   int64_t budget_tokens, const float *s, const arbor_params_t *params,
                   int32_t *k_out, int32_t *delta_out, uint8_t *on_path_out, int32_t *status,
                   void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * arbor_select -- retained set of every block whose count drops (Sec. 4
 * Execution: mandatory tail T_i and heavy hitters H_i by A_i(t), tail first on
 * overlap; Alg. 1 Evict).
 *
 * For every node with k[i] < c_i: tail = resident positions >= n_i - L_tail.
 * If k[i] <= |tail| or select_mode = TAIL_ONLY, the k[i] most recent resident
 * positions are kept; otherwise the tail plus the k[i] - |tail| other resident
 * positions with the largest A (fp32 compare, -0 == +0), ties to the lower
 * position.  The global sinks (resident positions < n_sinks of the root block
 * 0) come before everything else in the TAIL_HEAVY and SINKS_TAIL modes: the
 * root keeps its k[0] lowest sinks if k[0] is smaller, else all of them plus
 * the rule applied to its other tokens with k[0] - |sinks| (SINKS_TAIL: the
 * most recent ones).  sel_pos[tok_off[i] + s] (s < k[i]) receives the kept
 * positions in ascending order; entries of other nodes are not written.
 * Errors: ENONFINITE (NaN in A over a changed block), EINVAL (k < 0).
 */
int arbor_select(const arbor_geom_t *geom, const arbor_tree_t *tree, const arbor_pool_t *pool,
                 const float *A, const int32_t *k, const arbor_params_t *params,
                 int32_t *sel_pos, int32_t *status, hipStream_t stream);

/*
 * arbor_compact -- token-extractive compaction (Sec. 4 Execution: retained
 * entries stay, the rest are freed).  For every node with k[i] < c_i, slot s
 * (s < k[i]) afterwards holds position sel_pos[tok_off[i] + s], its K/V rows of
 * every layer and KV head copied bitwise from the slot that held it (in place,
 * order preserving).  The node keeps its first ceil(k[i]/P) pages; the rest go
 * on the free stack in (node, page) order; vacated slots and freed pages get
 * slot_pos = -1, unused page-table entries -1; n_kept[i] = k[i].
 * Errors: EINVAL (selection not a strictly increasing subset of the resident
 * positions), ECORRUPT (free stack would overflow).
 */
int arbor_compact(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                  const int32_t *k, const int32_t *sel_pos, int32_t *status, void *workspace,
                  size_t workspace_bytes, hipStream_t stream);

/*
 * arbor_select_compact -- arbor_select followed by arbor_compact on the same
 * k, in two launches instead of three to four (Sec. 4 Execution; Alg. 1
 * Evict): the wave that selects a block's retained set also writes its
 * compaction plan, as it knows the slot of every kept position, and the
 * free-stack scan runs in the same launch.  Writes exactly what
 * arbor_select then arbor_compact write (sel_pos included), from the same
 * arguments; the workspace is sized as for arbor_compact.
 * Errors: those of arbor_select (ENONFINITE, EINVAL) and ECORRUPT (free stack
 * would overflow); every error leaves the tree and pool unchanged.
 */
int arbor_select_compact(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                         const float *A, const int32_t *k, const arbor_params_t *params,
                         int32_t *sel_pos, int32_t *status, void *workspace,
                         size_t workspace_bytes, hipStream_t stream);

/*
 * arbor_compact_noalloc -- arbor_compact for callers that cannot allocate
 * memory: code under stream capture, tight serving loops, harnesses that
 * forbid allocation.  It takes no workspace; its scratch is a device array of
 * ARBOR_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends.  It allocates nothing (no hipMalloc, no hipFree, no
 * allocating library routine) and writes exactly what arbor_compact writes.
 * Limit: 12 bytes per token of the tree plus 16 per node (and 8 KiB) must fit
 * the array, which holds trees of up to about 2.7 M tokens; a larger tree is
 * refused with ARBOR_EWORKSPACE before anything is enqueued.  All calls on one
 * GPU share its array: calls that overlap on one GPU (unordered streams)
 * race and must not be issued.  Other errors as arbor_compact.
 */
#define ARBOR_NOALLOC_SCRATCH_BYTES (32u << 20)
int arbor_compact_noalloc(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                          const int32_t *k, const int32_t *sel_pos, int32_t *status,
                          hipStream_t stream);

/*
 * arbor_rehydrate -- lazy rehydration (Sec. 4 "Lazy rehydration"; Alg. 2
 * Transition): every node with on_path[i] != 0 and c_i < n_i is restored to
 * full retention before the next decode step, in ascending id (root first).
 * Its missing pages are popped from the top of the free stack in (node, page)
 * order; afterwards slot p holds position p.  Resident rows move bitwise;
 * evicted rows are copied bitwise from the token-span record host_k/host_v
 * ((pinned host) or device, layout [N][L][Hkv][head_dim], dtype), read by the
 * kernel over the host link.  Errors: ENOPAGES (checked before any change).
 */
int arbor_rehydrate(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
                    const uint8_t *on_path, const void *host_k, const void *host_v,
                    int32_t *status, void *workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * arbor_tree_decode_attn -- decode attention of each active leaf over the
 * resident tokens of its root-to-leaf chain (Sec. 1, Sec. 3).  For leaf
 * leaves[b], layer l in [layer_begin, layer_end) and query head h:
 *   out[b][l - layer_begin][h][:] = softmax(scale q K^T) V
 * over every resident slot of every chain node (the leaf's newest token is the
 * query's own position), q layout [n_leaves][Lr][Hq][head_dim] (dtype), out in
 * out_dtype, lse_out [n_leaves][Lr][Hq] fp32 natural-log LSE (nullable).
 * Each chain node is read once for all active leaves below it; partial results
 * are merged per leaf root to leaf, so results are bitwise reproducible.  A
 * leaf whose chain holds no resident token gets out = 0 and lse = -inf.
 * n_leaves = 0 (or layer_end = layer_begin) does nothing; leaves, q and out
 * may then be NULL.
 * Errors: EINVAL, EWORKSPACE, EUNSUPPORTED (a leaf deeper than
 * ARBOR_MAX_DEPTH).
 */
int arbor_tree_decode_attn(const arbor_geom_t *geom, const arbor_tree_t *tree,
                           const arbor_pool_t *pool, const int32_t *leaves, int32_t n_leaves,
                           int32_t layer_begin, int32_t layer_end, const void *q, void *out,
                           int32_t out_dtype, float *lse_out, float softmax_scale,
                           int32_t *status, void *workspace, size_t workspace_bytes,
                           hipStream_t stream);

/*
 * arbor_tree_decode_attn_scored -- arbor_tree_decode_attn that also grows the
 * accumulated attention A_i(t) from the weights of this decoding step (Sec. 4
 * Execution (iii): A is kept up to date from attention weights the decoding
 * already materialises, over a thin slice of layers and all heads).
 *
 * Outputs out / lse_out exactly as arbor_tree_decode_attn (bitwise the same
 * values).  In addition, for every leaf b, slice layer l = slice_layers[s]
 * (each in [layer_begin, layer_end)) and query head h, the decode softmax
 * weight of every resident key of a proper ancestor i of the leaf is added to
 * A[tok_off[i] + position] (the query sits at the leaf's newest position,
 * after every ancestor's end), and rows_seen[i] grows by n_slice * Hq per leaf
 * below i.  With self_window = 1 the leaf's own keys at positions below its
 * newest one (p < n_leaf - 1) are credited too and rows_seen[leaf] grows by
 * n_slice * Hq.  For leaves with at least one token this equals arbor_score
 * with the leaves as observers, window 1 and q_win taken from q's slice
 * layers.  The sums are formed in a fixed order per token (no atomics on A):
 * bitwise reproducible.  A is fp32 [N] and rows_seen int64 [V], both in/out;
 * nothing else of the tree or pool changes.
 */
typedef struct {
  const int32_t *slice_layers;  /* (host) n_slice layer ids in [layer_begin, layer_end) */
  int32_t n_slice;              /* 1..8                                              */
  int32_t self_window;          /* 0 or 1, as arbor_params_t.score_self_window        */
  float *A;                     /* device, fp32 [N], in/out                          */
  int64_t *rows_seen;           /* device, int64 [V], in/out                         */
} arbor_decode_credit_t;

/* The attention units keep the logits of the distinct slice layers (fp32,
 * CHUNK = 256 per unit row and kv head) in the workspace; the launch that
 * merges the partials also turns them into the credited weights, its credit
 * workgroups forming each row's log-sum-exp from the chain's partials
 * themselves.  The workspace must be sized with arbor_sizes_t.n_slice >=
 * n_slice.
 * Errors: those of arbor_tree_decode_attn; EINVAL for a slice layer outside
 * [layer_begin, layer_end), n_slice outside 1..8, self_window not 0 or 1, or A /
 * rows_seen NULL with n_leaves > 0; EWORKSPACE (device) when the workspace
 * cannot hold the kept logits. */
int arbor_tree_decode_attn_scored(const arbor_geom_t *geom, const arbor_tree_t *tree,
                                  const arbor_pool_t *pool, const int32_t *leaves,
                                  int32_t n_leaves, int32_t layer_begin, int32_t layer_end,
                                  const void *q, void *out, int32_t out_dtype, float *lse_out,
                                  float softmax_scale, const arbor_decode_credit_t *credit,
                                  int32_t *status, void *workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/*
 * arbor_walk -- the event-driven controller of Alg. 2 run on the device for a
 * sequence of Transition events (the active leaf switches by expansion or
 * backtracking), with no host round trip between events: the host enqueues
 * every kernel of every step at once and never waits, each step reading its
 * active leaf from targets[step] on the device.  Step e:
 *   1. Transition: arbor_allocate with active = {targets[e]} and the budget
 *      (Path* pinned -- or floored, params->k_protect -- and every other
 *      block lowered only where its new count is smaller, Alg. 2);
 *   2. lazy rehydration of the Path* blocks with evicted tokens from the
 *      token-span record (arbor_rehydrate; skipped when
 *      params->lazy_rehydration = 0);
 *   3. scoring (when q_win is not NULL): the window queries of the new
 *      active leaf, q_win + e * n_slice * Hq * window * head_dim, attend over
 *      its now restored chain and grow A, rows_seen, a and s (arbor_score
 *      with that one observer); the next step's allocation reads this s;
 *   4. arbor_select + arbor_compact of the blocks whose count drops;
 *   5. Pressure, when pressure_margin > 0: if the resident tokens M reach
 *      budget - pressure_margin (RaisePressureEvent of Alg. 2, margin delta),
 *      the allocation is redone for the budget budget - pressure_margin
 *      (off-path blocks lowered in priority order) and steps 4 run again.
 * stats (device int64 [n_steps][4], nullable) receives per step: the resident
 * tokens after the step, the tokens restored from the token store, the tokens
 * evicted, and 1 if a Pressure event fired.  k, delta, on_path (device [V])
 * and sel_pos (device [N]) are the caller's scratch for the step outputs and
 * hold those of the last step.  The results equal n_steps sequences of the
 * single-event entry points issued one by one.  A negative status stops every
 * later step on the device (the status is sticky).
 * Errors: those of the entry points above; EINVAL for n_steps < 0 or missing
 * buffers.
 */
typedef struct {
  const int32_t *targets;      /* device [n_steps]: active leaf of each step          */
  int32_t n_steps;
  int64_t budget_tokens;       /* B                                                   */
  int64_t pressure_margin;     /* delta of Alg. 2; 0: no Pressure events              */
  const void *q_win;           /* device [n_steps][n_slice][Hq][window][head_dim] or NULL */
  int32_t window;
  const int32_t *slice_layers; /* (host) n_slice layer ids (scoring only)             */
  int32_t n_slice;
  const float *v_in, *u_in;    /* device [V] (scoring only)                           */
  float *A;                    /* device [N], in/out                                  */
  int64_t *rows_seen;          /* device [V], in/out (scoring only)                   */
  float *a_out;                /* device [V] (scoring only)                           */
  float *s;                    /* device [V], in/out: the scores the allocations read */
  const void *host_k, *host_v; /* (pinned host) or device token store [N][L][Hkv][d]  */
  int32_t *k, *delta;          /* device [V] scratch / last step's outputs            */
  uint8_t *on_path;            /* device [V]                                          */
  int32_t *sel_pos;            /* device [N]                                          */
  int64_t *stats;              /* device [n_steps][4], nullable                       */
} arbor_walk_t;

int arbor_walk(const arbor_geom_t *geom, arbor_tree_t *tree, arbor_pool_t *pool,
               const arbor_walk_t *walk, const arbor_params_t *params, int32_t *status,
               void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * arbor_uncertainty -- the uncertainty signal of MSVE (Sec. 4, Eq. 1).  Row r of
 * logits ([n_rows][vocab], dtype ARBOR_BF16 or ARBOR_F32, rows contiguous) is
 * the next-token logit vector after closing a block; with p = softmax(row):
 *   top_k = 0 or >= vocab:  H = -sum_w p(w) ln p(w) over the whole vocabulary;
 *   0 < top_k < vocab:      H = -sum_{top} p ln p - p_o ln p_o over the top_k
 *                           largest probabilities and one "other" outcome with
 *                           the remaining mass p_o (omitted when p_o = 0);
 *   u_out[dst[r]] = 1 - H / ln(vocab)    (dst NULL: u_out[r]).
 * u_out is fp32 [n_out]; dst int32 [n_rows] (nullable), each in [0, n_out)
 * (typically the block ids whose u_in arbor_score reads).  The whole-vocabulary
 * form and the top-K form with top_k <= 256 split each row over several
 * workgroups and need `workspace` of at least
 * arbor_uncertainty_workspace_size(n_rows, vocab, dtype) bytes (a larger top_k
 * uses one workgroup per row and no workspace).  fp32 arithmetic with a fixed
 * reduction order: bitwise reproducible.  vocab must be a multiple of 8 (bf16) or 4 (fp32) and logits
 * 16-byte aligned (EUNSUPPORTED otherwise).
 * Errors: EINVAL (arguments, a dst entry out of range), ENONFINITE (a NaN or
 * infinite logit in a row; that row's u is not written), EWORKSPACE.
 */
int arbor_uncertainty(const void *logits, int32_t dtype, int32_t n_rows, int64_t vocab,
                      int32_t top_k, const int32_t *dst, float *u_out, int32_t n_out,
                      int32_t *status, void *workspace, size_t workspace_bytes,
                      hipStream_t stream);

/* Bytes of workspace arbor_uncertainty needs for n_rows rows of `vocab` logits. */
size_t arbor_uncertainty_workspace_size(int32_t n_rows, int64_t vocab, int32_t dtype);


#ifdef __cplusplus
}
#endif
#endif /* ARBOR_H */
