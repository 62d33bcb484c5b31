/*
 * dominotree.h -- C ABI of the MI355X (gfx950) DominoTree draft-tree builder.
 *
 * The library builds the conditional best-first draft tree of DominoTree
 * (arXiv 2607.08642, section 3, Algorithm 1) on one GPU:
 *
 *   S1  per depth, the top-M marginal candidates and the tail log-sum-exp
 *       (Alg. 1 step 1; section 3.2, candidate restriction);
 *   S2  the rows of the GRU input projection and of the correction head that
 *       the candidates need (section 3.2: gather the M rows once per depth);
 *       they depend on the model only, so the plan folds them for the whole
 *       vocabulary once and each call gathers them;
 *   S3  the root's children (Alg. 1 steps 2-3);
 *   S4  best-first expansion: pop, advance the GRU along the node's own path,
 *       score the next depth's slice with the path-dependent correction, push
 *       the top-k children (Alg. 1 step 4; Domino's correction, section 2.3);
 *   S5  emission of the tree in pop order with parent pointers, depths,
 *       position ids and the ancestor-only verification mask (section 3.5).
 *
 * Scoring of a node at depth d whose parent path has GRU state S (Fact B):
 *   delta_m = E[cand_d[m]] . (W_c S + b_c)          (correction head)
 *   z_m     = (x_d[m] + delta_m) / tau,  tau = T if T > 0 else 1
 *   logZ    = LSE_m(z_m) (SLICE)  or  LSE(LSE_m(z_m), R_d) (TAIL, default)
 *   ell_m   = z_m - logZ,  R_d = log sum_{v not in slice} exp(x_d[v] / tau)
 * The GRU follows PyTorch's GRUCell (gates r, z, n; W_ih = [W_ir; W_iz; W_in]).
 *
 * Ties: top-M by (logit desc, token id asc); children by (log-prob desc,
 * slot asc); pops by (score desc, insertion order asc).
 *
 * Conventions for every call:
 *   - all tensor arguments are DEVICE pointers (hipMalloc / torch CUDA tensors),
 *     row-major and contiguous, owned by the caller; the library never frees
 *     caller memory;
 *   - `stream` is a hipStream_t (NULL = the default stream); every call is
 *     stream-ordered and asynchronous: no host synchronisation happens inside
 *     dt_build_tree / dt_scan_topm, results are valid once the stream completes;
 *   - argument errors are detected on the host before any launch: a negative
 *     dt_status is returned and nothing is written; dt_last_error() gives a
 *     thread-local message;
 *   - data errors are per-tree status bits written on the device
 *     (DT_TREE_NONFINITE: a NaN or +inf logit; that tree gets n_nodes = 0);
 *   - no C++ exception crosses this interface.
 *
 * Envelope: 1 <= M <= min(V, 256); 1 <= B <= 256; 1 <= L <= 64;
 * 32 <= d_h <= 1024 with d_h % 32 == 0; 1 <= d_e <= 8192; 1 <= V < 2^31;
 * the per-row merge buffer, about 22 * ceil(V / 10240) * M + 20 * M bytes,
 * must fit 96 KiB (DT_ERR_UNSUPPORTED otherwise); the expansion kernel's LDS
 * layout must fit the device at some number of workgroups per tree (the plan
 * takes the largest that fits; on a 160 KiB device only d_h 864, 928 and 992
 * with M >= 128 fit at none).  Both are checked by dt_plan_create, the first
 * also by dt_scan_topm.
 */
#ifndef DOMINOTREE_H
#define DOMINOTREE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DT_ABI_VERSION 3

typedef enum { DT_F32 = 0, DT_BF16 = 1 } dt_dtype;

typedef enum {
  DT_OK = 0,
  DT_ERR_NULL = -1,        /* a required pointer is NULL */
  DT_ERR_SHAPE = -2,       /* a size is out of range or inconsistent */
  DT_ERR_DTYPE = -3,       /* unknown dtype code */
  DT_ERR_UNSUPPORTED = -4, /* outside the envelope above */
  DT_ERR_WORKSPACE = -5,   /* workspace missing or smaller than dt_workspace_size */
  DT_ERR_ALIGN = -6,       /* a pointer is not aligned as required */
  DT_ERR_HIP = -7          /* a HIP runtime call failed (see dt_last_error) */
} dt_status;

/* per-tree status bits, written to dt_tree.status[b] */
#define DT_TREE_NONFINITE 0x1 /* a NaN or +inf logit: the tree has no nodes */
#define DT_TREE_TRUNCATED 0x2 /* a capacity limit of the expansion was reached; only
                                 hundreds of exactly tied scores can cause it.  The tree
                                 is still a valid best-first tree but exact ties may be
                                 resolved differently from insertion order. */
#define DT_TREE_TIMEOUT 0x4   /* a cross-workgroup wait gave up after its spin limit
                                 (dt_options.debug_spin_limit): the tree is emitted
                                 with no nodes, like a non-finite one */

/* normalisation of the corrected slice (dt_options.norm_mode) */
#define DT_NORM_TAIL 0  /* logZ includes the uncorrected out-of-slice mass R_d */
#define DT_NORM_SLICE 1 /* logZ over the top-M slice only */

/* children function (dt_options.scorer); the three arms of the paper's
 * ablation (Appendix D) */
#define DT_SCORER_COND 0   /* DominoTree: the correction recomputed from each node's own
                              path state (Alg. 1, section 3.1) */
#define DT_SCORER_MARG 1   /* Marg: a depth's slice scored from the marginal logits alone
                              (no correction; the menu is shared by the depth's nodes) */
#define DT_SCORER_STATIC 2 /* Cond-static: the correction computed once per depth from
                              the state of Domino's greedy chain (the best corrected child
                              at every depth), its menu shared by the depth's nodes */

/* GRU of Domino's causal encoder (section 2.3), PyTorch GRUCell layout.
 * w_ih: [3*d_h, d_in] with d_in = the embedding width d_e; w_hh: [3*d_h, d_h];
 * b_ih, b_hh: [3*d_h] or NULL (treated as zeros).  dtype = the plan's
 * weights dtype. */
typedef struct {
  const void *w_ih, *w_hh, *b_ih, *b_hh;
  int d_in, d_h;
} dt_gru;

/* Correction head: q = w S + b with w: [d_e, d_h] (a Linear(d_h -> d_e)
 * weight), b: [d_e] or NULL.  delta(v) = E[v] . q. */
typedef struct {
  const void *w, *b;
} dt_head;

typedef struct {
  int max_children; /* k, children kept per expansion; 0 -> min(M, B).
                       The paper's headline setting is 8 (section 4.1). */
  int norm_mode;    /* DT_NORM_TAIL (default) or DT_NORM_SLICE */
  int pos_offset;   /* position_ids = pos_offset + depth */
  int scorer;       /* DT_SCORER_COND (default, 0), DT_SCORER_MARG or DT_SCORER_STATIC */
  int frontier_width;   /* 0 (default): the best-first heap of Alg. 1.  W >= 1: the
                           frontier builder of Appendix B (the serving builder of
                           section 4.5.1): depth by depth, only the W best nodes of
                           the depth (score desc, then the order in which they were
                           scored) are expanded, every scored child is a candidate,
                           and the tree is the B best candidates by (score desc,
                           depth asc, scoring order), emitted in that order.  W >= B
                           gives the heap's tree (exact score ties aside); W < B an
                           approximation of it.  Not with dt_build_tree_head or the
                           adaptive budget. */
  int debug_spin_limit; /* polls before a wait of the workgroups that build a tree
                           together gives up (0: the default, about 2^18 polls,
                           ~0.3 s); a tree whose wait gave up carries DT_TREE_TIMEOUT
                           and no nodes.  A small value exercises that path. */
} dt_options;

/* Output tree of every batch entry b (device pointers, caller-owned).
 * Nodes are in pop order, so a parent always precedes its children. */
typedef struct {
  int32_t *tokens;       /* [batch, B] token id; -1 in padding rows */
  int32_t *parents;      /* [batch, B] pop index of the parent; -1 = child of the root */
  int32_t *depth;        /* [batch, B] 1..L; 0 in padding rows */
  int32_t *position_ids; /* [batch, B] pos_offset + depth */
  uint8_t *mask;         /* [batch, B, B] mask[i][j] = 1 iff j is i or an ancestor of i */
  float *scores;         /* [batch, B] cumulative log-prob g; -inf in padding rows */
  int32_t *n_nodes;      /* [batch] nodes emitted (<= B) */
  int32_t *status;       /* [batch] DT_TREE_* bits */
} dt_tree;

typedef struct dt_plan dt_plan;

/* ABI version of the loaded library (DT_ABI_VERSION when it matches this header). */
int dt_abi_version(void);

/* Static text for a dt_status code. */
const char *dt_status_string(int status);

/* Thread-local detail of the last error returned on this host thread. */
const char *dt_last_error(void);

/* A drafter's model-level tables, shared by every plan made from it: the
 * embedding table folded through the GRU input projection and the correction
 * head for every token (W_ih E[v] + b_ih, W_c^T E[v], E[v] . b_c; section 2.3's
 * encoder input and head, precomputed per token as the candidate gather of
 * section 3.2 reads them), held in fp32, V * (4 d_h + 1) * 4 bytes of device
 * memory (1.24 GB for Qwen3's vocabulary at d_h = 512), and the repacked GRU.
 *   emb:  [V, d_e] token-embedding table (caller-owned; only read while the
 *         model is created);
 *   gru, head: the Domino encoder and correction head (copied and repacked
 *         into library-owned device memory; the caller may free them afterwards);
 *   weights_dtype: dtype of emb, GRU and head tensors.
 * The tables live on the device current at creation.  Runs packing kernels on
 * the default stream and waits for them.  On success *model is set; on
 * failure *model is NULL. */
typedef struct dt_model dt_model;
dt_status dt_model_create(dt_model **model, const void *emb, int V, int d_e, const dt_gru *gru,
                          const dt_head *head, int weights_dtype);

/* Release the caller's reference to the model (NULL is ignored).  Each plan
 * made from it holds a reference of its own: the tables are freed when the
 * model and all of its plans are destroyed, in any order. */
void dt_model_destroy(dt_model *model);

/* Create a plan for one (L, M, B) shape of a model: nothing is folded or
 * copied (a few small buffers are allocated later, for profiling and the
 * adaptive budget).  Plans of one model with different shapes, options or
 * batch limits share its tables.  The model's device must be current
 * (DT_ERR_SHAPE otherwise).
 *   logits_dtype: dtype of the marginal logits passed to dt_build_tree;
 *   max_batch: the largest batch dt_build_tree will be called with;
 *   opts: NULL for defaults.
 * On success *plan is set; on failure *plan is NULL. */
dt_status dt_plan_create_from_model(dt_plan **plan, dt_model *model, int L, int M, int B,
                                    int logits_dtype, int max_batch, const dt_options *opts);

/* Create a plan together with a model of its own (dt_model_create followed by
 * dt_plan_create_from_model; the plan holds the model's only reference, so
 * dt_plan_destroy frees its tables).  Arguments as for those two calls. */
dt_status dt_plan_create(dt_plan **plan, const void *emb, int V, int d_e, const dt_gru *gru,
                         const dt_head *head, int weights_dtype, int L, int M, int B,
                         int logits_dtype, int max_batch, const dt_options *opts);

/* Device workspace (bytes) dt_build_tree needs for `batch` trees. */
dt_status dt_workspace_size(const dt_plan *plan, int batch, size_t *bytes);

/* Build `batch` draft trees (Alg. 1) from marginal logits [batch, L, V].
 *   h0: [batch, d_h] fp32 root GRU states, or NULL for zeros;
 *   T:  temperature (T <= 0 scores with tau = 1);
 *   workspace: >= dt_workspace_size bytes, 256-byte aligned, caller-owned;
 *   out: output arrays as documented in dt_tree.
 * Launches on `stream` and returns without waiting; the call may be captured
 * into a HIP graph (it records no memset or copy nodes, only its two kernels,
 * whose arguments are fixed at capture).  For small batches several
 * workgroups (at most one per CU in total) build each tree together and wait
 * on one another; they rely on being resident at the same time, which holds on
 * a device that other work does not fill.  Each wait is bounded: a tree whose
 * workgroups could not meet carries DT_TREE_TIMEOUT.  A workspace must not be
 * shared by calls that can overlap. */
dt_status dt_build_tree(dt_plan *plan, const void *marginal_logits, int batch, const float *h0,
                        float T, void *workspace, size_t ws_bytes, dt_tree *out, void *stream);

/* For callers that cannot allocate (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): dt_build_tree without a workspace
 * argument.  The workspace is a 32 MiB array of library-owned device memory per
 * device (held until the process ends; enough for 32 trees per call at the
 * Qwen3-8B shape, L = 16, M = 64, B = 16, d_h = 512).  The call itself allocates
 * nothing; the array's address is resolved when a plan is created on the device.
 *   arguments: as dt_build_tree (the plan's device must be current);
 *   DT_ERR_WORKSPACE when dt_workspace_size(plan, batch) exceeds 32 MiB
 *   (use dt_build_tree with a workspace then), DT_ERR_SHAPE when the current
 *   device is not the plan's.
 * Every call on a device shares that device's array, which keeps the last
 * call's contents (the kernels clear what they need zeroed): calls that can
 * overlap on one device -- on different streams, or from several host threads
 * -- race and must not be made. */
dt_status dt_build_tree_noalloc(dt_plan *plan, const void *marginal_logits, int batch,
                                const float *h0, float T, dt_tree *out, void *stream);

/* Release the plan's device memory and its reference to the model (NULL is
 * ignored). */
void dt_plan_destroy(dt_plan *plan);

/* Stage timing (measurement aid).  With every = n > 0, every n-th dt_build_tree
 * call (the first one included) launches its two kernels with HIP events taken
 * at each kernel's start and end (hipExtLaunchKernel), so a stage is one
 * kernel's execution time: stage 0 = top-M scan of the logits (kernel 1),
 * 1 = per-row merge, expansion and emission (kernel 2).  every = 0
 * turns it off; enabling (again) starts a new count.  Calls made while the
 * stream is being captured into a HIP graph record no events and do not count.
 * dt_plan_stage_ms waits for the last profiled call and writes the mean stage
 * durations in milliseconds over the profiled calls (the most recent 1024) to
 * ms[0..1].  Returns DT_ERR_SHAPE if no profiled call has been made yet. */
dt_status dt_plan_set_profiling(dt_plan *plan, int every);
dt_status dt_plan_stage_ms(dt_plan *plan, float *ms);

/* The adaptive budget: CaDDTree's cost-aware stopping rule (section 2.5)
 * inlined into the conditional pop loop (section 3.4).  With it set, a tree
 * keeps popping best-first while
 *   theta(n) = (1 + Phi(n)) / (C_d + C_v(n)),  Phi(n) = sum_{s <= n} exp(g_s)
 * improves on theta(n - 1), g_s the cumulative log-prob of pop s; the first
 * pop that does not improve theta (theta(n) <= theta(n - 1)) is not kept, and
 * the plan's B is the cap.  The tree is the first n* pops of the fixed-budget
 * tree (n_nodes = n*, possibly 0; rows past it are padding).  For a convex C_v
 * theta is unimodal and n* is its argmax; otherwise n* is its first local
 * maximum.  The paper gives no cost model: the caller passes it.
 *   c_draft: C_d (the draft cost of a round, any unit);
 *   c_verify: host array of n = B + 1 floats, C_v(0), ..., C_v(B) (same unit);
 *   C_d + C_v(i) must be positive and finite (DT_ERR_SHAPE otherwise);
 *   c_verify = NULL turns the rule off (fixed budget B, the default).
 * Applies to dt_build_tree, dt_build_tree_noalloc and dt_build_tree_head calls
 * launched after it (waits for the copy; not a stream operation, so set it
 * before capturing calls into a graph: a captured call keeps the setting it
 * was captured with, reading the cost values current at replay). */
dt_status dt_plan_set_adaptive_budget(dt_plan *plan, float c_draft, const float *c_verify, int n);

/* Expansion statistics of the last profiled dt_build_tree call (measurement
 * aid; profiling on, see dt_plan_set_profiling): per tree, the dependent
 * expansion steps the kernel ran (the root's included; each step expands up to
 * 16 nodes of one depth) and the nodes it expanded (the root included, and the
 * speculative expansions of nodes that were not popped).  Writes n <= the last
 * profiled call's batch entries to the host arrays steps[] and expanded[];
 * waits for that call.  DT_ERR_SHAPE if no call was profiled since profiling
 * was enabled. */
dt_status dt_plan_expand_stats(dt_plan *plan, int32_t *steps, int32_t *expanded, int n);

/* Workspace (bytes) for dt_scan_topm over `rows` rows. */
dt_status dt_scan_workspace_size(int rows, int V, int M, size_t *bytes);

/* S1 alone: per row of logits [rows, V], the top-M ids (ordered by logit desc,
 * id asc), their logits widened to fp32, and the tail log-sum-exp
 * R = log sum_{v not in top-M} exp(x[v] / tau) (-inf when empty).
 *   ids: [rows, M] int32; vals: [rows, M] float; tail_lse: [rows] float;
 *   row_flags: [rows] int32 (DT_TREE_NONFINITE when the row holds NaN / +inf;
 *   the other outputs of such a row are unspecified).
 * Alg. 1 step 1; section 3.2. */
dt_status dt_scan_topm(const void *logits, int rows, int V, int logits_dtype, int M, float T,
                       int32_t *ids, float *vals, float *tail_lse, int32_t *row_flags,
                       void *workspace, size_t ws_bytes, void *stream);

/* Domino's own correction head (section 2.3): a rank-r bottleneck with SiLU
 * over the drafter's hidden state at the position and the path state,
 *   delta_m = W_2[cand_d[m]] . SiLU(W_1 [H_d; S])      (no biases)
 * which replaces the linear head's E[v] . (W_c S + b_c) in the scoring above.
 *   w1: [rank, d_H + d_h] (a Linear(d_H + d_h -> rank) weight; columns
 *       [0, d_H) act on H_d, the rest on S);
 *   w2: [V, rank] (a Linear(rank -> V) weight; row v is gathered for token v);
 * both device pointers in the plan's weights dtype, 16-byte aligned,
 * caller-owned and read by every dt_build_tree_head call.
 * 8 <= d_H <= 8192 and 8 <= rank <= 1024, both multiples of 8. */
typedef struct {
  const void *w1, *w2;
  int d_H, rank;
} dt_domino_head;

/* Workspace (bytes) dt_build_tree_head needs for `batch` trees with this head. */
dt_status dt_head_workspace_size(const dt_plan *plan, int batch, const dt_domino_head *head,
                                 size_t *bytes);

/* Build `batch` draft trees (Alg. 1) scored with Domino's own head.
 *   H: [batch, L, d_H] drafter hidden states (the plan's weights dtype,
 *      16-byte aligned); row d scores the children at depth d + 1, the same
 *      depth as logits row d;
 *   the other arguments are those of dt_build_tree; the plan's linear head
 *   (dt_head) is not used, its GRU is.
 * The plan must be created with DT_SCORER_COND and frontier_width 0.  Two
 * tree kernels exist; the call takes the first whose envelope holds:
 *  - dt_build_tree's expansion kernel with this head as the correction: the
 *    same G workgroups per tree as dt_build_tree (G = 16 at d_h = 512 and
 *    batch <= 16, 8 at batch 32), each owning rank / G ranks of the
 *    bottleneck; needs rank a multiple of 16 G with rank / G in {16, 32, 64},
 *    V * rank * (weight bytes) < 2^31 and its LDS to fit the device.  The
 *    envelope of dt_build_tree holds otherwise (any M, B the plan allows).
 *  - one workgroup per tree popping the heap one node at a time: M <= 64,
 *    the scan's segments per row <= 16 (true for V <= 163840 at any batch),
 *    k * (B + 1) <= 4096, and its LDS must fit the device.
 * DT_ERR_UNSUPPORTED when neither holds.  dt_head_workspace_size gives the
 * workspace of the kernel the call will take.  Stream-ordered and capturable
 * like dt_build_tree (three kernels, no memset or copy).  Stage timing
 * (dt_plan_set_profiling) counts these calls too: stage 0 = the scan,
 * stage 1 = the tree kernel (the projection between them is not timed);
 * dt_plan_expand_stats reports the expansion kernel's steps when it ran. */
dt_status dt_build_tree_head(dt_plan *plan, const void *marginal_logits, int batch, const void *H,
                             const dt_domino_head *head, const float *h0, float T,
                             void *workspace, size_t ws_bytes, dt_tree *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DOMINOTREE_H */
