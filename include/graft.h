/*
 * graft.h -- C ABI of the MI355X (gfx950) implementation of GRAFT's per-round
 * draft-tree construction (arXiv 2608.20375).
 *
 * One decoding round of a diffusion-LM drafter (DFlash) gives, for every
 * future depth d = 1..L, a full-vocabulary distribution q_{t,d} (the paper's
 * Preliminaries, "DFlash one-pass marginals").  graft_build_tree turns the
 * drafter logits of a batch of independent sequences into draft trees:
 *
 *   1. log-softmax statistics and the top-K candidate tokens of every depth
 *      (candidates = highest-probability tokens per position, DDTree paragraph);
 *   2. TDES edge scores of every parent -> child candidate pair between
 *      consecutive depths (Sec. "Target-Distilled Edge Scoring", eqs.
 *      tdes-score, tdes-center, tdes-bitower);
 *   3. the SABA budget B_t of every sequence (Sec. "State-Aware Budget
 *      Allocation", eqs. saba-objective, saba-gain, saba-cost);
 *   4. budgeted best-first selection of candidate prefixes ranked by their
 *      path score (DDTree paragraph and eq. ddtree-path-score; TDES
 *      "Inference", eq. tdes-path-score);
 *   5. emission of token ids, parent indices, depth position ids and the
 *      ancestor tree-attention mask (Preliminaries, tree-based speculative
 *      decoding).
 * graft_accept then performs the greedy acceptance walk against the target
 * model's tokens (same paragraph: commit the longest accepted draft path).
 *
 * Conventions
 *   - Every pointer is DEVICE memory unless its comment says (host).
 *   - Calls that take a stream enqueue work on it and return without
 *     synchronizing, except where stated.  All calls of one context must be
 *     ordered (one stream at a time); there is no internal locking.
 *   - The library never keeps a caller pointer past stream-ordered use.
 *   - Return values are graft_status codes.  Host-side validation happens
 *     before anything is enqueued: on an error the outputs are untouched and
 *     graft_last_error() (thread-local) describes it.  Nothing is thrown.
 *
 * Semantics fixed where the paper is silent (the CPU oracle uses the same):
 *   - The root (last committed token) is implicit: it is neither a node nor a
 *     mask row/column, and the budget counts draft nodes only.  A tree holds
 *     N = min(B_t, max_nodes, number of distinct prefixes) nodes.
 *   - Depth-1 edges have the root token as parent; every parent's children
 *     set C_{p,d} is all K candidates of depth d.
 *   - Prefix order (the heap order): higher path score, then smaller depth,
 *     then the lexicographically smaller token-id path from the root.  Path
 *     scores are fp64 sums, root to leaf, of fp32 edge scores.
 *   - Candidates of a depth are ordered by (logit descending, token id
 *     ascending); logits must be finite.
 *   - Nodes are numbered canonically: depth ascending, then token-id path
 *     lexicographically ascending.  parents[i] < i; parents[i] = -1 marks a
 *     child of the root.  pos_ids[i] = base_pos + depth(i).
 *   - mask row i has bit j set iff node j is node i or an ancestor of it;
 *     bit j of row i is bit (j & 63) of word (j >> 6).
 *   - acc_len counts accepted draft nodes and excludes the bonus token.
 */
#ifndef GRAFT_H
#define GRAFT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define GRAFT_API __attribute__((visibility("default")))
#else
#define GRAFT_API
#endif

/* Same type as HIP's hipStream_t; NULL is the default stream. */
typedef struct ihipStream_t *graft_stream_t;

typedef enum {
    GRAFT_OK = 0,
    GRAFT_ERR_INVALID_ARG = 1,   /* NULL where required, bad sizes, unsorted grid ... */
    GRAFT_ERR_UNSUPPORTED = 2,   /* a size beyond the limits below */
    GRAFT_ERR_OUT_OF_MEMORY = 3,
    GRAFT_ERR_HIP = 4,           /* a HIP runtime call or launch failed */
    GRAFT_ERR_DEVICE_DATA = 5    /* graft_get_device_status: kernels saw invalid data */
} graft_status;

typedef struct graft_ctx graft_ctx;

/* Problem sizes fixed for the life of a context. */
typedef struct {
    int32_t max_batch;   /* sequences per call, >= 1 */
    int32_t num_pos;     /* L: drafter block depth, 1..64 */
    int32_t vocab;       /* V: vocabulary size, >= top_k */
    int32_t top_k;       /* K: candidates per depth, 1..64 */
    int32_t max_nodes;   /* N_max: tree capacity, 1..1024 (mask row = ceil(N_max/64) words) */
    int32_t hist_window; /* w: acceptance-history window of the device ring, 1..64 (0 -> 4) */
} graft_dims;

/* TDES scorer, eq. tdes-bitower:
 *   f(p,c,d) = scale * (g_p(e_p) + u_d)^T (g_c(e_c) + u_d) / sqrt(score_dim),
 * g_p(e) = e^T g_parent, g_c(e) = e^T g_child (row-major, fp32);
 * edge score = log q_d(c) + beta * f~ where f~ is f minus its mean over the
 * K children of the same parent when center != 0 (eq. tdes-center), else f.
 * The benchmark stand-in score log q(c) + e_p^T U V^T e_c is
 * {emb, U, V, NULL, E, rank, sqrt(rank), 1, 0}. */
typedef struct {
    const float *emb;        /* [vocab, emb_dim] frozen token embeddings */
    const float *g_parent;   /* [emb_dim, score_dim] */
    const float *g_child;    /* [emb_dim, score_dim] */
    const float *depth_emb;  /* [num_pos, score_dim] u_d, or NULL for u = 0 */
    int32_t emb_dim;         /* E >= 1 */
    int32_t score_dim;       /* m, 1..64 */
    float scale;             /* s */
    float beta;              /* residual strength (the paper's default is 0.2) */
    int32_t center;          /* nonzero: subtract the per-parent mean */
} graft_scorer_desc;

/* SABA, eqs. saba-objective/gain/cost (host memory; copied into the context):
 *   tau = max(phi[0] + phi[1] conf + phi[2] feat + phi[3] hist, tau_min)
 *   U(B) = (1 - exp(-B / tau)) / (c0 + c1 B + c2 B prefix)
 *   B_t = the smallest budget of the grid with the largest U.
 * conf = mean over depths of the top-1 probability; hist = mean accepted
 * length over the window.  feat is the representation-degeneration signal of
 * the decoding state when the round passes the drafter's hidden states,
 *   degen = (1/(L-1)) sum_{d=1..L-1} r_d + (r_{L-1} - r_1),
 *   r_d = cos(h_d, h_{d+1}) (0 if either state is zero; degen = 0 if L = 1),
 * and otherwise the mean per-depth entropy of q, which stands in for it. */
typedef struct {
    const int32_t *budgets;  /* (host) strictly ascending, each in 1..max_nodes */
    int32_t n_budgets;       /* 1..64 */
    float phi[4];
    float tau_min;           /* > 0 */
    float c0, c1, c2;
} graft_saba_desc;

/* Per-round inputs. */
typedef struct {
    int32_t batch;               /* 1..max_batch */
    const uint16_t *logits;      /* [batch, L, V] bf16 bit patterns, contiguous,
                                    16-byte aligned base; finite values */
    const int32_t *root_token;   /* [batch] last committed token, in [0, V) */
    const int32_t *base_pos;     /* [batch] position id of the root */
    const int32_t *prefix_len;   /* [batch] prefix_t of eq. saba-cost, or NULL (0) */
    const float *hist;           /* [batch] hist_t, or NULL: mean of the context's ring */
    const int32_t *fixed_budget; /* [batch] fixed budgets (DDTree-style), or NULL: SABA */
    const uint16_t *hidden;      /* [batch, L, hidden_dim] bf16 bit patterns of the drafter's
                                    hidden state at each draft position, contiguous, 16-byte
                                    aligned base; or NULL (SABA then uses the mean entropy) */
    int32_t hidden_dim;          /* H: a multiple of 8, 8..1048576 (ignored without hidden) */
} graft_round_in;

/* Per-round outputs, caller-allocated.  Required: budget, n_nodes, tokens,
 * parents, pos_ids.  Every other field may be NULL. */
typedef struct {
    int32_t *budget;        /* [batch] B_t */
    int32_t *n_nodes;       /* [batch] N */
    int32_t *tokens;        /* [batch, max_nodes] canonical order, -1 padded */
    int32_t *parents;       /* [batch, max_nodes] -1 for root children and padding */
    int32_t *pos_ids;       /* [batch, max_nodes] -1 padded */
    uint64_t *mask;         /* [batch, max_nodes, ceil(max_nodes/64)] zero padded */
    int32_t *topk_ids;      /* [batch, L, K] candidates, rank order */
    float *topk_logq;       /* [batch, L, K] log q of the candidates */
    float *row_lse;         /* [batch, L] log-sum-exp of each logit row */
    float *row_maxprob;     /* [batch, L] top-1 probability */
    float *row_entropy;     /* [batch, L] entropy of q */
    float *edge_scores;     /* [batch, L, K, K] [depth-1][parent rank][child rank];
                               depth 1 uses parent row 0 only (others 0) */
    double *node_scores;    /* [batch, max_nodes] path score of each node, 0 padded */
    float *saba_state;      /* [batch, 4] conf, feat (degen with hidden states, else the
                               mean entropy), hist, tau (tau = 0 for fixed budgets) */
    float *adj_cos;         /* [batch, L - 1] cosines r_d of adjacent hidden states; written
                               only when the round passes hidden states */
} graft_tree_out;

/* Targets of the acceptance walk: exactly one of target_node / target_depth.
 *   per-node:  target(root) = target_root[b], target(node i) = target_node[b, i]
 *   per-depth: target(node at depth l) = target_depth[b, l], l = 0 (root) .. L */
typedef struct {
    const int32_t *target_root;   /* [batch] (per-node mode) */
    const int32_t *target_node;   /* [batch, max_nodes] or NULL */
    const int32_t *target_depth;  /* [batch, L + 1] or NULL */
} graft_targets;

/* Creates a context and allocates its workspace for `dims` (synchronous). */
GRAFT_API int graft_create(const graft_dims *dims /* host */, graft_ctx **out /* host */);

/* Destroys the context after synchronizing the device; NULL is a no-op. */
GRAFT_API void graft_destroy(graft_ctx *ctx);

/* Installs a TDES scorer: computes the cached projections g_p(e), g_c(e) of
 * every token once (the paper notes they depend only on the token id), on
 * `stream`.  The descriptor's arrays must stay valid until that work is done.
 * Must be called before the first graft_build_tree. */
GRAFT_API int graft_set_scorer(graft_ctx *ctx, const graft_scorer_desc *desc /* host */,
                     graft_stream_t stream);

/* Installs SABA parameters (host only, no device work). */
GRAFT_API int graft_set_saba(graft_ctx *ctx, const graft_saba_desc *desc /* host */);

/* Fills the device acceptance-history ring: init[b, i], i < hist_window,
 * are the accepted lengths of the previous rounds of sequence b. */
GRAFT_API int graft_set_history(graft_ctx *ctx, int32_t batch, const int32_t *init, graft_stream_t stream);

/* Copies the acceptance-history ring of the first `batch` sequences out (a
 * checkpoint of the decoding state that feeds hist_t of the SABA state, Sec.
 * SABA): ring [batch, hist_window] holds the stored accepted lengths in slot
 * order, pos [batch] (or NULL) the slot the next graft_accept with
 * update_history writes.  Both are device memory owned by the caller; the
 * copies are ordered on `stream`.  GRAFT_ERR_INVALID_ARG for a NULL ring, a
 * batch outside 1..max_batch or a context without a history ring. */
GRAFT_API int graft_get_history(graft_ctx *ctx, int32_t batch, int32_t *ring, int32_t *pos,
                                graft_stream_t stream);

/* One round of draft-tree construction for the batch (steps 1-5 above). */
GRAFT_API int graft_build_tree(graft_ctx *ctx, const graft_round_in *in /* host */,
                     const graft_tree_out *out /* host */, graft_stream_t stream);

/* Where steps 2 and 3 run (an execution choice; the results are the same
 * bits either way).  With enable != 0 (the default of a new context) the
 * selection kernel computes a sequence's edge scores and its budget itself
 * whenever the edge rows and the projection rows fit its on-chip memory:
 * num_pos * top_k^2 <= 4096, score_dim 16 or 32, and
 * L K <= 512 and L K (2 score_dim + 10) <= 24576 with L = num_pos, K = top_k; the round
 * then launches no separate edge stage.  With enable == 0
 * the edge stage always runs.  *active (host, may be NULL) receives 1 when
 * the fused path is taken for this context's sizes and installed scorer, else
 * 0.  Host only, no device work; the scorer's score_dim counts, so call it
 * after graft_set_scorer to read *active. */
GRAFT_API int graft_set_fusion(graft_ctx *ctx, int32_t enable, int32_t *active /* host */);

/* Size of the library's static scratch array used by graft_build_tree_static:
 * 24 MiB, the per-round intermediates of a batch of 128 sequences at L = 32
 * and K = 32 (about 18 MB).  Each GPU the library runs on holds one copy until
 * the process ends. */
#define GRAFT_STATIC_SCRATCH_BYTES (24ll * 1024 * 1024)

/* graft_build_tree without any device allocation: for callers that cannot
 * allocate memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, outputs and errors as
 * graft_build_tree, and the same kernels, but the round's intermediates
 * (split-row partials, candidates, row statistics, edge rows, candidate
 * tables in token-id order, positive flags, hidden-state cosines) live in a
 * static device array of GRAFT_STATIC_SCRATCH_BYTES per GPU instead of the
 * context's workspace; the context still provides the scorer's projections,
 * SABA parameters, the history ring and the device status.  The bytes needed grow with the batch:
 * 256-byte aligned parts of B*L*K*(4 + 4 + 4) + B*L*(12 + 1) + B*L*K*K*4 +
 * 4*B*max(L - 1, 1) bytes, plus 8*(3 + K) bytes per split-row partial when
 * rows are split (fewer than about 1024 rows).  A batch whose need exceeds
 * the array returns GRAFT_ERR_UNSUPPORTED before anything is enqueued.  The
 * call allocates nothing (the array's address on each device is resolved
 * once, when a context is created there).  Every call on one GPU shares that
 * GPU's array, which keeps the last call's contents: calls that overlap on one
 * GPU (on different streams, or from different contexts) race; calls ordered
 * on one stream do not.  Nothing in the array needs clearing between calls:
 * each round writes every intermediate before reading it. */
GRAFT_API int graft_build_tree_static(graft_ctx *ctx, const graft_round_in *in /* host */,
                                      const graft_tree_out *out /* host */,
                                      graft_stream_t stream);

/* Greedy acceptance walk over the trees of the batch.
 *   n_nodes [batch], tokens/parents [batch, max_nodes] as written by
 *   graft_build_tree (every node after its parent, as canonical numbering
 *   guarantees; a child listed before its parent is not found, and the walk
 *   stops there); acc_len [batch], acc_nodes [batch, L] (canonical node
 *   indices along the accepted path, -1 padded) and bonus [batch] (the target
 *   token after the last accepted node) are written.  With update_history
 *   nonzero, acc_len is pushed into the context's history ring. */
GRAFT_API int graft_accept(graft_ctx *ctx, int32_t batch, const int32_t *n_nodes, const int32_t *tokens,
                 const int32_t *parents, const graft_targets *targets /* host */,
                 int32_t *acc_len, int32_t *acc_nodes, int32_t *bonus,
                 int32_t update_history, graft_stream_t stream);

/* Verifier-side consumers of a round: the draft tree goes to the target model
 * under a tree-attention mask, and the longest accepted path is committed
 * (the paper's Preliminaries, tree-based speculative decoding). */

/* Expands the ancestor masks written by graft_build_tree into the additive
 * attention bias of the draft block: entry (i, j) of sequence b is 0 when i and
 * j are below n_nodes[b] and node j is node i or an ancestor of it, and -inf
 * otherwise (padding rows and columns included).  Entry (b, i, j), j <
 * max_nodes, is bias[b * batch_stride + i * ld + j]; dtype 0 writes fp32, 1 bf16
 * bit patterns.  bias is 16-byte aligned; ld >= max_nodes and batch_stride >=
 * max_nodes * ld are multiples of 4 (fp32) or 8 (bf16) elements.  Passing a
 * column offset into a wider [batch, max_nodes, prefix + max_nodes] bias, with
 * its full row stride as ld, fills that slice only.
 *   n_nodes [batch]; mask [batch, max_nodes, ceil(max_nodes/64)]. */
GRAFT_API int graft_mask_to_bias(graft_ctx *ctx, int32_t batch, const int32_t *n_nodes,
                                 const uint64_t *mask, void *bias, int32_t dtype, int64_t ld,
                                 int64_t batch_stride, graft_stream_t stream);

/* Commits the accepted path in the verifier's key/value rows: for i <
 * acc_len[b], destination row i of sequence b receives the row_bytes bytes of
 * row acc_nodes[b, i] (acc_len and acc_nodes [batch, L] as written by
 * graft_accept; acc_len is clamped to 0..L); other rows are untouched.
 * Row r of sequence b in plane p (p < n_planes, e.g. layer x {key, value}) is
 * at byte offset p * plane_stride + b * batch_stride + r * row_stride from the
 * source or destination base.  row_bytes, every stride and both bases are
 * multiples of 16.  Within a plane and sequence every source row is read
 * before a destination row that could alias it is written, so dst may be src
 * with the same strides (compaction in place) when the node indices increase
 * along the path and acc_nodes[b, i] >= i, which graft_accept guarantees;
 * other overlaps are not supported.  Node indices outside [0, max_nodes) are
 * skipped and reported by graft_get_device_status. */
GRAFT_API int graft_commit_accepted(graft_ctx *ctx, int32_t batch, const int32_t *acc_len,
                                    const int32_t *acc_nodes, const void *src, void *dst,
                                    int64_t row_bytes, int32_t n_planes,
                                    int64_t src_plane_stride, int64_t src_batch_stride,
                                    int64_t src_row_stride, int64_t dst_plane_stride,
                                    int64_t dst_batch_stride, int64_t dst_row_stride,
                                    graft_stream_t stream);

/* Synchronizes `stream` and reports data errors the kernels detected since
 * the last call (token ids outside [0, V), for example): GRAFT_OK or
 * GRAFT_ERR_DEVICE_DATA; the flag is then cleared. */
GRAFT_API int graft_get_device_status(graft_ctx *ctx, graft_stream_t stream);

/* Synthetic stand-in for the target model, for tests and benchmarks only: the
 * per-node targets of a counter-based draw keyed on each node's identity
 * (sequence, depth, parent token, token) with splitmix64.  With probability
 * 0.8 (24 hash bits under 13421773) the target is the candidate of
 * geometric(1/2) rank (capped at K-1) at the next depth, else, and always at
 * depth L, the identity hash modulo V.  topk_ids [batch, L, K] are the
 * candidates of the round; target_root [batch], target_node [batch, max_nodes]
 * are written (-1 padded). */
GRAFT_API int graft_synth_node_targets(graft_ctx *ctx, int32_t batch, uint64_t seed,
                             const int32_t *root_token, const int32_t *n_nodes,
                             const int32_t *tokens, const int32_t *parents,
                             const int32_t *topk_ids, int32_t *target_root,
                             int32_t *target_node, graft_stream_t stream);

/* Stage timing for benchmarks.  graft_profile_begin arms timing of the next
 * max_calls calls of graft_build_tree and of graft_accept (each counted
 * separately): timing-only HIP events (no system-scope fence) are recorded on
 * the call's stream around every stage, 0 = logits pass, 1 = hidden-state
 * cosines, edge scoring and the SABA budget, 2 = selection, emission and mask,
 * 3 = acceptance (with the fused path of graft_set_fusion, edge scoring and
 * the budget are timed in stage 2).  graft_profile_end synchronizes the events, writes
 * the summed milliseconds stage_ms[4] and the number of timed launches
 * stage_calls[4] (host arrays), and disarms.  Not for concurrent use. */
GRAFT_API int graft_profile_begin(graft_ctx *ctx, int32_t max_calls);
GRAFT_API int graft_profile_end(graft_ctx *ctx, double *stage_ms, int32_t *stage_calls);

/* ------------------------------------------------------------------------ */
/* TDES training (the paper's Target-Distilled Edge Scoring section: the       */
/* objectives KL, pairwise margin and class-balanced BCE, summed by eq.         */
/* tdes-training, and AdamW as in its training setup).                          */
/* ------------------------------------------------------------------------ */

typedef struct graft_tdes graft_tdes;

/* Sizes fixed for the life of a trainer.  Supported: emb_dim E in {32, 64,
 * 128}; score_dim m in 1..64 with E * M <= 4096 and num_pos * M <= 1024, where
 * M = m rounded up to a multiple of 16; top_k 1..64. */
typedef struct {
    int32_t vocab;       /* V, rows of the frozen embedding table */
    int32_t emb_dim;     /* E */
    int32_t score_dim;   /* m */
    int32_t num_pos;     /* L: depths 1..L */
    int32_t top_k;       /* K: children per group */
    int32_t max_groups;  /* >= 0 */
    int32_t max_pairs;   /* >= 0 */
} graft_tdes_dims;

/* One batch of target-model traces (device arrays, int32 / fp32).
 *   Groups g < n_groups (each an accepted parent and its candidate children
 *   C_{p,d}): parent[g], depth[g] in 1..L, child[g, K], logq[g, K] (drafter
 *   log-probabilities of the children), z_target[g, K] (target-model logits of
 *   the children), target[g] (the target's next token under the parent, -1 if
 *   none).  Every child is a verified edge of the BCE objective, labelled 1
 *   where it equals target[g].
 *   Pairs i < n_pairs: pairs[i, 0..5] = (p+, c+, d+, p-, c-, d-), a
 *   target-compatible edge and an incompatible alternative.
 * Token ids outside [0, V) or depths outside 1..L drop their group or pair
 * tile and are reported by graft_tdes_device_status. */
typedef struct {
    int32_t n_groups;
    const int32_t *parent;
    const int32_t *depth;
    const int32_t *child;
    const float *logq;
    const float *z_target;
    const int32_t *target;
    int32_t n_pairs;
    const int32_t *pairs;
} graft_tdes_batch;

/* L = lambda_kl * mean_groups KL(softmax(z) || softmax(logq + f))
 *   + lambda_pair * mean_pairs softplus(gamma - f(v+) + f(v-))
 *   - lambda_bce * mean_edges [w1 y log sigmoid(f) + (1 - y) log(1 - sigmoid(f))]
 * (an empty mean is 0).  The paper trains with lambda = (1, 1, 0.25), AdamW at
 * lr 2e-3 and weight decay 1e-4; beta1 = 0.9, beta2 = 0.999, eps = 1e-8 are
 * the usual AdamW defaults. */
typedef struct {
    float lambda_kl, lambda_pair, lambda_bce;
    float gamma;          /* margin of the pairwise objective */
    float w1;             /* weight of the positive edges in the BCE */
    float lr, weight_decay, beta1, beta2, eps;
} graft_tdes_hyper;

/* Creates a trainer and its workspace (block partial gradients; synchronous). */
GRAFT_API int graft_tdes_create(const graft_tdes_dims *dims /* host */, graft_tdes **out /* host */);
GRAFT_API void graft_tdes_destroy(graft_tdes *t);

/* Number of trainable parameters: 2 E m + L m + 1, laid out as
 *   g_parent [E, m] row-major | g_child [E, m] | depth_emb [L, m] (u_d at row
 *   d - 1) | scale s,
 * the arrays graft_scorer_desc takes (its scale is the last element). */
GRAFT_API int64_t graft_tdes_param_count(const graft_tdes_dims *dims /* host */);

/* One training step on `stream`: the objective and its gradient at theta for
 * the batch, then AdamW (decoupled weight decay on every parameter, bias
 * corrections for step `step` >= 1) updating theta, adam_m and adam_v in place
 * (device [param_count] fp32, theta 16-byte aligned; the moments start at
 * zero).  emb [V, E] fp32, 16-byte aligned, frozen.  loss (device, 4 doubles: L, L_KL, L_pair, L_BCE at
 * theta before the update) and grad (device [param_count] fp32: dL/dtheta) may
 * be NULL.  The step is deterministic: partial gradients are summed in a
 * fixed order. */
GRAFT_API int graft_tdes_step(graft_tdes *t, const float *emb, const graft_tdes_batch *batch /* host */,
                              const graft_tdes_hyper *hyper /* host */, int32_t step, float *theta,
                              float *adam_m, float *adam_v, double *loss, float *grad,
                              graft_stream_t stream);

/* Synchronizes `stream`; GRAFT_OK, or GRAFT_ERR_DEVICE_DATA if a step since the
 * last call dropped a group or pair tile for invalid ids (the flag is then
 * cleared). */
GRAFT_API int graft_tdes_device_status(graft_tdes *t, graft_stream_t stream);

/* ------------------------------------------------------------------------ */
/* SABA parameter fit by same-prefix budget replay (the paper's SABA section:  */
/* the gain and cost models are fitted on held-out replays and then fixed).     */
/* ------------------------------------------------------------------------ */

/* A replay log: round t of the validation set was decoded from one prefix with
 * every budget of the grid, giving its accepted length and round latency.
 * state, prefix, accepted, latency are device arrays; budgets is host. */
typedef struct {
    int32_t n_rounds;         /* T >= 1 */
    int32_t n_budgets;        /* 1..64 */
    const int32_t *budgets;   /* host [n_budgets], positive */
    const float *state;       /* [T, 3]: conf, degen (or the entropy stand-in), hist */
    const int32_t *prefix;    /* [T] prefix length of the round */
    const float *accepted;    /* [T, n_budgets] accepted length a_t(B_j) */
    const float *latency;     /* [T, n_budgets] round latency l_t(B_j), any unit */
    float tau_min;            /* > 0, as in graft_saba_desc */
} graft_saba_replay;

/* Fits the cost c = (c0, c1, c2) of eq. saba-cost by least squares of
 * l_t(B_j) on [1, B_j, B_j prefix_t], and phi of eq. saba-gain by
 * Levenberg-Marquardt from phi_init: phi minimises
 *   sum_{t,j} (A_t G_t(B_j) - a_t(B_j))^2,  G_t(B) = 1 - exp(-B / tau_t),
 *   tau_t = max(phi . [1, s_t], tau_min),
 * with each round's scale A_t eliminated in closed form (it cancels in the
 * budget rule's argmax); rounds that accept nothing contribute nothing.  The
 * sums over the log run on the device (fp64, fixed order: deterministic), the
 * 4 x 4 steps on the host; synchronous on `stream`.  phi_out and c_out (host,
 * 4 and 3 floats) are graft_saba_desc's phi and c0..c2; stats (host, 4 doubles,
 * or NULL): the gain and cost sums of squares, the iterations taken, and 1 if
 * the steps converged (0 if max_iter ran out or the system was singular, e.g.
 * every tau clamped). */
GRAFT_API int graft_saba_fit(const graft_saba_replay *log /* host */, const float *phi_init /* host [4] */,
                             int32_t max_iter, float *phi_out, float *c_out, double *stats,
                             graft_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Bandwidth reference                                                        */
/* ------------------------------------------------------------------------ */

#define GRAFT_READ_STREAM_SINK_WORDS 4096

/* A plain read of `bytes` bytes at src (device, 16-byte aligned, bytes a
 * positive multiple of 16) with the 16-byte non-temporal loads the logits pass
 * uses and no other work: the HBM read rate a streaming kernel reaches, timed
 * beside the logits pass in benchmarks.  sink (device, caller-owned,
 * GRAFT_READ_STREAM_SINK_WORDS uint32) receives per-workgroup xors of the
 * words read; the xor of all its words is the xor of every 32-bit word of the
 * buffer.  Asynchronous on `stream`; GRAFT_ERR_INVALID_ARG for NULL pointers,
 * misalignment or a bad size. */
GRAFT_API int graft_read_stream(const void *src, int64_t bytes, uint32_t *sink, graft_stream_t stream);

GRAFT_API const char *graft_status_string(int status);
GRAFT_API const char *graft_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GRAFT_H */
