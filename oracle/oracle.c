/*
 * oracle.c -- TEST INFRASTRUCTURE, not the product path.
 *
 * A plain, slow, fp64 CPU reference of GRAFT's per-round draft-tree
 * construction (arXiv 2608.20375).  Only the test-suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it.  It shares no code, header,
 * table or helper with the HIP library.
 *
 * Steps, each following the paper's text:
 *   O2  row statistics of each drafter distribution q_{t,d}
 *       (Preliminaries, "DFlash one-pass marginals"; SABA decoding state,
 *       conf_t uses the top-1 probability)
 *   O3  candidate nodes c^{(r)}_{t,d}: the K highest-scoring tokens per depth
 *       (Preliminaries, eq. dflash-top1 and the DDTree paragraph)
 *   O4  TDES edge scores (Sec. "Target-Distilled Edge Scoring",
 *       eqs. tdes-score, tdes-center, tdes-bitower)
 *   O5  SABA budget (Sec. "State-Aware Budget Allocation",
 *       eqs. saba-objective, saba-gain, saba-cost; budget grid), with the
 *       representation-degeneration signal of the decoding state when the
 *       drafter's hidden states are given (same section, degen_t)
 *   O6  best-first selection over a max-heap of candidate prefixes ranked by
 *       the path score (DDTree paragraph, eq. ddtree-path-score; TDES
 *       "Inference", eq. tdes-path-score)
 *   O7  emission: token ids, parent indices, depth position ids and the
 *       ancestor tree-attention mask (Preliminaries, tree-based speculative
 *       decoding)
 *   O8  greedy acceptance: longest accepted root path (same paragraph)
 *   V1  the verifier's additive attention bias of the draft block, expanded
 *       from the ancestor mask (Preliminaries, tree attention)
 *   V2  commit of the accepted path in the verifier's key/value rows: the
 *       rows of the accepted nodes moved to consecutive positions (same
 *       paragraph: the longest accepted path is committed)
 *
 * Readings where the paper is silent (all mirrored by the HIP library):
 *   - the budget counts draft nodes only; the root (last committed token) is
 *     implicit and is neither a node nor a mask row/column;
 *   - the heap order is: higher path score, then smaller depth, then the
 *     lexicographically smaller token-id path from the root;
 *   - nodes are numbered in canonical order (depth ascending, then token-id
 *     path lexicographically ascending);
 *   - depth-1 edges have the root token as parent; the children set of every
 *     parent is all K candidates of the next depth;
 *   - the SABA state is s = [1, conf, degen, hist] when hidden states are
 *     given and s = [1, conf, ent, hist] otherwise (mean per-depth entropy
 *     stands in for degen); tau = max(phi . s, tau_min); ties in the utility
 *     go to the smaller budget;
 *   - degen uses D = L hidden states h_1..h_L (one per drafted position); a
 *     cosine with a zero vector is 0; with L = 1 there is no adjacent pair and
 *     degen = 0;
 *   - acc_len excludes the bonus token.
 *
 * Parity pins: see tests/test_oracle_*.py.  The paper's trained TDES scorer is
 * not available; its stand-in weights are synthetic ("parity unpinned" for the
 * learned parameters themselves, the scoring formula is pinned).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_EXPORT __attribute__((visibility("default")))

/* ------------------------------------------------------------------------- */
/* O1: bf16 -> double (exact)                                                 */
/* ------------------------------------------------------------------------- */
static double bf16_value(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* ------------------------------------------------------------------------- */
/* O2: log-softmax statistics of one row                                      */
/*   m = max x, S = sum e^{x-m}, T = sum e^{x-m}(x-m)                         */
/*   LSE = m + ln S, top-1 probability = e^{m-LSE} = 1/S,                     */
/*   entropy = -sum q ln q = ln S - T/S                                       */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT void oracle_row_stats(const uint16_t *row, int64_t V,
                                    double *lse, double *maxprob, double *entropy)
{
    double m = -INFINITY;
    for (int64_t v = 0; v < V; ++v) {
        double x = bf16_value(row[v]);
        if (x > m) m = x;
    }
    double S = 0.0, T = 0.0;
    for (int64_t v = 0; v < V; ++v) {
        double d = bf16_value(row[v]) - m;
        double e = exp(d);
        S += e;
        T += e * d;
    }
    double lnS = log(S);
    *lse = m + lnS;
    *maxprob = 1.0 / S;
    *entropy = lnS - T / S;
}

/* ------------------------------------------------------------------------- */
/* O3: top-K candidates, ordered by (logit descending, token id ascending).   */
/* log q(c) = x_c - LSE is monotone in x_c within a row, so ranking the raw   */
/* logits ranks the probabilities.                                            */
/* ------------------------------------------------------------------------- */
typedef struct { double x; int32_t id; } oracle_item;

static int item_cmp(const void *pa, const void *pb)
{
    const oracle_item *a = (const oracle_item *)pa, *b = (const oracle_item *)pb;
    if (a->x > b->x) return -1;
    if (a->x < b->x) return 1;
    return (a->id < b->id) ? -1 : (a->id > b->id);
}

ORACLE_EXPORT int oracle_topk(const uint16_t *row, int64_t V, int32_t K,
                              int32_t *ids, double *x_out)
{
    if (K < 0 || K > V) return 1;
    oracle_item *it = (oracle_item *)malloc((size_t)V * sizeof *it);
    if (!it) return 2;
    for (int64_t v = 0; v < V; ++v) { it[v].x = bf16_value(row[v]); it[v].id = (int32_t)v; }
    qsort(it, (size_t)V, sizeof *it, item_cmp);
    for (int32_t r = 0; r < K; ++r) { ids[r] = it[r].id; if (x_out) x_out[r] = it[r].x; }
    free(it);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Parameters shared by the per-sequence entry points.                        */
/* ------------------------------------------------------------------------- */
typedef struct {
    int32_t L, K, n_max;
    int64_t V;
    /* TDES bi-tower f(p,c,d) = s (g_p(e_p)+u_d)^T (g_c(e_c)+u_d) / sqrt(m) */
    const float *emb;        /* [V, E] frozen token embeddings */
    int32_t emb_dim;         /* E */
    const float *g_parent;   /* [E, m]: g_p(e) = e^T G_p */
    const float *g_child;    /* [E, m] */
    const float *depth_emb;  /* [L, m] or NULL (u_d = 0) */
    int32_t score_dim;       /* m */
    double scale;            /* s */
    double beta;             /* residual strength */
    int32_t center;          /* subtract the mean over the children of a parent */
    /* SABA */
    int32_t use_saba;
    const int32_t *grid;     /* candidate budgets, ascending */
    int32_t n_grid;
    double phi[4];           /* tau = phi . [1, conf, degen (or ent), hist] */
    double tau_min, c0, c1, c2;
} oracle_params;

typedef struct {
    const uint16_t *logits;  /* [L, V] bf16 bits */
    int32_t root_token, base_pos, prefix_len, fixed_budget;
    double hist;
    const uint16_t *hidden;  /* [L, H] bf16 bits of the drafter's hidden states, or NULL */
    int32_t hidden_dim;      /* H */
} oracle_seq_in;

typedef struct {
    /* intermediates (all caller-allocated) */
    int32_t *topk_ids;       /* [L, K] */
    double *topk_logq;       /* [L, K] */
    double *row_lse, *row_maxprob, *row_entropy;  /* [L] */
    double *edge;            /* [L, K, K]; depth index 0 uses parent row 0 only */
    double conf, ent, tau;
    int32_t budget;
    double saba_relgap;      /* (U_best - U_second) / U_best, +inf if one budget */
    /* tree */
    int32_t n_nodes;
    int32_t *tokens, *parents, *pos_ids, *depth;  /* [n_max], -1 padded */
    double *node_scores;     /* [n_max], 0 padded */
    uint64_t *mask;          /* [n_max, ceil(n_max/64)] */
    /* audit of the floating-point decisions */
    double boundary_gap;     /* S(last selected) - S(best unselected frontier prefix) */
    double min_pop_gap;      /* min over pops of S(popped) - S(next best in heap) */
    /* representation degeneration (hidden states given) */
    double degen;
    double *adj_cos;         /* [L - 1] r_d, or NULL */
} oracle_seq_out;

/* ------------------------------------------------------------------------- */
/* O4: TDES edge scores of one sequence.                                      */
/*   edge[l][p][c], l = depth-1 in 0..L-1, child = candidate c of depth l+1,  */
/*   parent = root token (l = 0, row p = 0) or candidate p of depth l.        */
/*   S(v) = log q_{l+1}(c) + beta * f~(p,c,l+1)   (eq. tdes-score)            */
/*   f~ = f - mean_{c'} f(p,c',l+1)  when centering (eq. tdes-center)         */
/*   f  = s (g_p(e_p)+u)^T (g_c(e_c)+u) / sqrt(m)   (eq. tdes-bitower)        */
/* The projections depend only on the token, so they are computed once per   */
/* token as the paper notes; everything is fp64 from the fp32 parameters.     */
/* ------------------------------------------------------------------------- */
static void project(const oracle_params *P, const float *G, int32_t tok, double *out)
{
    const int E = P->emb_dim, m = P->score_dim;
    const float *e = P->emb + (int64_t)tok * E;
    for (int j = 0; j < m; ++j) {
        double acc = 0.0;
        for (int i = 0; i < E; ++i) acc += (double)e[i] * (double)G[(int64_t)i * m + j];
        out[j] = acc;
    }
}

ORACLE_EXPORT int oracle_edge_scores(const oracle_params *P, const int32_t *cand,
                                     const double *logq, int32_t root, double *edge,
                                     double *f_out)
{
    const int L = P->L, K = P->K, m = P->score_dim;
    double *gp = (double *)malloc(sizeof(double) * (size_t)m * (size_t)(1 + L * K));
    double *gc = (double *)malloc(sizeof(double) * (size_t)m * (size_t)(L * K));
    double *f = (double *)malloc(sizeof(double) * (size_t)K);
    if (!gp || !gc || !f) { free(gp); free(gc); free(f); return 2; }
    /* parent-side projections: root then every candidate; child-side: every candidate */
    project(P, P->g_parent, root, gp);
    for (int l = 0; l < L; ++l)
        for (int k = 0; k < K; ++k) {
            project(P, P->g_parent, cand[l * K + k], gp + (size_t)m * (1 + l * K + k));
            project(P, P->g_child, cand[l * K + k], gc + (size_t)m * (l * K + k));
        }
    const double inv_sqrt_m = 1.0 / sqrt((double)m);
    for (int l = 0; l < L; ++l) {
        const int n_par = (l == 0) ? 1 : K;
        for (int p = 0; p < K; ++p) {
            double *row = edge + ((size_t)l * K + p) * K;
            if (p >= n_par) {   /* depth 1 has the root as its only parent */
                for (int c = 0; c < K; ++c) {
                    row[c] = 0.0;
                    if (f_out) f_out[((size_t)l * K + p) * K + c] = 0.0;
                }
                continue;
            }
            const double *pv = (l == 0) ? gp : gp + (size_t)m * (1 + (l - 1) * K + p);
            double mean = 0.0;
            for (int c = 0; c < K; ++c) {
                const double *cv = gc + (size_t)m * (l * K + c);
                double dot = 0.0;
                for (int j = 0; j < m; ++j) {
                    double u = P->depth_emb ? (double)P->depth_emb[(size_t)l * m + j] : 0.0;
                    dot += (pv[j] + u) * (cv[j] + u);
                }
                f[c] = P->scale * dot * inv_sqrt_m;
                mean += f[c];
            }
            mean /= (double)K;
            for (int c = 0; c < K; ++c) {
                double ft = P->center ? f[c] - mean : f[c];
                row[c] = logq[l * K + c] + P->beta * ft;
                if (f_out) f_out[((size_t)l * K + p) * K + c] = f[c];
            }
        }
    }
    free(gp); free(gc); free(f);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* O5a: representation degeneration of the SABA decoding state.               */
/*   r_d = cos(h_d, h_{d+1}) for d = 1..D-1 (D = L hidden states, row-major    */
/*   [L, H] bf16), degen = (1/(D-1)) sum_d r_d + (r_{D-1} - r_1).             */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT double oracle_degen(const uint16_t *hidden, int32_t L, int32_t H, double *adj_cos)
{
    if (L < 2) return 0.0;
    double sum = 0.0, first = 0.0, last = 0.0;
    for (int d = 0; d + 1 < L; ++d) {
        const uint16_t *a = hidden + (size_t)d * (size_t)H;
        const uint16_t *b = a + H;
        double ab = 0.0, aa = 0.0, bb = 0.0;
        for (int i = 0; i < H; ++i) {
            double x = bf16_value(a[i]), y = bf16_value(b[i]);
            ab += x * y;
            aa += x * x;
            bb += y * y;
        }
        double r = (aa > 0.0 && bb > 0.0) ? ab / sqrt(aa * bb) : 0.0;
        if (adj_cos) adj_cos[d] = r;
        if (d == 0) first = r;
        last = r;
        sum += r;
    }
    return sum / (double)(L - 1) + (last - first);
}

/* ------------------------------------------------------------------------- */
/* O5: SABA.  B_t = argmax_B U(B),  U = G / C                                 */
/*   G(B) = 1 - exp(-B / tau)        (eq. saba-gain, tau = phi^T s_t)         */
/*   C(B) = c0 + c1 B + c2 B prefix  (eq. saba-cost)                          */
/* The grid is scanned in ascending order; a later budget replaces the        */
/* current best only when its utility is strictly larger.                     */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT int32_t oracle_saba(const oracle_params *P, double conf, double degen,
                                  double hist, int32_t prefix, double *tau_out,
                                  double *relgap_out, double *util_out)
{
    /* s = [1, conf, degen, hist]; callers without hidden states pass ent */
    double tau = P->phi[0] + P->phi[1] * conf + P->phi[2] * degen + P->phi[3] * hist;
    if (tau < P->tau_min) tau = P->tau_min;
    int32_t best = -1;
    double ubest = -INFINITY, usecond = -INFINITY;
    for (int i = 0; i < P->n_grid; ++i) {
        double B = (double)P->grid[i];
        double U = (1.0 - exp(-B / tau)) / (P->c0 + P->c1 * B + P->c2 * B * (double)prefix);
        if (util_out) util_out[i] = U;
        if (best < 0 || U > ubest) {
            if (best >= 0) usecond = ubest;
            ubest = U;
            best = P->grid[i];
        } else if (U > usecond) {
            usecond = U;
        }
    }
    if (tau_out) *tau_out = tau;
    if (relgap_out)
        *relgap_out = (usecond == -INFINITY) ? INFINITY : (ubest - usecond) / fabs(ubest);
    return best;
}

/* ------------------------------------------------------------------------- */
/* O6: best-first selection.                                                  */
/* Every candidate prefix lives in a pool with (score, depth, parent, slot);  */
/* its token path is recovered by walking the parents.  Popping a prefix      */
/* selects it and pushes all K of its children (eager expansion).             */
/* ------------------------------------------------------------------------- */
typedef struct { double score; int32_t depth, parent, slot; } oracle_prefix;

typedef struct {
    const oracle_prefix *pool;
    const int32_t *cand;     /* [L, K] */
    int32_t K;
} path_ctx;

/* token-id path of prefix i from the root, returns its depth */
static int token_path(const path_ctx *c, int32_t i, int32_t *out)
{
    int d = c->pool[i].depth;
    for (int32_t j = i; j >= 0; j = c->pool[j].parent)
        out[c->pool[j].depth - 1] = c->cand[(c->pool[j].depth - 1) * c->K + c->pool[j].slot];
    return d;
}

/* lexicographic comparison of the token paths of two prefixes (<0: a first) */
static int lex_cmp(const path_ctx *c, int32_t a, int32_t b)
{
    int32_t pa[64], pb[64];
    int da = token_path(c, a, pa), db = token_path(c, b, pb);
    int n = da < db ? da : db;
    for (int i = 0; i < n; ++i)
        if (pa[i] != pb[i]) return pa[i] < pb[i] ? -1 : 1;
    return (da > db) - (da < db);
}

/* the heap order: is prefix a ranked before prefix b? */
static int ranks_before(const path_ctx *c, int32_t a, int32_t b)
{
    const oracle_prefix *x = &c->pool[a], *y = &c->pool[b];
    if (x->score != y->score) return x->score > y->score;
    if (x->depth != y->depth) return x->depth < y->depth;
    return lex_cmp(c, a, b) < 0;
}

typedef struct { int32_t *a; int32_t n; } heap_t;

static void heap_push(const path_ctx *c, heap_t *h, int32_t v)
{
    int32_t i = h->n++;
    h->a[i] = v;
    while (i > 0) {
        int32_t p = (i - 1) / 2;
        if (!ranks_before(c, h->a[i], h->a[p])) break;
        int32_t t = h->a[i]; h->a[i] = h->a[p]; h->a[p] = t;
        i = p;
    }
}

static int32_t heap_pop(const path_ctx *c, heap_t *h)
{
    int32_t top = h->a[0];
    h->a[0] = h->a[--h->n];
    int32_t i = 0;
    for (;;) {
        int32_t l = 2 * i + 1, r = l + 1, best = i;
        if (l < h->n && ranks_before(c, h->a[l], h->a[best])) best = l;
        if (r < h->n && ranks_before(c, h->a[r], h->a[best])) best = r;
        if (best == i) break;
        int32_t t = h->a[i]; h->a[i] = h->a[best]; h->a[best] = t;
        i = best;
    }
    return top;
}

static _Thread_local const path_ctx *g_sort_ctx;

/* canonical order: depth ascending, then token path ascending */
static int canon_cmp(const void *pa, const void *pb)
{
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    const oracle_prefix *x = &g_sort_ctx->pool[a], *y = &g_sort_ctx->pool[b];
    if (x->depth != y->depth) return x->depth < y->depth ? -1 : 1;
    return lex_cmp(g_sort_ctx, a, b);
}

/* O6 + O7 from given edge scores (double) and budget. */
static int select_and_emit(const oracle_params *P, const int32_t *cand, const double *edge,
                           int32_t budget, int32_t base_pos, oracle_seq_out *o)
{
    const int L = P->L, K = P->K, n_max = P->n_max;
    const int words = (n_max + 63) / 64;
    int32_t n_target = budget < n_max ? budget : n_max;
    if (n_target < 0) n_target = 0;
    size_t cap = (size_t)K + (size_t)n_target * (size_t)K + 1;
    oracle_prefix *pool = (oracle_prefix *)malloc(cap * sizeof *pool);
    int32_t *heap_a = (int32_t *)malloc(cap * sizeof *heap_a);
    int32_t *sel = (int32_t *)malloc(((size_t)n_target + 1) * sizeof *sel);
    int32_t *canon = (int32_t *)malloc(cap * sizeof *canon);
    if (!pool || !heap_a || !sel || !canon) {
        free(pool); free(heap_a); free(sel); free(canon); return 2;
    }
    path_ctx ctx = { pool, cand, K };
    heap_t h = { heap_a, 0 };
    int32_t n_pool = 0;
    for (int c = 0; c < K; ++c) {
        pool[n_pool] = (oracle_prefix){ edge[c], 1, -1, c };   /* edge[0][0][c] */
        heap_push(&ctx, &h, n_pool++);
    }
    int32_t n_sel = 0;
    double min_pop_gap = INFINITY;
    while (n_sel < n_target && h.n > 0) {
        int32_t u = heap_pop(&ctx, &h);
        if (h.n > 0) {
            double g = pool[u].score - pool[h.a[0]].score;
            if (g < min_pop_gap) min_pop_gap = g;
        }
        sel[n_sel++] = u;
        const oracle_prefix pu = pool[u];
        if (pu.depth < L) {
            /* child at depth pu.depth+1 uses edge table index l = pu.depth,
               parent row = slot of u's last token */
            const double *row = edge + ((size_t)pu.depth * K + pu.slot) * K;
            for (int c = 0; c < K; ++c) {
                /* path score = running sum of edge scores from the root */
                pool[n_pool] = (oracle_prefix){ pu.score + row[c], pu.depth + 1, u, c };
                heap_push(&ctx, &h, n_pool++);
            }
        }
    }
    o->boundary_gap = (h.n > 0 && n_sel > 0) ? pool[sel[n_sel - 1]].score - pool[h.a[0]].score
                                              : INFINITY;
    o->min_pop_gap = min_pop_gap;

    /* O7: canonical numbering, parents, tokens, positions, ancestor mask */
    int32_t *order = (int32_t *)malloc(((size_t)n_sel + 1) * sizeof *order);
    if (!order) { free(pool); free(heap_a); free(sel); free(canon); return 2; }
    memcpy(order, sel, (size_t)n_sel * sizeof *order);
    g_sort_ctx = &ctx;
    qsort(order, (size_t)n_sel, sizeof *order, canon_cmp);
    for (size_t i = 0; i < cap; ++i) canon[i] = -1;
    for (int32_t i = 0; i < n_sel; ++i) canon[order[i]] = i;
    for (int32_t i = 0; i < n_max; ++i) {
        o->tokens[i] = -1; o->parents[i] = -1; o->pos_ids[i] = -1;
        if (o->depth) o->depth[i] = -1;
        if (o->node_scores) o->node_scores[i] = 0.0;
    }
    memset(o->mask, 0, sizeof(uint64_t) * (size_t)n_max * (size_t)words);
    for (int32_t i = 0; i < n_sel; ++i) {
        const oracle_prefix *p = &pool[order[i]];
        o->tokens[i] = cand[(p->depth - 1) * K + p->slot];
        o->parents[i] = (p->parent < 0) ? -1 : canon[p->parent];
        o->pos_ids[i] = base_pos + p->depth;
        if (o->depth) o->depth[i] = p->depth;
        if (o->node_scores) o->node_scores[i] = p->score;
    }
    /* row i holds node i and every ancestor of it (the root excluded) */
    for (int32_t i = 0; i < n_sel; ++i)
        for (int32_t j = i; j >= 0; j = o->parents[j])
            o->mask[(size_t)i * words + (j >> 6)] |= (uint64_t)1 << (j & 63);
    o->n_nodes = n_sel;
    free(order); free(pool); free(heap_a); free(sel); free(canon);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Whole round for one sequence: O2..O7.                                      */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT int oracle_build_sequence(const oracle_params *P, const oracle_seq_in *in,
                                        oracle_seq_out *o)
{
    const int L = P->L, K = P->K;
    double conf = 0.0, ent = 0.0;
    double *x = (double *)malloc(sizeof(double) * (size_t)K);
    if (!x) return 2;
    for (int l = 0; l < L; ++l) {
        const uint16_t *row = in->logits + (size_t)l * (size_t)P->V;
        oracle_row_stats(row, P->V, &o->row_lse[l], &o->row_maxprob[l], &o->row_entropy[l]);
        int rc = oracle_topk(row, P->V, K, o->topk_ids + l * K, x);
        if (rc) { free(x); return rc; }
        for (int k = 0; k < K; ++k) o->topk_logq[l * K + k] = x[k] - o->row_lse[l];
        conf += o->row_maxprob[l];
        ent += o->row_entropy[l];
    }
    free(x);
    conf /= (double)L;
    ent /= (double)L;
    o->conf = conf;
    o->ent = ent;
    /* the state's second feature: degen from the hidden states, else ent */
    double feat = ent;
    o->degen = 0.0;
    if (in->hidden) {
        o->degen = oracle_degen(in->hidden, L, in->hidden_dim, o->adj_cos);
        feat = o->degen;
    }
    int rc = oracle_edge_scores(P, o->topk_ids, o->topk_logq, in->root_token, o->edge, NULL);
    if (rc) return rc;
    if (P->use_saba) {
        o->budget = oracle_saba(P, conf, feat, in->hist, in->prefix_len, &o->tau,
                                &o->saba_relgap, NULL);
    } else {
        o->budget = in->fixed_budget;
        o->tau = 0.0;
        o->saba_relgap = INFINITY;
    }
    return select_and_emit(P, o->topk_ids, o->edge, o->budget, in->base_pos, o);
}

/* Staged entry: O6..O7 on externally supplied fp32 edge scores and budget.   */
ORACLE_EXPORT int oracle_select_staged(const oracle_params *P, const int32_t *cand,
                                       const float *edge32, int32_t budget, int32_t base_pos,
                                       oracle_seq_out *o)
{
    size_t n = (size_t)P->L * P->K * P->K;
    double *edge = (double *)malloc(n * sizeof *edge);
    if (!edge) return 2;
    for (size_t i = 0; i < n; ++i) edge[i] = (double)edge32[i];
    int rc = select_and_emit(P, cand, edge, budget, base_pos, o);
    free(edge);
    return rc;
}

/* ------------------------------------------------------------------------- */
/* O8: greedy acceptance.  From the root, repeatedly move to the child whose  */
/* token equals the target model's token after the current node; stop when   */
/* none matches.  target(root) = target_root (per-node) or target_depth[0];   */
/* target(node i) = target_node[i] or target_depth[depth(i)].                 */
/* Returns acc_len (accepted draft nodes, bonus excluded).                    */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT int32_t oracle_accept(int32_t n_nodes, const int32_t *tokens,
                                    const int32_t *parents, int32_t L,
                                    int32_t target_root, const int32_t *target_node,
                                    const int32_t *target_depth,
                                    int32_t *acc_nodes, int32_t *bonus)
{
    int32_t cur = -1, a = 0, depth = 0;
    for (int i = 0; i < L; ++i) acc_nodes[i] = -1;
    for (;;) {
        int32_t t = target_node ? (cur < 0 ? target_root : target_node[cur])
                                : target_depth[depth];
        int32_t next = -1;
        for (int32_t j = 0; j < n_nodes; ++j)
            if (parents[j] == cur && tokens[j] == t) { next = j; break; }
        if (next < 0) { *bonus = t; break; }
        acc_nodes[a++] = next;
        cur = next;
        ++depth;
    }
    return a;
}

/* ------------------------------------------------------------------------- */
/* V1: additive attention bias of the draft block.  Node i may attend to node */
/* j iff j is i or an ancestor of i (bit j of mask row i): bias 0, else -inf. */
/* Entries of padding rows or columns (i or j >= n) are -inf.  bias is        */
/* [n_max, n_max] doubles, row-major.                                          */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT void oracle_mask_to_bias(int32_t n, int32_t n_max, const uint64_t *mask,
                                       int32_t words, double *bias)
{
    for (int32_t i = 0; i < n_max; ++i)
        for (int32_t j = 0; j < n_max; ++j) {
            int visible = 0;
            if (i < n && j < n)
                visible = (int)((mask[(size_t)i * (size_t)words + (size_t)(j / 64)] >> (j % 64)) & 1u);
            bias[(size_t)i * (size_t)n_max + (size_t)j] = visible ? 0.0 : -INFINITY;
        }
}

/* ------------------------------------------------------------------------- */
/* V2: the accepted path's rows.  Destination row i (i < acc_len) receives    */
/* the row_bytes bytes of source row acc_nodes[i]; other rows are untouched.  */
/* Rows are read before any is written, so src and dst may be the same       */
/* buffer with the same stride (the accepted nodes then move down in place).  */
/* ------------------------------------------------------------------------- */
ORACLE_EXPORT int oracle_gather_rows(int32_t acc_len, const int32_t *acc_nodes,
                                     const uint8_t *src, int64_t src_row_stride, uint8_t *dst,
                                     int64_t dst_row_stride, int64_t row_bytes)
{
    if (acc_len <= 0) return 0;
    uint8_t *tmp = (uint8_t *)malloc((size_t)acc_len * (size_t)row_bytes);
    if (!tmp) return 1;
    for (int32_t i = 0; i < acc_len; ++i)
        memcpy(tmp + (size_t)i * (size_t)row_bytes,
               src + (size_t)acc_nodes[i] * (size_t)src_row_stride, (size_t)row_bytes);
    for (int32_t i = 0; i < acc_len; ++i)
        memcpy(dst + (size_t)i * (size_t)dst_row_stride, tmp + (size_t)i * (size_t)row_bytes,
               (size_t)row_bytes);
    free(tmp);
    return 0;
}
