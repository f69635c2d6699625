/* Drives every entry point of the CPU oracle on small seeded inputs and edge
 * cases, built together with oracle/oracle.c under AddressSanitizer and
 * UndefinedBehaviorSanitizer by tests/test_oracle_sanitize.py (host code only).
 * It checks memory safety and defined behaviour, not values: the values are
 * pinned by the Python tests.  Exit status 0 = every call returned normally. */
#include "../oracle/oracle.c"

#include <stdio.h>

static uint64_t g_state = 0x243F6A8885A308D3ull;

static uint64_t next_u64(void)
{
    /* splitmix64 (Steele, Lea, Flood 2014) as a plain stream of test inputs */
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static double uniform(void) { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }

static uint16_t bf16_bits(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static void *must(void *p)
{
    if (!p) {
        fprintf(stderr, "allocation failed\n");
        exit(3);
    }
    return p;
}

#define ALLOC(T, n) ((T *)must(calloc((size_t)(n) > 0 ? (size_t)(n) : 1, sizeof(T))))

typedef struct {
    int32_t *topk_ids, *tokens, *parents, *pos_ids, *depth;
    double *topk_logq, *row_lse, *row_maxprob, *row_entropy, *edge, *node_scores, *adj_cos;
    uint64_t *mask;
} bufs;

static void out_alloc(bufs *b, oracle_seq_out *o, int L, int K, int n_max)
{
    const int words = (n_max + 63) / 64;
    b->topk_ids = ALLOC(int32_t, L * K);
    b->topk_logq = ALLOC(double, L * K);
    b->row_lse = ALLOC(double, L);
    b->row_maxprob = ALLOC(double, L);
    b->row_entropy = ALLOC(double, L);
    b->edge = ALLOC(double, L * K * K);
    b->tokens = ALLOC(int32_t, n_max);
    b->parents = ALLOC(int32_t, n_max);
    b->pos_ids = ALLOC(int32_t, n_max);
    b->depth = ALLOC(int32_t, n_max);
    b->node_scores = ALLOC(double, n_max);
    b->mask = ALLOC(uint64_t, n_max * words);
    b->adj_cos = ALLOC(double, L > 1 ? L - 1 : 1);
    memset(o, 0, sizeof *o);
    o->topk_ids = b->topk_ids;
    o->topk_logq = b->topk_logq;
    o->row_lse = b->row_lse;
    o->row_maxprob = b->row_maxprob;
    o->row_entropy = b->row_entropy;
    o->edge = b->edge;
    o->tokens = b->tokens;
    o->parents = b->parents;
    o->pos_ids = b->pos_ids;
    o->depth = b->depth;
    o->node_scores = b->node_scores;
    o->mask = b->mask;
    o->adj_cos = b->adj_cos;
}

static void out_free(bufs *b)
{
    free(b->topk_ids); free(b->topk_logq); free(b->row_lse); free(b->row_maxprob);
    free(b->row_entropy); free(b->edge); free(b->tokens); free(b->parents); free(b->pos_ids);
    free(b->depth); free(b->node_scores); free(b->mask); free(b->adj_cos);
}

/* One case: L depths, K candidates, vocabulary V, N_max nodes, embedding
 * width E, score width m; quantised logits when ties (many exact ties). */
static int run_case(int L, int K, int64_t V, int n_max, int E, int m, int saba, int center,
                    int depth_emb, int hidden, int ties, int budget, double beta)
{
    float *emb = ALLOC(float, V * E), *gp = ALLOC(float, E * m), *gc = ALLOC(float, E * m);
    float *u = ALLOC(float, L * m);
    for (int64_t i = 0; i < V * E; ++i) emb[i] = (float)(uniform() - 0.5);
    for (int i = 0; i < E * m; ++i) {
        gp[i] = (float)(uniform() - 0.5);
        gc[i] = (float)(uniform() - 0.5);
    }
    for (int i = 0; i < L * m; ++i) u[i] = (float)(0.1 * (uniform() - 0.5));
    int32_t grid[5] = {1, 2, 4, 8, n_max};
    oracle_params P;
    memset(&P, 0, sizeof P);
    P.L = L; P.K = K; P.n_max = n_max; P.V = V;
    P.emb = emb; P.emb_dim = E; P.g_parent = gp; P.g_child = gc;
    P.depth_emb = depth_emb ? u : NULL; P.score_dim = m;
    P.scale = 1.5; P.beta = beta; P.center = center;
    P.use_saba = saba; P.grid = grid; P.n_grid = 5;
    P.phi[0] = 2.0; P.phi[1] = 3.0; P.phi[2] = 0.5; P.phi[3] = 0.25;
    P.tau_min = 1.0; P.c0 = 1.0; P.c1 = 0.05; P.c2 = 1e-4;

    uint16_t *logits = ALLOC(uint16_t, L * V);
    for (int64_t i = 0; i < L * V; ++i) {
        double x = 4.0 * (uniform() - 0.5);
        if (ties) x = (double)(int)(x * 2.0) * 0.5;
        logits[i] = bf16_bits((float)x);
    }
    const int H = 24;
    uint16_t *hid = ALLOC(uint16_t, L * H);
    for (int i = 0; i < L * H; ++i) hid[i] = bf16_bits(i % 7 == 0 ? 0.0f : (float)(uniform() - 0.5));
    if (hidden && L > 1)
        for (int i = 0; i < H; ++i) hid[i] = 0;   /* a zero state: cosine 0 */

    oracle_seq_in in = {logits, (int32_t)(V / 2), 100, 50, budget, 3.0, hidden ? hid : NULL, H};
    bufs b;
    oracle_seq_out o;
    out_alloc(&b, &o, L, K, n_max);
    int rc = oracle_build_sequence(&P, &in, &o);
    if (rc) return rc;
    if (o.n_nodes < 0 || o.n_nodes > n_max) return 10;

    /* staged selection on fp32 copies of the edges, also with positive scores */
    float *e32 = ALLOC(float, L * K * K);
    for (int i = 0; i < L * K * K; ++i) e32[i] = (float)b.edge[i];
    bufs b2;
    oracle_seq_out o2;
    out_alloc(&b2, &o2, L, K, n_max);
    rc = oracle_select_staged(&P, b.topk_ids, e32, o.budget, 7, &o2);
    if (rc) return rc;
    for (int i = 0; i < L * K * K; ++i) e32[i] = (float)(uniform() - 0.3);
    rc = oracle_select_staged(&P, b.topk_ids, e32, n_max, 7, &o2);
    if (rc) return rc;

    /* acceptance: per-depth and per-node targets */
    int32_t *acc = ALLOC(int32_t, L), bonus = 0;
    int32_t *td = ALLOC(int32_t, L + 1), *tn = ALLOC(int32_t, n_max);
    for (int i = 0; i <= L; ++i) td[i] = b.topk_ids[(i < L ? i : L - 1) * K];
    for (int i = 0; i < n_max; ++i) tn[i] = i < o.n_nodes ? b.topk_ids[0] : -1;
    int32_t a = oracle_accept(o.n_nodes, b.tokens, b.parents, L, -1, NULL, td, acc, &bonus);
    if (a < 0 || a > L) return 11;
    a = oracle_accept(o.n_nodes, b.tokens, b.parents, L, b.topk_ids[0], tn, NULL, acc, &bonus);
    if (a < 0 || a > L) return 12;

    /* verifier-side steps */
    double *bias = ALLOC(double, n_max * n_max);
    oracle_mask_to_bias(o.n_nodes, n_max, b.mask, (n_max + 63) / 64, bias);
    const int64_t row_bytes = 24;
    uint8_t *rows = ALLOC(uint8_t, n_max * row_bytes);
    for (int i = 0; i < n_max * row_bytes; ++i) rows[i] = (uint8_t)next_u64();
    rc = oracle_gather_rows(a, acc, rows, row_bytes, rows, row_bytes, row_bytes);
    if (rc) return rc;

    free(bias); free(rows); free(acc); free(td); free(tn); free(e32);
    out_free(&b); out_free(&b2);
    free(emb); free(gp); free(gc); free(u); free(logits); free(hid);
    return 0;
}

int main(void)
{
    /*            L  K   V    n_max E  m  saba cen demb hid ties budget beta */
    int rc = 0;
    rc |= run_case(4, 3, 50, 64, 8, 5, 1, 1, 1, 1, 0, 0, 0.2);
    rc |= run_case(4, 3, 50, 64, 8, 5, 0, 0, 0, 0, 1, 64, 1.0);
    rc |= run_case(3, 1, 9, 32, 4, 3, 0, 1, 1, 0, 0, 32, 0.5);     /* K = 1: a chain */
    rc |= run_case(2, 4, 4, 32, 4, 4, 0, 0, 0, 0, 1, 20, 0.0);     /* K = V, beta 0 */
    rc |= run_case(1, 5, 30, 32, 6, 2, 1, 1, 1, 1, 0, 0, 0.2);     /* L = 1 */
    rc |= run_case(5, 2, 40, 32, 6, 7, 0, 0, 1, 0, 1, 0, 1.0);     /* empty tree */
    rc |= run_case(5, 2, 40, 32, 6, 7, 0, 0, 1, 0, 1, 1, 1.0);     /* one node */
    rc |= run_case(6, 4, 200, 128, 16, 8, 1, 1, 1, 1, 1, 0, 0.2);
    rc |= run_case(3, 8, 100, 1024, 8, 4, 0, 0, 0, 0, 0, 1024, 1.0); /* every prefix fits */
    /* degeneration signal: L = 1 and zero states */
    uint16_t z[16] = {0};
    double r[2];
    if (oracle_degen(z, 1, 8, r) != 0.0) rc |= 20;
    if (oracle_degen(z, 2, 8, r) != 0.0) rc |= 21;
    /* top-K with K = V and statistics of a one-entry row */
    uint16_t one = bf16_bits(1.0f);
    int32_t id;
    double x, lse, mp, h;
    rc |= oracle_topk(&one, 1, 1, &id, &x);
    oracle_row_stats(&one, 1, &lse, &mp, &h);
    printf("oracle sanitizer driver: %s\n", rc ? "FAILED" : "ok");
    return rc ? 1 : 0;
}
