/*
 * kvr_ref.c -- plain fp64 CPU oracle for prefix-reuse attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is compiled and called by the test
 * suite, by the package smoke check and by the CPU-baseline leg of the
 * benchmark.  The GPU library never links, loads or calls it, and it shares
 * no code, header or constant with the GPU library.
 *
 * What it computes (paper: Background "Prefill and the KV cache"; Method
 * "Setup and notation", Alg. 1 and Alg. 2, Claim 1 and its argument):
 *
 *   A decoder layer's attention over a key sequence k_0, k_1, ... where the
 *   query at absolute position p may see exactly the keys j <= p (causal
 *   attention: the entry for a position depends only on earlier positions).
 *   Textbook scaled-dot-product attention, which the paper relies on but never
 *   writes out:
 *       z_j  = scale * sum_c q[c] * k_j[c]          for 0 <= j <= p
 *       m    = max_j z_j
 *       w_j  = exp(z_j - m)
 *       o    = sum_j w_j v_j / sum_j w_j
 *       lse  = m + log(sum_j w_j)
 *
 *   Grouped-query attention: query head h reads kv head g = h / G with
 *   G = n_q_heads / n_kv_heads (contiguous groups; the paper states 8 KV heads
 *   of width 128, Section "Artifact size").
 *
 *   Two modes, one definition:
 *     prefill   -- L tokens, query row i sits at position i, the key sequence is
 *                  the L new keys (Alg. 1's forward pass that fills the cache);
 *     continue  -- S new tokens after a cached prefix of L_prefix tokens; query
 *                  row i sits at position L_prefix + i (the position ids of
 *                  Alg. 2 start at the artifact's length), and the key sequence
 *                  is the cached rows 0..L_prefix-1 followed by the S new keys
 *                  (the mask spans the whole cached context plus the new
 *                  tokens, Section "Consuming an artifact").
 *
 * Layouts (row-major, fp64):
 *     Q, out       [rows][n_q_heads][head_dim]
 *     K, V (new)   [rows][n_kv_heads][head_dim]
 *     cache        [n_kv_heads][capacity][head_dim]
 *     lse          [rows][n_q_heads]
 *
 * Each output element is computed independently with a plain two-pass loop
 * over the visible keys, summing the head dimension in ascending order.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* One stretch of the key sequence: rows [0, count) of some buffer. */
typedef struct {
    const double *k, *v;
    int64_t count;       /* number of key rows in this stretch            */
    int64_t row_stride;  /* elements between consecutive key rows         */
    int64_t head_stride; /* elements between consecutive kv heads         */
} key_span;

typedef struct {
    int n_q_heads, n_kv_heads, head_dim;
    double scale;
    const double *q;         /* [q_rows][n_q_heads][head_dim]   */
    const int64_t *rows;     /* query rows to evaluate, or NULL */
    int64_t n_rows;
    int64_t q_pos0;          /* absolute position of query row 0 */
    key_span first, second;  /* the key sequence = first ++ second */
    int64_t k_lo, k_hi;      /* restrict to keys in [k_lo, k_hi)   */
    double *out, *lse;       /* [n_rows][n_q_heads][head_dim], [n_rows][n_q_heads] */
    int nthreads;
} job;

typedef struct {
    const job *j;
    int tid;
} worker_arg;

/* Pointer to key (or value) row `pos` of kv head `g` in the key sequence. */
static const double *seq_row(const job *j, int64_t pos, int g, int want_value) {
    const key_span *s = &j->first;
    if (pos >= s->count) {
        pos -= s->count;
        s = &j->second;
    }
    const double *base = want_value ? s->v : s->k;
    return base + (int64_t)g * s->head_stride + pos * s->row_stride;
}

static void one_row(const job *j, int64_t item, double *z) {
    const int H = j->n_q_heads, D = j->head_dim;
    const int G = j->n_q_heads / j->n_kv_heads;
    const int64_t r = item / H;        /* index into the row list */
    const int h = (int)(item % H);     /* query head              */
    const int g = h / G;               /* kv head it reads        */
    const int64_t qi = j->rows ? j->rows[r] : r;
    const double *q = j->q + (qi * H + h) * (int64_t)D;
    const int64_t pos = j->q_pos0 + qi;

    int64_t lo = j->k_lo;
    int64_t hi = pos + 1;              /* causal: keys 0..pos     */
    if (hi > j->k_hi) hi = j->k_hi;

    double *o = j->out + (r * H + h) * (int64_t)D;
    for (int c = 0; c < D; ++c) o[c] = 0.0;
    if (hi <= lo) {                    /* no visible key in range */
        j->lse[r * H + h] = -INFINITY;
        return;
    }

    double m = -INFINITY;
    for (int64_t t = lo; t < hi; ++t) {
        const double *k = seq_row(j, t, g, 0);
        double acc = 0.0;
        for (int c = 0; c < D; ++c) acc += q[c] * k[c];
        z[t - lo] = j->scale * acc;
        if (z[t - lo] > m) m = z[t - lo];
    }
    double l = 0.0;
    for (int64_t t = lo; t < hi; ++t) {
        const double w = exp(z[t - lo] - m);
        const double *v = seq_row(j, t, g, 1);
        for (int c = 0; c < D; ++c) o[c] += w * v[c];
        l += w;
    }
    for (int c = 0; c < D; ++c) o[c] /= l;
    j->lse[r * H + h] = m + log(l);
}

static void *worker(void *p) {
    const worker_arg *a = (const worker_arg *)p;
    const job *j = a->j;
    int64_t seq_len = j->first.count + j->second.count;
    double *z = (double *)malloc(sizeof(double) * (size_t)(seq_len > 0 ? seq_len : 1));
    const int64_t items = j->n_rows * j->n_q_heads;
    for (int64_t it = a->tid; it < items; it += j->nthreads) one_row(j, it, z);
    free(z);
    return NULL;
}

static int run(job *j) {
    if (j->n_q_heads <= 0 || j->n_kv_heads <= 0 || j->head_dim <= 0) return 1;
    if (j->n_q_heads % j->n_kv_heads != 0) return 1;
    if (j->nthreads < 1) j->nthreads = 1;
    if (j->nthreads > 256) j->nthreads = 256;
    if (j->n_rows == 0) return 0;
    pthread_t th[256];
    worker_arg args[256];
    for (int t = 0; t < j->nthreads; ++t) {
        args[t].j = j;
        args[t].tid = t;
        if (t > 0 && pthread_create(&th[t], NULL, worker, &args[t]) != 0) return 2;
    }
    worker(&args[0]);
    for (int t = 1; t < j->nthreads; ++t) pthread_join(th[t], NULL);
    return 0;
}

/*
 * Full causal prefill of L tokens (Alg. 1's forward pass, attention part).
 * rows == NULL evaluates every row 0..L-1 (n_rows must then equal L);
 * otherwise only the listed query rows, written densely in list order.
 */
int kvr_ref_prefill(int n_q_heads, int n_kv_heads, int head_dim, double scale,
                    const double *Q, const double *K, const double *V, int64_t L,
                    const int64_t *rows, int64_t n_rows,
                    double *out, double *lse, int nthreads) {
    job j;
    memset(&j, 0, sizeof j);
    j.n_q_heads = n_q_heads; j.n_kv_heads = n_kv_heads; j.head_dim = head_dim;
    j.scale = scale; j.q = Q; j.rows = rows; j.n_rows = n_rows; j.q_pos0 = 0;
    j.second.k = K; j.second.v = V; j.second.count = L;
    j.second.row_stride = (int64_t)n_kv_heads * head_dim;
    j.second.head_stride = head_dim;
    j.k_lo = 0; j.k_hi = L;
    j.out = out; j.lse = lse; j.nthreads = nthreads;
    return run(&j);
}

/*
 * Continuation of S new tokens over a cached prefix (Alg. 2, one forward call
 * with pos = L_prefix..L_prefix+S-1 and a mask spanning all of them).  The
 * cache is read only.  [k_lo, k_hi) restricts the key sequence (use 0 and
 * L_prefix + S for the plain definition); a row with no visible key in the
 * range gets out = 0 and lse = -inf.
 */
int kvr_ref_continue(int n_q_heads, int n_kv_heads, int head_dim, double scale,
                     const double *Qs, const double *Ks, const double *Vs, int64_t S,
                     const double *kcache, const double *vcache, int64_t capacity,
                     int64_t L_prefix, int64_t k_lo, int64_t k_hi,
                     const int64_t *rows, int64_t n_rows,
                     double *out, double *lse, int nthreads) {
    if (L_prefix > capacity) return 1;
    job j;
    memset(&j, 0, sizeof j);
    j.n_q_heads = n_q_heads; j.n_kv_heads = n_kv_heads; j.head_dim = head_dim;
    j.scale = scale; j.q = Qs; j.rows = rows; j.n_rows = n_rows; j.q_pos0 = L_prefix;
    j.first.k = kcache; j.first.v = vcache; j.first.count = L_prefix;
    j.first.row_stride = head_dim; j.first.head_stride = capacity * head_dim;
    j.second.k = Ks; j.second.v = Vs; j.second.count = S;
    j.second.row_stride = (int64_t)n_kv_heads * head_dim;
    j.second.head_stride = head_dim;
    j.k_lo = k_lo; j.k_hi = k_hi;
    j.out = out; j.lse = lse; j.nthreads = nthreads;
    return run(&j);
}

/*
 * Cache write: rows [L_cur, L_cur+S) of each kv head receive the S new K/V
 * rows, unchanged (Alg. 2's cache update; Claim 1's argument needs the stored
 * entries to be exactly what prefill produced).  Other rows are untouched.
 */
int kvr_ref_cache_append(int n_kv_heads, int head_dim, const double *Ks, const double *Vs,
                         int64_t S, double *kcache, double *vcache, int64_t capacity,
                         int64_t L_cur) {
    if (L_cur < 0 || S < 0 || L_cur + S > capacity) return 1;
    for (int64_t t = 0; t < S; ++t)
        for (int g = 0; g < n_kv_heads; ++g)
            for (int c = 0; c < head_dim; ++c) {
                const int64_t src = (t * n_kv_heads + g) * (int64_t)head_dim + c;
                const int64_t dst = ((int64_t)g * capacity + L_cur + t) * head_dim + c;
                kcache[dst] = Ks[src];
                vcache[dst] = Vs[src];
            }
    return 0;
}
