/*
 * oracle.c -- plain, slow fp64 CPU oracle for HeadWiseKV's grouped-cache
 * runtime (per-KV-head sink + recent-window residency, and the attention a
 * query computes over what is resident).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: it is used by the tests, by the smoke check and by the
 * benchmark's CPU-baseline leg, and by nothing else.  It shares no code,
 * header, table or helper with the HIP library; it is written from the
 * paper's definitions:
 *
 *   - window semantics J_t(w) = {max(1, t-w+1) .. t} (Method, "Sequential
 *     Prefix-Conditioned Calibration", definition of the available positions),
 *     here 0-based: a finite window w keeps positions s in [t+1-w, t];
 *   - "any w >= C is equivalent to full" (Method, "Structured Residency
 *     Model");
 *   - retained count r_C(w) = min(w, C), r_C(full) = C, nominal storage
 *     (Eq. nominal-storage) and the normalized rate (Eq. normalized-rate);
 *   - attention sinks as an additive prefix: the sink+recent control keeps
 *     4 sinks plus a 90,364-token window in a 90,368-token cache and starts
 *     evicting above 90,368 tokens (Appendix "Supplementary Evaluation",
 *     baseline controls).  The retained set of a finite unit at length n is
 *     therefore {p < S} U {p >= n - w}, of size min(n, S + w);
 *   - the attention output (Eqs. conditional-attention-weight and
 *     conditional-attention) with the exact scaled dot product logit
 *     z = gamma q.k.
 *
 * Readings taken where the paper is silent (all listed in the design notes):
 *   - the slot a resident token occupies in a unit's physical storage is
 *     slot(p) = p for full units and for sinks (p < S), and
 *     slot(p) = S + ((p - S) mod w) otherwise (a ring over the window);
 *   - a decode step appends token t and then attends with query t over the
 *     retained set at length t + 1 (the query's own token included, as J_t(w)
 *     includes t);
 *   - K/V/Q arrive as bf16 bit patterns and are widened exactly to fp64.
 *
 * Window encoding used throughout: w > 0 is a finite window, w == 0 is
 * "full history".  Positions and lengths are int64.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* bf16 -> fp64, exact: a bf16 value is the upper half of an IEEE fp32.      */
/* ------------------------------------------------------------------------- */
static double bf16_to_f64(uint16_t h)
{
    uint32_t bits = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

double orc_bf16_to_f64(uint16_t h) { return bf16_to_f64(h); }

/* ------------------------------------------------------------------------- */
/* Residency (Method, window semantics; sink+recent control).                */
/* ------------------------------------------------------------------------- */

/* Is position p (0-based) retained by a unit whose sequence has length n?
 * Full units keep every p < n.  Finite units keep the S sinks and the last w
 * positions. */
int orc_is_resident(int64_t p, int64_t n, int64_t n_sinks, int64_t window)
{
    if (p < 0 || p >= n)
        return 0;
    if (window == 0)
        return 1;
    if (p < n_sinks)
        return 1;
    return p >= n - window;
}

/* |R(n)| counted by enumeration (deliberately not the closed form, so that
 * the closed form min(n, S + w) can be tested against it). */
int64_t orc_resident_count(int64_t n, int64_t n_sinks, int64_t window)
{
    int64_t c = 0;
    for (int64_t p = 0; p < n; ++p)
        c += orc_is_resident(p, n, n_sinks, window);
    return c;
}

/* Physical capacity of one unit for one sequence, in token rows.  A finite
 * window whose sinks plus window reach max_ctx never evicts before max_ctx,
 * so it is the same as full ("any w >= C is equivalent to full"). */
int64_t orc_capacity(int64_t n_sinks, int64_t window, int64_t max_ctx)
{
    if (window == 0 || n_sinks + window >= max_ctx)
        return max_ctx;
    return n_sinks + window;
}

/* Canonical slot of position p (a reading: the paper fixes the retained set,
 * not its arrangement). */
int64_t orc_slot(int64_t p, int64_t n_sinks, int64_t window)
{
    if (window == 0 || p < n_sinks)
        return p;
    return n_sinks + (p - n_sinks) % window;
}

/* ------------------------------------------------------------------------- */
/* Accounting (Eq. nominal-storage, Eq. normalized-rate).                     */
/* r_C(w) counts the retained tokens at context C: min(S + w, C) for a finite */
/* window with S additive sinks, C for full.                                 */
/* ------------------------------------------------------------------------- */
int64_t orc_retained_tokens(int64_t ctx, int64_t n_sinks, int64_t window)
{
    if (window == 0)
        return ctx;
    return (n_sinks + window < ctx) ? n_sinks + window : ctx;
}

/* n_{lh,C}(w) = r_C(w) * (d^K b^K + d^V b^V), bytes. */
double orc_unit_bytes(int64_t ctx, int64_t n_sinks, int64_t window,
                      int64_t d_k, int64_t d_v, double b_k, double b_v)
{
    return (double)orc_retained_tokens(ctx, n_sinks, window) *
           ((double)d_k * b_k + (double)d_v * b_v);
}

/* N_C(a) summed over the units; windows[u] is the window of unit u. */
double orc_policy_bytes(int64_t ctx, int64_t n_sinks, int64_t n_units,
                        const int64_t *windows, int64_t d_k, int64_t d_v,
                        double b_k, double b_v)
{
    double total = 0.0;
    for (int64_t u = 0; u < n_units; ++u)
        total += orc_unit_bytes(ctx, n_sinks, windows[u], d_k, d_v, b_k, b_v);
    return total;
}

/* R_C(a) = N_C(a) / N_C(all full). */
double orc_rate(int64_t ctx, int64_t n_sinks, int64_t n_units,
                const int64_t *windows, int64_t d_k, int64_t d_v,
                double b_k, double b_v)
{
    double num = orc_policy_bytes(ctx, n_sinks, n_units, windows, d_k, d_v,
                                  b_k, b_v);
    double den = 0.0;
    for (int64_t u = 0; u < n_units; ++u)
        den += orc_unit_bytes(ctx, n_sinks, 0, d_k, d_v, b_k, b_v);
    return num / den;
}

/* ------------------------------------------------------------------------- */
/* Slot table of one unit and one sequence: table[j] is the position held in */
/* slot j, or -1 when the slot is empty.                                      */
/* ------------------------------------------------------------------------- */
void orc_table_init(int64_t *table, int64_t cap)
{
    for (int64_t j = 0; j < cap; ++j)
        table[j] = -1;
}

/* Materialise the chunk [p0, p1): every position of the chunk that is still
 * retained once the sequence has length p1 is stored in its slot; nothing
 * else is touched.  Returns 0, or -1 when a slot falls outside the table. */
int orc_table_prefill(int64_t *table, int64_t cap, int64_t n_sinks,
                      int64_t window, int64_t p0, int64_t p1)
{
    for (int64_t p = p0; p < p1; ++p) {
        if (!orc_is_resident(p, p1, n_sinks, window))
            continue;
        int64_t j = orc_slot(p, n_sinks, window);
        if (j < 0 || j >= cap)
            return -1;
        table[j] = p;
    }
    return 0;
}

/* Append position n (the sequence grows from n to n + 1).  Returns 0, or -1
 * when the slot falls outside the table. */
int orc_table_append(int64_t *table, int64_t cap, int64_t n_sinks,
                     int64_t window, int64_t n)
{
    int64_t j = orc_slot(n, n_sinks, window);
    if (j < 0 || j >= cap)
        return -1;
    table[j] = n;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Attention (Eqs. conditional-attention-weight, conditional-attention).      */
/* ------------------------------------------------------------------------- */

/* Output of one query head at query position t over the positions retained
 * at length t + 1, read from the FULL history ("masked full cache"):
 *   z_s = scale * sum_i q_i k_{s,i}      for retained s, ascending s
 *   o   = sum_s exp(z_s - m) v_s / sum_s exp(z_s - m),  m = max_s z_s
 * k_hist/v_hist point at row 0 of this KV head; row s starts at
 * s * row_stride elements.  All arithmetic in fp64. */
void orc_attend_row(const uint16_t *q, const uint16_t *k_hist,
                    const uint16_t *v_hist, int64_t row_stride, int64_t d,
                    int64_t t, int64_t n_sinks, int64_t window, double scale,
                    double *out)
{
    double m = -INFINITY;
    for (int64_t s = 0; s <= t; ++s) {
        if (!orc_is_resident(s, t + 1, n_sinks, window))
            continue;
        const uint16_t *k = k_hist + s * row_stride;
        double dot = 0.0;
        for (int64_t i = 0; i < d; ++i)
            dot += bf16_to_f64(q[i]) * bf16_to_f64(k[i]);
        double z = scale * dot;
        if (z > m)
            m = z;
    }
    double denom = 0.0;
    for (int64_t i = 0; i < d; ++i)
        out[i] = 0.0;
    for (int64_t s = 0; s <= t; ++s) {
        if (!orc_is_resident(s, t + 1, n_sinks, window))
            continue;
        const uint16_t *k = k_hist + s * row_stride;
        const uint16_t *v = v_hist + s * row_stride;
        double dot = 0.0;
        for (int64_t i = 0; i < d; ++i)
            dot += bf16_to_f64(q[i]) * bf16_to_f64(k[i]);
        double e = exp(scale * dot - m);
        denom += e;
        for (int64_t i = 0; i < d; ++i)
            out[i] += e * bf16_to_f64(v[i]);
    }
    for (int64_t i = 0; i < d; ++i)
        out[i] /= denom;
}

/* The same output computed from a compacted unit: cache_k/cache_v hold one
 * row of d elements per slot, and slot_pos[j] is the position stored in
 * slot j (-1 = empty).  Occupied slots are visited in ascending position
 * order, so the arithmetic is term-for-term that of orc_attend_row. */
typedef struct {
    int64_t pos;
    int64_t slot;
} pos_slot;

static int cmp_pos(const void *a, const void *b)
{
    int64_t x = ((const pos_slot *)a)->pos, y = ((const pos_slot *)b)->pos;
    return (x > y) - (x < y);
}

int orc_attend_slots(const uint16_t *q, const uint16_t *cache_k,
                     const uint16_t *cache_v, int64_t d,
                     const int64_t *slot_pos, int64_t n_slots, double scale,
                     double *out)
{
    pos_slot *order = (pos_slot *)malloc(sizeof(pos_slot) *
                                         (size_t)(n_slots > 0 ? n_slots : 1));
    if (!order)
        return -1;
    int64_t n = 0;
    for (int64_t j = 0; j < n_slots; ++j)
        if (slot_pos[j] >= 0) {
            order[n].pos = slot_pos[j];
            order[n].slot = j;
            ++n;
        }
    qsort(order, (size_t)n, sizeof(pos_slot), cmp_pos);
    double m = -INFINITY;
    for (int64_t r = 0; r < n; ++r) {
        const uint16_t *k = cache_k + order[r].slot * d;
        double dot = 0.0;
        for (int64_t i = 0; i < d; ++i)
            dot += bf16_to_f64(q[i]) * bf16_to_f64(k[i]);
        double z = scale * dot;
        if (z > m)
            m = z;
    }
    double denom = 0.0;
    for (int64_t i = 0; i < d; ++i)
        out[i] = 0.0;
    for (int64_t r = 0; r < n; ++r) {
        const uint16_t *k = cache_k + order[r].slot * d;
        const uint16_t *v = cache_v + order[r].slot * d;
        double dot = 0.0;
        for (int64_t i = 0; i < d; ++i)
            dot += bf16_to_f64(q[i]) * bf16_to_f64(k[i]);
        double e = exp(scale * dot - m);
        denom += e;
        for (int64_t i = 0; i < d; ++i)
            out[i] += e * bf16_to_f64(v[i]);
    }
    for (int64_t i = 0; i < d; ++i)
        out[i] /= denom;
    free(order);
    return (int)n;
}

/* ------------------------------------------------------------------------- */
/* One decode step of one layer, every sequence and every query head, split  */
/* over threads by (sequence, query head).  Query head qh reads KV head      */
/* qh / (n_q_heads / n_kv_heads) (contiguous GQA groups).                    */
/*   q        [batch][n_q_heads][d]                                          */
/*   k_hist[b], v_hist[b]  [>= t[b] + 1][n_kv_heads][d]                      */
/*   windows  [n_kv_heads] (0 = full), t[b] the query position of seq b      */
/*   out      [batch][n_q_heads][d]                                          */
/* ------------------------------------------------------------------------- */
typedef struct {
    int64_t batch, n_q_heads, n_kv_heads, d, n_sinks;
    const int64_t *windows;
    const int64_t *t;
    const uint16_t *q;
    const uint16_t *const *k_hist;
    const uint16_t *const *v_hist;
    double scale;
    double *out;
    int n_threads;
    int tid;
} layer_job;

static void *layer_worker(void *arg)
{
    layer_job *j = (layer_job *)arg;
    int64_t group = j->n_q_heads / j->n_kv_heads;
    int64_t items = j->batch * j->n_q_heads;
    for (int64_t it = j->tid; it < items; it += j->n_threads) {
        int64_t b = it / j->n_q_heads, qh = it % j->n_q_heads;
        int64_t h = qh / group;
        orc_attend_row(j->q + (b * j->n_q_heads + qh) * j->d,
                       j->k_hist[b] + h * j->d, j->v_hist[b] + h * j->d,
                       j->n_kv_heads * j->d, j->d, j->t[b], j->n_sinks,
                       j->windows[h], j->scale,
                       j->out + (b * j->n_q_heads + qh) * j->d);
    }
    return NULL;
}

int orc_decode_layer(int n_threads, int64_t batch, int64_t n_q_heads,
                     int64_t n_kv_heads, int64_t d, int64_t n_sinks,
                     const int64_t *windows, const int64_t *t,
                     const uint16_t *q, const uint16_t *const *k_hist,
                     const uint16_t *const *v_hist, double scale, double *out)
{
    if (n_threads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0)
        return -1;
    layer_job *jobs = (layer_job *)calloc((size_t)n_threads, sizeof *jobs);
    pthread_t *th = (pthread_t *)calloc((size_t)n_threads, sizeof *th);
    if (!jobs || !th) {
        free(jobs);
        free(th);
        return -1;
    }
    for (int i = 0; i < n_threads; ++i) {
        layer_job j = {batch, n_q_heads, n_kv_heads, d, n_sinks, windows, t,
                       q, k_hist, v_hist, scale, out, n_threads, i};
        jobs[i] = j;
    }
    int rc = 0;
    int started = 0;
    for (int i = 1; i < n_threads; ++i) {
        if (pthread_create(&th[i], NULL, layer_worker, &jobs[i]) != 0) {
            rc = -1;
            break;
        }
        started = i;
    }
    layer_worker(&jobs[0]);
    for (int i = 1; i <= started; ++i)
        pthread_join(th[i], NULL);
    if (rc != 0) /* a thread could not start: do its share here */
        for (int i = started + 1; i < n_threads; ++i)
            layer_worker(&jobs[i]);
    free(jobs);
    free(th);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Calibration score (Appendix, "Calibration Score and Fixed-Prefix         */
/* Selection", Eq. stabilized-cosine).                                       */
/* ------------------------------------------------------------------------ */

/* Stabilised cosine of u and v (length d): a vector whose Euclidean norm is
 * at most eps = 1e-12 counts as zero; two zero vectors score 1, exactly one
 * zero vector scores 0, otherwise the plain cosine u.v / (|u| |v|).  fp64. */
double orc_cos_eval(const double *u, const double *v, int64_t d)
{
    const double eps = 1e-12;
    double uu = 0.0, vv = 0.0, uv = 0.0;
    for (int64_t i = 0; i < d; ++i) {
        uu += u[i] * u[i];
        vv += v[i] * v[i];
        uv += u[i] * v[i];
    }
    const double nu = sqrt(uu), nv = sqrt(vv);
    const int zu = nu <= eps, zv = nv <= eps;
    if (zu && zv)
        return 1.0;
    if (zu || zv)
        return 0.0;
    return uv / (nu * nv);
}
