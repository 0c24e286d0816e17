/*
 * sfa_oracle.c -- plain fp64 CPU oracle for the Hidden Decoding hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or load
 * this file; it exists so that tests, the smoke check and the CPU-baseline leg of
 * the benchmark can compare the HIP kernels against an obviously correct,
 * independently written reference.  It shares no code, header or constant with
 * the HIP library.
 *
 * What it computes (paper: "Hidden Decoding at Scale", Sec. 2 "Method"):
 *   - multi-stream token expansion, eq. (expansion): expanded position of stream k
 *     of token i holds E_k(x_i); 0-based here: row p = t*n + s holds tables[s][ids[t]];
 *     and its gradient with respect to the tables (the adjoint of that gather: a sum of
 *     upstream rows per token id and stream);
 *   - cyclic replication of the tables when the expansion factor grows,
 *     eq. (cyclic_init): E_{n+k} <- E_k;
 *   - layers that run only the final stream (Sec. "Training Cost", KV-mirror: only
 *     the final stream of each token passes through the mirrored layers, whose keys
 *     and values cover all n streams): the same masks evaluated for the query
 *     positions t*n + n - 1 only;
 *   - token/stream index maps, eq. (indices), 0-based: t(p) = p / n, s(p) = p % n;
 *   - intra-stream attention mask, eq. (mask_intra): key p' visible from query p
 *     iff s(p') == s(p) and p' <= p (equivalently t(p') <= t(p));
 *   - full cross-stream ("mixing") mask, Fig. "masks" (a): the standard causal mask
 *     over the expanded sequence, written here in token/stream form:
 *     t(p') < t(p), or t(p') == t(p) and s(p') <= s(p);
 *   - local cross-stream mask, Fig. "masks" (b): the causal mask above restricted to
 *     a sliding window of w expanded positions, p - p' < w (its cost, O(nLw), is
 *     stated in the appendix on layouts; w itself is not given in the paper and is an
 *     argument here);
 *   - softmax attention under that mask, its log-sum-exp, and the analytic
 *     gradients with respect to q, k and v (standard softmax-attention calculus:
 *     dP = dO v^T, Delta = dO . O, dS = P (dP - Delta), dQ = scale dS K,
 *     dK = scale dS^T Q, dV = P^T dO; grouped-query heads sum dK/dV over the
 *     query heads that share a key/value head).
 *
 * Everything is fp64.  Inputs may be given as fp64, fp32 or bf16 bit patterns and
 * are upcast exactly.  The mask is evaluated from its definition for every
 * (query, key) pair; only visible pairs contribute.  No blocking, no online
 * softmax, no reordering beyond the plain definitions above.
 *
 * Layouts (row-major, 0-based):
 *   q, o, dO, dq : [B][N][Hq][D]     k, v, dk, dv : [B][N][Hkv][D]
 *   lse          : [B][Hq][N] (natural log)        N = n * L
 *   with ORC_FINAL or-ed into the mode (queries at the final stream only, keys and
 *   values from all n streams): q, o, dO, dq [B][L][Hq][D] and lse [B][Hq][L]; the
 *   row-selecting entry points still name query rows by expanded position.
 *   query head hq uses key/value head hq / (Hq / Hkv).
 *
 * Every function here is pinned by tests (closed forms, library reductions,
 * invariants and finite differences); none is "parity unpinned".
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_INTRA = 0, ORC_MIX = 1, ORC_LOCAL = 2 };
/* or-ed into a mode: only the final stream of each token carries a query row (the
 * layers of Sec. "Training Cost" that run only the final stream, with keys and values
 * from all n streams): q, o, dO and dq are [B][L][Hq][D], lse [B][Hq][L], and query row
 * t sits at expanded position t*n + n - 1 */
enum { ORC_FINAL = 4 };
enum { ORC_F64 = 0, ORC_F32 = 1, ORC_BF16 = 2 };

/* ---------------------------------------------------------------- inputs */

typedef struct {
    const void *q, *k, *v, *dout;
    int dtype;
    int64_t B, L, n, Hq, Hkv, D;
    int mode;
    int64_t window; /* local cross-stream layers only */
    double scale;
    int final_q; /* ORC_FINAL: queries at the final-stream positions only */
} problem_t;

static double load_elem(const void *base, int dtype, int64_t idx)
{
    if (dtype == ORC_F64) return ((const double *)base)[idx];
    if (dtype == ORC_F32) return (double)((const float *)base)[idx];
    /* bf16: the 16 stored bits are the top half of an fp32 */
    uint32_t bits = ((uint32_t)((const uint16_t *)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* ------------------------------------------------- index maps and masks */

/* eq. (indices), 0-based: token and stream of expanded position p */
static int64_t token_of(int64_t p, int64_t n) { return p / n; }
static int64_t stream_of(int64_t p, int64_t n) { return p % n; }

/* 1 if key position pk is visible from query position pq */
static int visible(int mode, int64_t n, int64_t window, int64_t pq, int64_t pk)
{
    int64_t t = token_of(pq, n), s = stream_of(pq, n);
    int64_t tk = token_of(pk, n), sk = stream_of(pk, n);
    if (mode == ORC_INTRA) /* eq. (mask_intra): same stream, not later */
        return sk == s && pk <= pq;
    /* full cross-stream layer: causal over the expanded sequence */
    int causal = tk < t || (tk == t && sk <= s);
    if (mode == ORC_LOCAL) /* ... and fewer than w expanded positions back */
        return causal && pq - pk < window;
    return causal;
}

/* element (b, p, h, d) of q, o, dO or dq; p is an expanded position, which for
 * final-stream queries is t*n + n - 1 and maps to row t of the [B][L] tensors */
static int64_t q_index(const problem_t *P, int64_t b, int64_t p, int64_t h, int64_t d)
{
    if (P->final_q) return ((b * P->L + token_of(p, P->n)) * P->Hq + h) * P->D + d;
    return ((b * (P->n * P->L) + p) * P->Hq + h) * P->D + d;
}

/* does expanded position p carry a query row? */
static int is_query(const problem_t *P, int64_t p)
{
    return !P->final_q || stream_of(p, P->n) == P->n - 1;
}

/* index of p's entry in lse [B][Hq][rows] */
static int64_t lse_index(const problem_t *P, int64_t b, int64_t hq, int64_t p)
{
    if (P->final_q) return (b * P->Hq + hq) * P->L + token_of(p, P->n);
    return (b * P->Hq + hq) * (P->n * P->L) + p;
}

static int64_t kv_index(const problem_t *P, int64_t b, int64_t p, int64_t h, int64_t d)
{
    return ((b * (P->n * P->L) + p) * P->Hkv + h) * P->D + d;
}

/* ------------------------------------------------------- one query row */

/*
 * Forward of one query row (b, hq, p).  x (length N) is caller scratch; on return
 * x[j] holds the probability P_pj for visible j and 0 otherwise.  o gets D values.
 */
static void row_forward(const problem_t *P, int64_t b, int64_t hq, int64_t p,
                        double *x, double *o, double *lse)
{
    const int64_t N = P->n * P->L, D = P->D;
    const int64_t hk = hq / (P->Hq / P->Hkv);
    double m = -INFINITY;
    for (int64_t j = 0; j < N; ++j) {
        if (!visible(P->mode, P->n, P->window, p, j)) { x[j] = -INFINITY; continue; }
        double dot = 0.0;
        for (int64_t d = 0; d < D; ++d)
            dot += load_elem(P->q, P->dtype, q_index(P, b, p, hq, d)) *
                   load_elem(P->k, P->dtype, kv_index(P, b, j, hk, d));
        x[j] = P->scale * dot;
        if (x[j] > m) m = x[j];
    }
    double l = 0.0;
    for (int64_t j = 0; j < N; ++j)
        if (x[j] != -INFINITY) l += exp(x[j] - m);
    for (int64_t j = 0; j < N; ++j)
        x[j] = (x[j] == -INFINITY) ? 0.0 : exp(x[j] - m) / l;
    for (int64_t d = 0; d < D; ++d) o[d] = 0.0;
    for (int64_t j = 0; j < N; ++j) {
        if (!visible(P->mode, P->n, P->window, p, j)) continue;
        for (int64_t d = 0; d < D; ++d)
            o[d] += x[j] * load_elem(P->v, P->dtype, kv_index(P, b, j, hk, d));
    }
    *lse = m + log(l);
}

/*
 * Backward of one query row.  Needs the row's probabilities (x from row_forward)
 * and its exact output o.  Writes dq (D values, may be NULL) and, when dk/dv are
 * non-NULL, adds this row's contributions into dk/dv rows laid out [N][D] for the
 * key/value head of hq (caller owns the per-head accumulation).
 */
static void row_backward(const problem_t *P, int64_t b, int64_t hq, int64_t p,
                         const double *x, const double *o, double *dq,
                         double *dk_head, double *dv_head, const int64_t *only_key,
                         int64_t n_only)
{
    const int64_t N = P->n * P->L, D = P->D;
    const int64_t hk = hq / (P->Hq / P->Hkv);
    double delta = 0.0; /* Delta_p = dO_p . O_p */
    for (int64_t d = 0; d < D; ++d)
        delta += load_elem(P->dout, P->dtype, q_index(P, b, p, hq, d)) * o[d];
    if (dq)
        for (int64_t d = 0; d < D; ++d) dq[d] = 0.0;
    for (int64_t j = 0; j < N; ++j) {
        if (!visible(P->mode, P->n, P->window, p, j)) continue;
        int64_t slot = j;
        if (only_key) { /* restrict dk/dv accumulation to listed keys */
            slot = -1;
            for (int64_t r = 0; r < n_only; ++r)
                if (only_key[r] == j) { slot = r; break; }
            if (slot < 0 && !dq) continue;
        }
        double dp = 0.0; /* dP_pj = dO_p . v_j */
        for (int64_t d = 0; d < D; ++d)
            dp += load_elem(P->dout, P->dtype, q_index(P, b, p, hq, d)) *
                  load_elem(P->v, P->dtype, kv_index(P, b, j, hk, d));
        double ds = x[j] * (dp - delta); /* dS_pj */
        if (dq)
            for (int64_t d = 0; d < D; ++d)
                dq[d] += P->scale * ds * load_elem(P->k, P->dtype, kv_index(P, b, j, hk, d));
        if (dk_head && slot >= 0)
            for (int64_t d = 0; d < D; ++d) {
                dk_head[slot * D + d] +=
                    P->scale * ds * load_elem(P->q, P->dtype, q_index(P, b, p, hq, d));
                dv_head[slot * D + d] +=
                    x[j] * load_elem(P->dout, P->dtype, q_index(P, b, p, hq, d));
            }
    }
}

/* ---------------------------------------------------------- threading */

typedef struct {
    const problem_t *P;
    int64_t first, count; /* work units */
    void *out[6];
    const int64_t *rows;
    int64_t nrows;
} job_t;

typedef void *(*job_fn)(void *);

static void run_jobs(job_fn fn, job_t *tmpl, int64_t units, int nthreads)
{
    if (nthreads < 1) nthreads = 1;
    if (nthreads > units) nthreads = (int)(units > 0 ? units : 1);
    pthread_t *th = calloc((size_t)nthreads, sizeof *th);
    job_t *jobs = calloc((size_t)nthreads, sizeof *jobs);
    int64_t per = units / nthreads, extra = units % nthreads, at = 0;
    for (int i = 0; i < nthreads; ++i) {
        jobs[i] = *tmpl;
        jobs[i].first = at;
        jobs[i].count = per + (i < extra ? 1 : 0);
        at += jobs[i].count;
    }
    for (int i = 1; i < nthreads; ++i) pthread_create(&th[i], NULL, fn, &jobs[i]);
    fn(&jobs[0]);
    for (int i = 1; i < nthreads; ++i) pthread_join(th[i], NULL);
    free(th);
    free(jobs);
}

/* ------------------------------------------------------------ forward */

/* unit = one (b, hq) head; all N rows */
static void *fwd_job(void *arg)
{
    job_t *J = arg;
    const problem_t *P = J->P;
    const int64_t N = P->n * P->L;
    double *o = J->out[0], *lse = J->out[1];
    double *x = malloc((size_t)N * sizeof *x);
    for (int64_t u = J->first; u < J->first + J->count; ++u) {
        int64_t b = u / P->Hq, hq = u % P->Hq;
        for (int64_t p = 0; p < N; ++p)
            if (is_query(P, p))
                row_forward(P, b, hq, p, x, &o[q_index(P, b, p, hq, 0)],
                            &lse[lse_index(P, b, hq, p)]);
    }
    free(x);
    return NULL;
}

static problem_t make_problem(const void *q, const void *k, const void *v, const void *dout,
                              int dtype, int64_t B, int64_t L, int64_t n, int64_t Hq,
                              int64_t Hkv, int64_t D, int mode, int64_t window, double scale)
{
    problem_t P = {q, k, v, dout, dtype, B, L, n, Hq, Hkv, D, mode & 3, window, scale,
                   (mode & ORC_FINAL) != 0};
    return P;
}

/* Full forward: o [B][N][Hq][D], lse [B][Hq][N]. */
void oracle_sfa_fwd(const void *q, const void *k, const void *v, int dtype, double *o,
                    double *lse, int64_t B, int64_t L, int64_t n, int64_t Hq, int64_t Hkv,
                    int64_t D, int mode, int64_t window, double scale, int nthreads)
{
    problem_t P = make_problem(q, k, v, NULL, dtype, B, L, n, Hq, Hkv, D, mode, window, scale);
    job_t J = {&P, 0, 0, {o, lse}, NULL, 0};
    run_jobs(fwd_job, &J, B * Hq, nthreads);
}

/* unit = one listed row (b, hq, p) */
static void *fwd_rows_job(void *arg)
{
    job_t *J = arg;
    const problem_t *P = J->P;
    const int64_t N = P->n * P->L, D = P->D;
    double *o = J->out[0], *lse = J->out[1];
    double *x = malloc((size_t)N * sizeof *x);
    for (int64_t r = J->first; r < J->first + J->count; ++r) {
        const int64_t *row = &J->rows[3 * r];
        row_forward(P, row[0], row[1], row[2], x, &o[r * D], &lse[r]);
    }
    free(x);
    return NULL;
}

/* Forward of selected rows: rows = nrows triplets (b, hq, p); o_rows [nrows][D]. */
void oracle_sfa_fwd_rows(const void *q, const void *k, const void *v, int dtype,
                         const int64_t *rows, int64_t nrows, double *o_rows,
                         double *lse_rows, int64_t B, int64_t L, int64_t n, int64_t Hq,
                         int64_t Hkv, int64_t D, int mode, int64_t window, double scale, int nthreads)
{
    problem_t P = make_problem(q, k, v, NULL, dtype, B, L, n, Hq, Hkv, D, mode, window, scale);
    job_t J = {&P, 0, 0, {o_rows, lse_rows}, rows, nrows};
    run_jobs(fwd_rows_job, &J, nrows, nthreads);
}

/* ----------------------------------------------------------- backward */

/* unit = one (b, hq) query head, all its rows; dq is written in place and the head's
 * dK/dV contributions go to its own [N][D] buffers (summed per key/value head after
 * all units have run, in ascending hq order) */
static void *bwd_job(void *arg)
{
    job_t *J = arg;
    const problem_t *P = J->P;
    const int64_t N = P->n * P->L, D = P->D;
    double *dq = J->out[0], *dk_part = J->out[3], *dv_part = J->out[4];
    double *x = malloc((size_t)N * sizeof *x);
    double *o = malloc((size_t)D * sizeof *o);
    for (int64_t u = J->first; u < J->first + J->count; ++u) {
        int64_t b = u / P->Hq, hq = u % P->Hq;
        double *dk_head = dk_part + u * N * D, *dv_head = dv_part + u * N * D;
        memset(dk_head, 0, (size_t)(N * D) * sizeof *dk_head);
        memset(dv_head, 0, (size_t)(N * D) * sizeof *dv_head);
        for (int64_t p = 0; p < N; ++p) {
            if (!is_query(P, p)) continue;
            double lse;
            row_forward(P, b, hq, p, x, o, &lse);
            row_backward(P, b, hq, p, x, o, &dq[q_index(P, b, p, hq, 0)], dk_head, dv_head,
                         NULL, 0);
        }
    }
    free(x);
    free(o);
    return NULL;
}

/* Full backward from (q, k, v, dO): dq [B][N][Hq][D], dk/dv [B][N][Hkv][D].  Threads
 * take whole query heads; dk/dv of a key/value head are the sum of its group's query
 * heads, added in ascending head order. */
void oracle_sfa_bwd(const void *q, const void *k, const void *v, const void *dout, int dtype,
                    double *dq, double *dk, double *dv, int64_t B, int64_t L, int64_t n,
                    int64_t Hq, int64_t Hkv, int64_t D, int mode, int64_t window, double scale, int nthreads)
{
    problem_t P = make_problem(q, k, v, dout, dtype, B, L, n, Hq, Hkv, D, mode, window, scale);
    const int64_t N = n * L, G = Hq / Hkv;
    double *dk_part = malloc((size_t)(B * Hq * N * D) * sizeof *dk_part);
    double *dv_part = malloc((size_t)(B * Hq * N * D) * sizeof *dv_part);
    job_t J = {&P, 0, 0, {dq, NULL, NULL, dk_part, dv_part}, NULL, 0};
    run_jobs(bwd_job, &J, B * Hq, nthreads);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t hk = 0; hk < Hkv; ++hk)
            for (int64_t j = 0; j < N; ++j)
                for (int64_t d = 0; d < D; ++d) {
                    double sk = 0.0, sv = 0.0;
                    for (int64_t hq = hk * G; hq < (hk + 1) * G; ++hq) {
                        sk += dk_part[((b * Hq + hq) * N + j) * D + d];
                        sv += dv_part[((b * Hq + hq) * N + j) * D + d];
                    }
                    dk[kv_index(&P, b, j, hk, d)] = sk;
                    dv[kv_index(&P, b, j, hk, d)] = sv;
                }
    free(dk_part);
    free(dv_part);
}

/* unit = one listed query row (b, hq, p) */
static void *dq_rows_job(void *arg)
{
    job_t *J = arg;
    const problem_t *P = J->P;
    const int64_t N = P->n * P->L, D = P->D;
    double *dq = J->out[0];
    double *x = malloc((size_t)N * sizeof *x);
    double *o = malloc((size_t)D * sizeof *o);
    for (int64_t r = J->first; r < J->first + J->count; ++r) {
        const int64_t *row = &J->rows[3 * r];
        double lse;
        row_forward(P, row[0], row[1], row[2], x, o, &lse);
        row_backward(P, row[0], row[1], row[2], x, o, &dq[r * D], NULL, NULL, NULL, 0);
    }
    free(x);
    free(o);
    return NULL;
}

/* dQ of selected query rows (b, hq, p); dq_rows [nrows][D]. */
void oracle_sfa_bwd_dq_rows(const void *q, const void *k, const void *v, const void *dout,
                            int dtype, const int64_t *rows, int64_t nrows, double *dq_rows,
                            int64_t B, int64_t L, int64_t n, int64_t Hq, int64_t Hkv,
                            int64_t D, int mode, int64_t window, double scale, int nthreads)
{
    problem_t P = make_problem(q, k, v, dout, dtype, B, L, n, Hq, Hkv, D, mode, window, scale);
    job_t J = {&P, 0, 0, {dq_rows}, rows, nrows};
    run_jobs(dq_rows_job, &J, nrows, nthreads);
}

/* dK/dV of the listed keys of one key/value head (b, hk).  Work units are the query
 * rows (hq, p) of its group; thread t takes units t, t + nthreads, ... (causal rows
 * differ in length) and adds each row's contributions to the listed keys into its own
 * [nkeys][D] buffers; the threads' buffers are summed in thread order afterwards.
 * Every query row's probabilities are formed once for all listed keys. */
typedef struct {
    const problem_t *P;
    int64_t b, hk, tid, nthreads;
    const int64_t *keys;
    int64_t nkeys;
    double *dk, *dv; /* this thread's [nkeys][D] */
} keyjob_t;

static void *dkdv_keys_job(void *arg)
{
    keyjob_t *J = arg;
    const problem_t *P = J->P;
    const int64_t N = P->n * P->L, D = P->D, G = P->Hq / P->Hkv;
    double *x = malloc((size_t)N * sizeof *x);
    double *o = malloc((size_t)D * sizeof *o);
    for (int64_t u = J->tid; u < G * N; u += J->nthreads) {
        const int64_t hq = J->hk * G + u / N, p = u % N;
        if (!is_query(P, p)) continue;
        int sees = 0; /* does this row see any listed key? */
        for (int64_t r = 0; r < J->nkeys && !sees; ++r)
            sees = visible(P->mode, P->n, P->window, p, J->keys[r]);
        if (!sees) continue;
        double lse;
        row_forward(P, J->b, hq, p, x, o, &lse);
        row_backward(P, J->b, hq, p, x, o, NULL, J->dk, J->dv, J->keys, J->nkeys);
    }
    free(x);
    free(o);
    return NULL;
}

/* dK/dV of selected key rows (b, hk, j); dk_rows, dv_rows [nrows][D]. */
void oracle_sfa_bwd_dkdv_rows(const void *q, const void *k, const void *v, const void *dout,
                              int dtype, const int64_t *rows, int64_t nrows, double *dk_rows,
                              double *dv_rows, int64_t B, int64_t L, int64_t n, int64_t Hq,
                              int64_t Hkv, int64_t D, int mode, int64_t window, double scale, int nthreads)
{
    problem_t P = make_problem(q, k, v, dout, dtype, B, L, n, Hq, Hkv, D, mode, window, scale);
    if (nthreads < 1) nthreads = 1;
    int64_t *keys = malloc((size_t)(nrows > 0 ? nrows : 1) * sizeof *keys);
    int64_t *slot = malloc((size_t)(nrows > 0 ? nrows : 1) * sizeof *slot);
    char *done = calloc((size_t)(nrows > 0 ? nrows : 1), 1);
    pthread_t *th = calloc((size_t)nthreads, sizeof *th);
    keyjob_t *jobs = calloc((size_t)nthreads, sizeof *jobs);
    for (int64_t r0 = 0; r0 < nrows; ++r0) {
        if (done[r0]) continue;
        const int64_t b = rows[3 * r0], hk = rows[3 * r0 + 1];
        /* the distinct keys listed for (b, hk); slot[r] = position of row r's key */
        int64_t nk = 0;
        for (int64_t r = r0; r < nrows; ++r) {
            if (rows[3 * r] != b || rows[3 * r + 1] != hk) continue;
            int64_t s = 0;
            while (s < nk && keys[s] != rows[3 * r + 2]) ++s;
            if (s == nk) keys[nk++] = rows[3 * r + 2];
            slot[r] = s;
            done[r] = 1;
        }
        double *buf = calloc((size_t)(2 * nthreads * nk * D), sizeof *buf);
        for (int t = 0; t < nthreads; ++t) {
            keyjob_t j = {&P, b, hk, t, nthreads, keys, nk, buf + (2 * t) * nk * D,
                          buf + (2 * t + 1) * nk * D};
            jobs[t] = j;
        }
        for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, dkdv_keys_job, &jobs[t]);
        dkdv_keys_job(&jobs[0]);
        for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
        for (int64_t r = r0; r < nrows; ++r) {
            if (rows[3 * r] != b || rows[3 * r + 1] != hk) continue;
            for (int64_t d = 0; d < D; ++d) {
                double sk = 0.0, sv = 0.0;
                for (int t = 0; t < nthreads; ++t) {
                    sk += jobs[t].dk[slot[r] * D + d];
                    sv += jobs[t].dv[slot[r] * D + d];
                }
                dk_rows[r * D + d] = sk;
                dv_rows[r * D + d] = sv;
            }
        }
        free(buf);
    }
    free(keys);
    free(slot);
    free(done);
    free(th);
    free(jobs);
}

/* ---------------------------------------------------- stream expansion */

/*
 * eq. (expansion), 0-based: out[b][t*n + s][:] = tables[s][ids[b][t]][:].
 * Element-size agnostic byte copy.  An id outside [0, V) gives n zero rows and
 * counts once (per token, not per stream); the count is returned.
 */
int64_t oracle_expand_embed(const int32_t *ids, const void *tables, void *out, int64_t B,
                            int64_t L, int64_t n, int64_t V, int64_t Dm, int64_t elem_bytes)
{
    int64_t bad = 0;
    const int64_t row_bytes = Dm * elem_bytes;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < L; ++t)
            for (int64_t s = 0; s < n; ++s) {
                int64_t p = t * n + s;
                int64_t id = ids[b * L + t];
                char *dst = (char *)out + (b * n * L + p) * row_bytes;
                if (id < 0 || id >= V) {
                    memset(dst, 0, (size_t)row_bytes);
                    if (s == 0) ++bad;
                    continue;
                }
                const char *src = (const char *)tables + (s * V + id) * row_bytes;
                memcpy(dst, src, (size_t)row_bytes);
            }
    return bad;
}

/*
 * Gradient of eq. (expansion) with respect to the n tables.  The expansion is a
 * gather, out[b][t*n + s] = tables[s][ids[b][t]], so for any upstream gradient dout
 *   dtables[s][x][:] = sum over tokens (b, t) with ids[b][t] == x of dout[b][t*n + s][:],
 * and tokens whose id lies outside [0, V) contribute nothing (their expanded rows are
 * constant zeros).  Dense fp64 [n][V][Dm] output, overwritten; tokens are visited in
 * (b, t) order.
 */
void oracle_expand_embed_bwd(const int32_t *ids, const void *dout, int dtype, double *dtables,
                             int64_t B, int64_t L, int64_t n, int64_t V, int64_t Dm)
{
    memset(dtables, 0, (size_t)(n * V * Dm) * sizeof(double));
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < L; ++t) {
            const int64_t id = ids[b * L + t];
            if (id < 0 || id >= V) continue;
            for (int64_t s = 0; s < n; ++s) {
                const int64_t row = b * n * L + t * n + s;
                double *dst = dtables + (s * V + id) * Dm;
                for (int64_t d = 0; d < Dm; ++d) dst[d] += load_elem(dout, dtype, row * Dm + d);
            }
        }
}

/*
 * The same gradient for a list of token ids only: drows[r][s][:] = dtables[s][req[r]][:]
 * above, each formed by scanning every token of the batch (for large vocabularies).
 */
void oracle_expand_embed_bwd_rows(const int32_t *ids, const void *dout, int dtype,
                                  const int32_t *req, int64_t nreq, double *drows, int64_t B,
                                  int64_t L, int64_t n, int64_t V, int64_t Dm)
{
    memset(drows, 0, (size_t)(nreq * n * Dm) * sizeof(double));
    for (int64_t r = 0; r < nreq; ++r) {
        const int64_t x = req[r];
        if (x < 0 || x >= V) continue;
        for (int64_t b = 0; b < B; ++b)
            for (int64_t t = 0; t < L; ++t) {
                if (ids[b * L + t] != x) continue;
                for (int64_t s = 0; s < n; ++s) {
                    const int64_t row = b * n * L + t * n + s;
                    double *dst = drows + (r * n + s) * Dm;
                    for (int64_t d = 0; d < Dm; ++d) dst[d] += load_elem(dout, dtype, row * Dm + d);
                }
            }
    }
}

/*
 * eq. (cyclic_init), 0-based: growing the expansion factor from n to m (a multiple of
 * n), the m tables are dst[s] = src[s mod n]; for m = 2n this is E_{n+k} <- E_k.
 * Element-size agnostic byte copy; src [n][V][Dm], dst [m][V][Dm].
 */
void oracle_cyclic_replicate(const void *src, void *dst, int64_t n, int64_t m, int64_t V,
                             int64_t Dm, int64_t elem_bytes)
{
    const size_t table = (size_t)(V * Dm * elem_bytes);
    for (int64_t s = 0; s < m; ++s)
        memcpy((char *)dst + s * table, (const char *)src + (s % n) * table, table);
}

/* Mask as bytes [N][N] straight from the definition (for probes and pins). */
void oracle_sfa_mask(unsigned char *mask, int64_t L, int64_t n, int mode, int64_t window)
{
    const int64_t N = n * L;
    for (int64_t p = 0; p < N; ++p)
        for (int64_t j = 0; j < N; ++j) mask[p * N + j] = (unsigned char)visible(mode, n, window, p, j);
}

/* Final-stream gather, eq. (hd_loss): the loss reads the hidden state of token i only at
 * the final stream of its block, expanded position i*n + n - 1 (0-based), so
 * out[b][i][:] = h[b][i*n + n - 1][:] for h [B][n*L][Dm] and out [B][L][Dm].  Elements
 * are copied as opaque elem_bytes-byte values. */
void oracle_final_gather(const void *h, void *out, int64_t B, int64_t L, int64_t n,
                         int64_t Dm, int64_t elem_bytes)
{
    const size_t row = (size_t)(Dm * elem_bytes);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < L; ++i)
            memcpy((char *)out + (size_t)(b * L + i) * row,
                   (const char *)h + (size_t)(b * n * L + i * n + n - 1) * row, row);
}

/* Its adjoint: the gradient w.r.t. h is dout at the final-stream positions and zero at
 * the other n - 1 positions of every token (those receive no direct loss). */
void oracle_final_gather_bwd(const void *dout, void *dh, int64_t B, int64_t L, int64_t n,
                             int64_t Dm, int64_t elem_bytes)
{
    const size_t row = (size_t)(Dm * elem_bytes);
    memset(dh, 0, (size_t)(B * n * L) * row);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < L; ++i)
            memcpy((char *)dh + (size_t)(b * n * L + i * n + n - 1) * row,
                   (const char *)dout + (size_t)(b * L + i) * row, row);
}
