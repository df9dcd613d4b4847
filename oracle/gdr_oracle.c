/*
 * fp64 CPU oracle for the gated delta rule prefill with state checkpoints.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * reference that the GPU library is checked against.  It shares no code,
 * header, table or constant with the GPU path, and nothing in the product
 * path may link, load or call it: only the test suite, the smoke check and
 * the benchmark's cpu_baseline leg do.
 *
 * What it computes (one sequence, every head independently, fp64):
 *
 *   The paper (section 2.2, "State position and scheduler position") fixes
 *   the position semantics: prefix lengths are counts, token indices are
 *   zero based, and a state representing prefix [0, B) supports continuation
 *   from B.  The paper names Flash Linear Attention kernels but never writes
 *   the recurrence; the recurrence taken here is the gated delta rule
 *
 *       S_t = exp(g_t) S_{t-1} + beta_t k_t (v_t - S_{t-1}^T k_t)^T,
 *       o_t = scale * S_t^T q_t,
 *
 *   with S a dk x dv matrix (the "literal" variant).  The "decayed delta"
 *   variant predicts with exp(g_t) S_{t-1} inside the bracket instead.
 *
 *   Checkpoints: after absorbing token t (zero based, absolute position
 *   start + t), the state represents prefix [0, start + t + 1).  Whenever
 *   that length is a multiple of the checkpoint interval C, the state is
 *   written out as a checkpoint (paper, section 2.2 and the checkpoint
 *   interval row of Table 1).  The checkpoint for absolute length P goes to
 *   row P / C - floor(start / C) - 1.
 *
 * Inputs are read from float32 arrays (the stored values, exact in fp64);
 * every operation afterwards is fp64 with libm exp.  Heads are spread over
 * POSIX threads; the arithmetic inside one head is a single sequential loop,
 * so results do not depend on the thread count.
 *
 * Build: gcc -O2 -shared -fPIC gdr_oracle.c -lm -lpthread
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int64_t T;
    int32_t H, dk, dv, variant;
    double scale;
    const float *q, *k, *v, *g, *beta;   /* [T,H,dk] [T,H,dk] [T,H,dv] [T,H] [T,H] */
    int64_t start, C;
    const double *state_in;              /* [H,dk,dv] or NULL (zero state) */
    double *o;                           /* [T,H,dv] or NULL */
    double *state_out;                   /* [H,dk,dv] or NULL */
    double *ckpt;                        /* [n_ckpt,H,dk,dv] or NULL */
    int32_t head_begin, head_end;
    double *S, *pred;                    /* per-thread scratch: [dk,dv], [dv] */
} oracle_job;

static void run_head(const oracle_job *j, int32_t h, double *S, double *pred)
{
    const int32_t H = j->H, dk = j->dk, dv = j->dv;
    const size_t state_elems = (size_t)dk * dv;
    if (j->state_in)
        memcpy(S, j->state_in + (size_t)h * state_elems, state_elems * sizeof(double));
    else
        memset(S, 0, state_elems * sizeof(double));

    for (int64_t t = 0; t < j->T; ++t) {
        const float *kt = j->k + ((size_t)t * H + h) * dk;
        const float *qt = j->q + ((size_t)t * H + h) * dk;
        const float *vt = j->v + ((size_t)t * H + h) * dv;
        const double alpha = exp((double)j->g[(size_t)t * H + h]);
        const double beta = (double)j->beta[(size_t)t * H + h];

        /* pred = S^T k_t  (prediction of v_t from the previous state) */
        for (int32_t c = 0; c < dv; ++c) pred[c] = 0.0;
        for (int32_t r = 0; r < dk; ++r) {
            const double kr = (double)kt[r];
            const double *Sr = S + (size_t)r * dv;
            for (int32_t c = 0; c < dv; ++c) pred[c] += Sr[c] * kr;
        }
        if (j->variant == 1)
            for (int32_t c = 0; c < dv; ++c) pred[c] *= alpha;

        /* u = beta (v_t - pred);  S = alpha S + k_t u^T */
        for (int32_t c = 0; c < dv; ++c) pred[c] = beta * ((double)vt[c] - pred[c]);
        for (int32_t r = 0; r < dk; ++r) {
            const double kr = (double)kt[r];
            double *Sr = S + (size_t)r * dv;
            for (int32_t c = 0; c < dv; ++c) Sr[c] = alpha * Sr[c] + kr * pred[c];
        }

        /* o_t = scale * S^T q_t  (read-out of the updated state) */
        if (j->o) {
            double *ot = j->o + ((size_t)t * H + h) * dv;
            for (int32_t c = 0; c < dv; ++c) ot[c] = 0.0;
            for (int32_t r = 0; r < dk; ++r) {
                const double qr = (double)qt[r];
                const double *Sr = S + (size_t)r * dv;
                for (int32_t c = 0; c < dv; ++c) ot[c] += Sr[c] * qr;
            }
            for (int32_t c = 0; c < dv; ++c) ot[c] *= j->scale;
        }

        /* checkpoint: the state now represents prefix [0, start + t + 1) */
        const int64_t len = j->start + t + 1;
        if (j->ckpt && j->C > 0 && len % j->C == 0) {
            const int64_t row = len / j->C - j->start / j->C - 1;
            memcpy(j->ckpt + ((size_t)row * H + h) * state_elems, S,
                   state_elems * sizeof(double));
        }
    }
    if (j->state_out)
        memcpy(j->state_out + (size_t)h * state_elems, S, state_elems * sizeof(double));
}

static void *run_heads(void *arg)
{
    const oracle_job *j = (const oracle_job *)arg;
    for (int32_t h = j->head_begin; h < j->head_end; ++h) run_head(j, h, j->S, j->pred);
    return NULL;
}

/*
 * Returns 0 on success, -1 on invalid arguments, -2 on allocation failure.
 * n_threads <= 0 means one thread per head.  The number of threads actually
 * used (min(n_threads, H)) is written to *threads_used when non-NULL.
 */
int oracle_gdr_prefill(int64_t T, int32_t H, int32_t dk, int32_t dv,
                       int32_t variant, double scale,
                       const float *q, const float *k, const float *v,
                       const float *g, const float *beta,
                       int64_t start, int64_t C, const double *state_in,
                       double *o, double *state_out, double *ckpt,
                       int32_t n_threads, int32_t *threads_used)
{
    if (T < 0 || H <= 0 || dk <= 0 || dv <= 0 || start < 0 || C < 0 ||
        (variant != 0 && variant != 1))
        return -1;
    if (n_threads <= 0 || n_threads > H) n_threads = H;
    if (threads_used) *threads_used = n_threads;

    oracle_job *jobs = (oracle_job *)calloc((size_t)n_threads, sizeof(oracle_job));
    pthread_t *tids = (pthread_t *)calloc((size_t)n_threads, sizeof(pthread_t));
    if (!jobs || !tids) { free(jobs); free(tids); return -2; }

    for (int32_t i = 0; i < n_threads; ++i) {
        oracle_job *j = &jobs[i];
        j->T = T; j->H = H; j->dk = dk; j->dv = dv; j->variant = variant;
        j->scale = scale; j->q = q; j->k = k; j->v = v; j->g = g; j->beta = beta;
        j->start = start; j->C = C; j->state_in = state_in;
        j->o = o; j->state_out = state_out; j->ckpt = ckpt;
        j->head_begin = (int32_t)((int64_t)H * i / n_threads);
        j->head_end = (int32_t)((int64_t)H * (i + 1) / n_threads);
        j->S = (double *)malloc((size_t)dk * dv * sizeof(double));
        j->pred = (double *)malloc((size_t)dv * sizeof(double));
    }
    int rc = 0;
    for (int32_t i = 0; i < n_threads; ++i)
        if (!jobs[i].S || !jobs[i].pred) rc = -2;
    if (rc != 0) goto done;
    if (n_threads == 1) {
        run_heads(&jobs[0]);
    } else {
        int32_t started = 0;
        for (; started < n_threads; ++started)
            if (pthread_create(&tids[started], NULL, run_heads, &jobs[started]) != 0) break;
        for (int32_t i = 0; i < started; ++i) pthread_join(tids[i], NULL);
        for (int32_t i = started; i < n_threads; ++i) run_heads(&jobs[i]);
    }
done:
    for (int32_t i = 0; i < n_threads; ++i) { free(jobs[i].S); free(jobs[i].pred); }
    free(jobs);
    free(tids);
    return rc;
}
