/*
 * CPU oracle for the key-only gated linear attention forward pass.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do. It shares no code, header or constant with the HIP path.
 *
 * What it computes (paper, Sec. 3.1 "Key-only gated recurrence"): for one head,
 * with the tokens visited in scan order,
 *
 *     S_t = Diag(gamma_t) S_{t-1} + k_t^T v_t,      o_t = scale * q_t S_t,
 *
 * where gamma_t = exp(g_t) is the per-key-dimension retention gate
 * (g_t = log gamma_t is the log-decay the chunkwise operator consumes,
 * Sec. 3.3 / App. "Custom CUDA Operator"), S_t is d_k x d_v, and each gate entry
 * scales one row of S_{t-1}. The paper fixes S_0 = 0 and scale = d_k^{-1/2};
 * here S_0 and scale are inputs (a zero S_0 and d_k^{-1/2} reproduce the paper).
 * S_final is the state after the last token in scan order.
 *
 * The scan order is an input: order[s] is the spatial index of the token visited
 * at scan position s (Sec. 3.1 "Directional scanning"). Outputs are written at
 * the token's spatial index, so the result is already in spatial order.
 *
 * Everything is float64 and strictly sequential over tokens, one token at a time,
 * exactly as the recurrence is written. Independent (batch, head) sequences run
 * on separate threads; that changes nothing about any sequence's arithmetic.
 */
#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    const double *q, *k, *v, *g, *s0;
    double *o, *s_final;
    long BH, L;
    int dk, dv;
    double scale;
    const long *order;
    int tid, nthreads;
    int status;
} job_t;

/* One (batch, head) sequence. S is caller-provided scratch of dk*dv doubles. */
static void run_sequence(const job_t *jb, long bh, double *S)
{
    const int dk = jb->dk, dv = jb->dv;
    const long L = jb->L;
    const double *q = jb->q + bh * L * dk;
    const double *k = jb->k + bh * L * dk;
    const double *v = jb->v + bh * L * dv;
    const double *g = jb->g + bh * L * dk;
    double *o = jb->o + bh * L * dv;

    if (jb->s0)
        memcpy(S, jb->s0 + bh * (long)dk * dv, sizeof(double) * (size_t)dk * dv);
    else
        memset(S, 0, sizeof(double) * (size_t)dk * dv);

    for (long s = 0; s < L; ++s) {
        const long t = jb->order[s];
        const double *qt = q + t * dk, *kt = k + t * dk, *gt = g + t * dk;
        const double *vt = v + t * dv;
        double *ot = o + t * dv;

        /* S <- Diag(exp(g_t)) S + k_t^T v_t */
        for (int i = 0; i < dk; ++i) {
            const double gamma = exp(gt[i]);
            double *row = S + (long)i * dv;
            for (int j = 0; j < dv; ++j)
                row[j] = gamma * row[j] + kt[i] * vt[j];
        }
        /* o_t <- scale * q_t S */
        for (int j = 0; j < dv; ++j)
            ot[j] = 0.0;
        for (int i = 0; i < dk; ++i) {
            const double *row = S + (long)i * dv;
            for (int j = 0; j < dv; ++j)
                ot[j] += qt[i] * row[j];
        }
        for (int j = 0; j < dv; ++j)
            ot[j] *= jb->scale;
    }
    if (jb->s_final)
        memcpy(jb->s_final + bh * (long)dk * dv, S, sizeof(double) * (size_t)dk * dv);
}

static void *worker(void *arg)
{
    job_t *jb = (job_t *)arg;
    double *S = (double *)malloc(sizeof(double) * (size_t)jb->dk * jb->dv);
    if (!S) {
        jb->status = 1;
        return NULL;
    }
    for (long bh = jb->tid; bh < jb->BH; bh += jb->nthreads)
        run_sequence(jb, bh, S);
    free(S);
    jb->status = 0;
    return NULL;
}

/*
 * q, k, g: [BH, L, dk]; v: [BH, L, dv]; s0: [BH, dk, dv] or NULL;
 * o: [BH, L, dv]; s_final: [BH, dk, dv] or NULL; order: [L] (a permutation).
 * Returns 0 on success, nonzero on allocation or thread failure.
 */
int oracle_gla_forward(const double *q, const double *k, const double *v, const double *g,
                       const double *s0, double *o, double *s_final, long BH, long L,
                       int dk, int dv, double scale, const long *order, int nthreads)
{
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > BH)
        nthreads = (int)(BH > 0 ? BH : 1);
    job_t *jobs = (job_t *)calloc((size_t)nthreads, sizeof(job_t));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !th) {
        free(jobs);
        free(th);
        return 1;
    }
    int rc = 0;
    for (int t = 0; t < nthreads; ++t) {
        job_t j = {q, k, v, g, s0, o, s_final, BH, L, dk, dv, scale, order, t, nthreads, 0};
        jobs[t] = j;
    }
    if (nthreads == 1) {
        worker(&jobs[0]);
        rc = jobs[0].status;
    } else {
        int started = 0;
        for (int t = 0; t < nthreads; ++t) {
            if (pthread_create(&th[t], NULL, worker, &jobs[t]) != 0) {
                rc = 2;
                break;
            }
            ++started;
        }
        for (int t = 0; t < started; ++t)
            pthread_join(th[t], NULL);
        for (int t = 0; t < started; ++t)
            rc |= jobs[t].status;
    }
    free(jobs);
    free(th);
    return rc;
}
