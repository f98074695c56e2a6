/*
 * Murmur decode-step attention oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU statement of what the decode hot path computes:
 *   (1) the retained KV set of each sequence at output step j, built by running
 *       the paper's eviction procedures literally (Section 3.2: Algorithm 1 for
 *       output tokens, Algorithm 2 and Equation 2 for speech tokens);
 *   (2) softmax attention of the current generation token over exactly that set
 *       (Section 3.2, Equation 1), with its log-sum-exp normaliser.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  It shares no code, header or helper with the GPU path and
 * includes nothing from it.  Every floating-point step is fp64; bf16 inputs are
 * widened exactly (bf16 bits << 16 is the fp32 bit pattern).
 *
 * Readings taken where the paper is silent or inconsistent (listed in the
 * design notes of the repository):
 *   - speech window width is w tokens (Algorithm 2), not w+1 (Equation 2);
 *   - the speech window start l advances before the set is formed whenever
 *     j >= d (Algorithm 2), and is clamped so the window ends at the last
 *     speech token;
 *   - speech sinks are Equation 2's first n_sink speech tokens;
 *   - Algorithm 1 is applied to the output region only, with 1-based output
 *     indices, j counting the current token;
 *   - both system prompts are always kept;
 *   - query head h reads KV head h / (Hq / Hkv).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Layout record of one sequence: [prompt_pre][speech][prompt_mid][output]. */
enum { SEG_PRE = 0, SEG_SPEECH = 1, SEG_MID = 2, SEG_OUT = 3, SEG_FIELDS = 4 };
/* Policy record: speech window, speech delay, speech sinks, output window,
 * output sinks.  A window of -1 disables eviction for that region. */
enum { POL_WS = 0, POL_D = 1, POL_NSS = 2, POL_WO = 3, POL_NSO = 4, POL_FIELDS = 5 };

int oracle_abi_version(void) { return 1; }

/* Algorithm 2, run literally: l starts at 0 and, at every decode step
 * jj = 1..j, is incremented when jj >= d, before the kept set is formed. */
static int64_t speech_window_start(int64_t j, int64_t d) {
    int64_t l = 0;
    for (int64_t jj = 1; jj <= j; ++jj) {
        if (jj >= d) l += 1;
    }
    return l;
}

/* Marks the retained positions of one sequence in keep[0 .. total).
 * Returns 0, or -1 on an invalid layout or policy. */
static int mark_retained(const int32_t *seg, const int32_t *pol, unsigned char *keep, int64_t total) {
    const int64_t p_pre = seg[SEG_PRE], l_s = seg[SEG_SPEECH], p_mid = seg[SEG_MID], j = seg[SEG_OUT];
    const int64_t w_s = pol[POL_WS], d = pol[POL_D], n_ss = pol[POL_NSS];
    const int64_t w_o = pol[POL_WO], n_so = pol[POL_NSO];
    if (p_pre < 0 || l_s < 0 || p_mid < 0 || j < 1) return -1;
    if (!(w_s == -1 || w_s >= 1) || d < 0 || n_ss < 0) return -1;
    if (!(w_o == -1 || w_o >= 1) || n_so < 0) return -1;
    const int64_t speech0 = p_pre, mid0 = p_pre + l_s, out0 = p_pre + l_s + p_mid;
    if (total != out0 + j) return -1;
    memset(keep, 0, (size_t)total);

    /* Both system prompts are kept at every step. */
    for (int64_t i = 0; i < p_pre; ++i) keep[i] = 1;
    for (int64_t i = 0; i < p_mid; ++i) keep[mid0 + i] = 1;

    /* Speech tokens (Algorithm 2 window united with Equation 2's sinks). */
    if (w_s == -1 || w_s >= l_s) {
        for (int64_t i = 0; i < l_s; ++i) keep[speech0 + i] = 1;
    } else {
        int64_t l = speech_window_start(j, d);
        if (l > l_s - w_s) l = l_s - w_s; /* window stays inside the speech region */
        for (int64_t i = l; i <= l + w_s - 1; ++i) keep[speech0 + i] = 1;
        for (int64_t i = 0; i < n_ss && i < l_s; ++i) keep[speech0 + i] = 1;
    }

    /* Output tokens (Algorithm 1), 1-based indices 1..j within the output region. */
    if (w_o == -1 || w_o >= j) {
        for (int64_t i = 1; i <= j; ++i) keep[out0 + i - 1] = 1;
    } else {
        for (int64_t i = 1; i <= n_so && i <= j; ++i) keep[out0 + i - 1] = 1;
        int64_t lo = j - w_o + 1;
        if (lo < 1) lo = 1;
        for (int64_t i = lo; i <= j; ++i) keep[out0 + i - 1] = 1;
    }
    return 0;
}

/* Retained-position lists for B sequences, ascending, padded with -1.
 * seg: [B][4]; pol: [B][5] if pol_per_seq else [1][5]; idx: [B][max_keep];
 * count: [B].  Returns 0; -1 on invalid input; -2 if some count exceeds
 * max_keep (count is still written, idx holds the first max_keep entries). */
int oracle_retained(const int32_t *seg, const int32_t *pol, int32_t pol_per_seq, int32_t B,
                    int32_t *idx, int32_t max_keep, int32_t *count) {
    if (B < 0 || max_keep < 0 || !seg || !pol || !count || (max_keep > 0 && !idx)) return -1;
    int status = 0;
    for (int32_t b = 0; b < B; ++b) {
        const int32_t *sg = seg + (int64_t)b * SEG_FIELDS;
        const int32_t *pl = pol + (pol_per_seq ? (int64_t)b * POL_FIELDS : 0);
        for (int32_t r = 0; r < max_keep; ++r) idx[(int64_t)b * max_keep + r] = -1;
        count[b] = 0;
        if (sg[SEG_PRE] < 0 || sg[SEG_SPEECH] < 0 || sg[SEG_MID] < 0 || sg[SEG_OUT] < 1) return -1;
        const int64_t total = (int64_t)sg[SEG_PRE] + sg[SEG_SPEECH] + sg[SEG_MID] + sg[SEG_OUT];
        unsigned char *keep = (unsigned char *)malloc((size_t)total);
        if (!keep) return -1;
        if (mark_retained(sg, pl, keep, total) != 0) {
            free(keep);
            return -1;
        }
        int64_t n = 0;
        for (int64_t i = 0; i < total; ++i) {
            if (!keep[i]) continue;
            if (n < max_keep) idx[(int64_t)b * max_keep + n] = (int32_t)i;
            ++n;
        }
        free(keep);
        count[b] = (int32_t)n;
        if (n > max_keep) status = -2;
    }
    return status;
}

/* ---- attention (Equation 1) ------------------------------------------------ */

static double bf16_to_double(uint16_t bits) {
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

typedef struct {
    const uint16_t *q, *k, *v;
    int32_t NL, B, Hq, Hkv, D, Lmax, max_keep;
    const int32_t *idx, *count;
    double scale;
    double *out, *lse;
    int32_t n_threads, thread_id;
    int status;
} attn_job;

/* One (layer, sequence, query head): softmax over the retained set R of the
 * scaled logits s_i = scale * q . k_i, then out = sum_i softmax_i * v_i and
 * lse = log sum_i exp(s_i). */
static int attend_one(const attn_job *a, int64_t layer, int64_t b, int64_t h) {
    const int64_t D = a->D, Lmax = a->Lmax;
    const int64_t group = a->Hq / a->Hkv;
    const int64_t g = h / group;
    const uint16_t *q = a->q + ((layer * a->B + b) * a->Hq + h) * D;
    const uint16_t *kb = a->k + ((layer * a->B + b) * a->Hkv + g) * Lmax * D;
    const uint16_t *vb = a->v + ((layer * a->B + b) * a->Hkv + g) * Lmax * D;
    const int32_t *R = a->idx + b * a->max_keep;
    const int64_t n = a->count[b];
    double *o = a->out + ((layer * a->B + b) * a->Hq + h) * D;
    double *lse = a->lse + (layer * a->B + b) * a->Hq + h;
    if (n < 1 || n > a->max_keep) return -1;

    double *s = (double *)malloc((size_t)n * sizeof(double));
    if (!s) return -1;
    for (int64_t t = 0; t < n; ++t) {
        const int64_t i = R[t];
        if (i < 0 || i >= Lmax) {
            free(s);
            return -1;
        }
        double dot = 0.0;
        for (int64_t e = 0; e < D; ++e) dot += bf16_to_double(q[e]) * bf16_to_double(kb[i * D + e]);
        s[t] = a->scale * dot;
    }
    double m = s[0];
    for (int64_t t = 1; t < n; ++t)
        if (s[t] > m) m = s[t];
    double z = 0.0;
    for (int64_t t = 0; t < n; ++t) {
        s[t] = exp(s[t] - m); /* unnormalised weight */
        z += s[t];
    }
    double wsum = 0.0;
    for (int64_t e = 0; e < D; ++e) o[e] = 0.0;
    for (int64_t t = 0; t < n; ++t) {
        const double w = s[t] / z;
        wsum += w;
        const int64_t i = R[t];
        for (int64_t e = 0; e < D; ++e) o[e] += w * bf16_to_double(vb[i * D + e]);
    }
    *lse = m + log(z);
    free(s);
    /* The weights of a softmax sum to one. */
    if (fabs(wsum - 1.0) > 1e-12) return -3;
    return 0;
}

static void *attn_worker(void *arg) {
    attn_job *a = (attn_job *)arg;
    const int64_t n_tasks = (int64_t)a->NL * a->B * a->Hq;
    for (int64_t t = a->thread_id; t < n_tasks; t += a->n_threads) {
        const int64_t h = t % a->Hq, b = (t / a->Hq) % a->B, layer = t / ((int64_t)a->Hq * a->B);
        const int rc = attend_one(a, layer, b, h);
        if (rc != 0 && a->status == 0) a->status = rc;
    }
    return NULL;
}

/* q: [NL][B][Hq][D]; k, v: [NL][B][Hkv][Lmax][D] (bf16 bits, contiguous);
 * idx: [B][max_keep] retained positions (shared by all layers and heads);
 * count: [B]; out: [NL][B][Hq][D] fp64; lse: [NL][B][Hq] fp64.
 * Tasks (layer, b, h) are spread over n_threads POSIX threads; each task is
 * computed exactly as stated above, independent of the thread count.
 * Returns 0; -1 on invalid input; -3 if a softmax failed to normalise. */
int oracle_attn(const uint16_t *q, const uint16_t *k, const uint16_t *v, int32_t NL, int32_t B, int32_t Hq,
                int32_t Hkv, int32_t D, int32_t Lmax, const int32_t *idx, const int32_t *count,
                int32_t max_keep, double scale, double *out, double *lse, int32_t n_threads) {
    if (!q || !k || !v || !idx || !count || !out || !lse) return -1;
    if (NL < 1 || B < 1 || Hq < 1 || Hkv < 1 || D < 1 || Lmax < 1 || max_keep < 1) return -1;
    if (Hq % Hkv != 0) return -1;
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    attn_job jobs[256];
    pthread_t tids[256];
    for (int32_t t = 0; t < n_threads; ++t) {
        attn_job a = {q, k, v, NL, B, Hq, Hkv, D, Lmax, max_keep, idx, count, scale, out, lse, n_threads, t, 0};
        jobs[t] = a;
    }
    int started = 0;
    for (int32_t t = 1; t < n_threads; ++t) {
        if (pthread_create(&tids[t], NULL, attn_worker, &jobs[t]) != 0) break;
        started = t;
    }
    /* Threads that could not be started are run on the calling thread. */
    for (int32_t t = started + 1; t < n_threads; ++t) attn_worker(&jobs[t]);
    attn_worker(&jobs[0]);
    for (int32_t t = 1; t <= started; ++t) pthread_join(tids[t], NULL);
    for (int32_t t = 0; t < n_threads; ++t)
        if (jobs[t].status != 0) return jobs[t].status;
    return 0;
}
