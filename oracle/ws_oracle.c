/*
 * ws_oracle.c -- plain fp64 CPU reference for block-causal attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no source with the GPU library.
 *
 * What it computes (Wan-Streamer v0.1, Abstract and Sec. 1 with Fig. 1:
 * the interleaved token stream is coordinated by block-causal attention;
 * Sec. 2.1, Eq. 1: the response of unit k is conditioned on every input of
 * units <= k and every response of units < k; Sec. 2.4: the performer
 * appends each received KV slice to a full-history cache):
 *
 *   a token whose block id is beta_q may see exactly the keys j whose block
 *   id beta_k(j) is <= beta_q, i.e. its own block in both directions and
 *   every earlier block;
 *
 *   optionally, each block ends in a token-causal segment (the thinker's
 *   language and state slots, decoded token by token: Sec. 1, Sec. 2.4;
 *   language tokens are trained by next-token prediction, Sec. 2.1) that
 *   starts at position tau of the block.  Inside such a block the tokens
 *   before tau still see each other in both directions but not the
 *   segment, and a segment token at position i sees the tokens before tau
 *   and the segment tokens at positions <= i.  Earlier blocks stay fully
 *   visible;
 *
 *   o_i   = sum_{j visible} softmax_j(scale * <q_i, k_j>) v_j
 *   lse_i = m_i + ln(sum_{j visible} exp(scale * <q_i, k_j> - m_i)),
 *           m_i = max_{j visible} scale * <q_i, k_j>.
 *
 * Everything is fp64.  bf16 inputs are widened exactly (bit pattern << 16 is
 * the fp32 value, and fp32 -> fp64 is exact).  Dot products are summed
 * sequentially over the head dimension; the mask row is materialised
 * explicitly for every query; masked keys never enter the max or the sums.
 * Grouped-query attention: query head h reads KV head floor(h / G) with
 * G = Hq / Hkv (contiguous groups).
 *
 * Rows are independent, so results do not depend on the thread count.
 *
 * Gradients (wso_prefill_bwd; training uses the same causal format as
 * inference, Sec. 2.3): for an upstream gradient dO of the output, with
 * P_ij the softmax weights above (0 for masked keys),
 *
 *   dP_ij = <dO_i, v_j>,   D_i = sum_j P_ij dP_ij,
 *   dS_ij = P_ij (dP_ij - D_i),
 *   dQ_i  = scale sum_j dS_ij k_j,
 *   dK_j  = scale sum_i dS_ij q_i,   dV_j = sum_i P_ij dO_i,
 *
 * where the sums over i run over every query row (and, with grouped-query
 * attention, every query head) that reads KV head g.
 *
 * Compile-time switch WSO_MUTANT (default 0) plants one deliberate mistake;
 * it exists only so the test suite can show that its pins catch such
 * mistakes.  A normal build never defines it.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef WSO_MUTANT
#define WSO_MUTANT 0
#endif

enum { WSO_F64 = 0, WSO_BF16 = 1 };

/* A 4-d token tensor [B][L][H][d] with the last dimension contiguous;
 * strides are in elements. */
typedef struct {
    const void *base;
    int dtype;
    int64_t sb, st, sh;
} wso_view;

static double wso_load(const wso_view *v, int64_t b, int64_t t, int64_t h, int64_t c)
{
    int64_t idx = b * v->sb + t * v->st + h * v->sh + c;
    if (v->dtype == WSO_F64)
        return ((const double *)v->base)[idx];
    uint16_t bits = ((const uint16_t *)v->base)[idx];
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* Which kind of problem a job describes. */
enum { WSO_PREFILL = 0, WSO_STEP = 1 };

typedef struct {
    int kind;
    int B, Lq, Hq, Hkv, d;
    double scale;
    /* prefill: queries and keys are the same L tokens; offsets [B][nb+1] */
    wso_view q, k, v;
    const int32_t *offsets;
    int nb;
    /* step: keys are cache tokens [0, Lc[b]) followed by the Lq new tokens */
    wso_view kc, vc;
    const int32_t *cache_lens;
    /* start of each block's token-causal segment, or NULL for none.
     * prefill: [B][nb] absolute positions; step: [B] positions within the
     * new block */
    const int32_t *text_starts;
    /* step only: tokens of stream b's new block (<= Lq), or NULL for Lq;
     * tokens past it are padding: never keys */
    const int32_t *new_lens;
    /* row list: nrows triples (b, h, i); NULL means every row */
    const int32_t *rows;
    int64_t nrows;
    /* outputs */
    double *out;   /* all rows: [B][Lq][Hq][d]; row list: [nrows][d] */
    double *lse;   /* all rows: [B][Hq][Lq];   row list: [nrows]; may be NULL */
    double *probs; /* optional, row list only: [nrows][Lk_max] */
    int64_t lk_max;
} wso_job;

/* Block id of token t given the block boundaries off[0..nb]:
 * the n with off[n] <= t < off[n+1]. */
static int wso_block_of(const int32_t *off, int nb, int64_t t)
{
    for (int n = 0; n < nb; ++n) {
#if WSO_MUTANT == 6
        if (off[n] < t && t <= off[n + 1])
            return n;
#else
        if (off[n] <= t && t < off[n + 1])
            return n;
#endif
    }
    return nb; /* past the end: later than every block */
}

/* Number of keys of stream b. */
static int64_t wso_num_keys(const wso_job *J, int b)
{
    if (J->kind == WSO_PREFILL)
        return J->Lq;
    return (int64_t)J->cache_lens[b] + J->Lq;
}

/* Element c of key (or value) j of stream b, KV head g. */
static double wso_key(const wso_job *J, int is_v, int b, int64_t j, int g, int c)
{
    if (J->kind == WSO_PREFILL)
        return wso_load(is_v ? &J->v : &J->k, b, j, g, c);
    int64_t lc = J->cache_lens[b];
    if (j < lc)
        return wso_load(is_v ? &J->vc : &J->kc, b, j, g, c);
    return wso_load(is_v ? &J->v : &J->k, b, j - lc, g, c);
}

/* Mask row of query i of stream b: mask[j] = 1 iff key j is visible, from
 * block ids (and the token-causal segment of the query's block).  Positions
 * are in key order: the query sits at key position iq, its block's segment
 * starts at key position tau (-1: the block has none). */
static void wso_mask_row(const wso_job *J, int b, int64_t i, unsigned char *mask)
{
    const int64_t Lk = wso_num_keys(J, b);
    int beta_q;
    int64_t iq, tau = -1;
    if (J->kind == WSO_PREFILL) {
        beta_q = wso_block_of(J->offsets + (int64_t)b * (J->nb + 1), J->nb, i);
        iq = i;
        if (J->text_starts)
            tau = J->text_starts[(int64_t)b * J->nb + beta_q];
    } else {
        beta_q = 1;
        iq = (int64_t)J->cache_lens[b] + i;
        if (J->text_starts)
            tau = (int64_t)J->cache_lens[b] + J->text_starts[b];
    }
    for (int64_t j = 0; j < Lk; ++j) {
        int beta_k;
        if (J->kind == WSO_PREFILL)
            beta_k = wso_block_of(J->offsets + (int64_t)b * (J->nb + 1), J->nb, j);
        else
            beta_k = (j < J->cache_lens[b]) ? 0 : 1;
#if WSO_MUTANT == 1
        int vis = beta_k < beta_q;
#elif WSO_MUTANT == 8
        int vis = beta_k >= beta_q;
#else
        int vis = beta_k <= beta_q;
#endif
#if WSO_MUTANT == 13
        if (J->kind == WSO_STEP && J->new_lens && j > (int64_t)J->cache_lens[b] + J->new_lens[b])
#else
        if (J->kind == WSO_STEP && J->new_lens && j >= (int64_t)J->cache_lens[b] + J->new_lens[b])
#endif
            vis = 0;   /* padding of the new block */
        if (vis && beta_k == beta_q && tau >= 0) {
            /* same block: a key of the segment is visible only to segment
             * queries at or after it */
#if WSO_MUTANT == 9
            vis = j < tau || j <= iq + 1;
#elif WSO_MUTANT == 10
            vis = j < tau || j <= iq || iq < tau;
#else
            vis = j < tau || j <= iq;
#endif
        }
        mask[j] = (unsigned char)vis;
    }
}

/* Scratch owned by one worker thread. */
typedef struct {
    double *s;
    unsigned char *mask;
    double *acc;
} wso_scratch;

/* One query row: materialise the mask row, then the softmax-weighted sum. */
static void wso_row(const wso_job *J, wso_scratch *S, int b, int h, int64_t i,
                    double *o, double *lse_out, double *p_out)
{
    const int G = J->Hq / J->Hkv;
#if WSO_MUTANT == 3
    const int g = h % J->Hkv;
#else
    const int g = h / G;
#endif
    const int64_t Lk = wso_num_keys(J, b);
    const int d = J->d;

    /* 1. explicit mask row */
    wso_mask_row(J, b, i, S->mask);

    /* 2. logits of visible keys, and their maximum */
    double m = -INFINITY;
    for (int64_t j = 0; j < Lk; ++j) {
        if (!S->mask[j])
            continue;
        double dot = 0.0;
        for (int c = 0; c < d; ++c) {
            double qv = wso_load(&J->q, b, i, h, c);
#if WSO_MUTANT == 4
            double kv = wso_key(J, 0, b, (j + 1) % Lk, g, c);
#else
            double kv = wso_key(J, 0, b, j, g, c);
#endif
            dot += qv * kv;
        }
#if WSO_MUTANT == 2
        S->s[j] = dot;
#else
        S->s[j] = J->scale * dot;
#endif
        if (S->s[j] > m)
            m = S->s[j];
    }

    /* 3. unnormalised weights and their sum */
    double l = 0.0;
    for (int64_t j = 0; j < Lk; ++j) {
        if (!S->mask[j]) {
            S->s[j] = 0.0;
            continue;
        }
        S->s[j] = exp(S->s[j] - m);
        l += S->s[j];
    }

    /* 4. weighted sum of values, normalised */
    for (int c = 0; c < d; ++c)
        S->acc[c] = 0.0;
    for (int64_t j = 0; j < Lk; ++j) {
        if (!S->mask[j])
            continue;
        for (int c = 0; c < d; ++c)
            S->acc[c] += S->s[j] * wso_key(J, 1, b, j, g, c);
    }
    for (int c = 0; c < d; ++c) {
#if WSO_MUTANT == 7
        o[c] = S->acc[c];
#else
        o[c] = S->acc[c] / l;
#endif
    }
    if (lse_out) {
#if WSO_MUTANT == 5
        *lse_out = m;
#else
        *lse_out = m + log(l);
#endif
    }
    if (p_out) {
        for (int64_t j = 0; j < Lk; ++j)
            p_out[j] = S->s[j] / l;
    }
}

typedef struct {
    const wso_job *J;
    int64_t first, last; /* half-open range of row indices */
    int status;
} wso_task;

static void *wso_worker(void *arg)
{
    wso_task *T = (wso_task *)arg;
    const wso_job *J = T->J;
    int64_t lk_cap = J->Lq;
    if (J->kind == WSO_STEP) {
        for (int b = 0; b < J->B; ++b)
            if (wso_num_keys(J, b) > lk_cap)
                lk_cap = wso_num_keys(J, b);
    }
    wso_scratch S;
    S.s = (double *)malloc(sizeof(double) * (size_t)(lk_cap > 0 ? lk_cap : 1));
    S.mask = (unsigned char *)malloc((size_t)(lk_cap > 0 ? lk_cap : 1));
    S.acc = (double *)malloc(sizeof(double) * (size_t)J->d);
    if (!S.s || !S.mask || !S.acc) {
        free(S.s);
        free(S.mask);
        free(S.acc);
        T->status = -1;
        return NULL;
    }
    for (int64_t r = T->first; r < T->last; ++r) {
        int b, h;
        int64_t i;
        double *o, *lse_out, *p_out = NULL;
        if (J->rows) {
            b = J->rows[3 * r + 0];
            h = J->rows[3 * r + 1];
            i = J->rows[3 * r + 2];
            o = J->out + r * J->d;
            lse_out = J->lse ? J->lse + r : NULL;
            if (J->probs)
                p_out = J->probs + r * J->lk_max;
        } else {
            /* r enumerates (b, i, h) in output order */
            h = (int)(r % J->Hq);
            i = (r / J->Hq) % J->Lq;
            b = (int)(r / ((int64_t)J->Hq * J->Lq));
            o = J->out + r * J->d;
            lse_out = J->lse ? J->lse + ((int64_t)b * J->Hq + h) * J->Lq + i : NULL;
        }
        wso_row(J, &S, b, h, i, o, lse_out, p_out);
    }
    free(S.s);
    free(S.mask);
    free(S.acc);
    T->status = 0;
    return NULL;
}

static int wso_run(const wso_job *J, int nthreads)
{
    int64_t total = J->rows ? J->nrows : (int64_t)J->B * J->Lq * J->Hq;
    if (total <= 0)
        return 0;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > total)
        nthreads = (int)total;
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    wso_task *tasks = (wso_task *)calloc((size_t)nthreads, sizeof(wso_task));
    if (!th || !tasks) {
        free(th);
        free(tasks);
        return -1;
    }
    for (int t = 0; t < nthreads; ++t) {
        tasks[t].J = J;
        tasks[t].first = total * t / nthreads;
        tasks[t].last = total * (t + 1) / nthreads;
        tasks[t].status = -1;
    }
    int started = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, wso_worker, &tasks[t]) != 0)
            break;
        started = t;
    }
    wso_worker(&tasks[0]);
    int rc = tasks[0].status;
    for (int t = 1; t <= started; ++t) {
        pthread_join(th[t], NULL);
        if (tasks[t].status != 0)
            rc = -1;
    }
    /* rows of threads that could not be started are done here */
    for (int t = started + 1; t < nthreads; ++t) {
        wso_worker(&tasks[t]);
        if (tasks[t].status != 0)
            rc = -1;
    }
    free(th);
    free(tasks);
    return rc;
}

static int wso_check_common(int B, int Lq, int Hq, int Hkv, int d)
{
    if (B < 0 || Lq < 0 || Hq <= 0 || Hkv <= 0 || d <= 0)
        return -2;
    if (Hq % Hkv != 0)
        return -2;
    return 0;
}

/*
 * Whole-sequence block-causal attention.  q, k, v: [B][L][H][d] contiguous
 * (dtype WSO_F64 or WSO_BF16 bit patterns).  offsets: [B][nb+1] block
 * boundaries, offsets[b][0] = 0, non-decreasing, offsets[b][nb] = L.
 * text_starts: NULL, or [B][nb] start of each block's token-causal segment
 * (offsets[b][n] <= text_starts[b][n] <= offsets[b][n+1]; equal to the
 * block end: no segment).
 * rows: NULL for every row, else nrows triples (b, h, i).  probs (row list
 * only, may be NULL): [nrows][L] normalised attention weights.
 * Returns 0 on success, -2 on bad arguments, -1 on allocation failure.
 */
int wso_prefill_text(const void *q, const void *k, const void *v, int dtype,
                     int B, int L, int Hq, int Hkv, int d,
                     const int32_t *offsets, int nb, const int32_t *text_starts, double scale,
                     const int32_t *rows, int64_t nrows,
                     double *out, double *lse, double *probs, int nthreads)
{
    if (wso_check_common(B, L, Hq, Hkv, d) || nb < 0 || !offsets || !out)
        return -2;
    for (int b = 0; b < B; ++b) {
        const int32_t *off = offsets + (int64_t)b * (nb + 1);
        if (off[0] != 0 || off[nb] != L)
            return -2;
        for (int n = 0; n < nb; ++n) {
            if (off[n + 1] < off[n])
                return -2;
            if (text_starts) {
                const int32_t t = text_starts[(int64_t)b * nb + n];
                if (t < off[n] || t > off[n + 1])
                    return -2;
            }
        }
    }
    wso_job J;
    memset(&J, 0, sizeof J);
    J.kind = WSO_PREFILL;
    J.B = B; J.Lq = L; J.Hq = Hq; J.Hkv = Hkv; J.d = d;
    J.scale = scale;
    J.q = (wso_view){q, dtype, (int64_t)L * Hq * d, (int64_t)Hq * d, d};
    J.k = (wso_view){k, dtype, (int64_t)L * Hkv * d, (int64_t)Hkv * d, d};
    J.v = (wso_view){v, dtype, (int64_t)L * Hkv * d, (int64_t)Hkv * d, d};
    J.offsets = offsets;
    J.nb = nb;
    J.text_starts = text_starts;
    J.rows = rows;
    J.nrows = nrows;
    J.out = out;
    J.lse = lse;
    J.probs = rows ? probs : NULL;
    J.lk_max = L;
    return wso_run(&J, nthreads);
}

/* The same with no token-causal segments (pure block-causal attention). */
int wso_prefill(const void *q, const void *k, const void *v, int dtype,
                int B, int L, int Hq, int Hkv, int d,
                const int32_t *offsets, int nb, double scale,
                const int32_t *rows, int64_t nrows,
                double *out, double *lse, double *probs, int nthreads)
{
    return wso_prefill_text(q, k, v, dtype, B, L, Hq, Hkv, d, offsets, nb, NULL, scale,
                            rows, nrows, out, lse, probs, nthreads);
}

/*
 * One streaming step: the Lq tokens of a new block attend to the cache
 * tokens [0, cache_lens[b]) of their stream (all earlier blocks) and to the
 * whole new block (their own block).  kc, vc: [B][Lc_max][Hkv][d]; q: [B][Lq][Hq][d];
 * kn, vn: [B][Lq][Hkv][d]; all contiguous.  probs rows have length
 * Lc_max + Lq (entries past the stream's own key count are left untouched).
 * text_starts: NULL, or [B] start of the new block's token-causal segment
 * within the block (0 <= text_starts[b] <= Lq; Lq: no segment).
 * new_lens: NULL, or [B] tokens of each stream's new block (1..Lq); the
 * block's tokens past new_lens[b] are padding and never keys (their own
 * rows are computed by the same rule).
 */
int wso_step_varlen(const void *q, const void *kc, const void *vc,
                    const void *kn, const void *vn, int dtype,
                    int B, int Lq, int Lc_max, const int32_t *cache_lens,
                    const int32_t *new_lens, const int32_t *text_starts,
                    int Hq, int Hkv, int d, double scale,
                    const int32_t *rows, int64_t nrows,
                    double *out, double *lse, double *probs, int nthreads)
{
    if (wso_check_common(B, Lq, Hq, Hkv, d) || Lc_max < 0 || !cache_lens || !out)
        return -2;
    for (int b = 0; b < B; ++b) {
        if (cache_lens[b] < 0 || cache_lens[b] > Lc_max)
            return -2;
        if (text_starts && (text_starts[b] < 0 || text_starts[b] > Lq))
            return -2;
        if (new_lens && (new_lens[b] < 1 || new_lens[b] > Lq))
            return -2;
    }
    wso_job J;
    memset(&J, 0, sizeof J);
    J.kind = WSO_STEP;
    J.B = B; J.Lq = Lq; J.Hq = Hq; J.Hkv = Hkv; J.d = d;
    J.scale = scale;
    J.q = (wso_view){q, dtype, (int64_t)Lq * Hq * d, (int64_t)Hq * d, d};
    J.k = (wso_view){kn, dtype, (int64_t)Lq * Hkv * d, (int64_t)Hkv * d, d};
    J.v = (wso_view){vn, dtype, (int64_t)Lq * Hkv * d, (int64_t)Hkv * d, d};
    J.kc = (wso_view){kc, dtype, (int64_t)Lc_max * Hkv * d, (int64_t)Hkv * d, d};
    J.vc = (wso_view){vc, dtype, (int64_t)Lc_max * Hkv * d, (int64_t)Hkv * d, d};
    J.cache_lens = cache_lens;
    J.text_starts = text_starts;
    J.new_lens = new_lens;
    J.rows = rows;
    J.nrows = nrows;
    J.out = out;
    J.lse = lse;
    J.probs = rows ? probs : NULL;
    J.lk_max = (int64_t)Lc_max + Lq;
    return wso_run(&J, nthreads);
}

/* Equal new-block lengths (new_lens = NULL). */
int wso_step_text(const void *q, const void *kc, const void *vc,
                  const void *kn, const void *vn, int dtype,
                  int B, int Lq, int Lc_max, const int32_t *cache_lens,
                  const int32_t *text_starts,
                  int Hq, int Hkv, int d, double scale,
                  const int32_t *rows, int64_t nrows,
                  double *out, double *lse, double *probs, int nthreads)
{
    return wso_step_varlen(q, kc, vc, kn, vn, dtype, B, Lq, Lc_max, cache_lens, NULL, text_starts, Hq, Hkv,
                           d, scale, rows, nrows, out, lse, probs, nthreads);
}

/* The same with no token-causal segment in the new block. */
int wso_step(const void *q, const void *kc, const void *vc,
             const void *kn, const void *vn, int dtype,
             int B, int Lq, int Lc_max, const int32_t *cache_lens,
             int Hq, int Hkv, int d, double scale,
             const int32_t *rows, int64_t nrows,
             double *out, double *lse, double *probs, int nthreads)
{
    return wso_step_text(q, kc, vc, kn, vn, dtype, B, Lq, Lc_max, cache_lens, NULL, Hq, Hkv, d,
                         scale, rows, nrows, out, lse, probs, nthreads);
}

/* ---------------------------------------------------------------------- */
/* Gradients of the whole-sequence path.                                   */

typedef struct {
    const wso_job *J;
    const void *dout;
    double *dq, *dk, *dv;
    int first, last; /* half-open range of (b, g) groups */
    int status;
} wso_bwd_task;

static void *wso_bwd_worker(void *arg)
{
    wso_bwd_task *T = (wso_bwd_task *)arg;
    const wso_job *J = T->J;
    const int d = J->d, G = J->Hq / J->Hkv;
    const int64_t L = J->Lq;
    const wso_view dov = {T->dout, J->q.dtype, J->q.sb, J->q.st, J->q.sh};
    double *p = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
    double *dp = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
    unsigned char *mask = (unsigned char *)malloc((size_t)(L > 0 ? L : 1));
    if (!p || !dp || !mask) {
        free(p);
        free(dp);
        free(mask);
        T->status = -1;
        return NULL;
    }
    for (int grp = T->first; grp < T->last; ++grp) {
        const int b = grp / J->Hkv, g = grp % J->Hkv;
        for (int hh = 0; hh < G; ++hh) {
            const int h = g * G + hh;
            for (int64_t i = 0; i < L; ++i) {
                /* softmax weights of row i over its visible keys */
                wso_mask_row(J, b, i, mask);
                double m = -INFINITY;
                for (int64_t j = 0; j < L; ++j) {
                    if (!mask[j])
                        continue;
                    double dot = 0.0;
                    for (int c = 0; c < d; ++c)
                        dot += wso_load(&J->q, b, i, h, c) * wso_load(&J->k, b, j, g, c);
                    p[j] = J->scale * dot;
                    if (p[j] > m)
                        m = p[j];
                }
                double l = 0.0;
                for (int64_t j = 0; j < L; ++j) {
                    p[j] = mask[j] ? exp(p[j] - m) : 0.0;
                    l += p[j];
                }
                for (int64_t j = 0; j < L; ++j)
                    p[j] /= l;
                /* dP_ij = <dO_i, v_j>, D_i = sum_j P_ij dP_ij */
                double D = 0.0;
                for (int64_t j = 0; j < L; ++j) {
                    dp[j] = 0.0;
                    if (!mask[j])
                        continue;
                    for (int c = 0; c < d; ++c)
                        dp[j] += wso_load(&dov, b, i, h, c) * wso_load(&J->v, b, j, g, c);
#if WSO_MUTANT == 16
                    D += dp[j];
#else
                    D += p[j] * dp[j];
#endif
                }
                /* dS_ij = P_ij (dP_ij - D_i) and the three gradients */
                double *dqi = T->dq + (((int64_t)b * L + i) * J->Hq + h) * d;
                for (int c = 0; c < d; ++c)
                    dqi[c] = 0.0;
                for (int64_t j = 0; j < L; ++j) {
                    if (!mask[j])
                        continue;
#if WSO_MUTANT == 11
                    const double ds = p[j] * dp[j];
#else
                    const double ds = p[j] * (dp[j] - D);
#endif
                    double *dkj = T->dk + (((int64_t)b * L + j) * J->Hkv + g) * d;
                    double *dvj = T->dv + (((int64_t)b * L + j) * J->Hkv + g) * d;
                    for (int c = 0; c < d; ++c) {
#if WSO_MUTANT == 14
                        dqi[c] += J->scale * ds * wso_load(&J->v, b, j, g, c);
#else
                        dqi[c] += J->scale * ds * wso_load(&J->k, b, j, g, c);
#endif
#if WSO_MUTANT == 12
                        dkj[c] += ds * wso_load(&J->q, b, i, h, c);
#else
                        dkj[c] += J->scale * ds * wso_load(&J->q, b, i, h, c);
#endif
#if WSO_MUTANT == 15
                        dvj[c] += p[j] * l * wso_load(&dov, b, i, h, c);
#else
                        dvj[c] += p[j] * wso_load(&dov, b, i, h, c);
#endif
                    }
                }
            }
        }
    }
    free(p);
    free(dp);
    free(mask);
    T->status = 0;
    return NULL;
}

/*
 * Gradients of whole-sequence block-causal attention (with optional
 * token-causal segments, as wso_prefill_text).  q, dout: [B][L][Hq][d];
 * k, v: [B][L][Hkv][d]; all contiguous, dtype WSO_F64 or WSO_BF16.
 * Outputs (fp64, overwritten): dq [B][L][Hq][d], dk and dv [B][L][Hkv][d].
 * Threads split the (stream, KV head) groups, so every gradient sum runs
 * in a fixed order whatever the thread count.
 * Returns 0 on success, -2 on bad arguments, -1 on allocation failure.
 */
int wso_prefill_bwd(const void *q, const void *k, const void *v, const void *dout, int dtype,
                    int B, int L, int Hq, int Hkv, int d,
                    const int32_t *offsets, int nb, const int32_t *text_starts, double scale,
                    double *dq, double *dk, double *dv, int nthreads)
{
    if (wso_check_common(B, L, Hq, Hkv, d) || nb < 0 || !offsets || !dq || !dk || !dv || !dout)
        return -2;
    for (int b = 0; b < B; ++b) {
        const int32_t *off = offsets + (int64_t)b * (nb + 1);
        if (off[0] != 0 || off[nb] != L)
            return -2;
        for (int n = 0; n < nb; ++n) {
            if (off[n + 1] < off[n])
                return -2;
            if (text_starts) {
                const int32_t t = text_starts[(int64_t)b * nb + n];
                if (t < off[n] || t > off[n + 1])
                    return -2;
            }
        }
    }
    wso_job J;
    memset(&J, 0, sizeof J);
    J.kind = WSO_PREFILL;
    J.B = B; J.Lq = L; J.Hq = Hq; J.Hkv = Hkv; J.d = d;
    J.scale = scale;
    J.q = (wso_view){q, dtype, (int64_t)L * Hq * d, (int64_t)Hq * d, d};
    J.k = (wso_view){k, dtype, (int64_t)L * Hkv * d, (int64_t)Hkv * d, d};
    J.v = (wso_view){v, dtype, (int64_t)L * Hkv * d, (int64_t)Hkv * d, d};
    J.offsets = offsets;
    J.nb = nb;
    J.text_starts = text_starts;
    const int64_t nkv = (int64_t)B * L * Hkv * d;
    for (int64_t x = 0; x < nkv; ++x) {
        dk[x] = 0.0;
        dv[x] = 0.0;
    }
    const int groups = B * Hkv;
    if (groups == 0 || L == 0)
        return 0;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > groups)
        nthreads = groups;
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    wso_bwd_task *tasks = (wso_bwd_task *)calloc((size_t)nthreads, sizeof(wso_bwd_task));
    if (!th || !tasks) {
        free(th);
        free(tasks);
        return -1;
    }
    for (int t = 0; t < nthreads; ++t) {
        tasks[t] = (wso_bwd_task){&J, dout, dq, dk, dv, groups * t / nthreads,
                                  groups * (t + 1) / nthreads, -1};
    }
    int started = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, wso_bwd_worker, &tasks[t]) != 0)
            break;
        started = t;
    }
    wso_bwd_worker(&tasks[0]);
    int rc = tasks[0].status;
    for (int t = 1; t <= started; ++t) {
        pthread_join(th[t], NULL);
        if (tasks[t].status != 0)
            rc = -1;
    }
    for (int t = started + 1; t < nthreads; ++t) {
        wso_bwd_worker(&tasks[t]);
        if (tasks[t].status != 0)
            rc = -1;
    }
    free(th);
    free(tasks);
    return rc;
}

int wso_mutant(void) { return WSO_MUTANT; }
