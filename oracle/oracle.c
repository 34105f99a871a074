/*
 * Test infrastructure, not product code: a plain CPU oracle for the batched
 * backoff n-gram query and the greedy shallow-fusion step.  Only the tests,
 * the smoke check and the CPU-baseline leg of the benchmark load it.  It shares
 * no code, header or table with the GPU library.
 *
 * What it computes, from the definitions and not from any trie layout:
 *
 *   score(c, v)  ARPA backoff rule (Section 2.1): if the n-gram c+(v) is listed,
 *                its weight W(c v); otherwise B(c) + score(c[1:], v), with
 *                B(c) = 0 for a context that is not listed, and the <unk>
 *                weight when even the unigram (v) is missing.  Two results
 *                are returned: the sum in double (the value of the definition
 *                for the fp32 inputs), and the fp32 sum taken in the order of
 *                the paper's Algorithm 1 (an accumulator that starts at 0 and
 *                adds each backoff weight from the query state downward, and
 *                one final add of the found weight).  Rounding decisions
 *                (argmax) use the fp32 value.
 *   next(c, v)   the state of the longest suffix of c+(v) that is a state
 *                (Section 2.1, graph representation: states are contexts,
 *                i.e. listed n-grams of order < N plus the empty context;
 *                highest-order arcs lead to the (N-1)-suffix state).
 *   state ids    0 is the empty context; the others are numbered by
 *                (order, token tuple in lexicographic order).  This is the
 *                order of arcs sorted by (from_state, token) in Section 2.2.
 *   greedy step  Section 2.3: plain fusion takes argmax_v of
 *                fmaf(lambda, lm(v), asr(v)); CTC first takes the plain ASR
 *                argmax over V+1 classes (blank = V) and keeps blank or the
 *                previous label unchanged without rescoring, otherwise it
 *                takes the fused argmax over the other tokens (not blank, not
 *                the previous label) and advances; the transducer mode keeps
 *                blank, otherwise takes the fused argmax over all V tokens;
 *                the AED mode adds class V = <eos>, scored with the LM's
 *                </s> weight of the state, and keeps the state when it wins.
 *                Ties go to the lowest index (strict '>' scan).
 *   repair       a list that is not closed (a pruned model) is closed by
 *                adding every missing prefix and suffix with backoff 0 and,
 *                as weight, score(c, v) on the list without the added n-gram,
 *                so that every history keeps its scores.
 *
 * Parity pins (no external implementation exists): hand-derived values on the
 * Figure 1 sentence, brute-force history recursion on tiny models (and on
 * pruned lists against the repaired ones), per-context normalisation of
 * generated models, and the N=1 / N=2 / lambda=0 reductions.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared -pthread (no fused multiply-add
 * is formed anywhere except the explicit fmaf of the fusion rule).
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_MAX_ORDER 10

enum {
    OR_OK = 0,
    OR_BAD_ARG = -1,
    OR_TOKEN = -2,
    OR_ORDER = -3,
    OR_DUP = -4,
    OR_NO_UNK = -7,
    OR_NOMEM = -20,
    OR_BAD_STATE = -12,
};

typedef struct {
    int32_t V, N;
    int64_t M;
    int32_t *ord;   /* [M] */
    int32_t *tok;   /* [M*N], row i uses its first ord[i] tokens */
    float *W, *B;   /* [M] */
    float unk;
    int has_unk;
    int64_t cap;    /* hash capacity (power of two) */
    int64_t *slot;  /* row index or -1 */
    int64_t S;
    int64_t *state_row; /* [S], state_row[0] = -1 (empty context) */
    int64_t *row_state; /* [M], -1 for n-grams that are no context */
    int special;        /* token V is <s>, token V + 1 is </s> */
} oracle_model;

static char g_err[256];
static const char *set_err(const char *msg) {
    snprintf(g_err, sizeof g_err, "%s", msg);
    return g_err;
}
const char *oracle_last_error(void) { return g_err; }

static uint64_t hash_tuple(const int32_t *t, int k) {
    uint64_t h = 1469598103934665603ull ^ (uint64_t)k;
    for (int i = 0; i < k; ++i) {
        h ^= (uint64_t)(uint32_t)t[i];
        h *= 1099511628211ull;
        h ^= h >> 29;
    }
    return h;
}

static int same_tuple(const oracle_model *m, int64_t row, const int32_t *t, int k) {
    if (m->ord[row] != k) return 0;
    return memcmp(m->tok + row * m->N, t, (size_t)k * sizeof(int32_t)) == 0;
}

/* Row of the listed n-gram t[0..k-1], or -1. */
static int64_t lookup(const oracle_model *m, const int32_t *t, int k) {
    uint64_t mask = (uint64_t)m->cap - 1;
    uint64_t i = hash_tuple(t, k) & mask;
    for (;;) {
        int64_t r = m->slot[i];
        if (r < 0) return -1;
        if (same_tuple(m, r, t, k)) return r;
        i = (i + 1) & mask;
    }
}

static int cmp_state(const void *a, const void *b, void *ctx) {
    const oracle_model *m = (const oracle_model *)ctx;
    int64_t ra = *(const int64_t *)a, rb = *(const int64_t *)b;
    if (m->ord[ra] != m->ord[rb]) return m->ord[ra] < m->ord[rb] ? -1 : 1;
    const int32_t *ta = m->tok + ra * m->N, *tb = m->tok + rb * m->N;
    for (int i = 0; i < m->ord[ra]; ++i)
        if (ta[i] != tb[i]) return ta[i] < tb[i] ? -1 : 1;
    return 0;
}

void oracle_free(oracle_model *m) {
    if (!m) return;
    free(m->ord); free(m->tok); free(m->W); free(m->B);
    free(m->slot); free(m->state_row); free(m->row_state);
    free(m);
}

/* flags & 1: the list uses token V for <s> and V + 1 for </s>.  A context
 * (state) is a listed n-gram of order < N that does not end in </s>. */
int oracle_create(int32_t V, int32_t N, int64_t M, const int32_t *order, const int32_t *tokens,
                  const float *logprob, const float *backoff, float unk_logprob, int flags,
                  oracle_model **out) {
    *out = NULL;
    if (V <= 0 || N < 1 || N > ORACLE_MAX_ORDER || M < 0) { set_err("bad sizes"); return OR_BAD_ARG; }
    oracle_model *m = (oracle_model *)calloc(1, sizeof *m);
    if (!m) return OR_NOMEM;
    m->V = V; m->N = N; m->M = M;
    m->special = flags & 1;
    m->unk = unk_logprob;
    m->has_unk = !isnan(unk_logprob);
    m->ord = (int32_t *)malloc(sizeof(int32_t) * (size_t)(M ? M : 1));
    m->tok = (int32_t *)malloc(sizeof(int32_t) * (size_t)(M ? M : 1) * (size_t)N);
    m->W = (float *)malloc(sizeof(float) * (size_t)(M ? M : 1));
    m->B = (float *)malloc(sizeof(float) * (size_t)(M ? M : 1));
    m->cap = 16;
    while (m->cap < 2 * M + 16) m->cap <<= 1;
    m->slot = (int64_t *)malloc(sizeof(int64_t) * (size_t)m->cap);
    m->row_state = (int64_t *)malloc(sizeof(int64_t) * (size_t)(M ? M : 1));
    if (!m->ord || !m->tok || !m->W || !m->B || !m->slot || !m->row_state) {
        oracle_free(m); set_err("out of memory"); return OR_NOMEM;
    }
    memcpy(m->ord, order, sizeof(int32_t) * (size_t)M);
    memcpy(m->tok, tokens, sizeof(int32_t) * (size_t)M * (size_t)N);
    memcpy(m->W, logprob, sizeof(float) * (size_t)M);
    memcpy(m->B, backoff, sizeof(float) * (size_t)M);
    memset(m->slot, 0xff, sizeof(int64_t) * (size_t)m->cap);

    int64_t n_states = 1;
    for (int64_t r = 0; r < M; ++r) {
        int k = m->ord[r];
        if (k < 1 || k > N) { oracle_free(m); set_err("order out of range"); return OR_ORDER; }
        const int32_t *t = m->tok + r * N;
        const int32_t vt = m->special ? V + 2 : V;
        for (int i = 0; i < k; ++i)
            if (t[i] < 0 || t[i] >= vt) { oracle_free(m); set_err("token out of range"); return OR_TOKEN; }
        uint64_t mask = (uint64_t)m->cap - 1, i = hash_tuple(t, k) & mask;
        while (m->slot[i] >= 0) {
            if (same_tuple(m, m->slot[i], t, k)) { oracle_free(m); set_err("duplicate n-gram"); return OR_DUP; }
            i = (i + 1) & mask;
        }
        m->slot[i] = r;
        if (k < N && !(m->special && t[k - 1] == V + 1)) ++n_states;
    }
    if (!m->has_unk) {
        for (int32_t v = 0; v < V; ++v)
            if (lookup(m, &v, 1) < 0) { oracle_free(m); set_err("missing unigram and no <unk>"); return OR_NO_UNK; }
    }
    /* canonical state numbering: empty context, then (order, tuple) ascending */
    m->S = n_states;
    m->state_row = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_states);
    if (!m->state_row) { oracle_free(m); return OR_NOMEM; }
    m->state_row[0] = -1;
    int64_t j = 1;
    for (int64_t r = 0; r < M; ++r)
        if (m->ord[r] < N && !(m->special && m->tok[r * N + m->ord[r] - 1] == V + 1)) m->state_row[j++] = r;
    qsort_r(m->state_row + 1, (size_t)(n_states - 1), sizeof(int64_t), cmp_state, m);
    for (int64_t r = 0; r < M; ++r) m->row_state[r] = -1;
    for (int64_t s = 1; s < n_states; ++s) m->row_state[m->state_row[s]] = s;
    *out = m;
    return OR_OK;
}

int64_t oracle_num_states(const oracle_model *m) { return m->S; }

/* Context tuple of state s into out[0..N-2]; returns its length, or -1. */
int oracle_state_context(const oracle_model *m, int64_t s, int32_t *out) {
    if (s < 0 || s >= m->S) return -1;
    if (s == 0) return 0;
    int64_t r = m->state_row[s];
    memcpy(out, m->tok + r * m->N, sizeof(int32_t) * (size_t)m->ord[r]);
    return m->ord[r];
}

/* State id of a context tuple, or -1 if the tuple is not a state. */
int64_t oracle_state_of(const oracle_model *m, const int32_t *ctx, int k) {
    if (k == 0) return 0;
    if (k < 0 || k >= m->N) return -1;
    int64_t r = lookup(m, ctx, k);
    return r < 0 ? -1 : m->row_state[r];
}

/* Longest suffix of g[0..len-1] (at most N-1 tokens) that is a state. */
static int64_t longest_state_suffix(const oracle_model *m, const int32_t *g, int len) {
    int jmax = len < m->N - 1 ? len : m->N - 1;
    for (int j = jmax; j >= 1; --j) {
        int64_t r = lookup(m, g + (len - j), j);
        if (r >= 0 && m->row_state[r] >= 0) return m->row_state[r];
    }
    return 0;
}

/* The backoff rule for context c[0..n-1] and token v. */
static void score_one(const oracle_model *m, const int32_t *c, int n, int32_t v,
                      float *s32, double *s64, int32_t *next) {
    int32_t g[ORACLE_MAX_ORDER + 1];
    float acc32 = 0.0f;
    double acc64 = 0.0;
    for (int k = n; k >= 0; --k) {
        /* g = last k tokens of the context, then v */
        memcpy(g, c + (n - k), sizeof(int32_t) * (size_t)k);
        g[k] = v;
        int64_t r = lookup(m, g, k + 1);
        if (r >= 0) {
            *s32 = acc32 + m->W[r];
            *s64 = acc64 + (double)m->W[r];
            *next = (int32_t)longest_state_suffix(m, g, k + 1);
            return;
        }
        if (k > 0) {
            int64_t rc = lookup(m, c + (n - k), k);
            float b = rc >= 0 ? m->B[rc] : 0.0f;
            acc32 = acc32 + b;
            acc64 = acc64 + (double)b;
        }
    }
    *s32 = acc32 + m->unk;
    *s64 = acc64 + (double)m->unk;
    *next = 0;
}

/* ---- closure repair (the definition behind the library's repair flag) ----
 *
 * A list that is not closed gets every missing prefix and suffix of a listed
 * n-gram (for an n-gram ending in </s>, its prefix) added with backoff 0;
 * added n-grams need their own prefixes and suffixes in turn, so the missing
 * ones are collected from the highest order down.  Each added n-gram c + v
 * then gets as weight the backoff rule's score of v after c on the list
 * without it, computed order by order from 1 up on a model that holds the
 * listed n-grams and the added ones of lower order.  An added unigram gets the
 * <unk> weight. */

typedef struct {
    int64_t n, cap;
    int32_t *ord, *tok;
    float *W, *B;
    char *added;
    int N;
} row_list;

static int rl_push(row_list *l, int k, const int32_t *t, float w, float b, char added) {
    if (l->n == l->cap) {
        int64_t c = l->cap ? 2 * l->cap : 1024;
        int32_t *o = (int32_t *)realloc(l->ord, sizeof(int32_t) * (size_t)c);
        if (o) l->ord = o;
        int32_t *tk = (int32_t *)realloc(l->tok, sizeof(int32_t) * (size_t)c * (size_t)l->N);
        if (tk) l->tok = tk;
        float *w2 = (float *)realloc(l->W, sizeof(float) * (size_t)c);
        if (w2) l->W = w2;
        float *b2 = (float *)realloc(l->B, sizeof(float) * (size_t)c);
        if (b2) l->B = b2;
        char *a2 = (char *)realloc(l->added, (size_t)c);
        if (a2) l->added = a2;
        if (!o || !tk || !w2 || !b2 || !a2) return OR_NOMEM;
        l->cap = c;
    }
    l->ord[l->n] = k;
    for (int i = 0; i < l->N; ++i) l->tok[l->n * l->N + i] = i < k ? t[i] : -1;
    l->W[l->n] = w;
    l->B[l->n] = b;
    l->added[l->n] = added;
    ++l->n;
    return OR_OK;
}

/* A model over the rows of l that are listed, or added with order below kmax. */
static int rl_model(const row_list *l, int32_t V, float unk, int flags, int kmax, oracle_model **m) {
    row_list sub = {0, 0, NULL, NULL, NULL, NULL, NULL, l->N};
    int rc = OR_OK;
    for (int64_t r = 0; r < l->n && rc == OR_OK; ++r)
        if (!l->added[r] || l->ord[r] < kmax)
            rc = rl_push(&sub, l->ord[r], l->tok + r * l->N, l->W[r], l->B[r], 0);
    if (rc == OR_OK) rc = oracle_create(V, l->N, sub.n, sub.ord, sub.tok, sub.W, sub.B, unk, flags, m);
    free(sub.ord); free(sub.tok); free(sub.W); free(sub.B); free(sub.added);
    return rc;
}

static int cmp_tuple_n;
static int cmp_tuple(const void *a, const void *b) {
    return memcmp(a, b, sizeof(int32_t) * (size_t)cmp_tuple_n);
}

int oracle_repair(int32_t V, int32_t N, int64_t M, const int32_t *order, const int32_t *tokens,
                  const float *logprob, const float *backoff, float unk_logprob, int flags,
                  int64_t *M_out, int32_t **order_out, int32_t **tokens_out, float **W_out, float **B_out) {
    if (V <= 0 || N < 1 || N > ORACLE_MAX_ORDER || M < 0) { set_err("bad sizes"); return OR_BAD_ARG; }
    const int special = flags & 1;
    row_list l = {0, 0, NULL, NULL, NULL, NULL, NULL, N};
    int rc = OR_OK;
    for (int64_t r = 0; r < M && rc == OR_OK; ++r)
        rc = rl_push(&l, order[r], tokens + r * N, logprob[r], backoff[r], 0);
    /* collect: prefixes and suffixes of order k, from the top down */
    for (int k = N; k >= 2 && rc == OR_OK; --k) {
        oracle_model *m = NULL;
        rc = rl_model(&l, V, unk_logprob, flags, ORACLE_MAX_ORDER + 1, &m);
        if (rc != OR_OK) break;
        int64_t nc = 0;
        int32_t *cand = (int32_t *)malloc(sizeof(int32_t) * (size_t)(2 * l.n + 1) * (size_t)(k - 1));
        if (!cand) { oracle_free(m); rc = OR_NOMEM; break; }
        for (int64_t r = 0; r < l.n; ++r) {
            if (l.ord[r] != k) continue;
            const int32_t *t = l.tok + r * N;
            memcpy(cand + nc++ * (k - 1), t, sizeof(int32_t) * (size_t)(k - 1));            /* prefix */
            if (!(special && t[k - 1] == V + 1))
                memcpy(cand + nc++ * (k - 1), t + 1, sizeof(int32_t) * (size_t)(k - 1));    /* suffix */
        }
        cmp_tuple_n = k - 1;
        qsort(cand, (size_t)nc, sizeof(int32_t) * (size_t)(k - 1), cmp_tuple);
        for (int64_t i = 0; i < nc && rc == OR_OK; ++i) {
            const int32_t *c = cand + i * (k - 1);
            if (i > 0 && memcmp(c, c - (k - 1), sizeof(int32_t) * (size_t)(k - 1)) == 0) continue;
            if (lookup(m, c, k - 1) < 0) rc = rl_push(&l, k - 1, c, 0.0f, 0.0f, 1);
        }
        free(cand);
        oracle_free(m);
    }
    /* weights: order by order from 1 up, by the backoff rule on the list without them */
    for (int k = 1; k < N && rc == OR_OK; ++k) {
        oracle_model *m = NULL;
        rc = rl_model(&l, V, unk_logprob, flags, k, &m);
        if (rc != OR_OK) break;
        for (int64_t r = 0; r < l.n; ++r) {
            if (!l.added[r] || l.ord[r] != k) continue;
            if (k == 1 && isnan(unk_logprob)) { set_err("repair needs a unigram and no <unk>"); rc = OR_NO_UNK; break; }
            float s32;
            double s64;
            int32_t nx;
            score_one(m, l.tok + r * N, k - 1, l.tok[r * N + k - 1], &s32, &s64, &nx);
            l.W[r] = s32;
        }
        oracle_free(m);
    }
    if (rc != OR_OK) {
        free(l.ord); free(l.tok); free(l.W); free(l.B); free(l.added);
        return rc;
    }
    free(l.added);
    *M_out = l.n;
    *order_out = l.ord;
    *tokens_out = l.tok;
    *W_out = l.W;
    *B_out = l.B;
    return OR_OK;
}

void oracle_free_buffer(void *p) { free(p); }

/* Full row for state s: scores and next states of all V tokens. */
static int score_row(const oracle_model *m, int64_t s, float *s32, double *s64, int32_t *next) {
    int32_t c[ORACLE_MAX_ORDER];
    int n = oracle_state_context(m, s, c);
    if (n < 0) return OR_BAD_STATE;
    double d;
    for (int32_t v = 0; v < m->V; ++v)
        score_one(m, c, n, v, &s32[v], s64 ? &s64[v] : &d, &next[v]);
    return OR_OK;
}

/* The </s> score of each state (Section 2.3, AED: the final weight), from
 * the same rule as any token; needs a model with <s>/</s>. */
int oracle_final(const oracle_model *m, const int32_t *states, int64_t B, float *out) {
    if (!m->special) return OR_BAD_ARG;
    int32_t c[ORACLE_MAX_ORDER], nx;
    double d;
    for (int64_t b = 0; b < B; ++b) {
        int n = oracle_state_context(m, states[b], c);
        if (n < 0) return OR_BAD_STATE;
        score_one(m, c, n, m->V + 1, &out[b], &d, &nx);
    }
    return OR_OK;
}

/* The state of the context <s> (0 without <s>/</s>). */
int64_t oracle_start_state(const oracle_model *m) {
    if (!m->special) return 0;
    int32_t bos = m->V;
    int64_t s = oracle_state_of(m, &bos, 1);
    return s < 0 ? 0 : s;
}

typedef struct {
    const oracle_model *m;
    const int32_t *states;
    int64_t b0, b1;
    float *s32;
    double *s64;
    int32_t *next;
    int rc;
} adv_job;

static void *adv_worker(void *p) {
    adv_job *j = (adv_job *)p;
    int64_t V = j->m->V;
    for (int64_t b = j->b0; b < j->b1; ++b) {
        int rc = score_row(j->m, j->states[b], j->s32 + b * V, j->s64 ? j->s64 + b * V : NULL,
                           j->next + b * V);
        if (rc) j->rc = rc;
    }
    return NULL;
}

static void run_jobs(void *(*fn)(void *), void *jobs, size_t job_size, int nthreads) {
    pthread_t th[256];
    int started = 1;
    for (; started < nthreads; ++started)
        if (pthread_create(&th[started], NULL, fn, (char *)jobs + job_size * (size_t)started) != 0) break;
    for (int t = started; t < nthreads; ++t) fn((char *)jobs + job_size * (size_t)t); /* no thread left */
    fn(jobs);
    for (int t = 1; t < started; ++t) pthread_join(th[t], NULL);
}

static int clamp_threads(int nthreads, int64_t work) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    if (work < nthreads) nthreads = work > 0 ? (int)work : 1;
    return nthreads;
}

/* scores32/next: [B, V]; scores64 may be NULL. */
int oracle_advance(const oracle_model *m, const int32_t *states, int64_t B, float *scores32,
                   double *scores64, int32_t *next, int nthreads) {
    nthreads = clamp_threads(nthreads, B);
    adv_job jobs[256];
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].m = m; jobs[t].states = states;
        jobs[t].b0 = B * t / nthreads; jobs[t].b1 = B * (t + 1) / nthreads;
        jobs[t].s32 = scores32; jobs[t].s64 = scores64; jobs[t].next = next; jobs[t].rc = 0;
    }
    run_jobs(adv_worker, jobs, sizeof(adv_job), nthreads);
    for (int t = 0; t < nthreads; ++t) if (jobs[t].rc) return jobs[t].rc;
    return OR_OK;
}

enum { MODE_PLAIN = 0, MODE_CTC = 1, MODE_TRANSDUCER = 2, MODE_AED = 3 };

/* One greedy step for one hypothesis.  asr has V+1 entries for CTC/transducer
 * (blank = V) and at least V for plain fusion.  Returns the label. */
static int32_t greedy_one(const oracle_model *m, const float *asr, int mode, float lambda,
                          int32_t *state, int32_t *prev, float *lm, int32_t *nx) {
    int32_t V = m->V;
    if (mode == MODE_CTC || mode == MODE_TRANSDUCER) {
        int32_t a = 0;
        for (int32_t v = 1; v <= V; ++v)
            if (asr[v] > asr[a]) a = v;
        if (a == V || (mode == MODE_CTC && a == *prev)) {
            if (mode == MODE_CTC) *prev = a;
            return a;
        }
    }
    score_row(m, *state, lm, NULL, nx);
    int32_t best = -1;
    float bestval = 0.0f;
    for (int32_t v = 0; v < V; ++v) {
        if (mode == MODE_CTC && v == *prev) continue;
        float f = fmaf(lambda, lm[v], asr[v]);
        if (best < 0 || f > bestval) { best = v; bestval = f; }
    }
    if (mode == MODE_AED) {   /* class V is <eos>: the LM's </s> score of the state */
        float fin;
        oracle_final(m, state, 1, &fin);
        float f = fmaf(lambda, fin, asr[V]);
        if (f > bestval) return V;   /* sentence ends: the state stays */
    }
    *state = nx[best];
    if (mode == MODE_CTC) *prev = best;
    return best;
}

/* One fused step over B hypotheses (in-place states/prev). */
int oracle_greedy_step(const oracle_model *m, const float *asr, int64_t B, int64_t ld, int mode,
                       float lambda, int32_t *states, int32_t *prev, int32_t *tokens_out) {
    if (mode < 0 || mode > 3 || (mode == MODE_AED && !m->special)) return OR_BAD_ARG;
    float *lm = (float *)malloc(sizeof(float) * (size_t)m->V);
    int32_t *nx = (int32_t *)malloc(sizeof(int32_t) * (size_t)m->V);
    if (!lm || !nx) { free(lm); free(nx); return OR_NOMEM; }
    int rc = OR_OK;
    for (int64_t b = 0; b < B; ++b) {
        if (states[b] < 0 || states[b] >= m->S) { rc = OR_BAD_STATE; break; }
        int32_t p = prev ? prev[b] : 0;
        tokens_out[b] = greedy_one(m, asr + b * ld, mode, lambda, &states[b], &p, lm, nx);
        if (prev) prev[b] = p;
    }
    free(lm); free(nx);
    return rc;
}

/* The k best fused scores fmaf(lambda, lm(v), asr(v)) over v < V of each
 * hypothesis, in descending order, ties to the lower index (a selection sort
 * over the definition's row); states are not changed. */
int oracle_fused_topk(const oracle_model *m, const float *asr, int64_t B, int64_t ld, float lambda, int k,
                      const int32_t *states, int32_t *tokens, float *scores, int32_t *next) {
    if (k < 1 || k > m->V) return OR_BAD_ARG;
    int32_t V = m->V;
    float *lm = (float *)malloc(sizeof(float) * (size_t)V);
    float *f = (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *nx = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    char *taken = (char *)malloc((size_t)V);
    if (!lm || !f || !nx || !taken) { free(lm); free(f); free(nx); free(taken); return OR_NOMEM; }
    int rc = OR_OK;
    for (int64_t b = 0; b < B && rc == OR_OK; ++b) {
        rc = score_row(m, states[b], lm, NULL, nx);
        if (rc) break;
        const float *row = asr + b * ld;
        for (int32_t v = 0; v < V; ++v) { f[v] = fmaf(lambda, lm[v], row[v]); taken[v] = 0; }
        for (int j = 0; j < k; ++j) {
            int32_t best = -1;
            for (int32_t v = 0; v < V; ++v)
                if (!taken[v] && (best < 0 || f[v] > f[best])) best = v;
            taken[best] = 1;
            tokens[b * k + j] = best;
            scores[b * k + j] = f[best];
            next[b * k + j] = nx[best];
        }
    }
    free(lm); free(f); free(nx); free(taken);
    return rc;
}

typedef struct {
    const oracle_model *m;
    const float *asr;
    int64_t T, ld, b0, b1;
    int mode;
    float lambda;
    const int32_t *starts, *lengths, *prev0;
    int32_t *labels, *states_out;
    int rc;
} dec_job;

static void *dec_worker(void *p) {
    dec_job *j = (dec_job *)p;
    const oracle_model *m = j->m;
    float *lm = (float *)malloc(sizeof(float) * (size_t)m->V);
    int32_t *nx = (int32_t *)malloc(sizeof(int32_t) * (size_t)m->V);
    if (!lm || !nx) { free(lm); free(nx); j->rc = OR_NOMEM; return NULL; }
    for (int64_t b = j->b0; b < j->b1; ++b) {
        int32_t s = j->starts ? j->starts[b] : 0, prev = j->prev0 ? j->prev0[b] : m->V;
        if (s < 0 || s >= m->S) { j->rc = OR_BAD_STATE; break; }
        int64_t len = j->lengths ? j->lengths[b] : j->T;
        if (len < 0) len = 0;
        if (len > j->T) len = j->T;
        for (int64_t t = 0; t < j->T; ++t) {
            const float *row = j->asr + (b * j->T + t) * j->ld;
            j->labels[b * j->T + t] = t < len ? greedy_one(m, row, j->mode, j->lambda, &s, &prev, lm, nx) : -1;
            j->states_out[b * j->T + t] = s;
        }
    }
    free(lm); free(nx);
    return NULL;
}

/* Whole greedy decode: asr [B, T, ld]; labels and states after each frame [B, T].
 * Hypothesis b starts at starts[b] (state 0 when starts is NULL) with previous
 * label prev0[b] (blank = V when prev0 is NULL) and runs lengths[b] frames (T
 * when lengths is NULL); later frames get label -1 and keep the state. */
int oracle_decode(const oracle_model *m, const float *asr, int64_t B, int64_t T, int64_t ld, int mode,
                  float lambda, const int32_t *starts, const int32_t *lengths, const int32_t *prev0,
                  int32_t *labels, int32_t *states_out, int nthreads) {
    if (mode < 0 || mode > 3 || (mode == MODE_AED && !m->special)) return OR_BAD_ARG;
    nthreads = clamp_threads(nthreads, B);
    dec_job jobs[256];
    for (int t = 0; t < nthreads; ++t) {
        dec_job d = {m, asr, T, ld, B * t / nthreads, B * (t + 1) / nthreads, mode, lambda, starts, lengths,
                     prev0, labels, states_out, 0};
        jobs[t] = d;
    }
    run_jobs(dec_worker, jobs, sizeof(dec_job), nthreads);
    for (int t = 0; t < nthreads; ++t) if (jobs[t].rc) return jobs[t].rc;
    return OR_OK;
}
