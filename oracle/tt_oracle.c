/*
 * TokenTiming verification hot path -- CPU ORACLE.
 *
 * This file is test infrastructure.  It is a plain, slow, deliberately simple
 * CPU implementation of what the GPU library computes, used only by the tests,
 * by the smoke check and by the benchmark's CPU-baseline leg.  It shares no code,
 * header, table or helper with the GPU library and must never be linked into it.
 *
 * Arithmetic: token distances and warping costs are int; probabilities are fp32
 * (the precision the inputs arrive in and in which the GPU takes every decision
 * that turns floating point into an integer); the sampling arithmetic is exact
 * integer.  Build with -O2 -ffp-contract=off and without fast-math.
 *
 * Sections of the paper followed:
 *   orc_levenshtein   App. H "Token Distance" (initialisation, recurrence, result)
 *   dtw_pair          Sec. 4.1 + Alg. 1 (Dynamic Token Warping, Sakoe-Chiba band,
 *                     backtrack from (k,m) to (0,0))
 *   mapping           App. A.2 Case 1 (terminal draft token) / Case 2 (copy)
 *   transfer          Sec. 4.2.2 / Alg. 2 "MapProbabilities"; App. A.2 draft
 *                     probability of the emitted token; Limitations (one-hot form)
 *   verify            Sec. 3 "Standard Speculative Sampling", Sec. 4.2.2 acceptance
 *                     rule, Sec. 4.2.3 / Alg. 2 bonus sample, App. D Alg. 4
 *                     (residual "modified distribution")
 *   orc_sd_verify     App. D Alg. 4 with dense proposals over one vocabulary (standard
 *                     speculative decoding, the homogeneous-vocabulary case)
 *   orc_delta_histogram  Sec. 5 Fig. CDF / App. K: position deviation |i - j| of the
 *                     matched pairs on the optimal paths
 *   orc_delta_quantile   App. K: the deviation where that distribution reaches a quantile
 *   orc_verify_logits the verification from bf16 logits and a temperature (App. F), the
 *                     target softmax formed with a specified base-2 exponential
 *
 * Readings where the paper is silent or ambiguous (each is listed in the design
 * notes of the repository):
 *   band      |i-j| <= w inclusive as in Alg. 1; w < 0 means no band; when
 *             |k-m| > w the corner (k,m) would be unreachable, so the half-width
 *             used is w_eff = max(w, |k-m|).
 *   ties      backtrack prefers the diagonal predecessor, then (i-1,j), then (i,j-1).
 *   mapping   target position j takes the largest draft index on the path in its
 *             column (the terminal draft token; a copy when one draft token spans
 *             several target tokens).
 *   accept    ratio = P_t / q in fp32 round-to-nearest; accept iff q <= 0 or u < ratio.
 *   residual  rejection at r < M: R = max(0, P_t[r] - q_r e_{t_r}); all accepted:
 *             R = P_t[M] (the bonus row).  R is clamped to [0,1] (NaN -> 0).
 *   sampling  R is quantised to Q62 fixed point by truncation, Z = sum, the
 *             threshold is T = floor(u * Z) computed exactly, and the token is the
 *             first index whose inclusive prefix sum exceeds T.  If Z = 0 the token
 *             is the first maximum of the row.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_INF 0x3fffffff

static int min_int(int a, int b) { return a < b ? a : b; }
static int max_int(int a, int b) { return a > b ? a : b; }

/* ------------------------------------------------------------------------------------ */
/* App. H: edit distance between byte strings s[0..m) and t[0..n), unit costs.          */
int orc_levenshtein(const uint8_t *s, int m, const uint8_t *t, int n) {
    int *D = (int *)malloc(sizeof(int) * (size_t)(m + 1) * (size_t)(n + 1));
#define DD(i, j) D[(size_t)(i) * (size_t)(n + 1) + (size_t)(j)]
    for (int i = 0; i <= m; ++i) DD(i, 0) = i;          /* Step 1, first column */
    for (int j = 0; j <= n; ++j) DD(0, j) = j;          /* Step 1, first row    */
    for (int i = 1; i <= m; ++i) {                      /* Step 2, recurrence   */
        for (int j = 1; j <= n; ++j) {
            int del = DD(i - 1, j) + 1;
            int ins = DD(i, j - 1) + 1;
            int sub = DD(i - 1, j - 1) + (s[i - 1] == t[j - 1] ? 0 : 1);
            DD(i, j) = min_int(del, min_int(ins, sub));
        }
    }
    int r = DD(m, n);                                   /* Step 3 */
#undef DD
    free(D);
    return r;
}

/* ------------------------------------------------------------------------------------ */
/* Vocabulary table: token id -> bytes[offsets[id] .. offsets[id+1]).                     */
typedef struct {
    const uint8_t *bytes;
    const int32_t *offsets;
    int32_t n_tokens;
    int32_t max_token_bytes;
} orc_vocab;

static int token_ok(const orc_vocab *v, int32_t id) {
    if (id < 0 || id >= v->n_tokens) return 0;
    int32_t len = v->offsets[id + 1] - v->offsets[id];
    return len >= 0 && len <= v->max_token_bytes;
}

static int token_distance(const orc_vocab *vd, int32_t a, const orc_vocab *vt, int32_t b) {
    const uint8_t *s = vd->bytes + vd->offsets[a];
    const uint8_t *t = vt->bytes + vt->offsets[b];
    return orc_levenshtein(s, vd->offsets[a + 1] - vd->offsets[a], t, vt->offsets[b + 1] - vt->offsets[b]);
}

/* Alg. 1 for one pair.  x = draft ids (K), y = proxy target ids (M).  Writes the cost
 * C*, the forward path as 0-based (i, j) pairs and the per-target-position map.
 * Returns the path length. */
static int dtw_pair(const orc_vocab *vd, const orc_vocab *vt, const int32_t *x, int K,
                    const int32_t *y, int M, int w, int32_t *cost, int32_t *path, int32_t *map) {
    int L = (w < 0) ? max_int(K, M) : max_int(w, abs(K - M));
    size_t cols = (size_t)M + 1;
    int *C = (int *)malloc(sizeof(int) * (size_t)(K + 1) * cols);
#define CC(i, j) C[(size_t)(i) * cols + (size_t)(j)]
    /* initialisation: C00 = 0, every other cell (borders and out-of-band) = inf */
    for (size_t e = 0; e < (size_t)(K + 1) * cols; ++e) C[e] = ORC_INF;
    CC(0, 0) = 0;
    for (int i = 1; i <= K; ++i) {
        for (int j = max_int(1, i - L); j <= min_int(M, i + L); ++j) {
            int best = min_int(CC(i - 1, j), min_int(CC(i, j - 1), CC(i - 1, j - 1)));
            if (best >= ORC_INF) continue; /* unreachable cell stays inf */
            CC(i, j) = token_distance(vd, x[i - 1], vt, y[j - 1]) + best;
        }
    }
    *cost = CC(K, M);

    /* backtrack from (K, M) to (0, 0): prepend, then move to the cheapest predecessor;
     * ties go to the diagonal, then (i-1, j), then (i, j-1). */
    int32_t *rev = (int32_t *)malloc(sizeof(int32_t) * 2 * (size_t)(K + M + 1));
    int n = 0, i = K, j = M;
    while (i != 0 || j != 0) {
        rev[2 * n] = i;
        rev[2 * n + 1] = j;
        ++n;
        int vd_ = (i >= 1 && j >= 1) ? CC(i - 1, j - 1) : ORC_INF;
        int vu = (i >= 1) ? CC(i - 1, j) : ORC_INF;
        int vl = (j >= 1) ? CC(i, j - 1) : ORC_INF;
        if (vd_ <= vu && vd_ <= vl) {
            --i;
            --j;
        } else if (vu <= vl) {
            --i;
        } else {
            --j;
        }
    }
#undef CC
    for (int p = 0; p < n; ++p) { /* forward order, 0-based */
        path[2 * p] = rev[2 * (n - 1 - p)] - 1;
        path[2 * p + 1] = rev[2 * (n - 1 - p) + 1] - 1;
    }
    /* App. A.2: each target position takes the terminal (largest) draft index aligned
     * with it; a draft token spanning several target positions is copied to each. */
    for (int t = 0; t < M; ++t) map[t] = -1;
    for (int p = 0; p < n; ++p) {
        int di = path[2 * p], tj = path[2 * p + 1];
        if (di > map[tj]) map[tj] = di;
    }
    free(rev);
    free(C);
    return n;
}

/* ------------------------------------------------------------------------------------ */
/* Static split of [0, n) over worker threads.                                          */
typedef void (*orc_range_fn)(void *ctx, int32_t lo, int32_t hi);
typedef struct {
    orc_range_fn fn;
    void *ctx;
    int32_t lo, hi;
} orc_job;

static void *orc_job_run(void *p) {
    orc_job *j = (orc_job *)p;
    j->fn(j->ctx, j->lo, j->hi);
    return NULL;
}

static void orc_parallel(int32_t n, int n_threads, orc_range_fn fn, void *ctx) {
    if (n_threads < 1) n_threads = 1;
    if (n_threads > n) n_threads = n > 0 ? n : 1;
    if (n_threads == 1) {
        fn(ctx, 0, n);
        return;
    }
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)n_threads);
    orc_job *jobs = (orc_job *)malloc(sizeof(orc_job) * (size_t)n_threads);
    for (int t = 0; t < n_threads; ++t) {
        jobs[t].fn = fn;
        jobs[t].ctx = ctx;
        jobs[t].lo = (int32_t)((int64_t)n * t / n_threads);
        jobs[t].hi = (int32_t)((int64_t)n * (t + 1) / n_threads);
        pthread_create(&th[t], NULL, orc_job_run, &jobs[t]);
    }
    for (int t = 0; t < n_threads; ++t) pthread_join(th[t], NULL);
    free(jobs);
    free(th);
}

/* ------------------------------------------------------------------------------------ */
/* Alignment of every pair.  Output layout:
 *   cost[b], path_len[b];
 *   path: pair b starts at int32 index 2*(draft_off[b] + target_off[b]), holding up to
 *         K_b + M_b (i, j) pairs, 0-based, forward order;
 *   map[target_off[b] + j] = i*(j), 0-based.
 * A pair with K_b or M_b outside [1, max], an id outside its vocabulary, or a token
 * longer than max_token_bytes gets cost -1, path_len 0 and map -1. */
typedef struct {
    orc_vocab vd, vt;
    const int32_t *draft_ids, *draft_off, *target_ids, *target_off;
    int32_t max_k, max_m, w;
    int32_t *cost, *path_len, *path, *map;
} orc_align_ctx;

static void orc_align_range(void *p, int32_t lo, int32_t hi) {
    orc_align_ctx *c = (orc_align_ctx *)p;
    for (int32_t b = lo; b < hi; ++b) {
        int32_t d0 = c->draft_off[b], t0 = c->target_off[b];
        int K = c->draft_off[b + 1] - d0, M = c->target_off[b + 1] - t0;
        int ok = K >= 1 && K <= c->max_k && M >= 1 && M <= c->max_m;
        for (int i = 0; ok && i < K; ++i) ok = token_ok(&c->vd, c->draft_ids[d0 + i]);
        for (int j = 0; ok && j < M; ++j) ok = token_ok(&c->vt, c->target_ids[t0 + j]);
        if (!ok) {
            c->cost[b] = -1;
            c->path_len[b] = 0;
            for (int j = 0; j < M; ++j) c->map[t0 + j] = -1;
            continue;
        }
        c->path_len[b] = dtw_pair(&c->vd, &c->vt, c->draft_ids + d0, K, c->target_ids + t0, M, c->w,
                                  &c->cost[b], c->path + 2 * ((size_t)d0 + (size_t)t0), c->map + t0);
    }
}

void orc_align(const uint8_t *vd_bytes, const int32_t *vd_off, int32_t vd_n, int32_t vd_maxlen,
               const uint8_t *vt_bytes, const int32_t *vt_off, int32_t vt_n, int32_t vt_maxlen,
               int32_t n_pairs, const int32_t *draft_ids, const int32_t *draft_off,
               const int32_t *target_ids, const int32_t *target_off, int32_t max_k, int32_t max_m,
               int32_t w, int32_t *cost, int32_t *path_len, int32_t *path, int32_t *map,
               int n_threads) {
    orc_align_ctx c = {{vd_bytes, vd_off, vd_n, vd_maxlen}, {vt_bytes, vt_off, vt_n, vt_maxlen},
                       draft_ids, draft_off, target_ids, target_off, max_k, max_m, w,
                       cost, path_len, path, map};
    orc_parallel(n_pairs, n_threads, orc_align_range, &c);
}

/* ------------------------------------------------------------------------------------ */
/* Transfer: q[target_off[b] + j] = P_d[row draft_off[b] + i][d_i] with i = map(j); the
 * draft's probability of the token it emitted at the aligned terminal position.
 * An index outside the pair or an id outside [0, v_d) gives NaN. */
void orc_transfer(int32_t n_pairs, int32_t v_d, const int32_t *draft_ids, const int32_t *draft_off,
                  const int32_t *target_off, const int32_t *map, const float *draft_probs,
                  int64_t draft_ld, float *q) {
    for (int32_t b = 0; b < n_pairs; ++b) {
        int32_t d0 = draft_off[b], K = draft_off[b + 1] - draft_off[b];
        for (int32_t t = target_off[b]; t < target_off[b + 1]; ++t) {
            int32_t i = map[t];
            float v = NAN;
            if (i >= 0 && i < K) {
                int32_t tok = draft_ids[d0 + i];
                if (tok >= 0 && tok < v_d) v = draft_probs[(int64_t)(d0 + i) * draft_ld + tok];
            }
            q[t] = v;
        }
    }
}

/* ------------------------------------------------------------------------------------ */
/* Sampling from a quantised row: exact threshold T = floor(u * Z), first index whose
 * inclusive prefix sum exceeds T.  u outside [0, 1) is clamped to the nearest end. */
static uint64_t exact_threshold(float u, uint64_t Z) {
    if (!(u > 0.0f)) return 0; /* u <= 0 or NaN */
    if (u >= 1.0f) return Z - 1;
    int e;
    float f = frexpf(u, &e);                          /* u = f * 2^e, f in [0.5, 1) */
    uint64_t mant = (uint64_t)ldexpf(f, 24);          /* exact: f has 24 significant bits */
    int shift = 24 - e;                               /* u = mant * 2^-shift */
    if (shift >= 128) return 0;
    unsigned __int128 prod = (unsigned __int128)mant * (unsigned __int128)Z;
    uint64_t T = (uint64_t)(prod >> shift);
    return T < Z ? T : Z - 1;
}

static int32_t sample_quantised(const uint64_t *Rq, int64_t V, uint64_t Z, float u) {
    uint64_t T = exact_threshold(u, Z);
    uint64_t prefix = 0;
    for (int64_t x = 0; x < V; ++x) {
        prefix += Rq[x];
        if (prefix > T) return (int32_t)x;
    }
    return (int32_t)(V - 1); /* unreachable when the sum equals Z > T */
}

static int32_t first_argmax(const float *row, int64_t V) {
    float best = -INFINITY;
    int32_t idx = 0;
    for (int64_t x = 0; x < V; ++x)
        if (row[x] > best) {
            best = row[x];
            idx = (int32_t)x;
        }
    return idx;
}

/* residual value at index x of a row: max(0, p - qx) clamped to [0, 1], NaN -> 0 */
static float residual_value(float p, float qx) {
    float r = fmaxf(p - qx, 0.0f);
    return fminf(r, 1.0f);
}

/* Verification of one stream (see the header comment for the readings). */
typedef struct {
    int32_t v_t;
    const int32_t *target_ids, *target_off;
    const float *q, *target_probs;
    int64_t target_ld;
    const float *u_accept, *u_sample;
    int32_t max_m;
    int32_t *n_accepted, *out_token;
    float *residual;
    uint64_t *z_out;
    const int32_t *select; /* optional list of streams to process */
} orc_verify_ctx;

static void orc_verify_stream(orc_verify_ctx *c, int32_t b) {
    int32_t t0 = c->target_off[b];
    int32_t M = c->target_off[b + 1] - t0;
    int ok = M >= 0 && M <= c->max_m;
    for (int32_t j = 0; ok && j < M; ++j) ok = c->target_ids[t0 + j] >= 0 && c->target_ids[t0 + j] < c->v_t;
    if (!ok) {
        c->n_accepted[b] = -1;
        c->out_token[b] = -1;
        if (c->z_out) c->z_out[b] = 0;
        return;
    }
    /* acceptance: t_j is accepted when u_j < P_t(t_j) / q_j; stop at the first rejection */
    int32_t gamma = M;
    for (int32_t j = 0; j < M; ++j) {
        int32_t tok = c->target_ids[t0 + j];
        float p = c->target_probs[(int64_t)(t0 + b + j) * c->target_ld + tok];
        float qj = c->q[t0 + j];
        float ratio = p / qj;
        int accept = (qj <= 0.0f) || (c->u_accept[t0 + j] < ratio);
        if (!accept) {
            gamma = j;
            break;
        }
    }
    /* residual (rejection) or bonus (all accepted) row */
    int32_t r = gamma;
    const float *row = c->target_probs + (int64_t)(t0 + b + r) * c->target_ld;
    int32_t rej_tok = (r < M) ? c->target_ids[t0 + r] : -1;
    float rej_q = (r < M) ? c->q[t0 + r] : 0.0f;
    int64_t V = c->v_t;
    uint64_t *Rq = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    uint64_t Z = 0;
    for (int64_t x = 0; x < V; ++x) {
        float qx = (x == rej_tok) ? rej_q : 0.0f;
        float R = residual_value(row[x], qx);
        Rq[x] = (uint64_t)(R * 0x1p62f); /* Q62, truncating */
        Z += Rq[x];
    }
    int32_t token = (Z == 0) ? first_argmax(row, V) : sample_quantised(Rq, V, Z, c->u_sample[b]);
    c->n_accepted[b] = gamma;
    c->out_token[b] = token;
    if (c->z_out) c->z_out[b] = Z;
    if (c->residual) {
        float *res = c->residual + (int64_t)b * c->target_ld;
        if (Z == 0) {
            for (int64_t x = 0; x < V; ++x) res[x] = (x == token) ? 1.0f : 0.0f;
        } else {
            float zf = (float)Z * 0x1p-62f;
            for (int64_t x = 0; x < V; ++x) {
                float qx = (x == rej_tok) ? rej_q : 0.0f;
                res[x] = residual_value(row[x], qx) / zf;
            }
        }
    }
    free(Rq);
}

static void orc_verify_range(void *p, int32_t lo, int32_t hi) {
    orc_verify_ctx *c = (orc_verify_ctx *)p;
    for (int32_t s = lo; s < hi; ++s) orc_verify_stream(c, c->select ? c->select[s] : s);
}

/* Verify streams (all n_streams, or only the n_select listed in `select`).  Outputs are
 * indexed by stream id.  residual (optional) is [n_streams x target_ld]; z_out
 * (optional) receives the Q62 residual mass per stream. */
void orc_verify(int32_t n_streams, int32_t v_t, const int32_t *target_ids, const int32_t *target_off,
                const float *q, const float *target_probs, int64_t target_ld, const float *u_accept,
                const float *u_sample, int32_t max_m, int32_t *n_accepted, int32_t *out_token,
                float *residual, uint64_t *z_out, const int32_t *select, int32_t n_select,
                int n_threads) {
    orc_verify_ctx c = {v_t, target_ids, target_off, q, target_probs, target_ld, u_accept, u_sample,
                        max_m, n_accepted, out_token, residual, z_out, select};
    orc_parallel(select ? n_select : n_streams, n_threads, orc_verify_range, &c);
}

/* ------------------------------------------------------------------------------------ */
/* Test-only: standard speculative sampling with a dense proposal over one vocabulary
 * (App. D Alg. 4, one drafted position).  p = target row, qd = draft row, x = drafted
 * token.  Accept when p(x) >= qd(x), else with probability p(x)/qd(x) (u < ratio);
 * on rejection sample norm(max(0, p - qd)); returns the emitted token, and sets
 * *accepted.  When accepted the caller emits x (the bonus sample is a separate step). */
int32_t orc_verify_dense(int32_t V, const float *p, const float *qd, int32_t x, float u_accept,
                         float u_sample, int32_t *accepted) {
    float ratio = p[x] / qd[x];
    if (qd[x] <= 0.0f || u_accept < ratio) {
        *accepted = 1;
        return x;
    }
    *accepted = 0;
    uint64_t *Rq = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    uint64_t Z = 0;
    for (int32_t y = 0; y < V; ++y) {
        Rq[y] = (uint64_t)(residual_value(p[y], qd[y]) * 0x1p62f);
        Z += Rq[y];
    }
    int32_t tok = (Z == 0) ? first_argmax(p, V) : sample_quantised(Rq, V, Z, u_sample);
    free(Rq);
    return tok;
}

/* ------------------------------------------------------------------------------------ */
/* Standard speculative sampling over one vocabulary (App. D Alg. 4) for a batch of
 * streams: the homogeneous-vocabulary case, where the proposal of drafted position j is
 * the draft model's whole distribution q_j over the same V tokens as the target.
 *
 * Stream b drafted M_b = off[b+1] - off[b] tokens x_j = draft_ids[off[b] + j], each
 * sampled from the dense row q_j = draft_probs[off[b] + j].  The target model scored the
 * M_b + 1 prefixes: p_j = target_probs[off[b] + b + j], j = 0..M_b.
 *   1. Alg. 4's loop: position j is kept when p_j(x_j) > q_j(x_j), or else with
 *      probability p_j(x_j) / q_j(x_j).  With u_j = u_accept[off[b] + j] in [0, 1) both
 *      cases are "u_j < p_j(x_j) / q_j(x_j)" (fp32 quotient); q_j(x_j) <= 0 keeps the
 *      token (the quotient is +inf), as in the one-hot reading.  gamma = the first
 *      position not kept, else M_b.
 *   2. The modified distribution: after a rejection at r = gamma < M_b it is
 *      max(0, p_r - q_r) (clamped to [0, 1], NaN -> 0), after full acceptance the plain
 *      bonus row p_{M_b}.
 *   3. The next token is drawn from it with u_sample[b] by the exact Q62 inverse CDF
 *      (same quantisation, threshold and tie rules as orc_verify).
 * A stream with M_b outside [0, max_m] or a drafted id outside [0, V) gets -1 outputs. */
typedef struct {
    int32_t V;
    const int32_t *draft_ids, *off;
    const float *draft_probs;
    int64_t draft_ld;
    const float *target_probs;
    int64_t target_ld;
    const float *u_accept, *u_sample;
    int32_t max_m;
    int32_t *n_accepted, *out_token;
    float *residual;
    uint64_t *z_out;
} orc_sd_ctx;

static void orc_sd_stream(orc_sd_ctx *c, int32_t b) {
    int32_t o = c->off[b];
    int32_t M = c->off[b + 1] - o;
    int ok = M >= 0 && M <= c->max_m;
    for (int32_t j = 0; ok && j < M; ++j) ok = c->draft_ids[o + j] >= 0 && c->draft_ids[o + j] < c->V;
    if (!ok) {
        c->n_accepted[b] = -1;
        c->out_token[b] = -1;
        if (c->z_out) c->z_out[b] = 0;
        return;
    }
    /* step 1: keep drafted tokens until the first rejection */
    int32_t gamma = M;
    for (int32_t j = 0; j < M; ++j) {
        int32_t x = c->draft_ids[o + j];
        float p = c->target_probs[(int64_t)(o + b + j) * c->target_ld + x];
        float qx = c->draft_probs[(int64_t)(o + j) * c->draft_ld + x];
        float ratio = p / qx;
        int keep = (qx <= 0.0f) || (c->u_accept[o + j] < ratio);
        if (!keep) {
            gamma = j;
            break;
        }
    }
    /* step 2: the modified distribution */
    int32_t r = gamma;
    const float *prow = c->target_probs + (int64_t)(o + b + r) * c->target_ld;
    const float *qrow = (r < M) ? c->draft_probs + (int64_t)(o + r) * c->draft_ld : NULL;
    int64_t V = c->V;
    uint64_t *Rq = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)V);
    uint64_t Z = 0;
    for (int64_t y = 0; y < V; ++y) {
        float R = residual_value(prow[y], qrow ? qrow[y] : 0.0f);
        Rq[y] = (uint64_t)(R * 0x1p62f); /* Q62, truncating */
        Z += Rq[y];
    }
    /* step 3: the next token */
    int32_t token = (Z == 0) ? first_argmax(prow, V) : sample_quantised(Rq, V, Z, c->u_sample[b]);
    c->n_accepted[b] = gamma;
    c->out_token[b] = token;
    if (c->z_out) c->z_out[b] = Z;
    if (c->residual) {
        float *res = c->residual + (int64_t)b * c->target_ld;
        if (Z == 0) {
            for (int64_t y = 0; y < V; ++y) res[y] = (y == token) ? 1.0f : 0.0f;
        } else {
            float zf = (float)Z * 0x1p-62f;
            for (int64_t y = 0; y < V; ++y) res[y] = residual_value(prow[y], qrow ? qrow[y] : 0.0f) / zf;
        }
    }
    free(Rq);
}

static void orc_sd_range(void *p, int32_t lo, int32_t hi) {
    for (int32_t s = lo; s < hi; ++s) orc_sd_stream((orc_sd_ctx *)p, s);
}

void orc_sd_verify(int32_t n_streams, int32_t V, const int32_t *draft_ids, const int32_t *off,
                   const float *draft_probs, int64_t draft_ld, const float *target_probs, int64_t target_ld,
                   const float *u_accept, const float *u_sample, int32_t max_m, int32_t *n_accepted,
                   int32_t *out_token, float *residual, uint64_t *z_out, int n_threads) {
    orc_sd_ctx c = {V, draft_ids, off, draft_probs, draft_ld, target_probs, target_ld, u_accept, u_sample,
                    max_m, n_accepted, out_token, residual, z_out};
    orc_parallel(n_streams, n_threads, orc_sd_range, &c);
}

/* ------------------------------------------------------------------------------------ */
/* Sec. 5 "DTW Bridges the Gap" (Fig. CDF) and App. K: the position deviation of a matched
 * draft / proxy target token pair (i, j) on an optimal warping path is |i - j|.  hist[d]
 * counts the path cells of all pairs with |i - j| = d for d < n_bins - 1; the last bin
 * counts every cell with |i - j| >= n_bins - 1.  Pair b's cells are path[2*(draft_off[b] +
 * target_off[b]) ...] (path_len[b] of them, as orc_align writes them).  A pair with
 * path_len <= 0 (a sentinel pair) contributes nothing, and so does one whose path_len
 * exceeds K_b + M_b: a warping path from (1,1) to (K,M) has at most K + M - 1 cells, and
 * the path area of pair b holds K_b + M_b of them. */
void orc_delta_histogram(int32_t n_pairs, const int32_t *draft_off, const int32_t *target_off,
                         const int32_t *path_len, const int32_t *path, int32_t n_bins, int64_t *hist) {
    for (int32_t d = 0; d < n_bins; ++d) hist[d] = 0;
    for (int32_t b = 0; b < n_pairs; ++b) {
        const int32_t K = draft_off[b + 1] - draft_off[b], M = target_off[b + 1] - target_off[b];
        if (path_len[b] > K + M) continue;
        const int32_t *cells = path + 2 * (int64_t)(draft_off[b] + target_off[b]);
        for (int32_t c = 0; c < path_len[b]; ++c) {
            int32_t dev = abs(cells[2 * c] - cells[2 * c + 1]);
            hist[dev < n_bins - 1 ? dev : n_bins - 1] += 1;
        }
    }
}

/* App. K "Settings of w": w is placed where the cumulative distribution of the position
 * deviation reaches 0.9 (read off the histogram above, collected without a band).  For a
 * quantile num/den (0 <= num <= den, 1 <= den <= 65536) this is the smallest d with
 * hist[0] + ... + hist[d] >= (num/den) * total, decided exactly as
 * (hist[0] + ... + hist[d]) * den >= num * total; 0 for an empty histogram.  If d is the
 * last bin the deviation at the quantile is at least n_bins - 1. */
int32_t orc_delta_quantile(const int64_t *hist, int32_t n_bins, int32_t num, int32_t den) {
    int64_t total = 0;
    for (int32_t d = 0; d < n_bins; ++d) total += hist[d];
    if (total == 0) return 0;
    int64_t cum = 0;
    for (int32_t d = 0; d < n_bins; ++d) {
        cum += hist[d];
        if (cum * (int64_t)den >= (int64_t)num * total) return d;
    }
    return n_bins - 1;
}

/* ------------------------------------------------------------------------------------ */
/* Verification from bf16 target logits with a temperature (the step before Sec. 3's target
 * distribution, App. F sampling temperatures): P_t = softmax(logit * inv_temp) formed inside
 * the verification, in base 2.  Readings (the paper fixes none of this arithmetic):
 *   c        = inv_temp * log2(e), one fp32 product per stream (log2(e) rounded to fp32);
 *   y        = fp32(bf16 logit) * c (fp32); NaN logits count as minus infinity;
 *   mu       = the largest y of the row, or, with a caller's log-sum-exp L of the row (in the
 *              natural units of logit * inv_temp), L * log2(e) (fp32);
 *   z        = fma(fp32(bf16 logit), c, 31 - mu) (31 - mu rounded to fp32 first), the base-2
 *              exponent of the logit's weight scaled by 2^31, held in [-1, 31] (NaN -> -1);
 *   2^z      = p * 2^k with k = rint(z), f = z - k in [-1/2, 1/2] and p the degree-5 Taylor
 *              polynomial of 2^f = exp(f ln 2) (coefficients (ln 2)^n / n! rounded to fp32,
 *              Horner's rule with fused multiply-adds; relative error below 3.3e-6);
 *   e31      = floor(p * 2^k), the logit's weight in Q31 (exact: p * 2^k < 2^32);
 *   E        = p * 2^(k - 31) as fp32 when z >= 0, else 0 (the weight as a fraction of the
 *              largest, cut where e31 is 0);
 *   S        = (sum of e31) * 2^-31 rounded once to the nearest fp32, ties to even;
 *   P_t(t_j) = E(t_j) / S (fp32), or E(t_j) when L is given (S = 1); accept iff q_j <= 0
 *              or u_j < P_t(t_j) / q_j;
 *   residual on rejection at r: the row's e31 with the entry at t_r replaced by
 *            floor(clamp(E(t_r) - q_r * S, 0, 1) * 2^31) (with L: clamp(P - q_r, 0, 1)) --
 *            proportional to max(0, P_t - q_r e_{t_r}); after full acceptance the bonus
 *            row's e31;
 *   sample   T = floor(u * Z) and the first index whose prefix exceeds T, as for the
 *            probability rows; if Z = 0 the first index of the largest y (0 if none).
 * Weights below 2^-31 of the largest count as 0.  Rows of at most 2^23 entries keep every
 * sum below 2^55. */
#define ORC_L2E 0x1.715476p+0f

/* 2^z = p * 2^k for z held in [-1, 31] (NaN -> -1): k = rint(z) (ties to even), f = z - k
 * (exact), p = 1 + f ln2 + (f ln2)^2/2! + ... + (f ln2)^5/5! by Horner's rule in f. */
static float orc_exp2_parts(float z, int *k) {
    z = fminf(fmaxf(z, -1.0f), 31.0f);
    const float kf = rintf(z);
    const float f = z - kf;
    float p = 0x1.5d87fep-10f;      /* (ln 2)^5 / 5! */
    p = fmaf(p, f, 0x1.3b2ab6p-7f); /* (ln 2)^4 / 4! */
    p = fmaf(p, f, 0x1.c6b08ep-5f); /* (ln 2)^3 / 3! */
    p = fmaf(p, f, 0x1.ebfbe0p-3f); /* (ln 2)^2 / 2! */
    p = fmaf(p, f, 0x1.62e430p-1f); /* ln 2 */
    p = fmaf(p, f, 1.0f);
    *k = (int)kf;
    return p;
}

/* Test hook: the specified 2^z as fp32 (z held in [-1, 31]). */
float orc_exp2(float z) {
    int k;
    const float p = orc_exp2_parts(z, &k);
    return ldexpf(p, k);
}

static uint32_t orc_e31(float z) { /* floor(2^z) */
    int k;
    const float p = orc_exp2_parts(z, &k);
    return (uint32_t)ldexpf(p, k);
}

static float orc_weight(float z) { /* E = 2^(z - 31), 0 when z < 0 or NaN */
    if (!(z >= 0.0f)) return 0.0f;
    int k;
    const float p = orc_exp2_parts(z, &k);
    return ldexpf(p, k - 31);
}

static uint32_t orc_q31(float r) { return (uint32_t)ldexpf(r, 31); } /* floor(r * 2^31), r in [0, 1] */

static float q31_to_f32(uint64_t n) { /* n * 2^-31 rounded to the nearest fp32, ties to even */
    if (n == 0) return 0.0f;
    int bl = 64;
    while (!((n >> (bl - 1)) & 1u)) --bl;
    if (bl <= 24) return ldexpf((float)n, -31);
    const int sh = bl - 24;
    uint64_t mant = n >> sh;
    const uint64_t rem = n & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    if (rem > half || (rem == half && (mant & 1u))) ++mant;
    return ldexpf((float)mant, sh - 31);
}

static float bf16_to_f32(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* Test hook: P_t of one logit x (fp32 value of its bf16) with a caller's log-sum-exp L. */
float orc_logit_prob(float x, float inv_temp, float L) {
    const float c = inv_temp * ORC_L2E;
    const float mu = L * ORC_L2E;
    return fminf(fmaxf(orc_weight(fmaf(x, c, 31.0f - mu)), 0.0f), 1.0f);
}

typedef struct {
    int32_t v;
    const int32_t *ids, *off;
    const float *q;
    const uint16_t *logits;
    int64_t ld;
    const float *inv_temp, *ua, *us;
    const float *lse; /* per row, or NULL */
    int32_t max_m;
    int32_t *nacc, *tok;
    uint64_t *z;
} orc_logits_ctx;

/* Sample row `row` of weights e31 (the entry at t replaced by adj when t >= 0): returns the
 * token and the mass Z. */
static int32_t orc_logits_sample(const uint16_t *lg, int32_t v, float c, float b31, int32_t t, uint32_t adj,
                                 float u, uint64_t *Zout) {
    uint64_t *w = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)v);
    uint64_t Z = 0;
    float best = -INFINITY;
    int32_t arg = 0;
    for (int32_t i = 0; i < v; ++i) {
        const float x = bf16_to_f32(lg[i]);
        float y = x * c;
        if (isnan(y)) y = -INFINITY;
        if (y > best) {
            best = y;
            arg = i;
        }
        w[i] = (i == t) ? adj : orc_e31(fmaf(x, c, b31));
        Z += w[i];
    }
    const int32_t token = Z == 0 ? arg : sample_quantised(w, v, Z, u);
    free(w);
    *Zout = Z;
    return token;
}

/* With per-row log-sum-exp values L_j supplied by the caller: mu = L_j * log2(e), S = 1, the
 * acceptance test on P = E(t_j), and one pass over the residual (or bonus) row. */
static void orc_logits_stream_lse(orc_logits_ctx *c, int32_t b) {
    const int32_t t0 = c->off[b], M = c->off[b + 1] - t0;
    const float cs = c->inv_temp[b] * ORC_L2E;
    int32_t r = M;
    float Pr = 0.0f;
    for (int32_t j = 0; j < M; ++j) {
        const int64_t row = t0 + b + j;
        const float mu = c->lse[row] * ORC_L2E;
        const float x = bf16_to_f32(c->logits[row * c->ld + c->ids[t0 + j]]);
        const float P = fminf(fmaxf(orc_weight(fmaf(x, cs, 31.0f - mu)), 0.0f), 1.0f);
        const float qj = c->q[t0 + j];
        if (!(qj <= 0.0f || c->ua[t0 + j] < P / qj)) {
            r = j;
            Pr = P;
            break;
        }
    }
    const int64_t row = t0 + b + r;
    const float mu = c->lse[row] * ORC_L2E;
    int32_t t = -1;
    uint32_t adj = 0;
    if (r < M) {
        t = c->ids[t0 + r];
        adj = orc_q31(fminf(fmaxf(Pr - c->q[t0 + r], 0.0f), 1.0f)); /* NaN -> 0 */
    }
    c->nacc[b] = r;
    c->tok[b] = orc_logits_sample(c->logits + row * c->ld, c->v, cs, 31.0f - mu, t, adj, c->us[b], &c->z[b]);
}

static void orc_logits_stream(orc_logits_ctx *c, int32_t b) {
    const int32_t t0 = c->off[b], M = c->off[b + 1] - t0;
    int ok = M >= 0 && M <= c->max_m && c->inv_temp[b] > 0.0f;
    for (int32_t j = 0; ok && j < M; ++j) ok = c->ids[t0 + j] >= 0 && c->ids[t0 + j] < c->v;
    if (!ok) {
        c->nacc[b] = -1;
        c->tok[b] = -1;
        c->z[b] = 0;
        return;
    }
    if (c->lse != NULL) {
        orc_logits_stream_lse(c, b);
        return;
    }
    const float cs = c->inv_temp[b] * ORC_L2E;
    for (int32_t j = 0; j <= M; ++j) {
        const uint16_t *row = c->logits + (int64_t)(t0 + b + j) * c->ld;
        float mu = -INFINITY;
        for (int32_t i = 0; i < c->v; ++i) {
            const float y = bf16_to_f32(row[i]) * cs;
            if (y > mu) mu = y; /* NaN never compares greater */
        }
        const float b31 = 31.0f - mu;
        uint64_t Sq = 0;
        for (int32_t i = 0; i < c->v; ++i) Sq += orc_e31(fmaf(bf16_to_f32(row[i]), cs, b31));
        const float S = q31_to_f32(Sq);
        int32_t t = -1;
        uint32_t adj = 0;
        if (j < M) {
            t = c->ids[t0 + j];
            const float qj = c->q[t0 + j];
            const float Et = orc_weight(fmaf(bf16_to_f32(row[t]), cs, b31));
            const float P = Et / S;
            if (qj <= 0.0f || c->ua[t0 + j] < P / qj) continue; /* accepted: next position */
            adj = orc_q31(fminf(fmaxf(Et - qj * S, 0.0f), 1.0f)); /* NaN -> 0 */
        }
        c->nacc[b] = j;
        c->tok[b] = orc_logits_sample(row, c->v, cs, b31, t, adj, c->us[b], &c->z[b]);
        return;
    }
}

static void orc_logits_range(void *p, int32_t lo, int32_t hi) {
    for (int32_t s = lo; s < hi; ++s) orc_logits_stream((orc_logits_ctx *)p, s);
}

void orc_verify_logits(int32_t n_streams, int32_t v, const int32_t *target_ids, const int32_t *target_off,
                       const float *q, const uint16_t *logits, int64_t ld, const float *inv_temp,
                       const float *lse, const float *u_accept, const float *u_sample, int32_t max_m,
                       int32_t *n_accepted, int32_t *out_token, uint64_t *z_out, int n_threads) {
    orc_logits_ctx c = {v, target_ids, target_off, q, logits, ld, inv_temp, u_accept, u_sample, lse, max_m,
                        n_accepted, out_token, z_out};
    orc_parallel(n_streams, n_threads, orc_logits_range, &c);
}

/* Test hook: the exact threshold floor(u * Z). */
uint64_t orc_threshold(float u, uint64_t Z) { return Z == 0 ? 0 : exact_threshold(u, Z); }
