/*
 * Test driver: runs every entry point of the CPU oracle on small seeded inputs, including
 * sentinel pairs and streams, empty strings, zero-mass rows and several threads.  The test
 * that builds it links it with the oracle under AddressSanitizer and UndefinedBehaviorSanitizer
 * (host code only), so an out-of-bounds access, a leak or undefined arithmetic in the oracle
 * fails the test.  Prints one line per stage and "done" at the end.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int orc_levenshtein(const uint8_t *s, int m, const uint8_t *t, int n);
void orc_align(const uint8_t *vd_bytes, const int32_t *vd_off, int32_t vd_n, int32_t vd_maxlen,
               const uint8_t *vt_bytes, const int32_t *vt_off, int32_t vt_n, int32_t vt_maxlen, int32_t n_pairs,
               const int32_t *draft_ids, const int32_t *draft_off, const int32_t *target_ids,
               const int32_t *target_off, int32_t max_k, int32_t max_m, int32_t w, int32_t *cost,
               int32_t *path_len, int32_t *path, int32_t *map, int n_threads);
void orc_transfer(int32_t n_pairs, int32_t v_d, const int32_t *draft_ids, const int32_t *draft_off,
                  const int32_t *target_off, const int32_t *map, const float *draft_probs, int64_t draft_ld,
                  float *q);
void orc_verify(int32_t n_streams, int32_t v_t, const int32_t *target_ids, const int32_t *target_off,
                const float *q, const float *target_probs, int64_t target_ld, const float *u_accept,
                const float *u_sample, int32_t max_m, int32_t *n_accepted, int32_t *out_token, float *residual,
                uint64_t *z_out, const int32_t *select, int32_t n_select, int n_threads);
int32_t orc_verify_dense(int32_t V, const float *p, const float *qd, int32_t x, float u_accept, float u_sample,
                         int32_t *accepted);
void orc_sd_verify(int32_t n_streams, int32_t V, const int32_t *draft_ids, const int32_t *off,
                   const float *draft_probs, int64_t draft_ld, const float *target_probs, int64_t target_ld,
                   const float *u_accept, const float *u_sample, int32_t max_m, int32_t *n_accepted,
                   int32_t *out_token, float *residual, uint64_t *z_out, int n_threads);
void orc_delta_histogram(int32_t n_pairs, const int32_t *draft_off, const int32_t *target_off,
                         const int32_t *path_len, const int32_t *path, int32_t n_bins, int64_t *hist);
uint64_t orc_threshold(float u, uint64_t Z);
float orc_exp2(float z);
void orc_verify_logits(int32_t n_streams, int32_t v, const int32_t *target_ids, const int32_t *target_off,
                       const float *q, const uint16_t *logits, int64_t ld, const float *inv_temp,
                       const float *lse, const float *u_accept, const float *u_sample, int32_t max_m,
                       int32_t *n_accepted, int32_t *out_token, uint64_t *z_out, int n_threads);

static uint32_t rng_state = 12345u;
static uint32_t next_u32(void) { /* xorshift32 */
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 17;
    rng_state ^= rng_state << 5;
    return rng_state;
}
static float next_unit(void) { return (float)(next_u32() >> 8) * 0x1p-24f; }

/* a vocabulary of n tokens of 1..maxlen bytes over a 6-letter alphabet, token t = t's digits */
static void make_vocab(int n, int maxlen, uint8_t **bytes, int32_t **off) {
    *off = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
    *bytes = (uint8_t *)malloc((size_t)n * (size_t)maxlen);
    int32_t pos = 0;
    for (int t = 0; t < n; ++t) {
        (*off)[t] = pos;
        int len = 1 + (int)(next_u32() % (uint32_t)maxlen);
        for (int k = 0; k < len; ++k) (*bytes)[pos++] = (uint8_t)('a' + next_u32() % 6u);
    }
    (*off)[n] = pos;
}

static void fill_rows(float *rows, int n, int width) {
    for (int r = 0; r < n; ++r) {
        double s = 0.0;
        for (int x = 0; x < width; ++x) s += (rows[(size_t)r * width + x] = next_unit() + 0.01f);
        for (int x = 0; x < width; ++x) rows[(size_t)r * width + x] = (float)(rows[(size_t)r * width + x] / s);
    }
}

int main(void) {
    /* Levenshtein: empty strings, equal strings, 64-byte strings */
    uint8_t a[64], b[64];
    for (int k = 0; k < 64; ++k) {
        a[k] = (uint8_t)(next_u32() & 0xFF);
        b[k] = (uint8_t)(next_u32() & 0xFF);
    }
    int d0 = orc_levenshtein(a, 0, b, 0), d1 = orc_levenshtein(a, 64, b, 0), d2 = orc_levenshtein(a, 64, a, 64);
    int d3 = orc_levenshtein(a, 64, b, 64);
    printf("levenshtein %d %d %d %d\n", d0, d1, d2, d3);
    if (d0 != 0 || d1 != 64 || d2 != 0 || d3 < 1 || d3 > 64) return 2;

    /* alignment, transfer, verify on a small batch with sentinel pairs */
    const int VD = 40, VT = 50, B = 6;
    uint8_t *vdb, *vtb;
    int32_t *vdo, *vto;
    make_vocab(VD, 4, &vdb, &vdo);
    make_vocab(VT, 5, &vtb, &vto);
    int32_t Ks[6] = {3, 7, 1, 9, 0, 12}, Ms[6] = {4, 2, 6, 9, 3, 20};  /* pair 4: K = 0 (sentinel) */
    int32_t doff[7] = {0}, toff[7] = {0};
    for (int p = 0; p < B; ++p) {
        doff[p + 1] = doff[p] + Ks[p];
        toff[p + 1] = toff[p] + Ms[p];
    }
    int32_t *dids = (int32_t *)malloc(sizeof(int32_t) * (size_t)doff[B]);
    int32_t *tids = (int32_t *)malloc(sizeof(int32_t) * (size_t)toff[B]);
    for (int k = 0; k < doff[B]; ++k) dids[k] = (int32_t)(next_u32() % VD);
    for (int k = 0; k < toff[B]; ++k) tids[k] = (int32_t)(next_u32() % VT);
    tids[toff[3]] = VT + 7; /* pair 3: an id outside the table (sentinel) */
    int32_t cost[6], plen[6];
    int32_t *path = (int32_t *)malloc(sizeof(int32_t) * (size_t)(2 * (doff[B] + toff[B])));
    int32_t *map = (int32_t *)malloc(sizeof(int32_t) * (size_t)toff[B]);
    for (int w = -1; w <= 4; w += 5) {
        orc_align(vdb, vdo, VD, 4, vtb, vto, VT, 5, B, dids, doff, tids, toff, 16, 24, w, cost, plen, path, map, 3);
        printf("align w=%d cost %d %d %d %d %d %d\n", w, cost[0], cost[1], cost[2], cost[3], cost[4], cost[5]);
    }
    int64_t hist[8];
    orc_delta_histogram(B, doff, toff, plen, path, 8, hist);
    printf("delta histogram %lld %lld\n", (long long)hist[0], (long long)hist[7]);

    float *dprobs = (float *)malloc(sizeof(float) * (size_t)doff[B] * VD);
    fill_rows(dprobs, doff[B], VD);
    float *q = (float *)malloc(sizeof(float) * (size_t)toff[B]);
    orc_transfer(B, VD, dids, doff, toff, map, dprobs, VD, q);
    float *tprobs = (float *)malloc(sizeof(float) * (size_t)(toff[B] + B) * VT);
    fill_rows(tprobs, toff[B] + B, VT);
    for (int x = 0; x < VT; ++x) tprobs[(size_t)(toff[1] + 1 + 2) * VT + x] = 0.0f; /* a zero-mass bonus row */
    float *ua = (float *)malloc(sizeof(float) * (size_t)toff[B]);
    for (int k = 0; k < toff[B]; ++k) ua[k] = next_unit();
    float us[6];
    for (int p = 0; p < B; ++p) us[p] = next_unit();
    int32_t nacc[6], tok[6];
    uint64_t z[6];
    float *res = (float *)malloc(sizeof(float) * (size_t)B * VT);
    orc_verify(B, VT, tids, toff, q, tprobs, VT, ua, us, 24, nacc, tok, res, z, NULL, 0, 2);
    int32_t sel[2] = {5, 0};
    orc_verify(B, VT, tids, toff, q, tprobs, VT, ua, us, 24, nacc, tok, NULL, NULL, sel, 2, 1);
    printf("verify %d/%d %d/%d %d/%d\n", nacc[0], tok[0], nacc[3], tok[3], nacc[5], tok[5]);

    /* dense proposals and single-position dense verification */
    int32_t soff[4] = {0, 2, 2, 5};
    int32_t sids[5] = {1, 3, 0, 49, 60}; /* stream 2: an id outside [0, V) */
    float *sq = (float *)malloc(sizeof(float) * 5 * VT);
    float *sp = (float *)malloc(sizeof(float) * 8 * VT);
    fill_rows(sq, 5, VT);
    fill_rows(sp, 8, VT);
    float sua[5] = {0.5f, 0.9f, 0.1f, 0.2f, 0.3f}, sus[3] = {0.25f, 0.75f, 0.0f};
    int32_t snacc[3], stok[3];
    uint64_t sz[3];
    float *sres = (float *)malloc(sizeof(float) * 3 * VT);
    orc_sd_verify(3, VT, sids, soff, sq, VT, sp, VT, sua, sus, 4, snacc, stok, sres, sz, 2);
    int32_t acc;
    int32_t t1 = orc_verify_dense(VT, sp, sq, 7, 0.99f, 0.5f, &acc);
    printf("dense %d/%d %d/%d %d/%d single %d/%d\n", snacc[0], stok[0], snacc[1], stok[1], snacc[2], stok[2], t1,
           acc);
    printf("threshold %llu %llu\n", (unsigned long long)orc_threshold(0.5f, 1000u),
           (unsigned long long)orc_threshold(1.0f - 0x1p-24f, ~0ull));

    /* logits: bf16 rows (random bit patterns of finite values, one NaN row), stream 1 invalid */
    uint16_t *lg = (uint16_t *)malloc(sizeof(uint16_t) * 8 * VT);
    for (int k = 0; k < 8 * VT; ++k) lg[k] = (uint16_t)(0x3c00u + (next_u32() % 0x0800u));
    for (int x = 0; x < VT; ++x) lg[2 * VT + x] = 0x7FC0u;
    int32_t loff[4] = {0, 2, 3, 5}, lids[5] = {1, 3, 70, 0, 49};
    float lq[5] = {0.5f, 0.9f, 0.1f, 0.2f, 0.3f}, lit[3] = {1.0f, 1.4f, 2.0f}, lus[3] = {0.25f, 0.75f, 0.5f};
    int32_t lnacc[3], ltok[3];
    uint64_t lz[3];
    orc_verify_logits(3, VT, lids, loff, lq, lg, VT, lit, NULL, sua, lus, 4, lnacc, ltok, lz, 2);
    float llse[8] = {3.0f, 3.5f, 2.0f, 4.0f, 3.0f, 3.0f, 3.0f, 3.0f};
    orc_verify_logits(3, VT, lids, loff, lq, lg, VT, lit, llse, sua, lus, 4, lnacc, ltok, lz, 2);
    printf("logits %d/%d %d/%d %d/%d exp2 %.7g\n", lnacc[0], ltok[0], lnacc[1], ltok[1], lnacc[2], ltok[2],
           (double)orc_exp2(-0.5f));
    free(lg);

    free(vdb); free(vtb); free(vdo); free(vto); free(dids); free(tids); free(path); free(map);
    free(dprobs); free(q); free(tprobs); free(ua); free(res); free(sq); free(sp); free(sres);
    printf("done\n");
    return 0;
}
