/*
 * tt.h -- TokenTiming verification hot path on AMD Instinct MI355X (gfx950).
 *
 * TokenTiming lets a draft model with vocabulary V_d propose tokens to a target
 * model with a different vocabulary V_t.  Per decode step and per stream:
 *   - the K draft tokens D are re-encoded into M proxy target tokens T with the
 *     same bytes (Sec. 4.2.1, App. A.1; done by the caller's tokenizer);
 *   - tt_align     Dynamic Token Warping aligns D with T (Sec. 4.1, Alg. 1) and
 *                  maps every target position to a draft position (App. A.2);
 *   - tt_transfer  gathers the draft probability of the aligned draft token for
 *                  every target position (Alg. 2 "MapProbabilities", App. A.2);
 *   - tt_verify    runs the speculative acceptance test on the target
 *                  probabilities and samples the next token from the residual
 *                  or bonus distribution (Sec. 3, Sec. 4.2.2-4.2.3, App. D Alg. 4).
 *
 * Conventions shared by every call
 *   - Every array pointer is a DEVICE pointer owned by the caller (e.g. a torch
 *     tensor's data_ptr()).  The library never allocates, frees or keeps them.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL is
 *     the default stream).  Nothing synchronises the host.
 *   - Calls return a status (TT_OK or a negative TT_E* code) and never throw.
 *     Host-visible argument errors are reported before anything is launched.
 *   - Errors only the device can see (a stream whose length is outside the
 *     caller's stated bound, an id outside its vocabulary) do not fail the call:
 *     that stream gets sentinel outputs (cost = -1, n_accepted = -1,
 *     out_token = -1, map = -1, q = NaN) and the other streams are unaffected.
 *   - Batches are CSR: stream b owns ids[off[b] .. off[b+1]).  Offsets are
 *     non-decreasing int32 with off[0] = 0.
 *   - The library holds no global state; calls on distinct workspaces are
 *     reentrant.
 */
#ifndef TT_H
#define TT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    TT_OK = 0,
    TT_EINVAL = -1,        /* null pointer, negative size, inconsistent scalar */
    TT_EUNSUPPORTED = -2,  /* valid request outside what the kernels implement */
    TT_ELAUNCH = -3,       /* the HIP runtime reported an error */
    TT_EWORKSPACE = -4     /* workspace missing or smaller than required */
};

/* Human-readable text for a status code (static storage, never NULL). */
const char *tt_status_string(int status);

/* Library version, major * 10000 + minor * 100 + patch. */
int tt_version(void);

/*
 * Token byte table (Sec. 4.1 token distance over UTF-8 bytes, App. H).
 * Token t is bytes[offsets[t] .. offsets[t+1]).  `bytes` and `offsets` are
 * device pointers; `offsets` has n_tokens + 1 entries.  max_token_bytes is an
 * upper bound on every token's length (1..64); a token found longer than it on
 * the device makes its pair a sentinel pair.
 */
typedef struct {
    const uint8_t *bytes;
    const int32_t *offsets;
    int32_t n_tokens;
    int32_t max_token_bytes;
} tt_vocab;

/*
 * Workspace bytes tt_align needs for these bounds: 0 when max_k <= 64 and
 * max_m <= 64 (each pair's working set stays in LDS), otherwise room for the
 * 2-bit predecessor codes of every pair's band (n_pairs * max_k *
 * (ceil(min(max_m, 2 L + 1) / 16) + 1) * 4 bytes, L the largest band half-width
 * the bounds allow), rounded up to 256 bytes and followed, for 2 to 2,048 pairs, by
 * one int per pair: the order in which the pairs are dispatched (descending band
 * work, so the longest pairs start first).  Returns TT_EUNSUPPORTED when the bounds need more LDS than
 * one MI355X workgroup can hold (token bytes (max_k + max_m) * slot, the slot
 * being max_token_bytes rounded up to 8, 16, 32 or 64, plus
 * 9 * (max_k + max_m) + about 11 KB).
 */
int tt_align_workspace_size(int32_t n_pairs, int32_t max_k, int32_t max_m, int32_t w,
                            int32_t max_token_bytes, size_t *bytes);

/*
 * tt_align -- Dynamic Token Warping (Sec. 4.1, Alg. 1) with the byte-level
 * Levenshtein token distance (App. H) and the Sakoe-Chiba band |i - j| <= w,
 * followed by the backtrack to the optimal path and the mapping of App. A.2.
 *
 *   vd, vt         draft / target token tables (host structs, device arrays)
 *   n_pairs        number of (draft, proxy target) sequence pairs, >= 0
 *   draft_ids      [sum K_b] draft token ids, CSR by draft_off[n_pairs + 1]
 *   target_ids     [sum M_b] proxy target ids, CSR by target_off[n_pairs + 1]
 *   max_k, max_m   bounds on K_b and M_b (1..4096); a pair with K_b or M_b
 *                  outside [1, bound] gets sentinel outputs
 *   w              band half-width; w < 0 means no band.  When |K_b - M_b| > w
 *                  the band is widened to |K_b - M_b| so the corner (K_b, M_b)
 *                  stays reachable.
 * Outputs (device):
 *   cost[b]        C* = C(K_b, M_b), sum of token distances along the path
 *   path_len[b]    number of cells on the optimal path (max(K,M)..K+M-1)
 *   path           int32 (i, j) pairs, 0-based, in forward order; pair b's
 *                  cells start at int32 index 2*(draft_off[b] + target_off[b])
 *                  (room for K_b + M_b cells per pair: size 2*(sum K + sum M))
 *   map            [sum M_b]: for target position j the largest draft index i
 *                  with (i, j) on the path (the terminal draft token of a
 *                  many-to-one block, the shared token of a one-to-many block)
 * Ties between equally cheap predecessors go to the diagonal step, then to
 * (i-1, j), then to (i, j-1).
 * workspace: device memory of tt_align_workspace_size bytes (may be NULL / 0 when
 * that size is 0); no initialisation needed; calls that overlap in time must not
 * share it.  TT_EWORKSPACE if it is missing or too small.
 */
int tt_align(const tt_vocab *vd, const tt_vocab *vt, int32_t n_pairs,
             const int32_t *draft_ids, const int32_t *draft_off,
             const int32_t *target_ids, const int32_t *target_off,
             int32_t max_k, int32_t max_m, int32_t w,
             int32_t *cost, int32_t *path_len, int32_t *path, int32_t *map,
             void *workspace, size_t workspace_bytes, void *stream);

/*
 * tt_transfer -- draft probabilities onto target positions (Alg. 2
 * "MapProbabilities", App. A.2 cases 1-2, Limitations: one-hot form).
 *
 *   q[target_off[b] + j] = draft_probs[(draft_off[b] + i) * draft_ld + d_i]
 *   with i = map[target_off[b] + j] and d_i = draft_ids[draft_off[b] + i],
 * i.e. the probability the draft model gave to the token it emitted at the
 * aligned draft position.  draft_probs is fp32 with one row of width >= v_d per
 * draft position (row stride draft_ld >= v_d elements).  i outside [0, K_b) or
 * d_i outside [0, v_d) gives q = NaN (a NaN proposal is always rejected).
 */
int tt_transfer(int32_t n_pairs, int32_t v_d,
                const int32_t *draft_ids, const int32_t *draft_off,
                const int32_t *target_off, const int32_t *map,
                const float *draft_probs, int64_t draft_ld,
                float *q, void *stream);

/* Workspace bytes tt_verify needs for n_streams rows of width v_t. */
int tt_verify_workspace_size(int32_t n_streams, int32_t v_t, size_t *bytes);

/*
 * tt_verify -- lossless speculative sampling over the full target vocabulary
 * (Sec. 3 "Standard Speculative Sampling", Sec. 4.2.2 acceptance rule,
 * Sec. 4.2.3 / Alg. 2 next-token sample, App. D Alg. 4 residual distribution).
 *
 * Inputs (device):
 *   target_ids   [sum M_b] proxy target tokens (CSR by target_off), ids index
 *                the target rows and must lie in [0, v_t)
 *   q            [sum M_b] transferred draft probabilities (tt_transfer)
 *   target_probs fp32 rows of width v_t, stride target_ld >= v_t elements;
 *                stream b owns M_b + 1 consecutive rows starting at row
 *                target_off[b] + b: row j is the target distribution after
 *                accepting t_1..t_j (row M_b is the bonus row)
 *   u_accept     [sum M_b] uniforms in [0,1) for the acceptance tests
 *   u_sample     [n_streams] uniforms in [0,1) for the final sample
 *   max_m        bound on M_b (0..65536); a stream outside [0, max_m] or with an
 *                id outside [0, v_t) gets sentinel outputs
 * Outputs (device):
 *   n_accepted[b]  gamma: t_j is accepted while u_j < P_t(t_j) / q_j (fp32,
 *                  round-to-nearest; q_j <= 0 always accepts), stopping at the
 *                  first rejection
 *   out_token[b]   next token: with r = gamma, sampled from
 *                  R(x) = max(0, P_t[r](x) - q_r [x == t_r]) if r < M_b
 *                  (rejection), or from P_t[M_b] (all accepted).  R is clamped
 *                  to [0,1] (NaN counts as 0), quantised to Q62 fixed point by
 *                  truncation, Z = sum, T = floor(u_sample * Z) exactly, and the
 *                  token is the first index whose inclusive prefix sum exceeds T.
 *                  If Z = 0 the token is the first maximum of the row.
 *   residual       optional (may be NULL): [n_streams x target_ld] fp32, row b
 *                  receives R(x) / Z_f (Z_f = Z * 2^-62 rounded to fp32) for
 *                  x < v_t, or a one-hot row at out_token when Z = 0.
 * Rows are expected to be probability distributions (entries in [0,1], sum
 * about 1); a row whose Q62 mass exceeds 2^64 gives an in-range but
 * unspecified token.
 * workspace: device memory of tt_verify_workspace_size bytes (per-chunk Q62
 * sums and per-stream scratch); it needs no initialisation.  Calls that overlap
 * in time must not share it.
 * Launches: with at least 256 streams (one per compute unit) and rows of at most
 * 2,097,152 floats, one kernel with a workgroup per stream; otherwise one streaming kernel
 * over B x S workgroups and one sampling kernel.  If residual != NULL, one more
 * kernel writes the residual rows.
 */
int tt_verify(int32_t n_streams, int32_t v_t,
              const int32_t *target_ids, const int32_t *target_off, const float *q,
              const float *target_probs, int64_t target_ld,
              const float *u_accept, const float *u_sample, int32_t max_m,
              int32_t *n_accepted, int32_t *out_token, float *residual,
              void *workspace, size_t workspace_bytes, void *stream);

/*
 * tt_verify_noalloc -- tt_verify for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments, kernels and results, without the workspace.
 * Its scratch is a device array of 8 MiB inside the library; each GPU the library
 * runs on holds its own copy until the process ends.  Batches whose workspace
 * (tt_verify_workspace_size) exceeds 8 MiB are refused with TT_EWORKSPACE (for
 * example 4,096 streams at v_t = 151,936 fit, 8,192 do not).  Nothing is
 * allocated: no hipMalloc, hipFree or allocating library call.  Every call on one
 * GPU shares that GPU's scratch, so calls that overlap in time on one GPU race;
 * calls in one stream (or otherwise ordered) do not.  TT_ELAUNCH if the scratch's
 * device address cannot be found.
 */
int tt_verify_noalloc(int32_t n_streams, int32_t v_t,
                      const int32_t *target_ids, const int32_t *target_off, const float *q,
                      const float *target_probs, int64_t target_ld,
                      const float *u_accept, const float *u_sample, int32_t max_m,
                      int32_t *n_accepted, int32_t *out_token, float *residual, void *stream);

/*
 * tt_verify_dense -- standard speculative sampling with dense proposals over one
 * vocabulary (App. D Alg. 4; the homogeneous-vocabulary case, where the draft
 * model's whole distribution over the target's tokens is the proposal).  It is
 * tt_verify with the one-hot transferred mass q_j replaced by a full draft row.
 *
 * Inputs (device):
 *   draft_ids    [sum M_b] drafted tokens x_j (CSR by off), ids in [0, v)
 *   off          [n_streams + 1] CSR offsets, M_b = off[b+1] - off[b]
 *   draft_probs  fp32 rows of width v, stride draft_ld >= v elements; row
 *                off[b] + j is the distribution q_j that x_j was drawn from
 *   target_probs fp32 rows of width v, stride target_ld >= v; stream b owns the
 *                M_b + 1 rows starting at row off[b] + b (row j: the target's
 *                distribution after x_1..x_j; row M_b is the bonus row)
 *   u_accept     [sum M_b] uniforms in [0,1), u_sample [n_streams] in [0,1)
 *   max_m        bound on M_b (0..65536); a stream outside [0, max_m] or with an
 *                id outside [0, v) gets n_accepted = out_token = -1
 * Outputs (device):
 *   n_accepted[b]  gamma: x_j is kept while u_j < p_j(x_j) / q_j(x_j) (fp32,
 *                  round-to-nearest; q_j(x_j) <= 0 keeps it), stopping at the
 *                  first rejection
 *   out_token[b]   with r = gamma, a sample of R(x) = max(0, p_r(x) - q_r(x))
 *                  if r < M_b, or of p_{M_b}(x) if every draft was kept; R is
 *                  clamped, quantised and sampled exactly as in tt_verify
 *   residual       optional (may be NULL): [n_streams x target_ld] fp32, the
 *                  normalised R as in tt_verify
 * workspace: tt_verify_workspace_size(n_streams, v) bytes, no initialisation;
 * calls that overlap in time must not share it.  Same launch shapes as
 * tt_verify; a rejected stream reads its target row and its draft row once each.
 */
int tt_verify_dense(int32_t n_streams, int32_t v,
                    const int32_t *draft_ids, const int32_t *off,
                    const float *draft_probs, int64_t draft_ld,
                    const float *target_probs, int64_t target_ld,
                    const float *u_accept, const float *u_sample, int32_t max_m,
                    int32_t *n_accepted, int32_t *out_token, float *residual,
                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * tt_verify_logits -- tt_verify with the target distributions given as bf16 logits and a
 * per-stream sampling temperature (App. F) instead of fp32 probability rows: the softmax
 * of Sec. 3's acceptance rule and of the residual (App. D Alg. 4) is formed inside.
 *
 * Inputs (device): target_ids, target_off, q, u_accept, u_sample as for tt_verify;
 * target_logits: bf16 bit patterns, row target_off[b] + b + j (j in [0, M_b]) at a stride
 * of target_ld elements; inv_temperature[n_streams] fp32 (1 / T, > 0).  max_m as for
 * tt_verify.  Outputs (device): n_accepted, out_token as for tt_verify (no residual rows).
 * Arithmetic, all of it order-independent, in base 2: c = inv_temperature * log2(e) (fp32);
 * y = logit * c (NaN counts as minus infinity); mu = the row's largest y; the scaled exponent
 * z = fma(logit, c, fp32(31 - mu)) held in [-1, 31]; 2^z = p * 2^k with k = rint(z) and p the
 * degree-5 Taylor polynomial of 2^(z - k) (coefficients (ln 2)^n / n! in fp32, Horner with
 * fused multiply-adds); the weight e31 = floor(p * 2^k) (Q31), summed exactly;
 * S = that sum * 2^-31 rounded once to fp32; E = p * 2^(k - 31) (0 for z < 0);
 * P_t(t_j) = E(t_j) / S in fp32; accept while q_j <= 0 or u_j < P_t(t_j) / q_j; after a
 * rejection at r the residual is the row's e31 with the entry at t_r replaced by
 * floor(clamp(E(t_r) - q_r * S, 0, 1) * 2^31), after full acceptance the bonus row's e31;
 * the token is the first index whose prefix exceeds floor(u_sample * Z) (the first largest
 * y when Z = 0).  A stream with M_b outside [0, max_m], an id outside [0, v_t) or
 * inv_temperature <= 0 gets n_accepted = out_token = -1.
 * lse (device, optional, one fp32 per logits row): the row's log-sum-exp of logit *
 * inv_temperature, as an LM head can emit it with its logits.  When given, mu = lse * log2(e)
 * and S = 1 (P = clamp(E, 0, 1), the residual entry at t_r is floor(clamp(P(t_r) - q_r, 0, 1)
 * * 2^31)): the acceptance test reads one logit per position and only the residual (or bonus)
 * row is read, once.  Without it each stream reads its rows 0 .. gamma twice (max, then
 * sums), one after another.
 * One kernel on `stream`, a workgroup per stream; no workspace.
 * TT_EINVAL on a bad size or a missing pointer, TT_EUNSUPPORTED for v_t > 2^23.
 */
int tt_verify_logits(int32_t n_streams, int32_t v_t, const int32_t *target_ids, const int32_t *target_off,
                     const float *q, const uint16_t *target_logits, int64_t target_ld,
                     const float *inv_temperature, const float *lse, const float *u_accept,
                     const float *u_sample, int32_t max_m, int32_t *n_accepted, int32_t *out_token,
                     void *stream);

/*
 * tt_delta_histogram -- position deviation of the matched tokens of aligned pairs
 * (Sec. 5 "DTW Bridges the Gap", Fig. CDF; App. K "Settings of w").  A cell (i, j)
 * of an optimal warping path matches draft token i with proxy target token j; it
 * deviates by |i - j| positions.  App. K aligns without a band (w < 0), reads the
 * offset where the CDF of this deviation reaches 0.9 and searches w below it.
 *
 * Inputs (device): draft_off, target_off, path_len and path exactly as tt_align
 * wrote them (pair b's path_len[b] cells start at int32 index
 * 2*(draft_off[b] + target_off[b])); a pair with path_len[b] <= 0 (a sentinel) or
 * longer than K_b + M_b contributes nothing.
 * Output (device): hist[n_bins] int32, overwritten: hist[d] = number of cells with
 * |i - j| = d for d < n_bins - 1, hist[n_bins - 1] = number with |i - j| >= n_bins - 1.
 * n_bins in [1, 8192].  Two kernels on `stream` (a fill, then the count); the
 * counts do not depend on scheduling.  TT_EINVAL on a bad size or a missing pointer.
 */
int tt_delta_histogram(int32_t n_pairs, const int32_t *draft_off, const int32_t *target_off,
                       const int32_t *path_len, const int32_t *path, int32_t n_bins,
                       int32_t *hist, void *stream);

/*
 * tt_delta_quantile -- App. K "Settings of w": where the cumulative distribution of
 * the deviation counted by tt_delta_histogram reaches a quantile (the paper reads it
 * at 0.9 from an alignment without a band and searches w at or below it).
 *
 * Inputs: hist[n_bins] int32 counts (device), n_bins in [1, 8192]; the quantile as a
 * fraction num/den of host integers, 0 <= num <= den, 1 <= den <= 65536 (0.9 is 9/10).
 * Output (device): *d_out = the smallest d with
 *     (hist[0] + ... + hist[d]) * den >= num * (hist[0] + ... + hist[n_bins - 1]),
 * compared exactly in 64-bit integers; 0 when the counts sum to 0.  d_out = n_bins - 1
 * means the deviation at the quantile is at least n_bins - 1 (the overflow bin).
 * One kernel on `stream`; nothing is allocated.  TT_EINVAL on a missing pointer or an
 * argument outside these ranges.
 */
int tt_delta_quantile(const int32_t *hist, int32_t n_bins, int32_t num, int32_t den, int32_t *d_out,
                      void *stream);

/*
 * Token index for longest-match lookups in a vocabulary (used by tt_retokenize for
 * the target vocabulary).  tt_token_index_size gives its bytes for n_tokens
 * (16 bytes per hash slot, a power of two >= 4 * n_tokens slots, then a filter of
 * 2 bits per slot that lets a lookup skip most byte strings that are no token);
 * n_tokens in [1, 2^28].  tt_token_index_build fills `index` (device, 16-byte aligned, at
 * least that many bytes, owned by the caller) from the table `v` in three kernels
 * on `stream`; tokens of length 0 or above v->max_token_bytes are left out, and of
 * several tokens with the same bytes only the lowest id can be found.  The index
 * stays valid while the table's device arrays are unchanged.  TT_EUNSUPPORTED if
 * v->max_token_bytes > 64, TT_EWORKSPACE if index_bytes is too small.
 */
int tt_token_index_size(int32_t n_tokens, size_t *bytes);
int tt_token_index_build(const tt_vocab *v, void *index, size_t index_bytes, void *stream);

/* Workspace bytes tt_retokenize needs: a count and max_m ids per stream. */
int tt_retokenize_workspace_size(int32_t n_streams, int32_t max_m, size_t *bytes);

/*
 * tt_retokenize -- proxy target tokens from the draft tokens (Sec. 4.2.1 "Draft Token
 * Calculation": S = Tokenizer_d.encode(D), T = Tokenizer_t.decode(S), also the
 * first lines of Alg. 2's loop; App. A.1: T spells the same string as D).  The
 * target tokenizer is greedy longest match over byte strings: S is the
 * concatenation of the draft tokens' bytes, and from its start the longest target
 * token that is a prefix of the rest of S is emitted (the lowest id among tokens
 * with equal bytes) until S is consumed.
 *
 * Inputs (device unless noted): vd, vt token tables (host structs); vt_index built
 * by tt_token_index_build for vt (index_bytes, host, its size); draft_ids /
 * draft_off CSR as for tt_align; max_bytes (host, 1..4096) bounds |S| per stream
 * and max_m (host, 1..4096) bounds |T|.
 * Outputs (device): target_off[n_streams + 1] CSR offsets and target_ids packed by
 * them (capacity n_streams * max_m ints is always enough).  A stream with a draft id
 * outside vd, |S| > max_bytes, more than max_m target tokens, or a byte of S that no
 * target token starts with gets zero tokens (target_off[b+1] = target_off[b]), which
 * tt_align then treats as a sentinel pair.
 * workspace: tt_retokenize_workspace_size bytes, no initialisation; calls that
 * overlap in time must not share it.  Two kernels up to 2,048 streams (one workgroup
 * per stream, then one that places and packs the ids), three beyond (the offsets get
 * a kernel of their own).
 */
int tt_retokenize(const tt_vocab *vd, const tt_vocab *vt, const void *vt_index, size_t index_bytes,
                  int32_t n_streams, const int32_t *draft_ids, const int32_t *draft_off,
                  int32_t max_bytes, int32_t max_m,
                  int32_t *target_ids, int32_t *target_off,
                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * tt_vocab_intersection -- the vocabulary intersection of the Token-Level
 * Intersection proposal (App. D Alg. 3, the set T ∩ D), each vocabulary taken as a
 * set of byte strings.
 *
 * Inputs: vd, vt token tables (host structs over device arrays) and their token
 * indexes vd_index, vt_index (device, built by tt_token_index_build from the same
 * tables; *_index_bytes their sizes, host).
 * Outputs (device, owned by the caller): d2t[vd->n_tokens] holds, for draft id x, the
 * id of the target token with the same bytes (the lowest such id), or -1 when vt has
 * no such token, x is not the lowest draft id holding its bytes, or x's length is 0
 * or above vd->max_token_bytes; t2d[vt->n_tokens] is the converse (d2t[x] = y exactly
 * when t2d[y] = x).
 * Two kernels on `stream`, no workspace.  TT_EINVAL for a missing or misaligned
 * pointer or an index smaller than tt_token_index_size gives, TT_EUNSUPPORTED if a
 * table's max_token_bytes is above 64.
 */
int tt_vocab_intersection(const tt_vocab *vd, const void *vd_index, size_t vd_index_bytes,
                          const tt_vocab *vt, const void *vt_index, size_t vt_index_bytes,
                          int32_t *d2t, int32_t *t2d, void *stream);

/*
 * tt_tli_proposal -- q' of App. D Alg. 3 for n_rows draft distributions: q'(y) =
 * q(x) / S where y = d2t[x] (x in the intersection), 0 at every other target id, and
 * S the mass q puts on the intersection.  Standard speculative sampling then runs
 * with q' as the dense proposal (tt_verify_dense).
 *
 * Inputs (device): d2t[v_d] and t2d[v_t] from tt_vocab_intersection (an entry of
 * t2d outside [0, v_d) counts as -1); draft_probs,
 * n_rows rows of v_d floats at a stride of draft_ld floats.  Output (device): q_out,
 * n_rows rows of v_t floats at a stride of q_ld floats, every element written.
 * q is clamped to [0, 1] (NaN -> 0); S is the sum of the intersected q(x), each
 * truncated to a multiple of 2^-62, formed exactly and rounded once to the nearest
 * fp32 (ties to even); q'(y) is the fp32 quotient.  A row with S = 0 is written as
 * zeros.  One kernel on `stream` (a workgroup per row), no workspace.  TT_EINVAL for
 * n_rows < 0, v_d or v_t < 1, a stride below its row length or a missing pointer.
 */
int tt_tli_proposal(int32_t n_rows, int32_t v_d, int32_t v_t, const int32_t *d2t, const int32_t *t2d,
                    const float *draft_probs, int64_t draft_ld, float *q_out, int64_t q_ld, void *stream);

/*
 * tt_verify_tli -- standard speculative sampling with the Token-Level Intersection
 * proposal (App. D Alg. 3 feeding Alg. 4) in one call, the proposal rows formed where they
 * are used instead of written: the result is that of tt_tli_proposal on the drafted
 * positions' rows followed by tt_verify_dense on its output, bit for bit.
 *
 * Inputs (device): d2t[v_d], t2d[v_t] from tt_vocab_intersection; target_ids / target_off
 * CSR proposals y_j (target ids, drawn from q'_j) as for tt_verify_dense; draft_probs: row
 * target_off[b] + j (stride draft_ld >= v_d floats) is the draft distribution q_j over
 * V_d; draft_mass (optional, may be NULL): one fp32 per draft row, S_j, the mass q_j puts
 * on the intersection as the drafter formed it when it normalised q'_j -- when NULL, S_j
 * is formed exactly as tt_tli_proposal forms it; target_probs: stream b owns the M_b + 1
 * rows from row target_off[b] + b (stride target_ld >= v_t); u_accept, u_sample, max_m as
 * for tt_verify_dense.
 * Proposal: q'_j(y) = clamp(q_j(t2d[y]), 0, 1) / S_j when t2d[y] lies in [0, v_d) and S_j > 0,
 * else 0.  Outputs (device): n_accepted, out_token as tt_verify_dense gives them for the
 * rows q'_j (a stream with M_b outside [0, max_m] or an id outside [0, v_t) gets -1, -1).
 * Reads: one gathered draft mass per tested position (with draft_mass; without it, draft
 * row j in full for every tested position, one after another), then target row gamma and,
 * after a rejection, the masses of draft row gamma gathered through t2d.  One kernel on
 * `stream`, a workgroup per stream, no workspace.  TT_EINVAL on a bad size or a missing
 * pointer, TT_EUNSUPPORTED for v_t > 2^21.
 */
int tt_verify_tli(int32_t n_streams, int32_t v_d, int32_t v_t, const int32_t *d2t, const int32_t *t2d,
                  const int32_t *target_ids, const int32_t *target_off, const float *draft_probs, int64_t draft_ld,
                  const float *draft_mass, const float *target_probs, int64_t target_ld, const float *u_accept,
                  const float *u_sample, int32_t max_m, int32_t *n_accepted, int32_t *out_token, void *stream);

/*
 * Workspace bytes tt_step needs: the larger of tt_align_workspace_size and
 * tt_verify_workspace_size for the same arguments (the two stages run one after
 * the other and share it).
 */
int tt_step_workspace_size(int32_t n_streams, int32_t v_t, int32_t max_k, int32_t max_m, int32_t w,
                           int32_t max_token_bytes, size_t *bytes);

/*
 * tt_step -- the whole verification path of one decode step: tt_align, then
 * tt_transfer, then tt_verify, with the same arguments and the same outputs as
 * those three calls made in sequence on `stream` (the target ids that are
 * aligned are also the ids verified against the target rows, and max_m bounds
 * both stages).  Sec. 4.1 / Alg. 1 / App. H (alignment), Alg. 2 / App. A.2
 * (transfer), Sec. 3, Sec. 4.2.2-4.2.3, App. D Alg. 4 (verification).
 *
 * When max_k <= 64, max_m <= 64, and either n_streams >= 256 with verify rows of
 * at most 2,097,152 floats or v_t <= 16384 (short rows, any batch size), the path runs as
 * ONE kernel with a workgroup per stream: the
 * pair is aligned in LDS, map and q never leave the chip before they are used,
 * and the selected target row is read once.  Other batches of pairs with
 * K, M <= 64 run that kernel up to the acceptance scan (alignment, transfer, gamma)
 * followed by the split verification kernels of tt_verify; larger pairs issue the
 * three calls' kernels in order.  Every output array (cost, path_len, path, map, q,
 * n_accepted, out_token, residual) is written exactly as by the three calls.
 * workspace: tt_step_workspace_size bytes, no initialisation needed.
 */
int tt_step(const tt_vocab *vd, const tt_vocab *vt, int32_t n_streams, int32_t v_d, int32_t v_t,
            const int32_t *draft_ids, const int32_t *draft_off,
            const int32_t *target_ids, const int32_t *target_off,
            int32_t max_k, int32_t max_m, int32_t w,
            const float *draft_probs, int64_t draft_ld,
            const float *target_probs, int64_t target_ld,
            const float *u_accept, const float *u_sample,
            int32_t *cost, int32_t *path_len, int32_t *path, int32_t *map, float *q,
            int32_t *n_accepted, int32_t *out_token, float *residual,
            void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* TT_H */
