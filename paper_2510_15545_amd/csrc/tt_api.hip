// C-ABI of the library: argument validation, workspace sizing and launches.
// Every entry point returns a status and never throws; nothing is launched when a
// host-visible argument is invalid.
#include "tt_internal.h"

#ifndef TT_STEP_FUSED
#define TT_STEP_FUSED 1  // 0: tt_step always issues the three calls' kernels
#endif

namespace {

constexpr int32_t kMaxAlignLen = 4096;   // bound on K_b / M_b accepted by tt_align
constexpr int32_t kMaxVerifyLen = 65536; // bound on M_b accepted by tt_verify
constexpr int32_t kMaxHistBins = 8192;   // bins of tt_delta_histogram (its LDS copy: 32 KB)
constexpr int32_t kMaxQuantileDen = 65536;  // denominator of tt_delta_quantile's quantile (int64-exact)
constexpr int32_t kMaxIndexTokens = 1 << 28;  // vocabulary size a token index accepts
constexpr int32_t kMaxTokenBytes = 64;        // longest target token the index and lookups handle
constexpr int32_t kMaxLogitsRow = 1 << 23;     // logits per row tt_verify_logits accepts (64-bit exact sums)
constexpr int32_t kMaxTliRow = 1 << 21;        // target row tt_verify_tli accepts (chunk sums in 16 KB of LDS)
constexpr int32_t kMaxRetokBytes = 4096;      // bytes of S (and tokens of T) per stream: 14 B of LDS each

bool vocab_ok(const tt_vocab *v) {
    return v != nullptr && v->bytes != nullptr && v->offsets != nullptr && v->n_tokens >= 1 &&
           v->max_token_bytes >= 1;
}

}  // namespace

extern "C" {

const char *tt_status_string(int status) {
    switch (status) {
        case TT_OK: return "ok";
        case TT_EINVAL: return "invalid argument";
        case TT_EUNSUPPORTED: return "unsupported configuration";
        case TT_ELAUNCH: return "HIP launch or runtime error";
        case TT_EWORKSPACE: return "workspace missing or too small";
        default: return "unknown status";
    }
}

int tt_version(void) { return 100; }

int tt_align_workspace_size(int32_t n_pairs, int32_t max_k, int32_t max_m, int32_t w,
                            int32_t max_token_bytes, size_t *bytes) {
    if (bytes == nullptr || n_pairs < 0 || max_k < 1 || max_m < 1 || max_k > kMaxAlignLen ||
        max_m > kMaxAlignLen || max_token_bytes < 1)
        return TT_EINVAL;
    const int tb = tt::align_token_slot(max_token_bytes);
    if (tb == 0 || tt::align_lds_bytes(max_k, max_m, w, tb) == 0) return TT_EUNSUPPORTED;
    *bytes = tt::align_workspace_bytes(n_pairs, max_k, max_m, w);
    return TT_OK;
}

int tt_align(const tt_vocab *vd, const tt_vocab *vt, int32_t n_pairs, const int32_t *draft_ids,
             const int32_t *draft_off, const int32_t *target_ids, const int32_t *target_off,
             int32_t max_k, int32_t max_m, int32_t w, int32_t *cost, int32_t *path_len, int32_t *path,
             int32_t *map, void *workspace, size_t workspace_bytes, void *stream) {
    if (!vocab_ok(vd) || !vocab_ok(vt) || n_pairs < 0) return TT_EINVAL;
    if (max_k < 1 || max_m < 1 || max_k > kMaxAlignLen || max_m > kMaxAlignLen) return TT_EINVAL;
    if (n_pairs == 0) return TT_OK;
    if (!draft_ids || !draft_off || !target_ids || !target_off || !cost || !path_len || !path || !map)
        return TT_EINVAL;
    const int32_t mt = vd->max_token_bytes > vt->max_token_bytes ? vd->max_token_bytes : vt->max_token_bytes;
    const int tb = tt::align_token_slot(mt);
    if (tb == 0 || tt::align_lds_bytes(max_k, max_m, w, tb) == 0) return TT_EUNSUPPORTED;
    tt::AlignArgs a;
    a.vd = *vd;
    a.vt = *vt;
    a.n_pairs = n_pairs;
    a.draft_ids = draft_ids;
    a.draft_off = draft_off;
    a.target_ids = target_ids;
    a.target_off = target_off;
    a.max_k = max_k;
    a.max_m = max_m;
    a.w = w;
    a.cost = cost;
    a.path_len = path_len;
    a.path = path;
    a.map = map;
    return tt::launch_align(a, workspace, workspace_bytes, static_cast<hipStream_t>(stream));
}

int tt_transfer(int32_t n_pairs, int32_t v_d, const int32_t *draft_ids, const int32_t *draft_off,
                const int32_t *target_off, const int32_t *map, const float *draft_probs, int64_t draft_ld,
                float *q, void *stream) {
    if (n_pairs < 0 || v_d < 1 || draft_ld < v_d) return TT_EINVAL;
    if (n_pairs == 0) return TT_OK;
    if (!draft_ids || !draft_off || !target_off || !map || !draft_probs || !q) return TT_EINVAL;
    tt::TransferArgs a;
    a.n_pairs = n_pairs;
    a.v_d = v_d;
    a.draft_ids = draft_ids;
    a.draft_off = draft_off;
    a.target_off = target_off;
    a.map = map;
    a.draft_probs = draft_probs;
    a.draft_ld = draft_ld;
    a.q = q;
    return tt::launch_transfer(a, static_cast<hipStream_t>(stream));
}

int tt_verify_workspace_size(int32_t n_streams, int32_t v_t, size_t *bytes) {
    if (bytes == nullptr || n_streams < 0 || v_t < 1) return TT_EINVAL;
    *bytes = tt::verify_layout(n_streams, v_t).total;
    return TT_OK;
}

int tt_verify(int32_t n_streams, int32_t v_t, const int32_t *target_ids, const int32_t *target_off,
              const float *q, const float *target_probs, int64_t target_ld, const float *u_accept,
              const float *u_sample, int32_t max_m, int32_t *n_accepted, int32_t *out_token,
              float *residual, void *workspace, size_t workspace_bytes, void *stream) {
    if (n_streams < 0 || v_t < 1 || target_ld < v_t || max_m < 0 || max_m > kMaxVerifyLen) return TT_EINVAL;
    if (n_streams == 0) return TT_OK;
    if (!target_ids || !target_off || !q || !target_probs || !u_accept || !u_sample || !n_accepted ||
        !out_token)
        return TT_EINVAL;
    tt::VerifyArgs a;
    a.n_streams = n_streams;
    a.v_t = v_t;
    a.target_ids = target_ids;
    a.target_off = target_off;
    a.q = q;
    a.target_probs = target_probs;
    a.target_ld = target_ld;
    a.u_accept = u_accept;
    a.u_sample = u_sample;
    a.max_m = max_m;
    a.n_accepted = n_accepted;
    a.out_token = out_token;
    a.residual = residual;
    a.workspace = workspace;
    a.workspace_bytes = workspace_bytes;
    return tt::launch_verify(a, static_cast<hipStream_t>(stream));
}

int tt_verify_dense(int32_t n_streams, int32_t v, const int32_t *draft_ids, const int32_t *off,
                    const float *draft_probs, int64_t draft_ld, const float *target_probs, int64_t target_ld,
                    const float *u_accept, const float *u_sample, int32_t max_m, int32_t *n_accepted,
                    int32_t *out_token, float *residual, void *workspace, size_t workspace_bytes, void *stream) {
    if (n_streams < 0 || v < 1 || draft_ld < v || target_ld < v || max_m < 0 || max_m > kMaxVerifyLen)
        return TT_EINVAL;
    if (n_streams == 0) return TT_OK;
    if (!draft_ids || !off || !draft_probs || !target_probs || !u_accept || !u_sample || !n_accepted || !out_token)
        return TT_EINVAL;
    tt::VerifyArgs a;
    a.n_streams = n_streams;
    a.v_t = v;
    a.target_ids = draft_ids;  // the proposals verified against the target rows
    a.target_off = off;
    a.q = nullptr;
    a.target_probs = target_probs;
    a.target_ld = target_ld;
    a.u_accept = u_accept;
    a.u_sample = u_sample;
    a.max_m = max_m;
    a.n_accepted = n_accepted;
    a.out_token = out_token;
    a.residual = residual;
    a.workspace = workspace;
    a.workspace_bytes = workspace_bytes;
    a.q_rows = draft_probs;
    a.q_ld = draft_ld;
    return tt::launch_verify(a, static_cast<hipStream_t>(stream));
}

int tt_verify_tli(int32_t n_streams, int32_t v_d, int32_t v_t, const int32_t *d2t, const int32_t *t2d,
                  const int32_t *target_ids, const int32_t *target_off, const float *draft_probs, int64_t draft_ld,
                  const float *draft_mass, const float *target_probs, int64_t target_ld, const float *u_accept,
                  const float *u_sample, int32_t max_m, int32_t *n_accepted, int32_t *out_token, void *stream) {
    if (n_streams < 0 || v_d < 1 || v_t < 1 || draft_ld < v_d || target_ld < v_t || max_m < 0 ||
        max_m > kMaxVerifyLen)
        return TT_EINVAL;
    if (v_t > kMaxTliRow) return TT_EUNSUPPORTED;
    if (n_streams == 0) return TT_OK;
    if (!d2t || !t2d || !target_ids || !target_off || !draft_probs || !target_probs || !u_accept || !u_sample ||
        !n_accepted || !out_token)
        return TT_EINVAL;
    tt::TliVerifyArgs a;
    a.n_streams = n_streams;
    a.v_d = v_d;
    a.v_t = v_t;
    a.d2t = d2t;
    a.t2d = t2d;
    a.target_ids = target_ids;
    a.target_off = target_off;
    a.draft_probs = draft_probs;
    a.draft_ld = draft_ld;
    a.draft_mass = draft_mass;
    a.target_probs = target_probs;
    a.target_ld = target_ld;
    a.u_accept = u_accept;
    a.u_sample = u_sample;
    a.max_m = max_m;
    a.n_accepted = n_accepted;
    a.out_token = out_token;
    return tt::launch_verify_tli(a, static_cast<hipStream_t>(stream));
}

int tt_verify_logits(int32_t n_streams, int32_t v_t, const int32_t *target_ids, const int32_t *target_off,
                     const float *q, const uint16_t *target_logits, int64_t target_ld, const float *inv_temperature,
                     const float *lse, const float *u_accept, const float *u_sample, int32_t max_m,
                     int32_t *n_accepted, int32_t *out_token, void *stream) {
    if (n_streams < 0 || v_t < 1 || target_ld < v_t || max_m < 0 || max_m > kMaxVerifyLen) return TT_EINVAL;
    if (v_t > kMaxLogitsRow) return TT_EUNSUPPORTED;
    if (n_streams == 0) return TT_OK;
    if (!target_ids || !target_off || !q || !target_logits || !inv_temperature || !u_accept || !u_sample ||
        !n_accepted || !out_token)
        return TT_EINVAL;
    tt::LogitsArgs a;
    a.n_streams = n_streams;
    a.v_t = v_t;
    a.target_ids = target_ids;
    a.target_off = target_off;
    a.q = q;
    a.logits = target_logits;
    a.ld = target_ld;
    a.inv_temp = inv_temperature;
    a.lse = lse;
    a.u_accept = u_accept;
    a.u_sample = u_sample;
    a.max_m = max_m;
    a.n_accepted = n_accepted;
    a.out_token = out_token;
    return tt::launch_verify_logits(a, static_cast<hipStream_t>(stream));
}

int tt_delta_histogram(int32_t n_pairs, const int32_t *draft_off, const int32_t *target_off,
                       const int32_t *path_len, const int32_t *path, int32_t n_bins, int32_t *hist, void *stream) {
    if (n_pairs < 0 || n_bins < 1 || n_bins > kMaxHistBins || hist == nullptr) return TT_EINVAL;
    if (n_pairs > 0 && (!draft_off || !target_off || !path_len || !path)) return TT_EINVAL;
    return tt::launch_delta_histogram(n_pairs, draft_off, target_off, path_len, path, n_bins, hist,
                                      static_cast<hipStream_t>(stream));
}

int tt_delta_quantile(const int32_t *hist, int32_t n_bins, int32_t num, int32_t den, int32_t *d_out,
                      void *stream) {
    if (hist == nullptr || d_out == nullptr || n_bins < 1 || n_bins > kMaxHistBins || den < 1 ||
        den > kMaxQuantileDen || num < 0 || num > den)
        return TT_EINVAL;
    return tt::launch_delta_quantile(hist, n_bins, num, den, d_out, static_cast<hipStream_t>(stream));
}

int tt_token_index_size(int32_t n_tokens, size_t *bytes) {
    if (bytes == nullptr || n_tokens < 1 || n_tokens > kMaxIndexTokens) return TT_EINVAL;
    *bytes = tt::token_index_bytes(n_tokens);
    return TT_OK;
}

int tt_token_index_build(const tt_vocab *v, void *index, size_t index_bytes, void *stream) {
    if (!vocab_ok(v) || v->n_tokens > kMaxIndexTokens || index == nullptr) return TT_EINVAL;
    if (v->max_token_bytes > kMaxTokenBytes) return TT_EUNSUPPORTED;
    if ((reinterpret_cast<uintptr_t>(index) & 15u) != 0) return TT_EINVAL;
    if (index_bytes < tt::token_index_bytes(v->n_tokens)) return TT_EWORKSPACE;
    return tt::launch_token_index_build(*v, index, static_cast<hipStream_t>(stream));
}

int tt_vocab_intersection(const tt_vocab *vd, const void *vd_index, size_t vd_index_bytes, const tt_vocab *vt,
                          const void *vt_index, size_t vt_index_bytes, int32_t *d2t, int32_t *t2d, void *stream) {
    if (!vocab_ok(vd) || !vocab_ok(vt) || vd->n_tokens > kMaxIndexTokens || vt->n_tokens > kMaxIndexTokens)
        return TT_EINVAL;
    if (vd->max_token_bytes > kMaxTokenBytes || vt->max_token_bytes > kMaxTokenBytes) return TT_EUNSUPPORTED;
    if (vd_index == nullptr || vt_index == nullptr || (reinterpret_cast<uintptr_t>(vd_index) & 15u) != 0 ||
        (reinterpret_cast<uintptr_t>(vt_index) & 15u) != 0)
        return TT_EINVAL;
    if (vd_index_bytes < tt::token_index_bytes(vd->n_tokens) || vt_index_bytes < tt::token_index_bytes(vt->n_tokens))
        return TT_EINVAL;
    if (d2t == nullptr || t2d == nullptr) return TT_EINVAL;
    return tt::launch_vocab_intersection(*vd, vd_index, *vt, vt_index, d2t, t2d, static_cast<hipStream_t>(stream));
}

int tt_tli_proposal(int32_t n_rows, int32_t v_d, int32_t v_t, const int32_t *d2t, const int32_t *t2d,
                    const float *draft_probs, int64_t draft_ld, float *q_out, int64_t q_ld, void *stream) {
    if (n_rows < 0 || v_d < 1 || v_t < 1 || draft_ld < v_d || q_ld < v_t) return TT_EINVAL;
    if (n_rows == 0) return TT_OK;
    if (!d2t || !t2d || !draft_probs || !q_out) return TT_EINVAL;
    tt::TliArgs a;
    a.n_rows = n_rows;
    a.v_d = v_d;
    a.v_t = v_t;
    a.d2t = d2t;
    a.t2d = t2d;
    a.draft_probs = draft_probs;
    a.draft_ld = draft_ld;
    a.q_out = q_out;
    a.q_ld = q_ld;
    return tt::launch_tli_proposal(a, static_cast<hipStream_t>(stream));
}

int tt_retokenize_workspace_size(int32_t n_streams, int32_t max_m, size_t *bytes) {
    if (bytes == nullptr || n_streams < 0 || max_m < 1 || max_m > kMaxRetokBytes) return TT_EINVAL;
    *bytes = tt::retok_workspace_bytes(n_streams, max_m);
    return TT_OK;
}

int tt_retokenize(const tt_vocab *vd, const tt_vocab *vt, const void *vt_index, size_t index_bytes,
                  int32_t n_streams, const int32_t *draft_ids, const int32_t *draft_off, int32_t max_bytes,
                  int32_t max_m, int32_t *target_ids, int32_t *target_off, void *workspace,
                  size_t workspace_bytes, void *stream) {
    if (!vocab_ok(vd) || !vocab_ok(vt) || vt->n_tokens > kMaxIndexTokens || n_streams < 0) return TT_EINVAL;
    if (max_bytes < 1 || max_bytes > kMaxRetokBytes || max_m < 1 || max_m > kMaxRetokBytes) return TT_EINVAL;
    if (vt->max_token_bytes > kMaxTokenBytes) return TT_EUNSUPPORTED;
    if (vt_index == nullptr || (reinterpret_cast<uintptr_t>(vt_index) & 15u) != 0) return TT_EINVAL;
    if (index_bytes < tt::token_index_bytes(vt->n_tokens)) return TT_EINVAL;
    if (!target_off) return TT_EINVAL;
    if (n_streams > 0 && (!draft_ids || !draft_off || !target_ids)) return TT_EINVAL;
    if (workspace == nullptr || workspace_bytes < tt::retok_workspace_bytes(n_streams, max_m)) return TT_EWORKSPACE;
    tt::RetokArgs a;
    a.vd = *vd;
    a.vt = *vt;
    a.index = vt_index;
    a.n_streams = n_streams;
    a.draft_ids = draft_ids;
    a.draft_off = draft_off;
    a.max_bytes = max_bytes;
    a.max_m = max_m;
    a.target_ids = target_ids;
    a.target_off = target_off;
    a.workspace = workspace;
    return tt::launch_retokenize(a, static_cast<hipStream_t>(stream));
}

int tt_step_workspace_size(int32_t n_streams, int32_t v_t, int32_t max_k, int32_t max_m, int32_t w,
                           int32_t max_token_bytes, size_t *bytes) {
    if (bytes == nullptr || v_t < 1 || max_m > kMaxVerifyLen) return TT_EINVAL;
    size_t ab = 0, vb = 0;
    const int st = tt_align_workspace_size(n_streams, max_k, max_m, w, max_token_bytes, &ab);
    if (st != TT_OK) return st;
    if (tt_verify_workspace_size(n_streams, v_t, &vb) != TT_OK) return TT_EINVAL;
    *bytes = ab > vb ? ab : vb;
    return TT_OK;
}

int tt_step(const tt_vocab *vd, const tt_vocab *vt, int32_t n_streams, int32_t v_d, int32_t v_t,
            const int32_t *draft_ids, const int32_t *draft_off, const int32_t *target_ids,
            const int32_t *target_off, int32_t max_k, int32_t max_m, int32_t w, const float *draft_probs,
            int64_t draft_ld, const float *target_probs, int64_t target_ld, const float *u_accept,
            const float *u_sample, int32_t *cost, int32_t *path_len, int32_t *path, int32_t *map, float *q,
            int32_t *n_accepted, int32_t *out_token, float *residual, void *workspace, size_t workspace_bytes,
            void *stream) {
    // the union of the three calls' host checks, all before anything is launched
    if (!vocab_ok(vd) || !vocab_ok(vt) || n_streams < 0) return TT_EINVAL;
    if (max_k < 1 || max_m < 1 || max_k > kMaxAlignLen || max_m > kMaxAlignLen) return TT_EINVAL;
    if (v_d < 1 || draft_ld < v_d || v_t < 1 || target_ld < v_t || max_m > kMaxVerifyLen) return TT_EINVAL;
    if (n_streams == 0) return TT_OK;
    if (!draft_ids || !draft_off || !target_ids || !target_off || !cost || !path_len || !path || !map ||
        !draft_probs || !q || !target_probs || !u_accept || !u_sample || !n_accepted || !out_token)
        return TT_EINVAL;
    const int32_t mt = vd->max_token_bytes > vt->max_token_bytes ? vd->max_token_bytes : vt->max_token_bytes;
    const int tb = tt::align_token_slot(mt);
    if (tb == 0 || tt::align_lds_bytes(max_k, max_m, w, tb) == 0) return TT_EUNSUPPORTED;
    size_t need = 0;
    if (tt_step_workspace_size(n_streams, v_t, max_k, max_m, w, mt, &need) != TT_OK) return TT_EUNSUPPORTED;
    if (workspace == nullptr || workspace_bytes < need) return TT_EWORKSPACE;

    tt::StepArgs s;
    s.al.vd = *vd;
    s.al.vt = *vt;
    s.al.n_pairs = n_streams;
    s.al.draft_ids = draft_ids;
    s.al.draft_off = draft_off;
    s.al.target_ids = target_ids;
    s.al.target_off = target_off;
    s.al.max_k = max_k;
    s.al.max_m = max_m;
    s.al.w = w;
    s.al.cost = cost;
    s.al.path_len = path_len;
    s.al.path = path;
    s.al.map = map;
    s.tr.n_pairs = n_streams;
    s.tr.v_d = v_d;
    s.tr.draft_ids = draft_ids;
    s.tr.draft_off = draft_off;
    s.tr.target_off = target_off;
    s.tr.map = map;
    s.tr.draft_probs = draft_probs;
    s.tr.draft_ld = draft_ld;
    s.tr.q = q;
    s.ve.n_streams = n_streams;
    s.ve.v_t = v_t;
    s.ve.target_ids = target_ids;
    s.ve.target_off = target_off;
    s.ve.q = q;
    s.ve.target_probs = target_probs;
    s.ve.target_ld = target_ld;
    s.ve.u_accept = u_accept;
    s.ve.u_sample = u_sample;
    s.ve.max_m = max_m;
    s.ve.n_accepted = n_accepted;
    s.ve.out_token = out_token;
    s.ve.residual = residual;
    s.ve.workspace = workspace;
    s.ve.workspace_bytes = workspace_bytes;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (TT_STEP_FUSED && tt::step_fused_fits(s, tb)) return tt::launch_step_fused(s, tb, st);
    if (TT_STEP_FUSED && tt::step_front_fits(s, tb)) return tt::launch_step_front(s, tb, st);
    int rc = tt::launch_align(s.al, workspace, workspace_bytes, st);
    if (rc == TT_OK) rc = tt::launch_transfer(s.tr, st);
    if (rc == TT_OK) rc = tt::launch_verify(s.ve, st);
    return rc;
}

}  // extern "C"
