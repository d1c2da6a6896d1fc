// Internal declarations shared by the library's translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "tt.h"

namespace tt {

// ---------------------------------------------------------------- alignment (dtw.hip)
struct AlignArgs {
    tt_vocab vd, vt;
    int32_t n_pairs;
    const int32_t *draft_ids, *draft_off, *target_ids, *target_off;
    int32_t max_k, max_m, w;
    int32_t *cost, *path_len, *path, *map;
};

// LDS bytes one alignment workgroup needs for these bounds; 0 if they exceed the
// per-workgroup LDS of gfx950.  `tb` is the token slot width chosen for the vocabularies.
size_t align_lds_bytes(int32_t max_k, int32_t max_m, int32_t w, int tb);
int align_token_slot(int32_t max_token_bytes);  // 8, 16, 32 or 64; 0 if unsupported
// Global workspace for the direction codes of finished 64-row strips (0 if max_k <= 64).
size_t align_workspace_bytes(int32_t n_pairs, int32_t max_k, int32_t max_m, int32_t w);
int launch_align(const AlignArgs &a, void *workspace, size_t workspace_bytes, hipStream_t stream);
// Row-scan kernel for short pairs (dtw_rows.hip): used when max_k and max_m are both <= 64.
bool align_rows_fits(int32_t max_k, int32_t max_m);
int launch_align_rows(const AlignArgs &a, int tb, hipStream_t stream);

// ---------------------------------------------------------------- transfer (transfer.hip)
struct TransferArgs {
    int32_t n_pairs, v_d;
    const int32_t *draft_ids, *draft_off, *target_off, *map;
    const float *draft_probs;
    int64_t draft_ld;
    float *q;
};
int launch_transfer(const TransferArgs &a, hipStream_t stream);

// ---------------------------------------------------------------- verify (verify.hip)
struct VerifyArgs {
    int32_t n_streams, v_t;
    const int32_t *target_ids, *target_off;
    const float *q, *target_probs;
    int64_t target_ld;
    const float *u_accept, *u_sample;
    int32_t max_m;
    int32_t *n_accepted, *out_token;
    float *residual;
    void *workspace;
    size_t workspace_bytes;
    // Dense proposals (tt_verify_dense): row target_off[b] + j of q_rows is the draft
    // distribution of position j over the same vocabulary; null for the one-hot proposal q.
    const float *q_rows = nullptr;
    int64_t q_ld = 0;
};

// Workspace layout for tt_verify: Q62 mass Z and selected row r per stream, Q62 sums of
// every 1024-float chunk of every stream's row.
struct VerifyLayout {
    size_t zsum, rsel, partials, total;
    int32_t n_chunks;
};
VerifyLayout verify_layout(int32_t n_streams, int32_t v_t);
int launch_verify(const VerifyArgs &a, hipStream_t stream);  // one-hot or dense by a.q_rows
// True when tt_verify runs one workgroup per stream (enough streams to fill the chip and
// the row's chunk sums fit in LDS); the fused step kernel uses the same shape.
bool verify_row_path(int32_t n_streams, int32_t v_t);
// Normalised residual rows from Z and r in the workspace (written by a previous launch).
int launch_verify_residual(const VerifyArgs &a, hipStream_t stream);
// The split path's streaming and sampling for the one-hot proposal with gamma already in the
// workspace (rsel, -1 for sentinel streams whose outputs are written), then the residual rows.
int launch_verify_after_gamma(const VerifyArgs &a, hipStream_t stream);

// ---------------------------------------------------------------- deviation histogram (delta.hip)
int launch_delta_histogram(int32_t n_pairs, const int32_t *draft_off, const int32_t *target_off,
                           const int32_t *path_len, const int32_t *path, int32_t n_bins, int32_t *hist,
                           hipStream_t stream);
int launch_delta_quantile(const int32_t *hist, int32_t n_bins, int32_t num, int32_t den, int32_t *d_out,
                          hipStream_t stream);

// ---------------------------------------------------------------- re-tokenisation (retok.hip)
uint32_t token_index_capacity(int32_t n_tokens);  // hash slots for a vocabulary of n_tokens
size_t token_index_bytes(int32_t n_tokens);
int launch_token_index_build(const tt_vocab &v, void *index, hipStream_t stream);
struct RetokArgs {
    tt_vocab vd, vt;
    const void *index;  // token index of vt (launch_token_index_build)
    int32_t n_streams;
    const int32_t *draft_ids, *draft_off;
    int32_t max_bytes, max_m;
    int32_t *target_ids, *target_off;
    void *workspace;
};
size_t retok_workspace_bytes(int32_t n_streams, int32_t max_m);
// d2t / t2d of the vocabulary intersection from the two tables' token indexes.
int launch_vocab_intersection(const tt_vocab &vd, const void *vd_index, const tt_vocab &vt, const void *vt_index,
                              int32_t *d2t, int32_t *t2d, hipStream_t stream);

// ---------------------------------------------------------------- verification from logits (logits.hip)
struct LogitsArgs {
    int32_t n_streams, v_t;
    const int32_t *target_ids, *target_off;
    const float *q;
    const uint16_t *logits;  // bf16 bit patterns
    int64_t ld;
    const float *inv_temp, *u_accept, *u_sample;
    const float *lse;  // per-row log-sum-exp of x, or nullptr
    int32_t max_m;
    int32_t *n_accepted, *out_token;
};
int launch_verify_logits(const LogitsArgs &a, hipStream_t stream);

// ---------------------------------------------------------------- TLI proposal rows (tli.hip)
struct TliArgs {
    int32_t n_rows, v_d, v_t;
    const int32_t *d2t, *t2d;
    const float *draft_probs;
    int64_t draft_ld;
    float *q_out;
    int64_t q_ld;
};
int launch_tli_proposal(const TliArgs &a, hipStream_t stream);
// Verification with the TLI proposal formed on the fly (tt_verify_tli): the proposal of
// position j is q' of draft row target_off[b] + j, with S from draft_mass when given.
struct TliVerifyArgs {
    int32_t n_streams, v_d, v_t;
    const int32_t *d2t, *t2d;
    const int32_t *target_ids, *target_off;
    const float *draft_probs;
    int64_t draft_ld;
    const float *draft_mass;  // per draft row, or null: formed as tt_tli_proposal forms it
    const float *target_probs;
    int64_t target_ld;
    const float *u_accept, *u_sample;
    int32_t max_m;
    int32_t *n_accepted, *out_token;
};
int launch_verify_tli(const TliVerifyArgs &a, hipStream_t stream);
size_t retok_lds_bytes(int32_t max_bytes);
int launch_retokenize(const RetokArgs &a, hipStream_t stream);

// ---------------------------------------------------------------- fused step (step.hip)
struct StepArgs {
    AlignArgs al;     // alignment inputs and outputs
    TransferArgs tr;  // transfer inputs and q (n_pairs, ids, offsets and map shared with al)
    VerifyArgs ve;    // verification inputs and outputs (q = tr.q, target ids = al.target_ids)
};
// One launch for align + transfer + verify when the batch fits both the row-scan alignment
// and the one-workgroup-per-stream verification; TT_EUNSUPPORTED otherwise.
bool step_fused_fits(const StepArgs &s, int tb);
int launch_step_fused(const StepArgs &s, int tb, hipStream_t stream);
// Otherwise, when the pairs fit the row-scan alignment: the same kernel up to gamma (alignment,
// transfer, acceptance) and the split verification path after it.
bool step_front_fits(const StepArgs &s, int tb);
int launch_step_front(const StepArgs &s, int tb, hipStream_t stream);

}  // namespace tt
