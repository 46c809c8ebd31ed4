// Host-side internals shared by the library's translation units: error
// state, dropout parameter setup and the launchers of the fused operators.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "../../include/dmtx.h"
#include "common.hpp"

// A configuration plan (plan_create): immutable once made.
struct dm_plan {
    std::vector<dm_contract_choice> entries;
    int attn_path;
    dm_layout_choice layout;
};

namespace dm {

// Records a message for dm_last_error() on the calling thread; returns code.
int set_error(int code, const char* fmt, ...);
int check_launch(const char* what);

// Per-launch timing (dm_trace_*): brackets the launches made in its scope
// with two events on `st` when tracing is enabled.
struct TraceScope {
    TraceScope(const char* label, hipStream_t st);
    ~TraceScope() { stop(); }
    void stop();                // records the end event now (idempotent)
    void next(const char* sub);  // ends the current record, starts one for the next launch of this scope
    int idx;
    hipStream_t st;
    const char* label;
    TraceScope* outer;
};
// Marks the start of a further launch of the innermost active scope (no-op
// when tracing is off), so every launch has a record of its own.
void trace_next(const char* sub);
// label of the innermost active scope ("" when timing is off)
const char* trace_current_label();
// The configuration plan of the entry-point call running on this thread
// (its descriptor's plan; nullptr = built-in choices), set for the call's
// duration by a PlanScope.
const dm_plan* current_plan();
struct PlanScope {
    explicit PlanScope(const dm_plan* p);
    ~PlanScope();
    const dm_plan* prev;
};
// attention-score launch grouping of the current plan: 0 automatic,
// 1 separate, 2 scores on chip, 3 scores and the next contraction together
int current_attn_path();
// launch record of the calling thread (plan_log)
void plan_log_set(bool on);
int plan_log_copy(dm_contract_choice* out, int cap);

// p in [0,1); seed/site/layer -> kernel parameters (thr, scale computed in double).
DropParams make_drop(float p, uint64_t seed, uint32_t site, uint32_t layer);
inline DropParams make_drop(const dm_dropout* d) {
    if (!d) return make_drop(0.f, 0, 0, 0);
    return make_drop(d->p, d->seed, d->site, d->layer);
}

// Column-sum scratch: partial sums of `nblk` row blocks (colsum_blocks for
// the column-sum and activation-backward kernels, ln_bwd_blocks for the
// LayerNorm backward; never more than colsum_blocks(rows)).
int colsum_blocks(int64_t rows);
// LayerNorm backward can take its column-split form for these row lengths
// (16-bit storage types)
inline bool ln_bwd_split_ok(int cols, int dtype) {
    return dtype != DM_F32 && cols % 64 == 0 && cols >= 320 && cols <= 1024;
}
// form: 0 = the library's choice (column split where allowed), 1 = one lane
// group per row, 2 = column split (where allowed)
inline bool ln_bwd_uses_split(int cols, int dtype, int form) {
    return form != 1 && ln_bwd_split_ok(cols, dtype);
}
int ln_bwd_blocks(int64_t rows, int cols, int dtype, int form = 0);
// partial rows of the activation backward (with the transposed copy, whole
// groups of 8 rows per block)
int act_bwd_blocks(int64_t rows, bool transposed);

// Layout and reduction choices of the fused operators for the running call:
// its plan's, with every "library's choice" field resolved for this shape.
struct FusedLayout {
    bool dO_t;      // LayerNorm-2 backward writes dO^T, the Linear-2 weight gradient reads it
    bool dH_t;      // activation backward writes dH^T, the Linear-1 weight gradient reads it
    int ln_form;    // LayerNorm backward reduction form (0/1/2 as ln_bwd_uses_split)
    int ln_lanes;   // lanes per row of the row-form LayerNorm kernels (0 = by length)
};
FusedLayout fused_layout(int dtype, int64_t T, int I, int F);

// ------------------------------------------------------- kernel launchers
// All take element counts, device pointers and a stream, and assume the
// caller validated alignment and sizes.  dtype: DM_F32 / DM_F16 / DM_BF16.
// lanes: lanes per row (0 = by row length; 16, 32 for rows of 257..1024)
void run_bdrln_fwd(int dtype, int64_t rows, int cols, const void* x, const void* bias,
                   const void* resid, const void* gamma, const void* beta, float eps,
                   const DropParams& dp, void* y, void* xhat, float* rstd, hipStream_t st, int lanes = 0);

// Attention scores without the score tensor in HBM (attn.hip).  Operand
// element (z = b*H + h, row r, contraction index d) sits at
// ptr + b*outer + h*inner + r*ld + d; P, alpha and d(beta) are [B][H][J][K].
// attn_fused_ok: dtype fp16 / bf16, K a multiple of 32 up to 960, D (the
// contraction length) in {16, 32, 48, 64, 96, 128}.
bool attn_fused_ok(int dtype, int K, int D);
// The contraction that follows in the same launch: out[z][j][n] =
// sum_k tile[z][j][k] x[z][k][n] with x element (z, k, n) at
// x + b*x_outer + h*x_inner + k*x_ld + n and out element (z, j, n) at
// out + b*o_outer + h*o_inner + j*o_ld + n; n < N.  attn_next_ok: the
// scores' own conditions, D (the first contraction's length) and N in
// {32, 64, 128}, x 16-byte aligned with strides that are multiples of 8
// elements, and the block's LDS within 64 KB.
struct AttnNext {
    const void* x = nullptr;
    int64_t x_outer = 0, x_inner = 0, x_ld = 0;
    void* out = nullptr;
    int64_t o_outer = 0, o_inner = 0, o_ld = 0;
    int N = 0;
    float* out_f32 = nullptr;  // optional fp32 copy of out before rounding (same strides)
};
bool attn_next_ok(int dtype, int K, int D, const AttnNext& n);
// P = softmax_k(round(scaler * Q K^T)), alpha = dropout(P); with `next`,
// also gamma = alpha V.  causal: query j sees keys k <= j only.
void run_attn_scores_fwd(int dtype, int B, int H, int J, int K, int D, float scaler, const void* q, int64_t q_outer,
                         int64_t q_inner, int64_t q_ld, const void* k, int64_t k_outer, int64_t k_inner, int64_t k_ld,
                         const DropParams& dp, void* prob, void* alpha, const AttnNext* next, hipStream_t st,
                         int causal = 0);
// d(beta) = scaler * P * (dP - sum_k dP P), dP = dropout(round(d(gamma) V^T));
// with `next`, also dQ = d(beta) K
void run_attn_scores_bwd(int dtype, int B, int H, int J, int K, int D, float scaler, const void* dgamma,
                         int64_t dg_outer, int64_t dg_inner, int64_t dg_ld, const void* v, int64_t v_outer,
                         int64_t v_inner, int64_t v_ld, const void* prob, const DropParams& dp, void* dbeta,
                         const AttnNext* next, hipStream_t st);

// Key-block backward of the attention scores (attn.hip): from d(gamma),
// gamma (fp32, before rounding), P and Q, K, V it writes dQ, dK, dV (the
// rows of Table 3 from Gamma dX1 to QK^T dX2) without materialising
// d(alpha), alpha or d(beta).
// Row operands as for the score kernels: element (z = b*H + h, row r, d) at
// ptr + b*outer + h*inner + r*ld + d.  attn_keys_ok: fp16 / bf16, P = W =
// 64, K a multiple of 128 (all rows 16-byte aligned).  part: fp32 scratch of
// attn_keys_part_bytes (nullptr allowed when that is 0).
struct AttnRows {
    const void* ptr;
    int64_t outer, inner, ld;
};
bool attn_keys_ok(int dtype, int K, int P, int W);
size_t attn_keys_part_bytes(int B, int H, int J, int K);
void run_attn_bwd_keys(int dtype, int B, int H, int J, int K, float scaler, AttnRows q, AttnRows k, AttnRows v,
                       AttnRows dgamma, AttnRows gamma, const void* prob, const DropParams& dp, AttnRows dq,
                       AttnRows dk, AttnRows dv, float* part, hipStream_t st);
// alpha = dropout(P) from the stored probabilities [B][H][J][K] (K % 8 == 0)
void run_alpha_from_prob(int dtype, int B, int H, int J, int K, const void* prob, const DropParams& dp, void* alpha,
                         hipStream_t st);

// causal: query row j sees keys k <= j only (probabilities after it exactly 0)
void run_softmax_fwd(int dtype, int B, int H, int J, int K, float scale, const void* beta,
                     const DropParams& dp, void* prob, void* alpha, hipStream_t st, int causal = 0);

void run_bias_act_fwd(int dtype, int64_t rows, int cols, const void* x, const void* bias, int act,
                      const DropParams& dp, void* y, hipStream_t st);

void run_attn_input_bias(int dtype, int64_t rows, int H, int P, const void* x, const void* bq,
                         const void* bk, const void* bv, void* y, hipStream_t st);

// LayerNorm backward row kernel, in the fused forms the layer uses:
//   dy = dya (+ dyb if non-null); optional dysum = dy written out;
//   optional ds = LN backward of dy; optional dsub = dropout(ds);
//   optional column partial sums of dy*xhat, dy and dsub into `part`
//   ([3][nblk][cols] floats) finished by run_colsum_finish.
struct LnBwdArgs {
    int dtype;
    int64_t rows;
    int cols;
    const void* dya;
    const void* dyb;
    const void* xhat;
    const void* gamma;
    const float* rstd;
    DropParams dp;
    void* dysum;
    void* ds;
    void* dsub;
    float* part;  // null: no column sums
    int want_dsub_sum;
    void* dsub_t;  // optional [cols][rows] copy of dsub (written when the column-split form runs)
    int form;      // 0 library's choice, 1 row form, 2 column split (ln_bwd_uses_split)
    int lanes;     // row form: lanes per row (0 = by row length)
};
void run_ln_bwd(const LnBwdArgs& a, hipStream_t st);

void run_softmax_bwd(int dtype, int B, int H, int J, int K, float scale, const void* dalpha,
                     const void* prob, const DropParams& dp, void* dbeta, hipStream_t st);

// dh = dropout'(da) * act'(h + b1) with column partials of dh into part
// (act_bwd_blocks(rows, dht != nullptr) partial rows); with dht also dh
// transposed, [F][rows] (rows a multiple of 8).
void run_act_bwd(int dtype, int64_t rows, int F, const void* da, const void* h, const void* b1,
                 int act, const DropParams& dp, void* dh, float* part, hipStream_t st, void* dht = nullptr);

// Column partial sums of x (rows x cols) into part[nblk][cols].
void run_colsum_partial(int dtype, int64_t rows, int cols, const void* x, float* part,
                        hipStream_t st);

// out[map(c)] = sum_b part[b][c] for c < cols.  With H, P > 0 the columns
// are (s, h, p) of a fused projection and go to outs[s][p*H + h].
// A job is one operator's partial sets (part[nsets][nblk][cols], all from
// `rows` rows); run_colsum_finish_jobs finishes several in one launch.
struct FinishJob {
    const float* part;
    float* out[3];
    int nblk, cols, nsets, qkv_H, qkv_P;
};
constexpr int MAX_FINISH_JOBS = 4;
struct FinishJobs {
    FinishJob job[MAX_FINISH_JOBS];
    int first[MAX_FINISH_JOBS];  // first block of each job
    int n;
};
inline FinishJob finish_job(const float* part, int nblk, int cols, float* out) {
    return FinishJob{part, {out, nullptr, nullptr}, nblk, cols, 1, 0, 0};
}
inline FinishJob finish_job3(const float* part, int nblk, int cols, float* o0, float* o1, float* o2) {
    return FinishJob{part, {o0, o1, o2}, nblk, cols, 3, 0, 0};
}
inline FinishJob finish_job_qkv(const float* part, int nblk, int H, int P, int nseg, float* dbq, float* dbk,
                                float* dbv) {
    return FinishJob{part, {dbq, dbk, dbv}, nblk, nseg * H * P, 1, H, P};
}
// bytes of `nsets` partial sets of `nblk` row blocks of `cols` columns
inline size_t colsum_part_bytes(int nblk, int64_t cols, int nsets) {
    return (size_t)nsets * (size_t)nblk * (size_t)cols * sizeof(float);
}
void run_colsum_finish_jobs(const FinishJob* jobs, int n, hipStream_t st);
// single jobs; nblk is the partial row count the producing kernel used
void run_colsum_finish(int nblk, int cols, const float* part, float* out, hipStream_t st);
void run_colsum_finish_qkv(int nblk, int H, int P, int nseg, const float* part, float* dbq,
                           float* dbk, float* dbv, hipStream_t st);

// out[r] = sum_c x[r][c] (float) for rows of length len (multiple of 8).
void run_rowsum(int dtype, int64_t rows, int len, const void* x, float* out, hipStream_t st);

void run_add(int dtype, int64_t n, const void* a, const void* b, void* out, hipStream_t st);

void run_dropout_mask(const DropParams& dp, uint64_t offset, uint64_t n, uint8_t* out,
                      hipStream_t st);

}  // namespace dm
