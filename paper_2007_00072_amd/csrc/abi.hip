// C ABI: error state, argument validation and the fused-operator entry
// points.  Every entry point validates all arguments before its first
// launch, so a call that fails has enqueued nothing.
#include <stdarg.h>
#include <stdio.h>
#include <math.h>

#include <new>
#include <vector>

#include "gemm.hpp"
#include "internal.hpp"

namespace dm {

static thread_local char g_err[512] = "";

int set_error(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int check_launch(const char* what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(DM_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
    return DM_OK;
}

// ------------------------------------------------------------ timing
namespace {
struct TraceRec {
    const char* label;
    const char* sub;
    hipEvent_t a, b;
};
// Timing switch, records and event pool of the calling thread.
thread_local TraceScope* g_active = nullptr;
thread_local bool g_trace_on = false;
thread_local std::vector<TraceRec> g_trace;     // records of the current session
thread_local std::vector<hipEvent_t> g_events;  // event pool, reused across sessions
thread_local size_t g_events_used = 0;

hipEvent_t pooled_event() {
    if (g_events_used == g_events.size()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        g_events.push_back(e);
    }
    return g_events[g_events_used++];
}
}  // namespace

static int trace_open(const char* label, const char* sub, hipStream_t st) {
    hipEvent_t a = pooled_event(), b = pooled_event();
    if (!a || !b) return -1;
    (void)hipEventRecord(a, st);
    g_trace.push_back({label, sub, a, b});
    return (int)g_trace.size() - 1;
}

const char* trace_current_label() { return g_active ? g_active->label : ""; }

TraceScope::TraceScope(const char* lab, hipStream_t s) : idx(-1), st(s), label(lab), outer(nullptr) {
    if (!g_trace_on) return;
    idx = trace_open(label, "", st);
    if (idx >= 0) {
        outer = g_active;
        g_active = this;
    }
}

void TraceScope::stop() {
    if (idx < 0) return;
    (void)hipEventRecord(g_trace[idx].b, st);
    idx = -1;
    if (g_active == this) g_active = outer;
}

void TraceScope::next(const char* sub) {
    if (idx < 0) return;
    (void)hipEventRecord(g_trace[idx].b, st);
    idx = trace_open(label, sub, st);
    if (idx < 0 && g_active == this) g_active = outer;
}

void trace_next(const char* sub) {
    if (g_active) g_active->next(sub);
}

DropParams make_drop(float p, uint64_t seed, uint32_t site, uint32_t layer) {
    DropParams d{};
    d.seed = seed;
    d.site = site;
    d.layer = layer;
    const double thr = floor((1.0 - (double)p) * 4294967296.0);
    // a p so small that 1 - p rounds to 1 keeps every word (thr = 2^32),
    // which a 32-bit threshold cannot express: no draws at all then
    d.enabled = p > 0.f && thr < 4294967296.0;
    d.thr = d.enabled ? (uint64_t)thr : (1ull << 32);
    d.scale = d.enabled ? (float)(1.0 / (1.0 - (double)p)) : 1.f;
    return d;
}

}  // namespace dm

using namespace dm;

namespace {

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_ptr(const void* p, const char* name) {
    if (!p) return set_error(DM_ERR_ARG, "%s is NULL", name);
    if (!aligned16(p)) return set_error(DM_ERR_ARG, "%s is not 16-byte aligned", name);
    return DM_OK;
}

int check_dtype(int32_t dt) {
    if (dt != DM_F32 && dt != DM_F16 && dt != DM_BF16)
        return set_error(DM_ERR_UNSUPPORTED, "unsupported dtype %d", dt);
    return DM_OK;
}

int check_drop(const dm_dropout* d) {
    if (d && !(d->p >= 0.f && d->p < 1.f)) return set_error(DM_ERR_ARG, "dropout p=%g outside [0,1)", d->p);
    return DM_OK;
}

int check_rows(int64_t rows, int32_t cols, int32_t max_cols) {
    if (rows < 0 || cols <= 0) return set_error(DM_ERR_ARG, "bad shape rows=%lld cols=%d", (long long)rows, cols);
    if (cols % 8) return set_error(DM_ERR_UNSUPPORTED, "row length %d is not a multiple of 8", cols);
    if (max_cols && cols > max_cols) return set_error(DM_ERR_UNSUPPORTED, "row length %d above %d", cols, max_cols);
    if (rows > (int64_t)INT32_MAX * 8) return set_error(DM_ERR_UNSUPPORTED, "too many rows");
    return DM_OK;
}

#define DM_TRY(x)                      \
    do {                               \
        int _rc = (x);                 \
        if (_rc != DM_OK) return _rc;  \
    } while (0)

hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

const char* dm_last_error(void) { return g_err; }

int plan_create(const dm_contract_choice* entries, int32_t n, int32_t attn_path, const dm_layout_choice* layout,
                dm_plan** plan) {
    if (!plan) return set_error(DM_ERR_ARG, "plan output pointer is NULL");
    *plan = nullptr;
    if (n < 0 || (n > 0 && !entries)) return set_error(DM_ERR_ARG, "plan entries missing");
    if (attn_path < 0 || attn_path > 3) return set_error(DM_ERR_ARG, "attn_path %d outside [0, 3]", attn_path);
    for (int i = 0; i < n; ++i) {
        const dm_contract_choice& e = entries[i];
        if (e.tile_cfg < 0 || e.tile_cfg > GEMM_MAX_CFG)
            return set_error(DM_ERR_ARG, "plan entry %d: tile_cfg %d", i, e.tile_cfg);
        if (e.splits < 1 || e.splits > 64) return set_error(DM_ERR_ARG, "plan entry %d: splits %d", i, e.splits);
        if (e.M <= 0 || e.N <= 0 || e.K <= 0 || e.batch <= 0) return set_error(DM_ERR_ARG, "plan entry %d: sizes", i);
    }
    dm_layout_choice lc = {-1, -1, -1, -1};
    if (layout) {
        lc = *layout;
        if (lc.dO_transposed < -1 || lc.dO_transposed > 1 || lc.dH_transposed < -1 || lc.dH_transposed > 1)
            return set_error(DM_ERR_ARG, "layout: transposed-copy fields must be -1, 0 or 1");
        if (lc.ln_bwd_form < -1 || lc.ln_bwd_form > 2)
            return set_error(DM_ERR_ARG, "layout: ln_bwd_form %d outside [-1, 2]", lc.ln_bwd_form);
        if (lc.ln_lanes != -1 && lc.ln_lanes != 0 && lc.ln_lanes != 16 && lc.ln_lanes != 32 && lc.ln_lanes != 64)
            return set_error(DM_ERR_ARG, "layout: ln_lanes %d not one of 16, 32, 64", lc.ln_lanes);
    }
    dm_plan* p = new (std::nothrow) dm_plan;
    if (!p) return set_error(DM_ERR_ARG, "out of host memory for the plan");
    p->entries.assign(entries, entries + n);
    p->attn_path = attn_path;
    p->layout = lc;
    *plan = p;
    return DM_OK;
}

int plan_destroy(dm_plan* plan) {
    delete plan;
    return DM_OK;
}

int plan_log(int32_t on) {
    plan_log_set(on != 0);
    return DM_OK;
}

int plan_log_read(dm_contract_choice* out, int32_t cap, int32_t* count) {
    if (cap < 0 || (cap > 0 && !out) || !count) return set_error(DM_ERR_ARG, "plan_log_read arguments");
    *count = plan_log_copy(out, cap);
    return DM_OK;
}

int dm_trace_enable(int32_t on) {
    if (on) {
        g_trace.clear();
        g_events_used = 0;
    }
    g_trace_on = on != 0;
    return DM_OK;
}

int32_t dm_trace_count(void) {
    return (int32_t)g_trace.size();
}

int dm_trace_get(int32_t i, const char** label, const char** sub, float* ms) {
    if (i < 0 || i >= (int32_t)g_trace.size()) return set_error(DM_ERR_ARG, "trace index %d out of range", i);
    hipError_t e = hipEventSynchronize(g_trace[i].b);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, g_trace[i].a, g_trace[i].b);
    if (e != hipSuccess) return set_error(DM_ERR_DEVICE, "trace event: %s", hipGetErrorString(e));
    if (label) *label = g_trace[i].label;
    if (sub) *sub = g_trace[i].sub;
    if (ms) *ms = t;
    return DM_OK;
}

size_t colsum_ws_bytes(int64_t rows, int32_t cols) {
    if (rows <= 0 || cols <= 0) return 0;
    return (size_t)3 * colsum_blocks(rows) * (size_t)cols * sizeof(float);
}

int bdrln_fwd(int32_t dtype, int64_t rows, int32_t cols, const void* x, const void* bias, const void* resid,
              const void* gamma, const void* beta, float eps, const dm_dropout* drop, void* y, void* xhat,
              float* rstd, void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, cols, 4096));
    DM_TRY(check_drop(drop));
    if (!(eps > 0.f)) return set_error(DM_ERR_ARG, "eps must be > 0");
    if (rows == 0) return DM_OK;
    DM_TRY(check_ptr(x, "x")); DM_TRY(check_ptr(bias, "bias")); DM_TRY(check_ptr(resid, "resid"));
    DM_TRY(check_ptr(gamma, "gamma")); DM_TRY(check_ptr(beta, "beta")); DM_TRY(check_ptr(y, "y"));
    if (xhat) DM_TRY(check_ptr(xhat, "xhat"));
    run_bdrln_fwd(dtype, rows, cols, x, bias, resid, gamma, beta, eps, make_drop(drop), y, xhat, rstd, S(stream));
    return check_launch("bdrln_fwd");
}

int softmax_dropout_fwd(int32_t dtype, int32_t B, int32_t H, int32_t J, int32_t K, float scale, const void* beta,
                        const dm_dropout* drop, void* prob, void* alpha, void* stream) {
    DM_TRY(check_dtype(dtype));
    if (B < 0 || H < 0 || J < 0) return set_error(DM_ERR_ARG, "negative size");
    DM_TRY(check_rows((int64_t)B * H * J, K, 4096));
    DM_TRY(check_drop(drop));
    if ((int64_t)B * H * J == 0) return DM_OK;
    DM_TRY(check_ptr(beta, "beta")); DM_TRY(check_ptr(prob, "prob")); DM_TRY(check_ptr(alpha, "alpha"));
    run_softmax_fwd(dtype, B, H, J, K, scale, beta, make_drop(drop), prob, alpha, S(stream));
    return check_launch("softmax_dropout_fwd");
}

int bias_act_fwd(int32_t dtype, int64_t rows, int32_t cols, const void* x, const void* bias, int32_t act,
                 const dm_dropout* drop, void* y, void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, cols, 0));
    DM_TRY(check_drop(drop));
    if (act != DM_GELU && act != DM_RELU) return set_error(DM_ERR_UNSUPPORTED, "unknown activation %d", act);
    if (rows == 0) return DM_OK;
    DM_TRY(check_ptr(x, "x")); DM_TRY(check_ptr(bias, "bias")); DM_TRY(check_ptr(y, "y"));
    run_bias_act_fwd(dtype, rows, cols, x, bias, act, make_drop(drop), y, S(stream));
    return check_launch("bias_act_fwd");
}

int attn_input_bias(int32_t dtype, int64_t rows, int32_t H, int32_t P, const void* x, const void* bq,
                    const void* bk, const void* bv, void* y, void* stream) {
    DM_TRY(check_dtype(dtype));
    if (H <= 0 || P <= 0 || P % 8) return set_error(DM_ERR_UNSUPPORTED, "P must be a positive multiple of 8");
    DM_TRY(check_rows(rows, 3 * H * P, 0));
    if (rows == 0) return DM_OK;
    DM_TRY(check_ptr(x, "x")); DM_TRY(check_ptr(y, "y"));
    if (!bq || !bk || !bv) return set_error(DM_ERR_ARG, "bias pointer is NULL");
    run_attn_input_bias(dtype, rows, H, P, x, bq, bk, bv, y, S(stream));
    return check_launch("attn_input_bias");
}

int ln_param_bwd(int32_t dtype, int64_t rows, int32_t cols, const void* dy, const void* xhat, float* dgamma,
                 float* dbeta, void* ws, size_t ws_bytes, void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, cols, 2048));
    if (rows == 0) return set_error(DM_ERR_ARG, "rows must be > 0");
    DM_TRY(check_ptr(dy, "dy")); DM_TRY(check_ptr(xhat, "xhat"));
    DM_TRY(check_ptr(dgamma, "dgamma")); DM_TRY(check_ptr(dbeta, "dbeta")); DM_TRY(check_ptr(ws, "ws"));
    if (ws_bytes < colsum_ws_bytes(rows, cols)) return set_error(DM_ERR_WORKSPACE, "workspace too small");
    LnBwdArgs a{};
    a.dtype = dtype; a.rows = rows; a.cols = cols; a.dya = dy; a.xhat = xhat;
    a.dp = make_drop(0.f, 0, 0, 0); a.part = (float*)ws;
    run_ln_bwd(a, S(stream));
    const int nb = ln_bwd_blocks(rows, cols, dtype);
    run_colsum_finish(nb, cols, (float*)ws, dgamma, S(stream));
    run_colsum_finish(nb, cols, (float*)ws + (size_t)nb * cols, dbeta, S(stream));
    return check_launch("ln_param_bwd");
}

int ln_dropout_bwd(int32_t dtype, int64_t rows, int32_t cols, const void* dy, const void* xhat, const void* gamma,
                   const float* rstd, const dm_dropout* drop, void* ds, void* dsub, void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, cols, 4096));
    DM_TRY(check_drop(drop));
    if (rows == 0) return DM_OK;
    DM_TRY(check_ptr(dy, "dy")); DM_TRY(check_ptr(xhat, "xhat")); DM_TRY(check_ptr(gamma, "gamma"));
    DM_TRY(check_ptr(rstd, "rstd")); DM_TRY(check_ptr(dsub, "dsub"));
    if (ds) DM_TRY(check_ptr(ds, "ds"));
    LnBwdArgs a{};
    a.dtype = dtype; a.rows = rows; a.cols = cols; a.dya = dy; a.xhat = xhat; a.gamma = gamma; a.rstd = rstd;
    a.dp = make_drop(drop); a.ds = ds; a.dsub = dsub;
    run_ln_bwd(a, S(stream));
    return check_launch("ln_dropout_bwd");
}

int residual_ln_param_bwd(int32_t dtype, int64_t rows, int32_t cols, const void* da, const void* db,
                          const void* xhat, void* dsum, float* dgamma, float* dbeta, void* ws, size_t ws_bytes,
                          void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, cols, 2048));
    if (rows == 0) return set_error(DM_ERR_ARG, "rows must be > 0");
    DM_TRY(check_ptr(da, "da")); DM_TRY(check_ptr(db, "db")); DM_TRY(check_ptr(xhat, "xhat"));
    DM_TRY(check_ptr(dsum, "dsum")); DM_TRY(check_ptr(dgamma, "dgamma")); DM_TRY(check_ptr(dbeta, "dbeta"));
    DM_TRY(check_ptr(ws, "ws"));
    if (ws_bytes < colsum_ws_bytes(rows, cols)) return set_error(DM_ERR_WORKSPACE, "workspace too small");
    LnBwdArgs a{};
    a.dtype = dtype; a.rows = rows; a.cols = cols; a.dya = da; a.dyb = db; a.xhat = xhat;
    a.dp = make_drop(0.f, 0, 0, 0); a.dysum = dsum; a.part = (float*)ws;
    run_ln_bwd(a, S(stream));
    const int nb = ln_bwd_blocks(rows, cols, dtype);
    run_colsum_finish(nb, cols, (float*)ws, dgamma, S(stream));
    run_colsum_finish(nb, cols, (float*)ws + (size_t)nb * cols, dbeta, S(stream));
    return check_launch("residual_ln_param_bwd");
}

int act_bias_bwd(int32_t dtype, int64_t rows, int32_t F, int32_t I, const void* da, const void* h, const void* b1,
                 int32_t act, const dm_dropout* drop, const void* dout, void* dh, float* db1, float* db2, void* ws,
                 size_t ws_bytes, void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, F, 16384));
    DM_TRY(check_rows(rows, I, 16384));
    DM_TRY(check_drop(drop));
    if (act != DM_GELU && act != DM_RELU) return set_error(DM_ERR_UNSUPPORTED, "unknown activation %d", act);
    if (rows == 0) return set_error(DM_ERR_ARG, "rows must be > 0");
    DM_TRY(check_ptr(da, "da")); DM_TRY(check_ptr(h, "h")); DM_TRY(check_ptr(b1, "b1"));
    DM_TRY(check_ptr(dout, "dout")); DM_TRY(check_ptr(dh, "dh")); DM_TRY(check_ptr(db1, "db1"));
    DM_TRY(check_ptr(db2, "db2")); DM_TRY(check_ptr(ws, "ws"));
    const int mx = F > I ? F : I;
    if (ws_bytes < colsum_ws_bytes(rows, mx)) return set_error(DM_ERR_WORKSPACE, "workspace too small");
    float* part = (float*)ws;
    run_act_bwd(dtype, rows, F, da, h, b1, act, make_drop(drop), dh, part, S(stream));
    run_colsum_finish(colsum_blocks(rows), F, part, db1, S(stream));
    run_colsum_partial(dtype, rows, I, dout, part, S(stream));
    run_colsum_finish(colsum_blocks(rows), I, part, db2, S(stream));
    return check_launch("act_bias_bwd");
}

int softmax_dropout_bwd(int32_t dtype, int32_t B, int32_t H, int32_t J, int32_t K, float scale,
                        const void* dalpha, const void* prob, const dm_dropout* drop, void* dbeta, void* stream) {
    DM_TRY(check_dtype(dtype));
    if (B < 0 || H < 0 || J < 0) return set_error(DM_ERR_ARG, "negative size");
    DM_TRY(check_rows((int64_t)B * H * J, K, 4096));
    DM_TRY(check_drop(drop));
    if ((int64_t)B * H * J == 0) return DM_OK;
    DM_TRY(check_ptr(dalpha, "dalpha")); DM_TRY(check_ptr(prob, "prob")); DM_TRY(check_ptr(dbeta, "dbeta"));
    run_softmax_bwd(dtype, B, H, J, K, scale, dalpha, prob, make_drop(drop), dbeta, S(stream));
    return check_launch("softmax_dropout_bwd");
}

int bias_grad(int32_t dtype, int64_t rows, int32_t cols, const void* x, float* db, void* ws, size_t ws_bytes,
              void* stream) {
    DM_TRY(check_dtype(dtype));
    DM_TRY(check_rows(rows, cols, 16384));
    if (rows == 0) return set_error(DM_ERR_ARG, "rows must be > 0");
    DM_TRY(check_ptr(x, "x")); DM_TRY(check_ptr(db, "db")); DM_TRY(check_ptr(ws, "ws"));
    if (ws_bytes < colsum_ws_bytes(rows, cols)) return set_error(DM_ERR_WORKSPACE, "workspace too small");
    run_colsum_partial(dtype, rows, cols, x, (float*)ws, S(stream));
    trace_next("finish");
    run_colsum_finish(colsum_blocks(rows), cols, (float*)ws, db, S(stream));
    return check_launch("bias_grad");
}

int attn_input_bias_grad(int32_t dtype, int64_t rows, int32_t H, int32_t P, const void* x, float* dbq, float* dbk,
                         float* dbv, void* ws, size_t ws_bytes, void* stream) {
    DM_TRY(check_dtype(dtype));
    if (H <= 0 || P <= 0 || P % 8) return set_error(DM_ERR_UNSUPPORTED, "P must be a positive multiple of 8");
    DM_TRY(check_rows(rows, 3 * H * P, 16384));
    if (rows == 0) return set_error(DM_ERR_ARG, "rows must be > 0");
    DM_TRY(check_ptr(x, "x")); DM_TRY(check_ptr(ws, "ws"));
    if (!dbq || !dbk || !dbv) return set_error(DM_ERR_ARG, "bias gradient pointer is NULL");
    if (ws_bytes < colsum_ws_bytes(rows, 3 * H * P)) return set_error(DM_ERR_WORKSPACE, "workspace too small");
    run_colsum_partial(dtype, rows, 3 * H * P, x, (float*)ws, S(stream));
    run_colsum_finish_qkv(colsum_blocks(rows), H, P, 3, (float*)ws, dbq, dbk, dbv, S(stream));
    return check_launch("attn_input_bias_grad");
}

int residual_add(int32_t dtype, int64_t n, const void* a, const void* b, void* out, void* stream) {
    DM_TRY(check_dtype(dtype));
    if (n < 0 || n % 8) return set_error(DM_ERR_UNSUPPORTED, "n must be a non-negative multiple of 8");
    if (n == 0) return DM_OK;
    DM_TRY(check_ptr(a, "a")); DM_TRY(check_ptr(b, "b")); DM_TRY(check_ptr(out, "out"));
    run_add(dtype, n, a, b, out, S(stream));
    return check_launch("residual_add");
}

int dropout_mask(uint64_t seed, uint32_t site, uint32_t layer, float p, uint64_t offset, uint64_t n, uint8_t* out,
                 void* stream) {
    if (!(p >= 0.f && p < 1.f)) return set_error(DM_ERR_ARG, "dropout p=%g outside [0,1)", p);
    if (offset % 8 || n % 8) return set_error(DM_ERR_ARG, "offset and n must be multiples of 8");
    if (n == 0) return DM_OK;
    if (!out) return set_error(DM_ERR_ARG, "out is NULL");
    if (((uintptr_t)out & 7u) != 0) return set_error(DM_ERR_ARG, "out is not 8-byte aligned");
    run_dropout_mask(make_drop(p, seed, site, layer), offset, n, out, S(stream));
    return check_launch("dropout_mask");
}

int contract(int32_t dtype, int32_t batch, int32_t M, int32_t N, int32_t K, float alpha, const void* A,
             int32_t a_trans, int64_t sa, const void* B, int32_t b_trans, int64_t sb, const void* bias, void* C,
             int32_t out_f32, int64_t sc, int32_t tile_cfg, int32_t splits, void* ws, size_t ws_bytes,
             void* stream) {
    DM_TRY(check_dtype(dtype));
    if (batch < 0 || M < 0 || N < 0 || K <= 0) return set_error(DM_ERR_ARG, "bad contraction shape");
    if ((int64_t)batch * M * N == 0) return DM_OK;
    if (dtype != DM_F32 && (M % 8 || N % 8 || K % 8))
        return set_error(DM_ERR_UNSUPPORTED, "M, N, K must be multiples of 8");
    DM_TRY(check_ptr(A, "A")); DM_TRY(check_ptr(B, "B")); DM_TRY(check_ptr(C, "C"));
    if (bias) DM_TRY(check_ptr(bias, "bias"));
    if (tile_cfg < -1 || tile_cfg > GEMM_MAX_CFG)
        return set_error(DM_ERR_ARG, "tile_cfg %d outside [-1, %d]", tile_cfg, GEMM_MAX_CFG);
    if (splits < 0 || splits > 64) return set_error(DM_ERR_ARG, "splits %d outside [0, 64]", splits);
    if (splits > 1 && (!ws || ws_bytes < gemm_split_ws_bytes(M, N, batch, splits)))
        return set_error(DM_ERR_WORKSPACE, "split-k workspace too small");
    if (ws) DM_TRY(check_ptr(ws, "ws"));
    if (dtype == DM_F32 && !out_f32) out_f32 = 1;
    GemmArgs g{};
    g.cfg = tile_cfg;
    g.splits = splits;
    g.split_ws = (float*)ws;
    g.split_cap = (int64_t)(ws_bytes / sizeof(float));
    g.M = M; g.N = N; g.K = K; g.batch = batch;
    g.a.ptr[0] = A; g.a.nseg = 1;
    g.a.kcontig = a_trans ? 0 : 1;
    g.a.row = linear_map(a_trans ? M : K);
    g.a.batch = linear_map(sa);
    g.b.ptr[0] = B; g.b.nseg = 1;
    g.b.kcontig = b_trans ? 1 : 0;
    g.b.row = linear_map(b_trans ? K : N);
    g.b.batch = linear_map(sb);
    g.c.ptr[0] = C; g.c.nseg = 1;
    g.c.mmap = linear_map(N); g.c.nmap = linear_map(1); g.c.batch = linear_map(sc);
    g.c.contig_n = 1; g.c.alpha = alpha;
    g.c.bias[0] = bias; g.c.bias_nseg = 1; g.c.bias_map = linear_map(1);
    g.c.out_f32 = out_f32;
    return launch_gemm(dtype, g, S(stream));
}

}  // extern "C"
