// Layer drivers: multi-head attention (Fig. 1a) and the post-LN encoder
// layer (Table 3), forward and backward, sequenced on one stream.
//
// Internal layouts (chosen so that every contraction reads its operands in
// place and every statistical normalisation reduces a contiguous row):
//   residual stream, LayerNorm outputs, FFN activations: token-major [T][.]
//   per-head projections Q, K, V:                         [B][H][J or K][P]
//   attention scores beta, probabilities, alpha:          [B][H][J][K]
//   attention context gamma:                              [T][H][W]
//   gradients of Q, K, V:                                 token-major [T][3][H][P]
// The paper's (p, h) ordering of projection rows and weights is reached by
// index maps inside the contraction kernel, never by a transpose pass.
#include <math.h>

#include "gemm.hpp"
#include "internal.hpp"

using namespace dm;

namespace {

constexpr size_t ALIGN = 256;
size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

struct Dims {
    int64_t B, J, K, H, P, W, I, F;
    int64_t Tq, Tk, N, S;
    int es;  // element size
    int dtype;
    int layout;
    int causal;      // query j sees keys k <= j only
    int qkv_fusion;  // self-attention projections: 0 one stacked contraction, 1 QK + V, 2 separate
};

Dims dims_of(const dm_layer_desc* d) {
    Dims x{};
    x.B = d->B; x.J = d->J; x.K = d->K; x.H = d->H; x.P = d->P; x.W = d->W; x.I = d->I; x.F = d->F;
    x.Tq = x.B * x.J; x.Tk = x.B * x.K; x.N = x.Tq * x.I; x.S = x.B * x.H * x.J * x.K;
    x.dtype = d->dtype;
    x.layout = d->layout;
    x.es = d->dtype == DM_F32 ? 4 : 2;
    x.causal = d->causal;
    x.qkv_fusion = d->qkv_fusion;
    return x;
}

// ------------------------------------------------------------ buffer plans
struct Carver {
    size_t total = 0;
    size_t take(size_t bytes) { size_t o = total; total += up(bytes); return o; }
};

struct MhaPlan {
    // saved (alpha is not: it is re-formed from P and the dropout keep
    // decisions where a step needs it); gamma32: gamma before rounding, in
    // fp32, for the key-block backward's row term (0 = not saved)
    size_t q, k, v, prob, gamma, gamma32;
    // forward workspace (alpha for the launch groupings that read it back)
    size_t beta, alpha_f;
    // backward workspace (alpha re-formed for the groupings that read it;
    // the key-block backward keeps its dQ partial sums in dalpha)
    size_t dgamma, dalpha, dbeta, alpha_b, dq, dk, dv, part;
    int64_t ldq, ldk, ldv;  // row strides (elements) of the Q/K/V gradient buffers
    size_t fused_dqkv;      // self-attention: one [T][3][H][P] buffer at dq
};

struct EncPlan {
    MhaPlan m;
    size_t xhat1, rstd1, y1, h, a, xhat2, rstd2, saved_total;
    size_t ao, o, fwd_split, fwd_total;
    size_t dS2, dO, dOT, dA, dH, dHT, dY1f, dS1, dAO, bwd_split, bwd_total;
    size_t part_ln2, part_act, part_ln1;  // column partials finished together at the end of the backward
    int64_t split_floats;
};

// Split-k scratch for the contractions of one call: room for four partial
// sums of the largest weight-sized output.
int64_t split_floats_for(int64_t a, int64_t b, int64_t c) { return 4 * (a > b ? (a > c ? a : c) : (b > c ? b : c)); }

// The contraction launches of one entry-point call take their split-k
// scratch from here (set for the duration of the call on this thread).
thread_local float* t_split_ws = nullptr;
thread_local int64_t t_split_cap = 0;
struct SplitScope {
    SplitScope(void* p, int64_t cap) { t_split_ws = reinterpret_cast<float*>(p); t_split_cap = cap; }
    ~SplitScope() { t_split_ws = nullptr; t_split_cap = 0; }
};

int64_t max3(int64_t a, int64_t b, int64_t c) { return a > b ? (a > c ? a : c) : (b > c ? b : c); }

// Input-projection modes of attention (dm_layer_desc.self_attention).
enum { PROJ_SEPARATE = 0, PROJ_QKV = 1, PROJ_KV = 2 };

void plan_attention(const Dims& x, int mode, Carver& sv, Carver& fw, Carver& bw, MhaPlan& p) {
    const size_t es = x.es;
    if (mode == PROJ_QKV) {
        // one [3][B][H][J][P] block (the saved-tensor view of Q, K, V);
        // every piece stays 16-byte aligned since J and P are multiples of 8
        const size_t one = es * x.B * x.H * x.J * x.P;
        p.q = sv.take(3 * one);
        p.k = p.q + one;
        p.v = p.k + one;
    } else {
        p.q = sv.take(es * x.B * x.H * x.J * x.P);
        p.k = sv.take(es * x.B * x.H * x.K * x.P);
        p.v = sv.take(es * x.B * x.H * x.K * x.W);
    }
    p.prob = sv.take(es * x.S);
    p.gamma = sv.take(es * x.Tq * x.H * x.W);
    p.gamma32 = attn_keys_ok(x.dtype, (int)x.K, (int)x.P, (int)x.W) ? sv.take(4 * x.Tq * x.H * x.W) : 0;
    p.beta = fw.take(es * x.S);
    p.alpha_f = fw.take(es * x.S);
    p.dgamma = bw.take(es * x.Tq * x.H * x.W);
    // (dQ partials of the key-block backward: at most 4 B x 64 per query
    // row and 128-key block, no more than 2 B per score)
    p.dalpha = bw.take(es * x.S > attn_keys_part_bytes((int)x.B, (int)x.H, (int)x.J, (int)x.K)
                           ? es * x.S
                           : attn_keys_part_bytes((int)x.B, (int)x.H, (int)x.J, (int)x.K));
    p.dbeta = bw.take(es * x.S);
    p.alpha_b = bw.take(es * x.S);
    if (mode == PROJ_QKV) {
        p.ldq = p.ldk = p.ldv = 3 * x.H * x.P;
        p.dq = bw.take(es * x.Tq * p.ldq);
        p.dk = p.dq;  // column offsets are added at use
        p.dv = p.dq;
    } else if (mode == PROJ_KV) {
        p.ldq = x.H * x.P;
        p.ldk = p.ldv = 2 * x.H * x.P;
        p.dq = bw.take(es * x.Tq * p.ldq);
        p.dk = bw.take(es * x.Tk * p.ldk);
        p.dv = p.dk;  // column offset added at use
    } else {
        p.ldq = x.H * x.P; p.ldk = x.H * x.P; p.ldv = x.H * x.W;
        p.dq = bw.take(es * x.Tq * p.ldq);
        p.dk = bw.take(es * x.Tk * p.ldk);
        p.dv = bw.take(es * x.Tk * p.ldv);
    }
}

EncPlan plan_encoder(const Dims& x) {
    EncPlan e{};
    Carver sv, fw, bw;
    plan_attention(x, PROJ_QKV, sv, fw, bw, e.m);
    const size_t es = x.es, T = x.Tq;
    e.xhat1 = sv.take(es * x.N);
    e.rstd1 = sv.take(4 * T);
    e.y1 = sv.take(es * x.N);
    e.h = sv.take(es * T * x.F);
    e.a = sv.take(es * T * x.F);
    e.xhat2 = sv.take(es * x.N);
    e.rstd2 = sv.take(4 * T);
    e.saved_total = sv.total;
    e.ao = fw.take(es * x.N);
    e.o = fw.take(es * x.N);
    e.split_floats = split_floats_for(3 * x.I * x.I, x.I * x.F, x.Tq * x.I);
    e.fwd_split = fw.take(4 * e.split_floats);
    e.fwd_total = fw.total;
    e.dS2 = bw.take(es * x.N);
    e.dO = bw.take(es * x.N);
    e.dOT = bw.take(es * x.N);  // dO transposed, [I][T]
    e.dA = bw.take(es * T * x.F);
    e.dH = bw.take(es * T * x.F);
    e.dHT = bw.take(es * T * x.F);  // dH transposed, [F][T] (when a plan asks for it)
    e.dY1f = bw.take(es * x.N);
    e.dS1 = bw.take(es * x.N);
    e.dAO = bw.take(es * x.N);
    // (either LayerNorm-backward form: colsum_blocks bounds both partial counts)
    e.part_ln2 = bw.take(colsum_part_bytes(colsum_blocks(T), x.I, 3));
    e.part_act = bw.take(colsum_part_bytes(colsum_blocks(T), x.F, 1));
    e.part_ln1 = bw.take(colsum_part_bytes(colsum_blocks(T), x.I, 3));
    e.m.part = bw.take(colsum_part_bytes(colsum_blocks(T), 3 * x.I, 1));
    e.bwd_split = bw.take(4 * e.split_floats);
    e.bwd_total = bw.total;
    return e;
}

struct MhaSizes { MhaPlan p; size_t saved, fwd, bwd, fwd_split, bwd_split; int64_t split_floats; };
MhaSizes plan_mha(const Dims& x, int mode) {
    MhaSizes s{};
    Carver sv, fw, bw;
    plan_attention(x, mode, sv, fw, bw, s.p);
    int64_t cols = max3(mode == PROJ_SEPARATE ? x.H * x.P : (3 - (mode == PROJ_KV)) * x.H * x.P, x.H * x.W, x.I);
    s.p.part = bw.take(colsum_ws_bytes(x.Tq > x.Tk ? x.Tq : x.Tk, (int32_t)cols) + 4 * x.I);
    s.split_floats = split_floats_for(3 * x.H * x.P * x.I, x.H * x.W * x.I, x.Tq * x.I);
    s.fwd_split = fw.take(4 * s.split_floats);
    s.bwd_split = bw.take(4 * s.split_floats);
    s.saved = sv.total; s.fwd = fw.total; s.bwd = bw.total;
    return s;
}

// ------------------------------------------------------------ validation
#define DM_TRY(x)                      \
    do {                               \
        int _rc = (x);                 \
        if (_rc != DM_OK) return _rc;  \
    } while (0)

int need(const void* p, const char* name) {
    if (!p) return set_error(DM_ERR_ARG, "%s is NULL", name);
    if ((uintptr_t)p & 15u) return set_error(DM_ERR_ARG, "%s is not 16-byte aligned", name);
    return DM_OK;
}

int check_desc(const dm_layer_desc* d, bool encoder) {
    if (!d) return set_error(DM_ERR_ARG, "descriptor is NULL");
    if (d->dtype != DM_F32 && d->dtype != DM_F16 && d->dtype != DM_BF16)
        return set_error(DM_ERR_UNSUPPORTED, "unsupported dtype %d", d->dtype);
    if (d->layout != DM_BJI && d->layout != DM_IBJ) return set_error(DM_ERR_UNSUPPORTED, "unsupported layout");
    if (d->B <= 0 || d->J <= 0 || d->K <= 0 || d->H <= 0 || d->P <= 0 || d->W <= 0 || d->I <= 0)
        return set_error(DM_ERR_ARG, "sizes must be positive");
    if (d->J % 8 || d->K % 8 || d->P % 8 || d->W % 8 || d->I % 8)
        return set_error(DM_ERR_UNSUPPORTED, "J, K, P, W, I must be multiples of 8");
    if (d->K > 4096) return set_error(DM_ERR_UNSUPPORTED, "key length above 4096");
    if ((int64_t)d->B * d->H > 65535) return set_error(DM_ERR_UNSUPPORTED, "B*H above 65535");
    if ((int64_t)d->B * d->H * d->J * d->K > ((int64_t)1 << 40)) return set_error(DM_ERR_UNSUPPORTED, "too large");
    if ((int64_t)d->B * (d->J > d->K ? d->J : d->K) * 3 * d->I >= ((int64_t)1 << 31))
        return set_error(DM_ERR_UNSUPPORTED, "token count too large");
    if (d->causal != 0 && d->causal != 1) return set_error(DM_ERR_ARG, "causal must be 0 or 1");
    if (d->qkv_fusion < 0 || d->qkv_fusion > 2) return set_error(DM_ERR_ARG, "qkv_fusion must be 0, 1 or 2");
    if (d->causal && d->J != d->K) return set_error(DM_ERR_UNSUPPORTED, "a causal mask needs J == K");
    const float ps[4] = {d->p_attn, d->p_attn_out, d->p_ffn_out, d->p_ffn_act};
    for (float p : ps)
        if (!(p >= 0.f && p < 1.f)) return set_error(DM_ERR_ARG, "dropout probability %g outside [0,1)", p);
    if (encoder) {
        if (d->layout != DM_BJI) return set_error(DM_ERR_UNSUPPORTED, "encoder layer supports layout BJI only");
        if (d->I != d->H * d->P || d->W != d->P) return set_error(DM_ERR_ARG, "encoder needs I == H*P and W == P");
        if (d->J != d->K) return set_error(DM_ERR_ARG, "encoder self-attention needs J == K");
        if (d->F <= 0 || d->F % 8) return set_error(DM_ERR_UNSUPPORTED, "F must be a positive multiple of 8");
        if (d->I > 2048) return set_error(DM_ERR_UNSUPPORTED, "I above 2048");
        if (d->F > 16384) return set_error(DM_ERR_UNSUPPORTED, "F above 16384");
        if (d->act != DM_GELU && d->act != DM_RELU) return set_error(DM_ERR_UNSUPPORTED, "unknown activation");
        if (!(d->ln_eps > 0.f)) return set_error(DM_ERR_ARG, "ln_eps must be > 0");
    } else {
        if (d->self_attention < PROJ_SEPARATE || d->self_attention > PROJ_KV)
            return set_error(DM_ERR_ARG, "self_attention must be 0, 1 or 2");
        if (d->self_attention == PROJ_QKV && (d->J != d->K || d->W != d->P))
            return set_error(DM_ERR_ARG, "self-attention needs J == K and W == P");
        if (d->self_attention == PROJ_KV && d->W != d->P)
            return set_error(DM_ERR_ARG, "a fused K/V projection needs W == P");
        if (3 * d->H * d->P > 16384 || d->I > 16384) return set_error(DM_ERR_UNSUPPORTED, "width above 16384");
    }
    return DM_OK;
}

int check_params(const dm_layer_params* p, bool encoder) {
    if (!p) return set_error(DM_ERR_ARG, "params is NULL");
    DM_TRY(need(p->wq, "wq")); DM_TRY(need(p->bq, "bq")); DM_TRY(need(p->wk, "wk")); DM_TRY(need(p->bk, "bk"));
    DM_TRY(need(p->wv, "wv")); DM_TRY(need(p->bv, "bv")); DM_TRY(need(p->wo, "wo")); DM_TRY(need(p->bo, "bo"));
    if (encoder) {
        DM_TRY(need(p->g1, "g1")); DM_TRY(need(p->be1, "be1")); DM_TRY(need(p->w1, "w1"));
        DM_TRY(need(p->b1, "b1")); DM_TRY(need(p->w2, "w2")); DM_TRY(need(p->b2, "b2"));
        DM_TRY(need(p->g2, "g2")); DM_TRY(need(p->be2, "be2"));
    }
    return DM_OK;
}

int check_grads(const dm_layer_grads* g, bool encoder) {
    if (!g) return set_error(DM_ERR_ARG, "grads is NULL");
    DM_TRY(need(g->dwq, "dwq")); DM_TRY(need(g->dbq, "dbq")); DM_TRY(need(g->dwk, "dwk"));
    DM_TRY(need(g->dbk, "dbk")); DM_TRY(need(g->dwv, "dwv")); DM_TRY(need(g->dbv, "dbv"));
    DM_TRY(need(g->dwo, "dwo")); DM_TRY(need(g->dbo, "dbo"));
    if (encoder) {
        DM_TRY(need(g->dg1, "dg1")); DM_TRY(need(g->dbe1, "dbe1")); DM_TRY(need(g->dw1, "dw1"));
        DM_TRY(need(g->db1, "db1")); DM_TRY(need(g->dw2, "dw2")); DM_TRY(need(g->db2, "db2"));
        DM_TRY(need(g->dg2, "dg2")); DM_TRY(need(g->dbe2, "dbe2"));
    }
    return DM_OK;
}

// ------------------------------------------------------------ GEMM builders
IdxMap zero_map() { return linear_map(0); }

Operand opnd(const void* p, bool kcontig, IdxMap row, IdxMap batch = zero_map()) {
    Operand o{};
    o.ptr[0] = p; o.nseg = 1; o.kcontig = kcontig; o.row = row; o.batch = batch;
    return o;
}
Operand opnd3(const void* p0, const void* p1, const void* p2, bool kcontig, IdxMap row) {
    Operand o = opnd(p0, kcontig, row);
    o.ptr[1] = p1; o.ptr[2] = p2; o.nseg = 3;
    return o;
}
Epilogue epi(void* p, IdxMap mmap, IdxMap nmap, bool contig_n, bool out_f32, IdxMap batch = zero_map()) {
    Epilogue e{};
    e.ptr[0] = p; e.nseg = 1; e.mmap = mmap; e.nmap = nmap; e.batch = batch;
    e.contig_n = contig_n; e.alpha = 1.f; e.out_f32 = out_f32; e.bias_nseg = 1;
    e.bias_map = linear_map(1);
    return e;
}
GemmArgs gemm(int64_t M, int64_t N, int64_t K, int64_t batch, const Operand& a, const Operand& b,
              const Epilogue& c) {
    GemmArgs g{};
    g.M = (int)M; g.N = (int)N; g.K = (int)K; g.batch = (int)batch;
    g.a = a; g.b = b; g.c = c;
    g.cfg = -1;
    g.splits = t_split_ws ? 0 : 1;
    g.split_ws = t_split_ws;
    g.split_cap = t_split_cap;
    return g;
}

// An activation x (t, i) in the given layout, as the (m, k) operand with m = t, k = i...
Operand act_mk(const void* p, int layout, int64_t T, int64_t I) {
    return layout == DM_BJI ? opnd(p, true, linear_map(I)) : opnd(p, false, linear_map(T));
}
// ... and as the (k, n) operand with k = t, n = i.
Operand act_kn(const void* p, int layout, int64_t T, int64_t I) {
    return layout == DM_BJI ? opnd(p, false, linear_map(I)) : opnd(p, true, linear_map(T));
}
// Output element (t, i) of an activation in the given layout.
Epilogue act_out(void* p, int layout, int64_t T, int64_t I) {
    return layout == DM_BJI ? epi(p, linear_map(I), linear_map(1), true, false)
                            : epi(p, linear_map(1), linear_map(T), false, false);
}

char* B8(void* base, size_t off) { return reinterpret_cast<char*>(base) + off; }
const char* B8(const void* base, size_t off) { return reinterpret_cast<const char*>(base) + off; }

float scaler_of(const dm_layer_desc* d) { return d->scaler > 0.f ? d->scaler : 1.0f / sqrtf((float)d->P); }

// ------------------------------------------------------------ attention pieces
// Projection of one input into a per-head tensor [B][H][L][n] (n = P or W),
// with the input bias in the epilogue.  w: [n][H][I] (paper order), b: [n][H].
int project(const Dims& x, int layout, const void* in, int64_t L, int64_t n, const void* w, const void* b,
            void* out, hipStream_t st) {
    const int64_t T = x.B * L;
    Operand A = act_mk(in, layout, T, x.I);
    Operand Bw = opnd(w, true, make_map((uint32_t)n, 0, x.H * x.I, x.I, 0));
    Epilogue c = epi(out, make_map((uint32_t)L, 0, n, x.H * L * n, 0), make_map((uint32_t)n, 0, 1, L * n, 0),
                     true, false);
    c.bias[0] = b; c.bias_map = make_map((uint32_t)n, 0, x.H, 1, 0);
    return launch_gemm(x.dtype, gemm(T, x.H * n, x.I, 1, A, Bw, c), st);
}

// Stacked input projections (Sec. "Algebraic Fusion"): the weights
// [Wq Wk Wv] of segments [s0, s1) times one input X of L tokens per
// sequence as one contraction, each segment's output going to its own
// [B][H][L][P] tensor with its bias.  Self-attention stacks Q, K and V
// (qkv_fusion picks the grouping: one stack, Q and K stacked plus V, or
// three separate contractions); encoder/decoder attention stacks K and V of
// the memory.
struct ProjGroup { int s0, s1; const char* sub; };
int proj_groups(int fusion, ProjGroup* g) {
    if (fusion == 1) { g[0] = {0, 2, ""}; g[1] = {2, 3, "v"}; return 2; }
    if (fusion == 2) { g[0] = {0, 1, ""}; g[1] = {1, 2, "k"}; g[2] = {2, 3, "v"}; return 3; }
    g[0] = {0, 3, ""};
    return 1;
}

int project_segments(const Dims& x, int layout, const void* in, int64_t L, const dm_layer_params* prm,
                     void* const* outs, int s0, int s1, hipStream_t st) {
    const int64_t T = x.B * L, P = x.P, H = x.H;
    const void* w[3] = {prm->wq, prm->wk, prm->wv};
    const void* b[3] = {prm->bq, prm->bk, prm->bv};
    const int ns = s1 - s0;
    Operand A = act_mk(in, layout, T, x.I);
    Operand Bw = opnd(w[s0], true, make_map((uint32_t)P, (uint32_t)H, H * x.I, x.I, 0));
    Epilogue c = epi(outs[s0], make_map((uint32_t)L, 0, P, H * L * P, 0),
                     make_map((uint32_t)P, (uint32_t)H, 1, L * P, 0), true, false);
    for (int i = 0; i < ns; ++i) {
        Bw.ptr[i] = w[s0 + i];
        c.ptr[i] = outs[s0 + i];
        c.bias[i] = b[s0 + i];
    }
    Bw.nseg = ns; c.nseg = ns; c.seg_on_m = 0; c.bias_nseg = ns;
    c.bias_map = make_map((uint32_t)P, (uint32_t)H, H, 1, 0);
    return launch_gemm(x.dtype, gemm(T, ns * H * P, x.I, 1, A, Bw, c), st);
}

// Q, K, V = projections of one input (self-attention), grouped by qkv_fusion.
int project_fused(const Dims& x, int layout, const void* in, const dm_layer_params* prm, void* q, void* k,
                  void* v, hipStream_t st) {
    void* outs[3] = {q, k, v};
    ProjGroup grp[3];
    const int n = proj_groups(x.qkv_fusion, grp);
    for (int i = 0; i < n; ++i) {
        if (i > 0) trace_next(grp[i].sub);
        DM_TRY(project_segments(x, layout, in, x.J, prm, outs, grp[i].s0, grp[i].s1, st));
    }
    return DM_OK;
}

// QK^T -> softmax + dropout -> alpha.V ; gamma token-major [Tq][H][W]
// (and, when gamma32 is not null, the same in fp32 before rounding).
int attention_core_fwd(const Dims& x, float scaler, const DropParams& dp, const void* q, const void* k,
                       const void* v, void* beta, void* prob, void* alpha, void* gamma, float* gamma32,
                       hipStream_t st) {
    const int64_t Z = x.B * x.H, J = x.J, K = x.K, P = x.P, W = x.W, HW = x.H * x.W;
    const int path = current_attn_path();
    if (path != 1 && attn_fused_ok(x.dtype, (int)K, (int)P)) {
        // QK^T and the softmax + dropout in one launch (beta stays on chip),
        // and Gamma in the same launch when its shape allows
        AttnNext nx;
        nx.x = v; nx.x_outer = x.H * K * W; nx.x_inner = K * W; nx.x_ld = W;
        nx.out = gamma; nx.o_outer = J * HW; nx.o_inner = W; nx.o_ld = HW; nx.N = (int)W;
        nx.out_f32 = gamma32;
        const bool with_gamma = path != 2 && attn_next_ok(x.dtype, (int)K, (int)P, nx);
        TraceScope t_(with_gamma ? "F2-4 qkt_softmax_gamma" : "F2-3 qkt_softmax", st);
        // (with Gamma in the same launch alpha stays on chip)
        run_attn_scores_fwd(x.dtype, (int)x.B, (int)x.H, (int)J, (int)K, (int)P, scaler, q, x.H * J * P, J * P, P, k,
                            x.H * K * P, K * P, P, dp, prob, with_gamma ? nullptr : alpha, with_gamma ? &nx : nullptr,
                            st, x.causal);
        DM_TRY(check_launch("attention scores"));
        if (with_gamma) return DM_OK;
    } else {
    // beta[z][j][k] = scaler * sum_p Q[z][j][p] K[z][k][p]
    Epilogue cb = epi(beta, linear_map(K), linear_map(1), true, false, linear_map(J * K));
    cb.alpha = scaler;
    {
        TraceScope t_("F2 qkt", st);
        DM_TRY(launch_gemm(x.dtype,
                           gemm(J, K, P, Z, opnd(q, true, linear_map(P), linear_map(J * P)),
                                opnd(k, true, linear_map(P), linear_map(K * P)), cb),
                           st));
    }
    {
        TraceScope t_("F3 softmax", st);
        run_softmax_fwd(x.dtype, (int)x.B, (int)x.H, (int)J, (int)K, 1.0f, beta, dp, prob, alpha, st, x.causal);
    }
    DM_TRY(check_launch("softmax"));
    }
    // gamma[(b,j)][(h,w)] = sum_k alpha[z][j][k] V[z][k][w]
    TraceScope t_("F4 gamma", st);
    for (int f32 = 0; f32 < (gamma32 ? 2 : 1); ++f32) {
        if (f32) trace_next("fp32");
        Epilogue cg = epi(f32 ? static_cast<void*>(gamma32) : gamma, linear_map(HW), linear_map(1), true, f32 != 0,
                          make_map((uint32_t)x.H, 0, W, J * HW, 0));
        DM_TRY(launch_gemm(x.dtype,
                           gemm(J, W, K, Z, opnd(alpha, true, linear_map(K), linear_map(J * K)),
                                opnd(v, false, linear_map(W), linear_map(K * W)), cg),
                           st));
    }
    return DM_OK;
}

// out(t, i) = sum_{h,w} gamma[t][(h,w)] wo[w][h][i] (+ bo)
int out_projection(const Dims& x, const void* gamma, const void* wo, const void* bo, void* out, int layout,
                   hipStream_t st) {
    const int64_t HW = x.H * x.W;
    Operand A = opnd(gamma, true, linear_map(HW));
    Operand Bw = opnd(wo, false, make_map((uint32_t)x.W, 0, x.H * x.I, x.I, 0));
    Epilogue c = act_out(out, layout, x.Tq, x.I);
    if (bo) { c.bias[0] = bo; c.bias_map = linear_map(1); }
    TraceScope t_("F5 out", st);
    return launch_gemm(x.dtype, gemm(x.Tq, x.I, HW, 1, A, Bw, c), st);
}

// Backward of attention from d(out) (layout `layout`) down to the gradients
// of Q, K, V (written token-major into dq/dk/dv at row strides ldq/ldk/ldv),
// plus dwo.
// Out dW: dwo[w][h][i] = sum_t gamma[t][(h,w)] dout(t,i)
GemmArgs out_dw_args(const Dims& x, const void* gamma, const void* dout, int layout, float* dwo) {
    const int64_t HW = x.H * x.W, I = x.I;
    return gemm(HW, I, x.Tq, 1, opnd(gamma, false, linear_map(HW)), act_kn(dout, layout, x.Tq, I),
                epi(dwo, make_map((uint32_t)x.W, 0, x.H * I, I, 0), linear_map(1), true, true));
}

// dwo == nullptr: the caller launches the output-projection weight gradient
// itself (the encoder pairs it with the Q/K/V weight gradient).  alpha:
// workspace of B*H*J*K elements where the groupings that read alpha
// re-form it from P.
int attention_core_bwd(const Dims& x, float scaler, const DropParams& dp, const void* dout, int layout,
                       const void* q, const void* k, const void* v, const void* prob, void* alpha,
                       const void* gamma, const float* gamma32, const void* wo, float* dwo, void* dgamma,
                       void* dalpha, void* dbeta,
                       void* dq, int64_t ldq, void* dk, int64_t ldk, void* dv, int64_t ldv, hipStream_t st) {
    const int64_t Z = x.B * x.H, J = x.J, K = x.K, P = x.P, W = x.W, H = x.H, HW = x.H * x.W, I = x.I;
    // Out dX: dgamma[t][(h,w)] = sum_i dout(t,i) wo[w][h][i]
    TraceScope t11("B11 out_dx", st);
    DM_TRY(launch_gemm(x.dtype,
                       gemm(x.Tq, HW, I, 1, act_mk(dout, layout, x.Tq, I),
                            opnd(wo, true, make_map((uint32_t)W, 0, H * I, I, 0)),
                            epi(dgamma, linear_map(HW), linear_map(1), true, false)),
                       st));
    t11.stop();
    if (dwo) {
        TraceScope t12("B12 out_dw", st);
        DM_TRY(launch_gemm(x.dtype, out_dw_args(x, gamma, dout, layout, dwo), st));
    }
    const IdxMap zg = make_map((uint32_t)H, 0, W, J * HW, 0);  // z=(b,h) -> gamma-like token-major offset
    const int path = current_attn_path();
    if ((path == 0 || path == 3) && gamma32 && attn_keys_ok(x.dtype, (int)K, (int)P, (int)W)) {
        // Gamma dX1, the softmax + dropout backward, Gamma dX2 and both QK^T
        // gradients in one launch over key blocks, reading P once (dQ
        // partial sums of several key blocks added by a second launch)
        TraceScope t_("B13-17 score_bwd_keys", st);
        run_attn_bwd_keys(x.dtype, (int)x.B, (int)H, (int)J, (int)K, scaler, AttnRows{q, H * J * P, J * P, P},
                          AttnRows{k, H * K * P, K * P, P}, AttnRows{v, H * K * W, K * W, W},
                          AttnRows{dgamma, J * HW, W, HW}, AttnRows{gamma32, J * HW, W, HW}, prob, dp,
                          AttnRows{dq, J * ldq, P, ldq}, AttnRows{dk, K * ldk, P, ldk}, AttnRows{dv, K * ldv, W, ldv},
                          reinterpret_cast<float*>(dalpha), st);
        return check_launch("attention key-block backward");
    }
    {
        TraceScope t_("B14a alpha", st);
        run_alpha_from_prob(x.dtype, (int)x.B, (int)H, (int)J, (int)K, prob, dp, alpha, st);
    }
    DM_TRY(check_launch("alpha from P"));
    const bool fused = path != 1 && attn_fused_ok(x.dtype, (int)K, (int)W);
    AttnNext nq;
    nq.x = k; nq.x_outer = H * K * P; nq.x_inner = K * P; nq.x_ld = P;
    nq.out = dq; nq.o_outer = J * ldq; nq.o_inner = P; nq.o_ld = ldq; nq.N = (int)P;
    const bool with_dq = fused && path != 2 && attn_next_ok(x.dtype, (int)K, (int)W, nq);
    if (fused) {
        // Gamma dX1 and the scaled softmax + dropout backward in one launch
        // (dalpha stays on chip): dbeta[z][j][k]; QK^T dX1 in the same
        // launch when its shape allows
        TraceScope t_(with_dq ? "B13+15+16 score_bwd_dq" : "B13-15 gamma_dx1_softmax_bwd", st);
        run_attn_scores_bwd(x.dtype, (int)x.B, (int)H, (int)J, (int)K, (int)W, scaler, dgamma, J * HW, W, HW, v,
                            H * K * W, K * W, W, prob, dp, dbeta, with_dq ? &nq : nullptr, st);
        DM_TRY(check_launch("attention score backward"));
    } else {
    // Gamma dX1: dalpha[z][j][k] = sum_w dgamma[(b,j)][(h,w)] V[z][k][w]
    TraceScope t13("B13 gamma_dx1", st);
    DM_TRY(launch_gemm(x.dtype,
                       gemm(J, K, W, Z, opnd(dgamma, true, linear_map(HW), zg),
                            opnd(v, true, linear_map(W), linear_map(K * W)),
                            epi(dalpha, linear_map(K), linear_map(1), true, false, linear_map(J * K))),
                       st));
    t13.stop();
    }
    // Gamma dX2: dV[z][k][w] = sum_j alpha[z][j][k] dgamma[(b,j)][(h,w)]
    TraceScope t14("B14 gamma_dx2", st);
    DM_TRY(launch_gemm(x.dtype,
                       gemm(K, W, J, Z, opnd(alpha, false, linear_map(K), linear_map(J * K)),
                            opnd(dgamma, false, linear_map(HW), zg),
                            epi(dv, linear_map(ldv), linear_map(1), true, false,
                                make_map((uint32_t)H, 0, W, K * ldv, 0))),
                       st));
    t14.stop();
    if (!fused) {
        // Scaled softmax dX
        TraceScope t15("B15 softmax_bwd", st);
        run_softmax_bwd(x.dtype, (int)x.B, (int)H, (int)J, (int)K, scaler, dalpha, prob, dp, dbeta, st);
        DM_TRY(check_launch("softmax backward"));
    }
    if (!with_dq) {
        // QK^T dX1: dQ[z][j][p] = sum_k dbeta[z][j][k] K[z][k][p]
        TraceScope t16("B16 qkt_dx1", st);
        DM_TRY(launch_gemm(x.dtype,
                           gemm(J, P, K, Z, opnd(dbeta, true, linear_map(K), linear_map(J * K)),
                                opnd(k, false, linear_map(P), linear_map(K * P)),
                                epi(dq, linear_map(ldq), linear_map(1), true, false,
                                    make_map((uint32_t)H, 0, P, J * ldq, 0))),
                           st));
    }
    // QK^T dX2: dK[z][k][p] = sum_j dbeta[z][j][k] Q[z][j][p]
    TraceScope t17("B17 qkt_dx2", st);
    DM_TRY(launch_gemm(x.dtype,
                       gemm(K, P, J, Z, opnd(dbeta, false, linear_map(K), linear_map(J * K)),
                            opnd(q, false, linear_map(P), linear_map(J * P)),
                            epi(dk, linear_map(ldk), linear_map(1), true, false,
                                make_map((uint32_t)H, 0, P, K * ldk, 0))),
                       st));
    return DM_OK;
}

// dX(t,i) = sum_{(h,n)} dproj[t][(h,n)] w[n][h][i] and dw[n][h][i] = sum_t dproj[t][(h,n)] X(t,i).
int project_bwd(const Dims& x, int layout, const void* in, int64_t T, int64_t n, const void* dproj, int64_t ld,
                const void* w, void* dx, float* dw, const void* resid, hipStream_t st) {
    const int64_t H = x.H, I = x.I;
    if (dx) {
        Epilogue c = act_out(dx, layout, T, I);
        c.resid = resid;
        DM_TRY(launch_gemm(x.dtype,
                           gemm(T, I, H * n, 1, opnd(dproj, true, linear_map(ld)),
                                opnd(w, false, make_map((uint32_t)n, 0, H * I, I, 0)), c),
                           st));
    }
    return launch_gemm(x.dtype,
                       gemm(H * n, I, T, 1, opnd(dproj, false, linear_map(ld)), act_kn(in, layout, T, I),
                            epi(dw, make_map((uint32_t)n, 0, H * I, I, 0), linear_map(1), true, true)),
                       st);
}

// Backward of stacked projections on a token-major [T][nseg][H][P]
// gradient dstk whose segment 0 is weight segment `seg0`: per group,
// dX += dstk[:, segments] [Wq Wk Wv][segments] (the first group adds
// `resid`, later ones add the dX written so far, each output element read
// and written by the same thread) and d[Wq Wk Wv][segments] = dstk[:,
// segments]^T X.
// pair: a further contraction launched together with the first group's
// weight gradient (one launch when both fit the chip at once).
// bias (optional, a single group of all nseg segments only): the weight
// gradient contraction also takes the input-bias gradients, as partial row
// sums of its dstk^T operand over the tokens (bias->part, at most
// bias->cap rows of nseg * H * P floats) where its kernel allows;
// bias->parts is the number of partial rows written (0: none).
struct BiasParts {
    float* part;
    int cap;
    int parts;
};
int project_stacked_bwd(const Dims& x, int layout, const void* in, int64_t T, const void* dstk, int nseg, int seg0,
                        const ProjGroup* grp, int n, const dm_layer_params* prm, void* dx, const dm_layer_grads* g,
                        const void* resid, hipStream_t st, const GemmArgs* pair = nullptr,
                        BiasParts* bias = nullptr) {
    const int64_t H = x.H, I = x.I, P = x.P, HP = H * P, ld = nseg * HP;
    const IdxMap wmap = make_map((uint32_t)P, (uint32_t)H, H * I, I, 0);
    const void* w[3] = {prm->wq, prm->wk, prm->wv};
    float* dw[3] = {g->dwq, g->dwk, g->dwv};
    {
        TraceScope t_("B18 qkv_dx", st);
        for (int i = 0; i < n; ++i) {
            const int s0 = grp[i].s0, ns = grp[i].s1 - grp[i].s0;
            if (i > 0) trace_next(grp[i].sub);
            Epilogue c = act_out(dx, layout, T, I);
            c.resid = i == 0 ? resid : dx;
            Operand Bw = opnd(w[s0], false, wmap);
            for (int j = 0; j < ns; ++j) Bw.ptr[j] = w[s0 + j];
            Bw.nseg = ns;
            const void* a = B8(dstk, (size_t)x.es * (s0 - seg0) * HP);
            DM_TRY(launch_gemm(x.dtype, gemm(T, I, ns * HP, 1, opnd(a, true, linear_map(ld)), Bw, c), st));
        }
    }
    TraceScope t_(pair ? "B12+19 out_dw+qkv_dw" : "B19 qkv_dw", st);
    if (bias) bias->parts = 0;
    const bool want_bias = bias && n == 1 && grp[0].s1 - grp[0].s0 == nseg;
    for (int i = 0; i < n; ++i) {
        const int s0 = grp[i].s0, ns = grp[i].s1 - grp[i].s0;
        if (i > 0) trace_next(grp[i].sub);
        Epilogue cw = epi(dw[s0], wmap, linear_map(1), true, true);
        for (int j = 0; j < ns; ++j) cw.ptr[j] = dw[s0 + j];
        cw.nseg = ns; cw.seg_on_m = 1;
        if (want_bias) {
            // row (s, h, p) of dstk^T, partial sums in the same column order
            cw.rsum = bias->part; cw.rsum_ld = (int)(ns * HP); cw.rsum_cap = bias->cap;
        }
        const void* a = B8(dstk, (size_t)x.es * (s0 - seg0) * HP);
        const GemmArgs gw = gemm(ns * HP, I, T, 1, opnd(a, false, linear_map(ld)), act_kn(in, layout, T, I), cw);
        if (i == 0 && pair) DM_TRY(launch_gemm_pair(x.dtype, gw, *pair, st));
        else DM_TRY(launch_gemm(x.dtype, gw, st));
        if (want_bias) bias->parts = gemm_rowsum_parts();
    }
    return DM_OK;
}

// Backward of project_fused on the token-major [T][3][H][P] gradient.
int project_fused_bwd(const Dims& x, int layout, const void* in, const void* dqkv, const dm_layer_params* prm,
                      void* dx, const dm_layer_grads* g, const void* resid, hipStream_t st,
                      const GemmArgs* pair = nullptr, BiasParts* bias = nullptr) {
    ProjGroup grp[3];
    const int n = proj_groups(x.qkv_fusion, grp);
    return project_stacked_bwd(x, layout, in, x.Tq, dqkv, 3, 0, grp, n, prm, dx, g, resid, st, pair, bias);
}

}  // namespace

extern "C" {

// ------------------------------------------------------------ encoder layer
int encoder_layer_sizes(const dm_layer_desc* d, size_t* saved_bytes, size_t* fwd_ws_bytes, size_t* bwd_ws_bytes) {
    DM_TRY(check_desc(d, true));
    EncPlan e = plan_encoder(dims_of(d));
    if (saved_bytes) *saved_bytes = e.saved_total;
    if (fwd_ws_bytes) *fwd_ws_bytes = e.fwd_total;
    if (bwd_ws_bytes) *bwd_ws_bytes = e.bwd_total;
    return DM_OK;
}

int attn_backward_form(const dm_layer_desc* d, int32_t* key_blocks) {
    DM_TRY(check_desc(d, false));
    if (!key_blocks) return set_error(DM_ERR_ARG, "key_blocks is NULL");
    PlanScope plan_(d->plan);
    const int path = current_attn_path();
    *key_blocks = (path == 0 || path == 3) && attn_keys_ok(d->dtype, d->K, d->P, d->W);
    return DM_OK;
}

int saved_tensor_view(const dm_layer_desc* d, int32_t id, size_t* offset, size_t* bytes) {
    DM_TRY(check_desc(d, true));
    const Dims x = dims_of(d);
    EncPlan e = plan_encoder(x);
    const size_t es = x.es;
    size_t o = 0, b = 0;
    switch (id) {
        case DM_SAVED_QKV: o = e.m.q; b = 3 * es * x.N; break;
        case DM_SAVED_PROB: o = e.m.prob; b = es * x.S; break;
        case DM_SAVED_ALPHA:
            return set_error(DM_ERR_ARG, "alpha is not saved: the backward re-forms it from P and the dropout mask");
        case DM_SAVED_GAMMA: o = e.m.gamma; b = es * x.N; break;
        case DM_SAVED_XHAT1: o = e.xhat1; b = es * x.N; break;
        case DM_SAVED_RSTD1: o = e.rstd1; b = 4 * x.Tq; break;
        case DM_SAVED_Y1: o = e.y1; b = es * x.N; break;
        case DM_SAVED_H: o = e.h; b = es * x.Tq * x.F; break;
        case DM_SAVED_A: o = e.a; b = es * x.Tq * x.F; break;
        case DM_SAVED_XHAT2: o = e.xhat2; b = es * x.N; break;
        case DM_SAVED_RSTD2: o = e.rstd2; b = 4 * x.Tq; break;
        default: return set_error(DM_ERR_ARG, "unknown saved tensor id %d", id);
    }
    if (offset) *offset = o;
    if (bytes) *bytes = b;
    return DM_OK;
}

int encoder_layer_fwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* x_in, void* y, void* saved,
                      void* ws, size_t ws_bytes, void* stream) {
    DM_TRY(check_desc(d, true));
    DM_TRY(check_params(prm, true));
    DM_TRY(need(x_in, "x")); DM_TRY(need(y, "y")); DM_TRY(need(saved, "saved")); DM_TRY(need(ws, "ws"));
    const Dims x = dims_of(d);
    const EncPlan e = plan_encoder(x);
    if (ws_bytes < e.fwd_total) return set_error(DM_ERR_WORKSPACE, "forward workspace too small");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    PlanScope plan_(d->plan);
    SplitScope split_(B8(ws, e.fwd_split), e.split_floats);
    const int dt = x.dtype;
    const int64_t T = x.Tq;
    void *q = B8(saved, e.m.q), *k = B8(saved, e.m.k), *v = B8(saved, e.m.v);
    void *prob = B8(saved, e.m.prob), *gamma = B8(saved, e.m.gamma), *alpha = B8(ws, e.m.alpha_f);
    void *xhat1 = B8(saved, e.xhat1), *y1 = B8(saved, e.y1), *hbuf = B8(saved, e.h), *abuf = B8(saved, e.a);
    void* xhat2 = B8(saved, e.xhat2);
    float *rstd1 = (float*)B8(saved, e.rstd1), *rstd2 = (float*)B8(saved, e.rstd2);
    void *beta = B8(ws, e.m.beta), *ao = B8(ws, e.ao), *o = B8(ws, e.o);

    // Q, K, V (algebraically fused) with the input bias
    {
        TraceScope t_("F1 qkv", st);
        DM_TRY(project_fused(x, DM_BJI, x_in, prm, q, k, v, st));
    }
    // QK^T, scaled softmax + dropout, Gamma
    float* gamma32 = e.m.gamma32 ? reinterpret_cast<float*>(B8(saved, e.m.gamma32)) : nullptr;
    DM_TRY(attention_core_fwd(x, scaler_of(d), make_drop(d->p_attn, d->seed, 0, d->layer_id), q, k, v, beta, prob,
                              alpha, gamma, gamma32, st));
    // Out
    DM_TRY(out_projection(x, gamma, prm->wo, nullptr, ao, DM_BJI, st));
    const FusedLayout fl = fused_layout(dt, T, (int)x.I, (int)x.F);
    // bias + dropout + residual + LayerNorm 1
    {
        TraceScope t_("F6 bdrln1", st);
        run_bdrln_fwd(dt, T, (int)x.I, ao, prm->bo, x_in, prm->g1, prm->be1, d->ln_eps,
                      make_drop(d->p_attn_out, d->seed, 1, d->layer_id), y1, xhat1, rstd1, st, fl.ln_lanes);
    }
    DM_TRY(check_launch("bdrln 1"));
    // Linear 1, with bias + activation (+ dropout) in its epilogue where
    // the contraction's kernel stages its output tile (else a launch of its
    // own): both write H and A = dropout(act(H + b1)) from the stored H
    {
        GemmArgs g1 = gemm(T, x.F, x.I, 1, opnd(y1, true, linear_map(x.I)), opnd(prm->w1, true, linear_map(x.I)),
                           epi(hbuf, linear_map(x.F), linear_map(1), true, false));
        g1.c.act_mode = 1; g1.c.act_out = abuf; g1.c.act_bias = prm->b1; g1.c.act = d->act;
        g1.c.act_dp = make_drop(d->p_ffn_act, d->seed, 3, d->layer_id);
        if (gemm_act_fusable(dt, g1)) {
            TraceScope t_("F7+8 linear1_bias_act", st);
            DM_TRY(launch_gemm(dt, g1, st));
        } else {
            g1.c.act_mode = 0;
            {
                TraceScope t_("F7 linear1", st);
                DM_TRY(launch_gemm(dt, g1, st));
            }
            TraceScope t_("F8 bias_act", st);
            run_bias_act_fwd(dt, T, (int)x.F, hbuf, prm->b1, d->act, g1.c.act_dp, abuf, st);
        }
    }
    DM_TRY(check_launch("bias+activation"));
    // Linear 2
    {
        TraceScope t_("F9 linear2", st);
        DM_TRY(launch_gemm(dt,
                           gemm(T, x.I, x.F, 1, opnd(abuf, true, linear_map(x.F)),
                                opnd(prm->w2, true, linear_map(x.F)),
                                epi(o, linear_map(x.I), linear_map(1), true, false)),
                           st));
    }
    // bias + dropout + residual + LayerNorm 2
    TraceScope t10("F10 bdrln2", st);
    run_bdrln_fwd(dt, T, (int)x.I, o, prm->b2, y1, prm->g2, prm->be2, d->ln_eps,
                  make_drop(d->p_ffn_out, d->seed, 2, d->layer_id), y, xhat2, rstd2, st, fl.ln_lanes);
    return check_launch("bdrln 2");
}

int encoder_layer_bwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* x_in, const void* saved,
                      const void* dy, void* dx, const dm_layer_grads* g, void* ws, size_t ws_bytes, void* stream) {
    DM_TRY(check_desc(d, true));
    DM_TRY(check_params(prm, true));
    DM_TRY(check_grads(g, true));
    DM_TRY(need(x_in, "x")); DM_TRY(need(saved, "saved")); DM_TRY(need(dy, "dy")); DM_TRY(need(dx, "dx"));
    DM_TRY(need(ws, "ws"));
    const Dims x = dims_of(d);
    const EncPlan e = plan_encoder(x);
    if (ws_bytes < e.bwd_total) return set_error(DM_ERR_WORKSPACE, "backward workspace too small");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    PlanScope plan_(d->plan);
    SplitScope split_(B8(ws, e.bwd_split), e.split_floats);
    const int dt = x.dtype;
    const int64_t T = x.Tq, I = x.I, F = x.F;
    const int es = x.es;
    const void *q = B8(saved, e.m.q), *k = B8(saved, e.m.k), *v = B8(saved, e.m.v);
    const void *prob = B8(saved, e.m.prob), *gamma = B8(saved, e.m.gamma);
    const float* gamma32 = e.m.gamma32 ? reinterpret_cast<const float*>(B8(saved, e.m.gamma32)) : nullptr;
    void* alpha = B8(ws, e.m.alpha_b);
    const void *xhat1 = B8(saved, e.xhat1), *y1 = B8(saved, e.y1), *hbuf = B8(saved, e.h), *abuf = B8(saved, e.a);
    const void* xhat2 = B8(saved, e.xhat2);
    const float *rstd1 = (const float*)B8(saved, e.rstd1), *rstd2 = (const float*)B8(saved, e.rstd2);
    void *dS2 = B8(ws, e.dS2), *dO = B8(ws, e.dO), *dA = B8(ws, e.dA), *dH = B8(ws, e.dH);
    void *dY1f = B8(ws, e.dY1f), *dS1 = B8(ws, e.dS1), *dAO = B8(ws, e.dAO);
    void *dgamma = B8(ws, e.m.dgamma), *dalpha = B8(ws, e.m.dalpha), *dbeta = B8(ws, e.m.dbeta);
    void* dqkv = B8(ws, e.m.dq);
    // Every column-sum partial set of the layer has its own region; one
    // launch at the end adds them all up (the parameter gradients they give
    // are read by no later step of the backward).
    float* part = (float*)B8(ws, e.m.part);
    float* part_ln2 = (float*)B8(ws, e.part_ln2);
    float* part_act = (float*)B8(ws, e.part_act);
    float* part_ln1 = (float*)B8(ws, e.part_ln1);

    const FusedLayout fl = fused_layout(dt, T, (int)I, (int)F);
    // LayerNorm-2 scale/shift grads, LayerNorm-2 dX, dropout dX, Linear-2 bias grad
    LnBwdArgs l2{};
    l2.form = fl.ln_form; l2.lanes = fl.ln_lanes;
    l2.dtype = dt; l2.rows = T; l2.cols = (int)I; l2.dya = dy; l2.xhat = xhat2; l2.gamma = prm->g2; l2.rstd = rstd2;
    l2.dp = make_drop(d->p_ffn_out, d->seed, 2, d->layer_id); l2.ds = dS2; l2.dsub = dO; l2.part = part_ln2;
    l2.want_dsub_sum = 1;
    // the column-split LayerNorm backward can also write dO transposed, so
    // the Linear-2 weight gradient reads one operand contiguous along the
    // tokens (the plan's layout choice; on by default)
    void* dOT = B8(ws, e.dOT);
    const bool have_dOT = fl.dO_t;
    l2.dsub_t = have_dOT ? dOT : nullptr;
    {
        TraceScope t_("B1-2 ln2_bwd", st);
        run_ln_bwd(l2, st);
    }
    DM_TRY(check_launch("LayerNorm-2 backward"));
    // (with the plan's layout choice, dH also transposed for the Linear-1
    // weight gradient)
    void* dHT = fl.dH_t ? B8(ws, e.dHT) : nullptr;
    // Linear 2 dX; where its kernel stages the output tile (and dH is not
    // wanted transposed), the dropout / activation backward runs in its
    // epilogue: dH is stored in place of dA, with the Linear-1 bias
    // gradient's partial column sums
    GemmArgs g3 = gemm(T, F, I, 1, opnd(dO, true, linear_map(I)), opnd(prm->w2, false, linear_map(F)),
                       epi(dA, linear_map(F), linear_map(1), true, false));
    g3.c.act_mode = 2; g3.c.act_in = hbuf; g3.c.act_bias = prm->b1; g3.c.act = d->act;
    g3.c.act_dp = make_drop(d->p_ffn_act, d->seed, 3, d->layer_id);
    g3.c.act_part = part_act; g3.c.act_part_cap = colsum_blocks(T);
    g3.c.ptr[0] = dH;
    int act_parts = 0;
    if (!dHT && gemm_act_fusable(dt, g3)) {
        TraceScope t_("B3+5 linear2_dx_act_bwd", st);
        DM_TRY(launch_gemm(dt, g3, st));
        act_parts = gemm_act_parts();
        if (act_parts <= 0) return set_error(DM_ERR_DEVICE, "activation backward epilogue not taken");
    } else {
        g3.c.act_mode = 0;
        g3.c.ptr[0] = dA;
        TraceScope t_("B3 linear2_dx", st);
        DM_TRY(launch_gemm(dt, g3, st));
    }
    {
        TraceScope t_("B4 linear2_dw", st);
        const Operand a_op = have_dOT ? opnd(dOT, true, linear_map(T)) : opnd(dO, false, linear_map(I));
        DM_TRY(launch_gemm(dt,
                           gemm(I, F, T, 1, a_op, opnd(abuf, false, linear_map(F)),
                                epi(g->dw2, linear_map(F), linear_map(1), true, true)),
                           st));
    }
    // dropout / activation backward, Linear-1 bias grad (unless in B3)
    if (!act_parts) {
        TraceScope t_("B5 act_bwd", st);
        run_act_bwd(dt, T, (int)F, dA, hbuf, prm->b1, d->act, g3.c.act_dp, dH, part_act, st, dHT);
    }
    DM_TRY(check_launch("activation backward"));
    // Linear 1 dX and dW
    {
        TraceScope t_("B6 linear1_dx", st);
        DM_TRY(launch_gemm(dt,
                           gemm(T, I, F, 1, opnd(dH, true, linear_map(F)), opnd(prm->w1, false, linear_map(I)),
                                epi(dY1f, linear_map(I), linear_map(1), true, false)),
                           st));
    }
    {
        TraceScope t_("B7 linear1_dw", st);
        const Operand a_op = dHT ? opnd(dHT, true, linear_map(T)) : opnd(dH, false, linear_map(F));
        DM_TRY(launch_gemm(dt,
                           gemm(F, I, T, 1, a_op, opnd(y1, false, linear_map(I)),
                                epi(g->dw1, linear_map(I), linear_map(1), true, true)),
                           st));
    }
    // residual + LayerNorm-1 scale/shift grads, LayerNorm-1 dX, dropout dX, output-bias grad
    LnBwdArgs l1{};
    l1.dtype = dt; l1.rows = T; l1.cols = (int)I; l1.dya = dY1f; l1.dyb = dS2; l1.xhat = xhat1; l1.gamma = prm->g1;
    l1.rstd = rstd1; l1.dp = make_drop(d->p_attn_out, d->seed, 1, d->layer_id); l1.ds = dS1; l1.dsub = dAO;
    l1.part = part_ln1; l1.want_dsub_sum = 1; l1.form = fl.ln_form; l1.lanes = fl.ln_lanes;
    {
        TraceScope t_("B8-10 ln1_bwd", st);
        run_ln_bwd(l1, st);
    }
    DM_TRY(check_launch("LayerNorm-1 backward"));
    // attention backward into the token-major [T][3][H][P] gradient
    const int64_t ld = 3 * I;
    // (the output-projection weight gradient waits for the Q/K/V weight
    // gradient: the two contractions share one launch)
    DM_TRY(attention_core_bwd(x, scaler_of(d), make_drop(d->p_attn, d->seed, 0, d->layer_id), dAO, DM_BJI, q, k, v,
                              prob, alpha, gamma, gamma32, prm->wo, nullptr, dgamma, dalpha, dbeta, dqkv, ld,
                              B8(dqkv, (size_t)es * I), ld, B8(dqkv, (size_t)es * 2 * I), ld, st));
    // Q, K, V dX (fused) + encoder-input residual; Q, K, V dW (fused) with Out dW
    const GemmArgs out_dw = out_dw_args(x, gamma, dAO, DM_BJI, g->dwo);
    // (the Q/K/V weight gradient also takes partial column sums of dQKV for
    // the input-bias gradients (B20), where its kernel allows)
    const int ncs = colsum_blocks(T);
    BiasParts bias = {part, ncs, 0};
    DM_TRY(project_fused_bwd(x, DM_BJI, x_in, dqkv, prm, dx, g, dS1, st, &out_dw, &bias));
    // input-bias partial sums otherwise
    if (bias.parts == 0) {
        TraceScope t20("B20 qkv_bias_grad", st);
        run_colsum_partial(dt, T, (int)(3 * I), dqkv, part, st);
    }
    // LayerNorm-2 (dgamma2, dbeta2, db2), activation (db1), LayerNorm-1
    // (dgamma1, dbeta1, dbo) and input-bias (dbq, dbk, dbv) column sums
    const int nln = ln_bwd_blocks(T, (int)I, dt, fl.ln_form);
    const FinishJob jobs[4] = {finish_job3(part_ln2, nln, (int)I, g->dg2, g->dbe2, g->db2),
                               finish_job(part_act, act_parts ? act_parts : act_bwd_blocks(T, dHT != nullptr),
                                          (int)F, g->db1),
                               finish_job3(part_ln1, nln, (int)I, g->dg1, g->dbe1, g->dbo),
                               finish_job_qkv(part, bias.parts ? bias.parts : ncs, (int)x.H, (int)x.P, 3, g->dbq,
                                              g->dbk, g->dbv)};
    TraceScope tf("B colsum finish", st);
    run_colsum_finish_jobs(jobs, 4, st);
    return check_launch("input-bias backward");
}

// ------------------------------------------------------------ attention only
int mha_sizes(const dm_layer_desc* d, size_t* saved_bytes, size_t* fwd_ws_bytes, size_t* bwd_ws_bytes) {
    DM_TRY(check_desc(d, false));
    MhaSizes s = plan_mha(dims_of(d), d->self_attention);
    if (saved_bytes) *saved_bytes = s.saved;
    if (fwd_ws_bytes) *fwd_ws_bytes = s.fwd;
    if (bwd_ws_bytes) *bwd_ws_bytes = s.bwd;
    return DM_OK;
}

int mha_fwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* qin, const void* kin, const void* vin,
            void* out, void* saved, void* ws, size_t ws_bytes, void* stream) {
    DM_TRY(check_desc(d, false));
    DM_TRY(check_params(prm, false));
    const int mode = d->self_attention;
    DM_TRY(need(qin, "q")); DM_TRY(need(out, "out")); DM_TRY(need(saved, "saved")); DM_TRY(need(ws, "ws"));
    if (mode == PROJ_QKV) {
        if ((kin && kin != qin) || (vin && vin != qin))
            return set_error(DM_ERR_ARG, "self-attention needs k and v NULL or equal to q");
    } else if (mode == PROJ_KV) {
        DM_TRY(need(kin, "k"));
        if (vin && vin != kin) return set_error(DM_ERR_ARG, "a fused K/V projection needs v NULL or equal to k");
    } else {
        DM_TRY(need(kin, "k")); DM_TRY(need(vin, "v"));
    }
    const Dims x = dims_of(d);
    const MhaSizes s = plan_mha(x, mode);
    if (ws_bytes < s.fwd) return set_error(DM_ERR_WORKSPACE, "forward workspace too small");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    PlanScope plan_(d->plan);
    SplitScope split_(B8(ws, s.fwd_split), s.split_floats);
    void *q = B8(saved, s.p.q), *k = B8(saved, s.p.k), *v = B8(saved, s.p.v);
    if (mode == PROJ_QKV) {
        TraceScope t_("F1 qkv", st);
        DM_TRY(project_fused(x, x.layout, qin, prm, q, k, v, st));
    } else if (mode == PROJ_KV) {
        // queries from q; keys and values of the one memory tensor k with
        // [Wk Wv] stacked (one contraction)
        TraceScope t_("F1 q,kv", st);
        DM_TRY(project(x, x.layout, qin, x.J, x.P, prm->wq, prm->bq, q, st));
        trace_next("kv");
        void* outs[3] = {q, k, v};
        DM_TRY(project_segments(x, x.layout, kin, x.K, prm, outs, 1, 3, st));
    } else {
        TraceScope t_("F1 q,k,v", st);
        DM_TRY(project(x, x.layout, qin, x.J, x.P, prm->wq, prm->bq, q, st));
        DM_TRY(project(x, x.layout, kin, x.K, x.P, prm->wk, prm->bk, k, st));
        DM_TRY(project(x, x.layout, vin, x.K, x.W, prm->wv, prm->bv, v, st));
    }
    DM_TRY(attention_core_fwd(x, scaler_of(d), make_drop(d->p_attn, d->seed, 0, d->layer_id), q, k, v,
                              B8(ws, s.p.beta), B8(saved, s.p.prob), B8(ws, s.p.alpha_f), B8(saved, s.p.gamma),
                              s.p.gamma32 ? reinterpret_cast<float*>(B8(saved, s.p.gamma32)) : nullptr, st));
    return out_projection(x, B8(saved, s.p.gamma), prm->wo, prm->bo, out, x.layout, st);
}

int mha_bwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* qin, const void* kin, const void* vin,
            const void* saved, const void* dout, void* dq, void* dk, void* dv, const dm_layer_grads* g, void* ws,
            size_t ws_bytes, void* stream) {
    DM_TRY(check_desc(d, false));
    DM_TRY(check_params(prm, false));
    DM_TRY(check_grads(g, false));
    const int mode = d->self_attention;
    const bool fused = mode == PROJ_QKV;
    DM_TRY(need(qin, "q")); DM_TRY(need(saved, "saved")); DM_TRY(need(dout, "dout")); DM_TRY(need(dq, "dq"));
    DM_TRY(need(ws, "ws"));
    if (fused) {
        if (dk || dv) return set_error(DM_ERR_ARG, "self-attention writes the total input gradient to dq; dk, dv must be NULL");
        if ((kin && kin != qin) || (vin && vin != qin))
            return set_error(DM_ERR_ARG, "self-attention needs k and v NULL or equal to q");
    } else if (mode == PROJ_KV) {
        DM_TRY(need(kin, "k")); DM_TRY(need(dk, "dk"));
        if (vin && vin != kin) return set_error(DM_ERR_ARG, "a fused K/V projection needs v NULL or equal to k");
        if (dv) return set_error(DM_ERR_ARG, "a fused K/V projection writes the memory gradient to dk; dv must be NULL");
    } else {
        DM_TRY(need(kin, "k")); DM_TRY(need(vin, "v")); DM_TRY(need(dk, "dk")); DM_TRY(need(dv, "dv"));
    }
    const Dims x = dims_of(d);
    const MhaSizes s = plan_mha(x, mode);
    if (ws_bytes < s.bwd) return set_error(DM_ERR_WORKSPACE, "backward workspace too small");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    PlanScope plan_(d->plan);
    SplitScope split_(B8(ws, s.bwd_split), s.split_floats);
    const int dt = x.dtype;
    const int es = x.es;
    const void *q = B8(saved, s.p.q), *k = B8(saved, s.p.k), *v = B8(saved, s.p.v);
    void* bq = B8(ws, s.p.dq);
    void* bk = fused ? B8(ws, s.p.dq + (size_t)es * x.H * x.P) : B8(ws, s.p.dk);
    void* bv = fused ? B8(ws, s.p.dq + (size_t)es * 2 * x.H * x.P)
                     : mode == PROJ_KV ? B8(ws, s.p.dk + (size_t)es * x.H * x.P) : B8(ws, s.p.dv);
    float* part = (float*)B8(ws, s.p.part);

    // output-bias grad
    TraceScope t10("B10 out_bias_grad", st);
    if (x.layout == DM_BJI) {
        run_colsum_partial(dt, x.Tq, (int)x.I, dout, part, st);
        trace_next("finish");
        run_colsum_finish(colsum_blocks(x.Tq), (int)x.I, part, g->dbo, st);
    } else {
        run_rowsum(dt, x.I, (int)x.Tq, dout, g->dbo, st);
    }
    DM_TRY(check_launch("output-bias backward"));
    t10.stop();
    DM_TRY(attention_core_bwd(x, scaler_of(d), make_drop(d->p_attn, d->seed, 0, d->layer_id), dout, x.layout, q, k, v,
                              B8(saved, s.p.prob), B8(ws, s.p.alpha_b), B8(saved, s.p.gamma),
                              s.p.gamma32 ? reinterpret_cast<const float*>(B8(saved, s.p.gamma32)) : nullptr,
                              prm->wo, g->dwo,
                              B8(ws, s.p.dgamma), B8(ws, s.p.dalpha), B8(ws, s.p.dbeta), bq, s.p.ldq, bk, s.p.ldk, bv,
                              s.p.ldv, st));
    if (fused) {
        BiasParts bias = {part, colsum_blocks(x.Tq), 0};
        DM_TRY(project_fused_bwd(x, x.layout, qin, bq, prm, dq, g, nullptr, st, nullptr, &bias));
        TraceScope t_("B20 qkv_bias_grad", st);
        if (bias.parts == 0) {
            run_colsum_partial(dt, x.Tq, (int)(3 * x.H * x.P), bq, part, st);
            trace_next("finish");
        }
        run_colsum_finish_qkv(bias.parts ? bias.parts : colsum_blocks(x.Tq), (int)x.H, (int)x.P, 3, part, g->dbq,
                              g->dbk, g->dbv, st);
    } else if (mode == PROJ_KV) {
        TraceScope t_("B18-20 q,kv_bwd", st);
        DM_TRY(project_bwd(x, x.layout, qin, x.Tq, x.P, bq, s.p.ldq, prm->wq, dq, g->dwq, nullptr, st));
        const ProjGroup kv = {1, 3, "kv"};
        DM_TRY(project_stacked_bwd(x, x.layout, kin, x.Tk, bk, 2, 1, &kv, 1, prm, dk, g, nullptr, st));
        run_colsum_partial(dt, x.Tq, (int)(x.H * x.P), bq, part, st);
        run_colsum_finish_qkv(colsum_blocks(x.Tq), (int)x.H, (int)x.P, 1, part, g->dbq, nullptr, nullptr, st);
        run_colsum_partial(dt, x.Tk, (int)(2 * x.H * x.P), bk, part, st);
        run_colsum_finish_qkv(colsum_blocks(x.Tk), (int)x.H, (int)x.P, 2, part, g->dbk, g->dbv, nullptr, st);
    } else {
        TraceScope t_("B18-20 q,k,v_bwd", st);
        DM_TRY(project_bwd(x, x.layout, qin, x.Tq, x.P, bq, s.p.ldq, prm->wq, dq, g->dwq, nullptr, st));
        DM_TRY(project_bwd(x, x.layout, kin, x.Tk, x.P, bk, s.p.ldk, prm->wk, dk, g->dwk, nullptr, st));
        DM_TRY(project_bwd(x, x.layout, vin, x.Tk, x.W, bv, s.p.ldv, prm->wv, dv, g->dwv, nullptr, st));
        run_colsum_partial(dt, x.Tq, (int)(x.H * x.P), bq, part, st);
        run_colsum_finish_qkv(colsum_blocks(x.Tq), (int)x.H, (int)x.P, 1, part, g->dbq, nullptr, nullptr, st);
        run_colsum_partial(dt, x.Tk, (int)(x.H * x.P), bk, part, st);
        run_colsum_finish_qkv(colsum_blocks(x.Tk), (int)x.H, (int)x.P, 1, part, g->dbk, nullptr, nullptr, st);
        run_colsum_partial(dt, x.Tk, (int)(x.H * x.W), bv, part, st);
        run_colsum_finish_qkv(colsum_blocks(x.Tk), (int)x.H, (int)x.W, 1, part, g->dbv, nullptr, nullptr, st);
    }
    return check_launch("input-bias backward");
}

}  // extern "C"
