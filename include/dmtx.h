/*
 * dmtx.h -- C ABI of the MI355X (gfx950) BERT encoder-layer library.
 *
 * The library computes the forward and backward pass of one post-LN BERT
 * encoder layer, and of multi-head attention alone, as restructured in
 * "Data Movement Is All You Need: A Case Study on Optimizing Transformers"
 * (Ivanov, Dryden, Ben-Nun, Li, Hoefler; MLSys 2021).  Index letters follow
 * the paper's problem statement (Fig. 1 caption): P/W key/value projection
 * size, H heads, I embedding size, B batch, J query length, K key/value
 * length.  F (feed-forward width) is this library's letter.
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless stated otherwise.  The caller owns
 *    and allocates every buffer (inputs, outputs, parameters, gradients,
 *    saved activations, workspace); the library never allocates or frees
 *    memory and keeps no pointer after a call returns.
 *  - All work is enqueued on `stream` (a hipStream_t; NULL = default
 *    stream).  Calls do not synchronise; device faults surface at the
 *    caller's next synchronisation.
 *  - Every argument is validated before the first launch: a call that
 *    returns an error has enqueued nothing.  Device pointers must be
 *    16-byte aligned; row lengths (I, F, K, P, W, cols) must be multiples
 *    of 8.  dm_last_error() describes the last failure of the calling thread.
 *  - Parameter gradients are float32 and are overwritten, not accumulated.
 *  - Outputs must not alias inputs.
 *  - Calls are thread-safe.  The library keeps no mutable process-wide
 *    state: configuration plans are immutable objects named by each call's
 *    descriptor, and the optional launch records (plan_log, dm_trace_*)
 *    belong to the calling thread.
 *  - Dropout masks are never stored: each is regenerated from a
 *    counter-based generator (Philox4x32-10, Salmon et al., SC'11) as a
 *    function of (seed, site, layer, logical element index), so a mask is
 *    independent of the physical layout.  Keep iff the element's 32-bit word
 *    < floor((1-p)*2^32); kept values are scaled by 1/(1-p); p = 0 is the
 *    identity.  Sites: 0 attention probabilities, logical order (h,b,j,k);
 *    1 attention-block output, (b,j,i); 2 feed-forward output, (b,j,i);
 *    3 after the feed-forward activation, (b,j,f).
 */
#ifndef DMTX_H
#define DMTX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DM_OK = 0,
    DM_ERR_ARG = 1,          /* null/misaligned pointer, bad size or probability   */
    DM_ERR_UNSUPPORTED = 2,  /* dtype, layout or shape outside the supported set   */
    DM_ERR_WORKSPACE = 3,    /* workspace smaller than the size query returned      */
    DM_ERR_DEVICE = 4        /* a HIP call failed (launch error)                    */
} dm_status;

typedef enum { DM_F32 = 0, DM_F16 = 1, DM_BF16 = 2 } dm_dtype;

/* Activation layouts: DM_BJI = row-major [B][J][I] (token-major);
 * DM_IBJ = row-major [I][B][J], the paper's printed order (Fig. 1a). */
typedef enum { DM_BJI = 0, DM_IBJ = 1 } dm_layout;

typedef enum { DM_GELU = 0, DM_RELU = 1 } dm_act;

/* Configuration plan (opaque, host memory; see plan_create).  A layer or
 * attention call uses the plan its descriptor points to; NULL selects the
 * library's built-in choices. */
typedef struct dm_plan dm_plan;

/* Layer description.  Encoder layer: I == H*P, W == P, J == K, layout BJI.
 * Attention only: any J, K; layout BJI or IBJ. */
typedef struct {
    int32_t B, J, K, H, P, W, I, F;
    int32_t dtype;           /* dm_dtype of activations and weights (accumulation is fp32) */
    int32_t layout;          /* dm_layout of x / y / dy / dx (q, k, v, out for attention)  */
    int32_t act;             /* dm_act of the feed-forward activation (GELU = exact erf)   */
    float scaler;            /* softmax input scale; <= 0 selects 1/sqrt(P)                */
    float ln_eps;            /* LayerNorm epsilon (inside the square root), > 0            */
    float p_attn;            /* dropout on attention probabilities (site 0)                */
    float p_attn_out;        /* dropout on the attention-block output (site 1)             */
    float p_ffn_out;         /* dropout on the feed-forward output (site 2)                */
    float p_ffn_act;         /* dropout after the activation (site 3; the paper's 4th)     */
    uint64_t seed;           /* dropout key                                                */
    uint32_t layer_id;       /* fourth counter word                                        */
    int32_t self_attention;  /* attention only: 1 = q, k, v are one tensor (fused QKV);    */
                             /* 2 = k, v are one memory tensor (fused KV, encoder/decoder */
                             /* attention, W == P); 0 = three tensors                      */
    int32_t causal;          /* 1 = query j attends to keys k <= j only (decoder self-     */
                             /* attention, as in GPT-style layers); needs J == K; 0 = all  */
    int32_t qkv_fusion;      /* self-attention input projections (Sec. "Algebraic Fusion")*/
                             /* 0: [Wq Wk Wv] X as one contraction each way; 1: [Wq Wk] X */
                             /* and Wv X; 2: three separate contractions                   */
    const dm_plan* plan;     /* configuration plan (plan_create), read during the call    */
                             /* only; NULL = built-in choices                              */
} dm_layer_desc;

/* Parameters in the paper's index order (Fig. 1a), row-major, dtype of the
 * layer: wq, wk [P][H][I]; wv, wo [W][H][I]; bq, bk [P][H]; bv [W][H];
 * bo [I]; g1, be1, g2, be2 [I] (LayerNorm scale/shift); w1 [F][I]; b1 [F];
 * w2 [I][F]; b2 [I].  Attention-only calls read wq..bo only. */
typedef struct {
    const void *wq, *bq, *wk, *bk, *wv, *bv, *wo, *bo;
    const void *g1, *be1, *w1, *b1, *w2, *b2, *g2, *be2;
} dm_layer_params;

/* Parameter gradients: float32, same shapes as dm_layer_params. */
typedef struct {
    float *dwq, *dbq, *dwk, *dbk, *dwv, *dbv, *dwo, *dbo;
    float *dg1, *dbe1, *dw1, *db1, *dw2, *db2, *dg2, *dbe2;
} dm_layer_grads;

/* Dropout of one site for the fused-operator entry points (NULL = none). */
typedef struct {
    float p;
    uint32_t site;
    uint32_t layer;
    uint64_t seed;
} dm_dropout;

/* ---------------------------------------------------------------- layer */

/* Byte sizes of the buffers an encoder layer needs: `saved` (written by
 * the forward, read by the backward, opaque), and the forward and backward
 * workspaces.  Returns DM_OK or a validation error. */
int encoder_layer_sizes(const dm_layer_desc* d, size_t* saved_bytes, size_t* fwd_ws_bytes,
                        size_t* bwd_ws_bytes);

/* Forward of one post-LN encoder layer (Table 3 forward rows):
 *   QKV projection with input bias; scaled QK^T; softmax over k with
 *   dropout (site 0); Gamma = alpha.V; Out projection; output bias, dropout
 *   (site 1), residual, LayerNorm 1; Linear 1; bias and activation
 *   (dropout site 3 if p_ffn_act > 0); Linear 2; bias, dropout (site 2),
 *   residual, LayerNorm 2.
 * x, y: [B][J][I] (DM_BJI).  `saved` must stay untouched until the
 * matching encoder_layer_bwd. */
int encoder_layer_fwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* x, void* y,
                      void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward of the same layer (Table 3 backward rows): given dy, writes dx
 * (same layout as x) and all parameter gradients.  x and `saved` are the
 * forward's input and saved buffer. */
int encoder_layer_bwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* x,
                      const void* saved, const void* dy, void* dx, const dm_layer_grads* g,
                      void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------ attention */

/* Sizes for attention only (multi-head attention of Fig. 1a). */
int mha_sizes(const dm_layer_desc* d, size_t* saved_bytes, size_t* fwd_ws_bytes,
              size_t* bwd_ws_bytes);

/* Multi-head attention forward (Fig. 1a) including the output bias:
 *   out = wo . (dropout(softmax(scaler * (wq q + bq)(wk k + bk))) . (wv v + bv)) + bo.
 * q: [I][B][J] or [B][J][I]; k, v: [I][B][K] or [B][K][I]; out like q.
 * With self_attention = 1, q == k == v is required (one fused projection);
 * k and v may then be NULL.  With self_attention = 2, k is the memory that
 * keys and values are both projected from ([Wk Wv] stacked, Sec.
 * "Algebraic Fusion"); v must be NULL or equal to k. */
int mha_fwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* q, const void* k,
            const void* v, void* out, void* saved, void* ws, size_t ws_bytes, void* stream);

/* Multi-head attention backward.  Writes dq, dk, dv (layouts of q, k, v)
 * and the gradients of wq..bo.  With self_attention = 1, dq receives the
 * total input gradient (dq + dk + dv) and dk, dv must be NULL.  With
 * self_attention = 2, dk receives the memory's total gradient (dk + dv)
 * and dv must be NULL. */
int mha_bwd(const dm_layer_desc* d, const dm_layer_params* prm, const void* q, const void* k,
            const void* v, const void* saved, const void* dout, void* dq, void* dk, void* dv,
            const dm_layer_grads* g, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------- fused operators
 * One entry point per fused operator of the paper's kernel list (Sec.
 * "Fusion Implementation"), named here by what it computes, with the
 * paper's kernel name in brackets.  "rows x cols" tensors are row-major
 * with the statistics/bias index as the contiguous `cols` axis; the
 * dropout logical index of element (r, c) is r*cols + c.  dtype is the
 * storage type of every non-float tensor argument.  Operators that reduce
 * over rows (column sums) need `ws` of colsum_ws_bytes(rows, cols) bytes. */

size_t colsum_ws_bytes(int64_t rows, int32_t cols);

/* [drln / bdrln] s = resid + dropout(x + bias); y = gamma * xhat + beta,
 * xhat = (s - mean_c s) * rstd, rstd = 1/sqrt(var_c s + eps) (biased
 * variance).  Writes y, xhat (dtype) and rstd (float [rows]); xhat / rstd
 * may be NULL. */
int bdrln_fwd(int32_t dtype, int64_t rows, int32_t cols, const void* x, const void* bias,
              const void* resid, const void* gamma, const void* beta, float eps,
              const dm_dropout* drop, void* y, void* xhat, float* rstd, void* stream);

/* [sm] rows of length K over a [B][H][J][K] tensor: prob = softmax_k(scale * beta);
 * alpha = dropout(prob) with logical index ((h*B + b)*J + j)*K + k. */
int softmax_dropout_fwd(int32_t dtype, int32_t B, int32_t H, int32_t J, int32_t K, float scale,
                        const void* beta, const dm_dropout* drop, void* prob, void* alpha,
                        void* stream);

/* [brd] y = dropout(act(x + bias)) over rows x cols (bias [cols]). */
int bias_act_fwd(int32_t dtype, int64_t rows, int32_t cols, const void* x, const void* bias,
                 int32_t act, const dm_dropout* drop, void* y, void* stream);

/* [aib] attention input bias on a token-major projection [rows][3][H][P]
 * (P == W): y[r][s][h][p] = x[r][s][h][p] + b_s[p][H-index h], with
 * b_0 = bq, b_1 = bk, b_2 = bv in the paper's [P][H] order. */
int attn_input_bias(int32_t dtype, int64_t rows, int32_t H, int32_t P, const void* x,
                    const void* bq, const void* bk, const void* bv, void* y, void* stream);

/* [bsb] dgamma = sum_r dy * xhat; dbeta = sum_r dy (float [cols]). */
int ln_param_bwd(int32_t dtype, int64_t rows, int32_t cols, const void* dy, const void* xhat,
                 float* dgamma, float* dbeta, void* ws, size_t ws_bytes, void* stream);

/* [blnrd] LayerNorm backward and dropout backward:
 *   ds = rstd * (g - mean_c g - xhat * mean_c(g * xhat)), g = dy * gamma;
 *   dsub = dropout(ds) (the gradient of the sublayer output and its bias).
 * Writes ds (the residual branch's gradient; may be NULL) and dsub. */
int ln_dropout_bwd(int32_t dtype, int64_t rows, int32_t cols, const void* dy, const void* xhat,
                   const void* gamma, const float* rstd, const dm_dropout* drop, void* ds,
                   void* dsub, void* stream);

/* [ebsb] dsum = da + db; dgamma = sum_r dsum * xhat; dbeta = sum_r dsum. */
int residual_ln_param_bwd(int32_t dtype, int64_t rows, int32_t cols, const void* da,
                          const void* db, const void* xhat, void* dsum, float* dgamma,
                          float* dbeta, void* ws, size_t ws_bytes, void* stream);

/* [bdrb] dh = dropout'(da) * act'(h + b1) over rows x F, db1 = sum_r dh;
 * db2 = sum_r dout over rows x I (the following layer's bias gradient). */
int act_bias_bwd(int32_t dtype, int64_t rows, int32_t F, int32_t I, const void* da,
                 const void* h, const void* b1, int32_t act, const dm_dropout* drop,
                 const void* dout, void* dh, float* db1, float* db2, void* ws, size_t ws_bytes,
                 void* stream);

/* [bs] rows of a [B][H][J][K] tensor: dp = dropout'(dalpha) (site/logical
 * index as softmax_dropout_fwd); dbeta = scale * prob * (dp - sum_k dp*prob). */
int softmax_dropout_bwd(int32_t dtype, int32_t B, int32_t H, int32_t J, int32_t K, float scale,
                        const void* dalpha, const void* prob, const dm_dropout* drop,
                        void* dbeta, void* stream);

/* [baob] db = sum_r x over rows x cols (float [cols]). */
int bias_grad(int32_t dtype, int64_t rows, int32_t cols, const void* x, float* db, void* ws,
              size_t ws_bytes, void* stream);

/* [baob] as bias_grad, for callers that cannot allocate device memory
 * (work recorded under stream capture, tight serving loops, harnesses that
 * forbid allocation): no workspace argument; the column partial sums live
 * in a fixed 8 MiB device array inside the library (one per GPU, held until
 * the process ends), enough for colsum_blocks(rows) * cols <= 2^21 floats,
 * i.e. up to 2048 columns at any row count or 4096 columns up to 4096
 * rows; larger shapes return DM_ERR_UNSUPPORTED before any launch.  The
 * call allocates nothing.  `stream` must belong to the current device.
 * Every call on one GPU shares that GPU's array: calls that overlap on a
 * GPU (on different streams, or from different threads) race; serialize
 * them.  Results are bit-identical to bias_grad's. */
int bias_grad_noalloc(int32_t dtype, int64_t rows, int32_t cols, const void* x, float* db,
                      void* stream);

/* [baib] input-bias gradients from a token-major [rows][3][H][P] gradient:
 * db_s[p][h] = sum_r x[r][s][h][p] for s = q, k, v (float, paper order). */
int attn_input_bias_grad(int32_t dtype, int64_t rows, int32_t H, int32_t P, const void* x,
                         float* dbq, float* dbk, float* dbv, void* ws, size_t ws_bytes,
                         void* stream);

/* [bei] out = a + b over n elements. */
int residual_add(int32_t dtype, int64_t n, const void* a, const void* b, void* out,
                 void* stream);

/* ------------------------------------------------------ test hooks */

/* Keep bits (0/1 bytes) of logical elements offset .. offset+n-1 of a
 * dropout site; offset and n multiples of 8.  p = 0 gives all ones. */
int dropout_mask(uint64_t seed, uint32_t site, uint32_t layer, float p, uint64_t offset,
                 uint64_t n, uint8_t* out, void* stream);

/* Location of one saved tensor inside `saved` (ids: see dm_saved_id). */
typedef enum {
    DM_SAVED_QKV = 0,    /* [3][B][H][J][P]: projections with input bias (head-major) */
    DM_SAVED_PROB = 1,   /* [B][H][J][K] softmax output                                */
    DM_SAVED_ALPHA = 2,  /* not saved (DM_ERR_ARG): re-formed from P and the mask      */
    DM_SAVED_GAMMA = 3,  /* [B][J][H][W] attention context                             */
    DM_SAVED_XHAT1 = 4,  /* [B][J][I]                                                  */
    DM_SAVED_RSTD1 = 5,  /* float [B*J]                                                */
    DM_SAVED_Y1 = 6,     /* [B][J][I] LayerNorm-1 output                               */
    DM_SAVED_H = 7,      /* [B][J][F] Linear-1 output before its bias                  */
    DM_SAVED_A = 8,      /* [B][J][F] activation output (after site-3 dropout)         */
    DM_SAVED_XHAT2 = 9,  /* [B][J][I]                                                  */
    DM_SAVED_RSTD2 = 10, /* float [B*J]                                                */
    DM_SAVED_COUNT = 11
} dm_saved_id;
int saved_tensor_view(const dm_layer_desc* d, int32_t id, size_t* offset, size_t* bytes);

/* Which attention-score backward the calls with this descriptor take (its
 * shape, dtype and plan decide): *key_blocks = 1 for the key-block form
 * (Gamma dX1, the softmax + dropout backward and both QK^T gradients in
 * one pass over key blocks: d(alpha) is never stored and the softmax
 * backward's row term is sum_k d(alpha) alpha, formed as d(gamma) . gamma
 * before gamma's rounding), 0 for the row form (d(alpha) stored in the
 * storage type, row term sum_k dP P).  The two differ only in rounding. */
int attn_backward_form(const dm_layer_desc* d, int32_t* key_blocks);

/* General contraction on the library's MFMA kernel, for op-level tests:
 * C[z][m][n] = alpha * sum_k A[z][m][k] * B[z][k][n] (+ bias[n]) with
 * row-major operands, `a_trans` / `b_trans` selecting A stored [K][M] /
 * B stored [N][K]; C dtype = dtype (out_f32 = 1: float C).  Strides in
 * elements between batches: sa, sb, sc.  tile_cfg selects kernel and block
 * tile (register-staged 16x16x32 MFMA kernel: 0: 256x256, 1: 256x128,
 * 2: 128x128, 3: 256x64, 4: 128x64; asynchronous-copy 16x16x32 kernel:
 * 5: 256x128, 6: 128x128, 7: 256x64, 8: 128x64; asynchronous-copy
 * 32x32x16 kernel: 9: 256x256, 10: 256x128 (4 waves), 11: 128x128,
 * 12: 256x128 (8 waves), 13: lean 256x256 kernel with 8 waves of 128x64
 * and 32-wide k-steps (K a multiple of 32, operand maps block-aligned;
 * otherwise run as 14), 14: 256x256 with 8 waves of 128x64, 15: lean
 * 128x128 kernel with 8 waves of 64x32 and 64-wide k-steps (K a multiple
 * of 64; otherwise run as 11), 16: the same tile with two groups of 4
 * waves of 64x64 each taking half of every k-step (otherwise run as 11),
 * 17: lean 256x256 kernel with 4 waves of 128x128 (as 13 otherwise 14),
 * 18: lean 128x128 kernel with 4 waves of 64x64 (as 15 otherwise 11),
 * 19: lean 256x192 kernel with 4 waves of 128x96, for a B operand
 * contiguous along k (otherwise run as 13); 20: the tile and waves of 17
 * with each MFMA issued next to its share of the next fragment reads and
 * operand copies (as 14 otherwise), 21: the same schedule on the tile and
 * waves of 19 (as 20 otherwise), 22: the same schedule on the tile and
 * waves of 18 (as 11 otherwise), 23 and 24: the tile and waves of 13
 * with the two wave rows alternating between reading a k-step's fragments
 * and multiplying them, four and five LDS stages (as 14 otherwise), 25: the
 * same schedule on a 256x192 tile of 8 waves of 64x96, for a B operand
 * contiguous along k (as 23 otherwise);
 * -1: chosen from the shape; other values are
 * DM_ERR_ARG); splits > 1 splits k, using `ws` (ws_bytes >=
 * splits*batch*M*N*4) for partial sums; splits = 0 chooses (no split
 * without ws). */
int contract(int32_t dtype, int32_t batch, int32_t M, int32_t N, int32_t K, float alpha,
             const void* A, int32_t a_trans, int64_t sa, const void* B, int32_t b_trans,
             int64_t sb, const void* bias, void* C, int32_t out_f32, int64_t sc,
             int32_t tile_cfg, int32_t splits, void* ws, size_t ws_bytes, void* stream);

/* ----------------------------------------------------- configuration plans
 * The configuration-selection step (Sec. "Configuration Selection"): the
 * layer and attention entry points choose each contraction's kernel, tile
 * and split factor from its shape, and the attention-score steps' launch
 * grouping by itself; a plan replaces those choices for the calls whose
 * descriptor names it.  A contraction is identified by its sizes, dtype and
 * which operands are contiguous along the contraction index
 * (dm_contract_choice without the label); a plan entry sets its tile_cfg
 * (0..19, as for contract) and split factor (1 = none; larger values are cut
 * to what the call's split-k scratch holds).  Entries that a contraction's
 * operands or epilogue do not allow fall back the way contract's tile_cfg
 * does, so a plan never changes results beyond the order of the fp32
 * accumulation.  attn_path: 0 = automatic, 1 = QK^T, softmax + dropout and
 * Gamma (and their backward steps) as separate launches, 2 = scores kept on
 * chip (QK^T with softmax + dropout, Gamma dX1 with its backward), 3 = as 2
 * with Gamma and QK^T dX1 in the same launches; a grouping a shape does not
 * allow falls back to the next smaller one.
 *
 * plan_create copies the entries into a new immutable plan (host memory,
 * owned by the caller until plan_destroy); it may be shared by any number
 * of descriptors and threads.  Destroy a plan only when no call that names
 * it is running.
 *
 * plan_log(1) clears and starts a record of the contractions the calling
 * thread's layer and attention calls launch (sizes, dtype, operand
 * contiguity, the tile_cfg and splits that ran, and the kernel-timing label
 * when timing is on); plan_log(0) stops it; plan_log_read copies up to `cap`
 * records of the calling thread and sets *count to the number recorded. */
typedef struct {
    int64_t M, N, K, batch;        /* contraction sizes; batch: contractions in one launch */
    int32_t dtype;                 /* dm_dtype                                             */
    int32_t a_kcontig, b_kcontig;  /* 1: operand contiguous along the contraction index   */
    int32_t tile_cfg;              /* 0..25 (contract's list)                              */
    int32_t splits;                /* split-k factor, 1 = none                             */
    char label[48];                /* log only: kernel-timing label, "" when timing is off */
} dm_contract_choice;
/* Layout and reduction choices of the memory-bound fused operators, the
 * plan's counterpart of the contraction entries (Sec. "Data Layout -- Fused
 * Operators"): which producers also write their output transposed, so
 * that the weight-gradient contraction consuming it reads it contiguous
 * along the tokens, and the reduction width of the LayerNorm kernels.
 * -1 in any field keeps the library's choice.  None of them changes
 * results beyond the order of fp32 sums. */
typedef struct {
    int32_t dO_transposed;  /* 1: the LayerNorm-2 backward also writes dO^T ([I][T]) and the    */
                            /* Linear-2 weight gradient reads it (column-split form only);     */
                            /* 0: not.  Library: 1 wherever the column-split form runs          */
    int32_t dH_transposed;  /* 1: the activation backward also writes dH^T ([F][T]) and the    */
                            /* Linear-1 weight gradient reads it (16-bit types); 0: not.        */
                            /* Library: 0                                                       */
    int32_t ln_bwd_form;    /* LayerNorm backward: 1 = one lane group per row, reduced across  */
                            /* its lanes; 2 = column slices of 16-row tiles (16-bit types, I a */
                            /* multiple of 64 in 320..1024).  Library: 2 where allowed         */
    int32_t ln_lanes;       /* lanes per row of the row-form LayerNorm kernels (the forward,   */
                            /* and the backward in form 1): 16, 32 or 64 for rows of 257..1024  */
                            /* elements (each lane holding 8-element vectors of its row).       */
                            /* Library: 64                                                      */
} dm_layout_choice;
/* layout: NULL keeps the library's choice for every field. */
int plan_create(const dm_contract_choice* entries, int32_t n, int32_t attn_path,
                const dm_layout_choice* layout, dm_plan** plan);
int plan_destroy(dm_plan* plan);
int plan_log(int32_t on);
int plan_log_read(dm_contract_choice* out, int32_t cap, int32_t* count);

/* ----------------------------------------------------- kernel timing
 * Optional per-launch timing for measurement: while enabled, every kernel
 * the layer and attention entry points enqueue is bracketed by two HIP
 * events on the call's stream and recorded under a short label naming the
 * paper's operator (e.g. "F7 linear1", "B15 softmax_bwd") and a sub-label
 * ("" for an operator's first launch, e.g. "reduce" or "finish" for the
 * second launch of a two-stage reduction).  Recording adds two event
 * records per launch; leave it off outside measurement.
 * dm_trace_enable(1) clears earlier records; dm_trace_get waits for the
 * i-th record to complete and returns its label and sub-label (static
 * storage) and its duration in milliseconds.  Switch, records and events
 * belong to the calling thread: each thread times its own calls. */
int dm_trace_enable(int32_t on);
int32_t dm_trace_count(void);
int dm_trace_get(int32_t i, const char** label, const char** sub, float* ms);

/* Message for the last non-OK status returned on the calling thread. */
const char* dm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DMTX_H */
