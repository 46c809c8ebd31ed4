"""Multi-head attention and the post-LN BERT encoder layer (oracle).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Everything here is float64 and follows the paper's statement of the problem:
the multi-head-attention einsums of Fig. 1a (index letters P/W, H, I, B, J, K),
and the encoder-layer operator sequence of Table 3 (forward: Q/K/V, input
bias, QK^T, scaled softmax + dropout, Gamma, Out, output bias + dropout +
residual + LayerNorm, Linear, bias + activation, Linear, bias + dropout +
residual + LayerNorm; backward: the same rows in reverse, each contraction
split into its dX and dW parts).  Activations are kept internally in the
paper's (i, b, j) index order.

Readings where the paper is silent or differs from the workloads built here:
  * softmax runs over k, the key index (the last index of beta[h,b,j,k]);
  * scaler = 1/sqrt(P) unless given;
  * the feed-forward activation is GELU in its exact erf form (ReLU is
    available as act="relu"); the paper's fourth dropout (after the
    activation) is the optional site 3, off unless p_ffn_act > 0;
  * inverted dropout: kept elements are scaled by 1/(1-p);
  * LayerNorm normalises over i per token with the biased variance and eps
    inside the square root;
  * post-LN: y = LN(x + dropout(sublayer(x) + bias));
  * the scaling of the softmax input is part of the softmax operator's
    backward (the paper's "bs" kernel: backward dropout and softmax with
    scaling), so d(beta)/d(qq.kk) carries the scaler there.

Mixed precision: the paper stores data in fp16 and accumulates in fp32
(Sec. "Evaluation Details" of the appendix) but does not fix which tensors
are materialised, which depends on the fusion.  With store_dtype set, each
tensor written by a fused operator or contraction is rounded to that
storage type (round-to-nearest-even) where it is written; values that stay
inside one fused operator are not rounded, and a fused operator that writes
two tensors derives both from its unrounded value (e.g. the softmax writes
the probabilities and, from the same unrounded values, the dropped-out
probabilities).  The fusion boundaries are the paper's kernel list, with
two further fusions: the residual + LayerNorm-scale/shift backward ("ebsb")
feeds the LayerNorm backward ("blnrd") directly, and the encoder-input
residual ("bei") is added where the Q/K/V input gradient is formed.  All
arithmetic stays float64; store_dtype "f64" gives the plain definition.

Parity: forward pinned to torch.nn.TransformerEncoderLayer and
torch.nn.MultiheadAttention at p = 0 (float64); forward and every gradient
pinned to float64 autograd of an independent torch composition at p > 0 and
to central finite differences on tiny shapes (tests/test_oracle_layer.py).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, Optional

import numpy as np
from scipy.special import erf

from . import philox


# ----------------------------------------------------------------- rounding
def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage type (RNE) and back to float64."""
    if dtype == "f64":
        return x
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    if dtype == "f16":
        return x.astype(np.float16).astype(np.float64)
    if dtype == "bf16":
        # bfloat16 keeps 8 significant bits; round the float64 significand
        # to 8 bits with ties to even (exact for the normal range).
        m, e = np.frexp(x)
        return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)
    raise ValueError(dtype)


# --------------------------------------------------------------- contraction
def contract(spec: str, a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Two-operand einsum evaluated with a batched matrix product.

    Indices present in both inputs and the output are batch indices, in
    both inputs but not the output are summed, and in one input only are
    free.  Equivalent to numpy.einsum(spec, a, b) (checked in the tests)."""
    ins, out = spec.split("->")
    sa, sb = ins.split(",")
    batch = [c for c in out if c in sa and c in sb]
    summed = [c for c in sa if c in sb and c not in out]
    fa = [c for c in sa if c not in sb]
    fb = [c for c in sb if c not in sa]
    dims = {c: a.shape[sa.index(c)] for c in sa}
    dims.update({c: b.shape[sb.index(c)] for c in sb})
    A = np.transpose(a, [sa.index(c) for c in batch + fa + summed])
    Bm = np.transpose(b, [sb.index(c) for c in batch + summed + fb])
    nb = int(np.prod([dims[c] for c in batch])) if batch else 1
    nfa = int(np.prod([dims[c] for c in fa])) if fa else 1
    nfb = int(np.prod([dims[c] for c in fb])) if fb else 1
    ns = int(np.prod([dims[c] for c in summed])) if summed else 1
    C = np.matmul(A.reshape(nb, nfa, ns), Bm.reshape(nb, ns, nfb))
    C = C.reshape([dims[c] for c in batch + fa + fb])
    order = batch + fa + fb
    return np.ascontiguousarray(np.transpose(C, [order.index(c) for c in out]))


# ----------------------------------------------------------- element-wise ops
def softmax_k(beta: np.ndarray, causal: bool = False) -> np.ndarray:
    """Softmax over the last index (k).  causal: query j (second-to-last
    index) sees keys k <= j only, as in decoder self-attention; the other
    probabilities are exactly zero."""
    if causal:
        J, K = beta.shape[-2], beta.shape[-1]
        if J != K:
            raise ValueError("a causal mask needs as many keys as queries")
        beta = np.where(np.arange(K)[None, :] <= np.arange(J)[:, None], beta, -np.inf)
    z = np.exp(beta - beta.max(axis=-1, keepdims=True))
    return z / z.sum(axis=-1, keepdims=True)


def gelu(u):
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def gelu_grad(u):
    # d/du [u * Phi(u)] = Phi(u) + u * phi(u)
    return 0.5 * (1.0 + erf(u / math.sqrt(2.0))) + u * np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)


def act_fwd(u, act):
    return gelu(u) if act == "gelu" else np.maximum(u, 0.0)


def act_grad(u, act):
    return gelu_grad(u) if act == "gelu" else (u > 0).astype(np.float64)


def layernorm_i(s: np.ndarray, eps: float):
    """Normalise over i (axis 0 of an [I,B,J] tensor): returns x_hat, rstd[b,j]."""
    mu = s.mean(axis=0)
    var = ((s - mu) ** 2).mean(axis=0)
    rstd = 1.0 / np.sqrt(var + eps)
    return (s - mu) * rstd, rstd


def layernorm_i_bwd(dy: np.ndarray, xhat: np.ndarray, rstd: np.ndarray, g: np.ndarray):
    """dS for y = g * x_hat + beta, x_hat = LN_i(S):
    dS = rstd * (gy - mean_i(gy) - x_hat * mean_i(gy * x_hat)), gy = dy * g."""
    gy = dy * g[:, None, None]
    return rstd * (gy - gy.mean(axis=0) - xhat * (gy * xhat).mean(axis=0))


# ------------------------------------------------------------------- config
@dataclass
class Config:
    B: int
    J: int
    K: int
    H: int
    P: int
    W: int
    I: int
    F: int = 0
    p_attn: float = 0.0
    p_attn_out: float = 0.0
    p_ffn_out: float = 0.0
    p_ffn_act: float = 0.0
    seed: int = 0
    layer: int = 0
    scaler: Optional[float] = None
    eps: float = 1e-12
    act: str = "gelu"
    store_dtype: str = "f64"
    causal: bool = False     # decoder self-attention: query j attends to keys k <= j
    # Storage emulation of the attention-score backward (no effect without
    # storage rounding): False, d(alpha) stays inside the fused score
    # backward (not rounded) and the softmax backward's row term is
    # sum_k d(alpha) alpha; True, Gamma dX1 stores d(alpha) in the storage
    # type and the row term is sum_k dP P over it.
    dalpha_stored: bool = False

    @property
    def s(self) -> float:
        return self.scaler if self.scaler is not None else 1.0 / math.sqrt(self.P)


def attn_dropout(cfg: Config) -> np.ndarray:
    """M/(1-p) on beta's logical (h, b, j, k) order."""
    return philox.dropout_factor(cfg.seed, philox.SITE_ATTN, cfg.layer, cfg.p_attn,
                                 (cfg.H, cfg.B, cfg.J, cfg.K))


def token_dropout(cfg: Config, site: int, p: float, width: int) -> np.ndarray:
    """M/(1-p) for a token-major (b, j, i) activation site, returned in the
    internal (i, b, j) order."""
    f = philox.dropout_factor(cfg.seed, site, cfg.layer, p, (cfg.B, cfg.J, width))
    return np.ascontiguousarray(f.transpose(2, 0, 1))


def f64(t) -> np.ndarray:
    """Storage-typed tensor (torch or numpy) -> float64 numpy array."""
    if hasattr(t, "detach"):
        return t.detach().to("cpu").double().numpy()
    return np.asarray(t, dtype=np.float64)


# ------------------------------------------------------ attention (Fig. 1a)
def mha_forward(q, k, v, prm: Dict[str, np.ndarray], cfg: Config, out_bias: bool = True):
    """Multi-head attention on q [I,B,J], k [I,B,K], v [I,B,K].

    Computed one sequence b and one head h at a time as plain matrix
    products, from the index definitions of the attention (Fig. 1a): the
    head's query, key and value rows are its slices of the projection
    weights applied to the token vectors plus the input bias; the scores are
    the scaled query-key dot products; the probabilities are their softmax
    over the keys; the head's context is the dropped-out probabilities
    times the value rows; the output sums every head's context through its
    slice of the output weights.

    Returns (out [I,B,J], cache); cached tensors are kept in the paper's
    index orders (qq, kk [P,H,B,len], vv and gamma [W,H,B,len], beta, prob
    and alpha [H,B,J,K]).  With out_bias=False the output bias bo is left
    out (the encoder layer adds it in its bias/dropout/residual/LayerNorm
    operator, Table 3)."""
    r = lambda x: store(x, cfg.store_dtype)
    B, J, K = q.shape[1], q.shape[2], k.shape[2]
    H, P, W, I = cfg.H, cfg.P, cfg.W, q.shape[0]
    m_attn = attn_dropout(cfg)                                  # [H,B,J,K]
    causal_ok = np.tril(np.ones((J, K), dtype=bool)) if cfg.causal else None
    head_q, head_k = np.empty((P, H, B, J)), np.empty((P, H, B, K))
    head_v, ctx = np.empty((W, H, B, K)), np.empty((W, H, B, J))
    scores, probs, dropped = np.empty((H, B, J, K)), np.empty((H, B, J, K)), np.empty((H, B, J, K))
    out = np.zeros((I, B, J))
    for b in range(B):
        tq, tk, tv = q[:, b, :].T, k[:, b, :].T, v[:, b, :].T   # token vectors, [len, I]
        for h in range(H):
            # rows "Q, K, V" and "Input bias" of Table 3
            Qh = r(tq @ prm["wq"][:, h, :].T + prm["bq"][:, h])    # [J, P]
            Kh = r(tk @ prm["wk"][:, h, :].T + prm["bk"][:, h])    # [K, P]
            Vh = r(tv @ prm["wv"][:, h, :].T + prm["bv"][:, h])    # [K, W]
            Sh = r(cfg.s * (Qh @ Kh.T))                             # [J, K]
            if causal_ok is not None:
                Sh_m = np.where(causal_ok, Sh, -np.inf)
            else:
                Sh_m = Sh
            e = np.exp(Sh_m - Sh_m.max(axis=1, keepdims=True))
            Ph = e / e.sum(axis=1, keepdims=True)                  # softmax over the keys
            # dropout of the probabilities as the operator stores them (rounded):
            # alpha is a function of the stored P and the mask alone
            Ah = r(r(Ph) * m_attn[h, b])
            Ch = r(Ah @ Vh)                                         # [J, W]
            out[:, b, :] += (Ch @ prm["wo"][:, h, :]).T             # the head's share of Out
            head_q[:, h, b, :], head_k[:, h, b, :], head_v[:, h, b, :] = Qh.T, Kh.T, Vh.T
            scores[h, b], probs[h, b], dropped[h, b], ctx[:, h, b, :] = Sh, r(Ph), Ah, Ch.T
    if out_bias:
        out = out + prm["bo"][:, None, None]
    out = r(out)
    cache = dict(q=q, k=k, v=v, qq=head_q, kk=head_k, vv=head_v, beta=scores, prob=probs,
                 m_attn=m_attn, alpha=dropped, gamma=ctx)
    return out, cache


def mha_backward(dout, cache, prm, cfg: Config, out_bias: bool = True):
    """Gradients of mha_forward.  Returns (dq, dk, dv, grads) with dq [I,B,J],
    dk, dv [I,B,K] and grads for wq, bq, wk, bk, wv, bv, wo (and bo)."""
    r = lambda x: store(x, cfg.store_dtype)
    wq, wk, wv, wo = prm["wq"], prm["wk"], prm["wv"], prm["wo"]
    g = {}
    if out_bias:
        g["bo"] = dout.sum(axis=(1, 2))                      # output bias dW
    # Out dX and dW.
    dgamma = r(contract("whi,ibj->whbj", wo, dout))
    g["wo"] = contract("whbj,ibj->whi", cache["gamma"], dout)
    # Gamma dX1 (w.r.t. alpha) and dX2 (w.r.t. vv).
    dalpha = contract("whbk,whbj->hbjk", cache["vv"], dgamma)
    if cfg.dalpha_stored:
        dalpha = r(dalpha)
    dvv = r(contract("hbjk,whbj->whbk", cache["alpha"], dgamma))
    # Scaled softmax dX: dropout backward, softmax backward, scaling.  The
    # row term sum_k dP P equals sum_k d(alpha) alpha (dP = m d(alpha) and
    # alpha = m P, m the dropout factor); with d(alpha) kept inside the
    # fused operator it is taken in that form, with alpha as stored.
    prob = cache["prob"]
    dprob = dalpha * cache["m_attn"]
    if cfg.dalpha_stored:
        row = (dprob * prob).sum(axis=-1, keepdims=True)
    else:
        row = (dalpha * cache["alpha"]).sum(axis=-1, keepdims=True)
    dbeta = r(cfg.s * prob * (dprob - row))
    # QK^T dX1 (w.r.t. qq) and dX2 (w.r.t. kk).
    dqq = r(contract("hbjk,phbk->phbj", dbeta, cache["kk"]))
    dkk = r(contract("hbjk,phbj->phbk", dbeta, cache["qq"]))
    # Q, K, V dX and dW; input-bias dW.
    dq = contract("phi,phbj->ibj", wq, dqq)
    dk = contract("phi,phbk->ibk", wk, dkk)
    dv = contract("whi,whbk->ibk", wv, dvv)
    g["wq"] = contract("phbj,ibj->phi", dqq, cache["q"])
    g["wk"] = contract("phbk,ibk->phi", dkk, cache["k"])
    g["wv"] = contract("whbk,ibk->whi", dvv, cache["v"])
    g["bq"] = dqq.sum(axis=(2, 3))
    g["bk"] = dkk.sum(axis=(2, 3))
    g["bv"] = dvv.sum(axis=(2, 3))
    inter = dict(dgamma=dgamma, dalpha=dalpha, dvv=dvv, dbeta=dbeta, dqq=dqq, dkk=dkk)
    return dq, dk, dv, g, inter


# ------------------------------------------------------------ encoder layer
def encoder_forward(x_bji, prm: Dict[str, np.ndarray], cfg: Config):
    """Post-LN encoder layer on a token-major input x [B,J,I].
    Returns (y [B,J,I], cache)."""
    r = lambda x: store(x, cfg.store_dtype)
    X = np.ascontiguousarray(np.transpose(x_bji, (2, 0, 1)))          # [I,B,J]
    ao, c = mha_forward(X, X, X, prm, cfg, out_bias=False)
    # Output bias, dropout, residual, LayerNorm ("drln"/"bdrln").
    m_ao = token_dropout(cfg, philox.SITE_ATTN_OUT, cfg.p_attn_out, cfg.I)
    s1 = X + (ao + prm["bo"][:, None, None]) * m_ao
    xhat1, rstd1 = layernorm_i(s1, cfg.eps)
    y1 = r(prm["g1"][:, None, None] * xhat1 + prm["be1"][:, None, None])
    # Linear, bias + activation (+ optional dropout), Linear.
    h = r(contract("fi,ibj->fbj", prm["w1"], y1))
    u = h + prm["b1"][:, None, None]
    m_act = token_dropout(cfg, philox.SITE_FFN_ACT, cfg.p_ffn_act, cfg.F)
    a = r(act_fwd(u, cfg.act) * m_act)
    o = r(contract("if,fbj->ibj", prm["w2"], a))
    # Bias, dropout, residual, LayerNorm.
    m_ffn = token_dropout(cfg, philox.SITE_FFN_OUT, cfg.p_ffn_out, cfg.I)
    s2 = y1 + (o + prm["b2"][:, None, None]) * m_ffn
    xhat2, rstd2 = layernorm_i(s2, cfg.eps)
    y = r(prm["g2"][:, None, None] * xhat2 + prm["be2"][:, None, None])
    c.update(X=X, ao=ao, m_ao=m_ao, s1=s1, xhat1=r(xhat1), rstd1=rstd1, y1=y1,
             h=h, u=u, m_act=m_act, a=a, o=o, m_ffn=m_ffn, s2=s2,
             xhat2=r(xhat2), rstd2=rstd2)
    return np.ascontiguousarray(np.transpose(y, (1, 2, 0))), c


def encoder_backward(dy_bji, cache, prm: Dict[str, np.ndarray], cfg: Config):
    """Gradients of encoder_forward.  Returns (dx [B,J,I], grads, intermediates);
    grads are keyed like the parameters and shaped like them."""
    r = lambda x: store(x, cfg.store_dtype)
    dY = np.ascontiguousarray(np.transpose(dy_bji, (2, 0, 1)))        # [I,B,J]
    g = {}
    # LayerNorm dW (bsb).
    g["g2"] = (dY * cache["xhat2"]).sum(axis=(1, 2))
    g["be2"] = dY.sum(axis=(1, 2))
    # LayerNorm dX and dropout dX (blnrd); dS2 also feeds the residual.
    dS2_x = layernorm_i_bwd(dY, cache["xhat2"], cache["rstd2"], prm["g2"])
    dS2 = r(dS2_x)
    dO = r(dS2_x * cache["m_ffn"])
    # Linear (second) dX and dW.
    dA = r(contract("if,ibj->fbj", prm["w2"], dO))
    g["w2"] = contract("ibj,fbj->if", dO, cache["a"])
    # Bias dW, dropout dX, activation dX, bias dW (bdrb).
    g["b2"] = dO.sum(axis=(1, 2))
    dH = r(dA * cache["m_act"] * act_grad(cache["u"], cfg.act))
    g["b1"] = dH.sum(axis=(1, 2))
    # Linear (first) dX and dW.
    dY1f = r(contract("fi,fbj->ibj", prm["w1"], dH))
    g["w1"] = contract("fbj,ibj->fi", dH, cache["y1"])
    # Residual and LayerNorm dW (ebsb), fused with the LayerNorm backward.
    dY1 = dY1f + dS2
    g["g1"] = (dY1 * cache["xhat1"]).sum(axis=(1, 2))
    g["be1"] = dY1.sum(axis=(1, 2))
    # LayerNorm dX and dropout dX (blnrd), output-bias dW (baob).
    dS1_x = layernorm_i_bwd(dY1, cache["xhat1"], cache["rstd1"], prm["g1"])
    dS1 = r(dS1_x)
    dAO = r(dS1_x * cache["m_ao"])
    g["bo"] = dAO.sum(axis=(1, 2))
    # Attention backward (Out ... Q,K,V dW, input-bias dW).
    dq, dk, dv, ga, inter = mha_backward(dAO, cache, prm, cfg, out_bias=False)
    g.update(ga)
    # Encoder-input residual (bei): self-attention sums the three input grads.
    dXa = dq + dk + dv
    dX = r(dXa + dS1)
    inter.update(dS2=dS2, dO=dO, dA=dA, dH=dH, dY1f=dY1f, dY1=dY1, dS1=dS1, dAO=dAO, dXa=dXa)
    return np.ascontiguousarray(np.transpose(dX, (1, 2, 0))), g, inter


# ------------------------------------------------------ attention-only entry
def mha_forward_ibj(q, k, v, prm, cfg: Config):
    """Attention on activations in the paper's [I,B,J] order (with bo)."""
    return mha_forward(q, k, v, prm, cfg, out_bias=True)


def mha_backward_ibj(dout, cache, prm, cfg: Config):
    return mha_backward(dout, cache, prm, cfg, out_bias=True)
