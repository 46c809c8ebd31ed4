"""Pins for the layer oracle (oracle/layer.py), none of which reuse its code.

* contract() equals numpy.einsum for every index spec the layer uses.
* Storage rounding equals torch's fp16 / bf16 casts.
* Forward at p = 0 equals torch.nn.TransformerEncoderLayer (post-LN, exact
  GELU) and torch.nn.MultiheadAttention in float64: library routines.
* Forward and every gradient at p > 0 equal float64 autograd of an
  independent token-major torch composition, with the oracle's dropout
  masks passed in as tensors.
* Every gradient equals central finite differences on tiny shapes, with all
  dropout sites active.
* Invariants: softmax rows sum to one, LayerNorm output has zero mean and
  unit variance before the affine step, the LayerNorm input gradient sums to
  zero over i, the softmax input gradient sums to zero over k.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

from oracle import layer as L
from oracle import philox

torch.set_default_dtype(torch.float64)


def rand_params(rng, cfg, kind="encoder", bias_std=0.1, ln_random=True):
    P, W, H, I, F = cfg.P, cfg.W, cfg.H, cfg.I, cfg.F
    prm = {
        "wq": rng.normal(0, 0.3, (P, H, I)), "bq": rng.normal(0, bias_std, (P, H)),
        "wk": rng.normal(0, 0.3, (P, H, I)), "bk": rng.normal(0, bias_std, (P, H)),
        "wv": rng.normal(0, 0.3, (W, H, I)), "bv": rng.normal(0, bias_std, (W, H)),
        "wo": rng.normal(0, 0.3, (W, H, I)), "bo": rng.normal(0, bias_std, (I,)),
    }
    if kind == "encoder":
        prm.update({
            "g1": 1 + rng.normal(0, 0.2, (I,)) if ln_random else np.ones(I),
            "be1": rng.normal(0, 0.2, (I,)) if ln_random else np.zeros(I),
            "w1": rng.normal(0, 0.3, (F, I)), "b1": rng.normal(0, bias_std, (F,)),
            "w2": rng.normal(0, 0.3, (I, F)), "b2": rng.normal(0, bias_std, (I,)),
            "g2": 1 + rng.normal(0, 0.2, (I,)) if ln_random else np.ones(I),
            "be2": rng.normal(0, 0.2, (I,)) if ln_random else np.zeros(I),
        })
    return prm


# ------------------------------------------------------------------ helpers
SPECS = ["phi,ibj->phbj", "whi,ibk->whbk", "phbk,phbj->hbjk", "whbk,hbjk->whbj",
         "whi,whbj->ibj", "fi,ibj->fbj", "if,fbj->ibj", "whi,ibj->whbj",
         "whbj,ibj->whi", "whbk,whbj->hbjk", "hbjk,whbj->whbk", "hbjk,phbk->phbj",
         "hbjk,phbj->phbk", "phi,phbj->ibj", "phbj,ibj->phi", "if,ibj->fbj",
         "ibj,fbj->if", "fi,fbj->ibj", "fbj,ibj->fi"]


@pytest.mark.parametrize("spec", SPECS)
def test_contract_equals_einsum(spec):
    rng = np.random.default_rng(abs(hash(spec)) % 2**31)
    dims = dict(p=3, w=3, h=2, i=5, b=2, j=4, k=6, f=7)
    sa, sb = spec.split("->")[0].split(",")
    a = rng.normal(size=[dims[c] for c in sa])
    b = rng.normal(size=[dims[c] for c in sb])
    np.testing.assert_allclose(L.contract(spec, a, b), np.einsum(spec, a, b), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dt,tdt", [("f16", torch.float16), ("bf16", torch.bfloat16),
                                    ("f32", torch.float32)])
def test_store_rounding_matches_torch(dt, tdt):
    rng = np.random.default_rng(1)
    x = rng.normal(0, 3, 20000).astype(np.float32).astype(np.float64)
    x = np.concatenate([x, [0.0, -0.0, 1.0, 1 + 2**-8, 1 + 3 * 2**-9, 1 + 2**-11, 1 + 3 * 2**-12]])
    want = torch.from_numpy(x).float().to(tdt).double().numpy()
    np.testing.assert_array_equal(L.store(x, dt), want)


# ------------------------------------------------------ library pins at p=0
def test_encoder_matches_torch_transformer_layer():
    rng = np.random.default_rng(3)
    cfg = L.Config(B=2, J=6, K=6, H=2, P=4, W=4, I=8, F=16, eps=1e-12)
    prm = rand_params(rng, cfg)
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    y, _ = L.encoder_forward(x, prm, cfg)

    I, H, P = cfg.I, cfg.H, cfg.P
    mod = torch.nn.TransformerEncoderLayer(d_model=I, nhead=H, dim_feedforward=cfg.F, dropout=0.0,
                                           activation="gelu", layer_norm_eps=cfg.eps,
                                           batch_first=True, norm_first=False)
    mod.train()  # the library's fused inference path is not float64-capable
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        # torch orders projected features head-major: row h*P + p.
        wqkv = [t(prm[n]).permute(1, 0, 2).reshape(H * P, I) for n in ("wq", "wk", "wv")]
        bqkv = [t(prm[n]).permute(1, 0).reshape(H * P) for n in ("bq", "bk", "bv")]
        mod.self_attn.in_proj_weight.copy_(torch.cat(wqkv))
        mod.self_attn.in_proj_bias.copy_(torch.cat(bqkv))
        mod.self_attn.out_proj.weight.copy_(t(prm["wo"]).permute(2, 1, 0).reshape(I, H * P))
        mod.self_attn.out_proj.bias.copy_(t(prm["bo"]))
        mod.linear1.weight.copy_(t(prm["w1"])); mod.linear1.bias.copy_(t(prm["b1"]))
        mod.linear2.weight.copy_(t(prm["w2"])); mod.linear2.bias.copy_(t(prm["b2"]))
        mod.norm1.weight.copy_(t(prm["g1"])); mod.norm1.bias.copy_(t(prm["be1"]))
        mod.norm2.weight.copy_(t(prm["g2"])); mod.norm2.bias.copy_(t(prm["be2"]))
        ref = mod(t(x)).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-10, atol=1e-10)


def test_mha_matches_torch_multihead_attention_general():
    # general attention: distinct q, k, v and J != K
    rng = np.random.default_rng(4)
    cfg = L.Config(B=2, J=5, K=7, H=2, P=3, W=3, I=6)
    prm = rand_params(rng, cfg, kind="mha")
    q = rng.normal(size=(cfg.I, cfg.B, cfg.J))
    k = rng.normal(size=(cfg.I, cfg.B, cfg.K))
    v = rng.normal(size=(cfg.I, cfg.B, cfg.K))
    out, _ = L.mha_forward_ibj(q, k, v, prm, cfg)
    I, H, P = cfg.I, cfg.H, cfg.P
    mha = torch.nn.MultiheadAttention(I, H, dropout=0.0, batch_first=False)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        mha.in_proj_weight.copy_(torch.cat([t(prm[n]).permute(1, 0, 2).reshape(H * P, I)
                                            for n in ("wq", "wk", "wv")]))
        mha.in_proj_bias.copy_(torch.cat([t(prm[n]).permute(1, 0).reshape(H * P)
                                          for n in ("bq", "bk", "bv")]))
        mha.out_proj.weight.copy_(t(prm["wo"]).permute(2, 1, 0).reshape(I, H * P))
        mha.out_proj.bias.copy_(t(prm["bo"]))
        # torch wants (L, N, E); ours are [I, B, J] -> (J, B, I)
        ref, _ = mha(t(q).permute(2, 1, 0), t(k).permute(2, 1, 0), t(v).permute(2, 1, 0),
                     need_weights=False)
    np.testing.assert_allclose(out, ref.permute(2, 1, 0).numpy(), rtol=1e-10, atol=1e-10)


# ------------------------------------- autograd of an independent composition
def torch_encoder(x, prm, cfg, m_attn, m_ao, m_act, m_ffn):
    """Token-major torch composition of the same layer (float64)."""
    B, J, H, P, W, I = cfg.B, cfg.J, cfg.H, cfg.P, cfg.W, cfg.I

    def proj(wname, bname, n):
        w = prm[wname].permute(1, 0, 2).reshape(H * n, I)       # row h*n + p
        b = prm[bname].permute(1, 0).reshape(H * n)
        return (x @ w.T + b).view(B, J, H, n).permute(0, 2, 1, 3)  # [B,H,J,n]

    q, k, v = proj("wq", "bq", P), proj("wk", "bk", P), proj("wv", "bv", W)
    att = torch.softmax(cfg.s * (q @ k.transpose(-1, -2)), dim=-1)
    att = att * m_attn.permute(1, 0, 2, 3)                       # mask given as [H,B,J,K]
    ctx = (att @ v).permute(0, 2, 1, 3).reshape(B, J, H * W)
    wo = prm["wo"].permute(2, 1, 0).reshape(I, H * W)
    s1 = x + (ctx @ wo.T + prm["bo"]) * m_ao
    y1 = Fnn.layer_norm(s1, (I,), prm["g1"], prm["be1"], cfg.eps)
    u = y1 @ prm["w1"].T + prm["b1"]
    a = (Fnn.gelu(u) if cfg.act == "gelu" else torch.relu(u)) * m_act
    o = a @ prm["w2"].T + prm["b2"]
    return Fnn.layer_norm(y1 + o * m_ffn, (I,), prm["g2"], prm["be2"], cfg.eps)


@pytest.mark.parametrize("act,p_act", [("gelu", 0.0), ("gelu", 0.25), ("relu", 0.25)])
def test_encoder_grads_match_autograd(act, p_act):
    rng = np.random.default_rng(11)
    cfg = L.Config(B=2, J=8, K=8, H=2, P=4, W=4, I=8, F=16, p_attn=0.2, p_attn_out=0.3,
                   p_ffn_out=0.15, p_ffn_act=p_act, seed=99, layer=5, act=act, eps=1e-5)
    prm = rand_params(rng, cfg)
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    dy = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    y, cache = L.encoder_forward(x, prm, cfg)
    dx, grads, _ = L.encoder_backward(dy, cache, prm, cfg)

    # masks straight from the generator, in token-major order
    fac = lambda site, p, shape: torch.from_numpy(philox.dropout_factor(cfg.seed, site, cfg.layer, p, shape))
    m_attn = fac(philox.SITE_ATTN, cfg.p_attn, (cfg.H, cfg.B, cfg.J, cfg.K))
    m_ao = fac(philox.SITE_ATTN_OUT, cfg.p_attn_out, (cfg.B, cfg.J, cfg.I))
    m_act = fac(philox.SITE_FFN_ACT, cfg.p_ffn_act, (cfg.B, cfg.J, cfg.F))
    m_ffn = fac(philox.SITE_FFN_OUT, cfg.p_ffn_out, (cfg.B, cfg.J, cfg.I))
    tp = {n: torch.from_numpy(v.copy()).requires_grad_(True) for n, v in prm.items()}
    tx = torch.from_numpy(x.copy()).requires_grad_(True)
    ty = torch_encoder(tx, tp, cfg, m_attn, m_ao, m_act, m_ffn)
    np.testing.assert_allclose(y, ty.detach().numpy(), rtol=1e-9, atol=1e-10)
    (ty * torch.from_numpy(dy)).sum().backward()
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-8, atol=1e-9)
    for n in prm:
        np.testing.assert_allclose(grads[n], tp[n].grad.numpy(), rtol=1e-8, atol=1e-9, err_msg=n)


# ------------------------------------------------------ finite differences
def _fd_check(f_loss, arrays, analytic, eps=1e-6, max_coords=None, rng=None, tol=2e-6):
    for name, arr in arrays.items():
        flat = arr.reshape(-1)
        idx = np.arange(flat.size)
        if max_coords is not None and flat.size > max_coords:
            idx = rng.choice(flat.size, max_coords, replace=False)
        ga = analytic[name].reshape(-1)
        for c in idx:
            old = flat[c]
            flat[c] = old + eps
            lp = f_loss()
            flat[c] = old - eps
            lm = f_loss()
            flat[c] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - ga[c]) <= tol * max(1.0, abs(num)), (name, int(c), num, ga[c])


def test_encoder_finite_differences_tiny():
    rng = np.random.default_rng(5)
    cfg = L.Config(B=1, J=4, K=4, H=2, P=2, W=2, I=4, F=8, p_attn=0.3, p_attn_out=0.3,
                   p_ffn_out=0.3, p_ffn_act=0.3, seed=7, eps=1e-5)
    prm = rand_params(rng, cfg)
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    dy = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    _, cache = L.encoder_forward(x, prm, cfg)
    dx, grads, _ = L.encoder_backward(dy, cache, prm, cfg)
    loss = lambda: float((L.encoder_forward(x, prm, cfg)[0] * dy).sum())
    grads = dict(grads, x=dx)
    _fd_check(loss, dict(prm, x=x), grads)


def test_encoder_finite_differences_sampled_small_config():
    # 200 sampled coordinates at the tiny fp32 workload's shapes
    rng = np.random.default_rng(6)
    cfg = L.Config(B=2, J=32, K=32, H=2, P=16, W=16, I=32, F=128, p_attn=0.1, p_attn_out=0.1,
                   p_ffn_out=0.1, seed=0, eps=1e-12)
    prm = rand_params(rng, cfg, bias_std=0.02)
    for n in ("wq", "wk", "wv", "wo", "w1", "w2"):
        prm[n] *= 0.2
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    dy = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    _, cache = L.encoder_forward(x, prm, cfg)
    dx, grads, _ = L.encoder_backward(dy, cache, prm, cfg)
    loss = lambda: float((L.encoder_forward(x, prm, cfg)[0] * dy).sum())
    arrays = dict(prm, x=x)
    grads = dict(grads, x=dx)
    names = list(arrays)
    per = max(1, 200 // len(names))
    _fd_check(loss, arrays, grads, max_coords=per, rng=rng, tol=1e-5)


def test_mha_general_finite_differences():
    rng = np.random.default_rng(8)
    cfg = L.Config(B=2, J=3, K=5, H=2, P=2, W=3, I=4, p_attn=0.3, seed=3)
    prm = rand_params(rng, cfg, kind="mha")
    q = rng.normal(size=(cfg.I, cfg.B, cfg.J))
    k = rng.normal(size=(cfg.I, cfg.B, cfg.K))
    v = rng.normal(size=(cfg.I, cfg.B, cfg.K))
    dout = rng.normal(size=(cfg.I, cfg.B, cfg.J))
    _, cache = L.mha_forward_ibj(q, k, v, prm, cfg)
    dq, dk, dv, grads, _ = L.mha_backward_ibj(dout, cache, prm, cfg)
    loss = lambda: float((L.mha_forward_ibj(q, k, v, prm, cfg)[0] * dout).sum())
    _fd_check(loss, dict(prm, q=q, k=k, v=v), dict(grads, q=dq, k=dk, v=dv))


# ------------------------------------------------------------- invariants
def test_invariants():
    rng = np.random.default_rng(9)
    cfg = L.Config(B=2, J=8, K=8, H=2, P=4, W=4, I=16, F=32, p_attn=0.1, p_attn_out=0.1,
                   p_ffn_out=0.1, eps=1e-12)
    prm = rand_params(rng, cfg)
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    dy = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    _, c = L.encoder_forward(x, prm, cfg)
    _, g, inter = L.encoder_backward(dy, c, prm, cfg)
    assert np.abs(c["prob"].sum(axis=-1) - 1).max() < 1e-13
    for xh in (c["xhat1"], c["xhat2"]):
        assert np.abs(xh.mean(axis=0)).max() < 1e-12
        assert np.abs((xh ** 2).mean(axis=0) - 1).max() < 1e-9
    for ds in (inter["dS1"], inter["dS2"]):
        assert np.abs(ds.sum(axis=0)).max() < 1e-11
    assert np.abs((inter["dS2"] * c["xhat2"]).sum(axis=0)).max() < 1e-9
    assert np.abs(inter["dbeta"].sum(axis=-1)).max() < 1e-12
    # dropped attention probabilities carry no value and no gradient of alpha's consumer
    dropped = c["m_attn"] == 0
    assert dropped.any() and np.all(c["alpha"][dropped] == 0)


def test_storage_emulation_close_to_f64():
    rng = np.random.default_rng(10)
    base = dict(B=2, J=16, K=16, H=2, P=8, W=8, I=16, F=64, p_attn=0.1, p_attn_out=0.1,
                p_ffn_out=0.1)
    prm = rand_params(rng, L.Config(**base), bias_std=0.02)
    x = rng.normal(size=(2, 16, 16))
    y64, _ = L.encoder_forward(x, prm, L.Config(**base))
    for dt, tol in (("f32", 1e-6), ("f16", 5e-3), ("bf16", 4e-2)):
        y, _ = L.encoder_forward(x, prm, L.Config(**base, store_dtype=dt))
        rel = np.linalg.norm(y - y64) / np.linalg.norm(y64)
        assert 0 < rel < tol, (dt, rel)
