"""Pins for the oracle's storage emulation (store_dtype = "f16" / "bf16").

The emulation rounds to the storage type exactly the tensors the GPU path
writes and nothing else (the materialisation reading of the layer: the
paper fixes fp16 data with fp32 accumulation but not which tensors are
written).  Two things are pinned here, neither by reusing the oracle's
arithmetic:

* the rounding itself: store() is round-to-nearest-even from float64,
  checked by brute force at every midpoint of the fp16 grid (and of a wide
  slice of the bf16 grid), just above and below it and at the tie;
* the rounding points: every tensor the emulation claims is written is
  recomputed by an independent token-major torch composition from the
  oracle's own rounded inputs of that step and rounded once, and must equal
  the oracle's value bit for bit; every value the emulation keeps inside a
  fused operator must not be rounded.  A rounding that is missing,
  misplaced (taken before instead of after a bias or a dropout) or taken
  from the wrong operand (alpha from the unrounded instead of the stored,
  rounded probabilities) fails one of these comparisons.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

from oracle import layer as L
from oracle import philox


# ------------------------------------------------------------ the rounding
def _f16_grid():
    bits = np.arange(0x0400, 0x7BFF, dtype=np.uint16)        # positive normals below the largest
    return bits.view(np.float16).astype(np.float64), (bits + 1).view(np.float16).astype(np.float64), bits


def _bf16_grid():
    exps = np.arange(127 - 40, 127 + 40, dtype=np.uint32)     # 2^-40 .. 2^39
    mant = np.arange(0, 127, dtype=np.uint32)                 # upper neighbour stays in the binade
    hi = (exps[:, None] << 7 | mant[None, :]).reshape(-1)
    lo = (hi.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    up = ((hi.astype(np.uint32) + 1) << 16).view(np.float32).astype(np.float64)
    return lo, up, hi


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_store_is_round_to_nearest_even(dt):
    lo, up, bits = _f16_grid() if dt == "f16" else _bf16_grid()
    mid = 0.5 * (lo + up)                      # exact in float64
    eps = (up - lo) * 2.0 ** -20               # far below half a spacing, far above float64's
    for sgn in (1.0, -1.0):
        np.testing.assert_array_equal(L.store(sgn * lo, dt), sgn * lo)
        np.testing.assert_array_equal(L.store(sgn * (mid - eps), dt), sgn * lo)
        np.testing.assert_array_equal(L.store(sgn * (mid + eps), dt), sgn * up)
        even = (bits & 1) == 0                 # ties go to the even significand
        np.testing.assert_array_equal(L.store(sgn * mid, dt), sgn * np.where(even, lo, up))


# --------------------------------------------------------- rounding points
def _setup(dt, act="gelu"):
    rng = np.random.default_rng(21)
    cfg = L.Config(B=2, J=8, K=8, H=2, P=4, W=4, I=8, F=16, p_attn=0.2, p_attn_out=0.3, p_ffn_out=0.15,
                   p_ffn_act=0.25, seed=99, layer=5, act=act, eps=1e-5, store_dtype=dt)
    shapes = {"wq": (4, 2, 8), "bq": (4, 2), "wk": (4, 2, 8), "bk": (4, 2), "wv": (4, 2, 8), "bv": (4, 2),
              "wo": (4, 2, 8), "bo": (8,), "g1": (8,), "be1": (8,), "w1": (16, 8), "b1": (16,), "w2": (8, 16),
              "b2": (8,), "g2": (8,), "be2": (8,)}
    prm = {}
    for n, s in shapes.items():
        base = 1.0 if n in ("g1", "g2") else 0.0
        prm[n] = L.store(base + rng.normal(0, 0.4 if n[0] == "w" else 0.2, s), dt)
    x = L.store(rng.normal(size=(2, 8, 8)), dt)
    dy = L.store(rng.normal(size=(2, 8, 8)), dt)
    return cfg, prm, x, dy


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a))


@pytest.mark.parametrize("dt,act,dalpha_stored", [("f16", "gelu", False), ("bf16", "gelu", False),
                                                  ("f16", "relu", False), ("bf16", "gelu", True)])
def test_rounding_points(dt, act, dalpha_stored):
    cfg, prm, x, dy = _setup(dt, act)
    cfg.dalpha_stored = dalpha_stored
    y, c = L.encoder_forward(x, prm, cfg)
    dx, g, it = L.encoder_backward(dy, c, prm, cfg)
    B, J, H, P, I = cfg.B, cfg.J, cfg.H, cfg.P, cfg.I
    R = lambda t: _t(L.store(t.numpy(), dt))
    p = {n: _t(v) for n, v in prm.items()}
    fac = lambda site, pr, shape: _t(philox.dropout_factor(cfg.seed, site, cfg.layer, pr, shape))
    m_attn = fac(philox.SITE_ATTN, cfg.p_attn, (H, B, J, J)).permute(1, 0, 2, 3)       # [b,h,j,k]
    m_ao = fac(philox.SITE_ATTN_OUT, cfg.p_attn_out, (B, J, I))
    m_act = fac(philox.SITE_FFN_ACT, cfg.p_ffn_act, (B, J, cfg.F))
    m_ffn = fac(philox.SITE_FFN_OUT, cfg.p_ffn_out, (B, J, I))

    # oracle tensors in the composition's token-major / head-major orders
    head = lambda a: _t(a).permute(2, 1, 3, 0)            # [p,h,b,j] -> [b,h,j,p]
    tok = lambda a: _t(a).permute(1, 2, 0)                # [i,b,j]   -> [b,j,i]
    hbjk = lambda a: _t(a).permute(1, 0, 2, 3)            # [h,b,j,k] -> [b,h,j,k]
    X = _t(x)
    qq, kk, vv = head(c["qq"]), head(c["kk"]), head(c["vv"])
    beta, prob, alpha = hbjk(c["beta"]), hbjk(c["prob"]), hbjk(c["alpha"])
    gamma = head(c["gamma"])
    ao, y1, h, a, o = tok(c["ao"]), tok(c["y1"]), tok(c["h"]), tok(c["a"]), tok(c["o"])
    xhat1, xhat2 = tok(c["xhat1"]), tok(c["xhat2"])

    def same(name, got, want):
        assert torch.equal(got, want), (name, float((got - want).abs().max()))

    # forward: each written tensor from the written tensors before it
    for name, w, b, got in (("qq", "wq", "bq", qq), ("kk", "wk", "bk", kk), ("vv", "wv", "bv", vv)):
        same(name, got, R(torch.einsum("bji,phi->bhjp", X, p[w]) + p[b].T[None, :, None, :]))
    same("beta", beta, R(cfg.s * torch.einsum("bhjp,bhkp->bhjk", qq, kk)))
    pr = torch.softmax(beta, dim=-1)                                   # unrounded inside `sm`
    same("prob", prob, R(pr))
    same("alpha", alpha, R(R(pr) * m_attn))                            # from the rounded (stored) probabilities
    same("gamma", gamma, R(torch.einsum("bhjk,bhkw->bhjw", alpha, vv)))
    ctx = gamma.permute(0, 2, 1, 3).reshape(B, J, H * cfg.W)
    same("ao", ao, R(ctx @ p["wo"].permute(1, 0, 2).reshape(H * cfg.W, I)))
    s1 = X + (ao + p["bo"]) * m_ao                                     # inside `bdrln`
    ln1 = Fnn.layer_norm(s1, (I,), eps=cfg.eps)
    same("xhat1", xhat1, R(ln1))
    same("y1", y1, R(ln1 * p["g1"] + p["be1"]))                       # from the unrounded x_hat
    same("h", h, R(y1 @ p["w1"].T))                                    # bias not yet added
    u = h + p["b1"]                                                    # inside `brd`
    av = Fnn.gelu(u) if act == "gelu" else torch.relu(u)
    same("a", a, R(av * m_act))
    same("o", o, R(a @ p["w2"].T))
    s2 = y1 + (o + p["b2"]) * m_ffn
    ln2 = Fnn.layer_norm(s2, (I,), eps=cfg.eps)
    same("xhat2", xhat2, R(ln2))
    same("y", _t(y), R(ln2 * p["g2"] + p["be2"]))

    # backward
    dY = _t(dy)
    rstd2 = _t(c["rstd2"])[..., None]
    rstd1 = _t(c["rstd1"])[..., None]

    def ln_bwd(d, xh, rstd, gm):
        gy = d * gm
        return rstd * (gy - gy.mean(-1, keepdim=True) - xh * (gy * xh).mean(-1, keepdim=True))

    dS2x = ln_bwd(dY, xhat2, rstd2, p["g2"])                            # from the written x_hat
    dS2, dO = tok(it["dS2"]), tok(it["dO"])
    same("dS2", dS2, R(dS2x))
    same("dO", dO, R(dS2x * m_ffn))                                    # from the unrounded dS2
    dA = tok(it["dA"])
    same("dA", dA, R(dO @ p["w2"]))
    dact = torch.autograd.functional.vjp(lambda t: Fnn.gelu(t) if act == "gelu" else torch.relu(t), u,
                                         dA * m_act)[1]
    dH = tok(it["dH"])
    same("dH", dH, R(dact))
    dY1f = tok(it["dY1f"])
    same("dY1f", dY1f, R(dH @ p["w1"]))
    dY1 = dY1f + dS2                                                   # `ebsb` feeds `blnrd` unrounded
    dS1x = ln_bwd(dY1, xhat1, rstd1, p["g1"])
    dS1, dAO = tok(it["dS1"]), tok(it["dAO"])
    same("dS1", dS1, R(dS1x))
    same("dAO", dAO, R(dS1x * m_ao))
    dgamma = head(it["dgamma"])
    wo_hw = p["wo"].permute(1, 0, 2)                                   # [h,w,i]
    same("dgamma", dgamma, R(torch.einsum("bji,hwi->bhjw", dAO, wo_hw)))
    dalpha = hbjk(it["dalpha"])
    dalpha_x = torch.einsum("bhjw,bhkw->bhjk", dgamma, vv)
    if dalpha_stored:                                                  # written by Gamma dX1
        same("dalpha", dalpha, R(dalpha_x))
    else:                                                              # inside the fused score backward
        assert torch.allclose(dalpha, dalpha_x, rtol=1e-12, atol=1e-14)
    same("dvv", head(it["dvv"]), R(torch.einsum("bhjk,bhjw->bhkw", alpha, dgamma)))
    dprob = dalpha * m_attn                                            # inside `bs`
    dbeta = hbjk(it["dbeta"])
    row_dp = (dprob * prob).sum(-1, keepdim=True)                      # sum_k dP P over the stored P
    row_da = (dalpha * alpha).sum(-1, keepdim=True)                    # sum_k d(alpha) alpha, alpha as stored
    same("dbeta", dbeta, R(cfg.s * prob * (dprob - (row_dp if dalpha_stored else row_da))))
    # the two row terms are different rounding readings of one number
    assert not torch.equal(R(cfg.s * prob * (dprob - row_dp)), R(cfg.s * prob * (dprob - row_da)))
    dqq, dkk = head(it["dqq"]), head(it["dkk"])
    same("dqq", dqq, R(torch.einsum("bhjk,bhkp->bhjp", dbeta, kk)))
    same("dkk", dkk, R(torch.einsum("bhjk,bhjp->bhkp", dbeta, qq)))
    dvv = head(it["dvv"])
    dXa = (torch.einsum("bhjp,phi->bji", dqq, p["wq"]) + torch.einsum("bhjp,phi->bji", dkk, p["wk"])
           + torch.einsum("bhjw,whi->bji", dvv, p["wv"]))
    same("dx", _t(dx), R(dXa + dS1))                                   # `bei` in the Q/K/V dX epilogue

    # values kept inside one fused operator are not rounded
    kept = [("s1", s1), ("u", u), ("s2", s2), ("dY1", dY1), ("dXa", dXa), ("dprob", dprob[m_attn != 0])]
    if not dalpha_stored:
        kept.append(("dalpha", dalpha))
    for name, v in kept:
        v = v.numpy()
        frac = float(np.mean(L.store(v, dt) == v))
        assert frac < 0.5, (name, frac)
