"""Pins for the oracle's causal (decoder) self-attention, none of which reuse
its masking code.

* Each softmax row j equals the plain softmax of that row's first j + 1
  scores, by brute force, with exact zeros after it.
* Causality: changing the input tokens after position t leaves every output
  at positions <= t unchanged (the whole encoder layer: attention, the
  residual streams, LayerNorms and the feed-forward block are per token
  except the attention, which may only look back).
* Every gradient of the causal layer equals central finite differences on a
  tiny shape with all dropout sites active; the softmax input gradient is
  exactly zero where the mask removed the score.
"""
import math

import numpy as np
import pytest

from oracle import layer as L
from test_oracle_layer import _fd_check, rand_params


def test_causal_softmax_rows_brute_force():
    rng = np.random.default_rng(3)
    beta = rng.normal(0, 2.0, (2, 3, 7, 7))
    got = L.softmax_k(beta, causal=True)
    for idx in np.ndindex(2, 3):
        for j in range(7):
            row = beta[idx + (j,)][: j + 1]
            e = [math.exp(v - max(row)) for v in row]
            want = [v / sum(e) for v in e] + [0.0] * (6 - j)
            np.testing.assert_allclose(got[idx + (j,)], want, rtol=1e-13, atol=0)
    assert np.all(got[..., 0, 1:] == 0.0) and np.allclose(got[..., 0, 0], 1.0)
    with pytest.raises(ValueError):
        L.softmax_k(rng.normal(size=(2, 3, 4)), causal=True)


@pytest.mark.parametrize("t", [0, 5, 10])
def test_causal_layer_does_not_look_ahead(t):
    rng = np.random.default_rng(11)
    cfg = L.Config(B=2, J=12, K=12, H=2, P=4, W=4, I=8, F=16, p_attn=0.2, p_attn_out=0.1,
                   p_ffn_out=0.1, seed=5, causal=True, eps=1e-5)
    prm = rand_params(rng, cfg)
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    y, _ = L.encoder_forward(x, prm, cfg)
    x2 = x.copy()
    x2[:, t + 1:, :] += rng.normal(0, 3.0, x2[:, t + 1:, :].shape)
    y2, _ = L.encoder_forward(x2, prm, cfg)
    np.testing.assert_allclose(y2[:, : t + 1], y[:, : t + 1], rtol=1e-12, atol=1e-12)
    if t + 1 < cfg.J:
        assert np.abs(y2[:, t + 1:] - y[:, t + 1:]).max() > 1e-3
    # without the mask the early positions do see the change
    ync, _ = L.encoder_forward(x, prm, L.Config(**{**cfg.__dict__, "causal": False}))
    ync2, _ = L.encoder_forward(x2, prm, L.Config(**{**cfg.__dict__, "causal": False}))
    if t + 1 < cfg.J:
        assert np.abs(ync2[:, : t + 1] - ync[:, : t + 1]).max() > 1e-6


def test_causal_finite_differences_tiny():
    rng = np.random.default_rng(6)
    cfg = L.Config(B=1, J=5, K=5, H=2, P=2, W=2, I=4, F=8, p_attn=0.3, p_attn_out=0.3,
                   p_ffn_out=0.3, p_ffn_act=0.3, seed=9, eps=1e-5, causal=True)
    prm = rand_params(rng, cfg)
    x = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    dy = rng.normal(size=(cfg.B, cfg.J, cfg.I))
    _, cache = L.encoder_forward(x, prm, cfg)
    dx, grads, inter = L.encoder_backward(dy, cache, prm, cfg)
    masked = np.arange(cfg.K)[None, :] > np.arange(cfg.J)[:, None]
    assert np.all(inter["dbeta"][..., masked] == 0.0)
    loss = lambda: float((L.encoder_forward(x, prm, cfg)[0] * dy).sum())
    _fd_check(loss, dict(prm, x=x), dict(grads, x=dx))
