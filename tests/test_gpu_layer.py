"""Layer-level parity on the GPU: encoder_layer_fwd/bwd and mha_fwd/bwd
against the oracle (storage-rounding emulation) on the same seeded inputs,
from the tiny fp32 layer through reduced shapes with ragged tiles up to the
full BERT-large / BERT-base / attention-only workloads."""
import numpy as np
import pytest
import torch

from oracle import layer as OL
from paper_2007_00072_amd.inputs import WORKLOADS, Shape, make_activation, make_params
from _util import assert_close, encoder_dx_scale, f64, oracle_config, params64

pytestmark = pytest.mark.gpu
DEV = "cuda"

ACT_KEYS = ("y",)
GRAD_NAMES = ("wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo", "g1", "be1", "w1", "b1", "w2", "b2", "g2", "be2")


def run_encoder(wl, layer=0, x=None, dy=None, **desc_over):
    from paper_2007_00072_amd.runner import EncoderLayer, desc_for
    params = make_params(wl, layer=layer)
    x = make_activation(wl, 0) if x is None else x
    dy = make_activation(wl, 1) if dy is None else dy
    L = EncoderLayer(desc_for(wl, layer, **desc_over), params, DEV)
    xd, dyd = x.to(DEV), dy.to(DEV)
    y = L.forward(xd)
    dx = L.backward(xd, dyd)
    torch.cuda.synchronize()
    return L, params, x, dy, y, dx


def check_encoder(wl, layer=0, x=None, dy=None, act="gelu", p_ffn_act=0.0, causal=False, **desc_over):
    L, params, x, dy, y, dx = run_encoder(wl, layer, x, dy, act=act, p_ffn_act=p_ffn_act, causal=causal,
                                          **desc_over)
    cfg = oracle_config(wl, layer, desc=L.desc, act=act, p_ffn_act=p_ffn_act, causal=causal)
    prm = params64(params)
    ry, cache = OL.encoder_forward(f64(x), prm, cfg)
    rdx, rg, inter = OL.encoder_backward(f64(dy), cache, prm, cfg)
    dt = wl.dtype
    assert_close("y", y, ry, dt)
    assert_close("dx", dx, rdx, dt, scale=encoder_dx_scale(cache, inter, prm))
    for n in GRAD_NAMES:
        if n == "bk":   # exactly zero: softmax is invariant to a per-row shift
            assert_close("dbk", L.grads[n], rg[n], dt, zero_ref=True, zero_scale=float(np.sqrt(np.mean(rg["bq"] ** 2))))
        else:
            assert_close("d" + n, L.grads[n], rg[n], dt, param_grad=True)
    return L, cache


def small(wl_name, **shape):
    wl = WORKLOADS[wl_name]
    return wl.with_(shape=Shape(**shape), name=wl_name + "_small")


def test_encoder_tiny_f32():
    check_encoder(WORKLOADS["tiny_f32"])


def test_encoder_tiny_f32_random_biases_and_ln():
    wl = WORKLOADS["tiny_f32"].with_(bias_std=0.1, random_ln=True, seed=12345, p_attn=0.3)
    check_encoder(wl, layer=3)


def test_encoder_tiny_f32_relu_with_activation_dropout():
    check_encoder(WORKLOADS["tiny_f32"].with_(bias_std=0.05), act="relu", p_ffn_act=0.2)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_reduced_ragged(name):
    # several tiles in every contraction plus ragged tile tails (T = 2*72)
    wl = small(name, B=2, J=72, K=72, H=4, P=64, W=64, I=256, F=1024).with_(random_ln=True)
    check_encoder(wl, layer=1)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_transposed_grad_ragged_tile(name):
    # 40 tokens: the LayerNorm-2 backward's transposed dO copy (read by the
    # Linear-2 weight gradient) ends with a partial 8-row tile
    check_encoder(small(name, B=1, J=40, K=40, H=6, P=64, W=64, I=384, F=768))


@pytest.mark.parametrize("name,shape", [
    ("bert_large_f16", dict(B=2, J=64, K=64, H=2, P=64, W=64, I=128, F=512)),
    ("bert_base_bf16", dict(B=2, J=64, K=64, H=2, P=64, W=64, I=128, F=512)),
    # 2 * B*H*J*P = 384 bytes per projection: not a multiple of 256
    ("bert_large_f16", dict(B=1, J=8, K=8, H=3, P=8, W=8, I=24, F=32)),
])
def test_encoder_saved_tensors(name, shape):
    wl = small(name, **shape)
    L, params, x, dy, y, dx = run_encoder(wl)
    cfg = oracle_config(wl)
    _, c = OL.encoder_forward(f64(x), params64(params), cfg)
    s = wl.shape
    tdt = {"f16": torch.float16, "bf16": torch.bfloat16}[wl.dtype]
    qkv = L.saved_tensor("qkv", (3, s.B, s.H, s.J, s.P), tdt)
    for i, key in enumerate(("qq", "kk", "vv")):
        assert_close(key, qkv[i], c[key].transpose(2, 1, 3, 0), wl.dtype)   # [p,h,b,j] -> [b,h,j,p]
    prob = L.saved_tensor("prob", (s.B, s.H, s.J, s.K), tdt)
    assert_close("prob", prob, c["prob"].transpose(1, 0, 2, 3), wl.dtype)
    y1 = L.saved_tensor("y1", (s.B, s.J, s.I), tdt)
    assert_close("y1", y1, c["y1"].transpose(1, 2, 0), wl.dtype)
    from paper_2007_00072_amd import lib
    with pytest.raises(lib.DmError):
        L.saved_tensor("alpha", (s.B, s.H, s.J, s.K), tdt)   # re-formed from P where needed, never saved


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_attention_masks_bit_exact(name):
    # alpha is not saved, but with one-hot token inputs and the identity as
    # value weights (V = I, no bias) the saved context gamma = alpha V is
    # alpha itself: the forward's dropout keep decisions show element by
    # element and must match the oracle's bit for bit
    from paper_2007_00072_amd.runner import EncoderLayer, desc_for
    wl = small(name, B=2, J=64, K=64, H=1, P=64, W=64, I=64, F=128).with_(p_attn=0.3)
    params = make_params(wl)
    tdt = params["wq"].dtype
    params["wv"] = torch.eye(64, dtype=tdt).reshape(64, 1, 64)
    params["bv"] = torch.zeros(64, 1, dtype=tdt)
    x = torch.eye(64, dtype=tdt).expand(2, 64, 64).contiguous()
    L = EncoderLayer(desc_for(wl, 0), params, DEV)
    L.forward(x.to(DEV))
    torch.cuda.synchronize()
    got = f64(L.saved_tensor("gamma", (2, 64, 1, 64), tdt))[:, :, 0, :]   # [B][J][H][W] -> [B][J][K]
    _, c = OL.encoder_forward(f64(x), params64(params), oracle_config(wl))
    ref = c["alpha"][0]                                                  # [H][B][J][K], H = 1
    assert (ref == 0).any() and (ref != 0).any()
    np.testing.assert_array_equal(got == 0, ref == 0)
    assert_close("alpha", got, ref, wl.dtype)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_full_size(name):
    check_encoder(WORKLOADS[name])


def test_encoder_deterministic():
    wl = small("bert_large_f16", B=2, J=64, K=64, H=4, P=64, W=64, I=256, F=1024)
    L1, _, _, _, y1, dx1 = run_encoder(wl)
    g1 = {n: t.clone() for n, t in L1.grads.items()}
    L2, _, _, _, y2, dx2 = run_encoder(wl)
    assert torch.equal(y1, y2) and torch.equal(dx1, dx2)
    for n in g1:
        assert torch.equal(g1[n], L2.grads[n]), n


# ----------------------------------------------------------- attention only
def check_mha(wl, self_attention=True, causal=False, **desc_over):
    from paper_2007_00072_amd.runner import MultiHeadAttention, desc_for
    s = wl.shape
    params = make_params(wl)
    q = make_activation(wl, 0)
    dout = make_activation(wl, 1)
    if self_attention is True:
        k = v = None
        kh = vh = q
    elif self_attention == 2:
        # encoder/decoder attention: keys and values from one memory tensor
        kh = vh = make_activation(wl, 2, length=s.K)
        k, v = kh.to(DEV), None
    else:
        kh = make_activation(wl, 2, length=s.K)
        vh = make_activation(wl, 3, length=s.K)
        k, v = kh.to(DEV), vh.to(DEV)
    M = MultiHeadAttention(desc_for(wl, self_attention=self_attention, causal=causal, **desc_over), params, DEV)
    qd = q.to(DEV)
    out = M.forward(qd, k, v)
    dq, dk, dv = M.backward(qd, dout.to(DEV), k, v)
    torch.cuda.synchronize()
    cfg = oracle_config(wl, desc=M.desc, causal=causal)
    prm = params64(params)
    to_ibj = (lambda a: a) if wl.layout == "ibj" else (lambda a: a.transpose(2, 0, 1))
    from_ibj = (lambda a: a) if wl.layout == "ibj" else (lambda a: a.transpose(1, 2, 0))
    rout, cache = OL.mha_forward_ibj(to_ibj(f64(q)), to_ibj(f64(kh)), to_ibj(f64(vh)), prm, cfg)
    rdq, rdk, rdv, rg, _ = OL.mha_backward_ibj(to_ibj(f64(dout)), cache, prm, cfg)
    dt = wl.dtype
    assert_close("out", out, from_ibj(rout), dt)
    if self_attention is True:
        assert_close("dx", dq, from_ibj(OL.store(rdq + rdk + rdv, dt)), dt)
    elif self_attention == 2:
        assert dv is None
        assert_close("dq", dq, from_ibj(OL.store(rdq, dt)), dt)
        assert_close("dmem", dk, from_ibj(OL.store(rdk + rdv, dt)), dt)
    else:
        assert_close("dq", dq, from_ibj(OL.store(rdq, dt)), dt)
        assert_close("dk", dk, from_ibj(OL.store(rdk, dt)), dt)
        assert_close("dv", dv, from_ibj(OL.store(rdv, dt)), dt)
    for n in ("wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo"):
        if n == "bk":
            assert_close("dbk", M.grads[n], rg[n], dt, zero_ref=True, zero_scale=float(np.sqrt(np.mean(rg["bq"] ** 2))))
        else:
            assert_close("d" + n, M.grads[n], rg[n], dt, param_grad=True)


@pytest.mark.parametrize("dtype,layout", [("f16", "bji"), ("bf16", "ibj"), ("f32", "bji")])
def test_mha_fused_kv_cross_attention(dtype, layout):
    # encoder/decoder attention with [Wk Wv] stacked over one memory tensor:
    # query length 72 against memory length 128 (scores kept on chip) and
    # the tiny fp32 case through the separate launches
    shape = Shape(B=2, J=72, K=128, H=4, P=32, W=32, I=128) if dtype != "f32" else \
        Shape(B=2, J=24, K=40, H=2, P=16, W=16, I=32)
    wl = WORKLOADS["mha_large_f16"].with_(shape=shape, dtype=dtype, layout=layout, p_attn=0.1)
    check_mha(wl, self_attention=2)


def test_mha_fused_kv_full_size():
    # BERT-large widths, 512 queries against a 384-token memory
    wl = WORKLOADS["mha_large_f16"]
    wl = wl.with_(shape=Shape(B=4, J=512, K=384, H=16, P=64, W=64, I=1024), layout="bji")
    check_mha(wl, self_attention=2)


def test_mha_full_size_ibj():
    check_mha(WORKLOADS["mha_large_f16"])


@pytest.mark.parametrize("layout", ["ibj", "bji"])
@pytest.mark.parametrize("self_attention", [True, False])
def test_mha_reduced(layout, self_attention):
    wl = WORKLOADS["mha_large_f16"]
    K = 64 if self_attention else 136
    wl = wl.with_(shape=Shape(B=2, J=64, K=K, H=4, P=32, W=32 if self_attention else 48, I=192),
                  layout=layout, p_attn=0.15)
    check_mha(wl, self_attention)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_mha_fused_scores_ragged_rows(dtype):
    # attention scores kept on chip (key length a multiple of 32): query
    # rows not a multiple of the kernels' 32-row blocks, contraction lengths
    # 48 (Q K^T) and 64 (dGamma V^T)
    wl = WORKLOADS["mha_large_f16"].with_(shape=Shape(B=2, J=72, K=96, H=3, P=48, W=64, I=144), dtype=dtype,
                                          layout="bji", p_attn=0.2)
    check_mha(wl, self_attention=False)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("shape", [
    # Gamma and dQ 64 wide: 34 k16 steps over 4 waves per column block, so
    # the key-side rows arrive in two register groups; ragged query rows
    dict(B=1, J=72, K=544, H=2, P=64, W=64, I=96),
    # Gamma 128 wide (4 column blocks, 2 waves each, two register groups),
    # dQ 64 wide after a 128-long Gamma dX1 contraction
    dict(B=2, J=40, K=320, H=2, P=64, W=128, I=160),
    # a single pair of k16 steps: most waves idle; one partial query block
    dict(B=1, J=24, K=32, H=3, P=128, W=32, I=96),
])
def test_mha_fused_next_contraction(dtype, shape):
    # Gamma = alpha V in the attention-score launch and dQ = dbeta K in the
    # score-backward launch, from the rounded row tile in LDS
    wl = WORKLOADS["mha_large_f16"].with_(shape=Shape(**shape), dtype=dtype, layout="bji", p_attn=0.1)
    check_mha(wl, self_attention=False)


@pytest.mark.parametrize("name,J", [("bert_large_f16", 96), ("bert_base_bf16", 96), ("bert_large_f16", 72)])
def test_encoder_causal(name, J):
    # decoder-style self-attention: J = 96 through the on-chip score kernels
    # (a partial last row block), J = 72 through the two-launch softmax
    wl = small(name, B=2, J=J, K=J, H=4, P=64, W=64, I=256, F=512).with_(p_attn=0.1)
    check_encoder(wl, layer=1, causal=True)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_head_size_32(name):
    # P = 32: the Q/K/V dX contraction with the encoder-input residual cannot
    # take the lean 128x128 kernel (its k-steps cross the weight map's lowest
    # radix) and falls back to the 128x64 tile, which must cover all of N
    wl = small(name, B=2, J=64, K=64, H=6, P=32, W=32, I=192, F=384)
    check_encoder(wl, layer=1)


@pytest.mark.parametrize("fusion", [1, 2])
@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_qkv_fusion_variants(name, fusion):
    # Q and K stacked + V, or three separate projections (Sec. "Algebraic
    # Fusion"); the backward accumulates dX over the groups in place
    wl = small(name, B=2, J=72, K=72, H=4, P=64, W=64, I=256, F=512).with_(p_attn=0.1)
    check_encoder(wl, layer=3, qkv_fusion=fusion)


@pytest.mark.parametrize("fusion", [1, 2])
@pytest.mark.parametrize("layout", ["ibj", "bji"])
def test_mha_qkv_fusion_variants(layout, fusion):
    wl = WORKLOADS["mha_large_f16"].with_(shape=Shape(B=2, J=64, K=64, H=4, P=32, W=32, I=192), layout=layout,
                                          p_attn=0.15)
    check_mha(wl, self_attention=True, qkv_fusion=fusion)


def test_encoder_causal_tiny_f32():
    check_encoder(WORKLOADS["tiny_f32"].with_(p_attn=0.2), causal=True)


@pytest.mark.parametrize("layout", ["ibj", "bji"])
def test_mha_causal(layout):
    wl = WORKLOADS["mha_large_f16"].with_(shape=Shape(B=2, J=128, K=128, H=2, P=64, W=64, I=128), layout=layout,
                                          p_attn=0.1)
    check_mha(wl, self_attention=True, causal=True)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_fused_scores(name):
    # several 32-row blocks per head through the on-chip score kernels
    wl = small(name, B=2, J=96, K=96, H=4, P=64, W=64, I=256, F=512)
    check_encoder(wl, layer=2)


def test_mha_tiny_f32_general():
    wl = WORKLOADS["mha_large_f16"].with_(shape=Shape(B=2, J=16, K=24, H=2, P=8, W=16, I=24), dtype="f32")
    check_mha(wl, self_attention=False)
