"""Further layer parity on the GPU: the 24-layer stack's layers (every
output, at a spread of layers, and the chained stack against standalone
calls), the ReLU layer with the activation dropout (the paper's own
dataflow) in 16-bit storage, extreme attention logits, LayerNorm rows with
a large mean, and the full BERT-large layer against the plain float64
definition (no storage emulation).

A large mean in the layer's *input* is not among the cases: it makes the
attention ill-conditioned in 16-bit storage (scores of size mean^2 stored
to a few units, and a dQ that cancels through the softmax's shift
invariance), so there the comparison measures the inputs' rounding, not
the kernels; LayerNorm rows with a large mean are tested at operator level."""
import numpy as np
import pytest
import torch

from oracle import layer as OL
from oracle import philox
from paper_2007_00072_amd.inputs import WORKLOADS, Shape, make_activation, make_params, make_tensor
from _util import assert_close, encoder_dx_scale, f64, oracle_config, params64
from test_gpu_layer import GRAD_NAMES, check_encoder, check_mha, run_encoder, small

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _compare_layer(tag, y, dx, grads, ry, rdx, rg, dt, dx_scale=None):
    assert_close(f"y{tag}", y, ry, dt)
    assert_close(f"dx{tag}", dx, rdx, dt, scale=dx_scale)
    for n in GRAD_NAMES:
        if n == "bk":
            assert_close(f"dbk{tag}", grads[n], rg[n], dt, zero_ref=True,
                         zero_scale=float(np.sqrt(np.mean(rg["bq"] ** 2))))
        else:
            assert_close(f"d{n}{tag}", grads[n], rg[n], dt, param_grad=True)


STACK_CHECK = [0, 4, 8, 12, 16, 20, 23]


@pytest.mark.parametrize("li", STACK_CHECK)
def test_encoder_stack_layer_parity(li):
    # layer li of the 24-layer BERT-large stack (bf16, B=4, L=512: its own
    # weights and dropout counter word) on seeded inputs: y, dx and all 16
    # parameter gradients against the oracle
    wl = WORKLOADS["bert_large_stack24_bf16"]
    x = make_activation(wl, 10 + 2 * li)
    dy = make_activation(wl, 11 + 2 * li)
    L, params, x, dy, y, dx = run_encoder(wl, layer=li, x=x, dy=dy)
    cfg = oracle_config(wl, li, desc=L.desc)
    prm = params64(params)
    ry, cache = OL.encoder_forward(f64(x), prm, cfg)
    rdx, rg, inter = OL.encoder_backward(f64(dy), cache, prm, cfg)
    _compare_layer(f"[{li}]", y, dx, L.grads, ry, rdx, rg, wl.dtype, encoder_dx_scale(cache, inter, prm))


def test_encoder_stack_chained_equals_standalone():
    # all 24 layers forward, then backward, in sequence on the GPU with one
    # shared workspace (activations of every layer kept for its backward):
    # each checked layer's outputs equal, bit for bit, a standalone call of
    # that layer on the same input and incoming gradient
    from paper_2007_00072_amd.runner import EncoderLayer, desc_for
    wl = WORKLOADS["bert_large_stack24_bf16"]
    x = make_activation(wl, 0).to(DEV)
    layers, inputs, outputs = [], [], []
    for li in range(wl.n_layers):
        L = EncoderLayer(desc_for(wl, li), make_params(wl, layer=li), DEV,
                         workspace=layers[0].ws if layers else None)
        inputs.append(x)
        x = L.forward(x)
        outputs.append(x)
        layers.append(L)
    dy = make_activation(wl, 1).to(DEV)
    dys, dxs = [None] * wl.n_layers, [None] * wl.n_layers
    for li in reversed(range(wl.n_layers)):
        dys[li] = dy
        dy = layers[li].backward(inputs[li], dy)
        dxs[li] = dy
    torch.cuda.synchronize()
    assert torch.isfinite(x.float()).all() and torch.isfinite(dy.float()).all()
    for li in (0, 11, 23):
        S = EncoderLayer(desc_for(wl, li), make_params(wl, layer=li), DEV)
        y1 = S.forward(inputs[li])
        dx1 = S.backward(inputs[li], dys[li])
        torch.cuda.synchronize()
        assert torch.equal(y1, outputs[li]) and torch.equal(dx1, dxs[li]), li
        for n, t in S.grads.items():
            assert torch.equal(t, layers[li].grads[n]), (li, n)


# |u| below which the GPU's and the oracle's ReLU branches may differ: u =
# h + b1 with h a rounded contraction over LayerNorm outputs, which differ
# by a unit of the storage type on some elements; this moves h near zero by
# up to ~1e-4 (fp16) or ~1e-3 (bf16) in absolute terms, not by units of
# h's own (tiny) spacing there.  Ten times that.
RELU_AMBIGUOUS = {"f16": 4e-3, "bf16": 3e-2}


def check_encoder_relu(wl, layer=0, p_ffn_act=0.1):
    """The ReLU layer in 16-bit storage.  ReLU's derivative jumps at 0, so
    where u = h + b1 lies within the rounding difference of h of zero, the
    GPU and the oracle may take different branches, both correct.  Which
    ambiguous elements the GPU took the other way is read off the first
    linear layer's weight gradient (flipping element (f, t) moves row f of
    it by a known vector, dH's change times token t's LayerNorm output),
    by greedy matching per row; the oracle's backward is then rerun with
    those branches, and every output must match it at the parity bar."""
    L, params, x, dy, y, dx = run_encoder(wl, layer, act="relu", p_ffn_act=p_ffn_act)
    dt = wl.dtype
    cfg = oracle_config(wl, layer, desc=L.desc, act="relu", p_ffn_act=p_ffn_act)
    prm = params64(params)
    ry, cache = OL.encoder_forward(f64(x), prm, cfg)
    assert_close("y", y, ry, dt)
    rdx, rg, inter = OL.encoder_backward(f64(dy), cache, prm, cfg)
    u = cache["u"]                                                    # [F, B, J]
    F = u.shape[0]
    u2d = u.reshape(F, -1)                                            # [F, T]
    dA = inter["dA"].reshape(F, -1)
    m_act = cache["m_act"].reshape(F, -1)
    y1t = np.ascontiguousarray(cache["y1"].reshape(cache["y1"].shape[0], -1).T)   # [T, I]
    diff = f64(L.grads["w1"]) - rg["w1"]                              # [F, I]
    flips = []
    n_amb = 0
    for f in range(F):
        ts = np.nonzero(np.abs(u2d[f]) <= RELU_AMBIGUOUS[dt])[0]
        n_amb += len(ts)
        if not len(ts):
            continue
        full = OL.store(dA[f, ts] * m_act[f, ts], dt)
        delta = np.where(u2d[f, ts] > 0, -full, full)
        cand = delta[:, None] * y1t[ts]                               # dW1 row change per flip
        r = diff[f].copy()
        taken = np.zeros(len(ts), dtype=bool)
        norms = (cand ** 2).sum(1)
        while True:
            gain = 2 * cand @ r - norms
            gain[taken] = -np.inf
            e = int(np.argmax(gain))
            if gain[e] <= 0:
                break
            taken[e] = True
            r -= cand[e]
        flips += [(f, int(t)) for t in ts[taken]]
    if flips:
        u2 = u2d.copy()
        for f, t in flips:
            u2[f, t] = -np.sign(u2d[f, t]) * 1e-30 if u2d[f, t] != 0 else 1e-30
        c2 = dict(cache, u=u2.reshape(u.shape))
        rdx, rg, inter = OL.encoder_backward(f64(dy), c2, prm, cfg)
    assert_close(f"dx (ambiguous ReLU branches {n_amb}, taken the other way {len(flips)})", dx, rdx, dt,
                 scale=encoder_dx_scale(cache, inter, prm))
    for n in GRAD_NAMES:
        if n == "bk":
            assert_close("dbk", L.grads[n], rg[n], dt, zero_ref=True, zero_scale=float(np.sqrt(np.mean(rg["bq"] ** 2))))
        else:
            assert_close("d" + n, L.grads[n], rg[n], dt, param_grad=True)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_relu_activation_dropout_ragged(name):
    # the paper's feed-forward (ReLU, then a fourth dropout), ragged tiles
    wl = small(name, B=2, J=72, K=72, H=4, P=64, W=64, I=256, F=1024).with_(random_ln=True, bias_std=0.05)
    check_encoder_relu(wl, layer=2)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_encoder_relu_activation_dropout_bert_large(dtype):
    # full BERT-large sizes (B=8, L=512) in both 16-bit storage types
    check_encoder_relu(WORKLOADS["bert_large_f16"].with_(dtype=dtype))


def test_encoder_full_size_vs_plain_f64():
    # BERT-large fp16 against the plain float64 definition (store_dtype
    # "f64": nothing rounded inside the oracle), at the stated bar
    wl = WORKLOADS["bert_large_f16"]
    L, params, x, dy, y, dx = run_encoder(wl)
    cfg = oracle_config(wl, desc=L.desc, store_dtype="f64")
    prm = params64(params)
    ry, cache = OL.encoder_forward(f64(x), prm, cfg)
    rdx, rg, inter = OL.encoder_backward(f64(dy), cache, prm, cfg)
    _compare_layer("(f64)", y, dx, L.grads, ry, rdx, rg, "f16", encoder_dx_scale(cache, inter, prm))


# --------------------------------------------------------- extreme inputs
@pytest.fixture(scope="module")
def lib():
    from paper_2007_00072_amd import lib as L
    return L


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("K", [64, 512])
def test_softmax_extreme_logits(lib, dt, K):
    # logits of magnitude up to ~2000: rows where one key dominates (the
    # others underflow to exactly zero), rows shifted far from zero, and
    # rows of equal values
    B, H, J = 2, 2, 16
    rng = np.random.default_rng(5)
    b = rng.normal(0, 30.0, (B, H, J, K))
    b[:, :, 0:4] += rng.normal(0, 1000.0, (B, H, 4, 1))       # large per-row offsets
    b[:, :, 4:6] = 7.0                                         # all equal
    b[:, :, 6:8] *= 20.0                                       # one key wins
    beta = torch.from_numpy(OL.store(b, dt)).to({"f32": torch.float32, "f16": torch.float16,
                                                 "bf16": torch.bfloat16}[dt])
    prob = torch.empty((B, H, J, K), dtype=beta.dtype, device=DEV)
    alpha = torch.empty_like(prob)
    DT = {"f32": 0, "f16": 1, "bf16": 2}
    lib.softmax_dropout_fwd(DT[dt], B, H, J, K, 1.0, beta.to(DEV), (0.1, 0, 0, 3), prob, alpha)
    torch.cuda.synchronize()
    p = OL.softmax_k(f64(beta))
    fac = philox.dropout_factor(3, 0, 0, 0.1, (H, B, J, K)).transpose(1, 0, 2, 3)
    assert_close("prob", prob, OL.store(p, dt), dt)
    assert_close("alpha", alpha, OL.store(OL.store(p, dt) * fac, dt), dt)
    assert torch.isfinite(prob.float()).all()


def test_mha_extreme_logits_on_chip_scores_f16():
    # projection weights of std 0.5 make the scaled scores |beta| ~ 30-100,
    # through the on-chip score kernels forward and backward
    wl = WORKLOADS["mha_large_f16"].with_(shape=Shape(B=2, J=64, K=128, H=2, P=32, W=32, I=128), dtype="f16",
                                          layout="bji", p_attn=0.1, weight_std=0.5)
    check_mha(wl, self_attention=False)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_mha_extreme_logits_exact_scores(dtype):
    # bf16 keeps 8 significant bits, so a score of 64 is stored to 0.5 and
    # a one-unit difference in a projection would move a probability by
    # e^0.5: the comparison is only meaningful where both sides hold the
    # same scores.  Integer inputs and weights in eighths make every
    # projection and score an exact fp32 (and float64) sum, rounded once
    # to the storage type identically on both sides; |beta| reaches ~60.
    from paper_2007_00072_amd.runner import MultiHeadAttention, desc_for
    s = Shape(B=2, J=64, K=128, H=2, P=64, W=64, I=128)
    wl = WORKLOADS["mha_large_f16"].with_(shape=s, dtype=dtype, layout="bji", p_attn=0.1)
    tdt = {"f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    gen = torch.Generator().manual_seed(4242)
    ints = lambda shape, lo, hi, scale: (torch.randint(lo, hi + 1, shape, generator=gen).double() * scale).to(tdt)
    params = make_params(wl)
    for n in ("wq", "wk", "wv"):
        params[n] = ints(tuple(params[n].shape), -2, 2, 0.125)
    for n in ("bq", "bk", "bv"):
        params[n] = torch.zeros_like(params[n])
    q = ints((s.B, s.J, s.I), -3, 3, 1.0)
    k = ints((s.B, s.K, s.I), -3, 3, 1.0)
    v = ints((s.B, s.K, s.I), -3, 3, 1.0)
    dout = make_activation(wl, 1)
    M = MultiHeadAttention(desc_for(wl, self_attention=False), params, DEV)
    out = M.forward(q.to(DEV), k.to(DEV), v.to(DEV))
    dq, dk, dv = M.backward(q.to(DEV), dout.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    cfg = oracle_config(wl, desc=M.desc)
    prm = params64(params)
    t = lambda a: f64(a).transpose(2, 0, 1)
    back = lambda a: a.transpose(1, 2, 0)
    rout, cache = OL.mha_forward_ibj(t(q), t(k), t(v), prm, cfg)
    assert np.abs(cache["beta"]).max() > 40
    rdq, rdk, rdv, rg, _ = OL.mha_backward_ibj(t(dout), cache, prm, cfg)
    assert_close("out", out, back(rout), dtype)
    assert_close("dq", dq, back(OL.store(rdq, dtype)), dtype)
    assert_close("dk", dk, back(OL.store(rdk, dtype)), dtype)
    assert_close("dv", dv, back(OL.store(rdv, dtype)), dtype)
    for n in ("wq", "bq", "wk", "wv", "bv", "wo", "bo"):
        assert_close("d" + n, M.grads[n], rg[n], dtype, param_grad=True)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("rows,cols", [(37, 768), (70, 1024)])
def test_bdrln_large_mean_rows(lib, dt, rows, cols):
    # residual rows with mean 1000 and unit spread: the variance must not
    # cancel (fp16 spacing at 1000 is 0.5, bf16 4; both sides see the same
    # rounded inputs)
    DT = {"f32": 0, "f16": 1, "bf16": 2}
    x = make_tensor((rows, cols), dt, 1)
    bias = make_tensor((cols,), dt, 2, 0.1)
    r = make_tensor((rows, cols), dt, 3, 8.0 if dt == "bf16" else 2.0, 1000.0)
    g = make_tensor((cols,), dt, 4, 0.1, 1.0)
    be = make_tensor((cols,), dt, 5, 0.1)
    y = torch.empty((rows, cols), dtype=x.dtype, device=DEV)
    xh = torch.empty_like(y)
    rs = torch.empty(rows, dtype=torch.float32, device=DEV)
    lib.bdrln_fwd(DT[dt], rows, cols, x.to(DEV), bias.to(DEV), r.to(DEV), g.to(DEV), be.to(DEV), 1e-12,
                  (0.1, 1, 0, 9), y, xh, rs)
    torch.cuda.synchronize()
    fac = philox.dropout_factor(9, 1, 0, 0.1, (rows, cols))
    s = f64(r) + (f64(x) + f64(bias)) * fac
    xhat, rstd = OL.layernorm_i(s.T, 1e-12)
    assert_close("y", y, OL.store(f64(g)[:, None] * xhat + f64(be)[:, None], dt).T, dt)
    assert_close("xhat", xh, OL.store(xhat, dt).T, dt)
    assert_close("rstd", rs, rstd, "f32" if dt == "f32" else dt)
