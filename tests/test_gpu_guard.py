"""Out-of-bounds writes: every entry point writes its outputs (and its saved
and workspace buffers) into views carved out of larger buffers filled with a
canary byte, at ragged shapes; the canary bands before and after each view
must come back unchanged."""
import numpy as np
import pytest
import torch

from paper_2007_00072_amd.inputs import WORKLOADS, Shape, make_activation, make_params, make_tensor

pytestmark = pytest.mark.gpu
DEV = "cuda"
CANARY = 0xA5
BAND = 4096          # bytes of canary on each side (a multiple of 16: views stay aligned)
TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
DT = {"f32": 0, "f16": 1, "bf16": 2}


class Guard:
    """Hands out canary-banded views and checks the bands afterwards."""

    def __init__(self):
        self.bufs = []

    def bytes(self, n):
        buf = torch.full((n + 2 * BAND,), CANARY, dtype=torch.uint8, device=DEV)
        self.bufs.append((buf, n))
        return buf[BAND:BAND + n]

    def tensor(self, shape, dtype):
        n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        return self.bytes(n).view(dtype).view(*shape)

    def like(self, t):
        return self.tensor(tuple(t.shape), t.dtype)

    def check(self):
        torch.cuda.synchronize()
        for i, (buf, n) in enumerate(self.bufs):
            head = buf[:BAND]
            tail = buf[BAND + n:]
            assert bool((head == CANARY).all()) and bool((tail == CANARY).all()), f"buffer {i} ({n} bytes) overwritten"


@pytest.fixture(scope="module")
def lib():
    from paper_2007_00072_amd import lib as L
    return L


@pytest.mark.parametrize("name,shape", [
    ("bert_large_f16", dict(B=1, J=40, K=40, H=6, P=64, W=64, I=384, F=768)),
    ("bert_base_bf16", dict(B=2, J=72, K=72, H=4, P=64, W=64, I=256, F=1024)),
    ("tiny_f32", dict(B=2, J=24, K=24, H=2, P=16, W=16, I=32, F=64)),
])
def test_encoder_layer_writes_stay_inside(lib, name, shape):
    wl = WORKLOADS[name].with_(shape=Shape(**shape))
    from paper_2007_00072_amd.runner import desc_for
    d = desc_for(wl, 0)
    g = Guard()
    params = {n: t.to(DEV) for n, t in make_params(wl).items()}
    cp = lib.make_params(params)
    saved_b, fwd_b, bwd_b = lib.encoder_layer_sizes(d)
    saved = g.bytes(saved_b)
    ws = g.bytes(max(fwd_b, bwd_b))
    x = make_activation(wl, 0).to(DEV)
    dy = make_activation(wl, 1).to(DEV)
    y = g.like(x)
    dx = g.like(x)
    grads = {n: g.tensor(tuple(t.shape), torch.float32) for n, t in params.items()}
    lib.encoder_layer_fwd(d, cp, x, y, saved, ws, max(fwd_b, bwd_b))
    lib.encoder_layer_bwd(d, cp, x, saved, dy, dx, lib.make_grads(grads), ws, max(fwd_b, bwd_b))
    g.check()
    assert torch.isfinite(y.float()).all() and torch.isfinite(dx.float()).all()


@pytest.mark.parametrize("self_attention,layout,dtype", [(True, "ibj", "f16"), (False, "bji", "bf16"),
                                                         (2, "bji", "f16")])
def test_mha_writes_stay_inside(lib, self_attention, layout, dtype):
    s = Shape(B=2, J=72, K=72 if self_attention is True else 96, H=3, P=48 if self_attention is not True else 32,
              W=48 if self_attention is not True else 32, I=144 if self_attention is not True else 96)
    wl = WORKLOADS["mha_large_f16"].with_(shape=s, dtype=dtype, layout=layout)
    from paper_2007_00072_amd.runner import desc_for
    d = desc_for(wl, self_attention=self_attention)
    g = Guard()
    params = {n: t.to(DEV) for n, t in make_params(wl).items()}
    cp = lib.make_params(params)
    saved_b, fwd_b, bwd_b = lib.mha_sizes(d)
    saved = g.bytes(saved_b)
    ws = g.bytes(max(fwd_b, bwd_b))
    q = make_activation(wl, 0).to(DEV)
    k = v = None
    if self_attention is not True:
        k = make_activation(wl, 2, length=s.K).to(DEV)
        v = None if self_attention == 2 else make_activation(wl, 3, length=s.K).to(DEV)
    dout = make_activation(wl, 1).to(DEV)
    out = g.like(q)
    lib.mha_fwd(d, cp, q, k, v, out, saved, ws, max(fwd_b, bwd_b))
    dq = g.like(q)
    dk = g.like(k) if self_attention is not True else None
    dv = g.like(v) if self_attention is False else None
    grads = {n: g.tensor(tuple(t.shape), torch.float32) for n, t in params.items()}
    lib.mha_bwd(d, cp, q, k, v, saved, dout, dq, dk, dv, lib.make_grads(grads), ws, max(fwd_b, bwd_b))
    g.check()


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_fused_operators_write_stay_inside(lib, dt):
    g = Guard()
    rows, cols = 37, 200
    t = TDT[dt]
    d = lambda *a: make_tensor(*a).to(DEV)
    x, b, r = d((rows, cols), dt, 1), d((cols,), dt, 2, 0.1), d((rows, cols), dt, 3)
    gm, be = d((cols,), dt, 4, 0.1, 1.0), d((cols,), dt, 5, 0.1)
    y, xh, rs = g.tensor((rows, cols), t), g.tensor((rows, cols), t), g.tensor((rows,), torch.float32)
    lib.bdrln_fwd(DT[dt], rows, cols, x, b, r, gm, be, 1e-5, (0.1, 1, 0, 3), y, xh, rs)
    ya = g.tensor((rows, cols), t)
    lib.bias_act_fwd(DT[dt], rows, cols, x, b, 0, (0.2, 3, 0, 3), ya)
    B, H, J, K = 2, 3, 5, 136
    beta = d((B, H, J, K), dt, 6)
    prob, alpha = g.tensor((B, H, J, K), t), g.tensor((B, H, J, K), t)
    lib.softmax_dropout_fwd(DT[dt], B, H, J, K, 0.5, beta, (0.1, 0, 0, 3), prob, alpha)
    dbeta = g.tensor((B, H, J, K), t)
    lib.softmax_dropout_bwd(DT[dt], B, H, J, K, 0.5, beta, prob, (0.1, 0, 0, 3), dbeta)
    Hh, P = 3, 16
    xq = d((rows, 3, Hh, P), dt, 7)
    bqkv = [d((P, Hh), dt, 8 + i) for i in range(3)]
    yq = g.tensor((rows, 3, Hh, P), t)
    lib.attn_input_bias(DT[dt], rows, Hh, P, xq, *bqkv, yq)
    wsb = lib.colsum_ws_bytes(rows, max(cols, 3 * Hh * P))
    ws = g.bytes(wsb)
    dg, db = g.tensor((cols,), torch.float32), g.tensor((cols,), torch.float32)
    lib.ln_param_bwd(DT[dt], rows, cols, x, xh, dg, db, ws, wsb)
    ds, dsub = g.tensor((rows, cols), t), g.tensor((rows, cols), t)
    lib.ln_dropout_bwd(DT[dt], rows, cols, x, xh, gm, rs, (0.1, 2, 0, 3), ds, dsub)
    dsum = g.tensor((rows, cols), t)
    dg2, db2 = g.tensor((cols,), torch.float32), g.tensor((cols,), torch.float32)
    lib.residual_ln_param_bwd(DT[dt], rows, cols, x, r, xh, dsum, dg2, db2, ws, wsb)
    F, I = 200, 40
    dout = d((rows, I), dt, 12)
    wsa = lib.colsum_ws_bytes(rows, F)
    ws2 = g.bytes(wsa)
    dh, db1, dbo = g.tensor((rows, F), t), g.tensor((F,), torch.float32), g.tensor((I,), torch.float32)
    lib.act_bias_bwd(DT[dt], rows, F, I, x, r, b, 0, (0.1, 3, 0, 3), dout, dh, db1, dbo, ws2, wsa)
    dbb = g.tensor((cols,), torch.float32)
    lib.bias_grad(DT[dt], rows, cols, x, dbb, ws, wsb)
    dq, dk, dv = (g.tensor((P, Hh), torch.float32) for _ in range(3))
    lib.attn_input_bias_grad(DT[dt], rows, Hh, P, xq, dq, dk, dv, ws, wsb)
    o = g.tensor((rows, cols), t)
    lib.residual_add(DT[dt], rows * cols, x, r, o)
    m = g.tensor((1000,), torch.uint8)
    lib.dropout_mask(5, 0, 1, 0.3, 8, 1000, m)
    g.check()


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("cfg,splits", [(-1, 0), (13, 1), (15, 2), (16, 1), (8, 3), (11, 1), (17, 1), (18, 2), (19, 1), (20, 1), (21, 2), (22, 3), (23, 1), (24, 2), (25, 1)])
@pytest.mark.parametrize("bt", [0, 1])
def test_contract_writes_stay_inside(lib, dt, cfg, splits, bt):
    g = Guard()
    batch, M, N, K = 2, 264, 392, 256
    A = make_tensor((batch, M, K), dt, 1).to(DEV)
    Bm = make_tensor((batch, N, K) if bt else (batch, K, N), dt, 2).to(DEV)
    C = g.tensor((batch, M, N), TDT[dt])
    wsb = max(1, splits) * batch * M * N * 4
    ws = g.bytes(wsb) if splits > 1 else None
    lib.contract(DT[dt], batch, M, N, K, 1.0, A, 0, M * K, Bm, bt, N * K, None, C, 0, M * N, cfg, splits, ws,
                 wsb if splits > 1 else 0)
    g.check()
