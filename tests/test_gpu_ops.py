"""Operator-level parity on the GPU: every fused-operator entry point, the
dropout-mask hook and the contraction kernel against the oracle's
definitions on the same seeded inputs (small sizes with ragged tails)."""
import numpy as np
import pytest
import torch

from oracle import layer as OL
from oracle import philox
from paper_2007_00072_amd.inputs import make_tensor
from _util import assert_close, f64

pytestmark = pytest.mark.gpu

DEV = "cuda"
DT = {"f32": 0, "f16": 1, "bf16": 2}


@pytest.fixture(scope="module")
def lib():
    from paper_2007_00072_amd import lib as L
    return L


def dev(t):
    return t.to(DEV)


def rnd(x, dt):
    return OL.store(x, dt)


# ------------------------------------------------------------------ dropout
@pytest.mark.parametrize("site,layer,p,seed,offset", [
    (0, 0, 0.1, 0, 0), (1, 3, 0.1, 0, 8), (2, 23, 0.5, 2**40 + 17, 4096),
    (3, 0, 0.3, 123456789, 2**33), (0, 7, 0.9, 5, 2**36 + 64)])
def test_dropout_mask_bit_exact(lib, site, layer, p, seed, offset):
    n = 1 << 16
    out = torch.empty(n, dtype=torch.uint8, device=DEV)
    lib.dropout_mask(seed, site, layer, p, offset, n, out)
    got = out.cpu().numpy().astype(bool)
    ref = philox.keep_mask(seed, site, layer, p, n, offset=offset)
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("p", [1e-20, 2.0 ** -33, 2.0 ** -24])
def test_dropout_mask_tiny_p(lib, p):
    # 1e-20: 1 - p rounds to 1 in double, so the threshold is 2^32 and every
    # element is kept; 2^-33: threshold 2^32 - 1, only the all-ones word drops
    n = 1 << 16
    out = torch.empty(n, dtype=torch.uint8, device=DEV)
    lib.dropout_mask(3, 1, 2, p, 0, n, out)
    np.testing.assert_array_equal(out.cpu().numpy().astype(bool), philox.keep_mask(3, 1, 2, p, n))
    if p == 1e-20:
        x = make_tensor((16, 64), "f16", 7)
        ys = []
        for pp in (0.0, p):
            y = torch.empty((16, 64), dtype=x.dtype, device=DEV)
            lib.bias_act_fwd(DT["f16"], 16, 64, dev(x), dev(make_tensor((64,), "f16", 8)), 1, (pp, 3, 0, 5), y)
            ys.append(y)
        torch.cuda.synchronize()
        assert torch.equal(ys[0], ys[1])


def test_dropout_mask_p0_all_ones(lib):
    out = torch.zeros(1024, dtype=torch.uint8, device=DEV)
    lib.dropout_mask(1, 0, 0, 0.0, 0, 1024, out)
    assert bool((out == 1).all())


# ------------------------------------------------------------ bdrln forward
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("rows,cols", [(37, 32), (21, 96), (9, 768), (70, 1024), (5, 2048)])
def test_bdrln_fwd(lib, dt, rows, cols):
    x = make_tensor((rows, cols), dt, 1)
    b = make_tensor((cols,), dt, 2, 0.1)
    r = make_tensor((rows, cols), dt, 3)
    g = make_tensor((cols,), dt, 4, 0.1, 1.0)
    be = make_tensor((cols,), dt, 5, 0.1)
    y = torch.empty((rows, cols), dtype=x.dtype, device=DEV)
    xh = torch.empty_like(y)
    rs = torch.empty(rows, dtype=torch.float32, device=DEV)
    drop = (0.1, 1, 2, 77)
    lib.bdrln_fwd(DT[dt], rows, cols, dev(x), dev(b), dev(r), dev(g), dev(be), 1e-5, drop, y, xh, rs)
    torch.cuda.synchronize()
    fac = philox.dropout_factor(77, 1, 2, 0.1, (rows, cols))
    s = f64(r) + (f64(x) + f64(b)) * fac
    xhat, rstd = OL.layernorm_i(s.T, 1e-5)
    ref_y = rnd(f64(g)[:, None] * xhat + f64(be)[:, None], dt).T
    assert_close("y", y, ref_y, dt)
    assert_close("xhat", xh, rnd(xhat, dt).T, dt)
    assert_close("rstd", rs, rstd, "f32" if dt == "f32" else dt)


# ----------------------------------------------------------- softmax forward
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("K", [32, 64, 128, 136, 512, 1024])
def test_softmax_dropout_fwd(lib, dt, K):
    B, H, J = 2, 3, 16
    beta = make_tensor((B, H, J, K), dt, 11, 3.0)
    prob = torch.empty((B, H, J, K), dtype=beta.dtype, device=DEV)
    alpha = torch.empty_like(prob)
    lib.softmax_dropout_fwd(DT[dt], B, H, J, K, 0.5, dev(beta), (0.2, 0, 4, 9), prob, alpha)
    torch.cuda.synchronize()
    p = OL.softmax_k(0.5 * f64(beta))
    # dropout factor on the logical (h, b, j, k) order
    fac = philox.dropout_factor(9, 0, 4, 0.2, (H, B, J, K)).transpose(1, 0, 2, 3)
    assert_close("prob", prob, rnd(p, dt), dt)
    a = f64(alpha)
    np.testing.assert_array_equal(a == 0, (fac == 0) | (rnd(rnd(p, dt) * fac, dt) == 0))
    assert_close("alpha", alpha, rnd(rnd(p, dt) * fac, dt), dt)


# ------------------------------------------------------------ bias + act
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("act,p", [(0, 0.0), (0, 0.25), (1, 0.25)])
def test_bias_act_fwd(lib, dt, act, p):
    rows, cols = 33, 200
    x = make_tensor((rows, cols), dt, 21, 2.0)
    b = make_tensor((cols,), dt, 22, 0.5)
    y = torch.empty((rows, cols), dtype=x.dtype, device=DEV)
    lib.bias_act_fwd(DT[dt], rows, cols, dev(x), dev(b), act, (p, 3, 1, 5), y)
    torch.cuda.synchronize()
    u = f64(x) + f64(b)
    ref = OL.act_fwd(u, "gelu" if act == 0 else "relu") * philox.dropout_factor(5, 3, 1, p, (rows, cols))
    assert_close("y", y, rnd(ref, dt), dt)


def test_attn_input_bias(lib):
    dt, rows, H, P = "f16", 40, 4, 16
    x = make_tensor((rows, 3, H, P), dt, 31)
    bs = [make_tensor((P, H), dt, 32 + s) for s in range(3)]
    y = torch.empty_like(x, device=DEV)
    lib.attn_input_bias(DT[dt], rows, H, P, dev(x), dev(bs[0]), dev(bs[1]), dev(bs[2]), y)
    torch.cuda.synchronize()
    ref = f64(x).copy()
    for s in range(3):
        ref[:, s] += f64(bs[s]).T[None]          # b[p][h] -> [h][p]
    assert_close("y", y, rnd(ref, dt), dt)


# ------------------------------------------------- LayerNorm backward family
def _ln_inputs(dt, rows, cols, seed=41):
    dy = make_tensor((rows, cols), dt, seed)
    s = f64(make_tensor((rows, cols), "f32", seed + 1, 2.0, 0.3))
    xhat, rstd = OL.layernorm_i(s.T, 1e-5)
    xh = torch.from_numpy(xhat.T.copy()).to(dy.dtype)
    rs = torch.from_numpy(rstd).float()
    g = make_tensor((cols,), dt, seed + 2, 0.2, 1.0)
    return dy, xh, rs, g


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("rows,cols", [(37, 32), (300, 768), (129, 1024), (8211, 384)])
def test_ln_dropout_bwd(lib, dt, rows, cols):
    dy, xh, rs, g = _ln_inputs(dt, rows, cols)
    ds = torch.empty((rows, cols), dtype=dy.dtype, device=DEV)
    dsub = torch.empty_like(ds)
    lib.ln_dropout_bwd(DT[dt], rows, cols, dev(dy), dev(xh), dev(g), dev(rs), (0.1, 2, 0, 3), ds, dsub)
    torch.cuda.synchronize()
    ref = OL.layernorm_i_bwd(f64(dy).T[:, :, None], f64(xh).T[:, :, None], f64(rs)[:, None], f64(g))[:, :, 0].T
    assert_close("ds", ds, rnd(ref, dt), dt)
    ref_sub = rnd(ref, dt) * philox.dropout_factor(3, 2, 0, 0.1, (rows, cols))
    assert_close("dsub", dsub, rnd(ref_sub, dt), dt)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("rows,cols", [(37, 32), (4096, 1024), (1000, 768)])
def test_ln_param_bwd(lib, dt, rows, cols):
    dy, xh, _, _ = _ln_inputs(dt, rows, cols, seed=51)
    dg = torch.empty(cols, dtype=torch.float32, device=DEV)
    db = torch.empty_like(dg)
    wsb = lib.colsum_ws_bytes(rows, cols)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    lib.ln_param_bwd(DT[dt], rows, cols, dev(dy), dev(xh), dg, db, ws, wsb)
    torch.cuda.synchronize()
    assert_close("dgamma", dg, (f64(dy) * f64(xh)).sum(0), dt, param_grad=True)
    assert_close("dbeta", db, f64(dy).sum(0), dt, param_grad=True)


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("rows,cols", [
    (333, 256),
    # column-split kernel: 8-lane groups, more 16-row tiles than blocks
    (9000, 512),
    # 6 vectors per 8-lane group (2 idle lanes), a single partial tile
    (20, 384),
    # 10 vectors per 16-lane group, tiles striding over 512 blocks
    (8250, 640),
])
def test_residual_ln_param_bwd(lib, dt, rows, cols):
    da = make_tensor((rows, cols), dt, 61)
    dbb = make_tensor((rows, cols), dt, 62)
    _, xh, _, _ = _ln_inputs(dt, rows, cols, seed=63)
    dsum = torch.empty((rows, cols), dtype=da.dtype, device=DEV)
    dg = torch.empty(cols, dtype=torch.float32, device=DEV)
    db = torch.empty_like(dg)
    wsb = lib.colsum_ws_bytes(rows, cols)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    lib.residual_ln_param_bwd(DT[dt], rows, cols, dev(da), dev(dbb), dev(xh), dsum, dg, db, ws, wsb)
    torch.cuda.synchronize()
    s = f64(da) + f64(dbb)
    assert_close("dsum", dsum, rnd(s, dt), dt)
    assert_close("dgamma", dg, (s * f64(xh)).sum(0), dt, param_grad=True)
    assert_close("dbeta", db, s.sum(0), dt, param_grad=True)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("act,p", [(0, 0.0), (0, 0.2), (1, 0.2)])
def test_act_bias_bwd(lib, dt, act, p):
    rows, F, I = 150, 512, 128
    da = make_tensor((rows, F), dt, 71)
    h = make_tensor((rows, F), dt, 72, 1.5)
    b1 = make_tensor((F,), dt, 73, 0.3)
    dout = make_tensor((rows, I), dt, 74)
    dh = torch.empty((rows, F), dtype=da.dtype, device=DEV)
    db1 = torch.empty(F, dtype=torch.float32, device=DEV)
    db2 = torch.empty(I, dtype=torch.float32, device=DEV)
    wsb = lib.colsum_ws_bytes(rows, F)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    lib.act_bias_bwd(DT[dt], rows, F, I, dev(da), dev(h), dev(b1), act, (p, 3, 2, 8), dev(dout), dh, db1, db2,
                     ws, wsb)
    torch.cuda.synchronize()
    u = f64(h) + f64(b1)
    ref = f64(da) * philox.dropout_factor(8, 3, 2, p, (rows, F)) * OL.act_grad(u, "gelu" if act == 0 else "relu")
    assert_close("dh", dh, rnd(ref, dt), dt)
    assert_close("db1", db1, rnd(ref, dt).sum(0), dt, param_grad=True)
    assert_close("db2", db2, f64(dout).sum(0), dt, param_grad=True)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("K", [32, 128, 512])
def test_softmax_dropout_bwd(lib, dt, K):
    B, H, J = 2, 2, 24
    p = OL.softmax_k(f64(make_tensor((B, H, J, K), "f32", 81, 2.0)))
    prob = torch.from_numpy(p).to(make_tensor((1,), dt, 0).dtype)
    da = make_tensor((B, H, J, K), dt, 82)
    dbeta = torch.empty((B, H, J, K), dtype=da.dtype, device=DEV)
    lib.softmax_dropout_bwd(DT[dt], B, H, J, K, 0.125, dev(da), dev(prob), (0.1, 0, 1, 4), dbeta)
    torch.cuda.synchronize()
    fac = philox.dropout_factor(4, 0, 1, 0.1, (H, B, J, K)).transpose(1, 0, 2, 3)
    dp = f64(da) * fac
    P = f64(prob)
    ref = 0.125 * P * (dp - (dp * P).sum(-1, keepdims=True))
    assert_close("dbeta", dbeta, rnd(ref, dt), dt)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_bias_grads_and_residual(lib, dt):
    rows, H, P = 517, 4, 32
    x = make_tensor((rows, 3 * H * P), dt, 91)
    wsb = lib.colsum_ws_bytes(rows, 3 * H * P)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    db = torch.empty(3 * H * P, dtype=torch.float32, device=DEV)
    lib.bias_grad(DT[dt], rows, 3 * H * P, dev(x), db, ws, wsb)
    dq = torch.empty((P, H), dtype=torch.float32, device=DEV)
    dk = torch.empty_like(dq)
    dv = torch.empty_like(dq)
    lib.attn_input_bias_grad(DT[dt], rows, H, P, dev(x), dq, dk, dv, ws, wsb)
    a = make_tensor((rows, 40), dt, 92)
    b = make_tensor((rows, 40), dt, 93)
    o = torch.empty((rows, 40), dtype=a.dtype, device=DEV)
    lib.residual_add(DT[dt], rows * 40, dev(a), dev(b), o)
    torch.cuda.synchronize()
    s = f64(x).sum(0)
    assert_close("db", db, s, dt, param_grad=True)
    per = s.reshape(3, H, P)
    for got, ref in zip((dq, dk, dv), per):
        assert_close("dbqkv", got, ref.T, dt, param_grad=True)
    assert_close("add", o, rnd(f64(a) + f64(b), dt), dt)


# --------------------------------------------------------------- contraction
def _contract_case(lib, dt, a_trans, b_trans, batch, M, N, K, cfg=-1, splits=0):
    A = make_tensor((batch, K, M) if a_trans else (batch, M, K), dt, 101)
    B = make_tensor((batch, N, K) if b_trans else (batch, K, N), dt, 102)
    bias = make_tensor((N,), dt, 103)
    C = torch.empty((batch, M, N), dtype=A.dtype, device=DEV)
    Cf = torch.empty((batch, M, N), dtype=torch.float32, device=DEV)
    ws, wsb = None, 0
    if splits > 1:
        wsb = splits * batch * M * N * 4
        ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    lib.contract(DT[dt], batch, M, N, K, 0.5, dev(A), a_trans, M * K, dev(B), b_trans, N * K, dev(bias), C, 0,
                 M * N, cfg, splits, ws, wsb)
    lib.contract(DT[dt], batch, M, N, K, 1.0, dev(A), a_trans, M * K, dev(B), b_trans, N * K, None, Cf, 1, M * N,
                 cfg, splits, ws, wsb)
    torch.cuda.synchronize()
    a = f64(A).transpose(0, 2, 1) if a_trans else f64(A)
    b = f64(B).transpose(0, 2, 1) if b_trans else f64(B)
    ref = np.matmul(a, b)
    assert_close("C", C, rnd(0.5 * ref + f64(bias), dt), dt)
    assert_close("Cf", Cf, ref, "f32" if dt == "f32" else dt)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("a_trans,b_trans", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("batch,M,N,K", [(1, 128, 128, 64), (3, 136, 200, 72), (2, 264, 40, 520), (1, 8, 8, 8)])
def test_contract_modes(lib, dt, a_trans, b_trans, batch, M, N, K):
    _contract_case(lib, dt, a_trans, b_trans, batch, M, N, K)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("cfg", list(range(26)))
@pytest.mark.parametrize("a_trans,b_trans", [(0, 1), (0, 0), (1, 0), (1, 1)])
def test_contract_tile_configs(lib, dt, cfg, a_trans, b_trans):
    # ragged in every dimension for every block tile
    _contract_case(lib, dt, a_trans, b_trans, 2, 264, 328, 200, cfg=cfg)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("a_trans,b_trans", [(0, 1), (0, 0), (1, 0), (1, 1)])
@pytest.mark.parametrize("batch,M,N,K,splits", [(2, 264, 328, 256, 1), (1, 512, 256, 512, 1), (1, 264, 520, 1152, 3),
                                                (3, 136, 40, 128, 1), (1, 8, 8, 64, 1), (2, 40, 200, 32, 1),
                                                (1, 296, 200, 96, 1)])
@pytest.mark.parametrize("cfg", [13, 15, 16, 17, 18, 19, 20, 21, 22, 23, 24, 25])
def test_contract_lean(lib, dt, a_trans, b_trans, batch, M, N, K, splits, cfg):
    # the lean kernels themselves (k a multiple of their 32- or 64-wide
    # step): ragged m and n, split k (single batch), bias and float output;
    # k of one and three 32-wide steps (fewer steps than the ping-pong
    # schedule keeps in flight)
    _contract_case(lib, dt, a_trans, b_trans, batch, M, N, K, cfg=cfg, splits=splits)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("a_trans,b_trans", [(0, 1), (0, 0), (1, 0), (1, 1)])
def test_contract_schedules_bit_identical(lib, dt, a_trans, b_trans):
    # the lean 32x32x16 kernels differ only in tiling and in how loads, reads
    # and MFMAs are scheduled: every output element takes the same MFMA
    # instruction over the same 16-wide k slices in the same order, so the
    # interleaved and ping-pong schedules (cfg 20, 23, 24; 21 and 25 on the
    # 192-wide tiles) reproduce the two-waves-per-SIMD kernel (cfg 13, 19)
    # bit for bit, also with bias and split partials; ragged m and n
    batch, M, N, K = 1, 520, 392, 1024
    A = make_tensor((batch, K, M) if a_trans else (batch, M, K), dt, 111)
    B = make_tensor((batch, N, K) if b_trans else (batch, K, N), dt, 112)
    bias = make_tensor((N,), dt, 113)

    def run(cfg, splits=1, out_f32=0):
        C = torch.empty((batch, M, N), dtype=torch.float32 if out_f32 else A.dtype, device=DEV)
        wsb = splits * batch * M * N * 4 if splits > 1 else 0
        ws = torch.empty(wsb, dtype=torch.uint8, device=DEV) if wsb else None
        lib.contract(DT[dt], batch, M, N, K, 0.5, dev(A), a_trans, M * K, dev(B), b_trans, N * K,
                     None if out_f32 else dev(bias), C, out_f32, M * N, cfg, splits, ws, wsb)
        torch.cuda.synchronize()
        return C.cpu()

    for out_f32 in (0, 1):
        for splits in (1, 2):
            ref = run(13, splits, out_f32)
            for cfg in (20, 23, 24):
                assert torch.equal(run(cfg, splits, out_f32), ref), (cfg, splits, out_f32)
            if b_trans:  # the 192-wide tiles take a B contiguous along k
                ref192 = run(19, splits, out_f32)
                assert torch.equal(ref192, ref)
                for cfg in (21, 25):
                    assert torch.equal(run(cfg, splits, out_f32), ref), (cfg, splits, out_f32)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("cfg,splits", [(2, 2), (4, 3), (0, 4), (3, 5), (5, 2), (6, 3), (7, 4), (8, 2), (9, 2), (10, 3), (11, 4), (12, 2), (13, 3), (14, 2), (15, 2), (16, 3), (17, 2), (18, 3), (19, 2), (20, 2), (21, 3), (22, 2), (23, 3), (24, 2), (25, 2)])
@pytest.mark.parametrize("a_trans,b_trans", [(0, 1), (1, 0)])
def test_contract_split_k(lib, dt, cfg, splits, a_trans, b_trans):
    _contract_case(lib, dt, a_trans, b_trans, 2, 136, 264, 1096, cfg=cfg, splits=splits)
