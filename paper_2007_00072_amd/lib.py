"""ctypes binding of libdmtx.so (the C ABI declared in include/dmtx.h).

Argument marshalling only: every function here passes device pointers and
sizes straight to the library, whose HIP kernels do all of the work.
Functions carry the C names.  Tensors may be passed wherever the C ABI
takes a pointer (their data_ptr() is used); None maps to NULL.  A nonzero
status raises DmError with the library's message.

Importing this module fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
# DMTX_LIB names another build of the same library (the host-sanitized one
# used by the CPU validation checks); by default the in-tree libdmtx.so
LIB_PATH = os.environ.get("DMTX_LIB") or os.path.join(PKG, "libdmtx.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2007_00072_amd.build` "
                      "(or __graft_entry__.build())")

# torch's HIP runtime is loaded first, so the library binds to the same one
# (loading the library first would bring a second runtime into the process)
import torch  # noqa: E402,F401

_lib = C.CDLL(LIB_PATH)

DM_OK, DM_ERR_ARG, DM_ERR_UNSUPPORTED, DM_ERR_WORKSPACE, DM_ERR_DEVICE = range(5)
DM_F32, DM_F16, DM_BF16 = 0, 1, 2
DM_BJI, DM_IBJ = 0, 1
DM_GELU, DM_RELU = 0, 1
DTYPE_CODES = {"f32": DM_F32, "f16": DM_F16, "bf16": DM_BF16}
LAYOUT_CODES = {"bji": DM_BJI, "ibj": DM_IBJ}
SAVED_IDS = {"qkv": 0, "prob": 1, "alpha": 2, "gamma": 3, "xhat1": 4, "rstd1": 5, "y1": 6,
             "h": 7, "a": 8, "xhat2": 9, "rstd2": 10}

EXPORTED = [
    "encoder_layer_sizes", "encoder_layer_fwd", "encoder_layer_bwd",
    "mha_sizes", "mha_fwd", "mha_bwd",
    "colsum_ws_bytes", "bdrln_fwd", "softmax_dropout_fwd", "bias_act_fwd", "attn_input_bias",
    "ln_param_bwd", "ln_dropout_bwd", "residual_ln_param_bwd", "act_bias_bwd",
    "softmax_dropout_bwd", "bias_grad", "bias_grad_noalloc", "attn_input_bias_grad", "residual_add",
    "dropout_mask", "saved_tensor_view", "attn_backward_form", "contract", "dm_last_error",
    "dm_trace_enable", "dm_trace_count", "dm_trace_get",
    "plan_create", "plan_destroy", "plan_log", "plan_log_read",
]


class ContractChoice(C.Structure):
    _fields_ = [("M", C.c_int64), ("N", C.c_int64), ("K", C.c_int64), ("batch", C.c_int64),
                ("dtype", C.c_int32), ("a_kcontig", C.c_int32), ("b_kcontig", C.c_int32),
                ("tile_cfg", C.c_int32), ("splits", C.c_int32), ("label", C.c_char * 48)]

    def key(self):
        return (self.M, self.N, self.K, self.batch, self.dtype, self.a_kcontig, self.b_kcontig)


class LayoutChoice(C.Structure):
    """Layout and reduction choices of the fused operators (-1: library's choice)."""
    _fields_ = [("dO_transposed", C.c_int32), ("dH_transposed", C.c_int32), ("ln_bwd_form", C.c_int32),
                ("ln_lanes", C.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class DmError(RuntimeError):
    def __init__(self, code: int, fn: str):
        self.code = code
        msg = _lib.dm_last_error().decode(errors="replace")
        super().__init__(f"{fn} returned {code}: {msg}")


class LayerDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("J", C.c_int32), ("K", C.c_int32), ("H", C.c_int32),
                ("P", C.c_int32), ("W", C.c_int32), ("I", C.c_int32), ("F", C.c_int32),
                ("dtype", C.c_int32), ("layout", C.c_int32), ("act", C.c_int32),
                ("scaler", C.c_float), ("ln_eps", C.c_float),
                ("p_attn", C.c_float), ("p_attn_out", C.c_float), ("p_ffn_out", C.c_float),
                ("p_ffn_act", C.c_float), ("seed", C.c_uint64), ("layer_id", C.c_uint32),
                ("self_attention", C.c_int32), ("causal", C.c_int32), ("qkv_fusion", C.c_int32),
                ("plan", C.c_void_p)]


_PNAMES = ["wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo", "g1", "be1", "w1", "b1", "w2", "b2",
           "g2", "be2"]


class LayerParams(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _PNAMES]


class LayerGrads(C.Structure):
    _fields_ = [("d" + n, C.c_void_p) for n in _PNAMES]


class Dropout(C.Structure):
    _fields_ = [("p", C.c_float), ("site", C.c_uint32), ("layer", C.c_uint32), ("seed", C.c_uint64)]


def _sig(name, res, *args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


P_ = C.c_void_p
I32, I64, U32, U64, F32, SZ = C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_float, C.c_size_t
PDESC, PPRM, PGRD, PDROP = C.POINTER(LayerDesc), C.POINTER(LayerParams), C.POINTER(LayerGrads), C.POINTER(Dropout)
PSZ = C.POINTER(C.c_size_t)

_f = {}
_f["encoder_layer_sizes"] = _sig("encoder_layer_sizes", I32, PDESC, PSZ, PSZ, PSZ)
_f["encoder_layer_fwd"] = _sig("encoder_layer_fwd", I32, PDESC, PPRM, P_, P_, P_, P_, SZ, P_)
_f["encoder_layer_bwd"] = _sig("encoder_layer_bwd", I32, PDESC, PPRM, P_, P_, P_, P_, PGRD, P_, SZ, P_)
_f["mha_sizes"] = _sig("mha_sizes", I32, PDESC, PSZ, PSZ, PSZ)
_f["mha_fwd"] = _sig("mha_fwd", I32, PDESC, PPRM, P_, P_, P_, P_, P_, P_, SZ, P_)
_f["mha_bwd"] = _sig("mha_bwd", I32, PDESC, PPRM, P_, P_, P_, P_, P_, P_, P_, P_, PGRD, P_, SZ, P_)
_f["colsum_ws_bytes"] = _sig("colsum_ws_bytes", SZ, I64, I32)
_f["bdrln_fwd"] = _sig("bdrln_fwd", I32, I32, I64, I32, P_, P_, P_, P_, P_, F32, PDROP, P_, P_, P_, P_)
_f["softmax_dropout_fwd"] = _sig("softmax_dropout_fwd", I32, I32, I32, I32, I32, I32, F32, P_, PDROP, P_, P_, P_)
_f["bias_act_fwd"] = _sig("bias_act_fwd", I32, I32, I64, I32, P_, P_, I32, PDROP, P_, P_)
_f["attn_input_bias"] = _sig("attn_input_bias", I32, I32, I64, I32, I32, P_, P_, P_, P_, P_, P_)
_f["ln_param_bwd"] = _sig("ln_param_bwd", I32, I32, I64, I32, P_, P_, P_, P_, P_, SZ, P_)
_f["ln_dropout_bwd"] = _sig("ln_dropout_bwd", I32, I32, I64, I32, P_, P_, P_, P_, PDROP, P_, P_, P_)
_f["residual_ln_param_bwd"] = _sig("residual_ln_param_bwd", I32, I32, I64, I32, P_, P_, P_, P_, P_, P_, P_, SZ, P_)
_f["act_bias_bwd"] = _sig("act_bias_bwd", I32, I32, I64, I32, I32, P_, P_, P_, I32, PDROP, P_, P_, P_, P_, P_, SZ, P_)
_f["softmax_dropout_bwd"] = _sig("softmax_dropout_bwd", I32, I32, I32, I32, I32, I32, F32, P_, P_, PDROP, P_, P_)
_f["bias_grad"] = _sig("bias_grad", I32, I32, I64, I32, P_, P_, P_, SZ, P_)
_f["bias_grad_noalloc"] = _sig("bias_grad_noalloc", I32, I32, I64, I32, P_, P_, P_)
_f["attn_input_bias_grad"] = _sig("attn_input_bias_grad", I32, I32, I64, I32, I32, P_, P_, P_, P_, P_, SZ, P_)
_f["residual_add"] = _sig("residual_add", I32, I32, I64, P_, P_, P_, P_)
_f["dropout_mask"] = _sig("dropout_mask", I32, U64, U32, U32, F32, U64, U64, P_, P_)
_f["saved_tensor_view"] = _sig("saved_tensor_view", I32, PDESC, I32, PSZ, PSZ)
_f["attn_backward_form"] = _sig("attn_backward_form", I32, PDESC, C.POINTER(C.c_int32))
_f["contract"] = _sig("contract", I32, I32, I32, I32, I32, I32, F32, P_, I32, I64, P_, I32, I64, P_, P_, I32, I64,
                      I32, I32, P_, SZ, P_)
_f["dm_last_error"] = _sig("dm_last_error", C.c_char_p)
_f["dm_trace_enable"] = _sig("dm_trace_enable", I32, I32)
_f["dm_trace_count"] = _sig("dm_trace_count", I32)
_f["dm_trace_get"] = _sig("dm_trace_get", I32, I32, C.POINTER(C.c_char_p), C.POINTER(C.c_char_p),
                          C.POINTER(C.c_float))
_f["plan_create"] = _sig("plan_create", I32, C.POINTER(ContractChoice), I32, I32, C.POINTER(LayoutChoice),
                         C.POINTER(C.c_void_p))
_f["plan_destroy"] = _sig("plan_destroy", I32, C.c_void_p)
_f["plan_log"] = _sig("plan_log", I32, I32)
_f["plan_log_read"] = _sig("plan_log_read", I32, C.POINTER(ContractChoice), I32, C.POINTER(I32))


def ptr(t) -> Optional[int]:
    """Device (or host) address of a tensor / int / None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def current_stream():
    import torch
    if torch.cuda.is_available():
        return torch.cuda.current_stream().cuda_stream
    return None


def _call(name, *args):
    rc = _f[name](*args)
    if rc != DM_OK:
        raise DmError(rc, name)
    return rc


def _drop(d):
    if d is None:
        return None
    if isinstance(d, Dropout):
        return C.byref(d)
    p, site, layer, seed = d
    return C.byref(Dropout(p, site, layer, seed))


def make_desc(shape, dtype: str, layout: str = "bji", act: str = "gelu", scaler: float = 0.0,
              ln_eps: float = 1e-12, p_attn=0.0, p_attn_out=0.0, p_ffn_out=0.0, p_ffn_act=0.0,
              seed: int = 0, layer_id: int = 0, self_attention=True, causal: bool = False,
              qkv_fusion: int = 0, plan: "Optional[Plan]" = None) -> LayerDesc:
    d = LayerDesc(shape.B, shape.J, shape.K, shape.H, shape.P, shape.W, shape.I, shape.F,
                  DTYPE_CODES[dtype], LAYOUT_CODES[layout], DM_GELU if act == "gelu" else DM_RELU,
                  scaler, ln_eps, p_attn, p_attn_out, p_ffn_out, p_ffn_act, seed, layer_id,
                  int(self_attention), 1 if causal else 0, qkv_fusion, None)
    set_plan(d, plan)
    return d


def set_plan(desc: LayerDesc, plan: "Optional[Plan]") -> None:
    """Points the descriptor at a plan (None: built-in choices); the
    descriptor keeps the Plan object alive."""
    desc.plan = plan.handle if plan is not None else None
    desc._plan_ref = plan


def make_params(tensors) -> LayerParams:
    return LayerParams(*[ptr(tensors.get(n)) for n in _PNAMES])


def make_grads(tensors) -> LayerGrads:
    return LayerGrads(*[ptr(tensors.get(n)) for n in _PNAMES])


# ---------------------------------------------------------------- layer
def encoder_layer_sizes(desc: LayerDesc):
    s, f, b = C.c_size_t(), C.c_size_t(), C.c_size_t()
    _call("encoder_layer_sizes", C.byref(desc), C.byref(s), C.byref(f), C.byref(b))
    return s.value, f.value, b.value


def encoder_layer_fwd(desc, params: LayerParams, x, y, saved, ws, ws_bytes, stream=None):
    return _call("encoder_layer_fwd", C.byref(desc), C.byref(params), ptr(x), ptr(y), ptr(saved), ptr(ws),
                 ws_bytes, stream if stream is not None else current_stream())


def encoder_layer_bwd(desc, params: LayerParams, x, saved, dy, dx, grads: LayerGrads, ws, ws_bytes, stream=None):
    return _call("encoder_layer_bwd", C.byref(desc), C.byref(params), ptr(x), ptr(saved), ptr(dy), ptr(dx),
                 C.byref(grads), ptr(ws), ws_bytes, stream if stream is not None else current_stream())


def mha_sizes(desc: LayerDesc):
    s, f, b = C.c_size_t(), C.c_size_t(), C.c_size_t()
    _call("mha_sizes", C.byref(desc), C.byref(s), C.byref(f), C.byref(b))
    return s.value, f.value, b.value


def mha_fwd(desc, params, q, k, v, out, saved, ws, ws_bytes, stream=None):
    return _call("mha_fwd", C.byref(desc), C.byref(params), ptr(q), ptr(k), ptr(v), ptr(out), ptr(saved),
                 ptr(ws), ws_bytes, stream if stream is not None else current_stream())


def mha_bwd(desc, params, q, k, v, saved, dout, dq, dk, dv, grads, ws, ws_bytes, stream=None):
    return _call("mha_bwd", C.byref(desc), C.byref(params), ptr(q), ptr(k), ptr(v), ptr(saved), ptr(dout),
                 ptr(dq), ptr(dk), ptr(dv), C.byref(grads), ptr(ws), ws_bytes,
                 stream if stream is not None else current_stream())


def saved_tensor_view(desc, name: str):
    o, b = C.c_size_t(), C.c_size_t()
    _call("saved_tensor_view", C.byref(desc), SAVED_IDS[name], C.byref(o), C.byref(b))
    return o.value, b.value


def attn_backward_form(desc) -> bool:
    """True when this descriptor's backward takes the key-block form of the
    attention-score backward (d(alpha) never stored), False for the row form."""
    kb = C.c_int32()
    _call("attn_backward_form", C.byref(desc), C.byref(kb))
    return bool(kb.value)


# ----------------------------------------------------- fused operators
def colsum_ws_bytes(rows: int, cols: int) -> int:
    return _f["colsum_ws_bytes"](rows, cols)


def _st(stream):
    return stream if stream is not None else current_stream()


def bdrln_fwd(dtype, rows, cols, x, bias, resid, gamma, beta, eps, drop, y, xhat, rstd, stream=None):
    return _call("bdrln_fwd", dtype, rows, cols, ptr(x), ptr(bias), ptr(resid), ptr(gamma), ptr(beta), eps,
                 _drop(drop), ptr(y), ptr(xhat), ptr(rstd), _st(stream))


def softmax_dropout_fwd(dtype, B, H, J, K, scale, beta, drop, prob, alpha, stream=None):
    return _call("softmax_dropout_fwd", dtype, B, H, J, K, scale, ptr(beta), _drop(drop), ptr(prob), ptr(alpha),
                 _st(stream))


def bias_act_fwd(dtype, rows, cols, x, bias, act, drop, y, stream=None):
    return _call("bias_act_fwd", dtype, rows, cols, ptr(x), ptr(bias), act, _drop(drop), ptr(y), _st(stream))


def attn_input_bias(dtype, rows, H, P, x, bq, bk, bv, y, stream=None):
    return _call("attn_input_bias", dtype, rows, H, P, ptr(x), ptr(bq), ptr(bk), ptr(bv), ptr(y), _st(stream))


def ln_param_bwd(dtype, rows, cols, dy, xhat, dgamma, dbeta, ws, ws_bytes, stream=None):
    return _call("ln_param_bwd", dtype, rows, cols, ptr(dy), ptr(xhat), ptr(dgamma), ptr(dbeta), ptr(ws),
                 ws_bytes, _st(stream))


def ln_dropout_bwd(dtype, rows, cols, dy, xhat, gamma, rstd, drop, ds, dsub, stream=None):
    return _call("ln_dropout_bwd", dtype, rows, cols, ptr(dy), ptr(xhat), ptr(gamma), ptr(rstd), _drop(drop),
                 ptr(ds), ptr(dsub), _st(stream))


def residual_ln_param_bwd(dtype, rows, cols, da, db, xhat, dsum, dgamma, dbeta, ws, ws_bytes, stream=None):
    return _call("residual_ln_param_bwd", dtype, rows, cols, ptr(da), ptr(db), ptr(xhat), ptr(dsum), ptr(dgamma),
                 ptr(dbeta), ptr(ws), ws_bytes, _st(stream))


def act_bias_bwd(dtype, rows, F, I, da, h, b1, act, drop, dout, dh, db1, db2, ws, ws_bytes, stream=None):
    return _call("act_bias_bwd", dtype, rows, F, I, ptr(da), ptr(h), ptr(b1), act, _drop(drop), ptr(dout), ptr(dh),
                 ptr(db1), ptr(db2), ptr(ws), ws_bytes, _st(stream))


def softmax_dropout_bwd(dtype, B, H, J, K, scale, dalpha, prob, drop, dbeta, stream=None):
    return _call("softmax_dropout_bwd", dtype, B, H, J, K, scale, ptr(dalpha), ptr(prob), _drop(drop), ptr(dbeta),
                 _st(stream))


def bias_grad(dtype, rows, cols, x, db, ws, ws_bytes, stream=None):
    return _call("bias_grad", dtype, rows, cols, ptr(x), ptr(db), ptr(ws), ws_bytes, _st(stream))


def bias_grad_noalloc(dtype, rows, cols, x, db, stream=None):
    return _call("bias_grad_noalloc", dtype, rows, cols, ptr(x), ptr(db), _st(stream))


def attn_input_bias_grad(dtype, rows, H, P, x, dbq, dbk, dbv, ws, ws_bytes, stream=None):
    return _call("attn_input_bias_grad", dtype, rows, H, P, ptr(x), ptr(dbq), ptr(dbk), ptr(dbv), ptr(ws),
                 ws_bytes, _st(stream))


def residual_add(dtype, n, a, b, out, stream=None):
    return _call("residual_add", dtype, n, ptr(a), ptr(b), ptr(out), _st(stream))


def dropout_mask(seed, site, layer, p, offset, n, out, stream=None):
    return _call("dropout_mask", seed, site, layer, p, offset, n, ptr(out), _st(stream))


def contract(dtype, batch, M, N, K, alpha, A, a_trans, sa, B, b_trans, sb, bias, Cout, out_f32, sc,
             tile_cfg=-1, splits=0, ws=None, ws_bytes=0, stream=None):
    return _call("contract", dtype, batch, M, N, K, alpha, ptr(A), a_trans, sa, ptr(B), b_trans, sb, ptr(bias),
                 ptr(Cout), out_f32, sc, tile_cfg, splits, ptr(ws), ws_bytes, _st(stream))


def dm_trace_enable(on: bool) -> None:
    _call("dm_trace_enable", 1 if on else 0)


def dm_trace_count() -> int:
    return _f["dm_trace_count"]()


def dm_trace_get(i: int):
    """(label, sub-label, ms) of the i-th launch record."""
    lab, sub, ms = C.c_char_p(), C.c_char_p(), C.c_float()
    _call("dm_trace_get", i, C.byref(lab), C.byref(sub), C.byref(ms))
    return lab.value.decode(), (sub.value or b"").decode(), ms.value


def trace_records():
    """All (label, sub-label, ms) records of the current timing session; an
    operator's second launch carries a sub-label (e.g. "reduce")."""
    return [dm_trace_get(i) for i in range(dm_trace_count())]


class Plan:
    """A configuration plan (plan_create) owned by Python: entries are
    ContractChoice records (or (M, N, K, batch, dtype, a_kcontig, b_kcontig,
    tile_cfg, splits) tuples); layout a LayoutChoice or a dict of its fields
    (missing ones: the library's choice).  Name it in a descriptor (make_desc(plan=...)
    or set_plan) to use it; destroyed with the object."""

    def __init__(self, entries=(), attn_path: int = 0, layout=None):
        recs = [e if isinstance(e, ContractChoice) else ContractChoice(*e) for e in entries]
        arr = (ContractChoice * max(1, len(recs)))(*recs)
        if isinstance(layout, dict):
            layout = LayoutChoice(**{f: int(layout.get(f, -1)) for f, _ in LayoutChoice._fields_})
        h = C.c_void_p()
        _call("plan_create", arr if recs else None, len(recs), attn_path,
              C.byref(layout) if layout is not None else None, C.byref(h))
        self.handle = h.value
        self.entries = recs
        self.attn_path = attn_path
        self.layout = layout

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h is not None and _f is not None:
            _f["plan_destroy"](h)


def plan_log(on: bool) -> None:
    _call("plan_log", 1 if on else 0)


def plan_log_read():
    """The contractions launched since plan_log(True), as ContractChoice records."""
    n = I32()
    _call("plan_log_read", None, 0, C.byref(n))
    arr = (ContractChoice * max(1, n.value))()
    _call("plan_log_read", arr, n.value, C.byref(n))
    return list(arr[: n.value])


def dm_last_error() -> str:
    return _lib.dm_last_error().decode(errors="replace")
