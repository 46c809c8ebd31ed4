"""Algorithmic work of every launch in the encoder layer (the analogue of
the paper's per-operator flop / I/O analysis, Table 3).

For each operator the model counts flop (2 per multiply-add of a
contraction; element-wise work is not counted as flop) and the minimum
bytes it must move: every input read once and every output written once,
in the storage dtype (float32 for statistics and parameter gradients).
Dropout masks cost no bytes (they are regenerated).  Scratch traffic of
the two-stage column reductions is not algorithmic and appears as zero.

Labels equal those the library records in its per-launch timing.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict

from .inputs import Shape

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_PEAK_TFLOPS = {"f16": 2516.6, "bf16": 2516.6, "f32": 157.3}   # dense MFMA / fp32 vector


@dataclass
class Work:
    flop: float
    bytes: float
    bound: str     # "mfma" or "hbm"
    cls: str = ""  # "fused" (memory-bound fused operator) or "contraction"; default from flop
    overhead: float = 0.0  # bytes the launch moves by design beyond the algorithmic minimum

    def __post_init__(self):
        if not self.cls:
            self.cls = "fused" if self.flop == 0.0 else "contraction"


def ridge(dtype: str) -> float:
    return MFMA_PEAK_TFLOPS[dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)


def _gemm(M, N, K, a_el, b_el, c_el, es, c_es=None, dtype="f16", extra=0.0) -> Work:
    c_es = es if c_es is None else c_es
    flop = 2.0 * M * N * K
    byt = (a_el + b_el) * es + c_el * c_es + extra
    return Work(flop, byt, "mfma" if flop / byt > ridge(dtype) else "hbm")


# Launch groups that stand in for several others when attention scores stay
# on chip; a layer runs either the group or all of the groups it replaces.
REPLACES = {
    "F2-3 qkt_softmax": ("F2 qkt", "F3 softmax"),
    "F2-4 qkt_softmax_gamma": ("F2 qkt", "F3 softmax", "F4 gamma"),
    "B13-15 gamma_dx1_softmax_bwd": ("B13 gamma_dx1", "B15 softmax_bwd"),
    "B13+15+16 score_bwd_dq": ("B13 gamma_dx1", "B15 softmax_bwd", "B16 qkt_dx1"),
    "B13-17 score_bwd_keys": ("B13 gamma_dx1", "B14 gamma_dx2", "B15 softmax_bwd", "B16 qkt_dx1", "B17 qkt_dx2"),
}
# Contractions the encoder layer issues as one launch (their tiles together
# fill the chip): the backward's output-projection and Q/K/V weight gradients.
PAIRED = {"B12+19 out_dw+qkv_dw": ("B12 out_dw", "B19 qkv_dw")}
# Operators that run inside a contraction's epilogue where its kernel
# allows (else as launches of their own): Linear 1 with bias + activation;
# the input-bias gradient's partial sums inside the Q/K/V weight gradient
# (that launch then also writes the three bias gradients).
EPILOGUE = {"F7+8 linear1_bias_act": ("F7 linear1", "F8 bias_act"),
            "B3+5 linear2_dx_act_bwd": ("B3 linear2_dx", "B5 act_bwd")}
FOLDED = {"B20 qkv_bias_grad": "B12+19 out_dw+qkv_dw"}
# The launch sets one layer can run: every score step separate, scores on
# chip, scores on chip with the next contraction in the same launch, and
# that forward with the key-block backward (head size 64, K a multiple of 128).
PATHS = {
    "separate": (),
    "scores": ("F2-3 qkt_softmax", "B13-15 gamma_dx1_softmax_bwd"),
    "scores_next": ("F2-4 qkt_softmax_gamma", "B13+15+16 score_bwd_dq"),
    "keys": ("F2-4 qkt_softmax_gamma", "B13-17 score_bwd_keys"),
}


def key_blocks(s: Shape, dtype: str):
    """Key-block backward of the shape: (possible, key blocks per head)."""
    if dtype == "f32" or s.P != 64 or s.W != 64 or s.K % 128:
        return False, 0
    kg = 8 if s.K % 256 == 0 and s.B * s.H * (s.K // 256) >= 192 else 4
    return True, s.K // (32 * kg)


def path_groups(w: Dict[str, "Work"], path: str, epilogue=(), folded: bool = False) -> Dict[str, "Work"]:
    """The launch groups of `w` that path `path` runs (epilogue: the EPILOGUE
    groups that ran, in place of their parts, True for all of them; folded:
    without the FOLDED launches)."""
    fused = PATHS[path]
    gone = {p for f in fused for p in REPLACES[f]} | {p for parts in PAIRED.values() for p in parts}
    ran = set(EPILOGUE) if epilogue is True else set(epilogue or ())
    for k, parts in EPILOGUE.items():
        gone |= set(parts) if k in ran else {k}
    if folded:
        gone |= set(FOLDED)
    return {k: v for k, v in w.items() if (k not in REPLACES or k in fused) and k not in gone}


def encoder_layer(s: Shape, dtype: str, elements: bool = False) -> Dict[str, Work]:
    """Work of each labelled launch group of one encoder-layer forward + backward.

    Holds both forms of the attention-score steps (see REPLACES).  With
    elements=True the `bytes` fields count elements instead (every tensor
    element once, whatever its type), the unit of the paper's I/O columns."""
    es = 4 if dtype == "f32" else 2
    f4 = 4
    if elements:
        es = f4 = 1
    T, I, F, H, P, W = s.B * s.J, s.I, s.F, s.H, s.P, s.W
    Z, J, K = s.B * s.H, s.J, s.K
    N, S, Fh = T * I, s.B * s.H * s.J * s.K, T * F
    g = lambda *a, **k: _gemm(*a, es=es, dtype=dtype, **k)
    m = lambda b: Work(0.0, float(b), "hbm")
    w = {}
    # forward
    w["F1 qkv"] = g(T, 3 * I, I, N, 3 * I * I, 3 * N, extra=3 * I * es)
    w["F2 qkt"] = _att(Z, J, K, P, es, dtype, S, N)
    w["F3 softmax"] = m(3 * S * es)
    # QK^T and softmax + dropout in one launch: Q, K read; P and alpha written
    w["F2-3 qkt_softmax"] = Work(2.0 * Z * J * K * P, float((2 * N + 2 * S) * es), "hbm", "fused")
    # ... and Gamma = alpha V in the same launch: V read, Gamma written, alpha
    # kept on chip (when the key-block backward can run, Gamma is also
    # written in fp32 before rounding: overhead)
    keys, nkb = key_blocks(s, dtype)
    w["F2-4 qkt_softmax_gamma"] = Work(2.0 * Z * J * K * (P + W), float((4 * N + S) * es), "hbm", "fused")
    if keys:
        w["F2-4 qkt_softmax_gamma"].overhead = f4 * N
    w["F4 gamma"] = _att(Z, J, W, K, es, dtype, S, N)
    w["F5 out"] = g(T, I, I, N, I * I, N)
    w["F6 bdrln1"] = m(4 * N * es + f4 * T + 3 * I * es)
    w["F7 linear1"] = g(T, F, I, N, F * I, Fh)
    w["F8 bias_act"] = m(2 * Fh * es + F * es)
    # Linear 1 writing H and A = act(H + b1) from its epilogue: H is not
    # read back
    w["F7+8 linear1_bias_act"] = Work(w["F7 linear1"].flop, w["F7 linear1"].bytes + Fh * es + F * es, "mfma",
                                      "contraction")
    w["F9 linear2"] = g(T, I, F, Fh, I * F, N)
    w["F10 bdrln2"] = m(4 * N * es + f4 * T + 3 * I * es)
    # backward
    # (the column-split LayerNorm backward also writes dO transposed for the
    # Linear-2 weight gradient: 16-bit, I a multiple of 64 in 320..1024; the
    # dataflow needs dO once, so that copy is overhead, not algorithmic)
    dot = N * es if dtype != "f32" and I % 64 == 0 and 320 <= I <= 1024 else 0
    w["B1-2 ln2_bwd"] = m(4 * N * es + f4 * T + I * es + 3 * I * f4)
    w["B1-2 ln2_bwd"].overhead = dot
    w["B3 linear2_dx"] = g(T, F, I, N, I * F, Fh)
    w["B4 linear2_dw"] = g(I, F, T, N, Fh, I * F, c_es=f4)
    w["B5 act_bwd"] = m(3 * Fh * es + F * es + F * f4)
    # Linear 2 dX with the activation backward in its epilogue: dA is
    # neither written nor read back (dH, H, b1 and db1 as in B5)
    w["B3+5 linear2_dx_act_bwd"] = Work(w["B3 linear2_dx"].flop,
                                        w["B3 linear2_dx"].bytes + Fh * es + F * es + F * f4, "mfma", "contraction")
    w["B6 linear1_dx"] = g(T, I, F, Fh, F * I, N)
    w["B7 linear1_dw"] = g(F, I, T, Fh, N, F * I, c_es=f4)
    w["B8-10 ln1_bwd"] = m(5 * N * es + f4 * T + I * es + 3 * I * f4)
    w["B11 out_dx"] = g(T, I, I, N, I * I, N)
    w["B12 out_dw"] = g(I, I, T, N, N, I * I, c_es=f4)
    w["B13 gamma_dx1"] = _att(Z, J, K, W, es, dtype, S, N)
    w["B14 gamma_dx2"] = _att(Z, K, W, J, es, dtype, S, N)
    w["B15 softmax_bwd"] = m(3 * S * es)
    # Gamma dX1 and the softmax + dropout backward in one launch: dGamma, V
    # and P read, dbeta written
    w["B13-15 gamma_dx1_softmax_bwd"] = Work(2.0 * Z * J * K * W, float((2 * N + 2 * S) * es), "hbm", "fused")
    # ... and dQ = dbeta K in the same launch: K read and dQ written too
    w["B13+15+16 score_bwd_dq"] = Work(2.0 * Z * J * K * (W + P), float((4 * N + 2 * S) * es), "hbm", "fused")
    # the key-block backward: dGamma, gamma, P, Q, K, V read; dQ, dK, dV
    # written (gamma read in fp32, and with several key blocks per head the
    # fp32 dQ partials written and read back: overhead)
    w["B13-17 score_bwd_keys"] = Work(2.0 * Z * J * K * 2 * (W + P), float((9 * N + S) * es), "hbm", "fused")
    if keys:
        w["B13-17 score_bwd_keys"].overhead = (f4 - es) * N + (2 * nkb * f4 * N if nkb > 1 else 0)
    w["B16 qkt_dx1"] = _att(Z, J, P, K, es, dtype, S, N)
    w["B17 qkt_dx2"] = _att(Z, K, P, J, es, dtype, S, N)
    w["B18 qkv_dx"] = g(T, I, 3 * I, 3 * N, 3 * I * I, N, extra=N * es)      # + residual read
    w["B19 qkv_dw"] = g(3 * I, I, T, 3 * N, N, 3 * I * I, c_es=f4)
    for lab, parts in PAIRED.items():
        w[lab] = Work(sum(w[p].flop for p in parts), sum(w[p].bytes for p in parts), "mfma", "contraction")
    w["B20 qkv_bias_grad"] = m(3 * N * es + 3 * I * f4)
    # column-sum partials of B1-2, B5, B8-10 and B20 finished in one launch
    w["B colsum finish"] = m(0)
    return w


def _att(Z, M, N, K, es, dtype, S, Ntok) -> Work:
    """Batched attention contraction: one S-sized operand and two N-sized ones."""
    flop = 2.0 * Z * M * N * K
    byt = (S + 2 * Ntok) * es
    return Work(flop, byt, "mfma" if flop / byt > ridge(dtype) else "hbm")


def contraction_gflop(s: Shape) -> Dict[str, float]:
    """Per-row contraction Gflop in the order of the paper's Table 3 rows."""
    T, I, F = s.B * s.J, s.I, s.F
    att = 2.0 * s.B * s.H * s.J * s.K * s.P / 1e9
    qkv = 2.0 * T * 3 * I * I / 1e9
    out = 2.0 * T * I * I / 1e9
    lin = 2.0 * T * F * I / 1e9
    return {
        "fwd Q,K,V": qkv, "fwd QK^T": att, "fwd Gamma": att, "fwd Out": out,
        "fwd Linear1": lin, "fwd Linear2": lin,
        "bwd Linear2 dX": lin, "bwd Linear2 dW": lin, "bwd Linear1 dX": lin, "bwd Linear1 dW": lin,
        "bwd Out dX": out, "bwd Out dW": out, "bwd Gamma dX1": att, "bwd Gamma dX2": att,
        "bwd QK^T dX1": att, "bwd QK^T dX2": att, "bwd Q,K,V dX": qkv, "bwd Q,K,V dW": qkv,
    }


def mha(s: Shape, dtype: str, layout: str = "ibj", elements: bool = False) -> Dict[str, Work]:
    """Work of each labelled launch group of multi-head self-attention alone
    (fused Q/K/V projection, output bias in the output projection's
    epilogue), forward + backward: the encoder layer's attention launches,
    with the output-bias gradient as its own launch and the Q/K/V input
    gradient written without a residual."""
    w = encoder_layer(s, dtype, elements)
    es = 1 if elements else (4 if dtype == "f32" else 2)
    f4 = 1 if elements else 4
    T, I = s.B * s.J, s.I
    N = T * I
    keep = ("F1 qkv", "F2 qkt", "F3 softmax", "F2-3 qkt_softmax", "F2-4 qkt_softmax_gamma", "F4 gamma",
            "F5 out", "B11 out_dx", "B12 out_dw", "B13 gamma_dx1", "B14 gamma_dx2", "B15 softmax_bwd",
            "B13-15 gamma_dx1_softmax_bwd", "B13+15+16 score_bwd_dq", "B13-17 score_bwd_keys", "B16 qkt_dx1",
            "B17 qkt_dx2",
            "B18 qkv_dx", "B19 qkv_dw", "B20 qkv_bias_grad")
    out = {k: w[k] for k in keep}
    f5 = w["F5 out"]
    out["F5 out"] = Work(f5.flop, f5.bytes + I * es, f5.bound)
    b18 = w["B18 qkv_dx"]
    out["B18 qkv_dx"] = Work(b18.flop, b18.bytes - N * es, b18.bound)
    out["B10 out_bias_grad"] = Work(0.0, float(N * es + I * f4), "hbm")
    return out


def unfused_table3(s: Shape, act_dropout: bool = False):
    """The layer's operators one by one, as the paper's Table 3 lists them
    (each its own kernel: every input read, every output written, dropout
    masks stored and read back as tensors of their own), with input and
    output element counts derived from the shapes.  The activation is the
    workload's; act_dropout adds the dropout after it (the paper's fourth).
    Returns [(row, inputs, outputs)]."""
    T, I, F, H, P = s.B * s.J, s.I, s.F, s.H, s.P
    N, S, Fh, I2 = T * I, s.B * s.H * s.J * s.K, T * F, I * I
    r = [("Q, K, V", N + 3 * I2, 3 * N), ("Input bias", 3 * N + 3 * I, 3 * N), ("QK^T", 2 * N, S),
         ("Scaled softmax", S, 3 * S), ("Gamma", S + N, N), ("Out", N + I2, N)]
    ln_block = lambda: [("Bias", N + I, N), ("Dropout", N, 2 * N), ("Residual", 2 * N, N), ("LayerNorm", N + 2 * I, N)]
    r += ln_block()
    r += [("Linear", N + I * F, Fh), ("Bias", Fh + F, Fh), ("Activation", Fh, Fh)]
    if act_dropout:
        r += [("Dropout", Fh, 2 * Fh)]
    r += [("Linear", Fh + I * F, N)]
    r += ln_block()
    # backward
    # (LayerNorm dX reads dY, x_hat, its scale and the per-token statistics)
    r += [("LayerNorm dW", 2 * N, 2 * I), ("LayerNorm dX", 2 * N + I + 2 * T, N), ("Dropout dX", 2 * N, N),
          ("Linear+Bias dX", N + I * F, Fh), ("Linear dW", N + Fh, I * F), ("Bias dW", N, I)]
    if act_dropout:
        r += [("Dropout dX", 2 * Fh, Fh)]
    r += [("Activation dX", 2 * Fh, Fh), ("Bias dW", Fh, F), ("Linear+Bias dX", Fh + I * F, N),
          ("Linear dW", Fh + N, I * F), ("Residual", 2 * N, N), ("LayerNorm dW", 2 * N, 2 * I),
          ("LayerNorm dX", 2 * N + I + 2 * T, N), ("Dropout dX", 2 * N, N), ("Output bias dW", N, I),
          ("Out dX", N + I2, N), ("Out dW", 2 * N, I2), ("Gamma dX1", 2 * N, S), ("Gamma dX2", S + N, N),
          ("Scaled softmax dX", 3 * S, S), ("QK^T dX1", S + N, N), ("QK^T dX2", S + N, N),
          ("Q, K, V dX", 3 * N + 3 * I2, N), ("Q, K, V dW", 4 * N, 3 * I2), ("Input bias dW", 3 * N, 3 * I),
          ("Residual", 2 * N, N)]
    return r


def data_movement(s: Shape, dtype: str, path: str = "scores_next", act_dropout: bool = False,
                  epilogue=(), folded: bool = False) -> Dict[str, float]:
    """The data-movement reduction of the fused layer against the operators
    one by one (the analogue of the paper's figure, from its Table 3 I/O
    columns): elements moved per forward + backward step, both ways."""
    unf = sum(i + o for _, i, o in unfused_table3(s, act_dropout))
    w = encoder_layer(s, dtype, elements=True)
    fused = sum(x.bytes for x in path_groups(w, path, epilogue, folded).values())
    if folded:
        # the weight-gradient launch also writes the three bias gradients
        fused += 3 * s.I
    return {"unfused_Melem": round(unf / 1e6, 2), "fused_Melem": round(fused / 1e6, 2),
            "reduction": round(1.0 - fused / unf, 4)}
