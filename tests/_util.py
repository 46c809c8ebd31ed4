"""Shared helpers for the parity tests: tolerance checks and oracle wiring."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import layer as OL

# Parity bar.  Float activations and input gradients: max |err| <= 2e-2 and
# relative L2 <= 5e-3 for fp16 / bf16 storage, relative <= 1e-5 for fp32.
# Parameter gradients are float32 sums over all tokens with magnitudes well
# above 1, so their absolute bound scales with max(1, rms(reference)).
TOL = {
    "f16": dict(max_abs=2e-2, rel_l2=5e-3),
    "bf16": dict(max_abs=2e-2, rel_l2=5e-3),
    "f32": dict(max_abs=1e-5, rel_l2=1e-5),
}


def f64(t) -> np.ndarray:
    if hasattr(t, "detach"):
        return t.detach().float().cpu().double().numpy() if t.dtype.is_floating_point else t.detach().cpu().numpy()
    return np.asarray(t, dtype=np.float64)


def errors(got, ref):
    got = f64(got)
    ref = f64(ref)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = got - ref
    max_abs = float(np.abs(d).max()) if d.size else 0.0
    nrm = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(d)) / nrm if nrm > 0 else float(np.linalg.norm(d))
    return max_abs, rel, float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0, float(np.abs(ref).max()) if ref.size else 0.0


def ulp(x: np.ndarray, dtype: str) -> np.ndarray:
    """Spacing of the storage type at |x| (bf16: 8 significant bits, fp16: 11)."""
    bits, emin = {"bf16": (8, -126), "f16": (11, -14), "f32": (24, -126)}[dtype]
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** emin)))
    return 2.0 ** (e - (bits - 1))


def assert_close(name, got, ref, dtype, param_grad=False, scale=None, zero_ref=False):
    """Checks `got` against the oracle `ref` at the parity bar of `dtype`.

    fp16 / bf16: every element within 2e-2 * s * max(1, |ref|) and relative
    L2 <= 5e-3.  s = 1 for activations and input gradients, max(1, rms(ref))
    for float32 parameter gradients (sums over all tokens).  The max(1, |ref|)
    factor matters only for elements of magnitude above 1, where the storage
    type's own spacing grows with the value (a bf16 value of 4 has spacing
    0.031, so one last-bit rounding difference already exceeds 2e-2).
    fp32: max |err| <= 1e-5 * max(1, max |ref|) and relative L2 <= 1e-5.
    zero_ref: the exact value is zero (e.g. the key-bias gradient, which
    softmax's shift invariance makes vanish), so only rounding noise is
    compared: |err| <= max-abs bound * max(1, scale), with `scale` the rms
    of a comparable nonzero gradient (the query-bias gradient)."""
    max_abs, rel, rms, amax = errors(got, ref)
    t = TOL[dtype]
    g, r = f64(got), f64(ref)
    if zero_ref:
        bound = t["max_abs"] * max(1.0, scale or 1.0)
        assert max_abs <= bound, f"{name}: max_abs={max_abs:.3e} (bound {bound:.3e}, exact value 0)"
        return max_abs, rel
    if dtype == "f32":
        bound = t["max_abs"] * max(1.0, amax)
        ok_abs = max_abs <= bound
    else:
        s = max(1.0, rms if scale is None else scale) if param_grad else (1.0 if scale is None else max(1.0, scale))
        bound = t["max_abs"] * s
        elem = bound * np.maximum(1.0, np.abs(r)) if not param_grad else bound
        ok_abs = bool(np.all(np.abs(g - r) <= elem))
    msg = f"{name}: max_abs={max_abs:.3e} (bound {bound:.3e}) rel_l2={rel:.3e} (bound {t['rel_l2']:.1e})"
    assert ok_abs and rel <= t["rel_l2"], msg
    return max_abs, rel


def oracle_config(wl, layer=0, **over):
    s = wl.shape
    kw = dict(B=s.B, J=s.J, K=s.K, H=s.H, P=s.P, W=s.W, I=s.I, F=s.F, p_attn=wl.p_attn,
              p_attn_out=wl.p_attn_out, p_ffn_out=wl.p_ffn_out, seed=wl.seed, layer=layer,
              eps=1e-12, store_dtype=wl.dtype)
    kw.update(over)
    return OL.Config(**kw)


def params64(params):
    return {n: f64(t) for n, t in params.items()}


requires_gpu = pytest.mark.gpu
