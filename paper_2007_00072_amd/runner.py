"""Device-buffer owners around the C ABI (allocation and marshalling only).

torch allocates device memory and supplies the stream; every computation
happens inside libdmtx.so.  Used by the tests, the smoke check and the
benchmark.
"""
from __future__ import annotations

from typing import Dict, Optional

import torch

from . import lib
from .inputs import Shape, Workload

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def desc_for(wl: Workload, layer: int = 0, **over) -> lib.LayerDesc:
    """Descriptor of a workload's layer; `plan=` names a lib.Plan."""
    kw = dict(layout=wl.layout, p_attn=wl.p_attn, p_attn_out=wl.p_attn_out, p_ffn_out=wl.p_ffn_out,
              seed=wl.seed, layer_id=layer, ln_eps=1e-12, self_attention=True)
    kw.update(over)
    return lib.make_desc(wl.shape, wl.dtype, **kw)


class EncoderLayer:
    """One encoder layer's device state: parameters, saved activations,
    workspace and fp32 gradients."""

    def __init__(self, desc: lib.LayerDesc, params: Dict[str, torch.Tensor], device="cuda",
                 workspace: Optional[torch.Tensor] = None):
        self.desc = desc
        self.device = torch.device(device)
        self.params = {n: t.to(self.device).contiguous() for n, t in params.items()}
        self.cparams = lib.make_params(self.params)
        self.saved_bytes, self.fwd_bytes, self.bwd_bytes = lib.encoder_layer_sizes(desc)
        self.saved = torch.empty(self.saved_bytes, dtype=torch.uint8, device=self.device)
        need = max(self.fwd_bytes, self.bwd_bytes)
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty(need, dtype=torch.uint8, device=self.device)
        self.ws = workspace
        self.grads = {n: torch.empty(t.shape, dtype=torch.float32, device=self.device)
                      for n, t in self.params.items()}
        self.cgrads = lib.make_grads(self.grads)

    def forward(self, x: torch.Tensor, y: Optional[torch.Tensor] = None) -> torch.Tensor:
        if y is None:
            y = torch.empty_like(x)
        lib.encoder_layer_fwd(self.desc, self.cparams, x, y, self.saved, self.ws, self.ws.numel())
        return y

    def backward(self, x: torch.Tensor, dy: torch.Tensor, dx: Optional[torch.Tensor] = None) -> torch.Tensor:
        if dx is None:
            dx = torch.empty_like(x)
        lib.encoder_layer_bwd(self.desc, self.cparams, x, self.saved, dy, dx, self.cgrads, self.ws,
                              self.ws.numel())
        return dx

    def saved_tensor(self, name: str, shape, dtype) -> torch.Tensor:
        off, nbytes = lib.saved_tensor_view(self.desc, name)
        return self.saved[off:off + nbytes].view(dtype).view(*shape)


class MultiHeadAttention:
    """Attention-only device state (multi-head attention of Fig. 1a)."""

    def __init__(self, desc: lib.LayerDesc, params: Dict[str, torch.Tensor], device="cuda"):
        self.desc = desc
        self.device = torch.device(device)
        self.params = {n: t.to(self.device).contiguous() for n, t in params.items()}
        self.cparams = lib.make_params(self.params)
        self.saved_bytes, self.fwd_bytes, self.bwd_bytes = lib.mha_sizes(desc)
        self.saved = torch.empty(self.saved_bytes, dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(max(self.fwd_bytes, self.bwd_bytes), dtype=torch.uint8, device=self.device)
        self.grads = {n: torch.empty(t.shape, dtype=torch.float32, device=self.device)
                      for n, t in self.params.items()}
        self.cgrads = lib.make_grads(self.grads)

    def forward(self, q, k=None, v=None, out=None):
        if out is None:
            out = torch.empty_like(q)
        lib.mha_fwd(self.desc, self.cparams, q, k, v, out, self.saved, self.ws, self.ws.numel())
        return out

    def backward(self, q, dout, k=None, v=None, dq=None, dk=None, dv=None):
        if dq is None:
            dq = torch.empty_like(q)
        if self.desc.self_attention != 1:
            dk = torch.empty_like(k) if dk is None else dk
        if self.desc.self_attention == 0:
            dv = torch.empty_like(v) if dv is None else dv
        lib.mha_bwd(self.desc, self.cparams, q, k, v, self.saved, dout, dq, dk, dv, self.cgrads, self.ws,
                    self.ws.numel())
        return dq, dk, dv
