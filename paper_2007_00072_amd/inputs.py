"""Seeded synthetic inputs for the encoder-layer workloads.

This module only draws numbers and names shapes.  It holds none of the
layer's arithmetic, so that both the HIP path and the CPU oracle can take
their inputs from it without sharing any computation.

Index letters follow the paper's problem statement (Fig. 1 caption):
P/W key/value projection size, H heads, I embedding size, B batch,
J query length, K key/value length; F is the feed-forward width (the paper
does not name it).  Parameter shapes follow the paper's einsum index order
(Fig. 1a): wq, wk [P,H,I]; wv, wo [W,H,I]; bq, bk [P,H]; bv [W,H]; bo [I];
the feed-forward weights are w1 [F,I] and w2 [I,F].

Every tensor is drawn in float64 from a CPU ``torch.Generator`` and then
rounded (round-to-nearest-even) to the storage dtype, so that the GPU and
the oracle consume identical bytes.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, Optional

import torch

DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

PARAM_NAMES = ("wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo",
               "g1", "be1", "w1", "b1", "w2", "b2", "g2", "be2")
MHA_PARAM_NAMES = ("wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo")


@dataclass(frozen=True)
class Shape:
    B: int
    J: int
    K: int
    H: int
    P: int
    W: int
    I: int
    F: int = 0

    @property
    def T(self) -> int:  # query tokens
        return self.B * self.J


@dataclass(frozen=True)
class Workload:
    """One workload: shapes, storage dtype, dropout rates and init recipe."""
    name: str
    kind: str               # "encoder" (full post-LN layer) or "mha" (attention only)
    shape: Shape
    dtype: str              # storage dtype: "f32", "f16", "bf16"
    layout: str             # activation layout: "bji" (token-major) or "ibj" (paper order)
    p_attn: float = 0.1     # dropout on attention probabilities
    p_attn_out: float = 0.1  # dropout on the attention-block output (before the residual)
    p_ffn_out: float = 0.1  # dropout on the feed-forward output (before the residual)
    seed: int = 0           # dropout seed
    n_layers: int = 1
    weight_std: float = 0.02
    bias_std: float = 0.0
    random_ln: bool = False  # gamma ~ 1+N(0,0.1), beta ~ N(0,0.1) instead of 1, 0
    input_seed: int = 1000

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads: a tiny fp32 layer, BERT-large multi-head attention,
# the BERT-large layer, the BERT-base layer at short sequences and large
# batch, and a 24-layer BERT-large stack.
WORKLOADS: Dict[str, Workload] = {
    "tiny_f32": Workload("tiny_f32", "encoder",
                         Shape(B=2, J=32, K=32, H=2, P=16, W=16, I=32, F=128),
                         "f32", "bji", bias_std=0.0, input_seed=1001),
    "mha_large_f16": Workload("mha_large_f16", "mha",
                              Shape(B=8, J=512, K=512, H=16, P=64, W=64, I=1024, F=0),
                              "f16", "ibj", p_attn_out=0.0, p_ffn_out=0.0,
                              bias_std=0.02, input_seed=1002),
    "bert_large_f16": Workload("bert_large_f16", "encoder",
                               Shape(B=8, J=512, K=512, H=16, P=64, W=64, I=1024, F=4096),
                               "f16", "bji", bias_std=0.02, input_seed=1003),
    "bert_base_bf16": Workload("bert_base_bf16", "encoder",
                               Shape(B=96, J=128, K=128, H=12, P=64, W=64, I=768, F=3072),
                               "bf16", "bji", bias_std=0.02, input_seed=1004),
    "bert_large_stack24_bf16": Workload("bert_large_stack24_bf16", "encoder",
                                        Shape(B=4, J=512, K=512, H=16, P=64, W=64, I=1024,
                                              F=4096),
                                        "bf16", "bji", bias_std=0.02, n_layers=24,
                                        input_seed=1005),
}


def _normal(gen: torch.Generator, shape, std: float, mean: float = 0.0) -> torch.Tensor:
    t = torch.empty(shape, dtype=torch.float64)
    t.normal_(mean=0.0, std=1.0, generator=gen)
    return t * std + mean


def _cast(t: torch.Tensor, dtype: str) -> torch.Tensor:
    return t.to(DTYPES[dtype]).contiguous()


def param_shapes(s: Shape, kind: str = "encoder") -> Dict[str, tuple]:
    shapes = {
        "wq": (s.P, s.H, s.I), "bq": (s.P, s.H),
        "wk": (s.P, s.H, s.I), "bk": (s.P, s.H),
        "wv": (s.W, s.H, s.I), "bv": (s.W, s.H),
        "wo": (s.W, s.H, s.I), "bo": (s.I,),
    }
    if kind == "encoder":
        shapes.update({
            "g1": (s.I,), "be1": (s.I,),
            "w1": (s.F, s.I), "b1": (s.F,),
            "w2": (s.I, s.F), "b2": (s.I,),
            "g2": (s.I,), "be2": (s.I,),
        })
    return shapes


def make_params(wl: Workload, layer: int = 0, seed: Optional[int] = None) -> Dict[str, torch.Tensor]:
    """Parameters of one layer in the storage dtype (CPU tensors)."""
    base = (wl.input_seed if seed is None else seed) * 1000 + 97 * layer
    out = {}
    for idx, (name, shp) in enumerate(param_shapes(wl.shape, wl.kind).items()):
        gen = torch.Generator().manual_seed(base + idx + 1)
        if name.startswith("w"):
            t = _normal(gen, shp, wl.weight_std)
        elif name in ("g1", "g2"):
            t = _normal(gen, shp, 0.1, 1.0) if wl.random_ln else torch.ones(shp, dtype=torch.float64)
        elif name in ("be1", "be2"):
            t = _normal(gen, shp, 0.1) if wl.random_ln else torch.zeros(shp, dtype=torch.float64)
        else:  # biases
            t = _normal(gen, shp, wl.bias_std) if wl.bias_std > 0 else torch.zeros(shp, dtype=torch.float64)
        out[name] = _cast(t, wl.dtype)
    return out


def activation_shape(s: Shape, layout: str, length: Optional[int] = None) -> tuple:
    L = s.J if length is None else length
    return (s.I, s.B, L) if layout == "ibj" else (s.B, L, s.I)


def make_activation(wl: Workload, stream: int, length: Optional[int] = None) -> torch.Tensor:
    """A N(0,1) activation in the workload's layout; `stream` picks the tensor
    (0: layer input x / query, 1: dY / dout, 2: key input, 3: value input)."""
    gen = torch.Generator().manual_seed(wl.input_seed * 7919 + 31 * stream + 5)
    t = _normal(gen, activation_shape(wl.shape, wl.layout, length), 1.0)
    return _cast(t, wl.dtype)


def make_tensor(shape, dtype: str, seed: int, std: float = 1.0, mean: float = 0.0) -> torch.Tensor:
    """A generic seeded N(mean, std) tensor in the storage dtype (for op-level tests)."""
    gen = torch.Generator().manual_seed(seed)
    return _cast(_normal(gen, shape, std, mean), dtype)

