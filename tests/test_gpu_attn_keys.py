"""The key-block attention backward (one launch from d(gamma) to dQ, dK, dV
over blocks of 128 or 256 keys; dQ partial sums of several key blocks per
head added by a second launch) against the oracle, at every block layout
it takes: 8 waves on 256 keys x 32 query rows (KG 8) or 128 keys x 64 rows
(KG 4), with one or several key blocks per head, ragged query lengths,
causal masking and no dropout; plus the other launch groupings, which
re-form alpha from the saved P, on the same shapes."""
import pytest
import torch

from paper_2007_00072_amd.inputs import WORKLOADS, Shape
from test_gpu_layer import check_encoder, check_mha, run_encoder, small

pytestmark = pytest.mark.gpu


def mha(dtype, p_attn=0.1, **shape):
    return WORKLOADS["mha_large_f16"].with_(shape=Shape(**shape), dtype=dtype, layout="bji", p_attn=p_attn)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("shape", [
    # KG 4, two key blocks per head (partials), 64-row steps, the second ragged
    dict(B=1, J=72, K=256, H=2, P=64, W=64, I=128),
    # KG 4, one key block per head, one partial step of 24 rows
    dict(B=3, J=24, K=128, H=2, P=64, W=64, I=128),
    # KG 8 (B*H*K/256 >= 192), one key block per head, 40 query rows
    dict(B=12, J=40, K=256, H=16, P=64, W=64, I=1024),
    # KG 8, two key blocks per head, 40 query rows
    dict(B=6, J=40, K=512, H=16, P=64, W=64, I=1024),
])
def test_mha_key_blocks(dtype, shape):
    check_mha(mha(dtype, **shape), self_attention=False)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_mha_key_blocks_no_dropout(dtype):
    check_mha(mha(dtype, p_attn=0.0, B=2, J=56, K=256, H=3, P=64, W=64, I=192), self_attention=False)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_mha_key_blocks_fused_kv(dtype):
    # keys and values from one memory tensor ([Wk Wv] stacked), 3 key blocks
    check_mha(mha(dtype, B=2, J=96, K=384, H=4, P=64, W=64, I=256), self_attention=2)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
@pytest.mark.parametrize("J", [128, 256])
def test_encoder_key_blocks(name, J):
    wl = small(name, B=2, J=J, K=J, H=4, P=64, W=64, I=256, F=512).with_(p_attn=0.1)
    check_encoder(wl, layer=2)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_key_blocks_causal(name):
    # key blocks past every query of a step see only zero probabilities
    wl = small(name, B=2, J=256, K=256, H=2, P=64, W=64, I=128, F=256).with_(p_attn=0.1)
    check_encoder(wl, layer=1, causal=True)


@pytest.mark.parametrize("path", [1, 2, 3])
@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_encoder_groupings_on_key_block_shape(name, path):
    # separate launches (1) and scores on chip (2) re-form alpha from P for
    # the Gamma dX2 contraction; 3 is the key-block backward
    from paper_2007_00072_amd import lib
    wl = small(name, B=2, J=128, K=128, H=4, P=64, W=64, I=256, F=512).with_(p_attn=0.2)
    check_encoder(wl, layer=1, plan=lib.Plan((), attn_path=path))


def test_key_blocks_deterministic():
    wl = small("bert_large_f16", B=2, J=256, K=256, H=4, P=64, W=64, I=256, F=512).with_(p_attn=0.1)
    L1, _, _, _, y1, dx1 = run_encoder(wl)
    g1 = {n: t.clone() for n, t in L1.grads.items()}
    L2, _, _, _, y2, dx2 = run_encoder(wl)
    assert torch.equal(y1, y2) and torch.equal(dx1, dx2)
    for n in g1:
        assert torch.equal(g1[n], L2.grads[n]), n
