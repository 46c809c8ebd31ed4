"""Configuration plans on the GPU: an installed plan changes the kernels and
launch grouping that run, results still match the oracle, and the tuner
(configuration selection) runs end to end."""
import json

import pytest
import torch

from paper_2007_00072_amd import lib, tune
from paper_2007_00072_amd.inputs import WORKLOADS, Shape
from test_gpu_layer import check_encoder, run_encoder, small

pytestmark = pytest.mark.gpu


def _launches(wl, plan=None):
    lib.dm_trace_enable(True)
    lib.plan_log(True)
    run_encoder(wl, plan=plan)
    recs = lib.plan_log_read()
    lib.plan_log(False)
    labels = [lab for lab, _, _ in lib.trace_records()]
    lib.dm_trace_enable(False)
    return recs, labels


def test_plan_entry_changes_the_kernel_and_keeps_parity():
    wl = small("bert_large_f16", B=2, J=96, K=96, H=4, P=64, W=64, I=256, F=512)
    recs, _ = _launches(wl)
    # Linear 1 (with bias + activation in its epilogue where its kernel allows)
    is_lin1 = lambda r: r.label.decode() in ("F7 linear1", "F7+8 linear1_bias_act")
    lin1 = next(r for r in recs if is_lin1(r))
    builtin = (lin1.tile_cfg, lin1.splits)
    want = 6 if builtin[0] != 6 else 2
    plan = lib.Plan([lib.ContractChoice(*lin1.key(), want, 1)], 0)
    recs2, _ = _launches(wl, plan)
    got = next(r for r in recs2 if is_lin1(r))
    assert (got.tile_cfg, got.splits) == (want, 1)
    # every other contraction kept its built-in choice
    for a, b in zip(recs, recs2):
        if not is_lin1(a):
            assert (a.tile_cfg, a.splits) == (b.tile_cfg, b.splits)
    check_encoder(wl, layer=1, plan=plan)


def test_plan_every_contraction_on_the_k_group_kernel():
    # every contraction of the layer that the lean kernels take runs on the
    # 128x128 kernel with two k groups (the residual epilogue of the Q/K/V
    # input gradient included); results still match the oracle
    wl = small("bert_large_f16", B=2, J=96, K=96, H=4, P=64, W=64, I=256, F=512)
    recs, _ = _launches(wl)
    plan = lib.Plan([lib.ContractChoice(*k, 16, 1) for k in {r.key() for r in recs}], 3)
    recs2, _ = _launches(wl, plan)
    assert sum(r.tile_cfg == 16 for r in recs2) >= 8
    assert any(r.tile_cfg == 16 and r.label.decode() == "B18 qkv_dx" for r in recs2)
    check_encoder(wl, layer=1, plan=plan)


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
def test_weight_gradients_share_one_launch(name):
    # the output-projection and Q/K/V weight gradients (both reduce over the
    # tokens) run as one launch of the lean 128x128 kernel; a plan entry
    # that gives one of them another kernel separates the launches again;
    # parity either way
    # (BERT-large widths: 192 + 64 tiles of 128 x 128, one per CU; 512
    # tokens, since bf16 parameter gradients summed over only 128 tokens sit
    # at the edge of the absolute bound whichever kernel computes them)
    wl = small(name, B=4, J=128, K=128, H=16, P=64, W=64, I=1024, F=1024)
    lab = "B12+19 out_dw+qkv_dw"
    recs, labels = _launches(wl)
    pair = [r for r in recs if r.label.decode() == lab]
    assert len(pair) == 2 and all((r.tile_cfg, r.splits) == (15, 1) for r in pair), pair
    assert labels.count(lab) == 1
    check_encoder(wl, layer=1)
    out_dw = next(r for r in pair if r.M == wl.shape.H * wl.shape.W)
    plan = lib.Plan([lib.ContractChoice(*out_dw.key(), 6, 1)], 0)
    recs2, labels2 = _launches(wl, plan)
    assert labels2.count(lab) == 2   # two launches under the one label
    assert any(r.label.decode() == lab and (r.tile_cfg, r.splits) == (6, 1) for r in recs2)
    check_encoder(wl, layer=1, plan=plan)
    # narrower layers (fewer tiles than 3/4 of the CUs) keep separate launches
    wl2 = small(name, B=2, J=128, K=128, H=4, P=64, W=64, I=256, F=1024)
    recs3, labels3 = _launches(wl2)
    assert labels3.count(lab) >= 2


@pytest.mark.parametrize("path,fwd,bwd", [
    (1, ["F2 qkt", "F3 softmax", "F4 gamma"], ["B13 gamma_dx1", "B15 softmax_bwd", "B16 qkt_dx1"]),
    (2, ["F2-3 qkt_softmax", "F4 gamma"], ["B13-15 gamma_dx1_softmax_bwd", "B16 qkt_dx1"]),
    (3, ["F2-4 qkt_softmax_gamma"], ["B13+15+16 score_bwd_dq"]),
])
def test_attention_groupings(path, fwd, bwd):
    wl = small("bert_base_bf16", B=2, J=64, K=64, H=4, P=64, W=64, I=256, F=512).with_(p_attn=0.1)
    plan = lib.Plan([], path)
    _, labels = _launches(wl, plan)
    for lab in fwd + bwd:
        assert lab in labels, (lab, labels)
    check_encoder(wl, layer=2, plan=plan)


def test_tuner_end_to_end(tmp_path):
    res = tune.tune("bert_large_f16", reps=1, log=lambda s: None,
                    shape=Shape(B=2, J=128, K=128, H=4, P=64, W=64, I=256, F=1024),
                    tile_cfgs=(8, 13, 15), splits=(1, 2))
    assert res["attn_path"] in (1, 2, 3)
    assert res["entries"] and all(0 <= e["tile_cfg"] <= 25 for e in res["entries"])
    for name in ("forward", "backward"):
        assert res["passes"][name]["predicted_ms"] > 0
    path = tmp_path / "plan.json"
    path.write_text(json.dumps(res))
    plan, cplan = tune.load_plan(str(path))
    assert plan["attn_path"] == res["attn_path"] == cplan.attn_path
    assert set(plan["layout"]) == {"ln_bwd_form", "dO_transposed", "dH_transposed", "ln_lanes"}
    assert len(res["layout_table"]) >= 2
    wl = small("bert_large_f16", B=2, J=128, K=128, H=4, P=64, W=64, I=256, F=1024)
    check_encoder(wl, layer=0, plan=cplan, qkv_fusion=int(plan["qkv_fusion"]))


def test_saved_bert_base_plan_keeps_parity():
    # the tuned BERT-base plan (long-k weight gradients split four ways on
    # the 4-wave 256x256 kernel, several contractions on other tiles) at
    # its full size: every planned contraction runs its entry's choice
    import os
    from paper_2007_00072_amd.inputs import WORKLOADS
    path = os.path.join(os.path.dirname(tune.__file__), "plans", "bert_base_bf16.json")
    plan, cplan = tune.load_plan(path)
    recs, _ = _launches(WORKLOADS["bert_base_bf16"], cplan)
    want = {(e["M"], e["N"], e["K"], e["batch"], e["dtype"], e["a_kcontig"], e["b_kcontig"]): (e["tile_cfg"], e["splits"])
            for e in plan["entries"]}
    planned = [r for r in recs if r.key() in want]
    assert planned and all((r.tile_cfg, r.splits) == want[r.key()] for r in planned)
    assert any(r.splits > 1 for r in planned)
    check_encoder(WORKLOADS["bert_base_bf16"], plan=cplan, qkv_fusion=int(plan.get("qkv_fusion", 0)))


@pytest.mark.parametrize("name", ["bert_large_f16", "bert_base_bf16"])
@pytest.mark.parametrize("layout", [
    {"dO_transposed": 0},
    {"dH_transposed": 1},
    {"ln_bwd_form": 1},
    {"ln_bwd_form": 1, "ln_lanes": 32},
    {"ln_lanes": 16, "dH_transposed": 1, "dO_transposed": 1},
])
def test_layout_choices_keep_parity(name, layout):
    # the fused operators' layout and reduction choices (transposed copies
    # for the weight gradients, LayerNorm backward form, lanes per row):
    # the contraction reading a transposed copy changes operand layout,
    # results match the oracle at every choice (144 tokens: ragged tiles)
    wl = small(name, B=2, J=72, K=72, H=6, P=64, W=64, I=384, F=768)
    plan = lib.Plan([], 0, layout)
    recs, _ = _launches(wl, plan)
    by = {r.label.decode(): r for r in recs}
    dot = layout.get("dO_transposed", -1) != 0 and layout.get("ln_bwd_form", -1) != 1
    assert by["B4 linear2_dw"].a_kcontig == (1 if dot else 0)
    assert by["B7 linear1_dw"].a_kcontig == (1 if layout.get("dH_transposed") == 1 else 0)
    check_encoder(wl, layer=1, plan=plan)


def test_layout_choice_validation():
    with pytest.raises(lib.DmError):
        lib.Plan([], 0, {"ln_lanes": 24})
    with pytest.raises(lib.DmError):
        lib.Plan([], 0, {"ln_bwd_form": 3})
    with pytest.raises(lib.DmError):
        lib.Plan([], 0, {"dH_transposed": 2})


@pytest.mark.parametrize("name,act,p_act", [("bert_large_f16", "gelu", 0.0), ("bert_base_bf16", "relu", 0.1)])
def test_epilogue_operators_change_no_value(name, act, p_act):
    # Linear 1 with bias + activation (+ dropout) in its epilogue and
    # Linear-2 dX with the activation backward in its epilogue, against the
    # same two contractions moved by a plan entry to the lean 4-wave 128x128
    # kernel (same MFMA instruction and k order, no epilogue operator), so
    # that the operators run as launches of their own: H, A, y, dx and every
    # weight gradient are bit for bit the same; db1, a column sum, differs
    # only in its summation order
    wl = small(name, B=2, J=128, K=128, H=4, P=64, W=64, I=256, F=1024)

    def run(plan=None):
        lib.dm_trace_enable(True)
        lib.plan_log(True)
        L, _, _, _, y, dx = run_encoder(wl, act=act, p_ffn_act=p_act, plan=plan)
        recs = lib.plan_log_read()
        lib.plan_log(False)
        labels = [lab for lab, _, _ in lib.trace_records()]
        lib.dm_trace_enable(False)
        T, F = wl.shape.B * wl.shape.J, wl.shape.F
        tdt = y.dtype
        saved = {n: L.saved_tensor(n, (T, F), tdt).clone() for n in ("h", "a")}
        return L, y, dx, recs, labels, saved

    L0, y0, dx0, recs, labels, s0 = run()
    assert "F7+8 linear1_bias_act" in labels and "B3+5 linear2_dx_act_bwd" in labels
    keys = {r.key() for r in recs if r.label.decode() in ("F7+8 linear1_bias_act", "B3+5 linear2_dx_act_bwd")}
    assert len(keys) == 2
    plan = lib.Plan([lib.ContractChoice(*k, 18, 1) for k in keys], 0)
    L1, y1, dx1, _, labels1, s1 = run(plan)
    assert {"F7 linear1", "F8 bias_act", "B3 linear2_dx", "B5 act_bwd"} <= set(labels1)
    for n in ("h", "a"):
        assert torch.equal(s0[n], s1[n]), n
    assert torch.equal(y0, y1) and torch.equal(dx0, dx1)
    for n, g in L0.grads.items():
        if n == "b1":
            assert torch.allclose(g, L1.grads[n], rtol=1e-5, atol=1e-5 * float(g.abs().max()))
        else:
            assert torch.equal(g, L1.grads[n]), n


@pytest.mark.parametrize("name,act,p_act", [("bert_large_f16", "gelu", 0.0), ("bert_base_bf16", "relu", 0.1)])
def test_bias_act_epilogue_on_the_192_wide_tile(name, act, p_act):
    # Linear 1 with its bias + activation epilogue moved by a plan entry to
    # the 256x192 ping-pong kernel (4 wave rows, ragged last tile column at
    # F = 1024): the same MFMA instruction and k order, the same epilogue
    # arithmetic, so H, A, y, dx and every weight gradient are bit for bit
    # those of the built-in kernel
    wl = small(name, B=2, J=128, K=128, H=4, P=64, W=64, I=256, F=1024)

    def run(plan=None):
        lib.dm_trace_enable(True)
        lib.plan_log(True)
        L, _, _, _, y, dx = run_encoder(wl, act=act, p_ffn_act=p_act, plan=plan)
        recs = lib.plan_log_read()
        lib.plan_log(False)
        labels = [lab for lab, _, _ in lib.trace_records()]
        lib.dm_trace_enable(False)
        T, F = wl.shape.B * wl.shape.J, wl.shape.F
        saved = {n: L.saved_tensor(n, (T, F), y.dtype).clone() for n in ("h", "a")}
        return L, y, dx, recs, labels, saved

    L0, y0, dx0, recs, labels, s0 = run()
    keys = [r.key() for r in recs if r.label.decode() == "F7+8 linear1_bias_act"]
    assert len(keys) == 1
    L1, y1, dx1, recs1, labels1, s1 = run(lib.Plan([lib.ContractChoice(*keys[0], 25, 1)], 0))
    assert "F7+8 linear1_bias_act" in labels1
    assert [r.tile_cfg for r in recs1 if r.label.decode() == "F7+8 linear1_bias_act"] == [25]
    for n in ("h", "a"):
        assert torch.equal(s0[n], s1[n]), n
    assert torch.equal(y0, y1) and torch.equal(dx0, dx1)
    for n, g in L0.grads.items():
        assert torch.equal(g, L1.grads[n]), n
