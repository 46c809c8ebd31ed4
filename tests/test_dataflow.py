"""The work model used for roofline reporting, pinned to the paper's
Table 3 contraction flop counts (tests/golden/table3_contraction_gflop.json)."""
import json
import os

import pytest

from paper_2007_00072_amd import dataflow
from paper_2007_00072_amd.inputs import WORKLOADS

GOLD = os.path.join(os.path.dirname(__file__), "golden", "table3_contraction_gflop.json")


def test_contraction_gflop_matches_table3():
    gold = json.load(open(GOLD))
    got = dataflow.contraction_gflop(WORKLOADS["bert_large_f16"].shape)
    for k, v in gold["rows"].items():
        assert got[k] == pytest.approx(v, abs=6e-4), k
    assert sum(got.values()) == pytest.approx(gold["total_tensor_contractions"], abs=2e-3)


def test_layer_model_flops_consistent():
    s = WORKLOADS["bert_large_f16"].shape
    w = dataflow.encoder_layer(s, "f16")
    table3 = sum(dataflow.contraction_gflop(s).values())
    for path in dataflow.PATHS:
        groups = dataflow.path_groups(w, path)
        assert sum(x.flop for x in groups.values()) / 1e9 == pytest.approx(table3, rel=1e-12), path
    assert "F4 gamma" in dataflow.path_groups(w, "scores")
    assert "F4 gamma" not in dataflow.path_groups(w, "scores_next")
    assert "B14 gamma_dx2" not in dataflow.path_groups(w, "keys") and "B17 qkt_dx2" not in dataflow.path_groups(w, "keys")
    # the key-block backward reads P once and writes no score-sized tensor
    N, S2 = s.B * s.J * s.I, s.B * s.H * s.J * s.K
    assert w["B13-17 score_bwd_keys"].bytes == (9 * N + S2) * 2
    for k, v in dataflow.PAIRED.items():
        assert w[k].flop == sum(w[p].flop for p in v) and w[k].bytes == sum(w[p].bytes for p in v)
        assert all(p not in dataflow.path_groups(w, "scores_next") for p in v)
    for k, v in dataflow.REPLACES.items():
        assert w[k].flop == sum(w[p].flop for p in v)
        assert w[k].cls == "fused"
        # a fused group moves less than the groups it stands in for
        assert w[k].bytes < sum(w[p].bytes for p in v)
    # the projection / feed-forward contractions are MFMA-bound, attention and fused ops HBM-bound
    assert w["F7 linear1"].bound == "mfma" and w["F1 qkv"].bound == "mfma"
    assert w["F2 qkt"].bound == "hbm" and w["F3 softmax"].bound == "hbm"
    # fused-operator algorithmic bytes: softmax fwd moves 3 S elements
    S = s.B * s.H * s.J * s.K
    assert w["F3 softmax"].bytes == 3 * S * 2


def test_unfused_accounting_matches_table3_io():
    # the operator-by-operator accounting behind the data-movement figure,
    # pinned to the paper's printed Input / Output cells (Table 3) for the
    # paper's own layer (ReLU with the fourth dropout)
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "table3_io.json")))
    rows = dataflow.unfused_table3(WORKLOADS["bert_large_f16"].shape, act_dropout=True)
    want = gold["forward"] + gold["backward"]
    assert [r[0] for r in rows] == [w[0] for w in want]
    checked = 0
    for (name, i, o), (_, wi, wo) in zip(rows, want):
        for got, ref in ((i, wi), (o, wo)):
            if ref is not None:
                assert round(got / 1e6, 2) == pytest.approx(ref, abs=0.011), (name, got / 1e6, ref)
                checked += 1
    assert checked >= 50


def test_data_movement_reduction_positive():
    s = WORKLOADS["bert_large_f16"].shape
    d = dataflow.data_movement(s, "f16")
    assert 0 < d["fused_Melem"] < d["unfused_Melem"] and 0 < d["reduction"] < 1
    # the transposed dO copy is overhead, not algorithmic traffic
    w = dataflow.encoder_layer(s, "f16")
    assert w["B1-2 ln2_bwd"].overhead == s.B * s.J * s.I * 2


def test_epilogue_and_folded_groups():
    # Linear 1 with bias + activation in its epilogue: the contraction's flop,
    # H not read back; the folded input-bias gradient leaves its launch out
    s = WORKLOADS["bert_large_f16"].shape
    w = dataflow.encoder_layer(s, "f16")
    T, F = s.B * s.J, s.F
    # H is not read back after Linear 1; dA is neither written nor read
    saved = {"F7+8 linear1_bias_act": T * F * 2, "B3+5 linear2_dx_act_bwd": 2 * T * F * 2}
    for k, parts in dataflow.EPILOGUE.items():
        assert w[k].flop == sum(w[p].flop for p in parts)
        assert w[k].bytes == sum(w[p].bytes for p in parts) - saved[k]
    g = dataflow.path_groups(w, "keys", epilogue=True, folded=True)
    assert "F7+8 linear1_bias_act" in g and "F7 linear1" not in g and "F8 bias_act" not in g
    assert "B3+5 linear2_dx_act_bwd" in g and "B5 act_bwd" not in g
    assert "B20 qkv_bias_grad" not in g
    g0 = dataflow.path_groups(w, "keys")
    assert "F7+8 linear1_bias_act" not in g0 and "F8 bias_act" in g0 and "B20 qkv_bias_grad" in g0
    g1 = dataflow.path_groups(w, "keys", epilogue={"F7+8 linear1_bias_act"})
    assert "F7+8 linear1_bias_act" in g1 and "B5 act_bwd" in g1 and "B3+5 linear2_dx_act_bwd" not in g1
    assert sum(x.flop for x in g.values()) == sum(x.flop for x in g0.values())
    d0 = dataflow.data_movement(s, "f16", "keys")
    d1 = dataflow.data_movement(s, "f16", "keys", epilogue=True, folded=True)
    # H (T*F) read once less, dA (T*F) neither written nor read, dQKV
    # (3*T*I) read once less; the bias gradients (3*I) move with the pair
    assert (d0["fused_Melem"] - d1["fused_Melem"]) * 1e6 == pytest.approx(3 * T * F + 3 * T * s.I - 3 * s.I,
                                                                          abs=1e4)
