"""The parity bar's per-element bound (tests/_util.py) on hand-computed
cases: units of the storage type at max(|ref|, scale), never below 2e-2."""
import numpy as np

from _util import element_bound, encoder_dx_scale, ulp


def test_ulp_spacing():
    assert ulp(np.array([0.82]), "bf16")[0] == 2.0 ** -8      # [0.5, 1): 8 significant bits
    assert ulp(np.array([2.17]), "bf16")[0] == 2.0 ** -6
    assert ulp(np.array([0.82]), "f16")[0] == 2.0 ** -11
    assert ulp(np.array([100.0]), "f16")[0] == 2.0 ** -4


def test_element_bound_takes_the_largest_term():
    ref = np.array([0.82, 0.82, 3.0, 100.0])
    assert np.array_equal(element_bound(ref, "bf16"), [0.02, 0.02, 4 * 2.0 ** -6, 4 * 2.0 ** -1])
    scale = np.array([0.0, 2.17, 0.0, 0.0])
    assert np.array_equal(element_bound(ref, "bf16", scale), [0.02, 4 * 2.0 ** -6, 4 * 2.0 ** -6, 4 * 2.0 ** -1])


def test_encoder_dx_scale_layout():
    # [I,B,J] oracle intermediates -> [B,J,I]; rstd per token, g1 per column
    I, B, J = 3, 2, 4
    inter = {"dY1f": np.zeros((I, B, J)), "dS2": np.zeros((I, B, J)), "dXa": np.zeros((I, B, J))}
    inter["dS2"][2, 1, 3] = -2.0
    inter["dY1f"][0, 0, 1] = 1.5
    inter["dXa"][1, 1, 0] = 0.25
    cache = {"rstd1": np.full((B, J), 2.0)}
    prm = {"g1": np.array([1.0, 1.0, 0.5])}
    s = encoder_dx_scale(cache, inter, prm)
    assert s.shape == (B, J, I)
    assert s[1, 3, 2] == 2.0 and s[0, 1, 0] == 3.0 and s[1, 0, 1] == 0.25
    assert np.count_nonzero(s) == 3
