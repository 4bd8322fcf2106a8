"""The parity helpers themselves: a non-finite result must never pass a closeness check."""
import numpy as np

from tests.helpers import allclose_report, bf16_layer_parity


def test_nan_and_inf_are_failures():
    ref = np.ones(8)
    for bad in (np.nan, np.inf, -np.inf):
        got = ref.copy()
        got[3] = bad
        rep = allclose_report(got, ref, atol=1e-2, rtol=1e-2)
        assert not rep["ok"] and rep["n_bad"] == 1
        assert not bf16_layer_parity(got, ref)["ok"]
    assert allclose_report(ref + 1e-3, ref, atol=1e-2, rtol=1e-2)["ok"]


def test_layer_gate_parts():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((64, 256))
    assert bf16_layer_parity(ref + 1e-3, ref)["ok"]
    # one row off by 5 % of its norm, everything else exact: the per-row bound catches it
    got = ref.copy()
    got[7] *= 1.05
    rep = bf16_layer_parity(got, ref, atol=1.0, rtol=1.0)
    assert not rep["ok"] and rep["row_norm_rel"] > 0.04 and rep["norm_rel"] < 1e-2
    # a single element far outside its bound (below the outlier fraction): the cap catches it
    got = ref.copy()
    got[3, 3] += 1.0
    rep = bf16_layer_parity(got, ref, outlier_frac=1e-3, row_norm_rel=1.0)
    assert not rep["ok"] and rep["n_bad"] == 1 and rep["worst_ratio"] > 4.0
    # the same element 2x over its bound is a tolerated outlier
    got = ref.copy()
    got[3, 3] += 2 * (2e-2 + 1e-2 * abs(ref[3, 3]))
    assert bf16_layer_parity(got, ref, outlier_frac=1e-3, row_norm_rel=1.0)["ok"]


def test_near_tie_window_is_capped():
    from tests.helpers import check_tokens, near_tie_window
    assert np.allclose(near_tie_window([0.001, 0.02, 0.3]), [0.002, 0.04, 0.05])
    z = np.array([[0.0, 1.0, 0.9], [0.0, 1.0, 0.99]])
    # row 0: margin 0.1 > capped window 0.05 although 2 x deviation (0.4) covers it
    gpu = z + np.array([[0.0, 0.0, 0.2], [0.0, 0.0, 0.0]])
    import pytest
    with pytest.raises(AssertionError):
        check_tokens([2, 1], z, gpu)
    assert check_tokens([1, 1], z, gpu) == 0
    assert check_tokens([1, 2], z, z + np.array([[0, 0, 0.0], [0, 0, 0.02]])) == 1
