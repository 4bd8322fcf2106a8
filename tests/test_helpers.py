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
