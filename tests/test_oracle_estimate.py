"""Pins of the oracle's latency (Eq. 1-3) and memory (M2 layer extrapolation) estimators."""
import numpy as np
import pytest

from oracle.estimate import fit_ttft_tpot, fit_l2, predict, extrapolate_layers


def _lat(n_layers, n_out, p):
    ttft = n_layers * p["ttft_layer"] + p["ttft_other"]
    tpot = n_layers * p["tpot_layer"] + p["tpot_other"]
    return ttft + n_out * tpot


@pytest.mark.parametrize("layers,n_out", [((1, 2), (16, 64)), ((1, 4), (10, 100)), ((2, 3), (1, 2))])
def test_l2_recovers_the_parameters_latencies_were_built_from(layers, n_out):
    p = dict(ttft_layer=7.25, tpot_layer=0.5, ttft_other=3.0, tpot_other=0.125)   # exact binary values
    lat = [[_lat(n, o, p) for o in n_out] for n in layers]
    m = fit_l2(layers, n_out, lat)
    for k in p:
        assert abs(m[k] - p[k]) < 1e-12, k
    # predictions at the observed points give the observed latencies
    for i, n in enumerate(layers):
        for j, o in enumerate(n_out):
            assert abs(predict(m, n, o)[2] - lat[i][j]) < 1e-9
    # and at a layer count and length not observed
    ttft, tpot, total = predict(m, 80, 100)
    assert abs(ttft - (80 * 7.25 + 3.0)) < 1e-9 and abs(tpot - (80 * 0.5 + 0.125)) < 1e-9
    assert abs(total - (ttft + 100 * tpot)) < 1e-9


def test_eq1_two_by_two():
    ttft, tpot = fit_ttft_tpot((16, 64), (20.0 + 16 * 1.5, 20.0 + 64 * 1.5))
    assert abs(ttft - 20.0) < 1e-12 and abs(tpot - 1.5) < 1e-12


def test_singular_designs_are_rejected():
    with pytest.raises(np.linalg.LinAlgError):
        fit_ttft_tpot((32, 32), (1.0, 2.0))
    with pytest.raises(np.linalg.LinAlgError):
        fit_l2((2, 2), (16, 64), [[1.0, 2.0], [1.0, 2.0]])
    with pytest.raises(np.linalg.LinAlgError):
        extrapolate_layers((3, 3), (1.0, 2.0), 5)


def test_memory_extrapolation_is_linear_in_layers():
    # footprint = fixed part + per-layer part
    fixed, per = 1_234_567_936.0, 400_556_032.0
    m = lambda n: fixed + n * per
    assert extrapolate_layers((1, 2), (m(1), m(2)), 80) == m(80)
    assert extrapolate_layers((1, 2), (m(1), m(2)), 1) == m(1)
    assert extrapolate_layers((2, 4), (m(2), m(4)), 3) == m(3)
