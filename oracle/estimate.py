"""Latency and memory estimation from fingerprints -- test infrastructure only.

Latency (Sec. 5.3).  A request's latency is the time to first token plus the output
length times the time per output token (Eq. 1):
    latency = TTFT + output_length * TPOT
L2 profiles two fingerprints, with n_a and n_b hidden layers, each under two output
lengths.  For each fingerprint the two latencies give a 2x2 system of Eq. 1 in
(TTFT, TPOT).  Both are split into the hidden layers' share and the other blocks'
share (Eq. 2 and Eq. 3):
    TTFT = num_layers * TTFT_layer + TTFT_other
    TPOT = num_layers * TPOT_layer + TPOT_other
and the four fingerprint values give a 4x4 system in (TTFT_layer, TPOT_layer,
TTFT_other, TPOT_other), from which TTFT and TPOT follow for any layer count.
Here a request of output length n is the prefill (which yields the first token)
followed by n decode steps.

Memory (Sec. 5.2, M2).  The footprint of a fingerprint grows linearly with its number
of hidden layers (Sec. 5, Fig. 7), so the footprints of two fingerprints extrapolate
linearly to any layer count.  (M2 then solves a 3x3 system over three parallelism
configurations; those need several GPUs and are not part of this build.)

Pins (tests/test_oracle_estimate.py): recovery of known parameters from latencies and
footprints built exactly from them, predictions at the observed points, singular
designs rejected.
"""
import numpy as np


def fit_ttft_tpot(n_out, lat):
    """Eq. 1 at two output lengths: solve [[1, n1], [1, n2]] (TTFT, TPOT) = (lat1, lat2)."""
    A = np.array([[1.0, float(n_out[0])], [1.0, float(n_out[1])]])
    return tuple(np.linalg.solve(A, np.asarray(lat, dtype=np.float64)))


def fit_l2(layers, n_out, lat):
    """L2: fingerprints with layers = (n_a, n_b) hidden layers, each timed at the output
    lengths n_out = (o1, o2); lat[i][j] is fingerprint i's latency at length j.  Returns
    dict(ttft_layer, tpot_layer, ttft_other, tpot_other)."""
    (ta, pa) = fit_ttft_tpot(n_out, lat[0])
    (tb, pb) = fit_ttft_tpot(n_out, lat[1])
    na, nb = float(layers[0]), float(layers[1])
    # unknowns (TTFT_layer, TPOT_layer, TTFT_other, TPOT_other); rows Eq. 2 then Eq. 3
    A = np.array([[na, 0.0, 1.0, 0.0],
                  [nb, 0.0, 1.0, 0.0],
                  [0.0, na, 0.0, 1.0],
                  [0.0, nb, 0.0, 1.0]])
    x = np.linalg.solve(A, np.array([ta, tb, pa, pb]))
    return dict(ttft_layer=x[0], tpot_layer=x[1], ttft_other=x[2], tpot_other=x[3])


def predict(model, num_layers, n_out):
    """(TTFT, TPOT, latency) of a stack of num_layers hidden layers at output length n_out."""
    ttft = num_layers * model["ttft_layer"] + model["ttft_other"]
    tpot = num_layers * model["tpot_layer"] + model["tpot_other"]
    return ttft, tpot, ttft + n_out * tpot


def extrapolate_layers(layers, values, num_layers):
    """The straight line through (layers[0], values[0]) and (layers[1], values[1]),
    evaluated at num_layers."""
    (na, nb), (va, vb) = layers, values
    if na == nb:
        raise np.linalg.LinAlgError("two distinct layer counts are needed")
    slope = (vb - va) / (nb - na)
    return va + (num_layers - na) * slope
