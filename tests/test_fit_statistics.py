"""Fit statistics on the workload tensors against independently probed values.

The per-tensor base b, shift s and the fraction of weights that encode to zero were probed for
the 2048x2048 (0.02 t4), 2048->8192 (0.02 t4 + 1e-4 outliers) and 8192->28672 (0.015 t3)
workloads, drawn on the CPU as ``default_rng([config, 0, 0, 0]).standard_t`` with configs 1, 2
and 5 (probe: b = 2.094, 2.241, 2.904; s = 7, 7, 5; zeros 29.7 %, 19.5 %, 37.9 %). They pin the
whole fit (energy pruning of Sec. 3.2 Eq. 5, Eq. 3, Eq. 4) and the zero boundary of Eq. 1 on
realistic sizes: a wrong energy quantile, exponent or rounding would move them.
"""
import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

PROBE = {
    "linear_2048x2048": (2.094, 7, 0.297),
    "up_2048x8192_outliers": (2.241, 7, 0.195),
    "layer_8192x28672": (2.904, 5, 0.379),
}


def _draw(name):
    wl = inputs.WORKLOADS[name]
    lin = wl["layers"][0]
    return inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                    outlier_frac=wl["outlier_frac"])


def test_oracle_fit_and_encode_match_probe_2048x2048():
    w = _draw("linear_2048x2048")
    r = O.fit(w)
    b, s, zf = PROBE["linear_2048x2048"]
    assert abs(r.base - b) < 5e-4 and r.shift == s
    codes = O.encode(w, r.base, r.shift)
    assert abs(float(np.mean((codes & 7) == 0)) - zf) < 5e-4


@pytest.mark.parametrize("name", ["up_2048x8192_outliers", "layer_8192x28672"])
def test_library_fit_matches_probe(name):
    """The library fit (bit-exact with the oracle on these tensors elsewhere) on the larger
    workloads; the zero fraction is |w| < thresholds[0], the first rounding boundary of Eq. 1."""
    w = _draw(name)
    p = L.fit(w)
    b, s, zf = PROBE[name]
    assert abs(p.base - b) < 5e-4 and p.shift == s
    thr0 = np.float32(p.thresholds_array()[0])
    assert abs(np.count_nonzero(np.abs(w) < thr0) / w.size - zf) < 5e-4
