"""Pins of the asymmetric linear baseline oracle (Sec. 2, Quant(s, z, x)) and of the quality
measures, against facts that do not come from the oracle itself: exact nearest-level search on
rationals, the end points of the range, the textbook SQNR of a uniform quantizer on uniformly
distributed data, and the host library's fit, which is an independent implementation."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import logbq_oracle as O
from oracle import uniform_oracle as U
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L


def _tensor(n, k, seed, nu=4, scale=0.02, outl=0.0):
    return np.asarray(inputs.student_t_weights(n, k, nu, scale, seed=seed, outlier_frac=outl))


def test_fit_definition_small():
    # min -1, max 2: s = 3 / 15 = 0.2, z = round(-1 / 0.2) = -5; code q stands for 0.2 (q - 5).
    w = np.array([-1.0, 0.0, 0.5, 2.0], dtype=np.float32)
    f = U.uniform_fit(w)
    assert f.scale == 3.0 / 15 and f.zero == -5
    lv = U.uniform_levels(f.scale, f.zero)
    assert lv[0] == np.float32(-1.0) and lv[5] == np.float32(0.0) and lv[15] == np.float32(2.0)
    assert U.uniform_encode(w, f.scale, f.zero).tolist() == [0, 5, 8, 15]   # 0.5 / 0.2 = 2.5 -> 3


def test_nearest_level_exact():
    """Every code is the level nearest to x (ties up), decided on exact rationals."""
    rng = np.random.default_rng(5)
    w = (rng.standard_t(3, 4000) * 0.03).astype(np.float32)
    f = U.uniform_fit(w)
    codes = U.uniform_encode(w, f.scale, f.zero)
    s = Fraction(f.scale)
    for x, c in zip(w.tolist(), codes.tolist()):
        v = Fraction(x) / s                           # exact x / s
        q = math.floor(v + Fraction(1, 2)) - f.zero   # nearest integer, ties up
        q = min(max(q, 0), 15)
        if abs(v - (math.floor(v) + Fraction(1, 2))) > Fraction(1, 10**9):
            assert c == q, (x, c, q)


def test_range_end_points():
    for seed in range(4):
        w = _tensor(64, 96, [21, seed, 0, 0], outl=1e-3)
        f = U.uniform_fit(w)
        c = U.uniform_encode(np.array([w.min(), w.max()], dtype=np.float32), f.scale, f.zero)
        assert c[0] == 0 and c[1] == 15
        lv = U.uniform_levels(f.scale, f.zero)
        assert abs(lv[0] - w.min()) <= f.scale / 2 and abs(lv[15] - w.max()) <= f.scale / 2


def test_idempotent():
    w = _tensor(50, 64, [21, 9, 0, 0])
    f = U.uniform_fit(w)
    c = U.uniform_encode(w, f.scale, f.zero)
    lv = U.uniform_levels(f.scale, f.zero)
    assert np.array_equal(U.uniform_encode(U.uniform_dequantize(c, lv), f.scale, f.zero), c)


def test_thresholds_reproduce_codes():
    w = _tensor(100, 64, [21, 3, 0, 0], outl=1e-3)
    f = U.uniform_fit(w)
    thr = U.uniform_thresholds(f.scale, f.zero)
    assert np.all(np.diff(thr) >= 0)
    probe = np.concatenate([w.ravel(), thr, np.nextafter(thr, np.float32(-np.inf)),
                            np.nextafter(thr, np.float32(np.inf))]).astype(np.float32)
    by_thr = (probe[:, None] >= thr[None, :]).sum(1)
    assert np.array_equal(by_thr, U.uniform_encode(probe, f.scale, f.zero))


def test_sqnr_textbook_uniform_data():
    """Uniform data over the range: error uniform in [-s/2, s/2], SQNR = 10 log10(15^2)."""
    rng = np.random.default_rng(8)
    w = rng.uniform(-1.0, 1.0, 2_000_000).astype(np.float32)
    f = U.uniform_fit(w)
    wh = U.uniform_dequantize(U.uniform_encode(w, f.scale, f.zero), U.uniform_levels(f.scale, f.zero))
    assert abs(U.sqnr_db(w, wh) - 20 * math.log10(15)) < 0.05


def test_quality_measures_basics():
    w = np.array([3.0, 4.0], dtype=np.float32)
    assert U.sqnr_db(w, np.zeros(2)) == 0.0
    assert abs(U.sqnr_db(w, w.astype(np.float64) * 0.9) - 20.0) < 1e-9   # error 0.1 w: 10 log10(100)
    assert abs(U.relative_error(np.array([3.0, 5.0]), np.array([3.0, 4.0])) - 0.2) < 1e-15


@pytest.mark.parametrize("nu,scale,outl", [(4, 0.02, 0.0), (4, 0.02, 1e-4), (3, 0.015, 0.0)])
def test_log_codebook_beats_linear_on_heavy_tails(nu, scale, outl):
    """The comparison the paper draws (Sec. 5): with a heavy-tailed weight distribution the
    linear codebook spends its levels on the rare large weights, the logarithmic one keeps
    precision near zero. Measured here as reconstruction SQNR and product error."""
    w = _tensor(512, 1024, [23, nu, 0, 0], nu, scale, outl)
    r = O.fit(w)
    wl = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
    f = U.uniform_fit(w)
    wu = U.uniform_dequantize(U.uniform_encode(w, f.scale, f.zero), U.uniform_levels(f.scale, f.zero))
    assert U.sqnr_db(w, wl) > U.sqnr_db(w, wu) + 6.0
    x = np.random.default_rng(3).standard_normal((4, 1024))
    y = x @ w.astype(np.float64).T
    assert U.relative_error(x @ wl.astype(np.float64).T, y) < 0.5 * U.relative_error(
        x @ wu.astype(np.float64).T, y)


@pytest.mark.parametrize("seed,nu,scale,outl", [([24, 0, 0, 0], 4, 0.02, 0.0),
                                                ([24, 1, 0, 0], 3, 0.015, 1e-4),
                                                ([24, 2, 0, 0], 6, 1.0, 0.0)])
def test_host_fit_uniform_matches_oracle(seed, nu, scale, outl):
    w = _tensor(300, 256, seed, nu, scale, outl)
    u = L.fit_uniform(w)
    f = U.uniform_fit(w)
    assert (u.bits, u.zero) == (4, f.zero)
    assert (u.wmin, u.wmax, u.scale) == (f.wmin, f.wmax, f.scale)
    assert u.codebook_array().view(np.uint32).tolist() == \
        U.uniform_levels(f.scale, f.zero).view(np.uint32).tolist()
    assert u.thresholds_array().view(np.uint32).tolist() == \
        U.uniform_thresholds(f.scale, f.zero).view(np.uint32).tolist()


def test_host_fit_uniform_errors():
    with pytest.raises(L.LogbqError) as e:
        L.fit_uniform(np.ones(10, dtype=np.float32))
    assert e.value.status == 3                       # DEGENERATE
    with pytest.raises(L.LogbqError) as e:
        L.fit_uniform(np.array([0.0, np.nan], dtype=np.float32))
    assert e.value.status == 2                       # NONFINITE
    with pytest.raises(L.LogbqError) as e:
        L.fit_uniform(np.array([1.0], dtype=np.float32))
    assert e.value.status == 1                       # INVALID_ARG
    with pytest.raises(L.LogbqError) as e:
        L.fit_uniform(np.array([0.0, 1.0], dtype=np.float32), bits=8)
    assert e.value.status == 4                       # UNSUPPORTED
