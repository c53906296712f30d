"""Pins of the exact-sum reading of Eq. 5 (Sec. 3.2) in the oracle (``fit_exact``), which the
device fit must reproduce bit for bit; host-side checks of logbq_fit_device's argument
validation; and the library's host run of the device fit's passes and exact selection
(logbq_fit_exact) bit for bit against the oracle (no GPU). The pins come from outside the function: hand-derived results, the
sequential float64 fit where the two readings cannot differ, a rational-arithmetic
certificate of w_min computed another way, and invariances of the definition."""
import ctypes
from fractions import Fraction

import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L


def test_hand_tie_case():
    # squares 1, 1, 1, 1, 4: total 8, eps 1/2 -> the prefix reaches 4 exactly at index 3.
    r = O.fit_exact(np.array([1, 1, 1, 1, 2], dtype=np.float32), eps=0.5)
    assert (r.wmin, r.wmax, r.wmin_index) == (1.0, 2.0, 3)


def test_hand_case_where_float64_sums_round():
    # 100 weights 2^-30 (squares 2^-60) and one 1.0: the exact total 1 + 100 2^-60 rounds to 1
    # in float64. With eps = 50 2^-60 the exact condition (i + 1) 2^-60 >= eps (1 + 100 2^-60)
    # first holds at i + 1 = 51; the sequential float64 reading stops at i + 1 = 50.
    w = np.array([2.0 ** -30] * 100 + [1.0], dtype=np.float32)
    eps = 50 * 2.0 ** -60
    assert O.fit_exact(w, eps=eps).wmin_index == 50
    assert O.fit(w, eps=eps).wmin_index == 49
    assert O.fit_exact(w, eps=eps).wmin == O.fit(w, eps=eps).wmin == 2.0 ** -30


def test_hand_subnormal_case():
    # |w| = k 2^-149 for k = 1, 2, 3, 4, 100: squares k^2 2^-298, total 10030 units; eps 1e-3
    # needs 10.03 units: prefixes 1, 5, 14 -> index 2, w_min = 3 2^-149.
    w = (np.array([1, 2, 3, 4, 100], dtype=np.float64) * 2.0 ** -149).astype(np.float32)
    assert np.all(w > 0)
    r = O.fit_exact(-w[::-1].copy(), eps=1e-3)
    assert r.wmin_index == 2 and r.wmin == 3 * 2.0 ** -149 and r.wmax == 100 * 2.0 ** -149


@pytest.mark.parametrize("name", ["linear_2048x2048", "up_2048x8192_outliers", "layer_8192x28672"])
def test_agrees_with_sequential_fit_on_workload_slices(name):
    """Far from a rounding boundary the two readings of Eq. 5 coincide."""
    wl = inputs.WORKLOADS[name]
    lin = wl["layers"][0]
    w = np.asarray(inputs.student_t_weights(256, lin.k, wl["nu"], wl["scale"],
                                            seed=[wl["cfg"], 0, 0, 0],
                                            outlier_frac=wl.get("outlier_frac", 0.0)))
    assert O.fit_exact(w) == O.fit(w)
    assert O.fit_exact(w, bits=8, eps=1e-6) == O.fit(w, bits=8, eps=1e-6)


def test_agrees_with_sequential_fit_random():
    rng = np.random.default_rng(77)
    for i in range(30):
        n = int(rng.integers(2, 3000))
        w = (rng.standard_t([2.5, 3, 4, 8][i % 4], n) * 10 ** rng.uniform(-30, 20)).astype(np.float32)
        if i % 5 == 0:
            w[rng.integers(0, n, n // 3)] = 0.0
        eps = [4e-3, 1e-6, 0.1][i % 3]
        try:
            a = O.fit(w, 4, eps)
        except O.OracleError as e:
            with pytest.raises(O.OracleError, match=e.kind):
                O.fit_exact(w, 4, eps)
            continue
        assert O.fit_exact(w, 4, eps) == a


def test_certificate_in_rationals():
    """w_min is present in |w|, the exact energy of |w| <= w_min reaches eps, that of
    |w| < w_min does not, and wmin_index counts the smaller weights plus the copies of w_min
    needed to reach eps."""
    rng = np.random.default_rng(5)
    for i in range(12):
        n = int(rng.integers(5, 400))
        w = (rng.standard_t(3, n) * 0.02).astype(np.float32)
        w = np.round(w, [2, 3, 6][i % 3]).astype(np.float32)   # ties
        eps = [4e-3, 0.05, 0.3][i % 3]
        try:
            r = O.fit_exact(w, 4, eps)
        except O.OracleError:
            continue
        a = np.abs(w.astype(np.float64))
        assert r.wmin in a.tolist()
        assert O.energy_ratio_exact(w, r.wmin) >= Fraction(eps)
        below = a[a < r.wmin]
        if below.size:
            assert O.energy_ratio_exact(w, float(below.max())) < Fraction(eps)
        sq = [Fraction(float(v)) ** 2 for v in a]
        total = sum(sq)
        e_below = sum(s for v, s in zip(a, sq) if v < r.wmin)
        v2 = Fraction(r.wmin) ** 2
        j = 1
        while e_below + j * v2 < Fraction(eps) * total:
            j += 1
        assert r.wmin_index == int(np.count_nonzero(a < r.wmin)) + j - 1


def test_invariances():
    w = np.asarray(inputs.student_t_weights(64, 96, 4, 0.02, seed=[40, 0, 0, 0]))
    r = O.fit_exact(w)
    perm = np.random.default_rng(1).permutation(w.size)
    assert O.fit_exact(w.ravel()[perm]) == r
    assert O.fit_exact(-w) == r
    r2 = O.fit_exact((w * np.float32(2.0 ** 10)).astype(np.float32))
    assert (r2.wmin, r2.wmax, r2.wmin_index) == (r.wmin * 2 ** 10, r.wmax * 2 ** 10, r.wmin_index)
    assert r2.base == r.base


def test_errors_match_sequential_fit():
    for w, kind in [(np.array([1.0, np.nan], dtype=np.float32), "nonfinite"),
                    (np.zeros(8, dtype=np.float32), "degenerate"),
                    (np.array([0.5, -0.5, 0.5, 0.0], dtype=np.float32), "degenerate"),
                    (np.array([0.5], dtype=np.float32), "invalid_arg")]:
        with pytest.raises(O.OracleError, match=kind):
            O.fit_exact(w)


def test_fit_device_validation_before_hip():
    h = L.lib()
    p = ctypes.byref(L.Params())
    a, ws = ctypes.c_void_p(4096), ctypes.c_void_p(8192)   # never dereferenced on these paths
    assert h.logbq_fit_device(None, 16, 4, 4e-3, ws, p, None) == L.ERR_INVALID_ARG
    assert h.logbq_fit_device(a, 16, 4, 4e-3, None, p, None) == L.ERR_INVALID_ARG
    assert h.logbq_fit_device(a, 16, 4, 4e-3, ws, None, None) == L.ERR_INVALID_ARG
    assert h.logbq_fit_device(a, 1, 4, 4e-3, ws, p, None) == L.ERR_INVALID_ARG
    for eps in (0.0, 1.0, -1.0, float("nan")):
        assert h.logbq_fit_device(a, 16, 4, eps, ws, p, None) == L.ERR_INVALID_ARG
    for bits in (2, 5, 16):
        assert h.logbq_fit_device(a, 16, bits, 4e-3, ws, p, None) == L.ERR_UNSUPPORTED
    assert h.logbq_fit_device(a, 2 ** 40, 4, 4e-3, ws, p, None) == L.ERR_UNSUPPORTED
    assert h.logbq_fit_device(ctypes.c_void_p(4100), 16, 4, 4e-3, ws, p, None) == L.ERR_UNSUPPORTED
    assert h.logbq_fit_device(a, 16, 4, 4e-3, ctypes.c_void_p(8196), p, None) == L.ERR_UNSUPPORTED
    assert L.FIT_WORKSPACE_BYTES == (1 + 3 * (2048 + 512 + 2048)) * 8


def _assert_exact_params(p, r, bits):
    q = 2 ** (bits - 1) - 1
    assert (p.bits, p.qmax) == (bits, q)
    assert (p.wmin, p.wmax, p.wmin_index) == (r.wmin, r.wmax, r.wmin_index)
    assert (p.base, p.shift) == (r.base, r.shift)
    assert p.codebook_array().view(np.uint32).tolist() == \
        O.codebook(r.base, r.shift, bits).view(np.uint32).tolist()
    assert p.thresholds_array()[:q].view(np.uint32).tolist() == \
        O.magnitude_thresholds(r.base, r.shift, bits).view(np.uint32).tolist()


@pytest.mark.parametrize("w,eps", [
    (np.array([1, 1, 1, 1, 2], np.float32), 0.5),
    (np.array([2.0 ** -30] * 100 + [1.0], np.float32), 50 * 2.0 ** -60),
    ((np.array([1, 2, 3, 4, 100.]) * 2.0 ** -149).astype(np.float32), 1e-3),
    (np.array([0.25, -1.0], np.float32), 0.05),
], ids=["tie", "float64-sums-round", "subnormals", "two-weights"])
def test_library_exact_fit_hand_cases(w, eps):
    _assert_exact_params(L.fit_exact(w, 4, eps), O.fit_exact(w, 4, eps), 4)


def test_library_exact_fit_random():
    """The device fit's passes and exact selection, run on the host, against the oracle."""
    rng = np.random.default_rng(91)
    for i in range(40):
        n = int(rng.integers(2, 40000))
        # magnitudes over the whole float32 range: 8-bit fits at 1e-35 or 1e30 have shifts s in
        # the thousands, where the exact thresholds need powers b^n with n near 2 s
        w = (rng.standard_t([2.5, 3, 4, 8][i % 4], n) * 10 ** rng.uniform(-42, 30)).astype(np.float32)
        if i % 5 == 0:
            w[rng.integers(0, n, n // 3)] = 0.0
        if i % 7 == 0:
            w = (np.round(w / np.abs(w).max() * 50) * 0.01).astype(np.float32)
        bits, eps = [4, 8][i % 2], [4e-3, 1e-6, 0.1, 0.5][i % 4]
        try:
            r = O.fit_exact(w, bits, eps)
        except O.OracleError as e:
            with pytest.raises(L.LogbqError) as err:
                L.fit_exact(w, bits, eps)
            assert err.value.status == {"nonfinite": L.ERR_NONFINITE,
                                        "degenerate": L.ERR_DEGENERATE}[e.kind]
            continue
        _assert_exact_params(L.fit_exact(w, bits, eps), r, bits)


@pytest.mark.parametrize("name", ["up_2048x8192_outliers", "layer_8192x28672"])
def test_library_exact_fit_workload_slices(name):
    wl = inputs.WORKLOADS[name]
    lin = wl["layers"][0]
    w = np.asarray(inputs.student_t_weights(512, lin.k, wl["nu"], wl["scale"],
                                            seed=[wl["cfg"], 1, 0, 0],
                                            outlier_frac=wl.get("outlier_frac", 0.0)))
    _assert_exact_params(L.fit_exact(w), O.fit_exact(w), 4)
    _assert_exact_params(L.fit_exact(w, 8, 1e-6), O.fit_exact(w, 8, 1e-6), 8)


def test_library_exact_fit_errors():
    for w, status in [(np.array([1.0, np.nan], np.float32), L.ERR_NONFINITE),
                      (np.array([1.0, -np.inf], np.float32), L.ERR_NONFINITE),
                      (np.zeros(8, np.float32), L.ERR_DEGENERATE),
                      (np.array([0.5, -0.5, 0.5, 0.0], np.float32), L.ERR_DEGENERATE),
                      (np.array([0.5], np.float32), L.ERR_INVALID_ARG)]:
        with pytest.raises(L.LogbqError) as e:
            L.fit_exact(w)
        assert e.value.status == status
    for eps in (0.0, 1.0, float("nan")):
        with pytest.raises(L.LogbqError) as e:
            L.fit_exact(np.array([0.5, 1.0], np.float32), eps=eps)
        assert e.value.status == L.ERR_INVALID_ARG
    with pytest.raises(L.LogbqError) as e:
        L.fit_exact(np.array([0.5, 1.0], np.float32), bits=5)
    assert e.value.status == L.ERR_UNSUPPORTED
