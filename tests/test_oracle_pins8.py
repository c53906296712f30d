"""Pins of the CPU oracle at 8 bits (q_max = 127, 256-entry codebook; no GPU).

Sec. 3.1-3.2 define the quantizer for any bit width n; the paper's other setting is n = 8 with
the energy fraction eps = 1e-6 (Sec. 3.2). The same kinds of checks as at 4 bits pin the oracle
against things other than itself: exact brute force of Eq. 5, closed forms of Eq. 3-4, the
log-domain / threshold equivalence of Eq. 1 around every one of the 127 boundaries, brute-force
log-nearest search over all 256 entries, round trips, special values; planted 8-bit mistakes
must each fail at least one of them.
"""
import math
from fractions import Fraction
from unittest import mock

import numpy as np
import pytest

from oracle import logbq_oracle as O

BITS = 8
EPS8 = 1e-6


def _tiny_tensors():
    rng = np.random.default_rng(8)
    out = []
    for i in range(60):
        n = int(rng.integers(8, 48))
        w = (rng.standard_t(3, size=n) * 10 ** rng.uniform(-3, 0)).astype(np.float32)
        if i % 4 == 0:
            w[rng.integers(0, n, 3)] = w[0]           # duplicates
        if i % 5 == 0:
            w[rng.integers(0, n, 2)] = 0.0            # zeros
        if i % 7 == 0:
            w[rng.integers(0, n)] = np.float32(50.0)  # an outlier
        out.append(w)
    return out


@pytest.mark.parametrize("eps", [EPS8, 1e-3, 0.2])
def test_fit8_wmin_wmax_bruteforce(eps):
    """w_min is the smallest |w_j| whose exact energy ratio reaches eps (Eq. 5) and w_max the
    largest |w| (Sec. 3.2), at 8 bits; b and s follow from them (checked below)."""
    checked = 0
    for w in _tiny_tensors():
        cands = sorted(set(float(v) for v in np.abs(w)))
        ratios = {t: O.energy_ratio_exact(w, t) for t in cands}
        if ratios[cands[-1]] == 0 or any(abs(float(r) - eps) < 1e-12 for r in ratios.values()):
            continue
        brute = min(t for t in cands if ratios[t] >= Fraction(eps))
        if brute == cands[-1]:
            continue
        r = O.fit(w, BITS, eps)
        assert r.wmin == brute and r.wmax == cands[-1]
        checked += 1
    assert checked > 30


def test_fit8_closed_forms():
    """Eq. 3: b^127 = w_max / w_min; Eq. 4: b^J <= w_max < b^(J+1) exactly with J = 127 - s;
    the 256-entry codebook is sign-symmetric and geometric with ratio b."""
    rng = np.random.default_rng(18)
    for i in range(20):
        w = (rng.standard_t([3, 4, 6][i % 3], size=8192) * 10 ** rng.uniform(-4, 1)).astype(np.float32)
        r = O.fit(w, BITS, EPS8)
        assert abs(r.base ** 127 / (r.wmax / r.wmin) - 1) < 1e-12
        J = 127 - r.shift
        bF = Fraction(r.base)
        assert bF ** J <= Fraction(r.wmax) < bF ** (J + 1)
        lut = O.codebook(r.base, r.shift, BITS)
        assert lut.shape == (256,) and lut[0] == 0 and lut[128] == 0 and not np.signbit(lut[128])
        assert np.array_equal(lut[129:], -lut[1:128])
        for k in (1, 2, 63, 64, 126, 127):
            exact = bF ** (k - r.shift)
            assert abs(Fraction(float(lut[k])) - exact) <= Fraction(float(np.spacing(lut[k]))) / 2
        ratios = lut[2:128].astype(np.float64) / lut[1:127].astype(np.float64) / r.base
        assert np.all(np.abs(ratios - 1) < 2.5e-7)
        assert float(lut[127]) <= r.wmax


def _params8():
    rng = np.random.default_rng(28)
    out = []
    for i in range(4):
        w = (rng.standard_t(3 + i % 3, size=50000) * 10 ** rng.uniform(-3, 0)).astype(np.float32)
        r = O.fit(w, BITS, EPS8)
        out.append((r.base, r.shift))
    return out


PARAMS8 = _params8()


@pytest.mark.parametrize("bs", PARAMS8[:2])
def test_encode8_log_domain_equals_thresholds(bs):
    """Eq. 1 at 8 bits is a monotone step function of |x| with 127 steps: the magnitude is
    the number of thresholds at or below |x|. Random magnitudes over the codebook range plus
    +-3 float32 ulps around every threshold."""
    b, s = bs
    thr = O.magnitude_thresholds(b, s, BITS)
    assert thr.shape == (127,) and np.all(np.diff(thr) > 0)
    rng = np.random.default_rng(int(b * 1e6) % 1000 + s)
    lo, hi = math.log(float(thr[0])) - 2, math.log(float(thr[-1])) + 2
    xs = [np.exp(rng.uniform(lo, hi, 100_000)).astype(np.float32)]
    for t in thr:
        v = np.array([t], dtype=np.float32).view(np.int32)[0]
        xs.append((np.arange(-3, 4, dtype=np.int32) + v).view(np.float32))
    x = np.concatenate(xs)
    x = np.concatenate([x, -x])
    codes = O.encode(x, b, s, BITS)
    mag = np.searchsorted(thr, np.abs(x), side="right")
    exp = np.where((x < 0) & (mag > 0), mag + 128, mag)
    assert np.array_equal(codes, exp.astype(np.uint8))


@pytest.mark.parametrize("bs", PARAMS8[:2])
def test_encode8_is_log_nearest_bruteforce(bs):
    """Every weight encodes to the log-nearest of all 256 entries with its own sign."""
    b, s = bs
    rng = np.random.default_rng(int(b * 1e5) % 997 + s)
    x = (rng.standard_t(3, size=300) * float(b) ** (64 - s)).astype(np.float32)
    x[:5] = [0.0, -0.0, np.inf, -np.inf, np.nan]
    assert O.encode(x, b, s, BITS).tolist() == [O.log_nearest_code(v, b, s, BITS) for v in x]


def test_dequant8_encode_idempotent():
    """encode(dequantize(c)) == c for all 256 codes (128, '-0', decodes to 0 -> code 0)."""
    for b, s in PARAMS8:
        lut = O.codebook(b, s, BITS)
        codes = np.arange(256, dtype=np.uint8)
        back = O.encode(O.dequantize(codes, lut), b, s, BITS)
        exp = codes.copy()
        exp[128] = 0
        assert back.tolist() == exp.tolist()


def test_encode8_special_values():
    b, s = PARAMS8[0]
    x = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 3e38, -3e38], dtype=np.float32)
    assert O.encode(x, b, s, BITS).tolist() == [0, 127, 255, 0, 0, 0, 0, 127, 255]


def test_pack_codes8_is_one_byte_per_weight():
    rng = np.random.default_rng(3)
    c = rng.integers(0, 256, size=(5, 64), dtype=np.uint8)
    p = O.pack_codes(c, 8)
    assert p.shape == (5, 64) and np.array_equal(p, c) and p is not c
    assert np.array_equal(O.unpack_codes(p, 8), c)
    c4 = c & 15
    assert np.array_equal(O.pack_codes(c4, 4), O.pack(c4))


# ---------------------------------------------------------------- planted 8-bit mistakes

def _run_pins8():
    failed = []
    checks = {
        "bruteforce": lambda: test_fit8_wmin_wmax_bruteforce(EPS8),
        "closed": test_fit8_closed_forms,
        "thresholds": lambda: test_encode8_log_domain_equals_thresholds(PARAMS8[0]),
        "nearest": lambda: test_encode8_is_log_nearest_bruteforce(PARAMS8[0]),
        "idempotent": test_dequant8_encode_idempotent,
        "special": test_encode8_special_values,
    }
    for name, fn in checks.items():
        try:
            fn()
        except (AssertionError, O.OracleError, ValueError, IndexError):
            failed.append(name)
    return failed


_REAL = {"fit": O.fit, "codebook": O.codebook, "encode": O.encode}


def _mut_fit_qmax4(w, bits=4, eps=4e-3):
    return _REAL["fit"](w, 4, eps)                       # the 4-bit q_max at every width


def _mut_encode_sign_nibble(x, base, shift, bits=4):
    c = _REAL["encode"](x, base, shift, bits).astype(np.int64)
    neg = c >= 2 ** (bits - 1)
    return np.where(neg, c - 2 ** (bits - 1) + 8, c).astype(np.uint8)   # sign bit at bit 3


def _mut_encode_clamp7(x, base, shift, bits=4):
    c = _REAL["encode"](x, base, shift, bits).astype(np.int64)
    half = 2 ** (bits - 1)
    mag, neg = c % half, c >= half
    mag = np.minimum(mag, 7)
    return (mag + half * (neg & (mag > 0))).astype(np.uint8)


def _mut_codebook_half8(base, shift, bits=4):
    lut = _REAL["codebook"](base, shift, bits)
    if bits == 8:
        lut = np.concatenate([lut[:8], lut[8:128], lut[128:]])   # shape kept...
        lut[129:] = lut[1:128]                                   # ...negatives lose the sign
    return lut


MUTANTS8 = {
    "fit_qmax_4bit": ("fit", _mut_fit_qmax4),
    "sign_bit_at_3": ("encode", _mut_encode_sign_nibble),
    "clamp_to_7": ("encode", _mut_encode_clamp7),
    "codebook_sign": ("codebook", _mut_codebook_half8),
}


def test_pins8_pass_on_real_oracle():
    assert _run_pins8() == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS8))
def test_pins8_catch_planted_mistakes(mutant):
    attr, fn = MUTANTS8[mutant]
    with mock.patch.object(O, attr, fn):
        assert _run_pins8(), f"planted mistake {mutant} passed every 8-bit pin"
