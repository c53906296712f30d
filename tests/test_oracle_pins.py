"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each test checks the oracle against something other than itself: the hand-derived worked
example (tests/golden/worked_b2.txt), brute force on tiny inputs in exact rational
arithmetic, closed forms of Eq. 3-4, the log-domain / threshold equivalence of Eq. 1, and
round trips. ``test_pins_catch_planted_mistakes`` plants plausible mistakes in the oracle and
checks that at least one pin fails for each.
"""
import math
import os
from fractions import Fraction
from unittest import mock

import numpy as np
import pytest

from oracle import logbq_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_b2.txt")


def f32(hexstr):
    return np.array([int(hexstr, 16)], dtype=np.uint32).view(np.float32)[0]


def load_golden():
    d = {"weights": [], "code": [], "pack": []}
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *rest = line.split()
            if key == "weights":
                d["weights"].append((int(rest[0]), f32(rest[1])))
            elif key == "code":
                d["code"].append((f32(rest[0]), int(rest[1])))
            elif key == "pack":
                arrow = rest.index("->")
                d["pack"].append(([int(v) for v in rest[:arrow]],
                                  [int(v, 16) for v in rest[arrow + 1:]]))
            else:
                d[key] = rest
    return d


# ---------------------------------------------------------------- worked example (golden)

@pytest.mark.parametrize("S", [0, 3, -10])
def test_worked_example(S):
    g = load_golden()
    scale = np.float32(2.0 ** S)
    w = np.concatenate([np.full(c, v, dtype=np.float32) for c, v in g["weights"]]) * scale
    w = np.random.default_rng(S + 100).permutation(w).astype(np.float32)
    eps = float(g["eps"][0])
    r = O.fit(w, 4, eps)
    assert r.wmin_index == int(g["wmin_index"][0])
    assert r.wmin == float(f32(g["wmin"][0]) * scale)
    assert r.wmax == float(f32(g["wmax"][0]) * scale)
    assert r.base == float(g["base"][0])
    assert r.shift == int(g["shift"][0]) - S
    lut = O.codebook(r.base, r.shift)
    exp_lut = np.array([f32(h) for h in g["codebook"]], dtype=np.float32) * scale
    assert lut.view(np.uint32).tolist() == exp_lut.view(np.uint32).tolist()
    thr = O.magnitude_thresholds(r.base, r.shift)
    exp_thr = np.array([f32(h) for h in g["thresholds"]], dtype=np.float32) * scale
    assert thr.view(np.uint32).tolist() == exp_thr.view(np.uint32).tolist()
    xs = np.array([x for x, _ in g["code"]], dtype=np.float32) * scale
    codes = O.encode(xs, r.base, r.shift)
    assert codes.tolist() == [c for _, c in g["code"]]
    for codes_in, bytes_out in g["pack"]:
        packed = O.pack(np.array([codes_in], dtype=np.uint8))
        assert packed[0].tolist() == bytes_out
        assert O.unpack(packed)[0].tolist() == codes_in


# ---------------------------------------------------------------- Eq. 5 brute force

def _tiny_tensors():
    rng = np.random.default_rng(7)
    out = []
    for i in range(60):
        n = int(rng.integers(2, 48))
        w = (rng.standard_t(3, size=n) * 0.05).astype(np.float32)
        if i % 3 == 0:                      # duplicates
            w[: n // 2] = w[0]
        if i % 4 == 1:                      # exact zeros
            w[rng.integers(0, n, size=max(1, n // 4))] = 0.0
        if i % 5 == 2:                      # one outlier
            w[rng.integers(0, n)] = np.float32(3.0)
        out.append(w)
    return out


@pytest.mark.parametrize("eps", [4e-3, 0.05, 0.3])
def test_fit_wmin_wmax_bruteforce(eps):
    """w_min is the smallest |w_j| whose exact energy ratio reaches eps (Eq. 5);
    w_max is the largest |w| (Sec. 3.2)."""
    checked = 0
    for w in _tiny_tensors():
        cands = sorted(set(float(v) for v in np.abs(w)))
        ratios = {t: O.energy_ratio_exact(w, t) for t in cands}
        if ratios[cands[-1]] == 0:
            continue
        # float64 rounding may only matter when a ratio is within 1e-12 of eps
        if any(abs(float(r) - eps) < 1e-12 for r in ratios.values()):
            continue
        brute = min(t for t in cands if ratios[t] >= Fraction(eps))
        if brute == cands[-1]:
            continue          # w_min == w_max: degenerate (tested separately)
        r = O.fit(w, 4, eps)
        assert r.wmin == brute
        assert r.wmax == cands[-1]
        # the pruned energy (strictly below w_min) is below eps (Sec. 3.2 "discard eps")
        below = [t for t in cands if t < brute]
        if below:
            assert ratios[below[-1]] < Fraction(eps)
        checked += 1
    assert checked > 30


def test_fit_closed_forms():
    """Eq. 3: b^q_max = w_max / w_min; Eq. 4: b^J <= w_max < b^(J+1) with J = q_max - s
    (exact); the codebook is symmetric, geometric with ratio b, and its top entry is the
    largest power of b not above w_max (Sec. 3.1)."""
    rng = np.random.default_rng(11)
    for i in range(40):
        nu = [3, 4, 6][i % 3]
        scale = float(10.0 ** rng.uniform(-4, 1))
        w = (rng.standard_t(nu, size=4096) * scale).astype(np.float32)
        r = O.fit(w, 4, 4e-3)
        q = O.qmax(4)
        assert abs(r.base ** q / (r.wmax / r.wmin) - 1) < 1e-12
        J = q - r.shift
        bF = Fraction(r.base)
        assert bF ** J <= Fraction(r.wmax) < bF ** (J + 1)
        lut = O.codebook(r.base, r.shift)
        assert lut[0] == 0 and lut[8] == 0 and not np.signbit(lut[8])
        for k in range(1, 8):
            assert lut[8 + k] == -lut[k]
            # entry k is b^(k - s) rounded to float32: within half an ulp
            exact = bF ** (k - r.shift)
            assert abs(Fraction(float(lut[k])) - exact) <= Fraction(float(np.spacing(lut[k]))) / 2
        for k in range(1, 7):
            assert abs(float(lut[k + 1]) / float(lut[k]) / r.base - 1) < 2.5e-7
        assert float(lut[7]) <= r.wmax
        assert r.wmin < float(lut[1]) * (1 + 1.2e-7) and float(lut[1]) <= r.base * r.wmin * (1 + 1.2e-7)


def test_fit_errors():
    with pytest.raises(O.OracleError, match="nonfinite"):
        O.fit(np.array([1, np.nan], dtype=np.float32))
    with pytest.raises(O.OracleError, match="nonfinite"):
        O.fit(np.array([1, np.inf], dtype=np.float32))
    with pytest.raises(O.OracleError, match="degenerate"):
        O.fit(np.zeros(8, dtype=np.float32))
    with pytest.raises(O.OracleError, match="degenerate"):
        O.fit(np.array([0.5, -0.5, 0.5], dtype=np.float32))
    with pytest.raises(O.OracleError, match="invalid_arg"):
        O.fit(np.array([0.5], dtype=np.float32))
    with pytest.raises(O.OracleError, match="invalid_arg"):
        O.fit(np.array([0.5, 1.0], dtype=np.float32), eps=0.0)
    with pytest.raises(O.OracleError, match="invalid_arg"):
        O.fit(np.array([0.5, 1.0], dtype=np.float32), eps=1.0)


def test_cumsum_is_sequential():
    """Eq. 5 prefix sums are sequential: np.cumsum must add left to right."""
    a = np.random.default_rng(3).random(50_000) ** 7
    acc, seq = 0.0, np.empty_like(a)
    for i, v in enumerate(a):
        acc += v
        seq[i] = acc
    assert np.array_equal(np.cumsum(a), seq)


# ---------------------------------------------------------------- Eq. 1 encode

def _params():
    rng = np.random.default_rng(5)
    out = [(2.0, 7)]
    for i in range(6):
        w = (rng.standard_t(3 + i % 3, size=20000) * 10 ** rng.uniform(-3, 0)).astype(np.float32)
        r = O.fit(w)
        out.append((r.base, r.shift))
    return out


@pytest.mark.parametrize("bs", _params())
def test_encode_log_domain_equals_thresholds(bs):
    """Rounding log_b|x| + s (Eq. 1) is a monotone step function of |x|: its magnitude is
    the number of thresholds at or below |x|. Checked on random magnitudes over the whole
    codebook range and on +-4 float32 ulps around every threshold."""
    b, s = bs
    thr = O.magnitude_thresholds(b, s)
    rng = np.random.default_rng(int(b * 1000) + s)
    lo, hi = math.log(float(thr[0])) - 3, math.log(float(thr[-1])) + 3
    xs = [np.exp(rng.uniform(lo, hi, 200_000)).astype(np.float32)]
    for t in thr:
        v = np.array([t], dtype=np.float32).view(np.int32)[0]
        xs.append((np.arange(-4, 5, dtype=np.int32) + v).view(np.float32))
    x = np.concatenate(xs)
    x = np.concatenate([x, -x])
    codes = O.encode(x, b, s)
    mag = np.searchsorted(thr, np.abs(x), side="right")
    exp = np.where((x < 0) & (mag > 0), mag + 8, mag)
    assert np.array_equal(codes, exp.astype(np.uint8))


def test_thresholds_are_rounding_boundaries():
    """tau_k has magnitude k+1 and the float32 just below it has magnitude k (Eq. 1, checked
    with float64 logs away from the exact boundary)."""
    for b, s in _params():
        thr = O.magnitude_thresholds(b, s)
        for k, t in enumerate(thr):
            below = np.nextafter(t, np.float32(0))
            tk = math.log(float(t)) / math.log(b) + s
            tb = math.log(float(below)) / math.log(b) + s
            assert tb <= k + 0.5 + 1e-12 and tk >= k + 0.5 - 1e-12
            assert abs(tk - (k + 0.5)) < 1e-6


@pytest.mark.parametrize("bs", _params()[:4])
def test_encode_is_log_nearest_bruteforce(bs):
    """Every weight encodes to the nearest codebook entry in log distance with its own sign
    (brute force over all 16 entries per weight, tiny tensor)."""
    b, s = bs
    rng = np.random.default_rng(int(b * 77) + s)
    x = (rng.standard_t(3, size=400) * float(b) ** (4 - s)).astype(np.float32)
    x[:5] = [0.0, -0.0, np.inf, -np.inf, np.nan]
    codes = O.encode(x, b, s)
    brute = [O.log_nearest_code(v, b, s) for v in x]
    assert codes.tolist() == brute


def test_encode_value_space_nearest():
    """Away from rounding boundaries, the decoded entry of x is the same-sign codebook entry
    minimising |ln|x| - ln|c|| over all float32 entries (zero's log position is b^-s)."""
    for b, s in _params()[:4]:
        lut = O.codebook(b, s)
        rng = np.random.default_rng(int(b * 31))
        x = (rng.standard_t(3, size=3000) * float(b) ** (4 - s)).astype(np.float32)
        codes = O.encode(x, b, s)
        t = np.log(np.abs(x.astype(np.float64))) / math.log(b) + s
        away = np.abs(t - np.floor(t) - 0.5) > 1e-4
        pos = np.concatenate([[b ** -s], lut[1:8].astype(np.float64)])
        for xi, ci, ok in zip(x, codes, away):
            if not ok or xi == 0:
                continue
            d = np.abs(np.log(abs(float(xi))) - np.log(pos))
            k = int(np.argmin(d))
            exp = k if (k == 0 or xi > 0) else k + 8
            assert ci == exp


def test_dequant_encode_idempotent():
    """encode(dequantize(c)) == c for every code (code 8, '-0', decodes to 0 -> code 0)."""
    for b, s in _params():
        lut = O.codebook(b, s)
        codes = np.arange(16, dtype=np.uint8)
        back = O.encode(O.dequantize(codes, lut), b, s)
        exp = codes.copy()
        exp[8] = 0
        assert back.tolist() == exp.tolist()


def test_encode_special_values():
    b, s = 2.0, 7
    x = np.array([np.nan, -np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 3e38, -3e38],
                 dtype=np.float32)
    assert O.encode(x, b, s).tolist() == [0, 0, 7, 15, 0, 0, 0, 0, 7, 15]


def test_pack_roundtrip():
    rng = np.random.default_rng(1)
    c = rng.integers(0, 16, size=(7, 64), dtype=np.uint8)
    p = O.pack(c)
    assert p.shape == (7, 32)
    assert np.array_equal(O.unpack(p), c)
    assert p[3, 5] == (c[3, 10] | (c[3, 11] << 4))


# ---------------------------------------------------------------- y = x W^T

def test_linear_bruteforce_exact():
    """The float64 matmul agrees with exact rational dot products to float64 rounding."""
    rng = np.random.default_rng(2)
    b, s = _params()[2]
    lut = O.codebook(b, s)
    for m, n, k in [(1, 3, 32), (2, 5, 64), (3, 2, 96)]:
        x = rng.standard_normal((m, k)).astype(np.float16)
        codes = rng.integers(0, 16, size=(n, k), dtype=np.uint8)
        wh = O.dequantize(codes, lut)
        y = O.linear(x, wh)
        for i in range(m):
            for j in range(n):
                terms = [Fraction(float(x[i, t])) * Fraction(float(wh[j, t])) for t in range(k)]
                exact = sum(terms, Fraction(0))
                mag = sum((abs(t) for t in terms), Fraction(0))
                assert abs(Fraction(y[i, j]) - exact) <= mag * Fraction(1, 2 ** 50)


# ---------------------------------------------------------------- planted mistakes

def _run_pins():
    """Run the main pins; return the names of those that fail."""
    failed = []
    checks = {
        "golden": lambda: [test_worked_example(S) for S in (0, 3, -10)],
        "bruteforce": lambda: test_fit_wmin_wmax_bruteforce(4e-3),
        "closed": test_fit_closed_forms,
        "thresholds": lambda: [test_encode_log_domain_equals_thresholds(p) for p in _params()[:3]],
        "nearest": lambda: [test_encode_is_log_nearest_bruteforce(p) for p in _params()[:2]],
        "idempotent": test_dequant_encode_idempotent,
        "pack": test_pack_roundtrip,
    }
    for name, fn in checks.items():
        try:
            fn()
        except (AssertionError, O.OracleError, ValueError, IndexError):
            failed.append(name)
    return failed


def _mut_fit_shift_sign(w, bits=4, eps=4e-3):
    r = _REAL["fit"](w, bits, eps)
    J = O.qmax(bits) - r.shift
    r.shift = O.qmax(bits) + J          # s = q_max + floor(log_b w_max): sign error
    return r


def _mut_fit_energy_not_squared(w, bits=4, eps=4e-3):
    # Eq. 5 with |w_i| in place of w_i^2 (a dropped square)
    return _REAL["fit"](np.sign(w) * np.sqrt(np.abs(w)).astype(np.float32), bits, eps)


def _mut_fit_strict(w, bits=4, eps=4e-3):
    r = _REAL["fit"](w, bits, eps)
    a = np.sort(np.abs(np.asarray(w, dtype=np.float64)).ravel())
    r.wmin = float(a[min(r.wmin_index + 1, a.size - 1)])   # off-by-one in Eq. 5 index
    r.wmin_index += 1
    return r


def _mut_codebook_offbyone(base, shift, bits=4):
    lut = _REAL["codebook"](base, shift + 1, bits)          # b^(k - s - 1)
    return lut


def _mut_encode_half_even(x, base, shift, bits=4):
    x = np.asarray(x, dtype=np.float32)
    ax = np.abs(x.astype(np.float64))
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.log(ax) / math.log(base) + shift
    m = np.clip(np.nan_to_num(np.floor(t), nan=0, neginf=0, posinf=7), 0, 7)   # truncation
    m = np.where(ax > 0, m, 0).astype(np.int64)
    return np.where((x < 0) & (m > 0), m + 8, m).astype(np.uint8)


def _mut_encode_signed_clamp(x, base, shift, bits=4):
    # the literal garbled clamp: sign(x) * clamp(round(t), -7, 7) in two's complement nibble
    x = np.asarray(x, dtype=np.float32)
    ax = np.abs(x.astype(np.float64))
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.log(ax) / math.log(base) + shift
    q = np.clip(np.nan_to_num(np.floor(t + 0.5), nan=0, neginf=-7, posinf=7), -7, 7)
    q = np.where(ax > 0, np.sign(x) * q, 0).astype(np.int64)
    return np.where(q < 0, 8 - q, q).astype(np.uint8)


def _mut_pack_swapped(codes):
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[:, 1::2] | (codes[:, 0::2] << 4)).astype(np.uint8)


def _mut_codebook_negzero(base, shift, bits=4):
    lut = _REAL["codebook"](base, shift, bits)
    lut[8 + 1:] = lut[1:8]                                     # dropped sign of negatives
    return lut


_REAL = {"fit": O.fit, "codebook": O.codebook, "encode": O.encode, "pack": O.pack}
MUTANTS = {
    "shift_sign": ("fit", _mut_fit_shift_sign),
    "energy_not_squared": ("fit", _mut_fit_energy_not_squared),
    "wmin_off_by_one": ("fit", _mut_fit_strict),
    "codebook_exponent": ("codebook", _mut_codebook_offbyone),
    "codebook_sign": ("codebook", _mut_codebook_negzero),
    "encode_truncates": ("encode", _mut_encode_half_even),
    "encode_signed_clamp": ("encode", _mut_encode_signed_clamp),
    "pack_nibble_order": ("pack", _mut_pack_swapped),
}


def test_pins_pass_on_real_oracle():
    assert _run_pins() == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistakes(mutant):
    attr, fn = MUTANTS[mutant]
    with mock.patch.object(O, attr, fn):
        failed = _run_pins()
    assert failed, f"planted mistake {mutant} passed every pin"
