"""Plain CPU oracle of LogbQuant (Bohn et al., "LogbQuant: Quantizing Language Models in
Logarithmic Space", arXiv 2607.01127).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or execute this
module: only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` use it. It shares no code with the HIP library and imports nothing from it.

Every function follows the paper's definitions step by step, in float64 numpy, with
Python ``fractions`` for the few decisions that must be exact:

* ``fit``          -- w_max (Sec. 3.2), w_min by energy-based pruning (Eq. 5), the base b
                      (Eq. 3) and the shift s (Eq. 4).
* ``fit_exact``    -- the same with the energy sums of Eq. 5 taken exactly (integers in
                      units of 2^-298, the square of the smallest float32 subnormal).
* ``codebook``     -- the 2^n-entry table of Dequant values (Eq. 2) for every n-bit code.
* ``encode``       -- Quant (Eq. 1): round log_b|x| + s to the nearest integer, clamp the
                      magnitude index to [0, q_max], attach the sign.
* ``magnitude_thresholds`` -- the smallest fp32 value whose Quant magnitude is k+1, for each
                      k; by monotonicity of Eq. 1 these describe the same quantizer.
* ``pack`` / ``unpack`` -- two 4-bit codes per byte (Sec. 3.3: weight packing);
                      ``pack_codes`` / ``unpack_codes`` also take 8-bit codes, one per byte.
* ``dequantize``   -- Dequant (Eq. 2) by table lookup (Sec. 3.3: LUT instead of b^x).
* ``linear``       -- y = x . W_hat^T in float64.

Readings of places where the paper is silent or garbled:

* Eq. 1 prints the clamp on the signed value; clamping sign(x)*round(...) to [-q_max, q_max]
  would send tiny weights to large values of the opposite sign. The magnitude index is
  clamped to [0, q_max] instead, and index 0 means the weight is zero (energy pruning).
* "Rounding to the nearest integer": ties round up in magnitude (floor(t + 1/2)).
* Eq. 4 writes floor(log_b w_max); the floor is taken exactly, as the largest integer J with
  b^J <= w_max, so that the top codebook entry never exceeds w_max.
* Eq. 5: the energy sums are sequential float64 prefix sums over |w| in ascending order,
  the total is the last prefix sum, and the ratio is a float64 division (``fit``). Read
  with exact sums instead (``fit_exact``): the first sorted position whose exact prefix
  energy is at least eps times the exact total, compared as rationals with eps taken as its
  exact double value. The two readings pick the same w_min unless the exact ratio lies within
  float64 rounding of eps.
* The sign+magnitude code has two zeros; code 2^(n-1) ("-0") is never produced and decodes
  to +0.0.
* The codebook is float32: entry k is pow(b, k - s) in double, rounded to float32.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from fractions import Fraction

import numpy as np

__all__ = [
    "OracleError", "FitResult", "qmax", "fit", "fit_exact", "codebook", "encode", "magnitude_thresholds",
    "pack", "unpack", "pack_codes", "unpack_codes", "dequantize", "linear", "energy_ratio_exact",
    "log_nearest_code",
]


class OracleError(ValueError):
    """Raised for inputs the method is not defined on (the library's error codes)."""

    def __init__(self, kind: str, msg: str):
        super().__init__(f"{kind}: {msg}")
        self.kind = kind


def qmax(bits: int) -> int:
    """q_max = 2^(n-1) - 1 (Sec. 3.1, after Eq. 2)."""
    return 2 ** (bits - 1) - 1


@dataclass
class FitResult:
    bits: int
    eps: float
    wmin: float
    wmax: float
    base: float
    shift: int
    wmin_index: int           # index of w_min in |w| sorted ascending
    extra: dict = field(default_factory=dict)


def fit(w, bits: int = 4, eps: float = 4e-3) -> FitResult:
    """Per-tensor codebook parameters (Sec. 3.1 Eq. 3-4, Sec. 3.2 Eq. 5).

    w: any array of float32 weights (flattened). eps: the pruned energy fraction
    (Sec. 3.2 gives 4e-3 for 4-bit codebooks).
    """
    w = _validate(w, bits, eps)

    # |w| ascending, in float64 (squares of float32 values are exact in float64).
    a = np.sort(np.abs(w.astype(np.float64)).ravel(), kind="stable")
    w_max = float(a[-1])                       # w_max := max_i |w_i|  (Sec. 3.2)
    if w_max == 0.0:
        raise OracleError("degenerate", "all weights are zero")

    # Eq. 5: w_min = min{ t : sum_{|w_i| <= t} w_i^2 / sum_i w_i^2 >= eps }.
    # The candidate t run over the sorted magnitudes; the prefix sum at index i is the
    # energy of every weight up to and including a[i].
    energy = a * a
    prefix = np.cumsum(energy)                 # sequential accumulation
    total = prefix[-1]
    ratio = prefix / total
    hit = np.nonzero(ratio >= eps)[0]
    i_star = int(hit[0])
    w_min = float(a[i_star])
    return _base_and_shift(bits, eps, w_min, w_max, i_star)


def _validate(w, bits: int, eps: float) -> np.ndarray:
    w = np.asarray(w)
    if w.dtype != np.float32:
        raise OracleError("invalid_arg", "weights must be float32")
    if bits < 2 or bits > 8:
        raise OracleError("invalid_arg", "bits out of range")
    if not (0.0 < eps < 1.0):
        raise OracleError("invalid_arg", "eps must lie in (0, 1)")
    if w.size < 2:
        raise OracleError("invalid_arg", "need at least two weights")
    if not np.all(np.isfinite(w)):
        raise OracleError("nonfinite", "weights contain NaN or Inf")
    return w


def fit_exact(w, bits: int = 4, eps: float = 4e-3) -> FitResult:
    """Per-tensor codebook parameters with the sums of Eq. 5 taken exactly.

    Every float32 |w_i| is an integer multiple n_i of 2^-149, so w_i^2 = n_i^2 2^-298 and
    both sums of Eq. 5 are integers in units of 2^-298. w_min is |w| at the first position i
    of |w| sorted ascending where sum_{j <= i} n_j^2 >= eps * sum_j n_j^2, decided on
    integers with eps as its exact double value. b and s follow as in ``fit``.
    """
    w = _validate(w, bits, eps)
    a = np.sort(np.abs(w.astype(np.float64)).ravel(), kind="stable")
    w_max = float(a[-1])
    if w_max == 0.0:
        raise OracleError("degenerate", "all weights are zero")
    n = [int(v) for v in np.ldexp(a, 149).tolist()]   # exact: scaling by a power of two
    energy = [v * v for v in n]
    total = sum(energy)
    num, den = float(eps).as_integer_ratio()
    prefix = 0
    i_star = len(energy) - 1
    for i, e in enumerate(energy):
        prefix += e
        if prefix * den >= num * total:               # prefix / total >= eps
            i_star = i
            break
    return _base_and_shift(bits, eps, float(a[i_star]), w_max, i_star)


def _base_and_shift(bits: int, eps: float, w_min: float, w_max: float, i_star: int) -> FitResult:
    """Eq. 3 and Eq. 4 from w_min and w_max."""
    q = qmax(bits)
    if not (w_min < w_max):
        raise OracleError("degenerate", "w_min == w_max: base would be 1")

    # Eq. 3: b = (w_max / w_min)^(1 / q_max)
    b = math.pow(w_max / w_min, 1.0 / q)
    if not (b > 1.0):
        raise OracleError("degenerate", "base rounds to 1")

    # Eq. 4: s = q_max - floor(log_b w_max), with the floor taken exactly.
    J = math.floor(math.log(w_max) / math.log(b))
    while math.pow(b, J + 1) <= w_max:
        J += 1
    while math.pow(b, J) > w_max:
        J -= 1
    s = q - J
    return FitResult(bits=bits, eps=eps, wmin=w_min, wmax=w_max, base=b, shift=int(s),
                     wmin_index=i_star)


def codebook(base: float, shift: int, bits: int = 4) -> np.ndarray:
    """Dequant (Eq. 2) of every n-bit sign+magnitude code, as float32.

    Code layout: bit (n-1) is the sign, the low n-1 bits the magnitude index |q|.
    Entry |q| = 0 is zero (both signs decode to +0.0); entry |q| = k > 0 is
    sign * b^(k - s).
    """
    half = 2 ** (bits - 1)
    lut = np.zeros(2 ** bits, dtype=np.float32)
    for k in range(1, qmax(bits) + 1):
        v = np.float32(math.pow(base, k - shift))
        lut[k] = v
        lut[half + k] = -v
    return lut


def _exact_ge_threshold(ax: float, base: float, shift: int, j: int) -> bool:
    """Exact test of |x| >= b^(j + 1/2 - s), i.e. whether log_b|x| + s rounds above j.

    Squared on both sides: x^2 >= b^(2j + 1 - 2s), in rational arithmetic with b taken as
    its exact double value.
    """
    lhs = Fraction(ax) ** 2
    rhs = Fraction(base) ** (2 * j + 1 - 2 * shift)
    return lhs >= rhs


def encode(x, base: float, shift: int, bits: int = 4) -> np.ndarray:
    """Quant (Eq. 1) of every element of x, returned as uint8 sign+magnitude codes.

    t = log_b|x| + s is rounded to the nearest integer (ties up), the magnitude index is
    clamped to [0, q_max]; index 0 encodes zero. Where t lies within 1e-9 of a rounding
    boundary the decision is made exactly (see ``_exact_ge_threshold``). NaN and +-0 give
    code 0; +-Inf give the largest magnitude with their sign.
    """
    x = np.asarray(x, dtype=np.float32)
    q = qmax(bits)
    half = 2 ** (bits - 1)
    ax = np.abs(x.astype(np.float64))
    mag = np.zeros(x.shape, dtype=np.int64)
    live = (ax > 0) & ~np.isnan(ax)
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.log(ax[live]) / math.log(base) + shift
        lo = np.floor(t)
        m = np.floor(t + 0.5)
        near = np.abs(t - (lo + 0.5)) < 1e-9
    if np.any(near):
        idx_live = np.nonzero(near)[0]
        vals = ax[live][idx_live]
        for pos, v, j in zip(idx_live, vals, lo[idx_live]):
            m[pos] = j + 1 if _exact_ge_threshold(float(v), base, shift, int(j)) else j
    m = np.clip(m, 0, q)
    mag[live] = m.astype(np.int64)
    neg = (x < 0) & (mag > 0)
    code = mag + half * neg
    return code.astype(np.uint8)


def magnitude_thresholds(base: float, shift: int, bits: int = 4) -> np.ndarray:
    """tau_k = smallest float32 f with Quant magnitude of f > k, for k = 0 .. q_max - 1.

    By Eq. 1 the magnitude of f exceeds k iff f >= b^(k + 1/2 - s); tau_k is found by
    stepping float32 neighbours around pow() with the exact rational test. Thresholds beyond
    the float32 range are +inf.
    """
    q = qmax(bits)
    out = np.empty(q, dtype=np.float32)
    f32max = np.float32(np.finfo(np.float32).max)
    for k in range(q):
        approx = math.pow(base, k + 0.5 - shift)
        if approx > float(f32max) * 2:
            out[k] = np.inf
            continue
        f = np.float32(min(approx, float(f32max)))
        inf32 = np.float32(np.inf)
        while not _exact_ge_threshold(float(f), base, shift, k):
            f = np.nextafter(f, inf32)
            if np.isinf(f):
                break
        while f > 0:
            g = np.nextafter(f, np.float32(0))
            if _exact_ge_threshold(float(g), base, shift, k):
                f = g
            else:
                break
        out[k] = f
    return out


def pack(codes: np.ndarray) -> np.ndarray:
    """Two 4-bit codes per byte (Sec. 3.3). codes: [N][K] with K even.

    Byte (n, j) holds code (n, 2j) in its low nibble and code (n, 2j+1) in its high nibble.
    """
    codes = np.asarray(codes, dtype=np.uint8)
    if codes.ndim != 2 or codes.shape[1] % 2:
        raise OracleError("invalid_arg", "pack needs [N][K] with even K")
    if np.any(codes > 15):
        raise OracleError("invalid_arg", "codes must be 4-bit")
    return (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)


def unpack(packed: np.ndarray) -> np.ndarray:
    """Inverse of ``pack``: [N][K/2] bytes -> [N][K] codes."""
    packed = np.asarray(packed, dtype=np.uint8)
    n, h = packed.shape
    out = np.empty((n, 2 * h), dtype=np.uint8)
    out[:, 0::2] = packed & 0x0F
    out[:, 1::2] = packed >> 4
    return out


def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    """Storage layout of n-bit codes: 4-bit codes two per byte (``pack``), 8-bit codes one per
    byte ([N][K] as is)."""
    if bits == 4:
        return pack(codes)
    if bits == 8:
        return np.array(codes, dtype=np.uint8, copy=True)
    raise OracleError("invalid_arg", "bits must be 4 or 8")


def unpack_codes(packed: np.ndarray, bits: int) -> np.ndarray:
    """Inverse of ``pack_codes``."""
    if bits == 4:
        return unpack(packed)
    if bits == 8:
        return np.array(packed, dtype=np.uint8, copy=True)
    raise OracleError("invalid_arg", "bits must be 4 or 8")


def dequantize(codes: np.ndarray, lut: np.ndarray) -> np.ndarray:
    """W_hat = Dequant(b, s, q) for every code, via the codebook table (Sec. 3.3)."""
    return np.asarray(lut, dtype=np.float32)[np.asarray(codes, dtype=np.int64)]


def linear(x: np.ndarray, w_hat: np.ndarray) -> np.ndarray:
    """y = x . W_hat^T in float64 (weight-only quantization: activations stay full precision).

    x: [M][K] (float16 activations), w_hat: [N][K] float32. The products of float16 and
    float32 values are exact in float64, so y is accurate to float64 rounding of the sums.
    """
    return np.asarray(x, dtype=np.float64) @ np.asarray(w_hat, dtype=np.float64).T


def energy_ratio_exact(w, t: float) -> Fraction:
    """sum_{|w_i| <= t} w_i^2 / sum_i w_i^2 in exact rational arithmetic (Eq. 5)."""
    vals = [Fraction(float(v)) for v in np.abs(np.asarray(w, dtype=np.float32).ravel())]
    tt = Fraction(t)
    num = sum((v * v for v in vals if v <= tt), Fraction(0))
    den = sum((v * v for v in vals), Fraction(0))
    return num / den


def log_nearest_code(x: float, base: float, shift: int, bits: int = 4) -> int:
    """Brute force over all codes: the entry nearest to x in log distance, same sign.

    Magnitude index k sits at position k - s on the log_b axis (Eq. 2); index 0 is the zero
    entry, placed at the virtual position -s. With t = log_b|x| + s the distance to index k
    is |t - k|; the nearest index is found by scanning all q_max + 1 of them (ties go to the
    larger index, matching round-half-up). When the two best distances agree to 1e-9 the
    choice between neighbours j, j+1 is made exactly through |x| >= b^(j + 1/2 - s).
    """
    q = qmax(bits)
    half = 2 ** (bits - 1)
    xf = float(np.float32(x))
    ax = abs(xf)
    if ax == 0.0 or math.isnan(ax):
        return 0
    if math.isinf(ax):
        best = q
    else:
        t = math.log(ax) / math.log(base) + shift
        dists = [abs(t - k) for k in range(q + 1)]
        order = sorted(range(q + 1), key=lambda k: (dists[k], -k))
        best, second = order[0], order[1]
        if abs(dists[best] - dists[second]) < 1e-9 and abs(best - second) == 1:
            j = min(best, second)
            best = j + 1 if _exact_ge_threshold(ax, base, shift, j) else j
    return int(best + (half if (xf < 0 and best > 0) else 0))
