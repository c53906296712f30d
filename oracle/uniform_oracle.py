"""Plain CPU oracle of the comparison baseline of LogbQuant (arXiv 2607.01127): asymmetric
linear ("uniform") quantization at tensor granularity, plus the quality measures used to
compare the two schemes on synthetic weights.

TEST INFRASTRUCTURE ONLY, like ``logbq_oracle``: only the tests, ``__graft_entry__.smoke()``
and ``bench.py``'s CPU legs may use it. It shares no code with the HIP library.

* ``uniform_fit``        -- scaling factor s and zero-point z of Quant(s, z, x) (Sec. 2) for
                            one tensor, from its full value range (asymmetric, tensor-wise, as
                            the baseline of Sec. 4 following LLM.int8).
* ``uniform_encode``     -- Quant(s, z, x) = round(x / s) - z, clamped to the n-bit range.
* ``uniform_levels``     -- the value s (q + z) each code q stands for, as float32.
* ``uniform_thresholds`` -- the smallest float32 whose code is at least j, for j = 1..2^n - 1;
                            by monotonicity these describe the same quantizer.
* ``sqnr_db``            -- reconstruction signal-to-quantization-noise ratio.
* ``relative_error``     -- ||y_hat - y|| / ||y|| of a product.

Readings:

* The paper gives Quant(s, z, x) = round(x / s) - z with a scaling factor and a zero-point and
  follows LLM.int8 for the asymmetric baseline; it does not print s and z. Read as min-max
  asymmetric quantization: s = (max w - min w) / (2^n - 1) and z = round(min w / s), so codes
  q = 0 .. 2^n - 1 decode to s (q + z), which spans [min w, max w] up to rounding.
* "A rounding function": ties round up (floor(v + 1/2)), the reading used for Eq. 1 as well.
* Codes outside 0 .. 2^n - 1 (only possible through the rounding of z) are clamped.
* Decisions are taken in float64 on float32 inputs: v = x / s, then floor(v + 1/2) - z.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

__all__ = ["UniformFit", "uniform_fit", "uniform_encode", "uniform_levels",
           "uniform_thresholds", "uniform_dequantize", "sqnr_db", "relative_error"]


class UniformError(ValueError):
    def __init__(self, kind: str, msg: str):
        super().__init__(f"{kind}: {msg}")
        self.kind = kind


@dataclass
class UniformFit:
    bits: int
    wmin: float      # min w (signed)
    wmax: float      # max w (signed)
    scale: float     # s
    zero: int        # z


def _round_half_up(v: float) -> float:
    return math.floor(v + 0.5)


def uniform_fit(w, bits: int = 4) -> UniformFit:
    """s and z of the asymmetric linear quantizer over the tensor's full range (Sec. 2)."""
    w = np.asarray(w)
    if w.dtype != np.float32:
        raise UniformError("invalid_arg", "weights must be float32")
    if bits < 2 or bits > 8:
        raise UniformError("invalid_arg", "bits out of range")
    if w.size < 2:
        raise UniformError("invalid_arg", "need at least two weights")
    if not np.all(np.isfinite(w)):
        raise UniformError("nonfinite", "weights contain NaN or Inf")
    lo = float(w.min())
    hi = float(w.max())
    if not (hi > lo):
        raise UniformError("degenerate", "all weights are equal")
    s = (hi - lo) / (2 ** bits - 1)
    z = int(_round_half_up(lo / s))
    return UniformFit(bits=bits, wmin=lo, wmax=hi, scale=s, zero=z)


def _code(x: float, s: float, z: int, bits: int) -> int:
    """Quant(s, z, x) = round(x / s) - z, clamped to [0, 2^n - 1] (Sec. 2)."""
    v = x / s
    if math.isnan(v):
        return 0
    if math.isinf(v):
        return 2 ** bits - 1 if v > 0 else 0
    q = int(_round_half_up(v)) - z
    return min(max(q, 0), 2 ** bits - 1)


def uniform_encode(x, s: float, z: int, bits: int = 4) -> np.ndarray:
    """Codes of every element of x (float32), uint8, by the definition above."""
    x = np.asarray(x, dtype=np.float32)
    v = x.astype(np.float64) / s                    # float64 division, correctly rounded
    q = np.floor(v + 0.5) - z
    q = np.where(np.isnan(q), 0, q)
    return np.clip(q, 0, 2 ** bits - 1).astype(np.uint8)


def uniform_levels(s: float, z: int, bits: int = 4) -> np.ndarray:
    """Dequantized value of every code: s (q + z), rounded to float32."""
    return np.array([np.float32(s * (q + z)) for q in range(2 ** bits)], dtype=np.float32)


def uniform_dequantize(codes: np.ndarray, levels: np.ndarray) -> np.ndarray:
    return levels[np.asarray(codes, dtype=np.int64)]


def uniform_thresholds(s: float, z: int, bits: int = 4) -> np.ndarray:
    """thr[j - 1] = smallest float32 x with code(x) >= j, j = 1 .. 2^n - 1 (+inf if none).

    The code is non-decreasing in x, so code(x) = #{j : x >= thr[j - 1]} for every float32 x
    that is not NaN. Found from the real boundary s (j + z - 1/2) by stepping through
    neighbouring float32 values with the exact rule above.
    """
    out = []
    for j in range(1, 2 ** bits):
        t = np.float32(s * (j + z - 0.5))
        if not np.isfinite(t):
            out.append(np.float32(np.inf) if t > 0 else np.float32(-np.inf))
            continue
        while _code(float(t), s, z, bits) >= j:
            t = np.nextafter(t, np.float32(-np.inf), dtype=np.float32)
        while _code(float(t), s, z, bits) < j:
            t = np.nextafter(t, np.float32(np.inf), dtype=np.float32)
            if not np.isfinite(t):
                break
        out.append(np.float32(t))
    return np.array(out, dtype=np.float32)


def sqnr_db(w, w_hat) -> float:
    """10 log10( sum w^2 / sum (w - w_hat)^2 ), in float64."""
    w = np.asarray(w, dtype=np.float64)
    e = w - np.asarray(w_hat, dtype=np.float64)
    return 10.0 * math.log10(float(np.sum(w * w)) / float(np.sum(e * e)))


def relative_error(y_hat, y) -> float:
    """||y_hat - y||_2 / ||y||_2, in float64."""
    y = np.asarray(y, dtype=np.float64)
    d = np.asarray(y_hat, dtype=np.float64) - y
    return float(np.linalg.norm(d) / np.linalg.norm(y))
