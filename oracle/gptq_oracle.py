"""Plain CPU oracle of GPTQ post-training calibration (Frantar et al., the calibration the
LogbQuant paper uses for every model, Sec. 2 and Sec. 4) with the LogbQuant quantizer (Eq. 1-2)
or the asymmetric linear baseline (Sec. 2) in its inner loop.

TEST INFRASTRUCTURE ONLY, like ``logbq_oracle``: only the tests and ``bench.py``'s CPU legs may
use it. It shares no code with the HIP library.

* ``hessian_factor`` -- from calibration inputs X [T][K]: H = 2 X^T X / T, columns that no
                        input touches get H_ii = 1, damping adds 1 % of the mean diagonal, and U
                        is the upper Cholesky factor of H^-1 (float64, returned as float32).
* ``gptq``           -- the column loop in blocks of 128 columns, in float32: quantize column i,
                        err = (w_i - q_i) / U_ii, subtract err * U_ij from every later column j
                        of the block; after the block, subtract sum_i err_i * U_i,j from every
                        column j after it.
* ``output_error``   -- ||(W - W_hat) X^T||_F / ||W X^T||_F, the layer-output error GPTQ reduces.

Readings:

* The paper calibrates with GPTQ but prints no algorithm; the steps are GPTQ's (Algorithm 1 of
  its paper, lazy batch updates with blocks of 128 columns, 1 % damping), in float32 as in its
  reference implementation.
* The quantizer's parameters (LogbQuant's b and s, the baseline's s and z) are fitted once on
  the original weights before the column loop, as GPTQ does for per-tensor quantizers; the loop
  only rounds columns to that fixed codebook.
* Operation order, which fixes every rounding: err = (w - q) / U_ii; in-block update
  w_j = w_j - err * U_ij (product rounded, then difference); the after-block update accumulates
  acc = acc + err_i * U_ij over the block's columns in increasing i starting from 0 (each
  product and sum rounded) and then w_j = w_j - acc. No fused multiply-add.
* Zero columns of W for inputs that are never active follow from the caller's data: here only
  the Hessian gets H_ii = 1 (the weights are kept), so the function is defined for any W.
"""
from __future__ import annotations

import numpy as np

__all__ = ["hessian_factor", "gptq", "output_error", "BLOCK"]

BLOCK = 128


def hessian_factor(x: np.ndarray, damp: float = 0.01) -> np.ndarray:
    """Upper Cholesky factor U of H^-1, H = 2 X^T X / T + damp * mean(diag H) * I (float32)."""
    x = np.asarray(x, dtype=np.float64)
    t, k = x.shape
    h = 2.0 * (x.T @ x) / t
    dead = np.diag(h) == 0
    h[dead, dead] = 1.0
    h += damp * float(np.mean(np.diag(h))) * np.eye(k)
    lower = np.linalg.cholesky(h)                      # H = L L^T
    hinv = np.linalg.inv(lower).T @ np.linalg.inv(lower)
    hinv = (hinv + hinv.T) / 2
    u = np.linalg.cholesky(hinv).T                     # H^-1 = U^T U, U upper triangular
    return np.triu(u).astype(np.float32)


def gptq(w: np.ndarray, u: np.ndarray, quantize, block: int = BLOCK):
    """GPTQ on W [N][K] (float32) with the upper factor U [K][K] (float32).

    quantize(column float32 [N]) -> (codes uint8 [N], values float32 [N]) rounds one column to
    the fixed codebook. Returns (codes [N][K] uint8, compensated weights [N][K] float32: every
    column as it was when it was quantized)."""
    w = np.array(w, dtype=np.float32, copy=True)
    u = np.asarray(u, dtype=np.float32)
    n, k = w.shape
    codes = np.zeros((n, k), dtype=np.uint8)
    for i1 in range(0, k, block):
        i2 = min(i1 + block, k)
        err = np.zeros((n, i2 - i1), dtype=np.float32)
        for i in range(i1, i2):
            c, q = quantize(w[:, i])
            codes[:, i] = c
            e = (w[:, i] - q.astype(np.float32)) / u[i, i]
            err[:, i - i1] = e
            if i + 1 < i2:
                w[:, i + 1:i2] = w[:, i + 1:i2] - e[:, None] * u[i, i + 1:i2][None, :]
        if i2 < k:
            acc = np.zeros((n, k - i2), dtype=np.float32)
            for i in range(i1, i2):
                acc = acc + err[:, i - i1][:, None] * u[i, i2:][None, :]
            w[:, i2:] = w[:, i2:] - acc
    return codes, w


def output_error(w: np.ndarray, w_hat: np.ndarray, x: np.ndarray) -> float:
    """||(W - W_hat) X^T||_F / ||W X^T||_F in float64."""
    w = np.asarray(w, dtype=np.float64)
    d = w - np.asarray(w_hat, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    return float(np.linalg.norm(d @ x.T) / np.linalg.norm(w @ x.T))
