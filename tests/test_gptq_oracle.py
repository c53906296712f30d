"""Pins of the GPTQ oracle (the calibration of Sec. 4, with LogbQuant's or the baseline's
quantizer in its loop) against facts that do not come from its own code: with U = I there is
nothing to compensate and GPTQ is round-to-nearest; one compensation step equals the
least-squares update computed directly from the calibration inputs; the layer-output error it
minimises drops against round-to-nearest. Also the library's argument checks (no GPU needed)."""
import ctypes
import math

import numpy as np
import pytest

from oracle import gptq_oracle as G
from oracle import logbq_oracle as O
from oracle import uniform_oracle as U
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L


def _weights(n, k, seed):
    return np.asarray(inputs.student_t_weights(n, k, 4, 0.02, seed=seed))


def _inputs(t, k, seed):
    """Correlated calibration inputs: per-channel scales and a shared low-rank part."""
    rng = np.random.default_rng(seed)
    scale = np.exp(rng.normal(0.0, 0.5, k))
    x = rng.standard_normal((t, k)) * scale + rng.standard_normal((t, 8)) @ rng.standard_normal((8, k)) * 0.5
    return x.astype(np.float32)


def _quantizers(w):
    r = O.fit(w)
    lut = O.codebook(r.base, r.shift)
    f = U.uniform_fit(w)
    lv = U.uniform_levels(f.scale, f.zero)

    def ql(col):
        c = O.encode(col, r.base, r.shift)
        return c, lut[c]

    def qu(col):
        c = U.uniform_encode(col, f.scale, f.zero)
        return c, lv[c]
    return (ql, lut, lambda ww: O.encode(ww, r.base, r.shift)), \
           (qu, lv, lambda ww: U.uniform_encode(ww, f.scale, f.zero))


@pytest.mark.parametrize("k", [96, 256, 300 // 32 * 32])
def test_identity_factor_is_round_to_nearest(k):
    w = _weights(40, k, [41, k, 0, 0])
    for q, lut, rtn in _quantizers(w):
        codes, wc = G.gptq(w, np.eye(k, dtype=np.float32), q)
        assert np.array_equal(codes, rtn(w))
        assert np.array_equal(wc, w)


def test_one_step_is_least_squares():
    """Two columns, no damping: after column 0 is rounded, column 1 becomes
    w1 + (w0 - q0) (x0 . x1) / (x1 . x1), the minimiser of ||(w0 - q0) x0 + (w1 - w1') x1||."""
    rng = np.random.default_rng(42)
    x = rng.standard_normal((500, 2)).astype(np.float32)
    x[:, 1] += np.float32(0.7) * x[:, 0]
    w = (rng.standard_normal((16, 2)) * 0.05).astype(np.float32)
    for q, lut, rtn in _quantizers(w):
        _, wc = G.gptq(w, G.hessian_factor(x, damp=0.0), q)
        xd = x.astype(np.float64)
        q0 = lut[rtn(w[:, :1])[:, 0]].astype(np.float64)
        ls = w[:, 1] + (w[:, 0] - q0) * (xd[:, 0] @ xd[:, 1]) / (xd[:, 1] @ xd[:, 1])
        assert np.max(np.abs(wc[:, 1] - ls)) <= 1e-6 * max(1.0, np.max(np.abs(ls)))


def test_factor_is_inverse_hessian_cholesky():
    x = _inputs(400, 64, 43)
    u = G.hessian_factor(x).astype(np.float64)
    h = 2.0 * x.astype(np.float64).T @ x.astype(np.float64) / 400
    h += 0.01 * np.mean(np.diag(h)) * np.eye(64)
    assert np.allclose(np.triu(u), u)
    assert np.allclose(u.T @ u @ h, np.eye(64), atol=1e-4)


@pytest.mark.parametrize("k", [256, 384])
def test_gptq_reduces_output_error(k):
    w = _weights(64, k, [44, k, 0, 0])
    x = _inputs(4 * k, k, 45)
    u = G.hessian_factor(x)
    for q, lut, rtn in _quantizers(w):
        codes, _ = G.gptq(w, u, q)
        e_gptq = G.output_error(w, lut[codes], x)
        e_rtn = G.output_error(w, lut[rtn(w)], x)
        assert e_gptq < 0.85 * e_rtn, (e_gptq, e_rtn)


def test_gptq_argument_checks():
    p = L.Params()
    u = L.Uniform()
    h = L.lib()
    ok = ctypes.c_void_p(16)
    # neither or both quantizers
    assert h.logbq_gptq(ok, 4, 32, ok, None, None, ok, ok, None) == 1
    assert h.logbq_gptq(ok, 4, 32, ok, ctypes.byref(p), ctypes.byref(u), ok, ok, None) == 1
    # bits / k % 32
    assert h.logbq_gptq(ok, 4, 32, ok, ctypes.byref(p), None, ok, ok, None) == 4   # p.bits = 0
    w = _weights(8, 64, [46, 0, 0, 0])
    fp = L.fit(w)
    assert h.logbq_gptq(ok, 4, 48, ok, ctypes.byref(fp), None, ok, ok, None) == 4
    assert h.logbq_gptq(None, 4, 64, ok, ctypes.byref(fp), None, ok, ok, None) == 1
    assert h.logbq_gptq(ok, 2 ** 21, 64, ok, ctypes.byref(fp), None, ok, ok, None) == 4
    assert h.logbq_gptq(None, 0, 64, None, ctypes.byref(fp), None, None, None, None) == 0


# ---------------------------------------------------------------- after-block path and mutants
#
# GPTQ's lazy batch updates apply a block's errors to the later columns only after the block
# (the after-block path). With no damping, the sequential update is ordinary least squares:
# once columns 0 .. i-1 are fixed at their rounded values q, column i becomes
#   w_i + sum_{j<i} (w_j - q_j) x_j . x_i / (x_i . x_i)   (for i = 1 with one column fixed)
# and, in general, the minimiser of ||sum_j (w_j - w'_j) x_j|| over the free column given the
# fixed ones. The pins below compute these minimisers from X with numpy least squares, so they
# do not depend on U or on the block structure, and run them with block sizes that send every
# update through the after-block path (block = 1), through both paths (block = 2 on three
# columns), and through the in-block path only (block = 128).

def _three_col_inputs(seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((600, 3))
    x[:, 1] += 0.7 * x[:, 0]
    x[:, 2] += 0.5 * x[:, 0] - 0.6 * x[:, 1]
    w = rng.standard_normal((24, 3)) * 0.05
    return x.astype(np.float32), w.astype(np.float32)


def _least_squares_column(x, w, fixed_vals, col):
    """Column `col` of the minimiser of ||sum_j (w_j - w'_j) x_j|| over the columns col, col + 1,
    ... (all still free when column col - 1 is rounded), every earlier column j fixed at
    fixed_vals[:, j]: numpy least squares from X directly (float64)."""
    xd = x.astype(np.float64)
    resid = (w[:, :col].astype(np.float64) - fixed_vals[:, :col]) @ xd[:, :col].T   # [N][T]
    delta, *_ = np.linalg.lstsq(xd[:, col:], resid.T, rcond=None)                  # [free][N]
    return w[:, col].astype(np.float64) + delta[0]


def _pin_sequential_least_squares(gptq_fn, block, seed):
    """True when every compensated column equals the least-squares minimiser given the rounded
    earlier columns (which the oracle reports through its codes)."""
    x, w = _three_col_inputs(seed)
    ok = True
    for q, lut, rtn in _quantizers(w):
        codes, wc = gptq_fn(w, G.hessian_factor(x, damp=0.0), q, block=block)
        qv = lut[codes].astype(np.float64)
        for col in (1, 2):
            ls = _least_squares_column(x, w, qv, col)
            ok &= bool(np.max(np.abs(wc[:, col] - ls)) <= 1e-7 * max(1.0, np.max(np.abs(ls))))
        # and every code is the rounding of the column it was taken from
        ok &= bool(np.array_equal(codes, rtn(wc)))
    return ok


@pytest.mark.parametrize("block", [1, 2, 128])
def test_sequential_updates_are_least_squares(block):
    assert _pin_sequential_least_squares(G.gptq, block, 47)
    assert _pin_sequential_least_squares(G.gptq, block, 48)


def test_one_step_least_squares_through_after_block_path():
    """The two-column pin above with block = 1: column 1 is compensated by the after-block
    update alone."""
    rng = np.random.default_rng(42)
    x = rng.standard_normal((500, 2)).astype(np.float32)
    x[:, 1] += np.float32(0.7) * x[:, 0]
    w = (rng.standard_normal((16, 2)) * 0.05).astype(np.float32)
    for q, lut, rtn in _quantizers(w):
        _, wc = G.gptq(w, G.hessian_factor(x, damp=0.0), q, block=1)
        xd = x.astype(np.float64)
        q0 = lut[rtn(w[:, :1])[:, 0]].astype(np.float64)
        ls = w[:, 1] + (w[:, 0] - q0) * (xd[:, 0] @ xd[:, 1]) / (xd[:, 1] @ xd[:, 1])
        assert np.max(np.abs(wc[:, 1] - ls)) <= 1e-6 * max(1.0, np.max(np.abs(ls)))


def test_blocked_equals_single_block():
    """Lazy batching reorders the same updates: blocks of 128 and one block of K give the same
    codes and weights equal to float32 rounding."""
    w = _weights(64, 384, [49, 0, 0, 0])
    x = _inputs(1536, 384, 50)
    u = G.hessian_factor(x)
    for q, lut, rtn in _quantizers(w):
        c1, w1 = G.gptq(w, u, q, block=128)
        c2, w2 = G.gptq(w, u, q, block=384)
        assert np.array_equal(c1, c2)
        assert np.max(np.abs(w1 - w2)) <= 1e-5 * np.max(np.abs(w))


def test_output_error_hand_value():
    """W = [[1, 2], [3, 4]], W_hat = [[1, 2], [3, 3]], X = [[1, 1], [0, 2], [1, 0]] (T = 3):
    W X^T = [[3, 4, 1], [7, 8, 3]], squared norm 9 + 16 + 1 + 49 + 64 + 9 = 148;
    (W - W_hat) X^T = [[0, 0, 0], [1, 2, 0]], squared norm 5; the error is sqrt(5 / 148)."""
    w = np.array([[1, 2], [3, 4]], dtype=np.float32)
    wh = np.array([[1, 2], [3, 3]], dtype=np.float32)
    x = np.array([[1, 1], [0, 2], [1, 0]], dtype=np.float32)
    assert G.output_error(w, wh, x) == pytest.approx(math.sqrt(5.0 / 148.0), rel=1e-15)
    assert G.output_error(w, w, x) == 0.0


def _mutant(kind):
    """A copy of the oracle's column loop with one plausible mistake planted."""
    def gptq(w, u, quantize, block=G.BLOCK):
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
                d = w[:, i] - q.astype(np.float32)
                e = d if kind == "no_divide" else d / u[i, i]
                err[:, i - i1] = e
                if i + 1 < i2:
                    upd = e[:, None] * u[i, i + 1:i2][None, :]
                    w[:, i + 1:i2] = w[:, i + 1:i2] + upd if kind == "in_block_sign" else \
                        w[:, i + 1:i2] - upd
            if i2 < k and kind != "drop_after_block":
                acc = np.zeros((n, k - i2), dtype=np.float32)
                for i in range(i1, i2):
                    row = u[i2:, i] if kind == "transposed_after_block" else u[i, i2:]
                    acc = acc + err[:, i - i1][:, None] * row[None, :]
                w[:, i2:] = w[:, i2:] - acc
        return codes, w
    return gptq


@pytest.mark.parametrize("kind", ["drop_after_block", "transposed_after_block", "no_divide",
                                  "in_block_sign"])
def test_pins_catch_planted_gptq_mistakes(kind):
    """Each planted mistake fails the least-squares pins at some block size (the block size
    decides which path a mistake in one of them can reach)."""
    fn = _mutant(kind)
    results = [_pin_sequential_least_squares(fn, b, s) for b in (1, 2, 128) for s in (47, 48)]
    assert not all(results), f"planted mistake {kind} passed every pin"
