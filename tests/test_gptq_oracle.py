"""Pins of the GPTQ oracle (the calibration of Sec. 4, with LogbQuant's or the baseline's
quantizer in its loop) against facts that do not come from its own code: with U = I there is
nothing to compensate and GPTQ is round-to-nearest; one compensation step equals the
least-squares update computed directly from the calibration inputs; the layer-output error it
minimises drops against round-to-nearest. Also the library's argument checks (no GPU needed)."""
import ctypes

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
