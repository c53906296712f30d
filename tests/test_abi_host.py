"""Host-side tests of liblogbq (no GPU): the library loads, exports every symbol the header
declares, validates arguments before any HIP call, and its host fit equals the oracle's
bit for bit (Sec. 3.1 Eq. 3-4, Sec. 3.2 Eq. 5)."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L
from stepped_rule import stepped_name, stepped_shape

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "logbq.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(logbq_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert {"logbq_fit", "logbq_encode", "logbq_linear", "logbq_dequantize", "logbq_linear8",
            "logbq_dequantize8", "logbq_status_str", "logbq_abi_version"} <= set(names)
    h = L.lib()
    for n in names:
        assert hasattr(h, n), n
    assert h.logbq_abi_version() == 2
    assert ctypes.sizeof(L.Params) == 4 + 4 + 8 * 4 + 4 + 4 + 8 + 4 * 256 + 4 * 128
    names_seen = {L.status_str(s) for s in range(7)}
    assert len(names_seen) == 7 and "unknown status" not in names_seen
    assert L.status_str(L.ERR_HOST_RESOURCE) == "host memory could not be allocated"
    assert L.status_str(99) == "unknown status"


def _cb():
    return (ctypes.c_float * 16)(*([0.0] + [2.0 ** (k - 7) for k in range(1, 8)] + [0.0] +
                                   [-(2.0 ** (k - 7)) for k in range(1, 8)]))


P = ctypes.c_void_p


def test_linear_validation_before_hip():
    h = L.lib()
    cb = _cb()
    a = P(4096)  # 16-byte aligned dummy address; never dereferenced on these paths
    assert h.logbq_linear(a, 1, 64, a, 4, None, a, None) == L.ERR_INVALID_ARG       # no codebook
    assert h.logbq_linear(a, -1, 64, a, 4, cb, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear(a, 1, -32, a, 4, cb, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear(a, 1, 64, a, -4, cb, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear(a, 1, 48, a, 4, cb, a, None) == L.ERR_UNSUPPORTED         # K % 32
    assert h.logbq_linear(a, 1, 64, a, 4, cb, None, None) == L.ERR_INVALID_ARG      # no y
    assert h.logbq_linear(None, 1, 64, a, 4, cb, a, None) == L.ERR_INVALID_ARG      # no x
    assert h.logbq_linear(a, 1, 64, None, 4, cb, a, None) == L.ERR_INVALID_ARG      # no codes
    assert h.logbq_linear(P(4100), 1, 64, a, 4, cb, a, None) == L.ERR_UNSUPPORTED   # misaligned
    assert h.logbq_linear(a, 1, 64, a, 4, cb, P(4104), None) == L.ERR_UNSUPPORTED
    bad = _cb()
    bad[3] = float("nan")
    assert h.logbq_linear(a, 1, 64, a, 4, bad, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear(a, 1, 2 ** 33, a, 4, cb, a, None) == L.ERR_UNSUPPORTED
    assert h.logbq_linear(a, 65535 * 64 + 1, 64, a, 4, cb, a, None) == L.ERR_UNSUPPORTED  # grid.y
    # empty calls succeed without touching the device
    assert h.logbq_linear(None, 0, 64, None, 4, cb, None, None) == L.OK
    assert h.logbq_linear(None, 3, 64, None, 0, cb, None, None) == L.OK


def test_encode_and_dequant_validation_before_hip():
    h = L.lib()
    p = L.fit(np.array([0.1, -0.5, 0.25, 1.0] * 8, dtype=np.float32))
    a = P(4096)
    assert h.logbq_encode(a, 4, 64, None, a, None, None) == L.ERR_INVALID_ARG
    assert h.logbq_encode(a, -1, 64, ctypes.byref(p), a, None, None) == L.ERR_INVALID_ARG
    assert h.logbq_encode(a, 4, 40, ctypes.byref(p), a, None, None) == L.ERR_UNSUPPORTED
    assert h.logbq_encode(None, 4, 64, ctypes.byref(p), a, None, None) == L.ERR_INVALID_ARG
    assert h.logbq_encode(P(4097), 4, 64, ctypes.byref(p), a, None, None) == L.ERR_UNSUPPORTED
    q = L.Params.from_buffer_copy(p)
    q.bits = 8                                                  # q_max still 7
    assert h.logbq_encode(a, 4, 64, ctypes.byref(q), a, None, None) == L.ERR_INVALID_ARG
    q.bits = 5
    assert h.logbq_encode(a, 4, 64, ctypes.byref(q), a, None, None) == L.ERR_UNSUPPORTED
    q = L.Params.from_buffer_copy(p)
    q.thresholds[2] = q.thresholds[1] / 2                      # not sorted
    assert h.logbq_encode(a, 4, 64, ctypes.byref(q), a, None, None) == L.ERR_INVALID_ARG
    cb = (ctypes.c_float * 16)()
    out = (ctypes.c_float * 16)()
    assert h.logbq_encode(None, 0, 64, ctypes.byref(p), None, out, None) == L.OK
    assert list(out) == list(p.codebook)[:16]
    assert h.logbq_dequantize(a, 4, 64, None, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_dequantize(a, 4, 33, cb, a, None) == L.ERR_UNSUPPORTED
    assert h.logbq_dequantize(None, 4, 64, cb, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_dequantize(a, 4, 64, cb, P(4098), None) == L.ERR_UNSUPPORTED
    assert h.logbq_dequantize(None, 0, 64, cb, None, None) == L.OK


def test_fit_errors_match_oracle():
    cases = [
        (np.array([1.0, np.nan], dtype=np.float32), L.ERR_NONFINITE, "nonfinite"),
        (np.array([1.0, -np.inf], dtype=np.float32), L.ERR_NONFINITE, "nonfinite"),
        (np.zeros(16, dtype=np.float32), L.ERR_DEGENERATE, "degenerate"),
        (np.array([0.5, -0.5, 0.5, 0.0], dtype=np.float32), L.ERR_DEGENERATE, "degenerate"),
        (np.array([0.5], dtype=np.float32), L.ERR_INVALID_ARG, "invalid_arg"),
    ]
    for w, status, kind in cases:
        with pytest.raises(L.LogbqError) as e:
            L.fit(w)
        assert e.value.status == status
        with pytest.raises(O.OracleError, match=kind):
            O.fit(w)
    for eps in (0.0, 1.0, -1e-3, float("nan")):
        with pytest.raises(L.LogbqError) as e:
            L.fit(np.array([0.5, 1.0], dtype=np.float32), eps=eps)
        assert e.value.status == L.ERR_INVALID_ARG
    for bits in (2, 3, 5, 16):
        with pytest.raises(L.LogbqError) as e:
            L.fit(np.array([0.5, 1.0], dtype=np.float32), bits=bits)
        assert e.value.status == L.ERR_UNSUPPORTED
    h = L.lib()
    assert h.logbq_fit(None, 4, 4, 4e-3, ctypes.byref(L.Params())) == L.ERR_INVALID_ARG


def _assert_fit_equal(w, eps=4e-3, bits=4):
    p = L.fit(w, bits, eps)
    r = O.fit(w, bits, eps)
    q = 2 ** (bits - 1) - 1
    assert p.bits == bits and p.qmax == q and p.eps == eps
    assert p.wmin == r.wmin and p.wmax == r.wmax
    assert p.wmin_index == r.wmin_index
    assert p.base == r.base, (p.base, r.base)
    assert p.shift == r.shift
    assert p.codebook_array().view(np.uint32).tolist() == \
        O.codebook(r.base, r.shift, bits).view(np.uint32).tolist()
    assert p.thresholds_array()[:q].view(np.uint32).tolist() == \
        O.magnitude_thresholds(r.base, r.shift, bits).view(np.uint32).tolist()
    assert all(np.isinf(p.thresholds[i]) for i in range(q, 128))
    assert all(p.codebook[i] == 0.0 for i in range(2 ** bits, 256))
    return p


def test_fit_bit_exact_random():
    rng = np.random.default_rng(123)
    for i in range(40):
        n = int(rng.integers(2, 5000))
        nu = [2.5, 3, 4, 8][i % 4]
        w = (rng.standard_t(nu, size=n) * 10 ** rng.uniform(-6, 2)).astype(np.float32)
        if i % 5 == 0:
            w[rng.integers(0, n, size=n // 3)] = 0.0
        if i % 7 == 0:
            w = np.round(w * 100) / 100                        # many duplicates
            w = w.astype(np.float32)
            if np.count_nonzero(w) < 2 or np.unique(np.abs(w[w != 0])).size < 2:
                continue
        eps = [4e-3, 1e-6, 0.1][i % 3]
        try:
            r = O.fit(w, 4, eps)
        except O.OracleError:
            continue
        del r
        _assert_fit_equal(w, eps)


def test_fit_golden_example():
    w = np.array([2.0 ** -7] * 66 + [1.0], dtype=np.float32)
    p = _assert_fit_equal(w)
    assert p.base == 2.0 and p.shift == 7 and p.wmin_index == 65


def test_fit_extreme_scales():
    rng = np.random.default_rng(9)
    base = rng.standard_t(3, size=3000).astype(np.float32)
    for s in (1e-30, 1e-12, 1e12, 1e30):
        _assert_fit_equal((base * np.float32(s)).astype(np.float32))
    sub = (rng.standard_t(3, size=3000) * 1e-41).astype(np.float32)   # subnormal weights
    sub = sub[np.abs(sub) > 0]
    try:
        O.fit(sub)
    except O.OracleError:
        return
    _assert_fit_equal(sub)


@pytest.mark.parametrize("name", ["linear_2048x2048", "up_2048x8192_outliers"])
def test_fit_bit_exact_workload_tensors(name):
    wl = inputs.WORKLOADS[name]
    lin = wl["layers"][0]
    w = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"],
                                 seed=[wl["cfg"], 0, 0, 0], outlier_frac=wl["outlier_frac"])
    _assert_fit_equal(w)


def test_fit8_bit_exact_random():
    """The 8-bit fit (q_max = 127, eps = 1e-6 as in Sec. 3.2) equals the oracle bit for bit:
    w_min, w_max, b, s, all 256 codebook entries and all 127 exact thresholds."""
    rng = np.random.default_rng(808)
    done = 0
    for i in range(16):
        n = int(rng.integers(64, 20000))
        w = (rng.standard_t([3, 4, 8][i % 3], size=n) * 10 ** rng.uniform(-5, 1)).astype(np.float32)
        eps = [1e-6, 1e-3, 0.05][i % 3]
        try:
            O.fit(w, 8, eps)
        except O.OracleError:
            continue
        _assert_fit_equal(w, eps, bits=8)
        done += 1
    assert done >= 10


def test_8bit_validation_before_hip():
    h = L.lib()
    cb = (ctypes.c_float * 256)(*([0.0] * 256))
    a = P(4096)
    assert h.logbq_linear8(a, 1, 64, a, 4, None, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear8(a, 1, 48, a, 4, cb, a, None) == L.ERR_UNSUPPORTED
    assert h.logbq_linear8(a, 1, 64, a, 4, cb, None, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear8(P(4100), 1, 64, a, 4, cb, a, None) == L.ERR_UNSUPPORTED
    bad = (ctypes.c_float * 256)(*([0.0] * 256))
    bad[200] = float("inf")                     # an entry only an 8-bit call reads
    assert h.logbq_linear8(a, 1, 64, a, 4, bad, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_linear8(None, 0, 64, None, 4, cb, None, None) == L.OK
    assert h.logbq_dequantize8(a, 4, 64, None, a, None) == L.ERR_INVALID_ARG
    assert h.logbq_dequantize8(a, 4, 48, cb, a, None) == L.ERR_UNSUPPORTED
    assert h.logbq_dequantize8(None, 0, 64, cb, None, None) == L.OK
    p = L.fit(np.array([0.1, -0.5, 0.25, 1.0] * 8, dtype=np.float32), bits=8)
    assert p.bits == 8 and p.qmax == 127
    out = (ctypes.c_float * 256)()
    assert h.logbq_encode(None, 0, 64, ctypes.byref(p), None, out, None) == L.OK
    assert list(out) == list(p.codebook)
    p.bits = 6
    assert h.logbq_encode(a, 1, 64, ctypes.byref(p), a, None, None) == L.ERR_UNSUPPORTED


def test_linear_path_rule():
    """Path choice is host logic: checked here without a device."""
    lp = L.linear_path
    assert lp(4, 1, 8192, 28672) == "gemv"
    assert lp(4, 0, 8192, 28672) == "none" and lp(4, 4, 0, 100) == "none"
    assert lp(4, 4, 64, 0) == "none"
    # split-K kernel: 4-bit, 2 <= m <= 16, K in {1, 2, 4, 8} Ki
    assert lp(4, 8, 8192, 28672) == "splitk"
    assert lp(4, 16, 2048, 8192) == "splitk"
    assert lp(4, 16, 8192, 28672) == "splitk"
    assert lp(4, 3, 4096, 4096) == "splitk" and lp(4, 3, 4096, 2048) == "gemv"
    assert lp(4, 4, 4096, 1024) == "splitk" and lp(4, 4, 8192, 1024) == "gemv"
    assert lp(4, 4, 8192, 2048) == "splitk" and lp(4, 2, 8192, 28672) == "gemv"
    assert lp(4, 8, 8192 + 32, 28672) == "mfma"    # K outside the split-K set
    assert lp(4, 17, 8192, 2048) == "splitk" and lp(4, 32, 8192, 16384) == "splitk"
    assert lp(4, 20, 8192, 28672) == "splitk" and lp(4, 21, 8192, 28672) == "mfma"
    assert lp(4, 32, 4096, 28672) == "splitk" and lp(4, 33, 4096, 4096) == "mfma"
    assert lp(4, 4, 14336, 4096) == "splitk" and lp(4, 16, 14336, 4096) == "splitk"
    assert lp(4, 17, 14336, 4096) == "mfma" and lp(4, 48, 14336, 4096) == "mfma"
    assert lp(4, 96, 8192, 28672) == "mfma"
    # K-quartered MFMA GEMM: 4-bit, m > 96 at N >= 4096, unless the stepped kernel's 64-row
    # grid fits on the chip (ceil(N / 64) x ceil(m / 128) <= 256 workgroups)
    assert lp(4, 128, 8192, 28672) == "mfma_kq" and lp(4, 97, 1024, 16448) == "mfma_kq"
    assert lp(4, 97, 1024, 4096) == "mfma" and lp(4, 128, 1024, 16384) == "mfma"
    assert lp(4, 129, 1024, 8192) == "mfma" and lp(4, 129, 1024, 8256) == "mfma_kq"
    assert lp(4, 128, 1024, 4095) == "mfma" and lp(8, 128, 8192, 28672) == "mfma_kq"
    assert lp(8, 65, 8192, 16384) == "mfma_kq" and lp(8, 64, 8192, 28672) == "mfma"
    assert lp(8, 128, 4096, 14336) == "mfma"
    # 8-bit codes: split-K for K in {2, 4, 8} Ki at 5 <= m <= 8 (not N <= 1024 at K >= 4096),
    # m = 3, 4 from N = 8192, 9 <= m <= 16 (not N > 16384 at K = 8192); else GEMV unless m >= 5
    # and m * N > 65536, else the stepped MFMA kernel
    assert lp(8, 1, 8192, 28672) == "gemv" and lp(8, 2, 8192, 28672) == "gemv"
    assert lp(8, 3, 8192, 28672) == "splitk" and lp(8, 4, 4096, 4096) == "gemv"
    assert lp(8, 5, 8192, 28672) == "splitk" and lp(8, 8, 2048, 8192) == "splitk"
    assert lp(8, 8, 8192, 1024) == "gemv" and lp(8, 8, 2048, 1024) == "splitk"
    assert lp(8, 16, 8192, 16384) == "splitk" and lp(8, 16, 8192, 28672) == "mfma"
    assert lp(8, 8, 6144, 28672) == "mfma" and lp(8, 17, 4096, 4096) == "mfma"
    for bad in ((4, -1, 64, 1), (4, 1, 64, -1)):
        with pytest.raises(L.LogbqError):
            lp(*bad)
    for bad in ((5, 1, 64, 1), (4, 1, 48, 1), (8, 1 << 40, 64, 1)):
        with pytest.raises(L.LogbqError):
            lp(*bad)


def test_stepped_shape_rule():
    """The library's stepped-kernel launch shapes agree with the rule stated in stepped_rule on
    every shape of a grid (ragged n, k from 1 to 56 steps, m from 3 to 256) that takes that
    kernel, for register tables, the 4-bit LDS table and 8-bit codes, and each rule reaches
    every kind of shape (64- and 128-row workgroups, one and two K parts)."""
    table = np.linspace(-0.07, 0.08, 16, dtype=np.float32)     # not sign-symmetric
    for kind in ("register", "table4", "bits8"):
        bits = 8 if kind == "bits8" else 4
        cb = table if kind == "table4" else None
        seen = set()
        for k in (1024, 2048, 3072, 4096, 8192, 14336):
            for n in (64, 1000, 2048, 4097, 8192, 14336, 16385, 28672):
                for m in (3, 9, 17, 33, 48, 64, 65, 96, 97, 128, 129, 200, 256):
                    if L.linear_path(bits, m, k, n) not in ("mfma", "mfma_kq"):
                        continue
                    name = L.linear_kernel(bits, m, k, n, cb)
                    if name.startswith("k_mfma_kq") or name.startswith("k_mfma_sk"):
                        continue
                    assert name == stepped_name(m, k, n, kind), (kind, m, k, n)
                    narrow, t, parts = stepped_shape(m, k, n, kind)
                    seen.add((narrow, parts))
        assert seen == {(True, 1), (True, 2), (False, 1), (False, 2)}, kind


def test_linear_kernel_names():
    """The kernel instance a call runs, named as the profiler lists it (host logic)."""
    lk = L.linear_kernel
    assert lk(4, 1, 8192, 28672) == "k_gemv<4, 1, 4, false, 2>"
    assert lk(4, 1, 14336, 4096) == "k_gemv<4, 1, 4, true, 2>"      # two wavefronts per row
    assert lk(4, 1, 2048, 2048) == "k_gemv<4, 1, 1, false, 3>"
    assert lk(4, 8, 8192, 28672) == "k_mfma_sk<16, 16, 2, 1, 1, false>"   # 2 batch groups
    assert lk(4, 12, 8192, 28672) == "k_mfma_sk<16, 16, 1, 1, 1, false>"
    assert lk(4, 4, 4096, 14336) == "k_mfma_sk<8, 16, 2, 1, 1, false>"
    assert lk(4, 8, 2048, 8192) == "k_mfma_sk<8, 8, 2, 1, 1, false>"
    assert lk(4, 32, 4096, 14336) == "k_mfma_sk<8, 16, 1, 2, 1, false>"   # two batch tiles
    assert lk(4, 32, 8192, 2048) == "k_mfma_sk<8, 16, 1, 2, 2, false>"    # K over 2 workgroups
    assert lk(4, 32, 1024, 4096) == "k_mfma_sk<4, 8, 1, 2, 1, false>"
    assert lk(4, 4, 14336, 4096) == "k_mfma_sk<16, 14, 2, 1, 2, false>"   # K over 2 workgroups
    # narrow layers split K over workgroup pairs (per linear, from its own n)
    assert lk(4, 4, 8192, 2048) == "k_mfma_sk<8, 16, 2, 1, 2, false>"
    assert lk(4, 8, 8192, 2049) == "k_mfma_sk<16, 16, 2, 1, 1, false>"
    assert lk(4, 16, 8192, 8192) == "k_mfma_sk<8, 16, 1, 1, 2, false>"
    assert lk(4, 16, 8192, 8193) == "k_mfma_sk<16, 16, 1, 1, 1, false>"
    assert lk(4, 16, 4096, 2048) == "k_mfma_sk<4, 16, 1, 1, 2, false>"
    assert lk(4, 12, 4096, 2048) == "k_mfma_sk<8, 16, 1, 1, 1, false>"
    assert lk(4, 32, 8192, 28672) == "k_mfma2<4, 2, 4, false, true>"
    assert lk(4, 128, 8192, 28672) == "k_mfma_kq"
    assert lk(4, 9, 14336, 4096) == "k_mfma_sk<16, 14, 1, 1, 2, false>"
    assert lk(4, 16, 14336, 4096) == "k_mfma_sk<16, 14, 1, 1, 2, false>"
    assert lk(4, 17, 14336, 4096) == "k_mfma2_narrow<4, 1, false, true>"
    # register tables: the cheapest launch shape whose grid fits on the chip (cost model)
    assert lk(4, 49, 14336, 4096) == "k_mfma2_narrow<4, 2, false, true>"
    assert lk(4, 64, 4096, 4096) == "k_mfma2_narrow<4, 1, false, true>"
    assert lk(4, 128, 4096, 4096) == "k_mfma2_narrow<4, 2, false, true>"
    assert lk(4, 128, 14336, 4096) == "k_mfma2<4, 2, 4, false, true>"
    assert lk(4, 256, 4096, 4096) == "k_mfma2<4, 2, 4, false, true>"
    assert lk(4, 64, 4096, 14336) == "k_mfma2<4, 2, 4, false, true>"
    assert lk(4, 128, 4096, 14336) == "k_mfma2<4, 4, 4, false, false>"
    assert lk(4, 33, 4096, 16384) == "k_mfma2_narrow<4, 3, false, false>"
    assert lk(4, 33, 4096, 16385) == "k_mfma2<4, 3, 4, false, false>"
    assert lk(4, 129, 1024, 8192) == "k_mfma2<4, 4, 4, false, false>"
    assert lk(4, 129, 1024, 8256) == "k_mfma_kq"
    for m, k, n in ((64, 8192, 28672), (96, 8192, 28672), (48, 8192, 16385), (200, 2048, 1000)):
        assert lk(4, m, k, n) == stepped_name(m, k, n), (m, k, n)
    assert lk(8, 1, 8192, 28672) == "k_gemv<8, 1, 8, false, 2>"
    assert lk(8, 128, 8192, 28672) == "k_mfma_kq8" and lk(8, 128, 4096, 14336) == "k_mfma2<8, 4, 4, true, false>"
    assert lk(8, 64, 4096, 14336) == "k_mfma2<8, 2, 4, true, true>"
    assert lk(8, 32, 8192, 28672) == "k_mfma2<8, 2, 4, true, true>"
    assert lk(8, 8, 8192, 28672) == "k_mfma_sk8<16, 2>" and lk(8, 12, 4096, 4096) == "k_mfma_sk8<8, 1>"
    assert lk(4, 0, 8192, 28672) == "none" and lk(4, 3, 0, 5) == "k_fill_zero"
    # a codebook that is not sign-symmetric takes the LDS table
    cb = np.arange(16, dtype=np.float32)
    assert lk(4, 8, 8192, 28672, cb) == "k_mfma_sk<32, 8, 1, 1, 1, true>"
    assert lk(4, 32, 4096, 14336, cb) == "k_mfma2<4, 1, 4, true, true>"   # above m = 16
    assert lk(4, 4, 14336, 4096, cb) == "k_mfma2_narrow<4, 1, true, true>"    # and at K = 14336
    assert lk(4, 128, 8192, 28672, cb) == "k_mfma2<4, 4, 4, true, false>"
    assert lk(4, 64, 4096, 4096, cb) == "k_mfma2_narrow<4, 1, true, true>"
    assert lk(4, 65, 4096, 16384, cb) == "k_mfma2<4, 4, 4, true, false>"   # two 64-row blocks
    assert lk(4, 64, 4096, 16384, cb) == "k_mfma2<4, 2, 4, true, true>"
    sym = np.array([0] + [2.0 ** k for k in range(1, 8)] + [0] + [-(2.0 ** k) for k in range(1, 8)],
                   dtype=np.float32)
    assert lk(4, 128, 8192, 28672, sym) == "k_mfma_kq"
    h = L.lib()
    small = ctypes.create_string_buffer(4)
    assert h.logbq_linear_kernel(4, 1, 64, 8, None, small, 4) == L.ERR_INVALID_ARG
    assert h.logbq_linear_kernel(4, 1, 64, 8, None, None, 96) == L.ERR_INVALID_ARG
    assert h.logbq_linear_kernel(5, 1, 64, 8, None, small, 4) == L.ERR_UNSUPPORTED


@pytest.mark.parametrize("scale", [1e-35, 1e30])
def test_fit8_extreme_shift_thresholds(scale):
    """An 8-bit codebook (b near 1) on weights far from 1 has a shift s in the thousands; its
    exact thresholds need b^n for n near 2 s. They equal the oracle's and take well under a
    second (the fit builds each power once by squaring)."""
    import time
    w = (np.random.default_rng(3).standard_t(3, 4000) * scale).astype(np.float32)
    t0 = time.perf_counter()
    p = L.fit(w, 8, 0.5)
    dt = time.perf_counter() - t0
    r = O.fit(w, 8, 0.5)
    assert abs(p.shift) > 1000 and p.shift == r.shift and p.base == r.base
    assert p.thresholds_array()[:127].view(np.uint32).tolist() == \
        O.magnitude_thresholds(r.base, r.shift, 8).view(np.uint32).tolist()
    assert dt < 5.0, dt


@pytest.mark.parametrize("threads", ["1", "3", "16"])
def test_fit_same_for_any_sort_thread_count(threads, monkeypatch):
    """The host fit's radix sort splits each pass over LOGBQ_HOST_THREADS ranges (one range
    runs without starting a thread); the parameters are the same for any count and equal the
    oracle's (3 * 2^20 + 5 weights, so the threaded path is taken)."""
    w = inputs.student_t_weights(3 * 2 ** 20 + 5, 1, 4, 0.02, seed=[71, 0, 0, 0]).reshape(-1)
    monkeypatch.setenv("LOGBQ_HOST_THREADS", threads)
    p = L.fit(w)
    r = O.fit(w)
    assert (p.wmin, p.wmax, p.wmin_index, p.base, p.shift) == \
        (r.wmin, r.wmax, r.wmin_index, r.base, r.shift)
