"""GPU parity of logbq_fit_device (Sec. 3.2 Eq. 5 with exact sums, Sec. 3.1 Eq. 3-4) through the
C ABI: every field of the parameters bit for bit against the oracle's ``fit_exact`` at sizes
it finishes in seconds (spanning several workgroups and a ragged tail), the error statuses,
and at the full 8192 x 28672 size a certificate of w_min in exact integer arithmetic plus
equality with the host run of the same passes (logbq_fit_exact) and with the host fit."""
import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
CHUNK = 1 << 18          # weights per workgroup of passes 2 and 3 (twice that in pass 1)


def _say(msg):
    print(msg, flush=True)


def _assert_params(p, r, bits):
    q = 2 ** (bits - 1) - 1
    assert p.bits == bits and p.qmax == q
    assert (p.wmin, p.wmax, p.wmin_index) == (r.wmin, r.wmax, r.wmin_index)
    assert p.base == r.base and p.shift == r.shift
    assert p.codebook_array().view(np.uint32).tolist() == \
        O.codebook(r.base, r.shift, bits).view(np.uint32).tolist()
    assert p.thresholds_array()[:q].view(np.uint32).tolist() == \
        O.magnitude_thresholds(r.base, r.shift, bits).view(np.uint32).tolist()


def _t(n, nu, scale, seed, outl=0.0):
    rng = np.random.default_rng(seed)
    w = (rng.standard_t(nu, n) * scale).astype(np.float32)
    if outl:
        pos = rng.choice(n, int(round(outl * n)), replace=False)
        w[pos] = np.float32(20 * scale) * rng.choice([-1, 1], pos.size).astype(np.float32)
    return w


def _cases():
    c = [("t4 1e6", _t(1_000_000, 4, 0.02, 1), 4, 4e-3),
         ("t3 outliers", _t(2048 * 512, 4, 0.02, 2, outl=1e-4), 4, 4e-3),
         ("8-bit", _t(768 * 1024, 3, 0.015, 3), 8, 1e-6),
         ("chunk + 3", _t(CHUNK + 3, 4, 0.02, 4), 4, 4e-3),
         ("3 chunks", _t(3 * CHUNK, 6, 1.0, 5), 4, 0.1),
         ("ragged 300001", _t(300_001, 4, 0.02, 6), 4, 4e-3),
         ("subnormal scale", _t(50_000, 4, 1e-41, 7), 4, 4e-3),
         ("large scale", _t(50_000, 3, 1e30, 8), 4, 4e-3),
         ("two weights", np.array([0.25, -1.0], np.float32), 4, 0.05),
         ("tie", np.array([1, 1, 1, 1, 2], np.float32), 4, 0.5),
         ("float64 sums round", np.array([2.0 ** -30] * 100 + [1.0], np.float32), 4, 50 * 2.0 ** -60),
         ("subnormals", (np.array([1, 2, 3, 4, 100.]) * 2.0 ** -149).astype(np.float32), 4, 1e-3)]
    w = _t(400_000, 4, 0.02, 9)
    w[np.random.default_rng(10).integers(0, w.size, w.size // 3)] = 0.0
    c.append(("zeros", w, 4, 4e-3))
    w = np.round(_t(500_000, 3, 0.02, 11) * 300).astype(np.float32) / np.float32(300)
    c.append(("duplicates", w.astype(np.float32), 4, 4e-3))
    return c


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c[0])
def test_fit_device_bit_exact(case):
    name, w, bits, eps = case
    _say(f"fit_device {name}: numel={w.size} bits={bits} eps={eps!r}")
    p = L.fit_device(torch.from_numpy(w).to(DEV), bits, eps)
    r = O.fit_exact(w, bits, eps)
    _assert_params(p, r, bits)


@pytest.mark.parametrize("pos", [0, 5, CHUNK + 1, 2 * CHUNK + 2])
@pytest.mark.parametrize("val", [np.nan, np.inf, -np.inf])
def test_fit_device_nonfinite(pos, val):
    _say(f"fit_device nonfinite {val} at {pos}")
    w = _t(2 * CHUNK + 3, 4, 0.02, 12)
    w[pos] = val
    with pytest.raises(L.LogbqError) as e:
        L.fit_device(torch.from_numpy(w).to(DEV))
    assert e.value.status == L.ERR_NONFINITE


def test_fit_device_degenerate():
    _say("fit_device degenerate")
    for w in (np.zeros(1001, np.float32), np.array([0.5, -0.5, 0.5, 0.0], np.float32)):
        with pytest.raises(L.LogbqError) as e:
            L.fit_device(torch.from_numpy(w).to(DEV))
        assert e.value.status == L.ERR_DEGENERATE


def test_fit_device_workspace_reuse():
    """One workspace serves consecutive fits of different tensors (every pass clears it)."""
    ws = torch.empty(L.FIT_WORKSPACE_BYTES, dtype=torch.uint8, device=DEV)
    for seed, n in ((13, 700_000), (14, 9)):
        w = _t(n, 4, 0.02, seed)
        _say(f"fit_device reuse n={n}")
        _assert_params(L.fit_device(torch.from_numpy(w).to(DEV), workspace=ws), O.fit_exact(w), 4)


def _exact_energy_by_exponent(keys):
    """Exact sum of |w|^2 in units of 2^-298 for float32 bit patterns `keys` (sign cleared):
    per exponent field, sum m^2 split into 24-bit halves, each sum exact in float64 (every
    partial sum is an integer below 2^53 for fewer than 2^28 weights)."""
    exp = (keys >> 23).astype(np.int64)
    m = (keys & 0x7FFFFF).astype(np.uint64) | np.where(exp > 0, np.uint64(0x800000), np.uint64(0))
    q = m * m
    hi = np.bincount(exp, weights=(q >> np.uint64(24)).astype(np.float64), minlength=256)
    lo = np.bincount(exp, weights=(q & np.uint64(0xFFFFFF)).astype(np.float64), minlength=256)
    total = 0
    for e in range(256):
        if hi[e] or lo[e]:
            ef = -149 if e == 0 else e - 150
            total += ((int(hi[e]) << 24) + int(lo[e])) << (2 * ef + 298)
    return total


def test_fit_device_full_layer_certificate():
    """8192 x 28672 weights (0.015 t_3): w_min satisfies Eq. 5 in exact arithmetic, w_max is
    max |w|, wmin_index is the first position reaching eps, and the host fit (float64
    sequential sums) picks the same parameters."""
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    _say(f"fit_device full layer {lin.n} x {lin.k}")
    wd = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                  device=DEV)
    eps = 4e-3
    p = L.fit_device(wd, 4, eps)
    w = wd.cpu().numpy().ravel()
    keys = w.view(np.uint32) & np.uint32(0x7FFFFFFF)
    assert p.wmax == float(np.abs(w).max())
    vkey = int(np.float32(p.wmin).view(np.uint32))
    assert np.float32(p.wmin) == p.wmin
    total = _exact_energy_by_exponent(keys)
    e_below = _exact_energy_by_exponent(keys[keys < vkey])
    copies = int(np.count_nonzero(keys == vkey))
    assert copies > 0
    v = int(np.ldexp(np.float64(p.wmin), 149))
    num, den = float(eps).as_integer_ratio()
    assert e_below * den < num * total <= (e_below + copies * v * v) * den
    j = -(-(num * total - den * e_below) // (den * v * v))
    assert p.wmin_index == int(np.count_nonzero(keys < vkey)) + j - 1
    _say("  the same passes on the host")
    e = L.fit_exact(w, 4, eps)
    assert (e.wmin, e.wmax, e.wmin_index, e.base, e.shift) == \
        (p.wmin, p.wmax, p.wmin_index, p.base, p.shift)
    assert e.thresholds_array().view(np.uint32).tolist() == \
        p.thresholds_array().view(np.uint32).tolist()
    _say("  host fit of the same tensor")
    h = L.fit(w, 4, eps)
    assert (h.wmin, h.wmax, h.wmin_index, h.base, h.shift) == \
        (p.wmin, p.wmax, p.wmin_index, p.base, p.shift)
    assert h.codebook_array().view(np.uint32).tolist() == p.codebook_array().view(np.uint32).tolist()
    assert h.thresholds_array().view(np.uint32).tolist() == \
        p.thresholds_array().view(np.uint32).tolist()
