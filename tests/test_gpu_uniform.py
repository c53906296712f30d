"""GPU parity of the asymmetric linear baseline (Sec. 2, Quant(s, z, x)) against its CPU oracle,
through the C ABI: codes and dequantized weights bit-exact, products within the same bar as
LogbQuant's (the codes run through logbq_linear with the baseline's codebook, which is not
sign-symmetric, so every kernel takes its LDS-table form), and the reconstruction SQNR of both
schemes computed from GPU-dequantized weights equal to the oracle's."""
import numpy as np
import pytest

from oracle import logbq_oracle as O
from oracle import uniform_oracle as U
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3
DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


def _tensor(n, k, seed, nu=4, scale=0.02, outl=0.0):
    return np.asarray(inputs.student_t_weights(n, k, nu, scale, seed=seed, outlier_frac=outl))


def _oracle_codes(w, f):
    return O.pack(U.uniform_encode(w, f.scale, f.zero))


@pytest.mark.parametrize("n,k,seed,nu,scale,outl", [
    (2048, 2048, [30, 0, 0, 0], 4, 0.02, 0.0),
    (8192, 2048, [30, 1, 0, 0], 4, 0.02, 1e-4),
    (37, 32, [30, 2, 0, 0], 3, 0.015, 0.0),
    (3, 14336, [30, 3, 0, 0], 6, 1.0, 0.0),
])
def test_encode_uniform_bit_exact(n, k, seed, nu, scale, outl):
    _say(f"uniform encode n={n} k={k}")
    w = _tensor(n, k, seed, nu, scale, outl)
    u = L.fit_uniform(w)
    f = U.uniform_fit(w)
    codes = L.encode_uniform(torch.from_numpy(w).to(DEV), u)
    torch.cuda.synchronize()
    got = codes.cpu().numpy()
    exp = _oracle_codes(w, f)
    assert np.array_equal(got, exp), f"{np.count_nonzero(got != exp)} bytes differ"
    wd = L.dequantize(codes, u.codebook_array())
    torch.cuda.synchronize()
    lv = U.uniform_levels(f.scale, f.zero)
    assert np.array_equal(wd.cpu().numpy().view(np.uint32),
                          U.uniform_dequantize(U.uniform_encode(w, f.scale, f.zero), lv).view(np.uint32))


def test_encode_uniform_boundaries():
    """Every threshold, its float32 neighbours, the range ends, +-inf and NaN."""
    _say("uniform encode boundaries")
    w = _tensor(64, 64, [30, 4, 0, 0])
    u = L.fit_uniform(w)
    f = U.uniform_fit(w)
    thr = U.uniform_thresholds(f.scale, f.zero)
    vals = np.concatenate([thr, np.nextafter(thr, np.float32(-np.inf)),
                           np.nextafter(thr, np.float32(np.inf)),
                           [w.min(), w.max(), 0.0, -0.0, np.inf, -np.inf, np.nan, 1e30, -1e30]])
    vals = np.resize(vals.astype(np.float32), 2 * 64)
    x = vals.reshape(2, 64)
    got = L.encode_uniform(torch.from_numpy(x).to(DEV), u).cpu().numpy()
    assert np.array_equal(got, O.pack(U.uniform_encode(x, f.scale, f.zero)))


# (4096, 1024, 128) has the K-quartered kernel's shape; this codebook is not sign-symmetric, so
# it falls back to the stepped kernel's LDS-table form.
@pytest.mark.parametrize("n,k,m", [(2048, 2048, 1), (8192, 2048, 4), (8192, 2048, 8),
                                   (4096, 4096, 32), (1000, 4128, 77), (2051, 1024, 128),
                                   (4096, 1024, 128)])
def test_linear_on_uniform_codes(n, k, m):
    _say(f"uniform linear n={n} k={k} m={m} path={L.linear_path(4, m, k, n)}")
    w = _tensor(n, k, [31, n, k, 0])
    u = L.fit_uniform(w)
    f = U.uniform_fit(w)
    x = np.asarray(inputs.activations(m, k, seed=[31, n, k, 1]))
    codes = L.encode_uniform(torch.from_numpy(w).to(DEV), u)
    y = L.linear(torch.from_numpy(x).to(DEV), codes, u.codebook_array())
    torch.cuda.synchronize()
    w_hat = U.uniform_dequantize(U.uniform_encode(w, f.scale, f.zero), U.uniform_levels(f.scale, f.zero))
    y_ref = O.linear(x, w_hat)
    yg = y.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(yg))
    xn = np.linalg.norm(x.astype(np.float64), axis=1)[:, None]
    wn = np.linalg.norm(w_hat.astype(np.float64), axis=1)[None, :]
    den = xn * wn
    zero_rows = int(np.count_nonzero(wn == 0))
    den[den == 0] = 1.0           # rows whose every weight sits on the zero level: y must be 0
    err = float(np.max(np.abs(yg - y_ref) / den))
    _say(f"  rel err {err:.3g}, rows with all weights on the zero level: {zero_rows}")
    assert err <= TOL, err


def test_quality_on_gpu_matches_oracle():
    """SQNR of both schemes from GPU-dequantized weights equals the oracle's value."""
    _say("quality parity")
    w = _tensor(2048, 2048, [32, 0, 0, 0])
    wd = torch.from_numpy(w).to(DEV)
    p = L.fit(w)
    codes, cb = L.encode(wd, p)
    wl = L.dequantize(codes, cb)
    u = L.fit_uniform(w)
    wu = L.dequantize(L.encode_uniform(wd, u), u.codebook_array())
    torch.cuda.synchronize()
    r = O.fit(w)
    wl_ref = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
    f = U.uniform_fit(w)
    wu_ref = U.uniform_dequantize(U.uniform_encode(w, f.scale, f.zero), U.uniform_levels(f.scale, f.zero))
    assert U.sqnr_db(w, wl.cpu().numpy()) == U.sqnr_db(w, wl_ref)
    assert U.sqnr_db(w, wu.cpu().numpy()) == U.sqnr_db(w, wu_ref)
    assert U.sqnr_db(w, wl_ref) > U.sqnr_db(w, wu_ref) + 6.0


def test_grouped_launch_with_uniform_codebooks():
    """Grouped calls whose codebooks are not sign-symmetric (the split-K kernel then launches
    per linear with its LDS table) equal single calls bit for bit."""
    k = 2048
    ws = [_tensor(n, k, [33, n, 0, 0]) for n in (4096, 300)]
    us = [L.fit_uniform(w) for w in ws]
    codes = [L.encode_uniform(torch.from_numpy(w).to(DEV), u) for w, u in zip(ws, us)]
    for m in (1, 4, 8, 16):
        _say(f"grouped uniform m={m}")
        x = torch.from_numpy(np.asarray(inputs.activations(m, k, seed=[33, m, 0, 1]))).to(DEV)
        ys = L.linear_multi(x, codes, [u.codebook_array() for u in us])
        for c, u, y in zip(codes, us, ys):
            y1 = L.linear(x, c, u.codebook_array())
            torch.cuda.synchronize()
            assert torch.equal(y, y1)
