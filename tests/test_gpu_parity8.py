"""GPU parity of the 8-bit variant (q_max = 127, one code per byte, Sec. 3.1 at n = 8 with the
eps = 1e-6 of Sec. 3.2) against the CPU oracle, through the C ABI.

Bars as for 4 bits: codes and dequantized weights bit-exact; y = x . W_hat^T within
max |y - y_ref| / (||x_m|| * ||W_hat_n||) <= 1e-3. Every expected value comes from the oracle
(or, for the exhaustive float32 sweep, from the oracle's 127 thresholds).
"""
import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3
DEV = "cuda:0"
EPS8 = 1e-6


def _say(msg):
    print(msg, flush=True)


def rel_err(y, x, w_hat):
    y_ref = O.linear(x, w_hat)
    xn = np.linalg.norm(x.astype(np.float64), axis=1)[:, None]
    wn = np.linalg.norm(w_hat.astype(np.float64), axis=1)[None, :]
    den = xn * wn
    den[den == 0] = 1.0
    return float(np.max(np.abs(y.astype(np.float64) - y_ref) / den)) if y.size else 0.0


def prepare(n, k, seed, nu=4, scale=0.02, outliers=0.0, eps=EPS8):
    w = inputs.student_t_weights(n, k, nu, scale, seed=seed, outlier_frac=outliers)
    p = L.fit(w, 8, eps)
    r = O.fit(w, 8, eps)
    assert (p.base, p.shift) == (r.base, r.shift)
    return w, p, r


def gpu_encode(w, p):
    codes, cb = L.encode(torch.from_numpy(w).to(DEV), p)
    torch.cuda.synchronize()
    return codes, cb


def oracle_codes(w, r):
    return O.pack_codes(O.encode(w, r.base, r.shift, 8), 8)


def oracle_w_hat(w, r):
    return O.dequantize(O.encode(w, r.base, r.shift, 8), O.codebook(r.base, r.shift, 8))


# ---------------------------------------------------------------- encode / dequantize

@pytest.mark.parametrize("n,k,seed,nu,scale,outl,eps", [
    (2048, 2048, [18, 0, 0, 0], 4, 0.02, 0.0, EPS8),
    (8192, 2048, [18, 1, 5, 0], 4, 0.02, 1e-4, EPS8),     # with +-20 sigma outliers
    (37, 32, [18, 1, 1, 0], 3, 0.015, 0.0, EPS8),          # ragged tiny
    (513, 352, [18, 2, 2, 0], 3, 1.0, 0.0, 1e-3),
    (3, 14336, [18, 3, 3, 0], 6, 1e-4, 0.0, 4e-3),
])
def test_encode8_bit_exact(n, k, seed, nu, scale, outl, eps):
    _say(f"encode8 n={n} k={k} seed={seed}")
    w, p, r = prepare(n, k, seed, nu, scale, outl, eps)
    codes, cb = gpu_encode(w, p)
    exp = oracle_codes(w, r)
    got = codes.cpu().numpy()
    assert got.shape == (n, k)
    assert np.array_equal(got, exp), f"{np.count_nonzero(got != exp)} codes differ"
    assert cb.view(np.uint32).tolist() == O.codebook(r.base, r.shift, 8).view(np.uint32).tolist()
    # w_max encodes to q_max; a large sample reaches most of the 128 magnitudes (the largest few
    # lie between the bulk and the single maximum of a heavy tail)
    if n * k >= 1 << 22:
        mags = set(np.unique(got & 127).tolist())
        assert {0, 1, 127} <= mags and len(mags) >= 100


def test_encode8_special_values():
    """NaN, +-0, +-Inf, denormals, float32 extremes, w_min, w_max, and every one of the 127
    thresholds with its neighbours at +-1 and +-2 ulps, both signs."""
    _say("encode8 special values")
    w, p, r = prepare(64, 1024, [18, 4, 4, 0])
    thr = O.magnitude_thresholds(r.base, r.shift, 8)
    specials = [np.nan, -np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 3.4e38, -3.4e38,
                float(r.wmin), -float(r.wmin), float(r.wmax), -float(r.wmax)]
    for t in thr:
        for d in (-2, -1, 0, 1, 2):
            v = np.array([t], dtype=np.float32).view(np.int32)[0] + d
            f = np.array([v], dtype=np.int32).view(np.float32)[0]
            specials += [float(f), -float(f)]
    assert len(specials) <= w.size
    flat = w.reshape(-1).copy()
    flat[: len(specials)] = np.array(specials, dtype=np.float32)
    w2 = flat.reshape(w.shape)
    codes, _ = gpu_encode(w2, p)
    assert np.array_equal(codes.cpu().numpy(), oracle_codes(w2, r))


@pytest.mark.parametrize("n,k", [(64, 32), (1000, 2048), (3, 96)])
def test_dequant8_bit_exact(n, k):
    _say(f"dequant8 n={n} k={k}")
    w, p, r = prepare(n, k, [18, 5, n, 0])
    rng = np.random.default_rng(n)
    c = rng.integers(0, 256, size=(n, k), dtype=np.uint8)        # every code, including 128
    out = L.dequantize8(torch.from_numpy(c).to(DEV), p)
    torch.cuda.synchronize()
    exp = O.dequantize(c, O.codebook(r.base, r.shift, 8))
    assert out.cpu().numpy().view(np.uint32).tolist() == exp.view(np.uint32).tolist()


def test_encode8_dequant8_roundtrip_idempotent():
    """encode(dequantize(codes)) == codes with code 128 (negative zero) mapped to 0."""
    _say("encode8(dequantize8(codes))")
    w, p, r = prepare(128, 512, [18, 6, 0, 0])
    rng = np.random.default_rng(5)
    c = rng.integers(0, 256, size=(128, 512), dtype=np.uint8)
    wh = L.dequantize8(torch.from_numpy(c).to(DEV), p)
    back, _ = L.encode(wh, p)
    torch.cuda.synchronize()
    exp = c.copy()
    exp[exp == 128] = 0
    assert np.array_equal(back.cpu().numpy(), exp)


@pytest.mark.parametrize("params", ["fit", "narrow"])
def test_encode8_every_float32(params):
    """Every float32 bit pattern with the sign clear (2^31 values) and a slice of negatives,
    against the oracle's 127 exact thresholds."""
    if params == "narrow":
        base, shift = 1.0625, 120        # thresholds straddle 1.0, steps of 6 %
    else:
        w = inputs.student_t_weights(1024, 1024, 4, 0.02, seed=[18, 7, 0, 0])
        r = O.fit(w, 8, EPS8)
        base, shift = r.base, r.shift
    thr = O.magnitude_thresholds(base, shift, 8)
    p = L.Params()
    p.bits, p.qmax, p.base, p.shift = 8, 127, base, shift
    for i in range(127):
        p.thresholds[i] = float(thr[i])
    p.thresholds[127] = float("inf")
    thr_t = torch.from_numpy(thr.astype(np.float32)).to(DEV)
    chunk = 1 << 28
    rows = chunk // 32768
    mism = 0
    for c0 in list(range(0, 1 << 31, chunk)) + ["neg"]:
        _say(f"sweep8 {params} chunk {c0}")
        if c0 == "neg":
            bits = torch.arange(0, chunk, device=DEV, dtype=torch.int64) * 7 + 0x80000000
            bits = (bits & 0xFFFFFFFF).to(torch.int64)
            bits = torch.where(bits >= 2 ** 31, bits - 2 ** 32, bits).to(torch.int32)
        else:
            bits = torch.arange(c0, c0 + chunk, device=DEV, dtype=torch.int64).to(torch.int32)
        x = bits.view(torch.float32).reshape(rows, 32768)
        codes, _ = L.encode(x, p)
        got = codes.reshape(-1).to(torch.int32)
        ax = x.reshape(-1).abs()
        mag = torch.bucketize(ax, thr_t, right=True, out_int32=True)
        mag = torch.where(torch.isnan(ax), torch.zeros_like(mag), mag)
        neg = (x.reshape(-1) < 0) & (mag > 0)
        exp = mag + 128 * neg.to(torch.int32)
        mism += int((got != exp).sum().item())
        del x, codes, got, ax, mag, neg, exp, bits
    assert mism == 0


def test_encode8_estimate_fallbacks():
    """The 8-bit encode estimates each magnitude index from log2|x| and corrects it against the
    thresholds; parameters whose thresholds do not sit where the estimate puts them (a base
    that disagrees with the thresholds) or whose base is too close to 1 for a float estimate
    take the binary search. Codes must equal the count of thresholds <= |x| either way."""
    rng = np.random.default_rng(31)
    for name, base, shift, claimed in (("consistent", 1.1, 100, None),
                                        ("base disagrees", 1.1, 100, 1.5),
                                        ("base near 1", 1.0001, 60000, None)):
        _say(f"encode8 estimate: {name}")
        thr = O.magnitude_thresholds(base, shift, 8)
        p = L.Params()
        p.bits, p.qmax, p.base, p.shift = 8, 127, claimed or base, shift
        for i in range(127):
            p.thresholds[i] = float(thr[i])
        p.thresholds[127] = float("inf")
        lo, hi = np.log2(float(thr[0])) - 2, np.log2(float(thr[126])) + 2
        mags = np.exp2(rng.uniform(lo, hi, size=64 * 4096)).astype(np.float32)
        x = (mags * rng.choice([-1.0, 1.0], size=mags.size)).astype(np.float32)
        x[:254] = np.repeat(thr, 2) * np.tile([1.0, -1.0], 127)          # thresholds themselves
        w = x.reshape(64, 4096)
        codes, _ = L.encode(torch.from_numpy(w).to(DEV), p)
        torch.cuda.synchronize()
        mag = np.searchsorted(thr, np.abs(w), side="right").astype(np.int64)
        exp = (mag + 128 * ((w < 0) & (mag > 0))).astype(np.uint8)
        assert np.array_equal(codes.cpu().numpy(), exp), name


# ---------------------------------------------------------------- linear

SHAPES = [(2048, 2048), (1000, 352), (37, 32), (512, 14336), (4096, 4096), (64, 8192),
          (8, 28672), (8197, 2048), (6145, 4096), (16, 32768), (3000, 6144)]
BATCH = [1, 2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 64, 100, 128, 129, 200]


@pytest.mark.parametrize("n,k", SHAPES)
def test_linear8_matches_oracle(n, k):
    w, p, r = prepare(n, k, [18, n, k % 1000, 0])
    codes, cb = gpu_encode(w, p)
    wh = oracle_w_hat(w, r)
    for m in BATCH:
        if m > 32 and n * k > 4096 * 4096:
            continue
        _say(f"linear8 n={n} k={k} m={m}")
        x = inputs.activations(m, k, seed=[18, n, k % 1000, 1 + m])
        y = L.linear8(torch.from_numpy(x).to(DEV), codes, cb)
        torch.cuda.synchronize()
        err = rel_err(y.cpu().numpy(), x, wh)
        assert err <= TOL, (m, err)
        assert err <= 2.5e-4, (m, err)


def test_linear8_unit_vectors_and_zero():
    n, k = 300, 1024
    w, p, r = prepare(n, k, [18, 1, 2, 3])
    codes, cb = gpu_encode(w, p)
    wh = oracle_w_hat(w, r)
    for m in (1, 8, 16, 64):
        _say(f"linear8 unit vectors m={m}")
        cols = np.arange(m) * 7 % k
        x = np.zeros((m, k), dtype=np.float16)
        x[np.arange(m), cols] = 1.0
        y = L.linear8(torch.from_numpy(x).to(DEV), codes, cb).cpu().numpy()
        exp = wh[:, cols].T.astype(np.float64)
        assert np.all(np.abs(y - exp) <= np.abs(exp) * 2.0 ** -11)
        assert np.all(np.sign(y) == np.sign(exp))
        y0 = L.linear8(torch.zeros((m, k), dtype=torch.float16, device=DEV), codes, cb)
        assert torch.all(y0 == 0).item()


def test_linear8_sign_flip_negates():
    n, k = 777, 1024
    w, p, r = prepare(n, k, [18, 2, 2, 2])
    codes, cb = gpu_encode(w, p)
    flipped = codes ^ 0x80
    wh = oracle_w_hat(w, r)
    for m in (1, 4, 8, 32, 128):
        _say(f"linear8 sign flip m={m}")
        xn = inputs.activations(m, k, seed=[18, 2, 2, m])
        x = torch.from_numpy(xn).to(DEV)
        y = L.linear8(x, codes, cb)
        yf = L.linear8(x, flipped, cb)
        torch.cuda.synchronize()
        absdot = np.abs(xn.astype(np.float64)) @ np.abs(wh.astype(np.float64)).T
        diff = np.abs(yf.cpu().numpy().astype(np.float64) + y.cpu().numpy().astype(np.float64))
        assert np.all(diff <= absdot * 2.0 ** -20), float(np.max(diff / absdot))


def test_linear8_constant_codes():
    n, k = 64, 512
    w, p, r = prepare(n, k, [18, 3, 3, 3])
    lut = O.codebook(r.base, r.shift, 8)
    for c in (1, 64, 127, 133, 255):
        codes = torch.full((n, k), c, dtype=torch.uint8, device=DEV)
        for m in (1, 16):
            _say(f"linear8 constant code {c} m={m}")
            x = inputs.activations(m, k, seed=[18, 3, c, m])
            y = L.linear8(torch.from_numpy(x).to(DEV), codes, p).cpu().numpy()
            exp = float(lut[c]) * x.astype(np.float64).sum(axis=1)
            bound = abs(float(lut[c])) * np.abs(x.astype(np.float64)).sum(axis=1) * 1e-3
            assert np.all(np.abs(y - exp[:, None]) <= bound[:, None])


def test_linear8_deterministic_and_empty():
    n, k = 4096, 4096
    w, p, r = prepare(n, k, [18, 4, 4, 4])
    codes, cb = gpu_encode(w, p)
    for m in (1, 3, 8, 32, 128):
        _say(f"linear8 determinism m={m}")
        x = torch.from_numpy(inputs.activations(m, k, seed=[18, 4, 4, m])).to(DEV)
        y1 = L.linear8(x, codes, cb)
        y2 = L.linear8(x, codes, cb)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2)
    _say("linear8 k = 0 and empty shapes")
    y = torch.full((3, 5), 7.0, device=DEV)
    L.linear8(torch.empty((3, 0), dtype=torch.float16, device=DEV),
              torch.empty((5, 0), dtype=torch.uint8, device=DEV), cb, out=y)
    torch.cuda.synchronize()
    assert torch.all(y == 0).item()
    y = L.linear8(torch.empty((0, 64), dtype=torch.float16, device=DEV),
                  torch.zeros((5, 64), dtype=torch.uint8, device=DEV), cb)
    assert y.shape == (0, 5)


def test_linear8_arbitrary_codebook():
    """Any 256 finite floats work as a codebook."""
    rng = np.random.default_rng(13)
    n, k = 300, 1024
    codes_np = rng.integers(0, 256, size=(n, k), dtype=np.uint8)
    codes = torch.from_numpy(codes_np).to(DEV)
    for trial in range(2):
        cb = rng.standard_normal(256).astype(np.float32) * np.float32(10.0 ** (3 * trial - 2))
        wh = O.dequantize(codes_np, cb)
        for m in (1, 5, 16, 33, 128):
            _say(f"linear8 arbitrary codebook trial {trial} m={m}")
            x = inputs.activations(m, k, seed=[18, 9, trial, m])
            y = L.linear8(torch.from_numpy(x).to(DEV), codes, cb)
            torch.cuda.synchronize()
            assert rel_err(y.cpu().numpy(), x, wh) <= TOL


def test_linear8_split_k():
    """The 8-bit split-K kernel at every K it serves, batch groups of two (m <= 8) and one, row
    counts that leave a partial last block, more blocks per workgroup than results held, a
    fitted and an arbitrary codebook; y prefilled with NaN so that every output must be
    written, and two calls bit-equal."""
    rng = np.random.default_rng(41)
    for n, k in ((3001, 8192), (6007, 4096), (20001, 2048)):
        w, p, r = prepare(n, k, [18, 41, k % 1000, 0])
        codes, cb = gpu_encode(w, p)
        wh = oracle_w_hat(w, r)
        cb2 = rng.standard_normal(256).astype(np.float32)
        wh2 = O.dequantize(codes.cpu().numpy(), cb2)
        for m in (3, 5, 8, 9, 16):
            if L.linear_path(8, m, k, n) != "splitk":
                continue
            _say(f"linear8 split-K n={n} k={k} m={m}")
            x = inputs.activations(m, k, seed=[18, 41, k % 1000, m])
            xd = torch.from_numpy(x).to(DEV)
            for book, ref, bar in ((cb, wh, 2.5e-4), (cb2, wh2, TOL)):
                y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
                L.linear8(xd, codes, book, out=y)
                y2 = L.linear8(xd, codes, book)
                torch.cuda.synchronize()
                assert torch.isfinite(y).all()
                assert torch.equal(y, y2)
                assert rel_err(y.cpu().numpy(), x, ref) <= bar, (n, k, m)
    assert L.linear_path(8, 8, 8192, 3001) == "splitk" and L.linear_path(8, 16, 2048, 20001) == "splitk"


def test_linear8_k_quartered():
    """The 8-bit K-quartered kernel (m > 64 at N >= 16384): a partial last 128-row workgroup,
    K not a multiple of its 128-k step, batch rows past the last full tile and two workgroup
    rows, a fitted and an arbitrary codebook; y prefilled with NaN, two calls bit-equal."""
    rng = np.random.default_rng(43)
    for n, k in ((16400, 1056), (16384, 4096)):
        w, p, r = prepare(n, k, [18, 43, k % 1000, 0])
        codes, cb = gpu_encode(w, p)
        wh = oracle_w_hat(w, r)
        cb2 = rng.standard_normal(256).astype(np.float32)
        wh2 = O.dequantize(codes.cpu().numpy(), cb2)
        for m in ((65, 100, 129) if k == 1056 else (128,)):
            assert L.linear_path(8, m, k, n) == "mfma_kq"
            _say(f"linear8 K-quartered n={n} k={k} m={m}")
            x = inputs.activations(m, k, seed=[18, 43, k % 1000, m])
            xd = torch.from_numpy(x).to(DEV)
            for book, ref, bar in ((cb, wh, 2.5e-4), (cb2, wh2, TOL)):
                y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
                L.linear8(xd, codes, book, out=y)
                y2 = L.linear8(xd, codes, book)
                torch.cuda.synchronize()
                assert torch.isfinite(y).all()
                assert torch.equal(y, y2)
                assert rel_err(y.cpu().numpy(), x, ref) <= bar, (n, k, m)


# ---------------------------------------------------------------- full-size, sampled

def test_full_size_layer8_8192x28672_sampled():
    """The 8192 x 28672 layer at 8 bits (eps = 1e-6) at every batch size of the sweep; codes and
    y compared on sampled rows."""
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    n, k = lin.n, lin.k
    _say("full-size layer8: generate")
    wd = inputs.student_t_weights(n, k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                  device=DEV)
    w = wd.cpu().numpy()
    _say("full-size layer8: oracle fit")
    r = O.fit(w, 8, EPS8)
    p = L.fit(w, 8, EPS8)
    assert (p.base, p.shift, p.wmin, p.wmax, p.wmin_index) == \
        (r.base, r.shift, r.wmin, r.wmax, r.wmin_index)
    rows = np.sort(np.random.default_rng(1).choice(n, size=48, replace=False))
    rows = np.concatenate([rows, [0, n - 1]])
    wsub = w[rows]
    del w
    _say("full-size layer8: encode")
    codes, cb = L.encode(wd, p)
    torch.cuda.synchronize()
    del wd
    got = codes[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    c_sub = O.encode(wsub, r.base, r.shift, 8)
    assert np.array_equal(got, c_sub)
    wh = O.dequantize(c_sub, O.codebook(r.base, r.shift, 8))
    for m in wl["batch"]:
        _say(f"full-size layer8: linear8 m={m}")
        x = inputs.activations(m, k, seed=[wl["cfg"], 0, 0, 1])
        y = L.linear8(torch.from_numpy(x).to(DEV), codes, cb)
        torch.cuda.synchronize()
        ys = y[:, torch.from_numpy(rows).to(DEV)].cpu().numpy()
        assert rel_err(ys, x, wh) <= TOL
