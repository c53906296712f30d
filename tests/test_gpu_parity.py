"""GPU parity of liblogbq against the CPU oracle, through the C ABI.

Bars: codes and dequantized weights bit-exact; y = x . W_hat^T within
max |y - y_ref| / (||x_m|| * ||W_hat_n||) <= 1e-3 (float32 accumulation). The same seeded
inputs go to both sides; every expected value comes from the oracle (or, for the exhaustive
float32 sweep, from the oracle's thresholds).
"""
import math

import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L
from stepped_rule import stepped_name, stepped_shape

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3
DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


def rel_err(y, x, w_hat):
    """max over (m, n) of |y - y_ref| / (||x_m|| ||W_hat_n||), with y_ref from the oracle."""
    y_ref = O.linear(x, w_hat)
    xn = np.linalg.norm(x.astype(np.float64), axis=1)[:, None]
    wn = np.linalg.norm(w_hat.astype(np.float64), axis=1)[None, :]
    den = xn * wn
    den[den == 0] = 1.0
    return float(np.max(np.abs(y.astype(np.float64) - y_ref) / den)) if y.size else 0.0


def prepare(n, k, seed, nu=4, scale=0.02, outliers=0.0):
    w = inputs.student_t_weights(n, k, nu, scale, seed=seed, outlier_frac=outliers)
    p = L.fit(w)
    r = O.fit(w)
    assert (p.base, p.shift) == (r.base, r.shift)
    return w, p, r


def gpu_encode(w, p):
    wd = torch.from_numpy(w).to(DEV)
    codes, cb = L.encode(wd, p)
    torch.cuda.synchronize()
    return codes, cb


def oracle_codes(w, r):
    return O.pack(O.encode(w, r.base, r.shift))


# ---------------------------------------------------------------- encode / dequantize

@pytest.mark.parametrize("n,k,seed,nu,scale,outl", [
    (2048, 2048, [0, 0, 0, 0], 4, 0.02, 0.0),          # 2048 x 2048 linear
    (8192, 2048, [1, 0, 5, 0], 4, 0.02, 1e-4),          # up-projection with outliers
    (37, 32, [9, 1, 1, 0], 3, 0.015, 0.0),              # ragged tiny
    (513, 352, [9, 2, 2, 0], 3, 1.0, 0.0),
    (3, 14336, [9, 3, 3, 0], 6, 1e-4, 0.0),
])
def test_encode_bit_exact(n, k, seed, nu, scale, outl):
    _say(f"encode n={n} k={k} seed={seed}")
    w, p, r = prepare(n, k, seed, nu, scale, outl)
    codes, cb = gpu_encode(w, p)
    exp = oracle_codes(w, r)
    got = codes.cpu().numpy()
    assert got.shape == exp.shape
    assert np.array_equal(got, exp), f"{np.count_nonzero(got != exp)} bytes differ"
    assert cb.view(np.uint32).tolist() == O.codebook(r.base, r.shift).view(np.uint32).tolist()


def test_encode_special_values():
    _say("encode special values")
    w, p, r = prepare(64, 64, [9, 4, 4, 0])
    thr = O.magnitude_thresholds(r.base, r.shift)
    specials = [np.nan, -np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 3.4e38, -3.4e38,
                float(r.wmin), -float(r.wmin), float(r.wmax), -float(r.wmax)]
    for t in thr:
        for d in (-2, -1, 0, 1, 2):
            v = np.array([t], dtype=np.float32).view(np.int32)[0] + d
            f = np.array([v], dtype=np.int32).view(np.float32)[0]
            specials += [float(f), -float(f)]
    flat = w.reshape(-1).copy()
    flat[: len(specials)] = np.array(specials, dtype=np.float32)
    w2 = flat.reshape(w.shape)
    codes, _ = gpu_encode(w2, p)
    assert np.array_equal(codes.cpu().numpy(), oracle_codes(w2, r))


@pytest.mark.parametrize("n,k", [(64, 32), (1000, 2048), (3, 96)])
def test_dequant_bit_exact(n, k):
    _say(f"dequant n={n} k={k}")
    w, p, r = prepare(n, k, [9, 5, n, 0])
    rng = np.random.default_rng(n)
    c = rng.integers(0, 16, size=(n, k), dtype=np.uint8)      # every code, including 8
    packed = torch.from_numpy(O.pack(c)).to(DEV)
    out = L.dequantize(packed, p)
    torch.cuda.synchronize()
    exp = O.dequantize(c, O.codebook(r.base, r.shift))
    assert out.cpu().numpy().view(np.uint32).tolist() == exp.view(np.uint32).tolist()


def test_encode_dequant_roundtrip_idempotent():
    """encode(dequantize(codes)) == codes with code 8 mapped to 0."""
    _say("encode(dequantize(codes))")
    w, p, r = prepare(128, 256, [9, 6, 0, 0])
    rng = np.random.default_rng(5)
    c = rng.integers(0, 16, size=(128, 256), dtype=np.uint8)
    packed = torch.from_numpy(O.pack(c)).to(DEV)
    wh = L.dequantize(packed, p)
    back, _ = L.encode(wh, p)
    torch.cuda.synchronize()
    exp = c.copy()
    exp[exp == 8] = 0
    assert np.array_equal(back.cpu().numpy(), O.pack(exp))


@pytest.mark.parametrize("params", ["b2", "c1", "heavy"])
def test_encode_every_float32(params):
    """Every float32 bit pattern with the sign clear (2^31 values) and a slice of negatives,
    against the oracle's exact thresholds."""
    if params == "b2":
        base, shift = 2.0, 7
    else:
        nu, scale = (4, 0.02) if params == "c1" else (3, 0.015)
        w = inputs.student_t_weights(1024, 1024, nu, scale, seed=[9, 7, len(params), 0])
        r = O.fit(w)
        base, shift = r.base, r.shift
    thr = O.magnitude_thresholds(base, shift)
    p = L.Params()
    p.bits, p.qmax, p.base, p.shift = 4, 7, base, shift
    for i in range(7):
        p.thresholds[i] = float(thr[i])
    p.thresholds[7] = float("inf")
    thr_t = torch.from_numpy(thr.astype(np.float32)).to(DEV)
    chunk = 1 << 28
    rows = chunk // 32768
    mism = 0
    shifts = torch.arange(0, 32, 4, device=DEV, dtype=torch.int32)
    for c0 in list(range(0, 1 << 31, chunk)) + ["neg"]:
        _say(f"sweep {params} chunk {c0}")
        if c0 == "neg":
            bits = torch.arange(0, chunk, device=DEV, dtype=torch.int64) * 7 + 0x80000000
            bits = (bits & 0xFFFFFFFF).to(torch.int64)
            bits = torch.where(bits >= 2 ** 31, bits - 2 ** 32, bits).to(torch.int32)
        else:
            bits = torch.arange(c0, c0 + chunk, device=DEV, dtype=torch.int64).to(torch.int32)
        x = bits.view(torch.float32).reshape(rows, 32768)
        codes, _ = L.encode(x, p)
        cw = codes.view(torch.int32).reshape(-1)
        nib = ((cw[:, None] >> shifts[None, :]) & 15).reshape(-1)
        ax = x.reshape(-1).abs()
        mag = torch.bucketize(ax, thr_t, right=True).to(torch.int32)
        mag = torch.where(torch.isnan(ax), torch.zeros_like(mag), mag)
        neg = (x.reshape(-1) < 0) & (mag > 0)
        exp = mag + 8 * neg.to(torch.int32)
        mism += int((nib != exp).sum().item())
        del x, codes, cw, nib, ax, mag, neg, exp, bits
    assert mism == 0


# ---------------------------------------------------------------- linear

SHAPES = [(2048, 2048), (1000, 352), (37, 32), (512, 14336), (4096, 4096), (64, 8192), (8, 28672),
          # row counts that leave 1 or 2 rows after the last full group of the code-buffer
          # ring; a K whose rows are split over four wavefronts; 3 chunks per lane
          (8197, 2048), (6145, 4096), (16, 32768), (3000, 6144),
          # more than 64 rows per wavefront (results are written 64 rows at a time)
          (140001, 32)]
BATCH = [1, 2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 64, 100, 128, 129, 200]


@pytest.mark.parametrize("n,k", SHAPES)
def test_linear_matches_oracle(n, k):
    w, p, r = prepare(n, k, [8, n, k % 1000, 0])
    codes, cb = gpu_encode(w, p)
    c = O.encode(w, r.base, r.shift)
    wh = O.dequantize(c, O.codebook(r.base, r.shift))
    for m in BATCH:
        if m > 32 and n * k > 4096 * 4096:
            continue
        _say(f"linear n={n} k={k} m={m}")
        x = inputs.activations(m, k, seed=[8, n, k % 1000, 1 + m])
        y = L.linear(torch.from_numpy(x).to(DEV), codes, cb)
        torch.cuda.synchronize()
        err = rel_err(y.cpu().numpy(), x, wh)
        assert err <= TOL, (m, err)
        assert err <= 2.5e-4, (m, err)   # float16 table + float32 accumulation headroom


def test_linear_unit_vectors_and_zero():
    """x = e_k gives column k of W_hat (up to the float16 table rounding); x = 0 gives +0."""
    n, k = 300, 256
    w, p, r = prepare(n, k, [8, 1, 2, 3])
    codes, cb = gpu_encode(w, p)
    wh = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
    for m in (1, 8, 16, 64):
        _say(f"unit vectors m={m}")
        cols = np.arange(m) * 7 % k
        x = np.zeros((m, k), dtype=np.float16)
        x[np.arange(m), cols] = 1.0
        y = L.linear(torch.from_numpy(x).to(DEV), codes, cb).cpu().numpy()
        exp = wh[:, cols].T.astype(np.float64)
        assert np.all(np.abs(y - exp) <= np.abs(exp) * 2.0 ** -11)
        assert np.all(np.sign(y) == np.sign(exp))
        y0 = L.linear(torch.zeros((m, k), dtype=torch.float16, device=DEV), codes, cb)
        assert torch.all(y0 == 0).item()


def test_linear_sign_flip_negates():
    """Flipping the sign bit of every code negates y. The products negate exactly; the float32
    accumulation (v_dot2_f32_f16 / MFMA) is not guaranteed sign-symmetric in its last bit, so
    the check is |y(flipped) + y| <= 2^-20 * sum_k |x_k w_k| per output."""
    n, k = 777, 1024
    w, p, r = prepare(n, k, [8, 2, 2, 2])
    codes, cb = gpu_encode(w, p)
    flipped = codes ^ 0x88
    wh = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
    for m in (1, 4, 8, 32, 128):
        _say(f"sign flip m={m}")
        xn = inputs.activations(m, k, seed=[8, 2, 2, m])
        x = torch.from_numpy(xn).to(DEV)
        y = L.linear(x, codes, cb)
        yf = L.linear(x, flipped, cb)
        torch.cuda.synchronize()
        absdot = np.abs(xn.astype(np.float64)) @ np.abs(wh.astype(np.float64)).T
        diff = np.abs(yf.cpu().numpy().astype(np.float64) + y.cpu().numpy().astype(np.float64))
        assert np.all(diff <= absdot * 2.0 ** -20), float(np.max(diff / absdot))
        _say(f"  bit-exact negation: {bool(torch.equal(yf, -y))}")


def test_linear_constant_codes():
    """All codes equal c: y_n = codebook[c] * sum(x) (float32 tolerance)."""
    n, k = 64, 512
    w, p, r = prepare(n, k, [8, 3, 3, 3])
    lut = O.codebook(r.base, r.shift)
    for c in (1, 7, 12):
        byte = c | (c << 4)
        codes = torch.full((n, k // 2), byte, dtype=torch.uint8, device=DEV)
        for m in (1, 16):
            _say(f"constant code {c} m={m}")
            x = inputs.activations(m, k, seed=[8, 3, c, m])
            y = L.linear(torch.from_numpy(x).to(DEV), codes, p).cpu().numpy()
            exp = float(lut[c]) * x.astype(np.float64).sum(axis=1)
            bound = abs(float(lut[c])) * np.abs(x.astype(np.float64)).sum(axis=1) * 1e-3
            assert np.all(np.abs(y - exp[:, None]) <= bound[:, None])


def test_linear_deterministic_and_empty():
    n, k = 4096, 4096
    w, p, r = prepare(n, k, [8, 4, 4, 4])
    codes, cb = gpu_encode(w, p)
    for m in (1, 3, 8, 32, 128):
        _say(f"determinism m={m}")
        x = torch.from_numpy(inputs.activations(m, k, seed=[8, 4, 4, m])).to(DEV)
        y1 = L.linear(x, codes, cb)
        y2 = L.linear(x, codes, cb)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2)
    _say("k = 0 and empty shapes")
    y = torch.full((3, 5), 7.0, device=DEV)
    L.linear(torch.empty((3, 0), dtype=torch.float16, device=DEV),
             torch.empty((5, 0), dtype=torch.uint8, device=DEV), cb, out=y)
    torch.cuda.synchronize()
    assert torch.all(y == 0).item()
    y = L.linear(torch.empty((0, 64), dtype=torch.float16, device=DEV),
                 torch.zeros((5, 32), dtype=torch.uint8, device=DEV), cb)
    assert y.shape == (0, 5)


def test_linear_arbitrary_codebook():
    """Any 16 finite floats work as a codebook (the table-lookup kernels); a fitted codebook is
    sign-symmetric and takes the register-dequant MFMA path, any other takes the pair table
    (at K = 14336 above m = 16 the stepped kernel, as for fitted codebooks)."""
    rng = np.random.default_rng(12)
    n = 300
    for k in (1024, 2048, 4096, 8192, 14336):
        codes_np = rng.integers(0, 16, size=(n, k), dtype=np.uint8)
        codes = torch.from_numpy(O.pack(codes_np)).to(DEV)
        for trial in range(2):
            cb = rng.standard_normal(16).astype(np.float32) * np.float32(10.0 ** (3 * trial - 2))
            wh = O.dequantize(codes_np, cb)
            for m in ((1, 5, 16, 33, 128) if k == 1024 else (5, 16, 24) if k == 14336 else (5, 16)):
                _say(f"arbitrary codebook k={k} trial {trial} m={m}")
                x = inputs.activations(m, k, seed=[8, 9, trial, m + k])
                y = L.linear(torch.from_numpy(x).to(DEV), codes, cb)
                torch.cuda.synchronize()
                assert rel_err(y.cpu().numpy(), x, wh) <= TOL


def test_linear_split_k_many_blocks():
    """The split-K MFMA path (2 <= m <= 16, K = 1, 2, 4 or 8 Ki) with more than 4 blocks of 16
    rows per workgroup (results are stored 4 blocks at a time) and a ragged last block, for a
    fitted (register dequantization, two batch groups up to m = 8) and an arbitrary codebook
    (pair table)."""
    n, k = 40003, 1024
    w, p, r = prepare(n, k, [8, 11, 1, 0])
    codes, cb = gpu_encode(w, p)
    wh = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
    rng = np.random.default_rng(13)
    cb2 = rng.standard_normal(16).astype(np.float32)
    wh2 = O.dequantize(O.unpack(codes.cpu().numpy()), cb2)
    for m in (5, 8, 13, 16):
        _say(f"split-K many blocks m={m}")
        x = inputs.activations(m, k, seed=[8, 11, 2, m])
        xd = torch.from_numpy(x).to(DEV)
        y = L.linear(xd, codes, cb)
        y2 = L.linear(xd, codes, cb2)
        torch.cuda.synchronize()
        assert rel_err(y.cpu().numpy(), x, wh) <= 2.5e-4
        assert rel_err(y2.cpu().numpy(), x, wh2) <= TOL


def test_linear_split_k_two_tiles():
    """Split-K with two batch tiles (17 <= m <= 32) at every supported K, on ragged row counts:
    at K = 8192 two workgroups add their K halves into y with float atomics after zeroing it,
    so y is prefilled with NaN (every output must be overwritten) and each call is repeated
    to check that the result is the same bit for bit. A grouped call equals single calls."""
    for k in (1024, 2048, 4096, 8192):
        ns = (300, 4099)
        tensors = [prepare(n, k, [8, 21, k % 1000, j]) for j, n in enumerate(ns)]
        codes = [gpu_encode(w, p) for w, p, r in tensors]
        whs = [O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
               for w, p, r in tensors]
        for m in (17, 24, 32):
            assert all(L.linear_path(4, m, k, n) == "splitk" for n in ns)
            _say(f"split-K two tiles k={k} m={m}")
            x = inputs.activations(m, k, seed=[8, 21, k % 1000, m])
            xd = torch.from_numpy(x).to(DEV)
            for (c, cb), wh, n in zip(codes, whs, ns):
                y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
                L.linear(xd, c, cb, out=y)
                y2 = L.linear(xd, c, cb)
                torch.cuda.synchronize()
                assert torch.isfinite(y).all()
                assert torch.equal(y, y2)
                assert rel_err(y.cpu().numpy(), x, wh) <= 2.5e-4
            ys = L.linear_multi(xd, [c for c, _ in codes], [cb for _, cb in codes])
            for (c, cb), yg in zip(codes, ys):
                y1 = L.linear(xd, c, cb)
                torch.cuda.synchronize()
                assert torch.equal(yg, y1)


def test_linear_long_rows_unsupported():
    """The stepped MFMA kernel reads a workgroup's 128 rows through one buffer descriptor, so
    it refuses rows of 2^31 / 128 bytes or more (k >= 2^25 at 4 bits, k >= 2^24 at 8 bits)
    with UNSUPPORTED before launching anything; the output buffer is left untouched."""
    m, n = 9, 1
    for bits, k in ((4, 1 << 25), (8, 1 << 24)):
        assert L.linear_path(bits, m, k, n) == "mfma"
        _say(f"long rows bits={bits} k={k}")
        x = torch.zeros((m, k), dtype=torch.float16, device=DEV)
        codes = torch.zeros((n, k // 2 if bits == 4 else k), dtype=torch.uint8, device=DEV)
        cb = np.zeros(16 if bits == 4 else 256, dtype=np.float32)
        y = torch.full((m, n), 7.0, dtype=torch.float32, device=DEV)
        fn = L.linear if bits == 4 else L.linear8
        with pytest.raises(L.LogbqError) as e:
            fn(x, codes, cb, out=y)
        assert e.value.status == L.ERR_UNSUPPORTED
        torch.cuda.synchronize()
        assert torch.all(y == 7.0).item()
        del x, codes


def test_linear_split_k_pairs_narrow():
    """Narrow layers split K over workgroup pairs (float atomic adds onto a zeroed y), chosen
    per linear from its own row count: K = 8192 with 2047 rows (128 blocks) at m <= 8 and up
    to 8192 rows above m = 8, K = 4096 above m = 12 with up to 2048 rows. y is prefilled with
    NaN, each call is repeated and must give the same bits. A grouped call equals single calls
    when its linears take different configurations (m = 8: 2047 rows split, 5000 rows not; two
    launches) and when they share one (m = 12: both split, one launch)."""
    cases = {8192: (2047, 5000), 4096: (1000,)}
    for k, ns in cases.items():
        tensors = [prepare(n, k, [8, 24, k % 1000, j]) for j, n in enumerate(ns)]
        codes = [gpu_encode(w, p) for w, p, r in tensors]
        whs = [O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
               for w, p, r in tensors]
        del tensors
        for m in ((4, 5, 8, 9, 12, 16) if k == 8192 else (13, 16)):
            x = inputs.activations(m, k, seed=[8, 24, k % 1000, m])
            xd = torch.from_numpy(x).to(DEV)
            for (c, cb), wh, n in zip(codes, whs, ns):
                assert L.linear_path(4, m, k, n) == "splitk"
                _say(f"split-K narrow k={k} n={n} m={m} kernel {L.linear_kernel(4, m, k, n)}")
                y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
                L.linear(xd, c, cb, out=y)
                y2 = L.linear(xd, c, cb)
                torch.cuda.synchronize()
                assert torch.isfinite(y).all()
                assert torch.equal(y, y2)
                assert rel_err(y.cpu().numpy(), x, wh) <= 2.5e-4
            if len(codes) > 1:
                ys = L.linear_multi(xd, [c for c, _ in codes], [cb for _, cb in codes])
                for (c, cb), yg in zip(codes, ys):
                    y1 = L.linear(xd, c, cb)
                    torch.cuda.synchronize()
                    assert torch.equal(yg, y1)


def test_linear_split_k_14336():
    """Split-K at K = 14336 on 4099 rows (257 blocks of 16, so a workgroup pair takes two or
    three blocks and the last block has 3 rows): workgroup pairs of 14 wavefronts add their K
    halves into y with float atomics after zeroing it, with two batch groups up to m = 8 and
    one above; above m = 16 the stepped kernel runs (64-row workgroups, K in two parts). y is
    prefilled with NaN (every output must be overwritten), each call is repeated and must give
    the same bits, and a grouped call (4099 and the first 4096 rows) equals single calls."""
    n, k = 4099, 14336
    w, p, r = prepare(n, k, [8, 23, 1, 0])
    c, cb = gpu_encode(w, p)
    wh = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
    del w
    c2 = c[:4096]
    for m in (3, 4, 5, 8, 9, 12, 16, 17, 33, 48):
        path = "splitk" if m <= 16 else "mfma"
        assert L.linear_path(4, m, k, n) == path and L.linear_path(4, m, k, 4096) == path
        _say(f"split-K k={k} m={m} kernel {L.linear_kernel(4, m, k, n)}")
        x = inputs.activations(m, k, seed=[8, 23, 2, m])
        xd = torch.from_numpy(x).to(DEV)
        y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
        L.linear(xd, c, cb, out=y)
        y2 = L.linear(xd, c, cb)
        torch.cuda.synchronize()
        assert torch.isfinite(y).all()
        assert torch.equal(y, y2)
        assert rel_err(y.cpu().numpy(), x, wh) <= 2.5e-4
        ys = L.linear_multi(xd, [c, c2], [cb, cb])
        y3 = L.linear(xd, c2, cb)
        torch.cuda.synchronize()
        assert torch.equal(ys[0], y) and torch.equal(ys[1], y3)


def test_linear_stepped_shapes():
    """The stepped MFMA kernel in the launch shapes its cost model picks: 64- and 128-row
    workgroups, one to eight batch tiles, K in one part or in two (outputs zeroed, then two
    atomic adds each), ragged row counts (1000, 2049, 4097), K outside the split-K set (3072)
    and in it, m from 9 to 200 (two batch blocks above 128). y is prefilled with NaN, each call
    is repeated and must give the same bits, and every output is within tolerance of the
    oracle."""
    parts_seen = set()
    for n, k in ((1000, 3072), (4097, 2048), (1000, 8192), (2049, 8192)):
        w, p, r = prepare(n, k, [8, 25, k % 1000, n])
        c, cb = gpu_encode(w, p)
        wh = O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
        del w
        for m in (9, 24, 33, 64, 96, 97, 128, 129, 200):
            if L.linear_path(4, m, k, n) != "mfma":
                continue   # split-K territory
            name = L.linear_kernel(4, m, k, n)
            narrow, tiles, parts = stepped_shape(m, k, n)
            _say(f"stepped n={n} k={k} m={m} kernel {name} K parts {parts}")
            assert name == stepped_name(m, k, n), name
            parts_seen.add((narrow, parts))
            x = inputs.activations(m, k, seed=[8, 25, n, m])
            xd = torch.from_numpy(x).to(DEV)
            y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
            L.linear(xd, c, cb, out=y)
            y2 = L.linear(xd, c, cb)
            torch.cuda.synchronize()
            assert torch.isfinite(y).all()
            assert torch.equal(y, y2)
            assert rel_err(y.cpu().numpy(), x, wh) <= 2.5e-4
    assert parts_seen == {(True, 1), (True, 2), (False, 1), (False, 2)}


@pytest.mark.parametrize("kind", ["table4", "bits8"])
def test_linear_stepped_shapes_lds_table(kind):
    """The stepped kernel with the LDS table (a 4-bit codebook that is not sign-symmetric, and
    8-bit codes) in the launch shapes its cost model picks, 64- and 128-row workgroups and K in
    one or two parts, on ragged row counts: each call is repeated and must give the same bits,
    and every output is within tolerance of the oracle's product with the dequantized codes."""
    rng = np.random.default_rng(31)
    bits = 8 if kind == "bits8" else 4
    seen = set()
    for n, k in ((1000, 3072), (1000, 8192), (2049, 8192)):
        codes_np = rng.integers(0, 1 << bits, size=(n, k), dtype=np.uint8)
        if bits == 8:
            cb = (rng.standard_normal(256) * 0.01).astype(np.float32)
            codes = torch.from_numpy(codes_np).to(DEV)
        else:
            cb = (rng.standard_normal(16) * 0.01).astype(np.float32)
            codes = torch.from_numpy(O.pack(codes_np)).to(DEV)
        wh = O.dequantize(codes_np, cb)
        lin = L.linear8 if bits == 8 else L.linear
        for m in (33, 64, 97, 128, 200):
            if L.linear_path(bits, m, k, n) != "mfma":
                continue
            name = L.linear_kernel(bits, m, k, n, cb)
            narrow, tiles, parts = stepped_shape(m, k, n, kind)
            _say(f"stepped {kind} n={n} k={k} m={m} kernel {name} K parts {parts}")
            assert name == stepped_name(m, k, n, kind), name
            seen.add((narrow, parts))
            x = inputs.activations(m, k, seed=[8, 31, n, m])
            xd = torch.from_numpy(x).to(DEV)
            y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
            lin(xd, codes, cb, out=y)
            y2 = lin(xd, codes, cb)
            torch.cuda.synchronize()
            assert torch.isfinite(y).all()
            assert torch.equal(y, y2)
            assert rel_err(y.cpu().numpy(), x, wh) <= TOL
    assert (True, 2) in seen and (False, 2) in seen and (True, 1) in seen


@pytest.mark.parametrize("kind", ["fitted4", "table4", "fitted8"])
def test_linear_stepped_narrow_equals_wide(kind):
    """With K in one part every launch shape gives every output the same K walk, so shapes
    agree bit for bit: a 16385-row linear (257 workgroups of 64 rows would not fit, so 128-row
    workgroups) against its first 16384 rows (256 workgroups of 64 rows, or, from m = 64 with a
    fitted codebook, 128-row workgroups with half the batch tiles), with register tables (a
    fitted 4-bit codebook) and with the LDS table (a 4-bit codebook that is not sign-symmetric,
    and 8-bit codes)."""
    n, k = 16385, 3072
    bits = 8 if kind == "fitted8" else 4
    w, _, _ = prepare(64, 256, [8, 26, 0, 0])
    if kind == "table4":
        cb = torch.linspace(-0.07, 0.08, 16, dtype=torch.float32)
    else:
        p = L.fit(w, 8, 1e-6) if bits == 8 else L.fit(w)
        _, cb = gpu_encode(w, p)
    lin = L.linear8 if bits == 8 else L.linear
    gen = torch.Generator(device=DEV)
    gen.manual_seed(26)
    c = torch.randint(0, 256, (n, k * bits // 8), dtype=torch.uint8, device=DEV, generator=gen)
    cbh = None if kind == "fitted4" else np.asarray(cb, dtype=np.float32)
    for m in ((9, 24, 33, 64, 96) if kind == "fitted4" else (9, 24, 33, 64)):
        wide = L.linear_kernel(bits, m, k, n, cbh)
        narrow = L.linear_kernel(bits, m, k, n - 1, cbh)
        _say(f"stepped {kind} wide {wide} vs narrow {narrow}, k={k} m={m}")
        assert wide.startswith("k_mfma2<") and narrow != wide
        # 12 steps of 256: one K part in both shapes
        assert kind != "fitted4" or m >= 64 or narrow.startswith("k_mfma2_narrow<")
        x = torch.from_numpy(inputs.activations(m, k, seed=[8, 26, 1, m])).to(DEV)
        y = lin(x, c, cb)
        y1 = lin(x, c[: n - 1], cb)
        torch.cuda.synchronize()
        assert torch.isfinite(y).all()
        assert torch.equal(y[:, : n - 1], y1)


def test_linear_multi_matches_single_launches():
    """Grouped launch of linears sharing x: every output equals the single-linear call bit for
    bit, and the oracle within tolerance (qkv-like and gate/up-like groups, ragged sizes)."""
    k = 2048
    # the last group mixes paths at m = 8 (8 * 8192 rows picks the MFMA kernel, 64 rows the GEMV)
    groups = [[2048, 512, 512], [4096, 4096], [37, 1000, 1, 64], [300], [8192, 64]]
    for gi, ns in enumerate(groups):
        tensors = [prepare(n, k, [8, 7, gi, j]) for j, n in enumerate(ns)]
        codes = [gpu_encode(w, p) for w, p, r in tensors]
        whs = [O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
               for w, p, r in tensors]
        for m in (1, 2, 3, 4, 8, 16):
            _say(f"linear_multi group {ns} m={m}")
            x = inputs.activations(m, k, seed=[8, 7, gi, 100 + m])
            xd = torch.from_numpy(x).to(DEV)
            ys = L.linear_multi(xd, [c for c, _ in codes], [cb for _, cb in codes])
            for (c, cb), y, wh in zip(codes, ys, whs):
                y1 = L.linear(xd, c, cb)
                torch.cuda.synchronize()
                assert torch.equal(y, y1)
                assert rel_err(y.cpu().numpy(), x, wh) <= TOL


def test_linear_multi_mixed_gemv_configurations():
    """At one batch row and k = 8192, linears of up to 4096 rows take two wavefronts per row and
    wider ones one; a grouped call then launches one GEMV per configuration, and every output
    still equals the single-linear call bit for bit (and the oracle within tolerance)."""
    k = 8192
    ns = [4096, 4160, 2048, 300]
    tensors = [prepare(n, k, [8, 9, 0, j]) for j, n in enumerate(ns)]
    codes = [gpu_encode(w, p) for w, p, r in tensors]
    whs = [O.dequantize(O.encode(w, r.base, r.shift), O.codebook(r.base, r.shift))
           for w, p, r in tensors]
    for m in (1, 2):
        _say(f"linear_multi mixed configurations {ns} m={m}")
        x = inputs.activations(m, k, seed=[8, 9, 1, m])
        xd = torch.from_numpy(x).to(DEV)
        ys = L.linear_multi(xd, [c for c, _ in codes], [cb for _, cb in codes])
        for (c, cb), y, wh in zip(codes, ys, whs):
            y1 = L.linear(xd, c, cb)
            torch.cuda.synchronize()
            assert torch.equal(y, y1)
            assert rel_err(y.cpu().numpy(), x, wh) <= 2.5e-4


# ---------------------------------------------------------------- full-size, sampled

def test_full_size_layer_8192x28672_sampled():
    """The 8192 x 28672 layer (t3 * 0.015 weights) at every batch size of the sweep, in the
    launch configuration the benchmark uses; codes and y compared on sampled rows."""
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    n, k = lin.n, lin.k
    _say("full-size layer: generate + fit")
    wd = inputs.student_t_weights(n, k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                  device=DEV)
    w = wd.cpu().numpy()
    _say("full-size layer: oracle fit")
    r = O.fit(w)
    p = L.fit(w)
    assert (p.base, p.shift, p.wmin, p.wmax, p.wmin_index) == \
        (r.base, r.shift, r.wmin, r.wmax, r.wmin_index)
    rows = np.sort(np.random.default_rng(0).choice(n, size=48, replace=False))
    rows = np.concatenate([rows, [0, n - 1]])
    wsub = w[rows]
    del w
    _say("full-size layer: encode")
    codes, cb = L.encode(wd, p)
    torch.cuda.synchronize()
    del wd
    got = codes[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    c_sub = O.encode(wsub, r.base, r.shift)
    assert np.array_equal(got, O.pack(c_sub))
    wh = O.dequantize(c_sub, O.codebook(r.base, r.shift))
    for m in wl["batch"]:
        _say(f"full-size layer: linear m={m}")
        x = inputs.activations(m, k, seed=[wl["cfg"], 0, 0, 1])
        y = L.linear(torch.from_numpy(x).to(DEV), codes, cb)
        torch.cuda.synchronize()
        ys = y[:, torch.from_numpy(rows).to(DEV)].cpu().numpy()
        assert rel_err(ys, x, wh) <= TOL
