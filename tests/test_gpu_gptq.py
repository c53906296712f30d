"""GPU parity of GPTQ calibration (logbq_gptq) against the float32 oracle, through the C ABI:
the codes and the error-compensated weights bit for bit (both follow the same fixed order of
separately rounded float32 operations), with LogbQuant's and with the asymmetric linear
baseline's quantizer, over ragged row counts and K with a partial last block of 128."""
import numpy as np
import pytest

from oracle import gptq_oracle as G
from oracle import logbq_oracle as O
from oracle import uniform_oracle as U
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


def _inputs(t, k, seed):
    rng = np.random.default_rng(seed)
    scale = np.exp(rng.normal(0.0, 0.5, k))
    x = rng.standard_normal((t, k)) * scale + rng.standard_normal((t, 8)) @ rng.standard_normal((8, k)) * 0.5
    return x.astype(np.float32)


@pytest.mark.parametrize("n,k", [(64, 256), (37, 160), (8, 32), (300, 544), (9, 1024)])
@pytest.mark.parametrize("scheme", ["logbquant", "uniform"])
def test_gptq_bit_exact(n, k, scheme):
    _say(f"gptq {scheme} n={n} k={k}")
    w = np.asarray(inputs.student_t_weights(n, k, 4, 0.02, seed=[47, n, k, 0]))
    x = _inputs(max(2 * k, 256), k, [47, n, k, 1])
    u = G.hessian_factor(x)
    if scheme == "logbquant":
        r = O.fit(w)
        lut = O.codebook(r.base, r.shift)
        params = L.fit(w)

        def q(col):
            c = O.encode(col, r.base, r.shift)
            return c, lut[c]
    else:
        f = U.uniform_fit(w)
        lut = U.uniform_levels(f.scale, f.zero)
        params = L.fit_uniform(w)

        def q(col):
            c = U.uniform_encode(col, f.scale, f.zero)
            return c, lut[c]
    codes_ref, w_ref = G.gptq(w, u, q)
    wd = torch.from_numpy(w).to(DEV)
    codes = L.gptq(wd, torch.from_numpy(u).to(DEV), params)
    torch.cuda.synchronize()
    got = codes.cpu().numpy()
    exp = O.pack(codes_ref)
    assert np.array_equal(got, exp), f"{np.count_nonzero(got != exp)} code bytes differ"
    wg = wd.cpu().numpy()
    assert np.array_equal(wg.view(np.uint32), w_ref.view(np.uint32)), \
        f"{np.count_nonzero(wg != w_ref)} compensated weights differ"
    # the calibrated codes decode through the library to the oracle's weights
    wq = L.dequantize(codes, params.codebook_array() if scheme == "uniform" else params)
    torch.cuda.synchronize()
    assert np.array_equal(wq.cpu().numpy().view(np.uint32), lut[codes_ref].view(np.uint32))


def test_gptq_identity_factor_equals_encode():
    """With U = I the GPU calibration gives the encoders' codes and leaves W unchanged."""
    n, k = 128, 512
    _say("gptq identity factor")
    w = np.asarray(inputs.student_t_weights(n, k, 3, 0.015, seed=[48, 0, 0, 0]))
    wd = torch.from_numpy(w).to(DEV)
    p = L.fit(w)
    codes = L.gptq(wd.clone(), torch.eye(k, device=DEV), p)
    enc, _ = L.encode(wd, p)
    torch.cuda.synchronize()
    assert torch.equal(codes, enc)
