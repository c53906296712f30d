"""logbq_gptq_noalloc (the GPTQ entry point that allocates nothing: its error workspace is a
fixed array in the library) against logbq_gptq with a caller-provided workspace, through the
C ABI: codes and error-compensated weights bit for bit, on two calls in a row (the second with
fewer rows and columns, so it runs over what the first left in the array), for LogbQuant's and
the baseline's quantizer; and the row limit."""
import ctypes

import numpy as np
import pytest

from oracle import gptq_oracle as G
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
MAX_ROWS = 16384


def _say(msg):
    print(msg, flush=True)


def _case(n, k, seed):
    w = inputs.student_t_weights(n, k, 4, 0.02, seed=[seed, n, k, 0])
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((2 * k, k)).astype(np.float32)
    u = G.hessian_factor(x)
    return w, u


def _run(fn_name, w, u, params, with_ws):
    h = L.lib()
    wd = torch.from_numpy(w).to(DEV)
    ud = torch.from_numpy(u).to(DEV)
    n, k = w.shape
    codes = torch.full((n, k // 2), 0xAB, dtype=torch.uint8, device=DEV)
    pp = ctypes.byref(params) if isinstance(params, L.Params) else None
    up = ctypes.byref(params) if isinstance(params, L.Uniform) else None
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if with_ws:
        ws = torch.empty((n, L.GPTQ_BLOCK), dtype=torch.float32, device=DEV)
        r = h.logbq_gptq(ctypes.c_void_p(wd.data_ptr()), n, k, ctypes.c_void_p(ud.data_ptr()), pp, up,
                         ctypes.c_void_p(ws.data_ptr()), ctypes.c_void_p(codes.data_ptr()), st)
    else:
        r = getattr(h, fn_name)(ctypes.c_void_p(wd.data_ptr()), n, k, ctypes.c_void_p(ud.data_ptr()),
                                pp, up, ctypes.c_void_p(codes.data_ptr()), st)
    assert r == L.OK, r
    torch.cuda.synchronize()
    return codes.cpu().numpy(), wd.cpu().numpy()


@pytest.mark.parametrize("scheme", ["logbquant", "uniform"])
def test_noalloc_equals_workspace_call(scheme):
    for n, k, seed in ((3000, 544, 61), (37, 160, 62)):
        _say(f"gptq_noalloc {scheme} n={n} k={k}")
        w, u = _case(n, k, seed)
        params = L.fit(w) if scheme == "logbquant" else L.fit_uniform(w)
        c_ref, w_ref = _run("logbq_gptq", w, u, params, with_ws=True)
        c_got, w_got = _run("logbq_gptq_noalloc", w, u, params, with_ws=False)
        assert np.array_equal(c_got, c_ref)
        assert np.array_equal(w_got.view(np.uint32), w_ref.view(np.uint32))


def test_noalloc_row_limit():
    h = L.lib()
    w = inputs.student_t_weights(8, 64, 4, 0.02, seed=[63, 0, 0, 0])
    p = L.fit(w)
    a = ctypes.c_void_p(4096)
    assert h.logbq_gptq_noalloc(a, MAX_ROWS + 1, 64, a, ctypes.byref(p), None, a, None) == \
        L.ERR_UNSUPPORTED
    assert h.logbq_gptq_noalloc(None, 0, 64, None, ctypes.byref(p), None, None, None) == L.OK
    assert h.logbq_gptq_noalloc(None, 4, 64, a, ctypes.byref(p), None, a, None) == L.ERR_INVALID_ARG
