"""Every output row at full size against the oracle: the 8192 -> 28672 layer (0.015 t3
weights) at every batch size of the sweep (m = 1, 8, 32, 128), and one 4096-wide decoder layer
(q, k, v, o, gate, up, down; 0.02 t4 weights) in the grouped launch configuration the decode
benchmark times, at m = 1 and 4 (Sec. 3.3 product, Eq. 1 codes).

Codes are compared bit for bit on every row; y on every element with the normalised bar
max |y - y_ref| / (||x_m|| ||W_hat_n||) <= 1e-3. Output buffers are filled with NaN before each
call, so an element no launch writes fails. The oracle (fit on the whole tensor, log-domain
encode, float64 product) runs in row chunks on a pool of host threads; its parameters come from
the oracle's own fit."""
import concurrent.futures as cf
import os

import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3
DEV = "cuda:0"
CHUNK = 1024


def _say(msg):
    print(msg, flush=True)


def _workers():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _check_rows(w, r, codes_host, xs, ys_host, label):
    """Oracle codes and products of every row, in chunks on a thread pool (BLAS limited to one
    thread per worker). Returns the largest normalised error per batch size."""
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:
        threadpool_limits = None
    lut = O.codebook(r.base, r.shift)
    n = w.shape[0]
    xns = {m: np.linalg.norm(x.astype(np.float64), axis=1)[:, None] for m, x in xs.items()}

    def one(i0):
        i1 = min(n, i0 + CHUNK)
        c = O.encode(w[i0:i1], r.base, r.shift)
        if not np.array_equal(O.pack(c), codes_host[i0:i1]):
            bad = int(np.count_nonzero(O.pack(c) != codes_host[i0:i1]))
            return i0, None, bad
        wh = O.dequantize(c, lut).astype(np.float64)
        wn = np.linalg.norm(wh, axis=1)[None, :]
        errs = {}
        for m, x in xs.items():
            y_ref = x.astype(np.float64) @ wh.T
            y = ys_host[m][:, i0:i1].astype(np.float64)
            if not np.all(np.isfinite(y)):
                errs[m] = float("inf")
                continue
            den = xns[m] * wn
            den[den == 0] = 1.0
            errs[m] = float(np.max(np.abs(y - y_ref) / den))
        return i0, errs, 0

    ctx = threadpool_limits(limits=1) if threadpool_limits else None
    worst = {m: 0.0 for m in xs}
    try:
        with cf.ThreadPoolExecutor(max_workers=_workers()) as pool:
            done = 0
            for i0, errs, bad in pool.map(one, range(0, n, CHUNK)):
                assert errs is not None, f"{label}: {bad} code bytes differ in rows {i0}.."
                for m, e in errs.items():
                    worst[m] = max(worst[m], e)
                done += 1
                if done % 8 == 0:
                    _say(f"  {label}: {min(n, done * CHUNK)} of {n} rows checked")
    finally:
        if ctx is not None:
            ctx.unregister()
    return worst


def test_layer_8192x28672_every_row():
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    n, k = lin.n, lin.k
    _say("layer 8192x28672: generate")
    wd = inputs.student_t_weights(n, k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                  device=DEV)
    w = wd.cpu().numpy()
    _say("layer 8192x28672: oracle fit and library fit")
    r = O.fit(w)
    p = L.fit(w)
    assert (p.base, p.shift) == (r.base, r.shift)
    codes, cb = L.encode(wd, p)
    torch.cuda.synchronize()
    del wd
    xs, ys = {}, {}
    for m in wl["batch"]:
        _say(f"layer 8192x28672: linear m={m} (path {L.linear_kernel(4, m, k, n, cb)})")
        xs[m] = inputs.activations(m, k, seed=[wl["cfg"], 0, 0, 1])
        y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
        L.linear(torch.from_numpy(xs[m]).to(DEV), codes, cb, out=y)
        torch.cuda.synchronize()
        ys[m] = y.cpu().numpy()
    codes_host = codes.cpu().numpy()
    del codes
    worst = _check_rows(w, r, codes_host, xs, ys, "layer 8192x28672")
    _say(f"layer 8192x28672: worst normalised error per m {worst}")
    for m, e in worst.items():
        assert e <= TOL, (m, e)


def test_decode_layer_4096_every_row():
    """Layer 0 of the 32-layer 4096-wide decode workload, launched as the benchmark launches it:
    q/k/v and gate/up grouped, o and down single (GEMV, grouped GEMV, split-row GEMV, and at
    m = 4 the grouped split-K MFMA kernel)."""
    name = "decode_8b_32x7"
    wl = inputs.WORKLOADS[name]
    lins = {lin.name: lin for lin in wl["layers"]}
    tensors = {}
    for lin in wl["layers"]:
        _say(f"{name}: {lin.name} {lin.k}->{lin.n}: generate, fit, encode")
        wd = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"],
                                      seed=[wl["cfg"], 0, inputs.PROJ[lin.name], 0], device=DEV)
        w = wd.cpu().numpy()
        r = O.fit(w)
        p = L.fit(w)
        assert (p.base, p.shift) == (r.base, r.shift)
        codes, cb = L.encode(wd, p)
        torch.cuda.synchronize()
        tensors[lin.name] = (w, r, codes, cb)
        del wd
    ms = (1, 4)
    xs = {(m, kk): inputs.activations(m, kk, seed=[wl["cfg"], 0, 98, kk + m])
          for m in ms for kk in {l.k for l in lins.values()}}
    ys = {g: {} for g in lins}
    for m in ms:
        for group in (["q", "k", "v"], ["o"], ["gate", "up"], ["down"]):
            kk = lins[group[0]].k
            xd = torch.from_numpy(xs[(m, kk)]).to(DEV)
            outs = [torch.full((m, lins[g].n), float("nan"), dtype=torch.float32, device=DEV)
                    for g in group]
            _say(f"{name} m={m} {'+'.join(group)}: "
                 f"{[L.linear_kernel(4, m, kk, lins[g].n, tensors[g][3]) for g in group]}")
            if len(group) == 1:
                L.linear(xd, tensors[group[0]][2], tensors[group[0]][3], out=outs[0])
            else:
                L.linear_multi(xd, [tensors[g][2] for g in group], [tensors[g][3] for g in group],
                               outs=outs)
            torch.cuda.synchronize()
            for g, y in zip(group, outs):
                ys[g][m] = y.cpu().numpy()
    for g, lin in lins.items():
        w, r, codes, _ = tensors[g]
        worst = _check_rows(w, r, codes.cpu().numpy(), {m: xs[(m, lin.k)] for m in ms}, ys[g],
                            f"{name} {g}")
        _say(f"{name} {g}: worst normalised error per m {worst}")
        for m, e in worst.items():
            assert e <= TOL, (g, m, e)
