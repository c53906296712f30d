"""Benchmark of the fused LogbQuant dequantize-and-multiply on one MI355X.

Default workload: the 8192 x 28672 layer (weights 0.015 * t3, 4-bit LogbQuant per tensor,
float16 N(0,1) activations) at batch M = 1. One step is one logbq_linear call on packed codes
already resident in HBM. The codes are held in several copies (>= 1 GiB together) and the
steps cycle through them, so every step streams its weights from HBM and not from the 256 MB
last-level cache. value = packed weight bytes (N * K / 2) per step / time per step.

The same run also measures, each in its own timed region:
  * decode weight passes: 16 layers x 7 linears (1B-shaped) and 32 x 7 (8B-shaped) at M = 1,
    and the 8B-shaped pass at M = 4, each captured once in a HIP graph and replayed per
    token (tokens/s = M / time per pass);
  * the same layer at M = 8, 32, 128 (GEMV and MFMA paths);
  * logbq_encode of the layer's float32 weights;
  * the 2048 x 8192 up-projection and the 2048 x 2048 linear at M = 1.
And, on the host, the CPU oracle (dequantize + float64 matmul) on a row sample of the layer.

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--quick]
"""
import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused LogbQuant GEMV effective weight GB/s (% HBM peak) + decode tokens/s, M=1"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
ROTATE_BYTES = 1 << 30


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Calls:
    """Pre-marshalled logbq_linear / logbq_linear_multi arguments, so that the timed loop (or the
    graph capture) only calls the library."""

    def __init__(self, L, stream):
        self.L = L
        self.fn = L.lib().logbq_linear
        self.fn8 = L.lib().logbq_linear8
        self.fn_multi = L.lib().logbq_linear_multi
        self.stream = ctypes.c_void_p(stream)
        self.args = []
        self.keep = []

    def add(self, x, codes, cb, y):
        """logbq_linear for 16-entry codebooks, logbq_linear8 for 256-entry ones."""
        cbarr = np.ascontiguousarray(cb, dtype=np.float32)
        self.keep.append(cbarr)
        fn = self.fn8 if cbarr.size == 256 else self.fn
        self.args.append((fn, (ctypes.c_void_p(x.data_ptr()), x.shape[0], x.shape[1],
                                    ctypes.c_void_p(codes.data_ptr()), codes.shape[0],
                                    cbarr.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                    ctypes.c_void_p(y.data_ptr()), self.stream)))

    def add_multi(self, x, codes_list, cbs, ys):
        cnt = len(codes_list)
        arrs = [np.ascontiguousarray(cb, dtype=np.float32) for cb in cbs]
        cptr = (ctypes.c_void_p * cnt)(*[c.data_ptr() for c in codes_list])
        ns = (ctypes.c_int64 * cnt)(*[c.shape[0] for c in codes_list])
        cbp = (ctypes.POINTER(ctypes.c_float) * cnt)(
            *[a.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for a in arrs])
        yp = (ctypes.c_void_p * cnt)(*[y.data_ptr() for y in ys])
        self.keep.append((arrs, cptr, ns, cbp, yp))
        self.args.append((self.fn_multi, (ctypes.c_void_p(x.data_ptr()), x.shape[0], x.shape[1],
                                          cnt, cptr, ns, cbp, yp, self.stream)))

    def run(self, idx):
        fn, a = self.args[idx]
        st = fn(*a)
        if st != 0:
            raise RuntimeError(f"logbq launch failed with status {st}")


def time_region(torch, stream, fn, steps, warmup):
    """Events around `steps` calls of fn on `stream`; returns ms per call."""
    for i in range(warmup):
        fn(i)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(steps):
        fn(i)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def _capture(torch, L, launches, count, offset=0):
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=cap):
        calls = Calls(L, torch.cuda.current_stream().cuda_stream)
        for a in launches:
            calls.add(*a)
        for i in range(count):
            calls.run((offset + i) % len(launches))
    return graph


WARM_CHUNK = 1000   # launches per captured warmup graph


def time_chain(torch, L, stream, rows):
    """Time several logbq_linear launch sequences back to back on one stream. `rows` is a list
    of (launches, steps, warmup): `launches` a list of (x, codes, cb, y), launch i of a row
    using entry i % len(launches); each row takes `warmup` untimed launches and then exactly
    `steps` timed ones between two events. The launches are captured in HIP graphs so that
    host launch cost cannot starve the GPU. All graphs are captured first; the rows are then
    replayed in order with no host synchronisation in between (one synchronisation after the
    last), so every row's timed launches run on a GPU that has been busy since the first
    row started, instead of after an idle gap in which its clocks drop. Returns ms per launch
    for each row."""
    plans = []
    for launches, steps, warmup in rows:
        full, rest = divmod(warmup, WARM_CHUNK)
        warm = _capture(torch, L, launches, WARM_CHUNK) if full else None
        warm_rest = _capture(torch, L, launches, rest) if rest else None
        timed = _capture(torch, L, launches, steps, offset=warmup)
        plans.append((full, warm, warm_rest, timed, steps))
    torch.cuda.synchronize()
    events = []
    with torch.cuda.stream(stream):
        for full, warm, warm_rest, timed, steps in plans:
            for _ in range(full):
                warm.replay()
            if warm_rest is not None:
                warm_rest.replay()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            timed.replay()
            e1.record(stream)
            events.append((e0, e1, steps))
    torch.cuda.synchronize()
    return [e0.elapsed_time(e1) / steps for e0, e1, steps in events]


def time_launches(torch, L, stream, launches, steps, warmup):
    """time_chain for one row: ms per launch of exactly `steps` launches after `warmup`."""
    return time_chain(torch, L, stream, [(launches, steps, warmup)])[0]


def aux_counts(steps, warmup):
    """Timed and warmup launches of a row other than the headline: at least 500 of each
    whatever --steps / --warmup ask for the headline (64 launches after one warmup launch ran
    7-17 % slower than the same rows timed over 500)."""
    return max(500, steps // 4), max(500, warmup // 4)


def make_tensor(torch, L, inputs, lin, wl, seed, dev):
    """Generate one weight tensor on the GPU, fit it on the host, encode it on the GPU."""
    wd = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"], seed=seed, device=dev,
                                  outlier_frac=wl.get("outlier_frac", 0.0))
    p = L.fit(wd.cpu().numpy())
    codes, cb = L.encode(wd, p)
    return codes, cb


def bench_layer(torch, L, inputs, dev, stream, ms, steps, warmup, with_encode=True):
    """The 8192 x 28672 layer: rotation copies, M sweep, encode timing."""
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    n, k = lin.n, lin.k
    log("layer 8192x28672: generate / fit / encode")
    wd = inputs.student_t_weights(n, k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                  device=dev)
    w = wd.cpu().numpy()
    t0 = time.perf_counter()
    p = L.fit(w)
    fit_s = time.perf_counter() - t0
    del w
    results = {}
    # device fit (exact sums of Eq. 5): three passes over the 0.94 GB tensor, each followed by a
    # copy of its bins to the host; wall clock of the blocking call
    ws = torch.empty(L.FIT_WORKSPACE_BYTES, dtype=torch.uint8, device=dev)
    L.fit_device(wd, workspace=ws, stream=stream)
    fit_times = []
    for _ in range(7):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pd = L.fit_device(wd, workspace=ws, stream=stream)
        fit_times.append(time.perf_counter() - t0)
    fit_dev_ms = float(np.median(fit_times)) * 1e3
    same = (pd.wmin, pd.wmax, pd.wmin_index, pd.base, pd.shift) == \
        (p.wmin, p.wmax, p.wmin_index, p.base, p.shift)
    log(f"device fit: {fit_dev_ms:.3f} ms (host fit {fit_s:.2f} s), same parameters: {same}")
    results["fit_device_8192x28672"] = {
        "ms": fit_dev_ms, "host_fit_ms": fit_s * 1e3, "speedup_vs_host_fit": fit_s * 1e3 / fit_dev_ms,
        "passes": 3, "read_GB_s": 3 * n * k * 4 / fit_dev_ms / 1e6,
        "hbm_frac": 3 * n * k * 4 / fit_dev_ms / 1e6 / HBM_PEAK_GBS,
        "same_params_as_host_fit": same}
    del ws
    codes, cb = L.encode(wd, p)
    torch.cuda.synchronize()
    packed = n * k // 2
    copies = max(2, -(-ROTATE_BYTES // packed))
    code_list = [codes] + [codes.clone() for _ in range(copies - 1)]
    # encode: 1 float32 tensor of 0.94 GB is read per call (larger than the last-level cache)
    if with_encode:
        enc_out = torch.empty_like(codes)

        def enc(i):
            L.encode(wd, p, out=enc_out, stream=stream)
        enc_ms = time_region(torch, stream, enc, max(5, steps // 20), 100)
        assert torch.equal(enc_out, codes)
        enc_bytes = n * k * 4 + packed
        results["encode_8192x28672"] = {"ms": enc_ms, "GB_s": enc_bytes / enc_ms / 1e6,
                                        "hbm_frac": enc_bytes / enc_ms / 1e6 / HBM_PEAK_GBS,
                                        "bytes": enc_bytes}
    del wd
    # The other batch sizes first, the headline (ms[0]) last, all back to back on one stream:
    # the headline's warmup launches start on a GPU that is already at its working clocks.
    order = list(ms[1:]) + [ms[0]]
    aux_steps, aux_warm = aux_counts(steps, warmup)
    plan = []
    for m in order:
        x = inputs.activations(m, k, seed=[wl["cfg"], 0, 0, 1], device=dev)
        launches = [(x, c, cb, torch.empty((m, n), dtype=torch.float32, device=dev))
                    for c in code_list]
        plan.append((launches, steps, warmup) if m == ms[0] else (launches, aux_steps, aux_warm))
    times = time_chain(torch, L, stream, plan)
    for m, (_, timed, warm), t in sorted(zip(order, plan, times), key=lambda r: ms.index(r[0])):
        log(f"layer m={m}: {t * 1e3:.2f} us per launch")
        algo = packed + 2 * m * k + 4 * m * n + 64
        flops = 2.0 * m * n * k
        results[f"linear_8192x28672_m{m}"] = {
            "ms": t, "us": t * 1e3, "launches_timed": timed, "warmup_launches": warm,
            "weight_GB_s": packed / t / 1e6,
            "algo_GB_s": algo / t / 1e6, "hbm_frac": algo / t / 1e6 / HBM_PEAK_GBS,
            "TFLOP_s": flops / t / 1e9, "mfma_frac": flops / t / 1e9 / MFMA_F16_PEAK_TFLOPS,
            "algo_bytes": algo,
            "path": L.linear_path(4, m, k, n), "kernel": L.linear_kernel(4, m, k, n, cb)}
        if m == ms[0] and len(ms) > 1:
            results[f"linear_8192x28672_m{m}"]["preceded_by"] = (
                "the m = " + ", ".join(str(v) for v in ms[1:]) + " rows on the same stream "
                "with no host synchronisation in between")
    return results, {"n": n, "k": k, "packed": packed, "copies": copies, "fit_s": fit_s,
                     "params": {"base": p.base, "shift": p.shift, "wmin": p.wmin,
                                "wmax": p.wmax}}, codes, cb


def bench_quality(torch, L, inputs, dev, stream, layer_codes, layer_cb, steps, warmup):
    """LogbQuant against the asymmetric linear baseline (Sec. 2, Quant(s, z, x); tensor-wise as
    in Sec. 4) on the single-tensor workloads: reconstruction SQNR, relative error of an M = 4
    product against the float64 product with the unquantized weights, the share of weights on
    the zero level, and, on the 8192 x 28672 layer, the time of the baseline's codes through
    the same linear kernels (their codebook is not sign-symmetric, so every kernel uses its
    LDS-table form)."""
    out = {}
    for name in ("linear_2048x2048", "up_2048x8192_outliers", "layer_8192x28672"):
        wl = inputs.WORKLOADS[name]
        lin = wl["layers"][0]
        log(f"quality {name}")
        w = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                     device=dev, outlier_frac=wl.get("outlier_frac", 0.0))
        w_host = w.cpu().numpy()
        if name == "layer_8192x28672":
            codes, cb = layer_codes, layer_cb
        else:
            codes, cb = L.encode(w, L.fit(w_host))
        u = L.fit_uniform(w_host)
        ucb = u.codebook_array()
        ucodes = L.encode_uniform(w, u)
        x = inputs.activations(4, lin.k, seed=[wl["cfg"], 0, 0, 2], device=dev)
        w64 = w.double()
        y_ref = x.double() @ w64.T
        row = {}
        for scheme, c, book in (("logbquant", codes, cb), ("uniform", ucodes, ucb)):
            wh = L.dequantize(c, book).double()
            err = float(((w64 - wh) ** 2).sum())
            sig = float((w64 ** 2).sum())
            y = L.linear(x, c, book).double()
            row[scheme] = {"sqnr_db": 10.0 * math.log10(sig / err),
                           "gemv_rel_err_m4": float((y - y_ref).norm() / y_ref.norm()),
                           "zero_level_frac": float((wh == 0).double().mean())}
            del wh
        row["uniform"]["params"] = {"scale": u.scale, "zero": u.zero, "wmin": u.wmin, "wmax": u.wmax}
        if name == "layer_8192x28672":
            packed = lin.n * lin.k // 2
            copies = max(2, -(-ROTATE_BYTES // packed))
            code_list = [ucodes] + [ucodes.clone() for _ in range(copies - 1)]
            aux_steps, aux_warm = aux_counts(steps, warmup)
            plan = []
            for m in (1, 8, 32):
                xm = inputs.activations(m, lin.k, seed=[wl["cfg"], 0, 0, 1], device=dev)
                launches = [(xm, c, ucb, torch.empty((m, lin.n), dtype=torch.float32, device=dev))
                            for c in code_list]
                plan.append((launches, aux_steps, aux_warm))
            for m, t in zip((1, 8, 32), time_chain(torch, L, stream, plan)):
                row["uniform"][f"linear_m{m}_us"] = t * 1e3
                row["uniform"][f"linear_m{m}_path"] = L.linear_path(4, m, lin.k, lin.n)
            del code_list
        out[name] = row
        del w, w64, ucodes, y_ref
        torch.cuda.empty_cache()
    return out


def bench_gptq(torch, L, inputs, dev, stream, with_cpu):
    """GPTQ calibration (logbq_gptq) of the 2048 x 2048 and 2048 -> 8192 tensors with seeded
    synthetic calibration inputs (16384 tokens; per-channel scales exp(N(0, 0.25)) plus a shared
    rank-8 part, so the Hessian is far from diagonal). The factor U of the damped inverse
    Hessian is the caller's input; it is formed here with torch in float64 (outside the timed
    region). Reported: GPU time of the calibration and the layer-output error
    ||(W - W_hat) X^T|| / ||W X^T|| of round-to-nearest and of GPTQ, for LogbQuant and for the
    asymmetric linear baseline."""
    out = {}
    tokens = 16384
    for name in ("linear_2048x2048", "up_2048x8192_outliers"):
        wl = inputs.WORKLOADS[name]
        lin = wl["layers"][0]
        n, k = lin.n, lin.k
        log(f"gptq {name}")
        w = inputs.student_t_weights(n, k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                     device=dev, outlier_frac=wl.get("outlier_frac", 0.0))
        gen = torch.Generator(device=dev)
        gen.manual_seed(wl["cfg"] * 1000 + 7)
        scale = torch.exp(0.5 * torch.randn(k, generator=gen, device=dev))
        x = (torch.randn(tokens, k, generator=gen, device=dev) * scale +
             torch.randn(tokens, 8, generator=gen, device=dev) @ torch.randn(8, k, generator=gen, device=dev) * 0.5)
        x64 = x.double()
        h = 2.0 * (x64.T @ x64) / tokens
        h += 0.01 * torch.mean(torch.diag(h)) * torch.eye(k, dtype=torch.float64, device=dev)
        u = torch.linalg.cholesky(torch.cholesky_inverse(torch.linalg.cholesky(h)), upper=True)
        u = u.float().contiguous()
        w_host = w.cpu().numpy()
        y_ref = w.double() @ x64.T
        ynorm = float(y_ref.norm())
        row = {"tokens": tokens}
        for scheme in ("logbquant", "uniform"):
            if scheme == "logbquant":
                params = L.fit(w_host)
                book = params
                rtn_codes, _ = L.encode(w, params)
            else:
                params = L.fit_uniform(w_host)
                book = params.codebook_array()
                rtn_codes = L.encode_uniform(w, params)
            ws = torch.empty((n, L.GPTQ_BLOCK), dtype=torch.float32, device=dev)
            codes = torch.empty((n, k // 2), dtype=torch.uint8, device=dev)
            times = []
            for rep in range(4):
                wc = w.clone()
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                L.gptq(wc, u, params, out_codes=codes, workspace=ws, stream=stream)
                e1.record(stream)
                torch.cuda.synchronize()
                times.append(e0.elapsed_time(e1))

            def err(c):
                wh = L.dequantize(c, book).double()
                return float(((w.double() - wh) @ x64.T).norm()) / ynorm
            row[scheme] = {"gptq_ms": sorted(times)[1], "launches": 2 * (-(-k // L.GPTQ_BLOCK)) - 1,
                           "out_err_rtn": err(rtn_codes), "out_err_gptq": err(codes)}
        if with_cpu:
            from oracle import gptq_oracle as G
            from oracle import logbq_oracle as O
            rows_sample = 128
            r = O.fit(w_host)
            lut = O.codebook(r.base, r.shift)

            def q(col):
                c = O.encode(col, r.base, r.shift)
                return c, lut[c]
            t0 = time.perf_counter()
            G.gptq(w_host[:rows_sample], u.cpu().numpy(), q)
            dt = time.perf_counter() - t0
            row["cpu_oracle"] = {"rows": rows_sample, "s": dt,
                                 "s_scaled_to_all_rows": dt * n / rows_sample}
        out[name] = row
        del w, x, x64, h, u, y_ref
        torch.cuda.empty_cache()
    return out


def bench_layer8(torch, L, inputs, dev, stream, ms, steps, warmup):
    """The 8192 x 28672 layer at 8 bits (q_max = 127, eps = 1e-6): one code byte per weight,
    256-entry table. Same weights and activations as the 4-bit layer."""
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    n, k = lin.n, lin.k
    log("layer 8192x28672 at 8 bits: generate / fit / encode")
    wd = inputs.student_t_weights(n, k, wl["nu"], wl["scale"], seed=[wl["cfg"], 0, 0, 0],
                                  device=dev)
    p = L.fit(wd.cpu().numpy(), 8, 1e-6)
    codes, cb = L.encode(wd, p)
    torch.cuda.synchronize()
    nbytes = n * k
    enc_out = torch.empty_like(codes)

    def enc(i):
        L.encode(wd, p, out=enc_out, stream=stream)
    enc_ms = time_region(torch, stream, enc, max(5, steps // 20), 100)
    assert torch.equal(enc_out, codes)
    del wd, enc_out
    enc_bytes = n * k * 4 + nbytes
    results = {"encode8_8192x28672": {"ms": enc_ms, "GB_s": enc_bytes / enc_ms / 1e6,
                                      "hbm_frac": enc_bytes / enc_ms / 1e6 / HBM_PEAK_GBS,
                                      "bytes": enc_bytes}}
    copies = max(2, -(-ROTATE_BYTES // nbytes))
    code_list = [codes] + [codes.clone() for _ in range(copies - 1)]
    aux_steps, aux_warm = aux_counts(steps, warmup)
    plan = []
    for m in ms:
        x = inputs.activations(m, k, seed=[wl["cfg"], 0, 0, 1], device=dev)
        launches = [(x, c, cb, torch.empty((m, n), dtype=torch.float32, device=dev))
                    for c in code_list]
        plan.append((launches, aux_steps, aux_warm))
    times = time_chain(torch, L, stream, plan)
    for m, t in zip(ms, times):
        timed = aux_steps
        log(f"layer8 m={m}: {t * 1e3:.2f} us per launch")
        algo = nbytes + 2 * m * k + 4 * m * n + 1024
        flops = 2.0 * m * n * k
        results[f"linear8_8192x28672_m{m}"] = {
            "ms": t, "us": t * 1e3, "launches_timed": timed, "weight_GB_s": nbytes / t / 1e6,
            "algo_GB_s": algo / t / 1e6, "hbm_frac": algo / t / 1e6 / HBM_PEAK_GBS,
            "TFLOP_s": flops / t / 1e9, "mfma_frac": flops / t / 1e9 / MFMA_F16_PEAK_TFLOPS,
            "algo_bytes": algo, "copies": copies,
            "path": L.linear_path(8, m, k, n), "kernel": L.linear_kernel(8, m, k, n, cb)}
    del code_list, codes
    return results


def read_ceiling(torch, stream, nbytes=1 << 32, steps=20, warmup=10):
    """HBM read ceiling: the pure streaming-read kernel of libhbmread.so (128-bit non-temporal
    loads, the GEMV's access pattern and prefetch depth, no compute) over a 4 GiB buffer."""
    path = os.path.join(ROOT, "paper_2607_01127_amd", "libhbmread.so")
    lib = ctypes.CDLL(path)
    lib.hbm_read.restype = ctypes.c_int32
    lib.hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
                             ctypes.c_void_p]
    grid = torch.cuda.get_device_properties(0).multi_processor_count
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    buf.fill_(1)
    sink = torch.zeros(grid * 512, dtype=torch.int32, device="cuda:0")
    st = ctypes.c_void_p(stream.cuda_stream)

    def one(i):
        r = lib.hbm_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()),
                         grid, st)
        assert r == 0, r
    ms = time_region(torch, stream, one, steps, warmup)
    del buf, sink
    return {"GB_s": nbytes / ms / 1e6, "bytes": nbytes, "ms": ms,
            "kernel": "k_read (libhbmread.so), 4 KiB per wavefront unit, 2 units in flight"}


def bench_batched(torch, L, inputs, dev, stream, ms, steps, warmup):
    """The distinct linear shapes of the 8B-shaped decoder layer (o: 4096 x 4096, gate/up:
    4096 -> 14336, down: 14336 -> 4096) run one at a time at batch sizes above decode (the
    split-K kernel, the stepped kernel with 64-row workgroups or the K-quartered kernel,
    whichever the path rule takes), codes rotated over copies larger than the last-level
    cache, all rows chained on one stream."""
    wl = inputs.WORKLOADS["decode_8b_32x7"]
    shapes = [lin for lin in wl["layers"] if lin.name in ("o", "gate", "down")]
    plan, keys = [], []
    for lin in shapes:
        log(f"batched {lin.name} {lin.k}->{lin.n}: generate / fit / encode")
        codes, cb = make_tensor(torch, L, inputs, lin, wl, [wl["cfg"], 1, inputs.PROJ[lin.name], 0],
                                dev)
        packed = lin.n * lin.k // 2
        copies = max(2, -(-ROTATE_BYTES // packed))
        code_list = [codes] + [codes.clone() for _ in range(copies - 1)]
        for m in ms:
            x = inputs.activations(m, lin.k, seed=[wl["cfg"], 1, inputs.PROJ[lin.name], m],
                                   device=dev)
            launches = [(x, c, cb, torch.empty((m, lin.n), dtype=torch.float32, device=dev))
                        for c in code_list]
            plan.append((launches, steps, warmup))
            keys.append((lin, m, packed, cb))
    times = time_chain(torch, L, stream, plan)
    out = {}
    for (lin, m, packed, cb), (_, timed, warm), t in zip(keys, plan, times):
        algo = packed + 2 * m * lin.k + 4 * m * lin.n + 64
        flops = 2.0 * m * lin.n * lin.k
        log(f"batched {lin.name} m={m}: {t * 1e3:.2f} us per launch")
        out[f"{lin.name}_{lin.k}x{lin.n}_m{m}"] = {
            "us": t * 1e3, "launches_timed": timed, "warmup_launches": warm,
            "algo_GB_s": algo / t / 1e6, "hbm_frac": algo / t / 1e6 / HBM_PEAK_GBS,
            "TFLOP_s": flops / t / 1e9, "mfma_frac": flops / t / 1e9 / MFMA_F16_PEAK_TFLOPS,
            "path": L.linear_path(4, m, lin.k, lin.n),
            "kernel": L.linear_kernel(4, m, lin.k, lin.n, cb)}
    return out


def bench_small(torch, L, inputs, dev, stream, name, steps, warmup):
    wl = inputs.WORKLOADS[name]
    lin = wl["layers"][0]
    codes, cb = make_tensor(torch, L, inputs, lin, wl, [wl["cfg"], 0, 0, 0], dev)
    packed = lin.n * lin.k // 2
    copies = max(2, -(-ROTATE_BYTES // packed))
    code_list = [codes] + [codes.clone() for _ in range(copies - 1)]
    x = inputs.activations(1, lin.k, seed=[wl["cfg"], 0, 0, 1], device=dev)
    y = torch.empty((1, lin.n), dtype=torch.float32, device=dev)
    timed = steps
    t = time_launches(torch, L, stream, [(x, c, cb, y) for c in code_list], steps, warmup)
    return {"ms": t, "us": t * 1e3, "launches_timed": timed, "weight_GB_s": packed / t / 1e6,
            "hbm_frac": packed / t / 1e6 / HBM_PEAK_GBS, "copies": copies,
            "path": L.linear_path(4, 1, lin.k, lin.n)}


def bench_decode(torch, L, inputs, dev, stream, name, batches, steps, warmup, traffic_only=False):
    """A full decode weight pass in dependency order, captured in a HIP graph. With
    traffic_only, the pass at the first batch size is only replayed four times (for a
    rocprofv3 --pmc FETCH_SIZE run) and nothing is timed."""
    wl = inputs.WORKLOADS[name]
    layers = wl["n_layers"]
    log(f"{name}: generating {layers} x {len(wl['layers'])} tensors")
    tensors = []
    # Quantize at load: every tensor is fitted on the device (logbq_fit_device, exact sums of
    # Eq. 5) and encoded there; only the parameters travel to the host.
    ws = torch.empty(L.FIT_WORKSPACE_BYTES, dtype=torch.uint8, device=dev)
    t0 = time.perf_counter()
    fit_s = 0.0
    for li in range(layers):
        for lin in wl["layers"]:
            wd = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"],
                                          seed=[wl["cfg"], li, inputs.PROJ[lin.name], 0],
                                          device=dev)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            p = L.fit_device(wd, workspace=ws, stream=stream)
            codes, cb = L.encode(wd, p, stream=stream)
            torch.cuda.synchronize()
            fit_s += time.perf_counter() - t1
            tensors.append((lin, codes, cb))
            del wd
        if li % 8 == 7:
            log(f"{name}: {li + 1} layers ready ({time.perf_counter() - t0:.1f} s)")
    setup_s = time.perf_counter() - t0
    del ws
    bytes_pass = sum(lin.n * lin.k // 2 for lin, _, _ in tensors)
    out = {}
    # Launch plan per layer, in dependency order: linears that read the same activations
    # (q, k, v) and (gate, up) go in one grouped launch.
    per_layer = len(wl["layers"])
    plan = []
    for li in range(layers):
        t = tensors[li * per_layer:(li + 1) * per_layer]
        names = [lin.name for lin, _, _ in t]
        groups = [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
        for g in groups:
            plan.append([t[names.index(nm)] for nm in g])
    for m in batches:
        xs = {}
        ys = {}
        leader = {"q": "q", "k": "q", "v": "q", "o": "o", "gate": "gate", "up": "gate",
                  "down": "down"}
        for lin, codes, cb in tensors:
            key = (lin.k, leader[lin.name])
            if key not in xs:
                xs[key] = inputs.activations(m, lin.k, seed=[wl["cfg"], 0, inputs.PROJ[key[1]], 1],
                                             device=dev)
            ys[id(codes)] = torch.empty((m, lin.n), dtype=torch.float32, device=dev)
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=cap):
            calls = Calls(L, torch.cuda.current_stream().cuda_stream)
            for grp in plan:
                x = xs[(grp[0][0].k, leader[grp[0][0].name])]
                if len(grp) == 1:
                    lin, codes, cb = grp[0]
                    calls.add(x, codes, cb, ys[id(codes)])
                else:
                    calls.add_multi(x, [c for _, c, _ in grp], [cb for _, _, cb in grp],
                                    [ys[id(c)] for _, c, _ in grp])
            for i in range(len(plan)):
                calls.run(i)
        if traffic_only:
            for _ in range(4):
                g.replay()
            torch.cuda.synchronize()
            return {"bytes_per_pass": bytes_pass, "launches": len(plan)}
        # check the replay against eager per-linear launches
        g.replay()
        torch.cuda.synchronize()
        ref = {key: y.clone() for key, y in ys.items()}
        for lin, codes, cb in tensors:
            L.linear(xs[(lin.k, leader[lin.name])], codes, cb, out=ys[id(codes)])
        torch.cuda.synchronize()
        assert all(torch.equal(ref[key], ys[key]) for key in ys), "graph replay differs"
        t = time_region(torch, stream, lambda i: g.replay(), steps, warmup)
        log(f"{name} m={m}: {t * 1e3:.1f} us per pass")
        # Sum of launch times: the launches of one group kind (e.g. every layer's gate/up) run
        # back to back in a graph of their own; the four kinds together are the pass's launches
        # without the switches between kinds.
        sum_ms = 0.0
        kinds = {}
        for grp in plan:
            kinds.setdefault(grp[0][0].name, []).append(grp)
        for kind, grps in kinds.items():
            gk = torch.cuda.CUDAGraph()
            torch.cuda.synchronize()
            with torch.cuda.graph(gk, stream=cap):
                ck = Calls(L, torch.cuda.current_stream().cuda_stream)
                for grp in grps:
                    x = xs[(grp[0][0].k, leader[grp[0][0].name])]
                    if len(grp) == 1:
                        ck.add(x, grp[0][1], grp[0][2], ys[id(grp[0][1])])
                    else:
                        ck.add_multi(x, [c for _, c, _ in grp], [cb for _, _, cb in grp],
                                     [ys[id(c)] for _, c, _ in grp])
                for i in range(len(grps)):
                    ck.run(i)
            sum_ms += time_region(torch, stream, lambda i: gk.replay(), max(10, steps // 4), 5)
            del gk
        out[f"m{m}"] = {"ms_per_token_pass": t, "tokens_per_s": m / (t * 1e-3),
                        "sum_launch_ms": sum_ms, "switch_overhead_frac": 1.0 - sum_ms / t,
                        "weight_GB_s": bytes_pass / t / 1e6,
                        "hbm_frac": bytes_pass / t / 1e6 / HBM_PEAK_GBS,
                        "launches": len(plan), "linears": len(tensors)}
        del g
    return {"bytes_per_pass": bytes_pass, "setup_s": setup_s, "quantize_at_load_s": fit_s,
            "quantize_at_load": "logbq_fit_device + logbq_encode per tensor", **out}


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "traffic_k_gemv_layer_8192x28672_m1.md")


def profiled_traffic(kernel):
    """HBM bytes per launch of the M = 1 layer GEMV from the committed rocprofv3 --pmc summary,
    or None when there is none, it covers another kernel instance, or the GEMV's device source
    changed since it was taken."""
    try:
        from paper_2607_01127_amd.prof_summary import source_hash
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        if line.startswith("- ") and ":" in line:
            key, val = line[2:].split(":", 1)
            fields[key.strip()] = val.strip()
    if fields.get("gemv_source_sha256_16") != source_hash():
        return None
    if f"kernel: `{kernel}`" not in text:
        return None
    try:
        return float(fields["traffic_bytes"])
    except (KeyError, ValueError):
        return None


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(L_unused, inputs, target_s=10.0):
    """The oracle on the host cores of this machine, as it stands (plain float64 numpy).

    Main figure: unpack + dequantize + float64 matmul on a 1024-row sample of the 8192x28672
    layer at M = 1, repeated for about `target_s` seconds with the BLAS threads pinned to the
    cores this process may run on. Also: the oracle fit and encode of the 2048x2048 linear, and
    one single-threaded dequantize + matmul of the 2048x2048, 2048x8192 and layer-sample
    tensors."""
    from oracle import logbq_oracle as O
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits, threadpool_info
    except ImportError:
        threadpool_limits = threadpool_info = None
    wl = inputs.WORKLOADS["layer_8192x28672"]
    lin = wl["layers"][0]
    rows = 1024
    w = inputs.student_t_weights(rows, lin.k, wl["nu"], wl["scale"], seed=[wl["cfg"], 99, 0, 0])
    r = O.fit(w)
    codes = O.pack(O.encode(w, r.base, r.shift))
    lut = O.codebook(r.base, r.shift)
    x = inputs.activations(1, lin.k, seed=[wl["cfg"], 0, 0, 1])

    def matvec(c, xx, lt):
        return O.linear(xx, O.dequantize(O.unpack(c), lt))

    ctx = threadpool_limits(limits=affinity) if threadpool_limits else None
    try:
        reps, t0 = 0, time.perf_counter()
        while True:
            matvec(codes, x, lut)
            reps += 1
            el = time.perf_counter() - t0
            if el >= target_s or reps >= 100000:
                break
        threads = 1
        if threadpool_info:
            threads = max([1] + [int(i.get("num_threads", 1)) for i in threadpool_info()])
    finally:
        if ctx is not None:
            ctx.unregister()
    per = el / reps
    packed = rows * lin.k // 2

    # oracle fit / encode / single-threaded matvec on the other workloads
    extra = {}
    small = inputs.WORKLOADS["linear_2048x2048"]
    sl = small["layers"][0]
    ws = inputs.student_t_weights(sl.n, sl.k, small["nu"], small["scale"], seed=[small["cfg"], 0, 0, 0])
    t0 = time.perf_counter()
    rs = O.fit(ws)
    extra["fit_s_2048x2048"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    cs = O.encode(ws, rs.base, rs.shift)
    extra["encode_s_2048x2048"] = time.perf_counter() - t0
    up = inputs.WORKLOADS["up_2048x8192_outliers"]
    ul = up["layers"][0]
    wu = inputs.student_t_weights(ul.n, ul.k, up["nu"], up["scale"], seed=[up["cfg"], 0, 0, 0],
                                  outlier_frac=up.get("outlier_frac", 0.0))
    ru = O.fit(wu)
    cu = O.pack(O.encode(wu, ru.base, ru.shift))
    ctx = threadpool_limits(limits=1) if threadpool_limits else None
    try:
        for name, c, lt, kk in (("2048x2048", O.pack(cs), O.codebook(rs.base, rs.shift), sl.k),
                                ("2048x8192", cu, O.codebook(ru.base, ru.shift), ul.k),
                                ("layer_sample_1024x8192", codes, lut, lin.k)):
            xx = inputs.activations(1, kk, seed=[0, 0, 0, 1])
            t0 = time.perf_counter()
            matvec(c, xx, lt)
            dt = time.perf_counter() - t0
            extra[f"linear_1thread_s_{name}"] = dt
            extra[f"linear_1thread_GB_s_{name}"] = c.size / dt / 1e9
    finally:
        if ctx is not None:
            ctx.unregister()
    return {"value": packed / per / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{rows} of 28672 rows of the 8192x28672 layer at M=1, {reps} reps, "
                      f"{el:.1f} s; unpack + dequantize + float64 matmul (numpy; BLAS threads "
                      f"{threads}, table lookup single-threaded)",
            "s_per_rep": per, "affinity_cores": affinity, "nproc": os.cpu_count(),
            "cpu_model": _cpu_model(), **{k: round(v, 4) for k, v in extra.items()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=10000,
                    help="untimed launches before the timed ones (about 0.2 s of GPU work at M = 1)")
    ap.add_argument("--quick", action="store_true", help="main layer only, no extra rows")
    ap.add_argument("--rows", default="layer,layer8,small,decode1b,decode8b,batched,quality,gptq",
                    help="comma list of extra rows: layer (M sweep + encode), layer8 (the same "
                         "layer at 8 bits), small, decode1b, decode8b, batched (the 8B-shaped "
                         "layer's linears at m = 16 .. 128), quality (LogbQuant against the "
                         "asymmetric linear baseline), gptq (calibration)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--decode-steps", type=int, default=0,
                    help="timed (and warmup) passes of each decode row (default 200 for the "
                         "1B-shaped pass, 100 for the 8B-shaped one)")
    ap.add_argument("--decode-traffic", action="store_true",
                    help="only build the 8B-shaped decode pass at M = 1 and replay it four times "
                         "(for rocprofv3 --pmc FETCH_SIZE per pass) and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 256 MiB device-to-device copy (calibrates the HBM byte "
                         "counters of rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration:
        src = torch.empty(1 << 28, dtype=torch.uint8, device="cuda:0").fill_(3)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel(), "copies": 5}))
        return
    from paper_2607_01127_amd import inputs
    from paper_2607_01127_amd import logbq as L
    L.lib()
    dev = "cuda:0"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    if args.decode_traffic:
        r = bench_decode(torch, L, inputs, dev, stream, "decode_8b_32x7", [1], 1, 1,
                         traffic_only=True)
        print(json.dumps(r))
        return

    want = set() if args.quick else set(args.rows.split(","))
    ms = [1, 8, 32, 128] if "layer" in want else [1]
    res, info, codes, cb = bench_layer(torch, L, inputs, dev, stream, ms, args.steps, args.warmup,
                                       with_encode="layer" in want)
    main_row = res["linear_8192x28672_m1"]
    t_ms = main_row["ms"]
    packed = info["packed"]
    algo = main_row["algo_bytes"]
    value = packed / t_ms / 1e6

    rows = dict(res)
    if "quality" in want:
        rows["quality_vs_uniform"] = bench_quality(torch, L, inputs, dev, stream, codes, cb,
                                                   args.steps, args.warmup)
    if "gptq" in want:
        rows["gptq"] = bench_gptq(torch, L, inputs, dev, stream, not args.no_cpu)
    log("HBM read ceiling (4 GiB)")
    ceiling = read_ceiling(torch, stream)
    torch.cuda.empty_cache()
    if "small" in want:
        for name in ("up_2048x8192_outliers", "linear_2048x2048"):
            log(name)
            rows[name + "_m1"] = bench_small(torch, L, inputs, dev, stream, name, 2000, 5000)
    del codes
    torch.cuda.empty_cache()
    if "layer8" in want:
        rows.update(bench_layer8(torch, L, inputs, dev, stream, [1, 8, 32, 128],
                                 args.steps // 2, args.warmup // 2))
        torch.cuda.empty_cache()
    if "decode1b" in want:
        n1 = args.decode_steps or 200
        rows["decode_1b_16x7"] = bench_decode(torch, L, inputs, dev, stream, "decode_1b_16x7",
                                              [1], n1, n1)
        torch.cuda.empty_cache()
    if "decode8b" in want:
        n8 = args.decode_steps or 100
        rows["decode_8b_32x7"] = bench_decode(torch, L, inputs, dev, stream, "decode_8b_32x7",
                                              [1, 4], n8, n8)
        torch.cuda.empty_cache()
    if "batched" in want:
        bs, bw = aux_counts(args.steps, args.warmup)
        rows["batched_8b_linears"] = bench_batched(torch, L, inputs, dev, stream,
                                                   [16, 32, 64, 128], bs, bw)
        torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu:
        log("cpu baseline (oracle)")
        cpu = cpu_baseline(None, inputs)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": t_ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "layer_8192x28672", "m": 1, "n_out": info["n"], "k_in": info["k"],
                   "weights": "0.015*StudentT(3) float32 -> 4-bit LogbQuant per tensor",
                   "activations": "float16 N(0,1)", "accumulate": "f32",
                   "rotation_copies": info["copies"], "params": info["params"],
                   "host_fit_s": info["fit_s"]},
        "roofline": {"bound": "hbm", "achieved": round(algo / t_ms / 1e6, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(algo / t_ms / 1e6 / HBM_PEAK_GBS, 4),
                     "traffic": profiled_traffic(main_row["kernel"]),
                     "kernel": main_row["kernel"], "algo_bytes_per_launch": algo,
                     "avg_launch_us": t_ms * 1e3,
                     "read_ceiling_GB_s": round(ceiling["GB_s"], 1),
                     "frac_of_read_ceiling": round(algo / t_ms / 1e6 / ceiling["GB_s"], 4)},
        "cpu_baseline": cpu,
        "rows": rows,
    }
    if "decode_8b_32x7" in rows:
        out["decode_tokens_per_s_m1"] = rows["decode_8b_32x7"]["m1"]["tokens_per_s"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
