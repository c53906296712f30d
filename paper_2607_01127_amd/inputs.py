"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers; it holds none of LogbQuant's arithmetic. The tests
feed the same arrays to the CPU oracle and to the HIP library.

The paper measures pretrained Llama-3.2-1B / Llama-3.1-8B weights (Sec. 4.1, Table 3), which
are not available here. In their place:

* weights: float32 ``scale * StudentT(nu)``, heavy tailed and densely centred on zero
  (Sec. 2 and Sec. 3 describe weight distributions that way), optionally with a fraction of
  outliers replaced by +-20 sigma (sigma = scale * sqrt(nu / (nu - 2)), the std of the
  scaled t distribution), random sign;
* activations: float16 N(0, 1) rows, M = batch rows per decode step.

Seeds are ``[config, layer, projection, stream]`` lists (stream 0 = weights,
1 = activations), so that every tensor of a multi-layer workload is independent and
reproducible. On the CPU the draw is numpy's ``Generator.standard_t``; on a GPU device it
is ``Z / sqrt(chi2_nu / nu)`` from torch's seeded device generator, with chi2_nu the sum of
nu squared standard normals (integer nu). Both are Student's t with nu degrees of freedom.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

PROJ = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6}


def _seed64(seed) -> int:
    ss = np.random.SeedSequence(list(seed) if isinstance(seed, (list, tuple)) else seed)
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def student_t_weights(n: int, k: int, nu: float, scale: float, seed, device=None,
                      outlier_frac: float = 0.0, outlier_sigmas: float = 20.0):
    """float32 [n][k] weights = scale * StudentT(nu), plus optional +-20 sigma outliers.

    device None -> numpy array; otherwise a torch tensor drawn on that device.
    The outlier count is round(outlier_frac * n * k); positions are distinct.
    """
    numel = n * k
    n_out = int(round(outlier_frac * numel))
    sigma = scale * math.sqrt(nu / (nu - 2.0)) if nu > 2 else scale
    if device is None:
        rng = np.random.default_rng(np.random.SeedSequence(list(seed)))
        w = (rng.standard_t(nu, size=(n, k)) * scale).astype(np.float32)
        if n_out:
            pos = rng.choice(numel, size=n_out, replace=False)
            sgn = rng.choice(np.array([-1.0, 1.0]), size=n_out)
            w.reshape(-1)[pos] = (sgn * outlier_sigmas * sigma).astype(np.float32)
        return w
    import torch
    if int(nu) != nu:
        raise ValueError("device draw needs an integer nu")
    g = torch.Generator(device=device)
    g.manual_seed(_seed64(seed))
    w = torch.empty((n, k), dtype=torch.float32, device=device)
    chi = torch.zeros((n, k), dtype=torch.float32, device=device)
    tmp = torch.empty((n, k), dtype=torch.float32, device=device)
    for _ in range(int(nu)):
        tmp.normal_(generator=g)
        chi.addcmul_(tmp, tmp)
    w.normal_(generator=g)
    w.mul_(torch.rsqrt(chi.div_(float(nu)))).mul_(scale)
    del chi, tmp
    if n_out:
        pos = torch.randperm(numel, generator=g, device=device)[:n_out]
        sgn = torch.randint(0, 2, (n_out,), generator=g, device=device).float() * 2 - 1
        w.view(-1)[pos] = sgn * float(outlier_sigmas * sigma)
    return w


def activations(m: int, k: int, seed, device=None):
    """float16 [m][k] activations drawn from N(0, 1)."""
    if device is None:
        rng = np.random.default_rng(np.random.SeedSequence(list(seed)))
        return rng.standard_normal((m, k)).astype(np.float16)
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_seed64(seed))
    return torch.randn((m, k), generator=g, device=device, dtype=torch.float32).half()


@dataclass(frozen=True)
class Linear:
    name: str
    k: int      # in features
    n: int      # out features


def decoder_linears(hidden: int, inter: int, kv: int):
    """The seven linears of one Llama-style decoder layer, in dependency order."""
    return [Linear("q", hidden, hidden), Linear("k", hidden, kv), Linear("v", hidden, kv),
            Linear("o", hidden, hidden), Linear("gate", hidden, inter),
            Linear("up", hidden, inter), Linear("down", inter, hidden)]


# The five synthetic workloads (weights: scale * t_nu; activations fp16 N(0,1)); cfg is the
# first seed element, numbered 1..5 in this order.
WORKLOADS = {
    "linear_2048x2048": dict(cfg=1, layers=[Linear("w", 2048, 2048)], nu=4, scale=0.02,
                             outlier_frac=0.0, batch=(1,)),
    "up_2048x8192_outliers": dict(cfg=2, layers=[Linear("up", 2048, 8192)], nu=4, scale=0.02,
                                  outlier_frac=1e-4, batch=(1,)),
    "decode_1b_16x7": dict(cfg=3, layers=decoder_linears(2048, 8192, 512) * 1, n_layers=16,
                           nu=4, scale=0.02, outlier_frac=0.0, batch=(1,)),
    "decode_8b_32x7": dict(cfg=4, layers=decoder_linears(4096, 14336, 1024), n_layers=32,
                           nu=4, scale=0.02, outlier_frac=0.0, batch=(1, 4)),
    "layer_8192x28672": dict(cfg=5, layers=[Linear("w", 8192, 28672)], nu=3, scale=0.015,
                             outlier_frac=0.0, batch=(1, 8, 32, 128)),
}
