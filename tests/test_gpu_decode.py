"""One decoder layer of each decode workload in the launch configuration bench.py times (grouped
q/k/v and gate/up launches, single o and down launches) at the batch sizes it times, against
the oracle on sampled output rows: the 2048-wide (16-layer) and 4096-wide (32-layer) shapes,
whose linears take the GEMV (single and grouped), the split-row GEMV (down, K = 8192 or
14336), and at M = 4 the split-K MFMA kernel (gate/up of the 4096-wide layer)."""
import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3
DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name", ["decode_1b_16x7", "decode_8b_32x7"])
def test_decode_layer_grouped_launches_sampled(name):
    wl = inputs.WORKLOADS[name]
    lins = {lin.name: lin for lin in wl["layers"]}
    rng = np.random.default_rng(50)
    tensors = {}
    for lin in wl["layers"]:
        _say(f"{name}: {lin.name} {lin.k}->{lin.n}: generate, fit, encode")
        wd = inputs.student_t_weights(lin.n, lin.k, wl["nu"], wl["scale"],
                                      seed=[wl["cfg"], 0, inputs.PROJ[lin.name], 0], device=DEV)
        p = L.fit(wd.cpu().numpy())
        codes, cb = L.encode(wd, p)
        rows = np.sort(rng.choice(lin.n, size=min(48, lin.n), replace=False))
        w_rows = wd[torch.from_numpy(rows).to(DEV)].cpu().numpy()
        c_rows = O.encode(w_rows, p.base, p.shift)
        torch.cuda.synchronize()
        assert np.array_equal(codes[torch.from_numpy(rows).to(DEV)].cpu().numpy(), O.pack(c_rows))
        tensors[lin.name] = (codes, cb, rows, O.dequantize(c_rows, O.codebook(p.base, p.shift)))
        del wd
    for m in (1, 4):
        xs = {k: inputs.activations(m, k, seed=[wl["cfg"], 0, 99, k + m]) for k in {l.k for l in lins.values()}}
        for group in (["q", "k", "v"], ["o"], ["gate", "up"], ["down"]):
            k = lins[group[0]].k
            x = xs[k]
            xd = torch.from_numpy(x).to(DEV)
            _say(f"{name} m={m} {'+'.join(group)}: path {L.linear_path(4, m, k, lins[group[0]].n)}")
            if len(group) == 1:
                ys = [L.linear(xd, tensors[group[0]][0], tensors[group[0]][1])]
            else:
                ys = L.linear_multi(xd, [tensors[g][0] for g in group], [tensors[g][1] for g in group])
            torch.cuda.synchronize()
            for g, y in zip(group, ys):
                _, _, rows, wh = tensors[g]
                ys_ = y[:, torch.from_numpy(rows).to(DEV)].cpu().numpy().astype(np.float64)
                y_ref = O.linear(x, wh)
                den = (np.linalg.norm(x.astype(np.float64), axis=1)[:, None] *
                       np.linalg.norm(wh.astype(np.float64), axis=1)[None, :])
                den[den == 0] = 1.0
                err = float(np.max(np.abs(ys_ - y_ref) / den))
                assert err <= TOL, (name, m, g, err)
