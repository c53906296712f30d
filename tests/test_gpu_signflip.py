"""Sign symmetry of the product at the level of single instructions (Eq. 2: the codebook is
symmetric, so flipping every sign bit negates every dequantized weight exactly).

With K = 32 and activations that are zero except at chosen positions, each output of the GEMV
is one v_dot2_f32_f16 (two products and a zero accumulator), two chained ones, or the full
chain of one 32-weight chunk; each output of the stepped MFMA kernel at m = 32 is one
v_mfma_f32_16x16x32_f16 over 2, 8 or 32 nonzero products (the later MFMAs of the step add
zero products). The tests count the outputs whose negated-code result is not exactly the
negation."""
import numpy as np
import pytest

from oracle import logbq_oracle as O
from paper_2607_01127_amd import inputs
from paper_2607_01127_amd import logbq as L

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


def _codes_and_book(n):
    w = inputs.student_t_weights(256, 256, 4, 0.02, seed=[12, 0, 0, 0])
    r = O.fit(w)
    book = O.codebook(r.base, r.shift)
    rng = np.random.default_rng(12)
    codes = rng.integers(0, 256, size=(n, 16), dtype=np.uint8)
    return torch.from_numpy(codes).to(DEV), book


@pytest.mark.parametrize("m", [1, 32])
@pytest.mark.parametrize("live", [[0, 1], [0, 1, 4, 5], list(range(8)), list(range(32))])
def test_sign_flip_single_instruction(m, live):
    n = 1 << 16
    codes, book = _codes_and_book(n)
    flipped = codes ^ 0x88
    rng = np.random.default_rng([13, m, len(live)])
    x = np.zeros((m, 32), dtype=np.float16)
    x[:, live] = rng.standard_normal((m, len(live))).astype(np.float16)
    xd = torch.from_numpy(x).to(DEV)
    y = L.linear(xd, codes, book)
    yf = L.linear(xd, flipped, book)
    torch.cuda.synchronize()
    y, yf = y.cpu().numpy(), yf.cpu().numpy()
    bad = int(np.count_nonzero(yf != -y))
    kern = L.linear_kernel(4, m, 32, n, book)
    _say(f"sign flip {kern} m={m} nonzero k={live}: {bad} of {y.size} outputs not exactly negated")
    wh = O.dequantize(O.unpack(codes.cpu().numpy()), book).astype(np.float64)
    absdot = np.abs(x.astype(np.float64)) @ np.abs(wh).T
    assert np.all(np.abs(yf.astype(np.float64) + y) <= absdot * 2.0 ** -20)
