"""Sign symmetry of the product at the level of single instructions (Eq. 2: the codebook is
symmetric, so flipping every sign bit negates every dequantized weight exactly).

With K = 32 and activations that are zero except at chosen positions, each output of the GEMV
(m = 1) is one v_dot2_f32_f16 with a zero accumulator (k = 0, 1), a second one accumulating
onto the first (k = 0, 1, 4, 5), or the chains of one 32-weight chunk; each output of the
stepped MFMA kernel (m = 32) is one v_mfma_f32_16x16x32_f16 with a zero accumulator over 2, 4
or 8 nonzero products (k < 8), or four MFMAs accumulating onto each other (k < 32). The other
instructions of the chain add products of zero activations, which leave the accumulator
unchanged. Measured on MI355X: with a zero accumulator both instructions negate exactly; once
they add onto a nonzero accumulator, a few per cent of the results differ from the negation in
the last bit of a partial sum (at most a few units of 2^-24 sum_k |x_k w_k|). So the float32
accumulation of these instructions is not sign-symmetric, and the general sign-flip test of the
linear kernels keeps a tolerance instead of bit equality."""
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
    wh = O.dequantize(O.unpack(codes.cpu().numpy()), book).astype(np.float64)
    absdot = np.abs(x.astype(np.float64)) @ np.abs(wh).T
    absdot[absdot == 0] = 1.0
    # differences in units of 2^-24 * sum_k |x_k w_k|: one last-bit difference in a partial sum
    # of that size is at most 2 units
    units = np.abs(yf.astype(np.float64) + y) / (absdot * 2.0 ** -24)
    kern = L.linear_kernel(4, m, 32, n, book)
    _say(f"sign flip {kern} m={m} nonzero k={live}: {bad} of {y.size} outputs not exactly negated, "
         f"largest difference {float(np.max(units)):.2f} x 2^-24 sum|x w|")
    one_instruction = max(live) < 2 if m == 1 else max(live) < 8
    if one_instruction:
        assert bad == 0        # zero accumulator: the result negates exactly
    else:
        assert bad > 0         # accumulating onto a nonzero value: not sign-symmetric
    assert float(np.max(units)) <= 8.0
