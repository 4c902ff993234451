"""Pins of the oracle's inference-side functions: the online reversion of BiIP around the
quantised matvec, the dequantisation, and the packed code format (CPU only)."""
import numpy as np
import pytest

import oracle as O


def rng(seed):
    return np.random.default_rng(seed)


def spd(n, seed, cond=50.0):
    r = rng(seed)
    q, _ = np.linalg.qr(r.standard_normal((n, n)))
    return (q * np.geomspace(1.0, cond, n)) @ q.T


# ------------------------------------------------------------------------------ online inference
@pytest.mark.parametrize("d_out,d_in", [(16, 32), (56, 64)])
def test_online_matvec_undoes_biip(d_out, d_in):
    # with W_rot the forward BiIP of W, the online product is the original layer's W x
    r = rng(20)
    W = r.standard_normal((d_out, d_in))
    HX, HG = spd(d_in, 21), spd(d_out, 22)
    rot_in = (np.where(r.random(d_in) < 0.5, -1, 1), None)
    q = np.linalg.qr(r.standard_normal((28, 28)))[0] if d_out % 28 == 0 else None
    rot_out = (np.where(r.random(d_out) < 0.5, -1, 1), q)
    b = O.biip_forward(W, HX, HG, rot_in, rot_out)
    x = r.standard_normal((d_in, 3))
    np.testing.assert_allclose(O.online_matvec(b["W"], b["sx"], b["sg"], b["V"], b["U"], x),
                               W @ x, rtol=1e-10, atol=1e-12)


def test_dequantize_matches_the_sweep():
    # the sweep's w_hat is scale * (code - zero) with the group's parameters
    r = rng(23)
    W = r.standard_normal((12, 256)) * 0.02
    U = O.inverse_cholesky_factor(O.damp(spd(256, 24, cond=1e2)))
    for group in (128, 256):
        res = O.obs_blocked(W, U, 3, group, 128)
        np.testing.assert_array_equal(
            O.dequantize(res["codes"], res["scales"], res["zeros"], group), res["w_hat"])


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_pack_codes_bit_layout(bits):
    # brute force: read every code back from the packed words as a bit string
    r = rng(bits)
    codes = r.integers(0, 2 ** bits, size=(3, 96))
    packed = O.pack_codes(codes, bits)
    assert packed.shape == (3, 96 * bits // 32)
    for i in range(3):
        stream = "".join(format(int(w), "032b")[::-1] for w in packed[i])  # LSB first
        for j in range(96):
            assert int(stream[j * bits:(j + 1) * bits][::-1], 2) == codes[i, j]
