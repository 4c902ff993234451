"""Pins of the oracle's diagnostics: the incoherence measures (Sec. 2.3), the norm variation of
Fig. 2b, the pivots and expected-loss factors of Prop. 2 and the optimality table.

Each pin checks the oracle against closed forms or brute force; the last group checks the
paper's qualitative claims about BiIP on synthetic layers.
"""
import numpy as np
import pytest

import oracle as O


def rng(seed):
    return np.random.default_rng(seed)


def spd(n, seed, cond=50.0):
    r = rng(seed)
    q, _ = np.linalg.qr(r.standard_normal((n, n)))
    return (q * np.geomspace(1.0, cond, n)) @ q.T


# ------------------------------------------------------------------------------ mu(W)
def test_incoherence_closed_forms():
    # a Hadamard matrix (any rows of it) is maximally incoherent, a one-hot matrix maximally
    # coherent; mu does not depend on the scale
    assert O.incoherence(O.hadamard(16)) == pytest.approx(1.0, rel=1e-15)
    assert O.incoherence(O.hadamard(16)[:4] * 3.5) == pytest.approx(1.0, rel=1e-15)
    M = np.zeros((6, 10))
    M[2, 7] = -4.0
    assert O.incoherence(M) == pytest.approx(np.sqrt(60.0), rel=1e-15)
    # two equal entries: sqrt(rc) * m / (sqrt(2) m)
    M[0, 0] = 4.0
    assert O.incoherence(M) == pytest.approx(np.sqrt(30.0), rel=1e-15)


def test_norm_cv_hand_cases():
    assert O.norm_cv(np.ones((5, 7))) == (0.0, 0.0)
    # column norms 1 and 3 (mean 2, std 1), and the same row norms
    M = np.array([[1.0, 0.0], [0.0, 3.0]])
    cv_in, cv_out = O.norm_cv(M)
    assert cv_in == pytest.approx(0.5, rel=1e-15) and cv_out == pytest.approx(0.5, rel=1e-15)
    M = np.array([[3.0, 4.0], [0.0, 0.0], [0.0, 5.0]])  # rows 5, 0, 5; columns 3, sqrt(41)
    cv_in, cv_out = O.norm_cv(M)
    n = np.array([3.0, np.sqrt(41.0)])
    assert cv_in == pytest.approx(np.std(n) / np.mean(n), rel=1e-14)
    # rows: mean 10/3, std sqrt(((5/3)^2 + (10/3)^2 + (5/3)^2) / 3) = 5 sqrt(2) / 3
    assert cv_out == pytest.approx(np.sqrt(2.0) / 2.0, rel=1e-14)


# ------------------------------------------------------------------------------ mu(H)
def test_hessian_incoherence_closed_forms():
    d = 16
    lam = np.geomspace(1.0, 100.0, d)
    # diagonal H: the eigenvectors are the axes
    assert O.hessian_incoherence(np.diag(lam)) == pytest.approx(np.sqrt(d), rel=1e-12)
    # H = Had diag(lam) Had^T / d: the eigenvectors are the normalised Hadamard columns
    Hn = O.hadamard(d) / np.sqrt(d)
    assert O.hessian_incoherence(Hn @ np.diag(lam) @ Hn.T) == pytest.approx(1.0, rel=1e-12)
    # 2 x 2 [[a, b], [b, a]]: eigenvectors (1, +-1) / sqrt(2)
    assert O.hessian_incoherence(np.array([[2.0, 0.5], [0.5, 2.0]])) == pytest.approx(1.0)


def test_hessian_incoherence_of_rotated_matrix():
    # the eigenvectors of Q H Q^T are Q times those of H: with distinct eigenvalues, mu is
    # sqrt(d) max |Q V| for any orthogonal Q; a permutation leaves it unchanged
    d = 24
    H = spd(d, 3, cond=1e3)
    _, V = O.eigenvectors(H)
    Q, _ = np.linalg.qr(rng(4).standard_normal((d, d)))
    assert O.hessian_incoherence(Q @ H @ Q.T) == pytest.approx(
        np.sqrt(d) * np.max(np.abs(Q @ V)), rel=1e-9)
    P = np.eye(d)[rng(5).permutation(d)]
    assert O.hessian_incoherence(P @ H @ P.T) == pytest.approx(O.hessian_incoherence(H), rel=1e-9)
    w, V = O.eigenvectors(H)
    np.testing.assert_allclose(H @ V, V * w, atol=1e-9 * w.max())


# ------------------------------------------------------------------------------ pivots
def test_sweep_pivots_brute_force():
    d = 10
    H = spd(d, 6, cond=1e3)
    D = O.sweep_pivots(H)
    for p in range(d):
        assert D[p] == pytest.approx(1.0 / np.linalg.inv(H[p:, p:])[0, 0], rel=1e-10)
    # product of the pivots is det(H); the last pivot is the last diagonal entry
    assert np.prod(D) == pytest.approx(np.linalg.det(H), rel=1e-9)
    assert D[-1] == pytest.approx(H[-1, -1], rel=1e-12)
    # a Schur complement never exceeds its diagonal entry: tr(D) <= tr(H), equal if diagonal
    assert np.all(D <= np.diag(H) * (1 + 1e-12))
    np.testing.assert_allclose(O.sweep_pivots(np.diag(np.arange(1.0, 6.0))),
                               np.arange(1.0, 6.0), rtol=1e-14)


# ------------------------------------------------------------------------------ Prop. 2
def test_rescale_objective_minimum_at_quarter():
    # Cauchy-Schwarz: (sum h/s^2)(sum s^2 a) >= (sum sqrt(h a))^2 with equality at
    # s = (h/a)^(1/4); alpha = 0 is the unscaled product (sum h)(sum a)
    r = rng(7)
    h = np.exp(2.0 * r.standard_normal(50))
    a = np.exp(0.5 * r.standard_normal(50))
    assert O.rescale_objective(h, a, 0.0) == pytest.approx(h.sum() * a.sum(), rel=1e-14)
    assert O.rescale_objective(h, a, 0.25) == pytest.approx(np.sum(np.sqrt(h * a)) ** 2,
                                                            rel=1e-13)
    grid = np.linspace(0.0, 0.5, 201)
    vals = [O.rescale_objective(h, a, al) for al in grid]
    assert grid[int(np.argmin(vals))] == pytest.approx(0.25)


def test_rescale_gain_cases():
    r = rng(8)
    h, a = np.exp(r.standard_normal(40)), np.exp(r.standard_normal(40))
    assert O.rescale_gain(h, a) <= 1.0
    assert O.rescale_gain(3.0 * a, a) == pytest.approx(1.0, rel=1e-14)  # h proportional to a
    # curvature on k of d channels with equal row energy: rho = k / d (appendix A.3)
    d, k = 64, 5
    h = np.zeros(d)
    h[:k] = 7.0
    assert O.rescale_gain(h, np.full(d, 2.0)) == pytest.approx(k / d, rel=1e-14)


def test_proxy_loss_factors_relations():
    r = rng(9)
    d_out, d_in = 12, 16
    W = r.standard_normal((d_out, d_in)) * np.exp(r.standard_normal(d_out))[:, None]
    HG = spd(d_out, 10, cond=1e4)
    Hd = O.damp(spd(d_in, 11, cond=1e3))
    f = O.proxy_loss_factors(HG, W, Hd)
    h, a = np.diag(HG), np.sum(W * W, axis=1)
    assert f["kronq"] == pytest.approx(f["rho"] * f["gptq"], rel=1e-13)
    assert f["gptq"] <= f["nearest"]
    assert f["kronq"] == pytest.approx(O.rescale_objective(h, a, 0.25) * f["trD"], rel=1e-13)
    assert f["gptq"] == pytest.approx(O.rescale_objective(h, a, 0.0) * f["trD"], rel=1e-13)
    # with a diagonal H~ GPTQ's factor equals nearest rounding's
    g = O.proxy_loss_factors(HG, W, np.diag(np.arange(1.0, d_in + 1)))
    assert g["gptq"] == pytest.approx(g["nearest"], rel=1e-13)


# ------------------------------------------------------------------------------ BiIP's effect
def _layer(d_out, d_in, n, seed):
    """A synthetic layer with structured scales: heavy per-channel gradient scales (as the bench
    workloads), weights with lognormal row and column scales."""
    r = rng(seed)
    X = r.standard_normal((n, d_in))
    X[:, :4] *= np.array([10.0, 20.0, 30.0, 40.0])  # separated outlier channels
    G = r.standard_normal((n, d_out)) * np.exp(1.5 * r.standard_normal(d_out))
    W = (0.02 * r.standard_normal((d_out, d_in)) * np.exp(0.7 * r.standard_normal(d_out))[:, None]
         * np.exp(0.7 * r.standard_normal(d_in))[None, :])
    sign = lambda d: np.where(r.random(d) < 0.5, -1, 1)
    return W, X.T @ X, G.T @ G, (sign(d_in), None), (sign(d_out), None)


def test_biip_makes_hessians_incoherent():
    # Sec. 4.2 / Fig. 2a: H_G is coherent (mu / sqrt(d) near 1) before BiIP and incoherent after;
    # after a random Hadamard rotation mu is of the order of a random orthogonal basis's,
    # sqrt(2 ln(d^2)) (1.5 times that is the bound here), and the same holds for H_X
    d = 256
    W, HX, HG, ri, ro = _layer(d, d, 2048, 12)
    b = O.biip_forward(W, HX, HG, ri, ro)
    bound = 1.5 * np.sqrt(2.0 * np.log(d * d)) / np.sqrt(d)
    assert O.hessian_incoherence(HG) / np.sqrt(d) > 0.9
    assert O.hessian_incoherence(b["HG"]) / np.sqrt(d) < bound
    assert O.hessian_incoherence(HX) / np.sqrt(d) > 0.9
    assert O.hessian_incoherence(b["HX"]) / np.sqrt(d) < bound
    assert O.incoherence(b["W"]) < O.incoherence(W)


def test_biip_equalises_row_and_column_norms():
    # Fig. 2b: input-side processing leaves the row norms' variation (CV_out) where the rescale
    # puts it (the rotation V keeps every row norm), the bidirectional one reduces both CVs
    W, HX, HG, ri, ro = _layer(128, 256, 1024, 13)
    cv_in0, cv_out0 = O.norm_cv(W)
    inp = O.biip_forward(W, HX, HG, ri, ro, O.RESCALE_IN | O.ROT_IN)
    both = O.biip_forward(W, HX, HG, ri, ro)
    sx, _ = O.rescale_factors(W, HX, HG, O.RESCALE_IN)
    assert O.norm_cv(inp["W"])[1] == pytest.approx(O.norm_cv(W * sx[None, :])[1], rel=1e-10)
    cv_in2, cv_out2 = O.norm_cv(both["W"])
    assert cv_in2 < 0.5 * cv_in0 and cv_out2 < 0.5 * cv_out0


def test_output_rescale_gain_on_synthetic_layer():
    # Prop. 2: with diag(H_G) spanning orders of magnitude rho is far below 1
    W, HX, HG, ri, ro = _layer(256, 128, 1024, 14)
    assert O.rescale_gain(np.diag(HG), np.sum(W * W, axis=1)) < 0.5
