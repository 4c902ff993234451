"""Pins of the oracle's drift-correction path (KronQ+GPTAQ) and of groups wider than one block.

Each pin checks the oracle against something other than its own formula: brute-force sums,
least-squares solutions on explicit token data, explicit sub-matrix inverses, or invariances the
paper states.
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


# ------------------------------------------------------------------------------ drift statistic
def test_cross_covariance_brute_force():
    r = rng(1)
    A, B = r.standard_normal((29, 4)), r.standard_normal((29, 4))
    D = O.cross_covariance(A, B, chunk=8)
    ref = np.zeros((4, 4))
    for t in range(29):
        for i in range(4):
            for j in range(4):
                ref[i, j] += A[t, i] * B[t, j]
    np.testing.assert_allclose(D, ref, rtol=1e-13)
    np.testing.assert_allclose(O.cross_covariance(A, A, chunk=5), O.covariance(A), rtol=1e-13)


# ------------------------------------------------------------------------------ P (Prop. 1)
@pytest.mark.parametrize("alpha", [1.0, 0.25])
def test_gptaq_rows_absorb_drift_by_least_squares(alpha):
    # row p of P is alpha D[p, p+1:] inv(H~[p+1:, p+1:]) (the remaining columns absorb column
    # p's drift), and P is strictly upper triangular
    d = 12
    H = O.damp(spd(d, 2, cond=1e3))
    U = O.inverse_cholesky_factor(H)
    D = rng(3).standard_normal((d, d))
    P = O.gptaq_correction(D, U, alpha)
    for p in range(d):
        np.testing.assert_array_equal(P[p, :p + 1], 0.0)
        if p + 1 < d:
            ref = alpha * D[p, p + 1:] @ np.linalg.inv(H[p + 1:, p + 1:])
            np.testing.assert_allclose(P[p, p + 1:], ref, rtol=1e-9, atol=1e-12)


def test_gptaq_rows_subset_equals_full():
    d = 40
    U = O.inverse_cholesky_factor(O.damp(spd(d, 4, cond=1e2)))
    D = rng(5).standard_normal((d, d))
    rows = [0, 7, 23, 39]
    np.testing.assert_allclose(O.gptaq_correction(D, U, 0.5, rows),
                               O.gptaq_correction(D, U, 0.5)[rows], rtol=1e-12, atol=1e-15)


def _token_problem(n, d_in, d_out, seed, lam_bar=0.5, drift=0.1):
    """Explicit tokens X, drift dX, and the damped H~ = X^T X + lam_bar I formed by appending
    sqrt(lam_bar) I as extra tokens (with zero drift), so D = dX^T X is unchanged."""
    r = rng(seed)
    X = r.standard_normal((n, d_in)) * np.linspace(0.5, 2.0, d_in)
    dX = drift * (r.standard_normal((n, d_in)) - 0.5 * X)
    Xa = np.vstack([X, np.sqrt(lam_bar) * np.eye(d_in)])
    dXa = np.vstack([dX, np.zeros((d_in, d_in))])
    W = r.standard_normal((d_out, d_in)) * 0.05
    return W, Xa, dXa


@pytest.mark.parametrize("group", [5, 10])
def test_drift_sweep_is_sequential_least_squares(group):
    # At step p the residual of column p against the full-precision target,
    # r = (w_p - w_hat_p) x_p + w_p dx_p, is absorbed by the later columns acting on X:
    # delta = argmin || r - X[:, p+1:] delta ||. The oracle's sweep with P (alpha = 1) must
    # reproduce this step by step (codes identical, weights to rounding).
    d_in, d_out, bits = 10, 7, 3
    W, Xa, dXa = _token_problem(80, d_in, d_out, 4)
    H = Xa.T @ Xa
    U = O.inverse_cholesky_factor(H)
    P = O.gptaq_correction(O.cross_covariance(dXa, Xa), U, 1.0)
    res = O.obs_unblocked(W, U, bits, group, P=P)

    Wt = W.copy()
    codes = np.zeros((d_out, d_in), dtype=np.int64)
    for p in range(d_in):
        if p % group == 0:
            s, z = O.group_params(Wt[:, p:p + group], bits)
        q, wh = O.quantize(Wt[:, p], s, z, bits)
        F = list(range(p + 1, d_in))
        if F:
            R = np.outer(Xa[:, p], Wt[:, p] - wh) + np.outer(dXa[:, p], Wt[:, p])
            delta, *_ = np.linalg.lstsq(Xa[:, F], R, rcond=None)
            Wt[:, F] += delta.T
        Wt[:, p] = wh
        codes[:, p] = q
    np.testing.assert_array_equal(res["codes"], codes)
    np.testing.assert_allclose(res["W"], Wt, rtol=1e-9, atol=1e-12)


def test_zero_drift_is_the_plain_sweep():
    r = rng(5)
    W = r.standard_normal((20, 128)) * 0.02
    U = O.inverse_cholesky_factor(O.damp(spd(128, 6, cond=1e3)))
    P = O.gptaq_correction(np.zeros((128, 128)), U, 1.0)
    a = O.obs_blocked(W, U, 3, 64, 32, P=P)
    b = O.obs_blocked(W, U, 3, 64, 32)
    for k in ("codes", "scales", "zeros", "err", "w_hat", "W"):
        np.testing.assert_array_equal(a[k], b[k])


@pytest.mark.parametrize("block,group", [(128, 128), (32, 128), (64, 256), (128, 256), (64, 64)])
def test_blocked_equals_unblocked_with_drift(block, group):
    # the lazy batch (reading R20: block columns as they stood when quantised) changes nothing
    r = rng(7)
    W = r.standard_normal((30, 256)) * 0.02
    H = O.damp(spd(256, 8, cond=1e3))
    U = O.inverse_cholesky_factor(H)
    P = O.gptaq_correction(0.05 * r.standard_normal((256, 256)) @ H, U, 1.0)
    a = O.obs_unblocked(W, U, 2, group, P=P)
    b = O.obs_blocked(W, U, 2, group, block, P=P)
    np.testing.assert_array_equal(a["codes"], b["codes"])
    np.testing.assert_allclose(b["W"], a["W"], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(b["err"], a["err"], rtol=1e-9, atol=1e-12)


# ------------------------------------------------------------------------------ BiIP with D
def test_biip_keeps_the_full_objective():
    # eq. kronq_full is unchanged by the rescaling and rotations when dX X^T is transformed
    # with H_X (Sec. 4.2, Thm. 1)
    r = rng(9)
    d_out, d_in = 8, 16
    W = r.standard_normal((d_out, d_in))
    W_hat = W + 0.1 * r.standard_normal((d_out, d_in))
    HX, HG = spd(d_in, 10), spd(d_out, 11)
    D = r.standard_normal((d_in, d_in))
    rot_in = (np.where(r.random(d_in) < 0.5, -1, 1), None)
    rot_out = (np.where(r.random(d_out) < 0.5, -1, 1), None)
    b = O.biip_forward(W, HX, HG, rot_in, rot_out, O.BIIP, D=D)
    What2 = b["U"] @ (b["sg"][:, None] * W_hat * b["sx"][None, :]) @ b["V"].T
    before = O.kronq_objective(W, W_hat, HX, HG, D)
    after = O.kronq_objective(b["W"], What2, b["HX"], b["HG"], b["D"])
    np.testing.assert_allclose(after, before, rtol=1e-10)
    # and the drift term alone is non-trivial here
    assert abs(O.kronq_objective(W, W_hat, HX, HG, D) - O.kronq_objective(W, W_hat, HX, HG)) > 1e-3


# ------------------------------------------------------------------------------ wide groups
def test_per_channel_grid_uses_the_initial_row():
    # group = d_in: one (scale, zero) per row, taken from the row before any compensation
    r = rng(12)
    W = r.standard_normal((25, 256)) * 0.02
    U = O.inverse_cholesky_factor(O.damp(spd(256, 13, cond=1e3)))
    res = O.obs_blocked(W, U, 3, 256, 128)
    s, z = O.group_params(W, 3)
    assert res["scales"].shape == (25, 1)
    np.testing.assert_array_equal(res["scales"][:, 0], s)
    np.testing.assert_array_equal(res["zeros"][:, 0], z)


def test_per_channel_rtn_when_hessian_is_diagonal():
    # diagonal H~: no propagation, so every code is the nearest point of the row's grid
    r = rng(14)
    W = r.standard_normal((30, 256)).astype(np.float32).astype(np.float64)
    U = O.inverse_cholesky_factor(O.damp(np.eye(256)))
    res = O.obs_blocked(W, U, 4, 256, 128)
    s, z = O.group_params(W, 4)
    grid = s[:, None] * (np.arange(16)[None, :] - z[:, None])
    for c in range(256):
        dist = np.abs(W[:, c, None] - grid)
        srt = np.sort(dist, axis=1)
        tie = srt[:, 1] - srt[:, 0] < 1e-15
        assert np.all((res["codes"][:, c] == np.argmin(dist, axis=1)) | tie)



# ------------------------------------------------------------------------------ eq. gptaq_obj
@pytest.mark.parametrize("kron_g", [False, True])
def test_full_objective_equals_output_error_on_explicit_tokens(kron_g):
    # eq. gptaq_obj: the drift-aware layer error ||W X~ - W_hat X||_F^2 on explicit tokens,
    # X~ = X + dX, expands to the objective's two terms plus the constant ||W dX||_F^2, which
    # does not depend on W_hat. With H_G = C^T C the output errors are weighted by C (each
    # output channel mixed by the rows of C, the K-FAC weighting of eq. kron_obj). A flipped
    # sign or a dropped factor 2 on the drift term breaks the equality.
    r = rng(15)
    n, d_out, d_in = 37, 6, 9
    X = r.standard_normal((n, d_in))          # token-major: row t is token t's input
    dX = 0.3 * r.standard_normal((n, d_in))
    W = r.standard_normal((d_out, d_in))
    W_hat = W + 0.2 * r.standard_normal((d_out, d_in))
    C = r.standard_normal((11, d_out)) if kron_g else np.eye(d_out)
    HX = X.T @ X
    HG = C.T @ C
    D = dX.T @ X                              # the drift statistic, token-major (reading R19)
    Xt = X + dX
    direct = 0.0
    const = 0.0
    for t in range(n):                        # token by token: y~_t - y_hat_t and W dx_t
        e = C @ (W @ Xt[t] - W_hat @ X[t])
        c = C @ (W @ dX[t])
        direct += float(e @ e)
        const += float(c @ c)
    got = O.kronq_objective(W, W_hat, HX, HG, D)
    np.testing.assert_allclose(got + const, direct, rtol=1e-11)
    # without the drift statistic it is the plain K-FAC loss, the error without drift
    plain = sum(float(np.sum((C @ ((W - W_hat) @ X[t])) ** 2)) for t in range(n))
    np.testing.assert_allclose(O.kronq_objective(W, W_hat, HX, HG), plain, rtol=1e-11)
