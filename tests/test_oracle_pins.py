"""Pins of the float64 oracle against what the paper and the mathematics fix (CPU only).

Each pin is independent of the oracle's own code path: brute force on tiny inputs, closed forms,
library routines, identities the paper states, or hand-derived values.
"""
import json
import os

import numpy as np
import pytest
import scipy.linalg

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed):
    return np.random.default_rng(seed)


def spd(n, seed, cond=50.0):
    r = rng(seed)
    q, _ = np.linalg.qr(r.standard_normal((n, n)))
    ev = np.geomspace(1.0, cond, n)
    return (q * ev) @ q.T


# ------------------------------------------------------------------------------------ O1
def test_widen_bf16_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x7F80, 0x0000, 0x8000, 0x4049],
                    dtype=np.uint16)
    v = O.widen_bf16(bits)
    assert v[0] == 1.0 and v[1] == -2.0
    assert v[2] == 1.0 + 2.0 ** -7
    assert v[3] == 2.0 ** -133  # smallest subnormal bf16
    assert np.isinf(v[4]) and v[5] == 0.0 and np.signbit(v[6])
    assert v[7] == 3.140625


def test_covariance_brute_force():
    r = rng(1)
    A = r.standard_normal((37, 5))
    H = O.covariance(A, chunk=8)  # several chunks and a ragged last one
    B = np.zeros((5, 5))
    for t in range(37):
        for i in range(5):
            for j in range(5):
                B[i, j] += A[t, i] * A[t, j]
    np.testing.assert_allclose(H, B, rtol=1e-13, atol=1e-13)
    assert np.array_equal(H, H.T)
    assert np.linalg.eigvalsh(H).min() > -1e-12


def test_covariance_bf16_exact():
    # bf16 inputs: every product is exact in float64, so chunking cannot change the result
    X = synth.gen_matrix(synth.small_spec(8, 16, 300).x)
    bits = synth.bf16_bits(X)
    h1 = O.covariance(bits, chunk=7)
    h2 = O.covariance(bits, chunk=300)
    xf = X.double().numpy()
    np.testing.assert_array_equal(h1, h2)
    np.testing.assert_array_equal(h1, xf.T @ xf)


def test_covariance_diag_is_brute_force_diagonal():
    # per-channel sums of squares by a plain loop, on bf16 bits (exact) and on floats
    X = synth.gen_matrix(synth.small_spec(8, 16, 300).x)
    bits = synth.bf16_bits(X)
    xf = X.double().numpy()
    ref = np.array([sum(xf[t, j] ** 2 for t in range(300)) for j in range(16)])
    np.testing.assert_array_equal(O.covariance_diag(bits, chunk=7), ref)
    A = rng(2).standard_normal((41, 6))
    ref = np.array([sum(A[t, j] * A[t, j] for t in range(41)) for j in range(6)])
    np.testing.assert_allclose(O.covariance_diag(A, chunk=5), ref, rtol=1e-14)


# ------------------------------------------------------------------------------------ O2/O3
def test_traces_closed_form():
    hx, hg = np.diag([1.0, 2.0, 3.0]), np.diag([4.0, 5.0])
    assert O.traces(hx, hg) == (6.0, 9.0, 54.0)


def _problem(d_out=12, d_in=8, seed=3):
    r = rng(seed)
    W = r.standard_normal((d_out, d_in)) * np.exp(r.standard_normal(d_in))[None, :]
    return W, spd(d_in, seed + 1), spd(d_out, seed + 2, cond=1e3)


def test_rescale_input_side_closed_form():
    # with only S_X, the squared column norms of W' equal diag(H_X') = sqrt(h_j a_j)
    W, HX, HG = _problem()
    out = O.biip_forward(W, HX, HG, flags=O.RESCALE_IN)
    a, h = np.sum(W * W, 0), np.diag(HX)
    np.testing.assert_allclose(np.sum(out["W"] ** 2, 0), np.diag(out["HX"]), rtol=1e-12)
    np.testing.assert_allclose(np.diag(out["HX"]), np.sqrt(h * a), rtol=1e-12)
    np.testing.assert_allclose(np.trace(out["HX"]), np.sum(np.sqrt(h * a)), rtol=1e-12)
    assert np.all(out["sg"] == 1.0)


def test_rescale_output_side_closed_form():
    W, HX, HG = _problem()
    out = O.biip_forward(W, HX, HG, flags=O.RESCALE_OUT)
    b, h = np.sum(W * W, 1), np.diag(HG)
    np.testing.assert_allclose(np.sum(out["W"] ** 2, 1), np.diag(out["HG"]), rtol=1e-12)
    np.testing.assert_allclose(np.diag(out["HG"]), np.sqrt(h * b), rtol=1e-12)
    assert np.all(out["sx"] == 1.0)


def test_rescale_from_diagonals_only():
    # only diag(H_X), diag(H_G) enter eq. rescale: the 1-D form gives identical factors
    W, HX, HG = _problem()
    sx, sg = O.rescale_factors(W, HX, HG)
    sx1, sg1 = O.rescale_factors(W, np.diag(HX).copy(), np.diag(HG).copy())
    assert np.array_equal(sx, sx1) and np.array_equal(sg, sg1)


def test_rescale_zero_norm_gives_one():
    W, HX, HG = _problem()
    W[:, 2] = 0.0
    W[5, :] = 0.0
    HX = HX.copy()
    sx, sg = O.rescale_factors(W, HX, HG)
    assert sx[2] == 1.0 and sg[5] == 1.0 and np.all(sx > 0) and np.all(sg > 0)


def _dw(shape, seed):
    return rng(seed).standard_normal(shape) * 1e-2


def test_loss_invariant_under_rescale():
    # eq. rescale leaves the K-FAC objective unchanged when W, H_X, H_G move together
    W, HX, HG = _problem()
    out = O.biip_forward(W, HX, HG, flags=O.RESCALE_IN | O.RESCALE_OUT)
    dW = _dw(W.shape, 9)
    dW2 = out["sg"][:, None] * dW * out["sx"][None, :]
    np.testing.assert_allclose(O.kfac_loss(dW2, out["HX"], out["HG"]),
                               O.kfac_loss(dW, HX, HG), rtol=1e-11)


# ------------------------------------------------------------------------------------ O4
@pytest.mark.parametrize("d", [64, 28 * 8])
def test_rht_rows_entrywise(d):
    """Rows formed entry by entry: equal to the dense builder's rows, and, for the 28-factor
    form, to rows of the explicit Kronecker product built here with a 2 x 2 block loop."""
    r = rng(d)
    sign = np.where(r.standard_normal(d) < 0, -1.0, 1.0)
    q28 = None
    if d % 28 == 0:
        q28, _ = np.linalg.qr(r.standard_normal((28, 28)))
    rows = [0, 1, d // 2 + 3, d - 1]
    V = O.rht_matrix(d, sign, q28)
    np.testing.assert_allclose(O.rht_rows(d, sign, q28, rows), V[rows], rtol=0, atol=1e-15)
    R = O.rht_rows(d, sign, q28, np.arange(d))
    np.testing.assert_allclose(R @ R.T, np.eye(d), atol=1e-12)
    if q28 is not None:
        m = d // 28
        for i in rows:
            a, b = divmod(i, m)
            for j in range(0, d, 37):
                a2, b2 = divmod(j, m)
                h = (-1.0) ** bin(b & b2).count("1")
                assert abs(R[i, j] - q28[a, a2] * h / np.sqrt(m) * sign[j]) < 1e-15


@pytest.mark.parametrize("m", [1, 2, 8, 64])
def test_hadamard_matches_scipy(m):
    assert np.array_equal(O.hadamard(m), scipy.linalg.hadamard(m).astype(float))


def test_hadamard_sylvester_recursion_and_orthogonality():
    h = np.array([[1.0]])
    for _ in range(5):
        h = np.block([[h, h], [h, -h]])
    assert np.array_equal(O.hadamard(32), h)
    np.testing.assert_array_equal(h @ h, 32 * np.eye(32))


@pytest.mark.parametrize("d", [16, 28 * 4, 28 * 8])
def test_rht_orthogonal(d):
    rot = synth.rotation_params(d, 5, "pin")
    V = O.rht_matrix(d, rot.sign, rot.q28_f64)
    np.testing.assert_allclose(V @ V.T, np.eye(d), atol=1e-13)
    # column k of V is sigma_k times column k of the unsigned core (signs act on the input)
    core = O.rht_matrix(d, np.ones(d), rot.q28_f64)
    np.testing.assert_array_equal(V, core * rot.sign[None, :])


def test_rht_kron_slow_index():
    # the 28-point factor mixes the slow index a of element a*m + b
    m = 4
    q = synth.rotation_params(28 * m, 1, "k").q28_f64
    V = O.rht_matrix(28 * m, np.ones(28 * m), q)
    x = np.zeros(28 * m)
    x[3 * m + 1] = 1.0  # a = 3, b = 1
    y = V @ x
    hm = O.hadamard(m) / np.sqrt(m)
    for a in range(28):
        np.testing.assert_allclose(y[a * m:(a + 1) * m], q[a, 3] * hm[:, 1], atol=1e-15)


def _rot_problem(d_out=28 * 2, d_in=16, seed=4):
    W, HX, HG = _problem(d_out, d_in, seed)
    ri = synth.rotation_params(d_in, seed, "in")
    ro = synth.rotation_params(d_out, seed, "out")
    return W, HX, HG, (ri.sign, ri.q28_f64), (ro.sign, ro.q28_f64)


def test_rotation_invariance_theorem1():
    W, HX, HG, ri, ro = _rot_problem()
    out = O.biip_forward(W, HX, HG, ri, ro, flags=O.ROT_IN | O.ROT_OUT)
    np.testing.assert_allclose(np.linalg.norm(out["W"]), np.linalg.norm(W), rtol=1e-13)
    np.testing.assert_allclose(np.linalg.eigvalsh(out["HX"]), np.linalg.eigvalsh(HX), rtol=1e-11)
    np.testing.assert_allclose(np.trace(out["HG"]), np.trace(HG), rtol=1e-12)
    dW = _dw(W.shape, 2)
    dW2 = out["U"] @ dW @ out["V"].T
    np.testing.assert_allclose(O.kfac_loss(dW2, out["HX"], out["HG"]),
                               O.kfac_loss(dW, HX, HG), rtol=1e-11)
    # W'' = U W V^T maps the rotated objective back: a transposed or swapped side would not
    np.testing.assert_allclose(out["U"].T @ out["W"] @ out["V"], W, atol=1e-13)


def test_full_biip_loss_invariance_and_revert():
    W, HX, HG, ri, ro = _rot_problem(28 * 4, 32, 7)
    out = O.biip_forward(W, HX, HG, ri, ro)
    dW = _dw(W.shape, 3)
    dW2 = out["U"] @ (out["sg"][:, None] * dW * out["sx"][None, :]) @ out["V"].T
    np.testing.assert_allclose(O.kfac_loss(dW2, out["HX"], out["HG"]),
                               O.kfac_loss(dW, HX, HG), rtol=1e-11)
    back = O.biip_revert(out["W"], out["sx"], out["sg"], out["V"], out["U"])
    np.testing.assert_allclose(back, W, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("shape,flags", [((28 * 4, 32), O.BIIP), ((64, 28 * 2), O.BIIP),
                                         ((28 * 4, 32), O.RESCALE_IN | O.ROT_IN)])
def test_biip_forward_rows_matches_dense(shape, flags):
    # the sampled-row form used at full size: the same rotated H_X, the listed rows of the
    # dense W'' and the post-BiIP traces of the dense matrices, with H_G given by its diagonal
    d_out, d_in = shape
    W, HX, HG, ri, ro = _rot_problem(d_out, d_in, 9)
    dense = O.biip_forward(W, HX, HG, ri, ro, flags)
    rows = [0, 5, d_out // 2, d_out - 1]
    part = O.biip_forward_rows(W, HX, np.diag(HG), ri, ro, rows, flags)
    np.testing.assert_allclose(part["HX"], dense["HX"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(part["W_rows"], dense["W"][rows], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(part["traces"], O.traces(dense["HX"], dense["HG"]), rtol=1e-12)
    np.testing.assert_array_equal(part["sx"], dense["sx"])
    np.testing.assert_array_equal(part["sg"], dense["sg"])


# ------------------------------------------------------------------------------------ O5/O6
def test_damp():
    H = spd(6, 1)
    Hd = O.damp(H, 0.01)
    np.testing.assert_array_equal(Hd - np.diag(np.diag(Hd)), H - np.diag(np.diag(H)))
    np.testing.assert_allclose(np.diag(Hd) - np.diag(H), 0.01 * np.mean(np.diag(H)), rtol=1e-12)


def test_inverse_cholesky_factor_routes():
    H = O.damp(spd(24, 2, cond=1e4))
    U = O.inverse_cholesky_factor(H)
    assert np.allclose(np.tril(U, -1), 0.0)
    np.testing.assert_allclose(U.T @ U @ H, np.eye(24), atol=1e-9)
    # independent route: H = R R^T with R upper (Cholesky of the index-reversed matrix), U = R^-1
    J = np.eye(24)[::-1]
    L = np.linalg.cholesky(J @ H @ J)
    R = J @ L @ J
    U2 = scipy.linalg.solve_triangular(R, np.eye(24), lower=False)
    np.testing.assert_allclose(U, U2, rtol=1e-9, atol=1e-12)


def test_inverse_cholesky_rows_are_obs_quantities():
    # [inv(H[p:, p:])]_{0, :} = U_pp U_{p, p:}: the sweep's row of U gives the OBS update
    H = O.damp(spd(20, 3, cond=1e3))
    U = O.inverse_cholesky_factor(H)
    for p in [0, 5, 19]:
        sub = np.linalg.inv(H[p:, p:])
        np.testing.assert_allclose(sub[0], U[p, p] * U[p, p:], rtol=1e-9, atol=1e-12)


# ------------------------------------------------------------------------------------ O7
def test_quantizer_hand_cases():
    # w = [-1, 0, 0.5, 1], 4 bits: scale = fp32(2/15) = 0.13333334 (rounded up), so
    # -xmin/scale = 7.4999996 and zero = 7; q(-1) = rint(-7.4999996) + 7 = 0, q(0) = 7,
    # q(0.5) = rint(3.7499998) + 7 = 11, q(1) = rint(7.4999996) + 7 = 14
    s, z = O.group_params(np.array([[-1.0, 0.0, 0.5, 1.0]]), 4)
    assert s[0] == float(np.float32(2.0 / 15.0)) and z[0] == 7.0
    q, wh = O.quantize(np.array([-1.0, 0.0, 0.5, 1.0]), np.repeat(s, 4), np.repeat(z, 4), 4)
    assert list(q) == [0, 7, 11, 14]
    assert wh[1] == 0.0  # zero is exactly representable
    # exact ties go half to even: w = [-1, 0.5, 1.5, 2], 2 bits: scale = 3/3 = 1, zero = 1,
    # q(0.5) = rint(0.5) + 1 = 1, q(1.5) = rint(1.5) + 1 = 3, q(2) = 3
    s, z = O.group_params(np.array([[-1.0, 0.5, 1.5, 2.0]]), 2)
    assert s[0] == 1.0 and z[0] == 1.0
    q, _ = O.quantize(np.array([-1.0, 0.5, 1.5, 2.0]), np.repeat(s, 4), np.repeat(z, 4), 2)
    assert list(q) == [0, 1, 3, 3]
    # all-positive group: xmin clamps to 0, zero = 0; 2 bits: scale = 3/3 = 1
    s, z = O.group_params(np.array([[0.5, 3.0, 1.5]]), 2)
    assert s[0] == 1.0 and z[0] == 0.0
    q, _ = O.quantize(np.array([0.5, 3.0, 1.5]), np.repeat(s, 3), np.repeat(z, 3), 2)
    assert list(q) == [0, 3, 2]
    # all-zero group uses the range (-1, 1): scale = fp32(2/3) (rounded up), zero = rint(1.4999999) = 1
    s, z = O.group_params(np.zeros((1, 4)), 2)
    assert s[0] == float(np.float32(2.0 / 3.0)) and z[0] == 1.0


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_quantizer_is_nearest_grid_point(bits):
    r = rng(bits)
    wg = r.standard_normal((50, 16))
    s, z = O.group_params(wg, bits)
    maxq = 2 ** bits - 1
    for col in range(16):
        q, wh = O.quantize(wg[:, col], s, z, bits)
        assert q.min() >= 0 and q.max() <= maxq
        # brute force over the grid points
        grid = s[:, None] * (np.arange(maxq + 1)[None, :] - z[:, None])
        best = np.min(np.abs(wg[:, col, None] - grid), axis=1)
        np.testing.assert_allclose(np.abs(wg[:, col] - wh), best, rtol=0, atol=1e-15)
        inside = (wg[:, col] >= grid[:, 0]) & (wg[:, col] <= grid[:, -1])
        assert np.all(np.abs(wg[inside, col] - wh[inside]) <= s[inside] / 2 * (1 + 1e-12))


def test_rtn_when_hessian_is_diagonal():
    # H_X = I and BiIP off: the factor is diagonal, nothing propagates, codes = RTN(W)
    r = rng(5)
    W = r.standard_normal((30, 256)).astype(np.float32).astype(np.float64)
    U = O.inverse_cholesky_factor(O.damp(np.eye(256)))
    res = O.obs_blocked(W, U, 4, 128, 128)
    for g in range(2):
        blk = W[:, g * 128:(g + 1) * 128]
        s, z = O.group_params(blk, 4)
        grid = s[:, None] * (np.arange(16)[None, :] - z[:, None])
        for c in range(128):
            dist = np.abs(blk[:, c, None] - grid)
            nearest = np.argmin(dist, axis=1)
            tie = np.sort(dist, axis=1)[:, 1] - np.sort(dist, axis=1)[:, 0] < 1e-15
            assert np.all((res["codes"][:, g * 128 + c] == nearest) | tie)
    np.testing.assert_allclose(res["W"], res["w_hat"], rtol=1e-14, atol=1e-15)


# ------------------------------------------------------------------------------------ O8
def _obs_problem(d_out, d_in, seed, cond=1e3):
    r = rng(seed)
    W = r.standard_normal((d_out, d_in)) * 0.02
    H = O.damp(spd(d_in, seed + 1, cond=cond))
    return W, H, O.inverse_cholesky_factor(H)


@pytest.mark.parametrize("block,group", [(128, 128), (32, 128), (256, 128), (64, 64)])
def test_blocked_equals_unblocked(block, group):
    W, H, U = _obs_problem(40, 256, 6)
    a = O.obs_unblocked(W, U, 3, group)
    b = O.obs_blocked(W, U, 3, group, block)
    np.testing.assert_array_equal(a["codes"], b["codes"])
    np.testing.assert_allclose(b["W"], a["W"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(b["err"], a["err"], rtol=1e-10, atol=1e-13)


def test_sweep_equals_textbook_obs():
    # eq. obs_update with the inverse of the remaining sub-Hessian re-formed at every step
    W, H, U = _obs_problem(16, 64, 8, cond=200.0)
    res = O.obs_unblocked(W, U, 4, 32)
    Wt = W.copy()
    codes = np.zeros_like(res["codes"])
    for p in range(64):
        if p % 32 == 0:
            s, z = O.group_params(Wt[:, p:p + 32], 4)
        q, wh = O.quantize(Wt[:, p], s, z, 4)
        hinv = np.linalg.inv(H[p:, p:])
        delta = (Wt[:, p] - wh) / hinv[0, 0]
        Wt[:, p + 1:] -= np.outer(delta, hinv[0, 1:])
        Wt[:, p] = wh
        codes[:, p] = q
    np.testing.assert_array_equal(codes, res["codes"])
    np.testing.assert_allclose(res["W"], Wt, rtol=1e-9, atol=1e-12)


def _kron_obs_step(W, What_p, p, HX, HG, F):
    """One OBS step on the full Kronecker Hessian restricted to columns F (p in F):
    dtheta = -H^-1 E_p (E_p^T H^-1 E_p)^-1 eps_p, with theta = vec(W[:, F]) stacking columns."""
    d_out = W.shape[0]
    Hf = np.kron(HX[np.ix_(F, F)], HG)
    Hinv = np.linalg.inv(Hf)
    k = F.index(p)
    E = np.kron(np.eye(len(F))[:, [k]], np.eye(d_out))
    eps = W[:, p] - What_p
    dtheta = -Hinv @ E @ np.linalg.solve(E.T @ Hinv @ E, eps)
    return dtheta.reshape(len(F), d_out).T  # back to [d_out x |F|] (column-stacked vec)


@pytest.mark.parametrize("p", [0, 2])
def test_prop1_hg_cancels(p):
    r = rng(10)
    d_out, d_in = 4, 6
    W = r.standard_normal((d_out, d_in))
    HX, HG = spd(d_in, 11), spd(d_out, 12, cond=1e3)
    What_p = np.round(W[:, p] * 2) / 2
    F = list(range(p, d_in))
    dW_kron = _kron_obs_step(W, What_p, p, HX, HG, F)
    hinv = np.linalg.inv(HX[np.ix_(F, F)])
    delta = (W[:, p] - What_p) / hinv[0, 0]
    dW_free = -np.outer(delta, hinv[0, :])
    np.testing.assert_allclose(dW_kron, dW_free, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(W[:, p] + dW_kron[:, 0], What_p, atol=1e-12)


def test_dw_equals_err_times_factor_and_ldl_identity():
    W, H, U = _obs_problem(24, 128, 13)
    res = O.obs_unblocked(W, U, 2, 128)
    dW = W - res["w_hat"]
    np.testing.assert_allclose(dW, res["err"] @ U, rtol=1e-10, atol=1e-13)
    HG = spd(24, 14, cond=1e2)
    lhs = O.kfac_loss(dW, H, HG)
    rhs = float(np.trace(res["err"].T @ HG @ res["err"]))
    np.testing.assert_allclose(lhs, rhs, rtol=1e-10)  # eq. app-decomp
    np.testing.assert_allclose(O.kfac_loss(dW, H, np.eye(24)), np.sum(res["err"] ** 2),
                               rtol=1e-10)


# ------------------------------------------------------------------------------------ O10
@pytest.mark.parametrize("shape", [(3, 5), (8, 16), (16, 7)])
def test_kfac_loss_equals_kronecker_form(shape):
    r = rng(sum(shape))
    dW = r.standard_normal(shape)
    HX, HG = spd(shape[1], 1), spd(shape[0], 2)
    v = dW.flatten(order="F")  # vec stacks columns (appendix A.1)
    direct = O.kfac_loss(dW, HX, HG)
    np.testing.assert_allclose(direct, v @ np.kron(HX, HG) @ v, rtol=1e-12)
    # row-major flattening pairs with the swapped Kronecker product
    vr = dW.flatten(order="C")
    np.testing.assert_allclose(direct, vr @ np.kron(HG, HX) @ vr, rtol=1e-12)


# ------------------------------------------------------------------------------------ O11
def test_allocation_equal_scores_is_uniform():
    bits, _ = O.allocate_bits([1.0] * 7, [1] * 7)
    assert bits == (3,) * 7


def test_allocation_hand_case():
    # one dominant layer: it gets 4 bits, paid for by one layer at 2 bits; among equal choices
    # the lexicographically smallest vector wins
    bits, val = O.allocate_bits([100.0, 1, 1, 1, 1, 1, 1], [1] * 7)
    assert bits == (4, 2, 3, 3, 3, 3, 3)
    np.testing.assert_allclose(val, 100 / 225 + 1 / 9 + 5 / 49, rtol=1e-15)


def test_allocation_respects_parameter_budget():
    specs = synth.block_layers(n_tokens=16)
    w = synth.param_count(specs)
    r = rng(3)
    s = np.exp(3 * r.standard_normal(7))
    bits, best = O.allocate_bits(s, w)
    assert np.dot(w, bits) <= 3.0 * np.sum(w)
    # brute force check that no feasible vector is better
    import itertools
    for cand in itertools.product((2, 3, 4), repeat=7):
        if np.dot(w, cand) <= 3.0 * np.sum(w):
            assert sum(si / (2 ** b - 1) ** 2 for si, b in zip(s, cand)) >= best - 1e-12 * abs(best)


def test_count_weighted_avg_bits_matches_paper_table():
    g = json.load(open(os.path.join(GOLDEN, "mp_avg_bits.json")))
    n = g["n_sublayer_types"]
    for row in g["rows"]:
        bits = [3] * row["upgraded"] + [2] * (n - row["upgraded"])
        assert round(O.count_avg_bits(bits), 2) == row["avg_bits_printed"]
