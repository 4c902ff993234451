"""Parity of the diagnostics (incoherence measures, norm variation, Jacobi eigendecomposition,
expected-loss factors) through the C ABI against the float64 oracle.

Matrix statistics are fp64 sums of exactly squared fp32 values: 1e-10 relative, the maximum
bit-exact. The eigendecomposition runs in fp32: eigenvalues to tol ||H||_F, residual and
orthogonality to tol, tol = max(1e-5, 5e-7 sqrt(sweeps d)) (the rounding accumulated over the
sweeps' rounds), and mu(H) to 1e-4 plus 1e-5 ||H|| / gap of the maximising eigenvector
(reading R25). The expected-loss factors take the same fp32 inputs as the
oracle: 1e-10.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import DEV, note, rot_oracle, to_np
from paper_2607_07964_amd import kronq as K

pytestmark = pytest.mark.gpu
ALPHAS = (0.0, 0.125, 0.25, 0.375, 0.5)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    K.load()
    assert torch.cuda.is_available(), "GPU tests need an MI355X"


def structured(rows, cols, seed, dtype=np.float32):
    r = np.random.default_rng(seed)
    M = (r.standard_normal((rows, cols)) * np.exp(0.7 * r.standard_normal(rows))[:, None]
         * np.exp(0.7 * r.standard_normal(cols))[None, :])
    return M.astype(dtype)


def spd_sep(d, seed, lo=1.0, hi=1e3):
    """SPD with geometrically spaced (separated) eigenvalues and a random eigenbasis."""
    r = np.random.default_rng(seed)
    q, _ = np.linalg.qr(r.standard_normal((d, d)))
    return ((q * np.geomspace(lo, hi, d)) @ q.T).astype(np.float32)


def check_stats(got, M64):
    cv_in, cv_out = O.norm_cv(M64)
    assert got[0] == np.max(np.abs(M64))
    np.testing.assert_allclose(got[1], np.sum(M64 * M64), rtol=1e-12)
    np.testing.assert_allclose(got[2], O.incoherence(M64), rtol=1e-12)
    np.testing.assert_allclose(got[3:5], [cv_in, cv_out], rtol=1e-10)


@pytest.mark.parametrize("rows,cols,bf16", [(37, 300, False), (300, 2100, True), (1, 5, False),
                                            (4100, 33, True), (64, 4096, False)])
def test_matrix_stats(rows, cols, bf16):
    M = torch.from_numpy(structured(rows, cols, rows + cols))
    if bf16:
        M = M.to(torch.bfloat16)
    note(f"matrix stats {rows}x{cols} bf16={bf16}")
    got = to_np(K.kronq_matrix_stats(M.to(DEV)))
    M64 = M.float().numpy().astype(np.float64)
    check_stats(got, M64)


def test_matrix_stats_strided_and_repeated():
    # a view with ld > cols; the same workspace reused for a second, smaller call
    big = torch.from_numpy(structured(50, 700, 3)).to(DEV)
    view = big[:, 100:613]
    ws = K.workspace(K.OP_STATS, 50, 700, 0, DEV)
    note("matrix stats strided view")
    a = to_np(K.kronq_matrix_stats(view, ws=ws))
    b = to_np(K.kronq_matrix_stats(big[:7, :300], ws=ws))
    check_stats(a, to_np(view).astype(np.float64))
    check_stats(b, to_np(big[:7, :300]).astype(np.float64))


def eigh_checks(H32, sweeps):
    """Eigenvalues, residual, orthogonality and convergence of the GPU eigendecomposition, and
    mu(H) against the oracle's. fp32 updates: a sweep has d/32 - 1 rounds, each a product of
    64-term dot products, so the rounding perturbation of A and V grows like sqrt(sweeps * d)
    unit roundoffs relative to ||H||_F; an eigenvector is determined to about eps ||H|| / gap,
    so mu's bound widens with 1 / (gap of the maximising eigenvector)."""
    d = H32.shape[0]
    note(f"jacobi eigh d={d} sweeps={sweeps}")
    w, Q, off = K.kronq_eigh(torch.from_numpy(H32).to(DEV), sweeps)
    torch.cuda.synchronize()
    w, Q, off = to_np(w).astype(np.float64), to_np(Q).astype(np.float64), float(off.item())
    H = H32.astype(np.float64)
    wr, Qr = O.eigenvectors(H)
    scale = np.max(np.abs(wr))
    tol = max(1e-5, 5e-7 * np.sqrt(sweeps * d))
    assert off < tol  # the off-diagonal mass left, relative: converged to rounding level
    # Weyl: each eigenvalue moves by at most the norm of the accumulated rounding perturbation
    err = np.max(np.abs(np.sort(w) - wr))
    print(f"eigh d={d}: max eigenvalue error {err:.3e} = {err / scale:.3e} max|lambda| = "
          f"{err / np.linalg.norm(H):.3e} ||H||_F (tol {tol:.2e})")
    np.testing.assert_allclose(np.sort(w), wr, rtol=0, atol=tol * np.linalg.norm(H))
    assert np.linalg.norm(H @ Q - Q * w) / np.linalg.norm(H) < tol
    assert np.max(np.abs(Q.T @ Q - np.eye(d))) < tol
    k = int(np.argmax(np.max(np.abs(Qr), axis=0)))  # the oracle's maximising eigenvector
    gap = np.min(np.abs(np.delete(wr, k) - wr[k])) if d > 1 else scale
    mu = np.sqrt(d) * np.max(np.abs(Q))
    np.testing.assert_allclose(mu, O.hessian_incoherence(H), rtol=1e-4 + 1e-5 * scale / gap)
    return mu


@pytest.mark.parametrize("d", [2, 3, 64, 130, 255])
def test_eigh_separated_spectrum(d):
    eigh_checks(spd_sep(d, d), 12)


def test_eigh_axis_aligned_and_diagonal():
    # a diagonal matrix is returned as is: Q = I (mu = sqrt(d)), the eigenvalues the diagonal
    d = 96
    lam = np.geomspace(1.0, 50.0, d).astype(np.float32)
    w, Q, off = K.kronq_eigh(torch.from_numpy(np.diag(lam)).to(DEV), 2)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(w), lam) and np.array_equal(to_np(Q), np.eye(d, dtype=np.float32))
    assert float(off.item()) == 0.0


def test_eigh_mu_before_and_after_biip_rotation():
    # Fig. 2a on a synthetic gradient covariance: coherent before, incoherent after the
    # randomised Hadamard rotation; mu from the GPU eigenvectors equals the oracle's
    spec = synth.small_spec(256, 256, 4096, seed=21)
    G = synth.gen_matrix(spec.g, DEV)
    HG = torch.empty(256, 256, device=DEV)
    K.kronq_accumulate_cov(G, HG)
    torch.cuda.synchronize()
    H32 = to_np(HG)
    mu0 = eigh_checks(H32, 12)
    ro = synth.rotation_params(256, 3, "diag:out")
    sgn, q = rot_oracle(ro)
    Vr = O.rht_matrix(256, sgn, q)
    Hr = (Vr @ H32.astype(np.float64) @ Vr.T).astype(np.float32)
    mu1 = eigh_checks(Hr, 14)
    assert mu0 / 16.0 > 0.9 and mu1 / 16.0 < 0.45


@pytest.mark.parametrize("bf16", [False, True])
def test_proxy_loss_factors(bf16):
    r = np.random.default_rng(5)
    d_out, d_in = 200, 384
    W = torch.from_numpy(structured(d_out, d_in, 6))
    if bf16:
        W = W.to(torch.bfloat16)
    W64 = W.float().numpy().astype(np.float64)
    G = r.standard_normal((1000, d_out)) * np.exp(1.5 * r.standard_normal(d_out))
    HG = (G.T @ G).astype(np.float32)
    Hd = O.damp(spd_sep(d_in, 7, 1.0, 1e2).astype(np.float64)).astype(np.float32)
    U = O.inverse_cholesky_factor(Hd.astype(np.float64)).astype(np.float32)
    note(f"proxy loss factors bf16={bf16}")
    got = to_np(K.kronq_proxy_loss_factors(
        torch.from_numpy(HG).to(DEV), W.to(DEV), torch.from_numpy(Hd).to(DEV),
        torch.from_numpy(np.ascontiguousarray(U)).to(DEV), ALPHAS))
    f = O.proxy_loss_factors(HG, W64, Hd, U)
    h, a = np.diag(HG).astype(np.float64), np.sum(W64 * W64, axis=1)
    ref = [f["nearest"], f["gptq"], f["kronq"], f["rho"], f["trD"], f["trH"]]
    ref += [O.rescale_objective(h, a, al) * f["trD"] for al in ALPHAS]
    np.testing.assert_allclose(got, ref, rtol=1e-10)
    # the sweep is minimal at 1/4 and brackets the GPTQ and KronQ rows
    assert int(np.argmin(got[6:])) == 2
    assert got[6] == pytest.approx(got[1], rel=1e-12) and got[8] == pytest.approx(got[2], rel=1e-12)


# ------------------------------------------------------------------------------ full size
@pytest.mark.slow
def test_matrix_stats_full_size_70b_weight():
    spec = synth.workload(4)
    note("matrix stats of the 70B up_proj weight 28672x8192 bf16")
    W = synth.gen_matrix(spec.w, DEV)
    got = to_np(K.kronq_matrix_stats(W))
    M64 = O.as_f64(synth.bf16_bits(W.cpu()))
    check_stats(got, M64)


@pytest.mark.slow
def test_eigh_full_size_q_proj_hessians():
    """H_X and H_G of the LLaMA-3-8B q_proj workload (d = 4096, N = 262144), with the sweep
    count bench.py --diagnostics uses."""
    spec = synth.workload(2)
    for name, ms in (("H_X", spec.x), ("H_G", spec.g)):
        A = synth.gen_matrix(ms, DEV)
        H = torch.empty(4096, 4096, device=DEV)
        K.kronq_accumulate_cov(A, H)
        torch.cuda.synchronize()
        del A
        note(f"full-size eigh of the q_proj {name}")
        eigh_checks(to_np(H), 12)
