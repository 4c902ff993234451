"""Stage-isolated parity: each HIP step through the C ABI against the float64 oracle.

Each stage gets inputs from the seeded generator or from the oracle (rounded to the fp32 the
library takes), never from another HIP step. Sizes span several tiles and ragged tails.
Tolerances: 1e-3 relative Frobenius error for covariances, traces and rotated matrices;
codes bit-exact in the round-to-nearest case and >= 99.5 % identical otherwise; loss 1e-3.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import DEV, note, oracle_view, rel_frob, rot_device, rot_oracle, to_np
from paper_2607_07964_amd import kronq as K
from paper_2607_07964_amd.layer import RotParams

pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _lib():
    K.load()
    assert torch.cuda.is_available(), "GPU tests need an MI355X"


def f32(a) -> torch.Tensor:
    """fp32 device copy with rows padded to 16 bytes (the library's layout contract)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if a.ndim == 2 and a.shape[1] % 4:
        buf = torch.zeros(a.shape[0], a.shape[1] + 4 - a.shape[1] % 4, device=DEV)
        buf[:, :a.shape[1]] = torch.from_numpy(a).to(DEV)
        return buf[:, :a.shape[1]]
    return torch.tensor(a, device=DEV)


def spd_from_tokens(d, n, seed, kind="normal_t3"):
    """An oracle covariance of generator tokens, rounded to fp32 (the form the library takes)."""
    spec = synth.small_spec(d, d, n, seed=seed, xkind=kind).x
    H = O.covariance(oracle_view(synth.gen_matrix(spec)))
    return H.astype(np.float32).astype(np.float64)


# ------------------------------------------------------------------------------ generator
def test_generator_gpu_matches_cpu():
    s = synth.small_spec(448, 256, 3000)
    for spec in (s.x, s.g, s.w):
        note(f"generator {spec.tag} {spec.rows}x{spec.cols}")
        assert torch.equal(synth.gen_matrix(spec, DEV).cpu(), synth.gen_matrix(spec))


# ------------------------------------------------------------------------------ covariance
@pytest.mark.parametrize("n,d", [(1000, 300), (5000, 600), (64, 8), (4099, 1024), (70, 257)])
def test_cov_bf16(n, d):
    dp = (d + 7) // 8 * 8  # rows padded to 16 bytes; the first d channels are used
    spec = synth.small_spec(dp, dp, n, seed=n + d).x
    X = synth.gen_matrix(spec, DEV)[:, :d]
    H = torch.full((d, d), float("nan"), device=DEV)
    note(f"cov bf16 n={n} d={d}")
    K.kronq_accumulate_cov(X, H)
    torch.cuda.synchronize()
    ref = O.covariance(oracle_view(synth.gen_matrix(spec))[:, :d])
    h = to_np(H)
    assert rel_frob(h, ref) < TOL
    assert np.array_equal(h, h.T)


@pytest.mark.parametrize("n", [7 * 1024 + 5, 9192, 10000, 12345, 16391, 20000])
def test_cov_bf16_stage_counts(n):
    """One 256-channel tile over 7 to 20 whole 32-token stages per slice (slices and their last
    one of varied length): the steady state of the stage ring with every remainder of stages
    left to its checked tail, and the loads of a stage split over two half-stages."""
    d = 256
    spec = synth.small_spec(d, d, n, seed=n).x
    X = synth.gen_matrix(spec, DEV)
    H = torch.full((d, d), float("nan"), device=DEV)
    note(f"cov bf16 stage counts n={n} d={d}")
    K.kronq_accumulate_cov(X, H)
    torch.cuda.synchronize()
    ref = O.covariance(oracle_view(synth.gen_matrix(spec)))
    assert rel_frob(to_np(H), ref) < TOL


def test_cov_chained_scaled_and_strided():
    n1, n2, d = 1500, 900, 520
    spec = synth.small_spec(d + 8, d + 8, n1 + n2, seed=5).x
    Xw = synth.gen_matrix(spec, DEV)  # [n, d + 8]; use the first d columns (lda = d + 8)
    X1, X2 = Xw[:n1, :d], Xw[n1:, :d]
    H = torch.empty(d, d, device=DEV)
    note("cov chained beta=1, alpha=1/N, lda > d")
    K.kronq_accumulate_cov(X1, H, alpha=1.0 / (n1 + n2), beta=0.0)
    K.kronq_accumulate_cov(X2, H, alpha=1.0 / (n1 + n2), beta=1.0)
    torch.cuda.synchronize()
    ref = O.covariance(oracle_view(synth.gen_matrix(spec))[:, :d]) / (n1 + n2)
    assert rel_frob(to_np(H), ref) < TOL


@pytest.mark.parametrize("max_cus", [8, 5, 24, 100000])
def test_cov_limited_matches_uncapped(max_cus):
    """The covariance holding at most max_cus CUs (persistent workgroups, several work items
    each) matches the oracle and the uncapped launch; 100000 exceeds the work items (no cap), 5
    is not a multiple of 8. The capped launch may cut the tokens into fewer slices (whole rounds
    of its own workgroups), so it agrees with the uncapped one up to the order of its fp32 sums."""
    n, d = 9000, 1280  # 5 x 5 channel blocks, 15 upper tiles, several token slices
    spec = synth.small_spec(d, d, n, seed=17).x
    X = synth.gen_matrix(spec, DEV)
    H0 = torch.empty(d, d, device=DEV)
    H1 = torch.full((d, d), float("nan"), device=DEV)
    note(f"cov limited max_cus={max_cus}")
    K.kronq_accumulate_cov(X, H0)
    K.kronq_accumulate_cov_limited(X, H1, max_cus)
    torch.cuda.synchronize()
    assert rel_frob(to_np(H1), to_np(H0)) < 1e-5
    assert torch.equal(H1, H1.T)
    ref = O.covariance(oracle_view(synth.gen_matrix(spec)))
    assert rel_frob(to_np(H1), ref) < TOL


@pytest.mark.parametrize("max_cus", [8, 5, 24])
def test_cov_limited_bits_when_the_plans_agree(max_cus):
    """At d = 1536, N = 8192 every one of these caps keeps the uncapped launch's 8 token slices
    (21 tiles x 8 slices fill whole rounds of 8, 24 and nearly of 5 workgroups, and more slices
    cost more partial tiles than they save), so the persistent workgroups, each walking several
    work items, must give exactly the uncapped launch's bits."""
    n, d = 8192, 1536
    spec = synth.small_spec(d, d, n, seed=23).x
    X = synth.gen_matrix(spec, DEV)
    H0 = torch.empty(d, d, device=DEV)
    H1 = torch.full((d, d), float("nan"), device=DEV)
    note(f"cov limited, same plan, max_cus={max_cus}")
    K.kronq_accumulate_cov(X, H0)
    K.kronq_accumulate_cov_limited(X, H1, max_cus)
    torch.cuda.synchronize()
    assert torch.equal(H0, H1)


@pytest.mark.parametrize("n,d,bf16", [(1000, 300, True), (5000, 600, True), (64, 8, True),
                                      (4099, 1030, True), (70, 257, True), (3000, 260, False),
                                      (200000, 64, True), (2, 4096, True), (3001, 2048, True),
                                      (1000, 6144, True), (2000, 4096, False)])
def test_cov_diag(n, d, bf16):
    """diag(A^T A) from one read of A: fp64 sums of exact bf16 squares (fp32 squares are exact
    in fp64 too), rounded once, so within one fp32 ulp of the oracle's diagonal; lda > d for
    ragged d; whole 4096-column blocks, a half block (2048, 6144) and ragged blocks; a second
    call gives the same bits."""
    dp = (d + 7) // 8 * 8
    spec = synth.small_spec(dp, dp, n, seed=n + 3 * d).x
    A = synth.gen_matrix(spec, DEV)
    if not bf16:
        g = torch.Generator().manual_seed(d)
        A = (A.float() * (1.0 + 1e-3 * torch.randn(A.shape, generator=g)).to(DEV)).contiguous()
    A = A[:, :d]
    note(f"cov diag n={n} d={d} bf16={bf16}")
    got = K.kronq_cov_diag(A)
    again = K.kronq_cov_diag(A, out=torch.full((d,), float("nan"), device=DEV))
    few = K.kronq_cov_diag(A, max_cus=8)  # fewer, longer chunks
    torch.cuda.synchronize()
    assert torch.equal(got, again)
    ref = np.diag(O.covariance(oracle_view(A.cpu().contiguous())))
    np.testing.assert_allclose(to_np(got), ref, rtol=1.2e-7, atol=0)
    np.testing.assert_allclose(to_np(few), ref, rtol=1.2e-7, atol=0)


def test_cov_diag_empty_and_matches_covariance():
    spec = synth.small_spec(512, 512, 3000, seed=8).x
    A = synth.gen_matrix(spec, DEV)
    note("cov diag n_rows=0")
    z = K.kronq_cov_diag(A[:0], out=torch.full((512,), 7.0, device=DEV))
    H = torch.empty(512, 512, device=DEV)
    K.kronq_accumulate_cov(A, H)
    dg = K.kronq_cov_diag(A)
    torch.cuda.synchronize()
    assert torch.equal(z, torch.zeros(512, device=DEV))
    # the covariance's diagonal (fp32 accumulation) agrees to its own rounding
    np.testing.assert_allclose(to_np(torch.diagonal(H)), to_np(dg), rtol=2e-6)


def test_cov_fp32_and_empty():
    s = synth.workload(1)
    X = synth.gen_matrix(s.x, DEV)
    H = torch.empty(256, 256, device=DEV)
    note("cov fp32 2048x256")
    K.kronq_accumulate_cov(X, H)
    torch.cuda.synchronize()
    ref = O.covariance(synth.gen_matrix(s.x).numpy())
    assert rel_frob(to_np(H), ref) < TOL
    note("cov n_rows=0")
    H2 = H.clone()
    K.kronq_accumulate_cov(X[:0], H2, beta=0.5)
    torch.cuda.synchronize()
    assert torch.equal(H2, H * 0.5)


# ------------------------------------------------------------------------------ traces
def test_traces():
    hx, hg = spd_from_tokens(300, 700, 1), spd_from_tokens(448, 900, 2)
    note("traces")
    out = K.kronq_traces(f32(hx), f32(hg))
    torch.cuda.synchronize()
    ref = np.array(O.traces(hx, hg))
    np.testing.assert_allclose(to_np(out), ref, rtol=1e-9)


# ------------------------------------------------------------------------------ rotation
ROT_CASES = [
    (448, 256, K.BIIP), (512, 224, K.BIIP), (256, 256, K.RESCALE_IN | K.RESCALE_OUT),
    (448, 256, K.ROT_IN | K.ROT_OUT), (448, 256, K.RESCALE_IN | K.ROT_IN),
    (448, 256, K.RESCALE_OUT | K.ROT_OUT), (2048, 1024, K.BIIP), (28 * 32, 4096, K.BIIP),
    # output sizes off the 16-row blocks of the norm kernel (its partial-block path)
    (200, 256, K.RESCALE_IN | K.RESCALE_OUT | K.ROT_IN), (132, 512, K.BIIP & ~K.ROT_OUT),
]


def _rot_problem(d_out, d_in, seed=3):
    s = synth.small_spec(d_out, d_in, 4 * max(d_in, d_out), seed=seed)
    W = synth.gen_matrix(s.w)
    hx = spd_from_tokens(d_in, 2 * d_in, seed + 1)
    hg = spd_from_tokens(d_out, 2 * d_out, seed + 2)
    ri = synth.rotation_params(d_in, seed, "in")
    try:
        ro = synth.rotation_params(d_out, seed, "out")
    except ValueError:  # an output size no transform takes: signs that are never read
        ro = synth.Rot(d_out, np.ones(d_out, dtype=np.int8), None, None)
    return s, W, hx, hg, ri, ro


@pytest.mark.parametrize("d_out,d_in,flags", ROT_CASES)
def test_rotate_forward(d_out, d_in, flags):
    s, W, hx, hg, ri, ro = _rot_problem(d_out, d_in)
    HX, HG = f32(hx), f32(hg)
    Wd = torch.empty(d_out, d_in, device=DEV)
    sx = torch.empty(d_in, device=DEV)
    sg = torch.empty(d_out, device=DEV)
    rin, rout = rot_device(ri), rot_device(ro)
    note(f"rotate {d_out}x{d_in} flags={flags}")
    K.kronq_rotate(W.to(DEV), Wd, HX, HG, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg, flags)
    torch.cuda.synchronize()
    ref = O.biip_forward(oracle_view(W), hx, hg, rot_oracle(ri), rot_oracle(ro), flags)
    assert rel_frob(to_np(Wd), ref["W"]) < TOL
    assert rel_frob(to_np(HX), ref["HX"]) < TOL
    assert rel_frob(to_np(HG), ref["HG"]) < TOL
    np.testing.assert_allclose(to_np(sx), ref["sx"], rtol=1e-5)
    np.testing.assert_allclose(to_np(sg), ref["sg"], rtol=1e-5)


@pytest.mark.parametrize("d_out", [16384, 28 * 1024])
def test_rotate_long_rows_sampled(d_out):
    """Output sides of 16384 and 28 * 1024: their row passes hold one workgroup per CU, each
    walking its rows (64 and 112) with the next row prefetched into registers. H from 64 tokens,
    so that an entry of U S^-1 H_G S^-1 U^T is a dot product of two rotated token rows (the
    oracle's rotated rows, as in the full-size sampled test); sampled entries of the rotated W."""
    d_in, ntok = 256, 64
    s = synth.small_spec(d_out, d_in, ntok, seed=5, name="long_rows")
    ax = O.as_f64(oracle_view(synth.gen_matrix(s.x)))
    ag = O.as_f64(oracle_view(synth.gen_matrix(s.g)))
    W = synth.gen_matrix(s.w)
    ri = synth.rotation_params(d_in, 5, "long_rows:in")
    ro = synth.rotation_params(d_out, 5, "long_rows:out")
    HX = f32(O.covariance(ax))
    HG = f32(O.covariance(ag))
    hx_diag = to_np(torch.diagonal(HX)).astype(np.float64)
    hg_diag = to_np(torch.diagonal(HG)).astype(np.float64)
    w = O.as_f64(oracle_view(W))
    sx, sg = O.rescale_factors(w, hx_diag, hg_diag)
    Wd = torch.empty(d_out, d_in, device=DEV)
    sxd = torch.empty(d_in, device=DEV)
    sgd = torch.empty(d_out, device=DEV)
    rin, rout = rot_device(ri), rot_device(ro)
    note(f"rotate long rows {d_out}x{d_in}")
    K.kronq_rotate(W.to(DEV), Wd, HX, HG, rin.sign, rout.sign, rin.q28, rout.q28, sxd, sgd,
                   K.BIIP)
    torch.cuda.synchronize()
    assert rel_frob(to_np(sgd), sg) < TOL
    rng = np.random.default_rng(12)
    sgn, q = rot_oracle(ro)
    rows = np.sort(rng.choice(d_out, 16, replace=False))
    Uo = O.rht_rows(d_out, sgn, q, rows)
    R = (Uo / sg[None, :]) @ ag.T
    ref = R @ R.T
    got = to_np(HG[rows][:, rows]).astype(np.float64)
    scale = np.sqrt(np.outer(np.diag(ref), np.diag(ref)))
    assert np.max(np.abs(got - ref) / scale) < TOL
    sgi, qi = rot_oracle(ri)
    cols = np.sort(rng.choice(d_in, 8, replace=False))
    Vo = O.rht_rows(d_in, sgi, qi, cols)
    ref_w = Uo @ (sg[:, None] * w * sx[None, :]) @ Vo.T
    got_w = to_np(Wd[rows][:, cols]).astype(np.float64)
    assert rel_frob(got_w, ref_w) < TOL


def test_rotate_inverse_and_in_place():
    d_out, d_in = 448, 256
    s, W, hx, hg, ri, ro = _rot_problem(d_out, d_in, 9)
    rin, rout = rot_device(ri), rot_device(ro)
    Wf = W.float().to(DEV)
    Wd = Wf.clone()
    sx = torch.empty(d_in, device=DEV)
    sg = torch.empty(d_out, device=DEV)
    note("rotate in place fp32, then inverse")
    K.kronq_rotate(Wd, Wd, f32(hx), f32(hg), rin.sign, rout.sign, rin.q28, rout.q28, sx, sg,
                   K.BIIP)
    back = torch.empty_like(Wd)
    K.kronq_rotate(Wd, back, None, None, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg,
                   K.BIIP | K.INVERSE)
    torch.cuda.synchronize()
    assert rel_frob(to_np(back), oracle_view(W.float())) < 1e-5
    # inverse of an arbitrary matrix against the oracle's revert (sx, sg as inputs)
    rng = np.random.default_rng(4)
    Wh = rng.standard_normal((d_out, d_in)).astype(np.float32)
    sxv = np.exp(rng.standard_normal(d_in) * 0.3).astype(np.float32)
    sgv = np.exp(rng.standard_normal(d_out) * 0.3).astype(np.float32)
    out = torch.empty(d_out, d_in, device=DEV)
    note("rotate inverse of a random matrix")
    K.kronq_rotate(f32(Wh), out, None, None, rin.sign, rout.sign, rin.q28, rout.q28, f32(sxv),
                   f32(sgv), K.BIIP | K.INVERSE)
    torch.cuda.synchronize()
    V = O.rht_matrix(d_in, *rot_oracle(ri))
    U = O.rht_matrix(d_out, *rot_oracle(ro))
    ref = O.biip_revert(Wh, sxv.astype(np.float64), sgv.astype(np.float64), V, U)
    assert rel_frob(to_np(out), ref) < TOL


# ------------------------------------------------------------------------------ Cholesky
# sizes cover one leaf, a ragged last leaf, odd leaf counts (uneven recursive splits) and
# several levels of the recursion; in 8392 the two largest levels take the split-bf16 path with
# ragged operand edges (4168 x 4224 products), in 8193 the top level's first three products do
# (4097 rows) while its last (K = 4097) falls back to the fp32 kernels (fewer tokens at these
# sizes: the oracle's covariance cost)
@pytest.mark.parametrize("d", [77, 128, 256, 300, 384, 640, 1000, 1024, 2112, 4096, 4200, 8193,
                               8392])
def test_cholesky_inverse_factor(d):
    h = spd_from_tokens(d, 3 * d if d <= 4200 else d + 512, d)
    H = f32(h)
    U = torch.full((d, d), float("nan"), device=DEV)
    note(f"cholesky_inv d={d}")
    info = K.kronq_cholesky_inv(H, U, 0.01)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    hd = O.damp(h, 0.01)
    np.testing.assert_allclose(to_np(H), hd, rtol=2e-6, atol=1e-6 * np.abs(hd).max())
    ref = O.inverse_cholesky_factor(hd)
    u = to_np(U)
    assert np.all(np.tril(u, -1) == 0.0)
    assert rel_frob(u, ref) < TOL


@pytest.mark.parametrize("d,bad", [(300, 5), (512, 200)])
def test_cholesky_not_pd_reports_pivot(d, bad):
    """A negative diagonal entry in a ragged last leaf (300) and inside a later panel of a full
    leaf (512): *info is the 1-based column of the failing pivot in the original order."""
    h = np.eye(d)
    h[bad, bad] = -1.0
    H = f32(h)
    U = torch.empty(d, d, device=DEV)
    note(f"cholesky_inv not PD d={d}")
    info = K.kronq_cholesky_inv(H, U, 0.01)
    torch.cuda.synchronize()
    assert int(info.item()) == bad + 1


# ------------------------------------------------------------------------------ OBS sweep
def _obs_run(W32: np.ndarray, U32: np.ndarray, bits: int, with_err=True):
    d_out, d_in = W32.shape
    W = f32(W32)
    codes = torch.empty(d_out, d_in, dtype=torch.uint8, device=DEV)
    scales = torch.empty(d_out, d_in // 128, device=DEV)
    zeros = torch.empty(d_out, d_in // 128, device=DEV)
    err = torch.empty(d_out, d_in, device=DEV) if with_err else None
    W_hat = torch.empty(d_out, d_in, device=DEV)
    K.kronq_obs_quantize_layer(W, f32(U32), bits, codes, scales, zeros, err, W_hat)
    torch.cuda.synchronize()
    return dict(W=to_np(W), codes=to_np(codes), scales=to_np(scales), zeros=to_np(zeros),
                err=None if err is None else to_np(err), w_hat=to_np(W_hat))


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_obs_rtn_bit_exact(bits):
    d_out, d_in = 200, 384
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=bits).w).float().numpy()
    U = O.inverse_cholesky_factor(O.damp(np.eye(d_in))).astype(np.float32)
    note(f"obs RTN bits={bits}")
    g = _obs_run(W, U, bits)
    ref = O.obs_blocked(W.astype(np.float64), U.astype(np.float64), bits, 128, 128)
    assert np.array_equal(g["codes"], ref["codes"])
    assert np.array_equal(g["scales"], ref["scales"].astype(np.float32))
    assert np.array_equal(g["zeros"], ref["zeros"])
    np.testing.assert_allclose(g["w_hat"], ref["w_hat"], rtol=1e-6, atol=1e-9)
    np.testing.assert_array_equal(g["W"], g["w_hat"])


@pytest.mark.parametrize("d_out,d_in,bits", [(200, 384, 4), (130, 512, 2), (64, 128, 3)])
def test_obs_general(d_out, d_in, bits):
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=d_out).w).float().numpy()
    h = O.damp(spd_from_tokens(d_in, 2 * d_in, d_in + 1))
    U = O.inverse_cholesky_factor(h).astype(np.float32)
    note(f"obs general {d_out}x{d_in} bits={bits}")
    g = _obs_run(W, U, bits)
    ref = O.obs_blocked(W.astype(np.float64), U.astype(np.float64), bits, 128, 128)
    same = g["codes"] == ref["codes"]
    agree = float(np.mean(same))
    print(f"code agreement {agree:.6f}")
    assert agree >= 0.995, agree
    rows = np.all(same, axis=1)  # rows whose codes all agree follow the same path
    assert rows.mean() > 0.5
    assert rel_frob(g["w_hat"][rows], ref["w_hat"][rows]) < TOL
    assert rel_frob(g["err"][rows], ref["err"][rows]) < TOL
    assert rel_frob(g["scales"], ref["scales"]) < TOL


def test_obs_without_err_output():
    d_out, d_in = 96, 256
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=8).w).float().numpy()
    U = O.inverse_cholesky_factor(O.damp(spd_from_tokens(d_in, 600, 3))).astype(np.float32)
    note("obs without err")
    a = _obs_run(W, U, 4, with_err=False)
    b = _obs_run(W, U, 4, with_err=True)
    assert np.array_equal(a["codes"], b["codes"]) and np.array_equal(a["W"], b["W"])


# ------------------------------------------------------------------------------ loss
@pytest.mark.parametrize("d_out,d_in", [(448, 256), (130, 203)])
def test_layer_loss(d_out, d_in):
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=1).w)
    rng = np.random.default_rng(0)
    Wh = (W.float().numpy() + 1e-3 * rng.standard_normal((d_out, d_in))).astype(np.float32)
    hx, hg = spd_from_tokens(d_in, 700, 4), spd_from_tokens(d_out, 700, 5)
    note(f"loss {d_out}x{d_in}")
    out = K.kronq_layer_loss(W.to(DEV), f32(Wh), f32(hx), f32(hg))
    torch.cuda.synchronize()
    ref = O.kfac_loss(oracle_view(W.float()) - Wh.astype(np.float64), hx, hg)
    assert abs(float(out.item()) / ref - 1.0) < TOL


def test_rotate_split_equals_one_call():
    """H_X half then the W / H_G half (the two-stream schedule) gives the one-call result."""
    d_out, d_in = 448, 512
    s, W, hx, hg, ri, ro = _rot_problem(d_out, d_in, 12)
    rin, rout = rot_device(ri), rot_device(ro)
    Wb = W.to(DEV)
    outs = []
    for split in (False, True):
        HX, HG = f32(hx), f32(hg)
        Wd = torch.empty(d_out, d_in, device=DEV)
        sx = torch.empty(d_in, device=DEV)
        sg = torch.empty(d_out, device=DEV)
        note(f"rotate split={split}")
        if split:
            K.kronq_rotate(Wb, None, HX, None, rin.sign, None, rin.q28, None, sx, sg,
                           K.BIIP | K.HX_ONLY)
            K.kronq_rotate(Wb, Wd, None, HG, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg,
                           K.BIIP | K.SX_GIVEN)
        else:
            K.kronq_rotate(Wb, Wd, HX, HG, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg, K.BIIP)
        torch.cuda.synchronize()
        outs.append([to_np(t) for t in (Wd, HX, HG, sx, sg)])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("d_out,d_in,flags", [(448, 512, K.BIIP), (2048, 896, K.BIIP),
                                              (448, 256, K.RESCALE_OUT | K.ROT_OUT),
                                              (256, 256, K.RESCALE_IN | K.RESCALE_OUT)])
def test_rotate_hg_split_equals_one_call(d_out, d_in, flags):
    """H_X half, then W with S_G from diag(H_G) (HG_DIAG), then H_G from the given sg
    (SG_GIVEN) -- the sweep no longer waits for H_G -- gives the one-call result bit for bit
    when the diagonal passed is H_G's own; also HG_DIAG without SX_GIVEN (W and H_X at once)."""
    s, W, hx, hg, ri, ro = _rot_problem(d_out, d_in, 21)
    rin, rout = rot_device(ri), rot_device(ro)
    Wb = W.to(DEV)
    outs = []
    for mode in ("one", "three", "two"):
        HX, HG = f32(hx), f32(hg)
        hgd = torch.diagonal(HG).contiguous()
        Wd = torch.full((d_out, d_in), float("nan"), device=DEV)
        sx = torch.empty(d_in, device=DEV)
        sg = torch.empty(d_out, device=DEV)
        note(f"rotate H_G split mode={mode} {d_out}x{d_in} flags={flags}")
        if mode == "one":
            K.kronq_rotate(Wb, Wd, HX, HG, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg, flags)
        else:
            if mode == "three":
                K.kronq_rotate(Wb, None, HX, None, rin.sign, None, rin.q28, None, sx, sg,
                               flags | K.HX_ONLY)
                K.kronq_rotate(Wb, Wd, None, hgd, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg,
                               flags | K.SX_GIVEN | K.HG_DIAG)
            else:
                K.kronq_rotate(Wb, Wd, HX, hgd, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg,
                               flags | K.HG_DIAG)
            hg_before = HG.clone()
            K.kronq_rotate(None, None, None, HG, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg,
                           flags | K.SX_GIVEN | K.SG_GIVEN)
            torch.cuda.synchronize()
            assert not torch.equal(HG, hg_before) or not (flags & (K.RESCALE_OUT | K.ROT_OUT))
        torch.cuda.synchronize()
        outs.append([to_np(t) for t in (Wd, HX, HG, sx, sg)])
    for other in outs[1:]:
        for a, b in zip(outs[0], other):
            np.testing.assert_array_equal(a, b)


def test_traces_split_across_calls():
    hx, hg = spd_from_tokens(300, 700, 1), spd_from_tokens(448, 900, 2)
    out = torch.zeros(3, dtype=torch.float64, device=DEV)
    note("traces split")
    K.kronq_traces(f32(hx), None, out)
    K.kronq_traces(None, f32(hg), out)
    torch.cuda.synchronize()
    np.testing.assert_allclose(to_np(out), np.array(O.traces(hx, hg)), rtol=1e-9)
