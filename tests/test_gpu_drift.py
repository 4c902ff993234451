"""Parity of the drift-corrected path (KronQ+GPTAQ) and of quantisation groups wider than one
block, through the C ABI against the float64 oracle.

Inputs come from the seeded generator or from the oracle (rounded to the fp32 the library takes),
never from another HIP step. Sizes span several tiles and ragged tails. Tolerances as for the
plain path: 1e-3 relative Frobenius error for matrices (1e-4 for the drift statistic, whose
products are exact), codes bit-exact in the round-to-nearest case and >= 99.5 % identical
otherwise.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import DEV, note, oracle_view, rel_frob, rot_device, rot_oracle, to_np
from paper_2607_07964_amd import kronq as K
from paper_2607_07964_amd import layer as L

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


def as32(a) -> np.ndarray:
    """The fp32 value the library receives, widened again for the oracle."""
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def tokens(d, n, seed, kind="normal_t3"):
    """(spec, X, dX) of a small generator layer with d input channels (CPU tensors)."""
    spec = synth.small_spec(d, d, n, seed=seed, xkind=kind)
    X = synth.gen_matrix(spec.x)
    return spec, X, synth.gen_drift(spec, X=X)


def hd_u_d(d, seed, alpha=1.0):
    """A damped H~ and its factor U from generator tokens, the drift statistic D and P."""
    _, X, dX = tokens(d, 3 * d, seed)
    h = as32(O.covariance(oracle_view(X)))
    U = as32(O.inverse_cholesky_factor(O.damp(h)))
    D = as32(O.cross_covariance(oracle_view(dX), oracle_view(X)))
    return U, D, as32(O.gptaq_correction(D, U, alpha))


# ------------------------------------------------------------------------------ drift statistic
@pytest.mark.parametrize("n,d", [(1000, 300), (5000, 600), (64, 8), (4099, 1024), (70, 257),
                                 (3000, 512)])
def test_cross_bf16(n, d):
    dp = (d + 7) // 8 * 8  # rows padded to 16 bytes; the first d channels are used
    spec, X, dX = tokens(dp, n, n + d)
    C = torch.full((d, d), float("nan"), device=DEV)
    note(f"cross bf16 n={n} d={d}")
    K.kronq_accumulate_cross(dX.to(DEV)[:, :d], X.to(DEV)[:, :d], C)
    torch.cuda.synchronize()
    ref = O.cross_covariance(oracle_view(dX)[:, :d], oracle_view(X)[:, :d])
    assert rel_frob(to_np(C), ref) < 1e-4


@pytest.mark.parametrize("max_cus", [8, 5, 24])
def test_cross_limited_matches_uncapped(max_cus):
    """The drift statistic on at most max_cus CUs (persistent workgroups, several work items
    each): at d = 1536, N = 8192 every one of these caps keeps the uncapped launch's 8 token
    slices (36 tiles x 8 slices), so the bits must be the uncapped launch's; and it matches the
    oracle."""
    n, d = 8192, 1536
    spec, X, dX = tokens(d, n, 31)
    C0 = torch.empty(d, d, device=DEV)
    C1 = torch.full((d, d), float("nan"), device=DEV)
    note(f"cross limited max_cus={max_cus}")
    K.kronq_accumulate_cross(dX.to(DEV), X.to(DEV), C0)
    K.kronq_accumulate_cross_limited(dX.to(DEV), X.to(DEV), C1, max_cus)
    torch.cuda.synchronize()
    assert torch.equal(C0, C1)
    ref = O.cross_covariance(oracle_view(dX), oracle_view(X))
    assert rel_frob(to_np(C1), ref) < 1e-4


@pytest.mark.parametrize("max_cus", [8, 40])
def test_cross_limited_fewer_slices(max_cus):
    """At d = 768, N = 20000 the uncapped drift statistic cuts the tokens into 24 slices and a
    launch capped to 8 or 40 CUs into 8 (whole rounds of its own workgroups): the same sums in
    another order, so it agrees with the uncapped launch to fp32 rounding and with the oracle."""
    n, d = 20000, 768
    spec, X, dX = tokens(d, n, 37)
    C0 = torch.empty(d, d, device=DEV)
    C1 = torch.full((d, d), float("nan"), device=DEV)
    note(f"cross limited, fewer slices, max_cus={max_cus}")
    K.kronq_accumulate_cross(dX.to(DEV), X.to(DEV), C0)
    K.kronq_accumulate_cross_limited(dX.to(DEV), X.to(DEV), C1, max_cus)
    torch.cuda.synchronize()
    assert rel_frob(to_np(C1), to_np(C0)) < 1e-5
    ref = O.cross_covariance(oracle_view(dX), oracle_view(X))
    assert rel_frob(to_np(C1), ref) < 1e-4


def test_cross_chained_scaled_fp32_and_symmetric_case():
    n1, n2, d = 1500, 900, 520
    spec, X, dX = tokens(d + 8, n1 + n2, 7)
    Xd, dXd = X.to(DEV)[:, :d], dX.to(DEV)[:, :d]
    C = torch.empty(d, d, device=DEV)
    note("cross chained beta=1, alpha=1/N, ld > d")
    K.kronq_accumulate_cross(dXd[:n1], Xd[:n1], C, alpha=1.0 / (n1 + n2), beta=0.0)
    K.kronq_accumulate_cross(dXd[n1:], Xd[n1:], C, alpha=1.0 / (n1 + n2), beta=1.0)
    torch.cuda.synchronize()
    ref = O.cross_covariance(oracle_view(dX)[:, :d], oracle_view(X)[:, :d]) / (n1 + n2)
    assert rel_frob(to_np(C), ref) < 1e-4
    # fp32 inputs
    A = torch.randn(777, 200, generator=torch.Generator().manual_seed(1))
    B = torch.randn(777, 200, generator=torch.Generator().manual_seed(2))
    C2 = torch.empty(200, 200, device=DEV)
    note("cross fp32 777x200")
    K.kronq_accumulate_cross(A.to(DEV), B.to(DEV), C2)
    torch.cuda.synchronize()
    assert rel_frob(to_np(C2), O.cross_covariance(A.numpy(), B.numpy())) < 1e-4
    # A = B: the covariance
    H = torch.empty(d, d, device=DEV)
    note("cross of X with itself vs covariance")
    K.kronq_accumulate_cross(Xd, Xd, C)
    K.kronq_accumulate_cov(Xd, H)
    torch.cuda.synchronize()
    assert rel_frob(to_np(C), to_np(H)) < 1e-5


# ------------------------------------------------------------------------------ BiIP of D
@pytest.mark.parametrize("d,flags", [(256, K.RESCALE_IN | K.ROT_IN), (28 * 16, K.RESCALE_IN | K.ROT_IN),
                                     (1024, K.ROT_IN), (512, K.RESCALE_IN)])
def test_rotate_drift(d, flags):
    spec, X, dX = tokens(d, 3 * d, 40 + d)
    h = as32(O.covariance(oracle_view(X)))
    D = as32(O.cross_covariance(oracle_view(dX), oracle_view(X)))
    W = synth.gen_matrix(synth.small_spec(64, d, 16, seed=d).w)
    ri = synth.rotation_params(d, 5, "in")
    ref = O.biip_forward(oracle_view(W), h, None, rot_oracle(ri), None, flags, D=D)
    sx = f32(ref["sx"])
    rin = rot_device(ri)
    Dd = f32(D)
    note(f"rotate drift d={d} flags={flags}")
    K.kronq_rotate_drift(Dd, sx, rin.sign, rin.q28, flags)
    torch.cuda.synchronize()
    assert rel_frob(to_np(Dd), ref["D"]) < TOL


# ------------------------------------------------------------------------------ P
@pytest.mark.parametrize("d,alpha", [(128, 1.0), (300, 1.0), (640, 0.25), (1000, 1.0),
                                     (2112, 1.0)])
def test_gptaq_correction(d, alpha):
    _, X, dX = tokens(d, 3 * d, d + 3)
    U = as32(O.inverse_cholesky_factor(O.damp(as32(O.covariance(oracle_view(X))))))
    D = as32(O.cross_covariance(oracle_view(dX), oracle_view(X)))
    P = torch.full((d, d), float("nan"), device=DEV)
    note(f"gptaq correction d={d} alpha={alpha}")
    K.kronq_gptaq_correction(f32(D), f32(U), P, alpha)
    torch.cuda.synchronize()
    p = to_np(P)
    assert np.all(np.tril(p) == 0.0)
    assert rel_frob(p, O.gptaq_correction(D, U, alpha)) < TOL


# ------------------------------------------------------------------------------ sweeps
def _sweep(W32, U32, bits, group=128, P32=None):
    d_out, d_in = W32.shape
    W = f32(W32)
    codes = torch.empty(d_out, d_in, dtype=torch.uint8, device=DEV)
    scales = torch.empty(d_out, d_in // group, device=DEV)
    zeros = torch.empty(d_out, d_in // group, device=DEV)
    err = torch.empty(d_out, d_in, device=DEV)
    W_hat = torch.empty(d_out, d_in, device=DEV)
    if P32 is None:
        K.kronq_obs_quantize_layer(W, f32(U32), bits, codes, scales, zeros, err, W_hat,
                                   group=group)
    else:
        K.kronq_obs_quantize_layer_drift(W, f32(U32), f32(P32), bits, codes, scales, zeros, err,
                                         W_hat, group=group)
    torch.cuda.synchronize()
    return dict(W=to_np(W), codes=to_np(codes), scales=to_np(scales), zeros=to_np(zeros),
                err=to_np(err), w_hat=to_np(W_hat))


def _agree(g, ref):
    same = g["codes"] == ref["codes"]
    agree = float(np.mean(same))
    print(f"code agreement {agree:.6f}")
    assert agree >= 0.995, agree
    rows = np.all(same, axis=1)  # rows whose codes all agree follow the same path
    assert rows.mean() > 0.5
    assert rel_frob(g["w_hat"][rows], ref["w_hat"][rows]) < TOL
    assert rel_frob(g["err"][rows], ref["err"][rows]) < TOL
    assert rel_frob(g["scales"], ref["scales"]) < TOL


@pytest.mark.parametrize("d_out,d_in,bits,group", [(200, 384, 4, 128), (130, 512, 2, 128),
                                                  (96, 768, 3, 256), (64, 768, 2, 768)])
def test_obs_drift(d_out, d_in, bits, group):
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=d_out + 1).w).float().numpy()
    U, D, P = hd_u_d(d_in, d_in + 9)
    note(f"obs drift {d_out}x{d_in} bits={bits} group={group}")
    g = _sweep(W, U, bits, group, P)
    ref = O.obs_blocked(W.astype(np.float64), U, bits, group, 128, P=P)
    _agree(g, ref)


def test_obs_drift_with_zero_p_is_the_plain_sweep():
    # the two entry points batch the trailing updates differently (the plain sweep applies a
    # block's pending updates inside its own launch), so they agree up to the fp32 summation
    # order: the same codes up to near ties, and the floats to rounding
    d_out, d_in = 100, 512
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=3).w).float().numpy()
    U, _, _ = hd_u_d(d_in, 4)
    note("obs drift with P = 0")
    a = _sweep(W, U, 3, 128, np.zeros((d_in, d_in)))
    b = _sweep(W, U, 3, 128)
    assert np.mean(a["codes"] == b["codes"]) >= 0.995
    for k in ("scales", "W", "err"):
        assert rel_frob(a[k], b[k]) < 1e-5, k


# ------------------------------------------------------------------------------ wide groups
@pytest.mark.parametrize("bits,group", [(4, 768), (3, 256), (2, 384)])
def test_wide_group_rtn_bit_exact(bits, group):
    d_out, d_in = 150, 768
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=bits).w).float().numpy()
    U = O.inverse_cholesky_factor(O.damp(np.eye(d_in))).astype(np.float32)
    note(f"obs RTN group={group} bits={bits}")
    g = _sweep(W, U, bits, group)
    ref = O.obs_blocked(W.astype(np.float64), U.astype(np.float64), bits, group, 128)
    assert np.array_equal(g["codes"], ref["codes"])
    assert np.array_equal(g["scales"], ref["scales"].astype(np.float32))
    assert np.array_equal(g["zeros"], ref["zeros"])


@pytest.mark.parametrize("d_out,d_in,bits,group", [(200, 768, 3, 768), (130, 1024, 2, 512),
                                                  (96, 768, 4, 384), (64, 640, 3, 640)])
def test_wide_group_general(d_out, d_in, bits, group):
    W = synth.gen_matrix(synth.small_spec(d_out, d_in, 16, seed=d_out + 2).w).float().numpy()
    _, X, _ = tokens(d_in, 2 * d_in, d_in + 5)
    U = as32(O.inverse_cholesky_factor(O.damp(as32(O.covariance(oracle_view(X))))))
    note(f"obs general group={group} {d_out}x{d_in} bits={bits}")
    g = _sweep(W, U, bits, group)
    ref = O.obs_blocked(W.astype(np.float64), U, bits, group, 128)
    _agree(g, ref)


# ------------------------------------------------------------------------------ whole layer
def _layer_case(spec, alpha, overlap, group=128):
    X = synth.gen_matrix(spec.x, DEV)
    G = synth.gen_matrix(spec.g, DEV)
    W0 = synth.gen_matrix(spec.w, DEV)
    dX = synth.gen_drift(spec, DEV, X=X)
    ri = synth.rotation_params(spec.d_in, spec.seed, spec.name + ":in")
    ro = synth.rotation_params(spec.d_out, spec.seed, spec.name + ":out")
    st = L.LayerState.allocate(spec.d_out, spec.d_in, spec.n_tokens, DEV, keep_err=True,
                               group=group, drift=True)
    note(f"layer drift {spec.d_out}x{spec.d_in} N={spec.n_tokens} overlap={overlap}")
    L.quantize_layer(st, X, G, W0, rot_device(ri), rot_device(ro), spec.bits, spec.damp,
                     overlap=overlap, dX=dX, alpha=alpha)
    L.check(st)
    return st, (X, G, W0, dX), (ri, ro)


@pytest.mark.parametrize("group", [128, 512])
def test_layer_with_drift_end_to_end(group):
    spec = synth.small_spec(448, 512, 3000, bits=3, seed=17)
    alpha = 0.5
    st, (X, G, W0, dX), (ri, ro) = _layer_case(spec, alpha, True, group)
    torch.cuda.synchronize()
    hx, hg = O.covariance(oracle_view(X.cpu())), O.covariance(oracle_view(G.cpu()))
    D = O.cross_covariance(oracle_view(dX.cpu()), oracle_view(X.cpu()))
    b = O.biip_forward(oracle_view(W0.cpu()), hx, hg, rot_oracle(ri), rot_oracle(ro), K.BIIP, D=D)
    U = O.inverse_cholesky_factor(O.damp(b["HX"], spec.damp))
    P = O.gptaq_correction(b["D"], U, alpha)
    q = O.obs_blocked(b["W"], U, spec.bits, group, 128, P=P)
    assert rel_frob(to_np(st.D), b["D"]) < TOL
    assert rel_frob(to_np(st.U), U) < TOL
    assert rel_frob(to_np(st.P), P) < TOL
    agree = float(np.mean(to_np(st.codes) == q["codes"]))
    print(f"group {group}: code agreement {agree:.6f}")
    assert agree >= 0.995


def test_layer_with_drift_overlap_matches_serial():
    spec = synth.small_spec(448, 256, 2000, bits=2, seed=23)
    outs = []
    for overlap in (False, True):
        st, _, _ = _layer_case(spec, 1.0, overlap)
        torch.cuda.synchronize()
        outs.append([to_np(t) for t in (st.codes, st.W, st.U, st.P, st.D, st.sx, st.sg)])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)
