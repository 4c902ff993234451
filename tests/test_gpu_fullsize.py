"""Parity at full size, in the launch configuration bench.py times (the LLaMA-3-8B q_proj layer:
W 4096 x 4096, N = 262144 tokens, 4-bit, group 128).

The oracle cannot redo a 4.4e12-flop covariance in seconds, so it checks what it can compute
one by one (sampled covariance entries, exact traces, rows of the solve, which are independent
given U) and stage-isolated steps fed with oracle-made inputs at the real shapes.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import DEV, note, oracle_view, rel_frob, rot_device, rot_oracle, to_np
from paper_2607_07964_amd import kronq as K
from paper_2607_07964_amd import layer as L

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
TOL = 1e-3


@pytest.fixture(scope="module")
def q_proj():
    K.load()
    spec = synth.workload(2)
    note("full-size inputs: q_proj 4096x4096, N=262144")
    X = synth.gen_matrix(spec.x, DEV)
    G = synth.gen_matrix(spec.g, DEV)
    W0 = synth.gen_matrix(spec.w, DEV)
    ri = synth.rotation_params(spec.d_in, spec.seed, spec.name + ":in")
    ro = synth.rotation_params(spec.d_out, spec.seed, spec.name + ":out")
    return spec, X, G, W0, ri, ro


def test_covariance_sampled_entries_and_traces(q_proj):
    spec, X, G, W0, ri, ro = q_proj
    d, n = spec.d_in, spec.n_tokens
    for name, A, mspec in (("X", X, spec.x), ("G", G, spec.g)):
        H = torch.empty(d, d, device=DEV)
        note(f"full-size covariance of {name}")
        K.kronq_accumulate_cov(A, H)
        tr = K.kronq_traces(H, H)
        torch.cuda.synchronize()
        h = to_np(H)
        assert np.array_equal(h, h.T)
        rng = np.random.default_rng(7)
        idx = rng.choice(d, 24, replace=False)
        pairs = [(idx[k], idx[(k * 7 + 3) % 24]) for k in range(24)] + [(i, i) for i in idx[:6]]
        cols = sorted(set(int(c) for p in pairs for c in p))
        sub = O.as_f64(oracle_view(synth.gen_columns(mspec, cols)))
        pos = {c: k for k, c in enumerate(cols)}
        ref = np.array([sub[:, pos[i]] @ sub[:, pos[j]] for i, j in pairs])
        got = np.array([h[i, j] for i, j in pairs])
        scale = np.sqrt([h[i, i] * h[j, j] for i, j in pairs])
        assert np.max(np.abs(got - ref) / scale) < TOL
        # exact trace: sum of squares of every token in float64, over CPU copies of the
        # generator's tensor (the generator is bit-identical on CPU and GPU)
        acc = 0.0
        for t0 in range(0, n, 16384):
            blk = O.as_f64(oracle_view(A[t0:t0 + 16384].cpu()))
            acc += float(np.sum(blk * blk))
        assert abs(float(tr[0].item()) / acc - 1.0) < TOL


@pytest.fixture(scope="module")
def rotated(q_proj):
    """Stage-isolated BiIP at full shape: oracle covariances of the first 4096 tokens as H."""
    spec, X, G, W0, ri, ro = q_proj
    nsub = 4096
    hx = O.covariance(oracle_view(synth.gen_matrix(spec.x, "cpu", rows=(0, nsub))))
    hg = O.covariance(oracle_view(synth.gen_matrix(spec.g, "cpu", rows=(0, nsub))))
    hx32, hg32 = hx.astype(np.float32), hg.astype(np.float32)
    ref = O.biip_forward(oracle_view(W0.cpu()), hx32.astype(np.float64), hg32.astype(np.float64),
                         rot_oracle(ri), rot_oracle(ro))
    return hx32, hg32, ref


def test_rotation_full_shape(q_proj, rotated):
    spec, X, G, W0, ri, ro = q_proj
    hx32, hg32, ref = rotated
    HX = torch.from_numpy(hx32).to(DEV)
    HG = torch.from_numpy(hg32).to(DEV)
    Wd = torch.empty(spec.d_out, spec.d_in, device=DEV)
    sx = torch.empty(spec.d_in, device=DEV)
    sg = torch.empty(spec.d_out, device=DEV)
    rin, rout = rot_device(ri), rot_device(ro)
    note("full-size rotate")
    K.kronq_rotate(W0, Wd, HX, HG, rin.sign, rout.sign, rin.q28, rout.q28, sx, sg, K.BIIP)
    torch.cuda.synchronize()
    assert rel_frob(to_np(Wd), ref["W"]) < TOL
    assert rel_frob(to_np(HX), ref["HX"]) < TOL
    assert rel_frob(to_np(HG), ref["HG"]) < TOL


def test_factor_and_sweep_full_shape(q_proj, rotated):
    spec, X, G, W0, ri, ro = q_proj
    _, _, ref = rotated
    h = np.ascontiguousarray(ref["HX"], dtype=np.float32)
    H = torch.from_numpy(h).to(DEV)
    U = torch.empty_like(H)
    note("full-size cholesky_inv")
    info = K.kronq_cholesky_inv(H, U, spec.damp)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    Uo = O.inverse_cholesky_factor(O.damp(h.astype(np.float64), spec.damp))
    assert rel_frob(to_np(U), Uo) < TOL
    # the sweep on the oracle's rotated W and factor; rows are independent given U
    W32 = np.ascontiguousarray(ref["W"], dtype=np.float32)
    U32 = np.ascontiguousarray(Uo, dtype=np.float32)
    Wd = torch.from_numpy(W32).to(DEV)
    codes = torch.empty(spec.d_out, spec.d_in, dtype=torch.uint8, device=DEV)
    scales = torch.empty(spec.d_out, spec.d_in // 128, device=DEV)
    zeros = torch.empty_like(scales)
    err = torch.empty(spec.d_out, spec.d_in, device=DEV)
    note("full-size obs sweep")
    K.kronq_obs_quantize_layer(Wd, torch.from_numpy(U32).to(DEV), spec.bits, codes, scales, zeros,
                               err)
    torch.cuda.synchronize()
    rows = np.random.default_rng(3).choice(spec.d_out, 48, replace=False)
    q = O.obs_blocked(W32[rows].astype(np.float64), U32.astype(np.float64), spec.bits, 128, 128)
    agree = float(np.mean(to_np(codes)[rows] == q["codes"]))
    print(f"full-size sampled-row code agreement {agree:.6f}")
    assert agree >= 0.995
    # dW' = E U holds for every row at any size (the LDL loss identity rests on it)
    r2 = rows[:8]
    dW = W32[r2].astype(np.float64) - to_np(Wd)[r2].astype(np.float64)
    EU = to_np(err)[r2].astype(np.float64) @ U32.astype(np.float64)
    assert rel_frob(EU, dW) < TOL


def test_layer_pipeline_full_size(q_proj):
    """The bench's launch sequence; outputs checked by properties that hold at any size."""
    spec, X, G, W0, ri, ro = q_proj
    rin, rout = rot_device(ri), rot_device(ro)
    st = L.LayerState.allocate(spec.d_out, spec.d_in, spec.n_tokens, DEV, keep_err=True)
    note("full-size layer pipeline")
    L.quantize_layer(st, X, G, W0, rin, rout, spec.bits, spec.damp)
    L.check(st)
    torch.cuda.synchronize()
    codes = to_np(st.codes)
    assert codes.max() <= 2 ** spec.bits - 1
    pre, post = to_np(st.tr_pre), to_np(st.tr_post)
    # post-BiIP trace of H_X has the closed form sum_j sqrt(h_jj a_j) (rotation keeps traces)
    assert np.all(np.isfinite(post)) and post[0] > 0 and post[1] > 0
    u = to_np(st.U)
    assert np.all(np.tril(u, -1) == 0) and np.all(np.diag(u) > 0)
    rows = [0, 1, 2047, 4095]
    w_hat = to_np(st.W)[rows]
    s = np.repeat(to_np(st.scales)[rows], 128, axis=1)
    z = np.repeat(to_np(st.zeros)[rows], 128, axis=1)
    np.testing.assert_allclose(w_hat, (s.astype(np.float64) * (codes[rows] - z)).astype(np.float32),
                               rtol=0, atol=0)
