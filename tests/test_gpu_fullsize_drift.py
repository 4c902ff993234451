"""Parity of the drift-corrected path at full size, in the launch configuration bench.py times
with --drift: the LLaMA-3-8B q_proj (W 4096 x 4096) and the LLaMA-3-70B up_proj
(W 28672 x 8192), N = 262144 tokens, with the synthetic input drift.

As for the plain path, the oracle checks what it can compute one by one: sampled entries of the
drift statistic over all tokens, sampled entries of its transform, rows of P and of the sweep
(rows are independent given U and P), and properties of the whole pipeline.
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
WORKLOADS = {"q_proj": 2, "up_proj_70b": 4}
ALPHA = 1.0


@pytest.fixture(scope="module", params=list(WORKLOADS))
def wl(request):
    K.load()
    spec = synth.workload(WORKLOADS[request.param])
    note(f"full-size drift inputs: {spec.name} {spec.d_out}x{spec.d_in}, N={spec.n_tokens}")
    X = synth.gen_matrix(spec.x, DEV)
    dX = synth.gen_drift(spec, DEV, X=X)
    ri = synth.rotation_params(spec.d_in, spec.seed, spec.name + ":in")
    yield spec, X, dX, ri
    del X, dX
    torch.cuda.empty_cache()


def test_drift_statistic_sampled_entries(wl):
    spec, X, dX, ri = wl
    d = spec.d_in
    C = torch.empty(d, d, device=DEV)
    note(f"full-size drift statistic d={d}")
    K.kronq_accumulate_cross(dX, X, C)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    idx = rng.choice(d, 20, replace=False)
    pairs = [(idx[k], idx[(k * 7 + 3) % 20]) for k in range(20)] + [(i, i) for i in idx[:6]]
    got = np.array([C[i, j].item() for i, j in pairs])
    cols = sorted(set(int(c) for p in pairs for c in p))
    pos = {c: k for k, c in enumerate(cols)}
    a = O.as_f64(oracle_view(synth.gen_drift_columns(spec, cols)))
    b = O.as_f64(oracle_view(synth.gen_columns(spec.x, cols)))
    ref = np.array([a[:, pos[i]] @ b[:, pos[j]] for i, j in pairs])
    scale = np.sqrt([(a[:, pos[i]] @ a[:, pos[i]]) * (b[:, pos[j]] @ b[:, pos[j]])
                     for i, j in pairs])
    assert np.max(np.abs(got - ref) / scale) < TOL


def test_drift_biip_sampled(wl):
    """D = dA^T A over the first 64 tokens (rank 64), so an entry of V S^-1 D S^-1 V^T is the
    dot product of rows of V S^-1 dA^T and V S^-1 A^T."""
    spec, X, dX, ri = wl
    d, ntok = spec.d_in, 64
    a = O.as_f64(oracle_view(synth.gen_matrix(spec.x, "cpu", rows=(0, ntok))))
    da = O.as_f64(oracle_view(synth.gen_drift(spec, "cpu", rows=(0, ntok))))
    D = torch.from_numpy(O.cross_covariance(da, a).astype(np.float32)).to(DEV)
    sx = np.exp(0.3 * np.random.default_rng(2).standard_normal(d)).astype(np.float32)
    rin = rot_device(ri)
    note(f"full-size drift BiIP d={d}")
    K.kronq_rotate_drift(D, torch.from_numpy(sx).to(DEV), rin.sign, rin.q28)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(3).choice(d, 12, replace=False))
    sgn, q = rot_oracle(ri)
    V = O.rht_rows(d, sgn, q, rows) / sx.astype(np.float64)[None, :]
    ref = (V @ da.T) @ (V @ a.T).T
    got = to_np(D[rows][:, rows]).astype(np.float64)
    assert rel_frob(got, ref) < TOL


def test_correction_and_drift_sweep_rows(wl):
    """P at the real d from an oracle-made U and D (tokens: 4096 or 2 d), checked on sampled rows;
    then the drift sweep with the oracle's U and P on 48 sampled rows of W."""
    spec, X, dX, ri = wl
    d = spec.d_in
    ntok = 4096 if d <= 4096 else 2 * d
    xs = oracle_view(synth.gen_matrix(spec.x, "cpu", rows=(0, ntok)))
    dxs = oracle_view(synth.gen_drift(spec, "cpu", rows=(0, ntok)))
    h = O.covariance(xs).astype(np.float32).astype(np.float64)
    U32 = np.ascontiguousarray(O.inverse_cholesky_factor(O.damp(h, spec.damp)), dtype=np.float32)
    D32 = np.ascontiguousarray(O.cross_covariance(dxs, xs), dtype=np.float32)
    U64, D64 = U32.astype(np.float64), D32.astype(np.float64)
    Ud, Dd = torch.from_numpy(U32).to(DEV), torch.from_numpy(D32).to(DEV)
    P = torch.empty(d, d, device=DEV)
    note(f"full-size gptaq correction d={d}")
    K.kronq_gptaq_correction(Dd, Ud, P, ALPHA)
    torch.cuda.synchronize()
    prow = np.sort(np.random.default_rng(4).choice(d, 16, replace=False))
    pref = O.gptaq_correction(D64, U64, ALPHA, prow)
    assert rel_frob(to_np(P[prow]), pref) < TOL
    assert float(torch.tril(P).abs().max().item()) == 0.0
    del Dd, P
    # the sweep, with the oracle's P (rounded to fp32) as its input
    P32 = np.ascontiguousarray(O.gptaq_correction(D64, U64, ALPHA), dtype=np.float32)
    W0 = synth.gen_matrix(spec.w)
    W32 = np.ascontiguousarray(O.as_f64(oracle_view(W0)), dtype=np.float32)
    Wd = torch.from_numpy(W32).to(DEV)
    codes = torch.empty(spec.d_out, d, dtype=torch.uint8, device=DEV)
    scales = torch.empty(spec.d_out, d // 128, device=DEV)
    zeros = torch.empty_like(scales)
    note("full-size drift sweep")
    K.kronq_obs_quantize_layer_drift(Wd, Ud, torch.from_numpy(P32).to(DEV), spec.bits, codes,
                                     scales, zeros)
    torch.cuda.synchronize()
    rows = np.random.default_rng(3).choice(spec.d_out, 48, replace=False)
    q = O.obs_blocked(W32[rows].astype(np.float64), U64, spec.bits, 128, 128,
                      P=P32.astype(np.float64))
    agree = float(np.mean(to_np(codes[rows]) == q["codes"]))
    print(f"{spec.name}: full-size drift sweep sampled-row code agreement {agree:.6f}")
    assert agree >= 0.995


def test_drift_pipeline_full_size(wl):
    """The bench's launch sequence with --drift; outputs checked by properties that hold at any
    size."""
    spec, X, dX, ri = wl
    G = synth.gen_matrix(spec.g, DEV)
    W0 = synth.gen_matrix(spec.w, DEV)
    ro = synth.rotation_params(spec.d_out, spec.seed, spec.name + ":out")
    st = L.LayerState.allocate(spec.d_out, spec.d_in, spec.n_tokens, DEV, drift=True)
    note(f"full-size drift pipeline {spec.name}")
    L.quantize_layer(st, X, G, W0, rot_device(ri), rot_device(ro), spec.bits, spec.damp, dX=dX,
                     alpha=ALPHA)
    L.check(st)
    torch.cuda.synchronize()
    assert int(st.codes.max().item()) <= 2 ** spec.bits - 1
    assert bool(torch.isfinite(st.P).all()) and bool(torch.isfinite(st.W).all())
    assert float(torch.tril(st.P).abs().max().item()) == 0.0
    # the sweep leaves W at its dequantised values: scale * (code - zero) on sampled rows
    rows = [0, spec.d_out // 3, spec.d_out - 1]
    w = to_np(st.W[rows]).astype(np.float64)
    c = to_np(st.codes[rows]).astype(np.float64)
    s = np.repeat(to_np(st.scales[rows]).astype(np.float64), 128, axis=1)
    z = np.repeat(to_np(st.zeros[rows]).astype(np.float64), 128, axis=1)
    np.testing.assert_allclose(w, s * (c - z), rtol=1e-6, atol=0)
