"""Parity of the inference-side path (packed codes, online rotations around the packed-code
matvec) through the C ABI against the float64 oracle.

Codes, scales and zeros are seeded random values of the sweep's output format (the matvec does
not depend on where they came from), rotation draws come from the generator. Tolerance 1e-4
relative (fp32 arithmetic on exact inputs); the packed format is checked bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import DEV, note, rel_frob, rot_device, rot_oracle, to_np
from paper_2607_07964_amd import kronq as K
from paper_2607_07964_amd import layer as L

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _lib():
    K.load()
    assert torch.cuda.is_available(), "GPU tests need an MI355X"


def quantised_layer(d_out, d_in, bits, group, seed):
    r = np.random.default_rng(seed)
    codes = r.integers(0, 2 ** bits, size=(d_out, d_in)).astype(np.uint8)
    ng = d_in // group
    scales = (np.exp(0.3 * r.standard_normal((d_out, ng))) * 0.01).astype(np.float32)
    zeros = r.integers(0, 2 ** bits, size=(d_out, ng)).astype(np.float32)
    sx = np.exp(0.2 * r.standard_normal(d_in)).astype(np.float32)
    sg = np.exp(0.2 * r.standard_normal(d_out)).astype(np.float32)
    return codes, scales, zeros, sx, sg


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_pack_codes_bit_exact(bits):
    d_out, d_in = 37, 384
    codes = np.random.default_rng(bits).integers(0, 2 ** bits, size=(d_out, d_in)).astype(np.uint8)
    note(f"pack codes bits={bits}")
    packed = K.kronq_pack_codes(torch.from_numpy(codes).to(DEV), bits)
    torch.cuda.synchronize()
    ref = O.pack_codes(codes, bits)
    assert np.array_equal(to_np(packed).view(np.uint32), ref)


def _run(codes, scales, zeros, sx, sg, bits, group, ri, ro, flags, x):
    d_out, d_in = codes.shape
    rin, rout = rot_device(ri), rot_device(ro)
    mul_in = K.kronq_online_factors(torch.from_numpy(sx).to(DEV),
                                    rin.sign if flags & K.ROT_IN else None, d_in)
    mul_out = K.kronq_online_factors(torch.from_numpy(sg).to(DEV),
                                     rout.sign if flags & K.ROT_OUT else None, d_out)
    packed = K.kronq_pack_codes(torch.from_numpy(codes).to(DEV), bits)
    y = K.kronq_online_matvec(packed, torch.from_numpy(scales).to(DEV),
                              torch.from_numpy(zeros).to(DEV), bits, group, d_in, mul_in, mul_out,
                              rin.q28, rout.q28, x, flags=flags)
    torch.cuda.synchronize()
    return to_np(y)


def _ref(codes, scales, zeros, sx, sg, group, ri, ro, flags, x64):
    d_out, d_in = codes.shape
    V = O.rht_matrix(d_in, *rot_oracle(ri)) if flags & K.ROT_IN else np.eye(d_in)
    U = O.rht_matrix(d_out, *rot_oracle(ro)) if flags & K.ROT_OUT else np.eye(d_out)
    Wr = O.dequantize(codes, scales.astype(np.float64), zeros.astype(np.float64), group)
    return O.online_matvec(Wr, sx.astype(np.float64), sg.astype(np.float64), V, U, x64.T).T


@pytest.mark.parametrize("d_out,d_in,bits,group,batch,flags,xdt", [
    (448, 256, 4, 128, 1, K.BIIP, torch.bfloat16),
    (512, 896, 2, 128, 2, K.BIIP, torch.float32),
    (256, 1024, 3, 1024, 3, K.BIIP, torch.bfloat16),
    (448, 512, 8, 256, 4, K.BIIP, torch.float32),
    (300, 256, 4, 128, 1, K.ROT_IN | K.RESCALE_IN, torch.float32),
    (448, 384, 2, 384, 2, K.ROT_OUT | K.RESCALE_OUT, torch.bfloat16),
    (200, 640, 4, 128, 1, 0, torch.float32),
    # one vector: the persistent GEMV, with the input transform inside (power-of-two or no
    # input rotation, d_in <= 8192) or after a separate transform (larger d_in);
    # several tiles per workgroup, several tiles per row, a ragged last row block
    (9000, 512, 2, 128, 1, K.ROT_IN | K.RESCALE_IN | K.RESCALE_OUT, torch.bfloat16),
    (14336, 256, 4, 128, 1, K.BIIP, torch.float32),
    (256, 896, 2, 128, 1, K.BIIP, torch.bfloat16),
    (64, 16384, 4, 128, 1, K.BIIP, torch.float32),
    (1024, 8192, 2, 256, 1, K.BIIP, torch.float32),
    (130, 1024, 4, 1024, 1, K.RESCALE_IN | K.RESCALE_OUT, torch.bfloat16),
    # one vector with a 28 * m input rotation (the separate input transform, then the persistent
    # GEMV on its digits): m = 64, 256 without an output rotation, 128 with a 28 * m output, and
    # 1024 (the largest input one vector allows)
    (300, 1792, 4, 256, 1, K.ROT_IN | K.RESCALE_IN | K.RESCALE_OUT, torch.float32),
    (130, 7168, 2, 1792, 1, K.ROT_IN | K.RESCALE_IN, torch.bfloat16),
    (896, 3584, 2, 128, 1, K.BIIP, torch.bfloat16),
    (64, 28672, 4, 128, 1, K.BIIP, torch.float32),
])
def test_online_matvec(d_out, d_in, bits, group, batch, flags, xdt):
    codes, scales, zeros, sx, sg = quantised_layer(d_out, d_in, bits, group, d_out + d_in)
    ri = synth.rotation_params(d_in, 3, "in") if flags & K.ROT_IN else synth.Rot(d_in, np.ones(d_in, np.int8), None, None)
    ro = synth.rotation_params(d_out, 3, "out") if flags & K.ROT_OUT else synth.Rot(d_out, np.ones(d_out, np.int8), None, None)
    x = torch.randn(batch, d_in, generator=torch.Generator().manual_seed(batch)).to(xdt)
    note(f"online matvec {d_out}x{d_in} bits={bits} group={group} batch={batch} flags={flags}")
    y = _run(codes, scales, zeros, sx, sg, bits, group, ri, ro, flags, x.to(DEV))
    ref = _ref(codes, scales, zeros, sx, sg, group, ri, ro, flags, x.float().numpy().astype(np.float64))
    assert rel_frob(y, ref) < TOL


def test_online_matvec_serves_the_quantised_layer():
    """After the GPU sweep, the online matvec on its packed codes equals the dense product with
    the reverted dequantised weights (both on the GPU): the format and the transforms agree."""
    spec = synth.small_spec(448, 512, 2000, bits=3, seed=29)
    X = synth.gen_matrix(spec.x, DEV)
    G = synth.gen_matrix(spec.g, DEV)
    W0 = synth.gen_matrix(spec.w, DEV)
    ri = synth.rotation_params(spec.d_in, spec.seed, spec.name + ":in")
    ro = synth.rotation_params(spec.d_out, spec.seed, spec.name + ":out")
    rin, rout = rot_device(ri), rot_device(ro)
    st = L.LayerState.allocate(spec.d_out, spec.d_in, spec.n_tokens, DEV)
    note("online matvec of a GPU-quantised layer")
    L.quantize_layer(st, X, G, W0, rin, rout, spec.bits, spec.damp)
    L.check(st)
    Wrev = L.revert(st, rin, rout)
    mul_in = K.kronq_online_factors(st.sx, rin.sign, spec.d_in)
    mul_out = K.kronq_online_factors(st.sg, rout.sign, spec.d_out)
    packed = K.kronq_pack_codes(st.codes, spec.bits)
    x = torch.randn(2, spec.d_in, generator=torch.Generator().manual_seed(0)).to(DEV)
    y = K.kronq_online_matvec(packed, st.scales, st.zeros, spec.bits, 128, spec.d_in, mul_in,
                              mul_out, rin.q28, rout.q28, x)
    dense = x @ Wrev.T
    torch.cuda.synchronize()
    assert rel_frob(to_np(y), to_np(dense)) < 1e-4


@pytest.mark.slow
@pytest.mark.parametrize("d_out,d_in,bits", [(4096, 4096, 4), (4096, 14336, 2), (28672, 8192, 2)])
def test_online_matvec_full_shape(d_out, d_in, bits):
    """The LLaMA-3-8B q_proj, down_proj and LLaMA-3-70B up_proj shapes (bench configurations);
    the oracle forms W_hat' and the input transform densely, and the output transform on sampled
    rows (a column of U^T is a signed row of the transposed factor)."""
    codes, scales, zeros, sx, sg = quantised_layer(d_out, d_in, bits, 128, 7)
    ri = synth.rotation_params(d_in, 5, "in")
    ro = synth.rotation_params(d_out, 5, "out")
    x = torch.randn(1, d_in, generator=torch.Generator().manual_seed(1)).to(torch.bfloat16)
    note(f"online matvec full shape {d_out}x{d_in} bits={bits}")
    y = _run(codes, scales, zeros, sx, sg, bits, 128, ri, ro, K.BIIP, x.to(DEV))[0]
    x64 = x.float().numpy().astype(np.float64)[0]
    sgn_in, q_in = rot_oracle(ri)
    xr = O.rht_rows(d_in, sgn_in, q_in, np.arange(d_in)) @ (x64 / sx.astype(np.float64))
    Wr = O.dequantize(codes, scales.astype(np.float64), zeros.astype(np.float64), 128)
    yr = Wr @ xr
    del Wr
    rows = np.sort(np.random.default_rng(2).choice(d_out, 24, replace=False))
    sgn_out, q_out = rot_oracle(ro)
    # U^T = diag(sign) (Q^T (x) H) / sqrt(m): row i of U^T is sign_i times row i of the unsigned
    # transposed factor
    qt = None if q_out is None else np.ascontiguousarray(q_out.T)
    Ut_rows = O.rht_rows(d_out, np.ones(d_out), qt, rows) * sgn_out[rows, None]
    ref = (Ut_rows @ yr) / sg.astype(np.float64)[rows]
    assert rel_frob(y[rows], ref) < TOL
