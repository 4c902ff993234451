"""The C-ABI library: loads, exports every declared symbol, host-side logic (CPU only).

No call here launches GPU work: only symbol lookup, workspace queries, argument checks that fail
before any HIP call, and the host-only bit allocation.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
from paper_2607_07964_amd import kronq as K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kronq.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kronq_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = K.load()
    names = declared_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(K.EXPORTS)


def test_version_and_workspace_queries():
    assert K.kronq_version() >= 100
    assert K.kronq_workspace_bytes(K.OP_COV, 0, 4096, 262144) > 0
    assert K.kronq_workspace_bytes(K.OP_CHOL, 0, 4096, 0) >= 2 * 4096 * 4096 * 4
    assert K.kronq_workspace_bytes(K.OP_OBS, 4096, 4096, 0) > 0
    assert K.kronq_workspace_bytes(K.OP_CROSS, 0, 4096, 262144) >= 256 * 256 * 256 * 4
    assert K.kronq_workspace_bytes(K.OP_ROTATE_DRIFT, 0, 4096, 0) >= 4096 * 4
    assert K.kronq_workspace_bytes(K.OP_GPTAQ, 0, 4096, 0) >= 4096 * 4096 * 4
    # split U^T (and -P^T with the drift correction), two bf16 planes each; without the drift
    # correction U^T is kept row-major and in MFMA-fragment order
    assert K.kronq_workspace_bytes(K.OP_OBS_DRIFT, 4096, 4096, 0) >= 2 * 2 * 4096 * 4096 * 2
    assert K.kronq_workspace_bytes(K.OP_OBS, 4096, 4096, 0) >= 2 * 2 * 4096 * 4096 * 2
    assert K.kronq_workspace_bytes(99, 1, 1, 1) == 0
    assert K.kronq_workspace_bytes(K.OP_COV, 0, -1, 10) == 0


def _err(rc):
    return rc, K.load().kronq_last_error().decode()


def test_argument_checks_fail_before_any_launch():
    lib = K.load()
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: checks fail first
    # unsupported group / block / bits
    rc, msg = _err(lib.kronq_obs_quantize_layer(fake, 8, 256, 256, fake, 256, 4, 64, 128, fake,
                                                fake, fake, nul, nul, nul, 0, nul))
    assert rc == -6 and "group" in msg
    rc, _ = _err(lib.kronq_obs_quantize_layer(fake, 8, 256, 256, fake, 256, 9, 128, 128, fake,
                                              fake, fake, nul, nul, nul, 0, nul))
    assert rc == -6
    rc, _ = _err(lib.kronq_obs_quantize_layer(fake, 8, 256, 256, fake, 256, 4, 128, 64, fake,
                                              fake, fake, nul, nul, nul, 0, nul))
    assert rc == -6
    # bad dtype, null H
    rc, _ = _err(lib.kronq_accumulate_cov(fake, 7, 10, 8, 8, fake, 8, 1.0, 0.0, nul, 0, nul))
    assert rc == -1
    rc, _ = _err(lib.kronq_accumulate_cov(fake, 1, 10, 8, 8, nul, 8, 1.0, 0.0, nul, 0, nul))
    assert rc == -1
    # too small a workspace
    rc, msg = _err(lib.kronq_accumulate_cov(fake, 1, 1000, 64, 64, fake, 64, 1.0, 0.0, nul, 16,
                                            nul))
    assert rc == -5 and "workspace" in msg
    # rotation of a dimension that is neither 2^k nor 28 * 2^k
    ws = ctypes.c_void_p(1 << 30)
    rc, msg = _err(lib.kronq_rotate(fake, 2, 96, fake, 8, 96, 96, fake, 96, nul, 0, fake, nul,
                                    nul, nul, fake, fake, K.ROT_IN, ws, 1 << 30, nul))
    assert rc == -6 and "96" in msg
    # 28 * 2^k without the 28 x 28 factor
    rc, msg = _err(lib.kronq_rotate(fake, 2, 112, fake, 8, 112, 112, fake, 112, nul, 0, fake, nul,
                                    nul, nul, fake, fake, K.ROT_IN, ws, 1 << 30, nul))
    assert rc == -1 and "28" in msg
    # W_in rows not 16-byte aligned (bf16 with ldw_in % 8 != 0; a misaligned base pointer)
    rc, msg = _err(lib.kronq_rotate(fake, 1, 132, fake, 8, 128, 128, fake, 128, nul, 0, fake,
                                    nul, nul, nul, fake, fake, K.ROT_IN, ws, 1 << 30, nul))
    assert rc == -1 and "W_in" in msg
    odd = ctypes.c_void_p((1 << 20) + 8)
    rc, msg = _err(lib.kronq_rotate(odd, 2, 128, fake, 8, 128, 128, fake, 128, nul, 0, fake,
                                    nul, nul, nul, fake, fake, K.ROT_IN, ws, 1 << 30, nul))
    assert rc == -1 and "W_in" in msg
    # d_in not a multiple of the group
    rc, _ = _err(lib.kronq_obs_quantize_layer(fake, 8, 200, 200, fake, 200, 4, 128, 128, fake,
                                              fake, fake, nul, nul, nul, 0, nul))
    assert rc == -2
    # Cholesky output aliasing its input
    rc, _ = _err(lib.kronq_cholesky_inv(fake, 8, 8, 0.01, fake, 8, fake, ws, 1 << 30, nul))
    assert rc == -1
    # the sweep's workspace is checked also when the caller keeps the errors
    rc, msg = _err(lib.kronq_obs_quantize_layer(fake, 8, 256, 256, ctypes.c_void_p(1 << 21), 256,
                                                4, 128, 128, fake, fake, fake, fake, nul, nul, 16,
                                                nul))
    assert rc == -5 and "workspace" in msg


def test_drift_and_group_argument_checks():
    lib = K.load()
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    other = ctypes.c_void_p(1 << 21)
    ws = ctypes.c_void_p(1 << 30)
    # groups: multiples of 128 that divide d_in (any of them); others are unsupported
    rc, msg = _err(lib.kronq_obs_quantize_layer(fake, 8, 768, 768, other, 768, 3, 192, 128, fake,
                                                fake, fake, nul, nul, nul, 0, nul))
    assert rc == -6 and "group" in msg
    rc, msg = _err(lib.kronq_obs_quantize_layer(fake, 8, 768, 768, other, 768, 3, 512, 128, fake,
                                                fake, fake, nul, nul, nul, 0, nul))
    assert rc == -2
    # (a supported wide group gets past the group checks and stops at the workspace)
    rc, msg = _err(lib.kronq_obs_quantize_layer(fake, 8, 768, 768, other, 768, 3, 384, 128, fake,
                                                fake, fake, nul, nul, nul, 0, nul))
    assert rc == -5
    # the drift sweep needs P, and P must not alias W
    rc, msg = _err(lib.kronq_obs_quantize_layer_drift(fake, 8, 256, 256, other, 256, nul, 256, 3,
                                                      128, 128, fake, fake, fake, nul, nul, ws,
                                                      1 << 30, nul))
    assert rc == -1 and "P" in msg
    rc, msg = _err(lib.kronq_obs_quantize_layer_drift(fake, 8, 256, 256, other, 256, fake, 256, 3,
                                                      128, 128, fake, fake, fake, nul, nul, ws,
                                                      1 << 30, nul))
    assert rc == -1 and "alias" in msg
    # drift statistic: B missing, rows not 16-byte aligned
    rc, _ = _err(lib.kronq_accumulate_cross(fake, nul, 1, 100, 64, 64, fake, 64, 1.0, 0.0, ws,
                                            1 << 30, nul))
    assert rc == -1
    rc, _ = _err(lib.kronq_accumulate_cross(fake, other, 1, 100, 64, 68, fake, 64, 1.0, 0.0, ws,
                                            1 << 30, nul))
    assert rc == -1
    # its BiIP takes only the input-side flags
    rc, msg = _err(lib.kronq_rotate_drift(fake, 64, 64, fake, fake, nul, K.ROT_OUT, ws, 1 << 30,
                                          nul))
    assert rc == -1 and "RESCALE_IN" in msg
    # P must not alias D
    rc, msg = _err(lib.kronq_gptaq_correction(fake, 64, 64, other, 64, 1.0, fake, 64, ws, 1 << 30,
                                              nul))
    assert rc == -1 and "alias" in msg


def test_cov_limited_argument_checks():
    lib = K.load()
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    rc, msg = _err(lib.kronq_accumulate_cov_limited(fake, 1, 100, 64, 64, fake, 64, 1.0, 0.0, -1,
                                                    nul, 0, nul))
    assert rc == -1 and "max_cus" in msg
    rc, msg = _err(lib.kronq_accumulate_cov_limited(fake, 1, 1000, 64, 64, fake, 64, 1.0, 0.0, 8,
                                                    nul, 16, nul))
    assert rc == -5 and "workspace" in msg


def test_cov_diag_and_split_rotation_argument_checks():
    lib = K.load()
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    ws = ctypes.c_void_p(1 << 30)
    assert K.kronq_workspace_bytes(K.OP_COV_DIAG, 0, 4096, 262144) >= 4096 * 8
    # cov_diag: bad dtype, lda < d, bf16 lda not divisible by 8, workspace too small
    rc, _ = _err(lib.kronq_cov_diag(fake, 3, 100, 64, 64, fake, 0, ws, 1 << 30, nul))
    assert rc == -1
    rc, msg = _err(lib.kronq_cov_diag(fake, 1, 100, 64, 32, fake, 0, ws, 1 << 30, nul))
    assert rc == -1 and "lda" in msg
    rc, msg = _err(lib.kronq_cov_diag(fake, 1, 100, 60, 60, fake, 0, ws, 1 << 30, nul))
    assert rc == -1 and "aligned" in msg
    rc, msg = _err(lib.kronq_cov_diag(fake, 1, 100000, 64, 64, fake, 0, ws, 16, nul))
    assert rc == -5 and "workspace" in msg
    rc, msg = _err(lib.kronq_cov_diag(fake, 1, 100, 64, 64, nul, 0, ws, 1 << 30, nul))
    assert rc == -1 and "hdiag" in msg
    rc, msg = _err(lib.kronq_cov_diag(fake, 1, 100, 64, 64, fake, -1, ws, 1 << 30, nul))
    assert rc == -1 and "max_cus" in msg

    def rot(flags, W_in=fake, W=fake):
        return _err(lib.kronq_rotate(W_in, 2, 128, W, 64, 128, 128, fake, 128, fake, 64, fake,
                                     fake, nul, nul, fake, fake, flags, ws, 1 << 30, nul))
    # HG_DIAG excludes HX_ONLY and SG_GIVEN; SG_GIVEN needs SX_GIVEN
    for flags in (K.HG_DIAG | K.HX_ONLY, K.HG_DIAG | K.SX_GIVEN | K.SG_GIVEN,
                  K.HG_DIAG | K.INVERSE):
        rc, msg = rot(K.BIIP | flags)
        assert rc == -1 and "HG_DIAG" in msg
    rc, msg = rot(K.BIIP | K.SG_GIVEN)
    assert rc == -1 and "SX_GIVEN" in msg
    # an H_G-only call reads neither W_in nor W, but needs H_G
    rc, msg = _err(lib.kronq_rotate(nul, 2, 0, nul, 64, 128, 0, nul, 0, nul, 64, fake, fake, nul,
                                    nul, fake, fake, K.BIIP | K.SX_GIVEN | K.SG_GIVEN, ws,
                                    1 << 30, nul))
    assert rc == -1 and "H_G" in msg
    # a W-transforming call still needs W_in
    rc, msg = rot(K.BIIP | K.SX_GIVEN | K.HG_DIAG, W_in=nul)
    assert rc == -1 and "W_in" in msg


def test_cov_diag_noalloc_checks_fail_before_any_launch():
    lib = K.load()
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    # the same argument checks as kronq_cov_diag
    rc, _ = _err(lib.kronq_cov_diag_noalloc(fake, 3, 100, 64, 64, fake, 0, nul))
    assert rc == -1
    rc, msg = _err(lib.kronq_cov_diag_noalloc(fake, 1, 100, 64, 32, fake, 0, nul))
    assert rc == -1 and "lda" in msg
    rc, msg = _err(lib.kronq_cov_diag_noalloc(fake, 1, 100, 64, 64, nul, 0, nul))
    assert rc == -1 and "hdiag" in msg
    # partials beyond the fixed 16 MiB array: rejected with the workspace error, by size alone
    d = 1 << 23
    rc, msg = _err(lib.kronq_cov_diag_noalloc(fake, 1, 4096, d, d, fake, 0, nul))
    assert rc == -5 and "scratch" in msg


def test_diagnostics_argument_checks():
    lib = K.load()
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    other = ctypes.c_void_p(1 << 28)
    ws = ctypes.c_void_p(1 << 30)
    assert K.kronq_workspace_bytes(K.OP_EIGH, 0, 4096, 0) >= 2 * 4096 * 4096 * 4
    assert K.kronq_workspace_bytes(K.OP_STATS, 4096, 4096, 0) > 0
    assert K.kronq_workspace_bytes(K.OP_PROXY, 4096, 4096, 0) > 0
    assert K.kronq_workspace_bytes(K.OP_EIGH, 0, 0, 0) == 0
    # stats: bad dtype, ld < cols, workspace too small
    rc, _ = _err(lib.kronq_matrix_stats(fake, 3, 8, 8, 8, other, ws, 1 << 30, nul))
    assert rc == -1
    rc, _ = _err(lib.kronq_matrix_stats(fake, 2, 8, 8, 4, other, ws, 1 << 30, nul))
    assert rc == -1
    rc, msg = _err(lib.kronq_matrix_stats(fake, 2, 64, 64, 64, other, ws, 16, nul))
    assert rc == -5 and "workspace" in msg
    # eigh: Q overlapping H, too many sweeps, too large an order
    rc, msg = _err(lib.kronq_eigh(fake, 64, 64, 10, other, ctypes.c_void_p((1 << 20) + 256), 64,
                                  other, ws, 1 << 30, nul))
    assert rc == -1 and "overlap" in msg
    rc, _ = _err(lib.kronq_eigh(fake, 64, 64, 65, other, other, 64, other, ws, 1 << 30, nul))
    assert rc == -1
    rc, _ = _err(lib.kronq_eigh(fake, 20000, 20000, 10, other, other, 20000, other, ws, 1 << 40,
                                nul))
    assert rc == -6
    # proxy factors: more exponents than the kernel's argument block holds
    al = (ctypes.c_double * 17)(*([0.25] * 17))
    rc, _ = _err(lib.kronq_proxy_loss_factors(fake, 8, 8, fake, 2, 8, 8, fake, 8, fake, 8, al, 17,
                                              other, ws, 1 << 30, nul))
    assert rc == -1


@pytest.mark.parametrize("seed", range(6))
def test_allocation_matches_oracle(seed):
    r = np.random.default_rng(seed)
    n = int(r.integers(2, 8))
    scores = np.exp(3 * r.standard_normal(n))
    weights = r.integers(1, 1000, size=n)
    avg = float(r.choice([2.5, 3.0, 3.5]))
    lib_bits, lib_val = K.kronq_allocate_bits(scores, weights, (2, 3, 4), avg)
    ora_bits, ora_val = O.allocate_bits(scores, weights, (2, 3, 4), avg)
    assert lib_bits == ora_bits
    assert lib_val == ora_val  # same float64 operations in the same order


def test_allocation_infeasible_budget():
    with pytest.raises(K.KronqError):
        K.kronq_allocate_bits([1.0, 2.0], [1, 1], (3, 4), 2.0)
