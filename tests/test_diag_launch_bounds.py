"""Host-side bounds check of the eigendecomposition's launches (kronq_eigh, diag.hip), on the CPU.

Every global index the block-Jacobi kernels form is enumerated for each launch of a full sweep
(every round r, every workgroup) from the same launch geometry and index arithmetic the host
code and the kernels use, and checked against the size of the buffer it addresses: the padded
N x N matrices A0/A1/V, the rotation buffer zbuf (np 64 x 64 blocks), the caller's H, Q and the
fp64 row sums. Within a workgroup an index is monotone in the element index inside each of the
two 32-index halves of a block pair, so the first and last element of each half bound it.
"""
import numpy as np
import pytest

BJ, BT = 32, 64


def circle(k, r, n):
    k = np.asarray(k, dtype=np.int64)
    return np.where(k == 0, 0, 1 + (k - 1 + r) % (n - 1))


def pair_rows(P, Q):
    """All indices of block pair (P, Q): [P*32, P*32+31] and [Q*32, Q*32+31] (min, max)."""
    lo = np.minimum(P, Q) * BJ
    hi = np.maximum(P, Q) * BJ + BJ - 1
    return lo, hi


@pytest.mark.parametrize("d", [4096, 4093, 100, 64, 1, 8191])
def test_block_jacobi_indices_stay_in_their_buffers(d):
    N = -(-d // BT) * BT
    nb, np_ = N // BJ, N // BT
    size_A = N * N                      # A0, A1, V (each N x N)
    size_z = np_ * BT * BT              # zbuf
    ldh = ldq = d
    # bjac_init: grid (ceil(N/256), N), j < N checked in the kernel
    i = np.arange(N)
    j_max = N - 1
    assert (i.max() * N + j_max) < size_A
    # the H read is guarded by i < d and j < d
    assert ((d - 1) * ldh + d - 1) < d * ldh
    for r in range(nb - 1):
        # bjac_solve: one workgroup per pair, j < np
        jj = np.arange(np_)
        P, Q = circle(jj, r, nb), circle(nb - 1 - jj, r, nb)
        assert P.min() >= 0 and Q.min() >= 0 and max(P.max(), Q.max()) < nb
        assert np.all(P != Q)
        lo, hi = pair_rows(P, Q)
        assert lo.min() >= 0 and (hi.max() * N + hi.max()) < size_A
        assert ((np_ - 1) * BT * BT + BT * BT - 1) < size_z
        # the pairs of a round are disjoint: every block appears once
        assert np.array_equal(np.sort(np.concatenate([P, Q])), np.arange(nb))
        # bjac_apply: grid (np, np + N/64)
        kx = np.arange(np_)
        P2, Q2 = circle(kx, r, nb), circle(nb - 1 - kx, r, nb)
        _, chi = pair_rows(P2, Q2)
        ky = np.arange(np_ + N // BT)
        vt = ky >= np_
        # V tiles: rows 64 (ky - np) .. + 63, read and written in place
        vrow_hi = (ky[vt] - np_) * BT + BT - 1
        assert vrow_hi.max() < N and (vrow_hi.max() * N + chi.max()) < size_A
        # A / B tiles
        P1, Q1 = circle(ky[~vt], r, nb), circle(nb - 1 - ky[~vt], r, nb)
        _, rhi = pair_rows(P1, Q1)
        assert (rhi.max() * N + chi.max()) < size_A
        assert (kx.max() * BT * BT + BT * BT - 1) < size_z
        assert (ky[~vt].max() * BT * BT + BT * BT - 1) < size_z
    # bjac_out: grid (ceil(d/256), d), j < d: V[i*N+j] and Q[i*ldq+j]
    assert ((d - 1) * N + d - 1) < size_A and ((d - 1) * ldq + d - 1) < d * ldq
    # row_squares / jacobi_finish: i < d, j < d with lda = N; sums of d entries
    assert ((d - 1) * N + d - 1) < size_A
    # grid dimensions within the hardware limits (y <= 65535)
    assert N <= 65535 and np_ + N // BT <= 65535
