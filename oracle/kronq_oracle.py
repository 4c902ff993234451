"""Float64 reference of the KronQ per-layer quantisation path, written from the paper.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg, never by the product path. Plain numpy in float64; a matmul, a Cholesky or
an inverse from numpy/LAPACK serves as a step where the paper's definition is that operation.

Paper references (arxiv 2607.07964, "KronQ"):

* layer objective, Sec. 3.1 eq. (ptq_obj); K-FAC factors, Sec. 4.1 eq. (kfac), objective eq.
  (kron_obj);
* OBS compensation, Sec. 3.1 eq. (obs_update) and Proposition 1 eq. (kronq_update);
* BiIP rescaling, Sec. 4.2 eq. (rescale); rotations eq. (biip); Algorithm 1 (appendix B);
* sensitivity score, Sec. 4.3 eq. (sensitivity);
* quantisation loop, Algorithm 2 (appendix B);
* LDL loss identity, appendix A.3 eq. (app-decomp).

Readings taken where the paper is silent or garbled:

R1  covariances are plain sums, H_X = X^T X, H_G = G^T G (token-major X, G).
R3  the inverse-Cholesky factor is the UPPER U with inv(H~) = U^T U; the sweep uses rows of U
    (Algorithm 2 prints rows of a lower L, which would be zero blocks).
R5  the drift correction P of Algorithm 2 is optional: zero ("KronQ+GPTQ") unless the drift
    statistic D = dX^T X is given (the paper's default "KronQ+GPTAQ").
R6  damping lambda = 0.01 of the mean diagonal, on the post-BiIP H_X.
R7  asymmetric min-max grid per row and group (GPTQ convention): xmin = min(0, min w),
    xmax = max(0, max w), (-1, 1) if both are 0; scale = float32((xmax - xmin) / (2^b - 1));
    zero = rint(-xmin / scale); q = clamp(rint(w / scale) + zero, 0, 2^b - 1);
    w_hat = scale * (q - zero). rint is round-half-to-even; divisions are float64 IEEE.
    Group parameters are taken when the sweep reaches the group's first column.
R8  natural column order.
R10 a zero column/row norm or zero diagonal gives a scale of 1.
R11 V = H_d diag(sigma) / sqrt(d) (Sylvester H), or (Q28 kron H_m / sqrt(m)) diag(sigma) for
    d = 28 m, with the 28-point factor on the slow index.
R12 H_G is rotated too (Algorithm 1 does so before releasing it).
R13 traces are reported before and after BiIP; the sensitivity score uses post-BiIP traces.
R14 bit allocation: exhaustive search minimising sum_l s_l (2^b_l - 1)^-2 under a
    parameter-weighted average-bit budget, ties to the lexicographically smallest vector.
R15 the reported loss is taken in the original space with undamped H_X, H_G.
R19 drift correction (Prop. 1, Algorithm 2): the paper's L with inv(H~) = L L^T is the
    transpose of the upper U of R3, so P = alpha ((D U^T) . M_U) U, where M_U is the STRICTLY
    upper mask (Prop. 1 says strictly, Algorithm 2's comment drops the word). Row p of P is then
    alpha D[p, p+1:] inv(H~[p+1:, p+1:]), which is the least-squares absorption of column p's
    drift by the columns after it. D is the token-major dX^T X (dX = X~ - X).
R20 the W in the drift term of the sweep is the column as it stands when it is quantised; in
    the trailing update the block's columns enter with those same values, so that the lazy batch
    equals the per-column update of eq. kronq_update. (Read literally, Algorithm 2's trailing
    update would use the block after its sweep, which holds the quantised values.)
R21 alpha is an input; 1 is the value for which the update is the exact least-squares
    absorption. The paper leaves alpha's value to GPTAQ.
R22 packed codes: each run of 32 consecutive codes of a row is one 32*b-bit little-endian
    string (code j at bits [j*b, (j+1)*b)) held in b uint32 words.
R23 the online product is the original-space layer S_G^-1 U^T W_hat' V S_X^-1 x, applied factor
    by factor.
R24 CV_in and CV_out are population coefficients of variation (std / mean, std over n, not
    n - 1) of the column norms ||W_:,j|| and the row norms ||W_i,:|| (norms, not squared).
R25 mu(H) = sqrt(d) max |Q_ij| over the eigenvector matrix Q (unit columns) of the symmetric H.
    Within a repeated eigenvalue Q is not unique and neither is mu; comparisons are made where
    the maximising eigenvector belongs to a simple, separated eigenvalue.
R26 Prop. 2 and the optimality table: h_i = [H_G]_ii and a_i = ||W_i,:||^2 of the layer before
    BiIP; D holds the pivots the natural-order sweep sees, D_p = 1 / [inv(H~[p:, p:])]_00 for the
    damped post-BiIP H~ (the paper's "LDL diagonal"); the nearest-rounding row takes tr(H~) of
    the same matrix. A channel with h_i a_i = 0 takes s_i = 1 (as R10).
"""
from __future__ import annotations

import itertools

import numpy as np

__all__ = [
    "widen_bf16", "as_f64", "covariance", "covariance_diag", "cross_covariance", "traces",
    "rescale_factors", "hadamard", "rht_matrix", "rht_rows",
    "biip_forward", "biip_forward_rows", "biip_revert", "damp", "inverse_cholesky_factor",
    "gptaq_correction",
    "group_params", "quantize", "obs_unblocked", "obs_blocked", "kfac_loss", "kronq_objective",
    "allocate_bits", "count_avg_bits", "dequantize", "online_matvec", "pack_codes",
    "incoherence", "norm_cv", "eigenvectors", "hessian_incoherence", "sweep_pivots",
    "rescale_objective", "rescale_gain", "proxy_loss_factors",
    "RESCALE_IN", "RESCALE_OUT", "ROT_IN", "ROT_OUT", "BIIP",
]

# BiIP switches (the ablation of Table "ablation" toggles these)
RESCALE_IN, RESCALE_OUT, ROT_IN, ROT_OUT = 1, 2, 4, 8
BIIP = RESCALE_IN | RESCALE_OUT | ROT_IN | ROT_OUT


# ----------------------------------------------------------------------------------------------
# input widening
# ----------------------------------------------------------------------------------------------
def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exact float64 values (bits go to the high half of an
    IEEE float32, which widens exactly)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def as_f64(a) -> np.ndarray:
    """float16/32/64 numpy array -> float64 (exact)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return widen_bf16(a)
    return a.astype(np.float64)


# ----------------------------------------------------------------------------------------------
# O1: covariances  (Sec. 3.1: H_X = X X^T for column-stacked samples; Algorithm 1 first line;
#                   Sec. 4.1 eq. kfac for H_G)
# ----------------------------------------------------------------------------------------------
def covariance(A, chunk: int = 8192) -> np.ndarray:
    """H = A^T A for token-major A [N x d], summed over token chunks in float64 (reading R1)."""
    A = np.asarray(A)
    n, d = A.shape
    H = np.zeros((d, d), dtype=np.float64)
    for t0 in range(0, n, chunk):
        C = as_f64(A[t0:t0 + chunk])
        H += C.T @ C
    return H


def cross_covariance(A, B, chunk: int = 8192) -> np.ndarray:
    """D = A^T B for token-major A, B [N x d], summed over token chunks in float64. With A the
    input drift dX = X~ - X and B the input X this is the drift statistic of Algorithm 1's first
    line (the paper's dX X^T for column-stacked samples; eq. gptaq_obj)."""
    A, B = np.asarray(A), np.asarray(B)
    if A.shape != B.shape:
        raise ValueError("A and B must have the same shape")
    n, d = A.shape
    D = np.zeros((d, d), dtype=np.float64)
    for t0 in range(0, n, chunk):
        D += as_f64(A[t0:t0 + chunk]).T @ as_f64(B[t0:t0 + chunk])
    return D


# ----------------------------------------------------------------------------------------------
# O2: traces and the sensitivity score  (Sec. 4.3 eq. sensitivity)
# ----------------------------------------------------------------------------------------------
def covariance_diag(A, chunk: int = 8192) -> np.ndarray:
    """diag(A^T A) in float64: each channel's sum of squares over the tokens (the diagonal of
    O1, without the off-diagonal products)."""
    n, d = A.shape
    out = np.zeros(d, dtype=np.float64)
    for t0 in range(0, n, chunk):
        blk = as_f64(A[t0:t0 + chunk])
        out += np.einsum("ij,ij->j", blk, blk)
    return out


def traces(HX: np.ndarray, HG: np.ndarray) -> tuple[float, float, float]:
    """(tr H_X, tr H_G, s = tr H_G * tr H_X)."""
    tx = float(np.sum(np.diag(HX)))
    tg = float(np.sum(np.diag(HG)))
    return tx, tg, tx * tg


# ----------------------------------------------------------------------------------------------
# O3: BiIP diagonal rescaling  (Sec. 4.2 eq. rescale; Algorithm 1 rescaling lines)
# ----------------------------------------------------------------------------------------------
def _quarter_ratio(h: np.ndarray, a: np.ndarray) -> np.ndarray:
    ok = (h > 0) & (a > 0)
    s = np.ones_like(h)
    s[ok] = (h[ok] / a[ok]) ** 0.25
    return s  # reading R10: 1 where a norm or a diagonal entry is zero


def _diag(H) -> np.ndarray:
    H = np.asarray(H)
    return (H if H.ndim == 1 else np.diag(H)).astype(np.float64)


def rescale_factors(W: np.ndarray, HX: np.ndarray, HG: np.ndarray | None, flags: int = BIIP):
    """s^X_j = (H_X,jj / ||W_:,j||^2)^(1/4) and s^G_i = (H_G,ii / ||W_i,:||^2)^(1/4), both from
    the original W (1 for a side whose rescale is off). Only the diagonals of H_X and H_G enter,
    so either the matrices or their diagonals (1-D) may be passed."""
    W = as_f64(W)
    a = np.sum(W * W, axis=0)  # squared column norms (input side)
    b = np.sum(W * W, axis=1)  # squared row norms (output side)
    sx = _quarter_ratio(_diag(HX), a) if flags & RESCALE_IN else np.ones(W.shape[1])
    if flags & RESCALE_OUT:
        if HG is None:
            raise ValueError("output-side rescaling needs H_G")
        sg = _quarter_ratio(_diag(HG), b)
    else:
        sg = np.ones(W.shape[0])
    return sx, sg


# ----------------------------------------------------------------------------------------------
# O4: randomised Hadamard rotations  (Sec. 4.2 eq. biip; reading R11)
# ----------------------------------------------------------------------------------------------
def hadamard(m: int) -> np.ndarray:
    """Sylvester-ordered Hadamard matrix, entry (i, j) = (-1)^popcount(i & j)."""
    if m <= 0 or m & (m - 1):
        raise ValueError("Hadamard order must be a power of two")
    i = np.arange(m)
    x = i[:, None] & i[None, :]
    par = np.zeros_like(x)
    while np.any(x):
        par ^= x & 1
        x = x >> 1
    return np.where(par == 1, -1.0, 1.0)


def rht_matrix(d: int, sign, q28=None) -> np.ndarray:
    """Dense orthogonal V = H_d diag(sigma) / sqrt(d), or (Q28 kron H_m / sqrt(m)) diag(sigma)
    when d = 28 m (Q28 on the slow index: element index = a * m + b)."""
    sign = np.asarray(sign, dtype=np.float64)
    if q28 is None:
        core = hadamard(d) / np.sqrt(d)
    else:
        m = d // 28
        if 28 * m != d:
            raise ValueError("d must be 28 * 2^k when a 28-point factor is given")
        core = np.kron(np.asarray(q28, dtype=np.float64), hadamard(m) / np.sqrt(m))
    return core * sign[None, :]


def rht_rows(d: int, sign, q28, rows) -> np.ndarray:
    """Selected rows of the V of ``rht_matrix``, entry by entry from the same definition:
    V[i, j] = (-1)^popcount(i & j) sigma_j / sqrt(d), or, when d = 28 m with i = a m + b and
    j = a' m + b', V[i, j] = Q28[a, a'] (-1)^popcount(b & b') sigma_j / sqrt(m). For sizes whose
    dense matrix is too large to form (d = 28672 is 6.6 GB)."""
    sign = np.asarray(sign, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    j = np.arange(d, dtype=np.int64)
    if q28 is None:
        m, lo_i, lo_j, scale = d, rows, j, np.ones((len(rows), d))
    else:
        m = d // 28
        if 28 * m != d:
            raise ValueError("d must be 28 * 2^k when a 28-point factor is given")
        q = np.asarray(q28, dtype=np.float64)
        lo_i, lo_j = rows % m, j % m
        scale = q[(rows // m)[:, None], (j // m)[None, :]]
    x = lo_i[:, None] & lo_j[None, :]
    par = np.zeros_like(x)
    while np.any(x):
        par ^= x & 1
        x = x >> 1
    return scale * np.where(par == 1, -1.0, 1.0) / np.sqrt(m) * sign[None, :]


def biip_forward(W, HX, HG, rot_in=None, rot_out=None, flags: int = BIIP, D=None):
    """Algorithm 1:
    W' = S_G W S_X; H_X' = S_X^-1 H_X S_X^-1; H_G' = S_G^-1 H_G S_G^-1; D' = S_X^-1 D S_X^-1;
    then W'' = U W' V^T, H_X'' = V H_X' V^T, H_G'' = U H_G' U^T, D'' = V D' V^T.

    ``rot_in`` / ``rot_out`` are (sign, q28-or-None); ``D`` is the optional drift statistic
    (reading R5). Returns a dict with W, HX, HG, D, sx, sg, V, U (V, U are identities for a
    side whose rotation is off; D is None when not given)."""
    W = as_f64(W)
    HX = np.asarray(HX, dtype=np.float64)
    HG = None if HG is None else np.asarray(HG, dtype=np.float64)
    d_out, d_in = W.shape
    sx, sg = rescale_factors(W, HX, HG, flags)
    W1 = sg[:, None] * W * sx[None, :]
    HX1 = HX / np.outer(sx, sx)
    HG1 = None if HG is None else HG / np.outer(sg, sg)
    V = rht_matrix(d_in, *rot_in) if flags & ROT_IN else np.eye(d_in)
    U = rht_matrix(d_out, *rot_out) if flags & ROT_OUT else np.eye(d_out)
    D1 = None if D is None else np.asarray(D, dtype=np.float64) / np.outer(sx, sx)
    return {
        "W": U @ W1 @ V.T,
        "HX": V @ HX1 @ V.T,
        "HG": None if HG1 is None else U @ HG1 @ U.T,
        "D": None if D1 is None else V @ D1 @ V.T,
        "sx": sx, "sg": sg, "V": V, "U": U,
    }


def biip_forward_rows(W, HX, HG_diag, rot_in, rot_out, rows, flags: int = BIIP):
    """Algorithm 1 for a layer whose output side is too large to rotate densely: the full
    V H_X' V^T, but only the listed rows of W'' = U W' V^T (rows of U from ``rht_rows``) and the
    post-BiIP traces. The output side enters only through diag(H_G) (S_G, eq. rescale) and
    tr(U H_G' U^T) = tr(H_G') = sum_i H_G,ii / s^G_i^2 (an orthogonal similarity keeps the
    trace). Returns dict(HX, W_rows, sx, sg, traces)."""
    W = as_f64(W)
    HX = np.asarray(HX, dtype=np.float64)
    hg = _diag(HG_diag)
    d_out, d_in = W.shape
    sx, sg = rescale_factors(W, HX, hg, flags)
    HX1 = HX / np.outer(sx, sx)
    V = rht_matrix(d_in, *rot_in) if flags & ROT_IN else np.eye(d_in)
    rows = np.asarray(rows, dtype=np.int64)
    if flags & ROT_OUT:
        Ur = rht_rows(d_out, rot_out[0], rot_out[1], rows)
    else:
        Ur = np.eye(d_out)[rows]
    W1 = sg[:, None] * W * sx[None, :]
    HX2 = V @ HX1 @ V.T
    tx = float(np.trace(HX2))
    tg = float(np.sum(hg / sg ** 2))
    return {"HX": HX2, "W_rows": (Ur @ W1) @ V.T, "sx": sx, "sg": sg,
            "traces": (tx, tg, tx * tg)}


def biip_revert(W_hat, sx, sg, V, U) -> np.ndarray:
    """Algorithm 2's final line: W = S_G^-1 U^T W_hat V S_X^-1."""
    W_hat = np.asarray(W_hat, dtype=np.float64)
    return (U.T @ W_hat @ V) / sg[:, None] / sx[None, :]


# ----------------------------------------------------------------------------------------------
# O5, O6: damping and the inverse-Cholesky factor  (Algorithm 2 first two lines; Prop. 1)
# ----------------------------------------------------------------------------------------------
def damp(H, lam: float = 0.01) -> np.ndarray:
    """H~ = H + lam * mean(diag H) * I (reading R6)."""
    H = np.asarray(H, dtype=np.float64)
    return H + lam * np.mean(np.diag(H)) * np.eye(H.shape[0])


def inverse_cholesky_factor(Hd) -> np.ndarray:
    """Upper-triangular U with inv(H~) = U^T U (reading R3), by the LAPACK route
    U = cholesky(inv(H~))^T."""
    Hinv = np.linalg.inv(np.asarray(Hd, dtype=np.float64))
    Hinv = 0.5 * (Hinv + Hinv.T)
    return np.linalg.cholesky(Hinv).T


def gptaq_correction(D, U, alpha: float = 1.0, rows=None) -> np.ndarray:
    """The drift correction of Prop. 1 and Algorithm 2's third line,
    P = alpha ((D L) . M_U) L^T with L = U^T (readings R19, R21): strictly upper triangular.
    ``rows`` (optional) returns only those rows of P, each from the same row of D."""
    D = np.asarray(D, dtype=np.float64)
    U = np.asarray(U, dtype=np.float64)
    if rows is None:
        return alpha * (np.triu(D @ U.T, 1) @ U)
    rows = np.asarray(rows)
    T = D[rows] @ U.T
    T[np.arange(U.shape[0])[None, :] <= rows[:, None]] = 0.0  # keep columns after each row
    return alpha * (T @ U)


# ----------------------------------------------------------------------------------------------
# O7: the asymmetric min-max quantiser  (reading R7)
# ----------------------------------------------------------------------------------------------
def group_params(wg: np.ndarray, bits: int):
    """Per-row (scale, zero) of a [rows x g] group; scale rounded once to float32."""
    wg = np.asarray(wg, dtype=np.float64)
    maxq = float(2 ** bits - 1)
    xmin = np.minimum(wg.min(axis=1), 0.0)
    xmax = np.maximum(wg.max(axis=1), 0.0)
    flat = xmax == xmin
    xmin = np.where(flat, -1.0, xmin)
    xmax = np.where(flat, 1.0, xmax)
    scale = ((xmax - xmin) / maxq).astype(np.float32).astype(np.float64)
    zero = np.rint(-xmin / scale)
    return scale, zero


def quantize(w: np.ndarray, scale: np.ndarray, zero: np.ndarray, bits: int):
    """Codes q and dequantised values w_hat of one column w (per-row scale and zero)."""
    maxq = float(2 ** bits - 1)
    q = np.clip(np.rint(np.asarray(w, dtype=np.float64) / scale) + zero, 0.0, maxq)
    return q.astype(np.int64), scale * (q - zero)


# ----------------------------------------------------------------------------------------------
# O8: the column-wise OBS sweep  (eq. obs_update; Prop. 1 with P = 0; Algorithm 2)
# ----------------------------------------------------------------------------------------------
def _outputs(d_out, d_in, group):
    ng = d_in // group
    return (np.zeros((d_out, d_in), np.int64), np.zeros((d_out, ng)), np.zeros((d_out, ng)),
            np.zeros((d_out, d_in)), np.zeros((d_out, d_in)))


def obs_unblocked(W, U, bits: int, group: int = 128, P=None):
    """Sequential OBS: for each column p, quantise it (group parameters taken at the group's
    first column from the current W), form the scaled error e_p = (w_p - w_hat_p) / U_pp and
    subtract e_p U_{p, p:} from the columns p onward; with the drift correction P also add
    w_p P_{p, p:}, w_p being column p before it is quantised (eq. kronq_update; R20). Column p
    then holds w_hat_p.

    Returns dict(codes, scales, zeros, err, w_hat, W) with W the final compensated matrix."""
    W = as_f64(W).copy()
    U = np.asarray(U, dtype=np.float64)
    P = None if P is None else np.asarray(P, dtype=np.float64)
    d_out, d_in = W.shape
    if d_in % group:
        raise ValueError("d_in must be a multiple of the group size")
    codes, scales, zeros, err, w_hat = _outputs(d_out, d_in, group)
    for p in range(d_in):
        if p % group == 0:
            s, z = group_params(W[:, p:p + group], bits)
            scales[:, p // group], zeros[:, p // group] = s, z
        q, wh = quantize(W[:, p], s, z, bits)
        x = W[:, p].copy()
        e = (x - wh) / U[p, p]
        W[:, p:] -= np.outer(e, U[p, p:])
        if P is not None:
            W[:, p:] += np.outer(x, P[p, p:])
        codes[:, p], err[:, p], w_hat[:, p] = q, e, wh
    return {"codes": codes, "scales": scales, "zeros": zeros, "err": err, "w_hat": w_hat, "W": W}


def obs_blocked(W, U, bits: int, group: int = 128, block: int = 128, P=None):
    """Algorithm 2: in-block sequential updates restricted to the block, then one trailing
    update W[:, i+B:] -= E U[i:i+B, i+B:] - W_blk P[i:i+B, i+B:] per block (lazy batch), where
    W_blk holds the block's columns as they stood when each was quantised (R20). P = None is
    the P = 0 case."""
    W = as_f64(W).copy()
    U = np.asarray(U, dtype=np.float64)
    P = None if P is None else np.asarray(P, dtype=np.float64)
    d_out, d_in = W.shape
    if d_in % group:
        raise ValueError("d_in must be a multiple of the group size")
    codes, scales, zeros, err, w_hat = _outputs(d_out, d_in, group)
    for i in range(0, d_in, block):
        j_end = min(i + block, d_in)
        E = np.zeros((d_out, j_end - i))
        Wq = np.zeros((d_out, j_end - i))
        for j in range(i, j_end):
            if j % group == 0:
                s, z = group_params(W[:, j:j + group], bits)
                scales[:, j // group], zeros[:, j // group] = s, z
            q, wh = quantize(W[:, j], s, z, bits)
            x = W[:, j].copy()
            e = (x - wh) / U[j, j]
            W[:, j:j_end] -= np.outer(e, U[j, j:j_end])
            if P is not None:
                W[:, j:j_end] += np.outer(x, P[j, j:j_end])
            E[:, j - i], Wq[:, j - i] = e, x
            codes[:, j], err[:, j], w_hat[:, j] = q, e, wh
        if j_end < d_in:
            W[:, j_end:] -= E @ U[i:j_end, j_end:]
            if P is not None:
                W[:, j_end:] += Wq @ P[i:j_end, j_end:]
    return {"codes": codes, "scales": scales, "zeros": zeros, "err": err, "w_hat": w_hat, "W": W}


# ----------------------------------------------------------------------------------------------
# Inference with the quantised layer  (Sec. 3.2 and 4.2: the rotations are applied online; Alg. 2
# last line gives the original-space weights; Limitations: O(d log d) online reversion)
# ----------------------------------------------------------------------------------------------
def dequantize(codes, scales, zeros, group: int) -> np.ndarray:
    """W_hat' = scale * (q - zero) per row and group (the rotated-space dequantised weights)."""
    codes = np.asarray(codes, dtype=np.float64)
    s = np.repeat(np.asarray(scales, dtype=np.float64), group, axis=1)
    z = np.repeat(np.asarray(zeros, dtype=np.float64), group, axis=1)
    return s * (codes - z)


def online_matvec(W_rot, sx, sg, V, U, x) -> np.ndarray:
    """y = S_G^-1 U^T W_rot V S_X^-1 x for the columns of x [d_in x B], applied factor by factor
    from the right (the original-space product of Alg. 2's last line without forming it)."""
    x = np.asarray(x, dtype=np.float64)
    xr = V @ (x / np.asarray(sx, dtype=np.float64)[:, None])
    yr = np.asarray(W_rot, dtype=np.float64) @ xr
    return (U.T @ yr) / np.asarray(sg, dtype=np.float64)[:, None]


def pack_codes(codes, bits: int) -> np.ndarray:
    """Storage format of the codes: each run of 32 consecutive codes of a row becomes a
    32*bits-bit little-endian string (code j at bits [j*bits, (j+1)*bits)), held in `bits`
    uint32 words. Returns uint32 [d_out x d_in*bits/32]."""
    codes = np.asarray(codes, dtype=np.uint64)
    d_out, d_in = codes.shape
    if d_in % 32:
        raise ValueError("d_in must be a multiple of 32")
    out = np.zeros((d_out, d_in * bits // 32), dtype=np.uint64)
    for j in range(d_in):
        pos = (j // 32) * 32 * bits + (j % 32) * bits  # bit position in the row
        w, off = pos // 32, pos % 32
        out[:, w] |= (codes[:, j] << np.uint64(off)) & np.uint64(0xFFFFFFFF)
        if off + bits > 32:
            out[:, w + 1] |= codes[:, j] >> np.uint64(32 - off)
    return out.astype(np.uint32)


# ----------------------------------------------------------------------------------------------
# O10: the K-FAC loss  (Sec. 4.1 eq. kron_obj)
# ----------------------------------------------------------------------------------------------
def kfac_loss(dW, HX, HG) -> float:
    """tr(H_G dW H_X dW^T) = sum_ij (H_G dW)_ij (dW H_X)_ij."""
    dW = np.asarray(dW, dtype=np.float64)
    return float(np.sum((np.asarray(HG, np.float64) @ dW) * (dW @ np.asarray(HX, np.float64))))


def kronq_objective(W, W_hat, HX, HG, D=None) -> float:
    """The full layer objective of eq. kronq_full without its constant term:
    tr(H_G (dW H_X dW^T + 2 W D dW^T)) with dW = W - W_hat (D = None drops the drift term)."""
    W = np.asarray(W, dtype=np.float64)
    dW = W - np.asarray(W_hat, dtype=np.float64)
    HG = np.asarray(HG, dtype=np.float64)
    val = kfac_loss(dW, HX, HG)
    if D is not None:
        val += 2.0 * float(np.sum((HG @ W @ np.asarray(D, dtype=np.float64)) * dW))
    return val


# ----------------------------------------------------------------------------------------------
# O11: mixed-precision allocation  (Sec. 4.3; Sec. 5.5; reading R14)
# ----------------------------------------------------------------------------------------------
def allocate_bits(scores, weights, choices=(2, 3, 4), avg_bits: float = 3.0):
    """Exhaustive search over every assignment (lexicographic order of ``choices``) of
    sum_l s_l / (2^b_l - 1)^2 subject to sum_l w_l b_l <= avg_bits * sum_l w_l.
    Returns (bits tuple, objective)."""
    scores = [float(s) for s in scores]
    weights = [int(w) for w in weights]
    budget = avg_bits * float(sum(weights))
    best, best_val = None, None
    for bits in itertools.product(sorted(choices), repeat=len(scores)):
        if float(sum(w * b for w, b in zip(weights, bits))) > budget:
            continue
        val = 0.0
        for s, b in zip(scores, bits):
            val += s / float((2 ** b - 1) ** 2)
        if best_val is None or val < best_val:
            best, best_val = bits, val
    if best is None:
        raise ValueError("no assignment meets the bit budget")
    return best, best_val


def count_avg_bits(bits) -> float:
    """Count-weighted average bit width (the 'Avg bits' column of the mixed-precision table)."""
    return float(np.mean(np.asarray(bits, dtype=np.float64)))


# ----------------------------------------------------------------------------------------------
# Diagnostics  (Sec. 2.3 eq. incoherence_measure; Sec. 4.2 with Fig. 2; Prop. 2 eq. biip-bound,
# appendix A.3 and the optimality table)
# ----------------------------------------------------------------------------------------------
def incoherence(M) -> float:
    """mu(M) = sqrt(rows * cols) max_ij |M_ij| / ||M||_F (eq. incoherence_measure, left)."""
    M = as_f64(M)
    r, c = M.shape
    return float(np.sqrt(r * c) * np.max(np.abs(M)) / np.sqrt(np.sum(M * M)))


def norm_cv(M) -> tuple[float, float]:
    """(CV_in, CV_out): coefficient of variation of the column norms and of the row norms
    (Fig. 2b; reading R24)."""
    M = as_f64(M)

    def cv(n):
        mean = np.mean(n)
        return float(np.sqrt(np.mean((n - mean) ** 2)) / mean)

    return cv(np.sqrt(np.sum(M * M, axis=0))), cv(np.sqrt(np.sum(M * M, axis=1)))


def eigenvectors(H) -> tuple[np.ndarray, np.ndarray]:
    """Eigenvalues and the eigenvector matrix Q (unit columns) of the symmetric H (LAPACK)."""
    return np.linalg.eigh(np.asarray(H, dtype=np.float64))


def hessian_incoherence(H) -> float:
    """mu(H) = sqrt(d) max_ij |Q_ij| (eq. incoherence_measure, right; reading R25)."""
    _, Q = eigenvectors(H)
    return float(np.sqrt(H.shape[0]) * np.max(np.abs(Q)))


def sweep_pivots(Hd, U=None) -> np.ndarray:
    """D_p = 1 / [inv(H~[p:, p:])]_00, the pivots the natural-order sweep divides by (R26).
    [inv(H~[p:, p:])]_00 = U_pp^2 for the factor of R3, so the diagonal of that factor is used
    (``U`` if given, else the oracle's own factor of Hd)."""
    U = inverse_cholesky_factor(Hd) if U is None else np.asarray(U, dtype=np.float64)
    return 1.0 / np.diag(U) ** 2


def _powered_ratio(h, a, alpha: float) -> np.ndarray:
    h, a = np.asarray(h, dtype=np.float64), np.asarray(a, dtype=np.float64)
    ok = (h > 0) & (a > 0)
    s = np.ones_like(h)
    s[ok] = (h[ok] / a[ok]) ** alpha
    return s


def rescale_objective(h, a, alpha: float) -> float:
    """(sum_i h_i / s_i^2)(sum_i s_i^2 a_i) for s_i = (h_i / a_i)^alpha: the rescaling-dependent
    factor of the expected loss in Prop. 2 (eq. biip-bound; the exponent sweep of appendix A.3)."""
    h, a = np.asarray(h, dtype=np.float64), np.asarray(a, dtype=np.float64)
    s2 = _powered_ratio(h, a, alpha) ** 2
    return float(np.sum(h / s2) * np.sum(s2 * a))


def rescale_gain(h, a) -> float:
    """rho = (sum_i sqrt(h_i a_i))^2 / (sum_i h_i sum_i a_i) (Prop. 2)."""
    h, a = np.asarray(h, dtype=np.float64), np.asarray(a, dtype=np.float64)
    return float(np.sum(np.sqrt(h * a)) ** 2 / (np.sum(h) * np.sum(a)))


def proxy_loss_factors(HG, W, Hd, U=None) -> dict:
    """The three rows of the optimality table for a layer: nearest rounding
    (sum h)(sum a) tr(H~), GPTQ (sum h)(sum a) tr(D), KronQ (sum sqrt(h a))^2 tr(D), with
    h = diag(H_G) and a the squared row norms of W before BiIP, H~ the damped post-BiIP H_X
    (reading R26). Also rho and tr(D)."""
    h = _diag(HG)
    W = as_f64(W)
    a = np.sum(W * W, axis=1)
    trD = float(np.sum(sweep_pivots(Hd, U)))
    trH = float(np.trace(np.asarray(Hd, dtype=np.float64)))
    return {"nearest": float(np.sum(h) * np.sum(a) * trH),
            "gptq": float(np.sum(h) * np.sum(a) * trD),
            "kronq": float(np.sum(np.sqrt(h * a)) ** 2 * trD),
            "rho": rescale_gain(h, a), "trD": trD, "trH": trH}
