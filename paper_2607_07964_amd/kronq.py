"""Python binding of libkronq (the KronQ per-layer path on MI355X).

Argument marshalling only: every function checks tensor placement and dtype, supplies the
workspace and the current HIP stream, and calls the C-ABI entry point of the same name
(declared in include/kronq.h). PyTorch provides device memory and streams; all arithmetic runs
in the library's HIP kernels. There is no fallback: if libkronq.so is missing or a call fails,
an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkronq.so")

KRONQ_BF16, KRONQ_FP32 = 1, 2
RESCALE_IN, RESCALE_OUT, ROT_IN, ROT_OUT, INVERSE = 1, 2, 4, 8, 16
HX_ONLY, SX_GIVEN, HG_DIAG, SG_GIVEN = 32, 64, 128, 256
BIIP = RESCALE_IN | RESCALE_OUT | ROT_IN | ROT_OUT
OP_COV, OP_ROTATE, OP_CHOL, OP_OBS, OP_LOSS = 1, 2, 3, 4, 5
OP_CROSS, OP_ROTATE_DRIFT, OP_GPTAQ, OP_OBS_DRIFT, OP_ONLINE = 6, 7, 8, 9, 10
OP_STATS, OP_EIGH, OP_PROXY, OP_COV_DIAG = 11, 12, 13, 14
MAX_ALPHAS = 16
ERRORS = {0: "OK", -1: "INVALID_ARG", -2: "SHAPE", -3: "NOT_PD", -4: "HIP", -5: "WORKSPACE",
          -6: "UNSUPPORTED"}

EXPORTS = (
    "kronq_workspace_bytes", "kronq_last_error", "kronq_version", "kronq_accumulate_cov",
    "kronq_traces", "kronq_rotate", "kronq_cholesky_inv", "kronq_obs_quantize_layer",
    "kronq_layer_loss", "kronq_allocate_bits", "kronq_profile_enable", "kronq_profile_only",
    "kronq_profile_reset", "kronq_profile_read", "kronq_profile_names", "kronq_accumulate_cross",
    "kronq_rotate_drift",    "kronq_gptaq_correction", "kronq_obs_quantize_layer_drift", "kronq_pack_codes",
    "kronq_online_factors", "kronq_online_matvec", "kronq_matrix_stats", "kronq_eigh",
    "kronq_proxy_loss_factors", "kronq_accumulate_cov_limited", "kronq_cov_diag",
    "kronq_cov_diag_noalloc", "kronq_probe_mfma_bf16", "kronq_accumulate_cross_limited",
)


class KronqError(RuntimeError):
    def __init__(self, code: int, func: str, msg: str):
        super().__init__(f"{func}: {ERRORS.get(code, code)}: {msg}")
        self.code = code


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libkronq.so (once). Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2607_07964_amd.build`")
    lib = ctypes.CDLL(path)
    P, I64, I, F, D, SZ = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float,
                           ctypes.c_double, ctypes.c_size_t)
    sig = {
        "kronq_workspace_bytes": (SZ, [I, I64, I64, I64]),
        "kronq_last_error": (ctypes.c_char_p, []),
        "kronq_version": (I, []),
        "kronq_accumulate_cov": (I, [P, I, I64, I64, I64, P, I64, F, F, P, SZ, P]),
        "kronq_accumulate_cov_limited": (I, [P, I, I64, I64, I64, P, I64, F, F, I, P, SZ, P]),
        "kronq_cov_diag": (I, [P, I, I64, I64, I64, P, I, P, SZ, P]),
        "kronq_cov_diag_noalloc": (I, [P, I, I64, I64, I64, P, I, P]),
        "kronq_probe_mfma_bf16": (I, [P, I, P, I64, P, P]),
        "kronq_accumulate_cross": (I, [P, P, I, I64, I64, I64, P, I64, F, F, P, SZ, P]),
        "kronq_accumulate_cross_limited": (I, [P, P, I, I64, I64, I64, P, I64, F, F, I, P, SZ,
                                               P]),
        "kronq_rotate_drift": (I, [P, I64, I64, P, P, P, I, P, SZ, P]),
        "kronq_gptaq_correction": (I, [P, I64, I64, P, I64, F, P, I64, P, SZ, P]),
        "kronq_obs_quantize_layer_drift": (I, [P, I64, I64, I64, P, I64, P, I64, I, I, I, P, P, P,
                                               P, P, P, SZ, P]),
        "kronq_pack_codes": (I, [P, I64, I64, I64, I, P, I64, P]),
        "kronq_online_factors": (I, [P, P, I64, P, P]),
        "kronq_online_matvec": (I, [P, I64, P, P, I64, I, I, I64, I64, P, P, P, P, I, P, I, I64,
                                    I64, P, I64, P, SZ, P]),
        "kronq_matrix_stats": (I, [P, I, I64, I64, I64, P, P, SZ, P]),
        "kronq_eigh": (I, [P, I64, I64, I, P, P, I64, P, P, SZ, P]),
        "kronq_proxy_loss_factors": (I, [P, I64, I64, P, I, I64, I64, P, I64, P, I64, P, I, P, P,
                                         SZ, P]),
        "kronq_traces": (I, [P, I64, I64, P, I64, I64, P, P]),
        "kronq_rotate": (I, [P, I, I64, P, I64, I64, I64, P, I64, P, I64, P, P, P, P, P, P, I, P,
                             SZ, P]),
        "kronq_cholesky_inv": (I, [P, I64, I64, F, P, I64, P, P, SZ, P]),
        "kronq_obs_quantize_layer": (I, [P, I64, I64, I64, P, I64, I, I, I, P, P, P, P, P, P, SZ,
                                         P]),
        "kronq_layer_loss": (I, [P, I, I64, P, I64, I64, I64, P, I64, P, I64, P, P, SZ, P]),
        "kronq_allocate_bits": (I, [P, P, I, P, I, D, P, P]),
        "kronq_profile_enable": (I, [I]),
        "kronq_profile_only": (I, [ctypes.c_char_p]),
        "kronq_profile_reset": (None, []),
        "kronq_profile_read": (I, [ctypes.c_char_p, P, P]),
        "kronq_profile_names": (I64, [ctypes.c_char_p, SZ]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(rc: int, func: str):
    if rc != 0:
        raise KronqError(rc, func, load().kronq_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libkronq works on device tensors only")


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a row-major 2-D tensor (unit column stride)")
    return t.stride(0)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return KRONQ_BF16
    if t.dtype == torch.float32:
        return KRONQ_FP32
    raise ValueError(f"unsupported dtype {t.dtype}")


def workspace(op: int, d_out: int, d_in: int, n_rows: int, device) -> torch.Tensor:
    n = load().kronq_workspace_bytes(op, d_out, d_in, n_rows)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def kronq_workspace_bytes(op: int, d_out: int, d_in: int, n_rows: int) -> int:
    return int(load().kronq_workspace_bytes(op, d_out, d_in, n_rows))


def kronq_version() -> int:
    return int(load().kronq_version())


# ------------------------------------------------------------------------------------ steps
def kronq_accumulate_cov(A: torch.Tensor, H: torch.Tensor, alpha: float = 1.0, beta: float = 0.0,
                         ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """H <- beta H + alpha A^T A (token-major A [N x d], bf16 or fp32; H fp32 [d x d])."""
    _dev(A, H)
    n, d = A.shape
    if ws is None:
        ws = workspace(OP_COV, 0, d, n, A.device) if A.dtype == torch.bfloat16 else \
            torch.empty(256, dtype=torch.uint8, device=A.device)
    rc = load().kronq_accumulate_cov(_ptr(A), _dtype_code(A), n, d, _ld(A), _ptr(H), _ld(H),
                                     alpha, beta, _ptr(ws), ws.numel(), _stream(A.device))
    _check(rc, "kronq_accumulate_cov")
    return H


def kronq_accumulate_cov_limited(A: torch.Tensor, H: torch.Tensor, max_cus: int,
                                 alpha: float = 1.0, beta: float = 0.0,
                                 ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """kronq_accumulate_cov holding at most ``max_cus`` compute units at once (0: all)."""
    _dev(A, H)
    n, d = A.shape
    if ws is None:
        ws = workspace(OP_COV, 0, d, n, A.device) if A.dtype == torch.bfloat16 else \
            torch.empty(256, dtype=torch.uint8, device=A.device)
    rc = load().kronq_accumulate_cov_limited(_ptr(A), _dtype_code(A), n, d, _ld(A), _ptr(H),
                                             _ld(H), alpha, beta, int(max_cus), _ptr(ws),
                                             ws.numel(), _stream(A.device))
    _check(rc, "kronq_accumulate_cov_limited")
    return H


def kronq_cov_diag(A: torch.Tensor, out: Optional[torch.Tensor] = None,
                   ws: Optional[torch.Tensor] = None, max_cus: int = 0) -> torch.Tensor:
    """diag(A^T A) as fp32 [d] (token-major A [N x d], bf16 or fp32), without the covariance;
    ``max_cus`` > 0 bounds its workgroups."""
    _dev(A, out)
    n, d = A.shape
    if out is None:
        out = torch.empty(d, dtype=torch.float32, device=A.device)
    if ws is None:
        ws = workspace(OP_COV_DIAG, 0, d, n, A.device)
    rc = load().kronq_cov_diag(_ptr(A), _dtype_code(A), n, d, _ld(A), _ptr(out), int(max_cus),
                               _ptr(ws), ws.numel(), _stream(A.device))
    _check(rc, "kronq_cov_diag")
    return out


def kronq_cov_diag_noalloc(A: torch.Tensor, out: torch.Tensor, max_cus: int = 0) -> torch.Tensor:
    """kronq_cov_diag with the library's fixed device scratch array instead of a workspace:
    nothing is allocated (``out`` fp32 [d] is the caller's). Overlapping calls on one GPU race."""
    _dev(A, out)
    n, d = A.shape
    rc = load().kronq_cov_diag_noalloc(_ptr(A), _dtype_code(A), n, d, _ld(A), _ptr(out),
                                       int(max_cus), _stream(A.device))
    _check(rc, "kronq_cov_diag_noalloc")
    return out


def kronq_traces(HX: Optional[torch.Tensor], HG: Optional[torch.Tensor],
                 out: Optional[torch.Tensor] = None):
    """Device float64 tensor [tr H_X, tr H_G, tr H_X * tr H_G] (a None side leaves its slot)."""
    _dev(HX, HG)
    ref = HX if HX is not None else HG
    if out is None:
        out = torch.empty(3, dtype=torch.float64, device=ref.device)
    rc = load().kronq_traces(_ptr(HX), HX.shape[0] if HX is not None else 0,
                             _ld(HX) if HX is not None else 0, _ptr(HG),
                             HG.shape[0] if HG is not None else 0,
                             _ld(HG) if HG is not None else 0, _ptr(out), _stream(ref.device))
    _check(rc, "kronq_traces")
    return out


def kronq_rotate(W_in: Optional[torch.Tensor], W: Optional[torch.Tensor],
                 HX: Optional[torch.Tensor],
                 HG: Optional[torch.Tensor], sign_in: Optional[torch.Tensor],
                 sign_out: Optional[torch.Tensor], q28_in: Optional[torch.Tensor],
                 q28_out: Optional[torch.Tensor], sx: torch.Tensor, sg: torch.Tensor,
                 flags: int = BIIP, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """BiIP forward (W <- U S_G W_in S_X V^T, H_X and H_G in place) or, with INVERSE, the revert.
    With HG_DIAG, HG is the 1-D diagonal of H_G; with SG_GIVEN, W_in and W may be None (the
    sizes then come from sg and sx)."""
    _dev(W_in, W, HX, HG, sign_in, sign_out, q28_in, q28_out, sx, sg)
    d_out, d_in = W_in.shape if W_in is not None else (sg.numel(), sx.numel())
    dev = sx.device
    if ws is None:
        ws = workspace(OP_ROTATE, d_out, d_in, 0, dev)
    rc = load().kronq_rotate(
        _ptr(W_in), _dtype_code(W_in) if W_in is not None else KRONQ_FP32,
        _ld(W_in) if W_in is not None else 0, _ptr(W), d_out, d_in,
        _ld(W) if W is not None else 0, _ptr(HX),
        _ld(HX) if HX is not None else 0, _ptr(HG),
        _ld(HG) if HG is not None and HG.dim() == 2 else 0,
        _ptr(sign_in), _ptr(sign_out), _ptr(q28_in), _ptr(q28_out), _ptr(sx), _ptr(sg), flags,
        _ptr(ws), ws.numel(), _stream(dev))
    _check(rc, "kronq_rotate")
    return W


def kronq_cholesky_inv(H: torch.Tensor, U: torch.Tensor, damp: float = 0.01,
                       info: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Damp H in place and write the upper U with inv(H~) = U^T U. Returns the device info."""
    _dev(H, U)
    d = H.shape[0]
    if info is None:
        info = torch.empty(1, dtype=torch.int32, device=H.device)
    if ws is None:
        ws = workspace(OP_CHOL, 0, d, 0, H.device)
    rc = load().kronq_cholesky_inv(_ptr(H), d, _ld(H), damp, _ptr(U), _ld(U), _ptr(info),
                                   _ptr(ws), ws.numel(), _stream(H.device))
    _check(rc, "kronq_cholesky_inv")
    return info


def kronq_obs_quantize_layer(W: torch.Tensor, U: torch.Tensor, bits: int, codes: torch.Tensor,
                             scales: torch.Tensor, zeros: torch.Tensor,
                             err: Optional[torch.Tensor] = None,
                             W_hat: Optional[torch.Tensor] = None, group: int = 128,
                             block: int = 128, ws: Optional[torch.Tensor] = None):
    """Lazy-block OBS sweep with group quantisation; W ends as the dequantised W_hat."""
    _dev(W, U, codes, scales, zeros, err, W_hat)
    d_out, d_in = W.shape
    if ws is None:
        ws = workspace(OP_OBS, d_out, d_in, 0, W.device)
    rc = load().kronq_obs_quantize_layer(
        _ptr(W), d_out, d_in, _ld(W), _ptr(U), _ld(U), bits, group, block, _ptr(codes),
        _ptr(scales), _ptr(zeros), _ptr(err), _ptr(W_hat), _ptr(ws), ws.numel(),
        _stream(W.device))
    _check(rc, "kronq_obs_quantize_layer")


def kronq_accumulate_cross(A: torch.Tensor, B: torch.Tensor, C: torch.Tensor, alpha: float = 1.0,
                           beta: float = 0.0, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """C <- beta C + alpha A^T B (token-major A, B [N x d] of one dtype and row stride)."""
    _dev(A, B, C)
    n, d = A.shape
    if B.shape != A.shape or B.dtype != A.dtype or _ld(B) != _ld(A):
        raise ValueError("A and B must have the same shape, dtype and row stride")
    if ws is None:
        ws = workspace(OP_CROSS, 0, d, n, C.device)
    rc = load().kronq_accumulate_cross(_ptr(A), _ptr(B), _dtype_code(A), n, d, _ld(A), _ptr(C),
                                       _ld(C), alpha, beta, _ptr(ws), ws.numel(),
                                       _stream(C.device))
    _check(rc, "kronq_accumulate_cross")
    return C


def kronq_accumulate_cross_limited(A: torch.Tensor, B: torch.Tensor, C: torch.Tensor,
                                   max_cus: int, alpha: float = 1.0, beta: float = 0.0,
                                   ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """kronq_accumulate_cross holding at most ``max_cus`` compute units at once (0: all)."""
    _dev(A, B, C)
    n, d = A.shape
    if B.shape != A.shape or B.dtype != A.dtype or _ld(B) != _ld(A):
        raise ValueError("A and B must have the same shape, dtype and row stride")
    if ws is None:
        ws = workspace(OP_CROSS, 0, d, n, C.device)
    rc = load().kronq_accumulate_cross_limited(_ptr(A), _ptr(B), _dtype_code(A), n, d, _ld(A),
                                               _ptr(C), _ld(C), alpha, beta, int(max_cus),
                                               _ptr(ws), ws.numel(), _stream(C.device))
    _check(rc, "kronq_accumulate_cross_limited")
    return C


def kronq_rotate_drift(D: torch.Tensor, sx: Optional[torch.Tensor], sign_in: Optional[torch.Tensor],
                       q28_in: Optional[torch.Tensor], flags: int = RESCALE_IN | ROT_IN,
                       ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """D <- V diag(1/sx) D diag(1/sx) V^T in place (the input-side BiIP of H_X)."""
    _dev(D, sx, sign_in, q28_in)
    d = D.shape[0]
    if ws is None:
        ws = workspace(OP_ROTATE_DRIFT, 0, d, 0, D.device)
    rc = load().kronq_rotate_drift(_ptr(D), d, _ld(D), _ptr(sx), _ptr(sign_in), _ptr(q28_in),
                                   flags, _ptr(ws), ws.numel(), _stream(D.device))
    _check(rc, "kronq_rotate_drift")
    return D


def kronq_gptaq_correction(D: torch.Tensor, U: torch.Tensor, P: torch.Tensor, alpha: float = 1.0,
                           ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """P = alpha ((D U^T) . M_U) U, strictly upper triangular."""
    _dev(D, U, P)
    d = D.shape[0]
    if ws is None:
        ws = workspace(OP_GPTAQ, 0, d, 0, D.device)
    rc = load().kronq_gptaq_correction(_ptr(D), d, _ld(D), _ptr(U), _ld(U), alpha, _ptr(P), _ld(P),
                                       _ptr(ws), ws.numel(), _stream(D.device))
    _check(rc, "kronq_gptaq_correction")
    return P


def kronq_obs_quantize_layer_drift(W: torch.Tensor, U: torch.Tensor, P: torch.Tensor, bits: int,
                                   codes: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
                                   err: Optional[torch.Tensor] = None,
                                   W_hat: Optional[torch.Tensor] = None, group: int = 128,
                                   block: int = 128, ws: Optional[torch.Tensor] = None):
    """The lazy-block OBS sweep with the drift correction P; W ends as the dequantised W_hat."""
    _dev(W, U, P, codes, scales, zeros, err, W_hat)
    d_out, d_in = W.shape
    if ws is None:
        ws = workspace(OP_OBS_DRIFT, d_out, d_in, 0, W.device)
    rc = load().kronq_obs_quantize_layer_drift(
        _ptr(W), d_out, d_in, _ld(W), _ptr(U), _ld(U), _ptr(P), _ld(P), bits, group, block,
        _ptr(codes), _ptr(scales), _ptr(zeros), _ptr(err), _ptr(W_hat), _ptr(ws), ws.numel(),
        _stream(W.device))
    _check(rc, "kronq_obs_quantize_layer_drift")


def kronq_pack_codes(codes: torch.Tensor, bits: int, packed: Optional[torch.Tensor] = None
                     ) -> torch.Tensor:
    """Packed uint32 storage [d_out x d_in * bits / 32] (as int32) of uint8 codes."""
    _dev(codes, packed)
    d_out, d_in = codes.shape
    if packed is None:
        packed = torch.empty(d_out, d_in * bits // 32, dtype=torch.int32, device=codes.device)
    rc = load().kronq_pack_codes(_ptr(codes), d_out, d_in, _ld(codes), bits, _ptr(packed),
                                 _ld(packed), _stream(codes.device))
    _check(rc, "kronq_pack_codes")
    return packed


def kronq_online_factors(s: Optional[torch.Tensor], sign: Optional[torch.Tensor], d: int,
                         mul: Optional[torch.Tensor] = None, device=None) -> torch.Tensor:
    """mul = sign / s (the multipliers of the online transforms)."""
    _dev(s, sign, mul)
    dev = device or (s if s is not None else sign).device
    if mul is None:
        mul = torch.empty(d, dtype=torch.float32, device=dev)
    rc = load().kronq_online_factors(_ptr(s), _ptr(sign), d, _ptr(mul), _stream(mul.device))
    _check(rc, "kronq_online_factors")
    return mul


def kronq_online_matvec(packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
                        bits: int, group: int, d_in: int, mul_in: Optional[torch.Tensor],
                        mul_out: Optional[torch.Tensor], q28_in: Optional[torch.Tensor],
                        q28_out: Optional[torch.Tensor], x: torch.Tensor,
                        y: Optional[torch.Tensor] = None, flags: int = BIIP,
                        ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y = diag(mul_out) T_out W_hat' T_in diag(mul_in) x for the rows of x [batch x d_in]."""
    _dev(packed, scales, zeros, mul_in, mul_out, q28_in, q28_out, x, y)
    d_out = packed.shape[0]
    if x.dim() == 1:
        x = x.view(1, -1)
    batch = x.shape[0]
    if y is None:  # rows padded to a multiple of 4 floats (16-byte aligned rows)
        y = torch.empty(batch, (d_out + 3) // 4 * 4, dtype=torch.float32,
                        device=x.device)[:, :d_out]
    if ws is None:
        ws = workspace(OP_ONLINE, d_out, d_in, batch, x.device)
    rc = load().kronq_online_matvec(
        _ptr(packed), _ld(packed), _ptr(scales), _ptr(zeros), _ld(scales), bits, group, d_out,
        d_in, _ptr(mul_in), _ptr(mul_out), _ptr(q28_in), _ptr(q28_out), flags, _ptr(x),
        _dtype_code(x), _ld(x), batch, _ptr(y), _ld(y), _ptr(ws), ws.numel(), _stream(x.device))
    _check(rc, "kronq_online_matvec")
    return y


def kronq_layer_loss(W: torch.Tensor, W_hat: Optional[torch.Tensor], HX: torch.Tensor,
                     HG: torch.Tensor, out: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Device float64 scalar tr(H_G dW H_X dW^T), dW = W - W_hat."""
    _dev(W, W_hat, HX, HG)
    d_out, d_in = W.shape
    if out is None:
        out = torch.empty(1, dtype=torch.float64, device=W.device)
    if ws is None:
        ws = workspace(OP_LOSS, d_out, d_in, 0, W.device)
    rc = load().kronq_layer_loss(
        _ptr(W), _dtype_code(W), _ld(W), _ptr(W_hat), _ld(W_hat) if W_hat is not None else 0,
        d_out, d_in, _ptr(HX), _ld(HX), _ptr(HG), _ld(HG), _ptr(out), _ptr(ws), ws.numel(),
        _stream(W.device))
    _check(rc, "kronq_layer_loss")
    return out


def kronq_matrix_stats(M: torch.Tensor, out: Optional[torch.Tensor] = None,
                       ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Device float64 [5]: max |M|, ||M||_F^2, mu(M), CV of the column norms, CV of the row
    norms."""
    _dev(M)
    rows, cols = M.shape
    if out is None:
        out = torch.empty(5, dtype=torch.float64, device=M.device)
    if ws is None:
        ws = workspace(OP_STATS, rows, cols, 0, M.device)
    rc = load().kronq_matrix_stats(_ptr(M), _dtype_code(M), rows, cols, _ld(M), _ptr(out),
                                   _ptr(ws), ws.numel(), _stream(M.device))
    _check(rc, "kronq_matrix_stats")
    return out


def kronq_eigh(H: torch.Tensor, sweeps: int = 12, evals: Optional[torch.Tensor] = None,
               Q: Optional[torch.Tensor] = None, off: Optional[torch.Tensor] = None,
               ws: Optional[torch.Tensor] = None):
    """Jacobi eigendecomposition of the symmetric fp32 H: (evals, Q with unit eigenvector
    columns, device float64 off-diagonal residual)."""
    _dev(H)
    d = H.shape[0]
    if evals is None:
        evals = torch.empty(d, device=H.device)
    if Q is None:
        Q = torch.empty(d, d, device=H.device)
    if off is None:
        off = torch.empty(1, dtype=torch.float64, device=H.device)
    if ws is None:
        ws = workspace(OP_EIGH, 0, d, 0, H.device)
    rc = load().kronq_eigh(_ptr(H), d, _ld(H), int(sweeps), _ptr(evals), _ptr(Q), _ld(Q), _ptr(off),
                           _ptr(ws), ws.numel(), _stream(H.device))
    _check(rc, "kronq_eigh")
    return evals, Q, off


def kronq_proxy_loss_factors(HG: torch.Tensor, W: torch.Tensor, Hd: torch.Tensor, U: torch.Tensor,
                             alphas=(), out: Optional[torch.Tensor] = None,
                             ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Device float64 [6 + len(alphas)]: nearest, GPTQ and KronQ expected-loss factors, rho,
    tr(D), tr(H~), then the exponent sweep."""
    _dev(HG, W, Hd, U)
    d_out, d_in = W.shape
    n = len(alphas)
    if out is None:
        out = torch.empty(6 + n, dtype=torch.float64, device=W.device)
    if ws is None:
        ws = workspace(OP_PROXY, d_out, d_in, 0, W.device)
    al = (ctypes.c_double * max(n, 1))(*[float(a) for a in alphas])
    rc = load().kronq_proxy_loss_factors(
        _ptr(HG), d_out, _ld(HG), _ptr(W), _dtype_code(W), _ld(W), d_in, _ptr(Hd), _ld(Hd), _ptr(U),
        _ld(U), al, n, _ptr(out), _ptr(ws), ws.numel(), _stream(W.device))
    _check(rc, "kronq_proxy_loss_factors")
    return out


def kronq_allocate_bits(scores, weights, choices=(2, 3, 4), avg_bits: float = 3.0):
    """Host-side exhaustive bit allocation. Returns (bits tuple, objective)."""
    n = len(scores)
    s = (ctypes.c_double * n)(*[float(x) for x in scores])
    w = (ctypes.c_int64 * n)(*[int(x) for x in weights])
    c = (ctypes.c_int * len(choices))(*[int(x) for x in choices])
    out = (ctypes.c_int * n)()
    obj = ctypes.c_double()
    rc = load().kronq_allocate_bits(s, w, n, c, len(choices), avg_bits, out, ctypes.byref(obj))
    _check(rc, "kronq_allocate_bits")
    return tuple(out[i] for i in range(n)), obj.value


# ------------------------------------------------------------------------------------ profiler
def kronq_probe_mfma_bf16(data: torch.Tensor, iters: int, out: torch.Tensor) -> int:
    """Launch the register-resident bf16 MFMA loop on ``data`` (bf16, >= 4096 elements) on the
    current stream; returns the workgroup count (flops = wgs * 4 * iters * 8 * 32768)."""
    _dev(data, out)
    if data.dtype != torch.bfloat16 or data.numel() < 4096:
        raise ValueError("data must be bf16 with at least 4096 elements")
    wgs = ctypes.c_int()
    rc = load().kronq_probe_mfma_bf16(_ptr(data), int(iters), _ptr(out), out.numel(),
                                      ctypes.byref(wgs), _stream(data.device))
    _check(rc, "kronq_probe_mfma_bf16")
    return wgs.value


def kronq_profile_enable(on: bool = True):
    _check(load().kronq_profile_enable(int(on)), "kronq_profile_enable")


def kronq_profile_only(kernel: Optional[str]):
    _check(load().kronq_profile_only(None if kernel is None else kernel.encode()),
           "kronq_profile_only")


def kronq_profile_reset():
    load().kronq_profile_reset()


def kronq_profile_read(kernel: str):
    """(total milliseconds, launches) of the named kernel since the last reset."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(load().kronq_profile_read(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)),
           "kronq_profile_read")
    return ms.value, n.value


def kronq_profile_names() -> list:
    """Kernel names recorded since the last reset."""
    lib = load()
    need = int(lib.kronq_profile_names(None, 0))
    buf = ctypes.create_string_buffer(need + 1)
    lib.kronq_profile_names(buf, need + 1)
    return [n for n in buf.value.decode().split(",") if n]
