"""Seeded synthetic inputs for the KronQ per-layer path.

This module is the only code shared by the HIP path's callers (tests, bench) and the float64
oracle. It holds random draws, their distributions and shapes, and nothing of the method's
arithmetic.

Counter-based element generator
-------------------------------
Element (t, i) of a generated [N x d] matrix is a pure function of a 64-bit stream key and the
flat index c = t*d + i:

* ``h = mix32(mix32(lo32(c) ^ k1) ^ mix32(hi32(c) ^ k2))``. ``mix32`` is the "lowbias32" integer
  finaliser (xor-shift 16, multiply 0x7feb352d, xor-shift 15, multiply 0x846ca68b, xor-shift 16),
  a bijection on 32-bit words.
* The top 16 bits of ``h`` select one of 65536 quantiles, F^-1((u + 1/2) / 65536), of the target
  distribution. The quantile table is computed once in float64 and rounded to float32.
* The value is multiplied by a per-channel float32 scale (one IEEE multiply) and rounded to
  bfloat16 (round to nearest even) where the workload is bf16.

Every step is integer arithmetic or a single correctly rounded float32 operation. The same torch
code therefore gives identical bytes on a CPU tensor and on a GPU tensor. Any subset of
columns can be regenerated on its own, which is how full-size parity checks sample the
covariances.

The workloads stand in for the paper's calibration set of 128 sequences x 2048 tokens on LLaMA-3
layer shapes (experimental setup, Section 5.1). Outlier, heavy-tail and log-normal channel scales
mimic the column outliers and the gradient-scale spread the paper shows (Figure 1(a); appendix
on LLaMA-3-70B weight outliers).
"""
from __future__ import annotations

import dataclasses
import math
from functools import lru_cache
from typing import Optional

import numpy as np
import torch

__all__ = [
    "LayerSpec", "WORKLOADS", "workload", "block_layers", "quantile_table", "gen_matrix",
    "gen_columns", "layer_inputs", "rotation_params", "bf16_bits", "Rot", "drift_noise_spec",
    "gen_drift", "gen_drift_columns",
]

NQ = 65536  # quantile levels (16 bits of the hash)


# --------------------------------------------------------------------------------------------
# quantile tables
# --------------------------------------------------------------------------------------------
@lru_cache(maxsize=None)
def quantile_table(dist: str) -> torch.Tensor:
    """float32 table of the 65536 mid-point quantiles of ``dist`` (CPU tensor)."""
    u = (np.arange(NQ, dtype=np.float64) + 0.5) / NQ
    if dist == "normal":
        from scipy.special import ndtri
        q = ndtri(u)
    elif dist == "t3":
        from scipy.stats import t as student_t
        q = student_t.ppf(u, 3)
    elif dist == "laplace":
        q = np.where(u < 0.5, np.log(2.0 * u), -np.log(2.0 - 2.0 * u))
    else:
        raise ValueError(dist)
    return torch.from_numpy(q.astype(np.float32))


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    # (x * c) mod 2^32 for 0 <= x < 2^32, split so that no product exceeds 2^48 (int64-safe)
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & 0xFFFFFFFF


def _mix32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def _hash16(flat: torch.Tensor, k1: int, k2: int) -> torch.Tensor:
    lo = flat & 0xFFFFFFFF
    hi = flat >> 32
    h = _mix32(_mix32(lo ^ k1) ^ _mix32(hi ^ k2))
    return h >> 16


def _keys(seed: int, tag: str) -> tuple[int, int]:
    ss = np.random.SeedSequence([seed, *(ord(ch) for ch in tag)])
    k = ss.generate_state(2, dtype=np.uint32)
    return int(k[0]), int(k[1])


# --------------------------------------------------------------------------------------------
# matrix description
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class MatSpec:
    """A seeded [rows x cols] matrix: element (t, i) = table[col_dist[i]][hash(t, i)] * col_scale[i]."""
    seed: int
    tag: str
    rows: int
    cols: int
    dists: tuple  # names of the tables used
    dist_idx: Optional[np.ndarray]  # per column index into dists (None: all 0)
    col_scale: np.ndarray  # float32 [cols]
    dtype: torch.dtype  # torch.bfloat16 or torch.float32


def _tables(spec: MatSpec, device) -> torch.Tensor:
    return torch.cat([quantile_table(d) for d in spec.dists]).to(device)


def _gen_block(spec: MatSpec, r0: int, r1: int, cols: torch.Tensor, device) -> torch.Tensor:
    """Rows [r0, r1) of ``spec`` restricted to column indices ``cols`` (int64 tensor)."""
    k1, k2 = _keys(spec.seed, spec.tag)
    t = torch.arange(r0, r1, dtype=torch.int64, device=device)
    flat = t[:, None] * spec.cols + cols[None, :]
    u = _hash16(flat, k1, k2)
    if spec.dist_idx is not None:
        sel = torch.from_numpy(spec.dist_idx.astype(np.int64)).to(device)[cols]
        u = u + sel[None, :] * NQ
    vals = _tables(spec, device)[u]
    scale = torch.from_numpy(spec.col_scale).to(device)[cols]
    vals = vals * scale[None, :]
    return vals.to(spec.dtype)


def gen_matrix(spec: MatSpec, device="cpu", rows: Optional[tuple] = None,
               chunk_elems: Optional[int] = None) -> torch.Tensor:
    """Generate rows [r0, r1) (default all) of ``spec`` on ``device``, chunked over rows."""
    r0, r1 = rows if rows is not None else (0, spec.rows)
    if chunk_elems is None:  # cache-sized chunks on the CPU, large ones on the GPU
        chunk_elems = (1 << 20) if torch.device(device).type == "cpu" else (1 << 27)
    out = torch.empty((r1 - r0, spec.cols), dtype=spec.dtype, device=device)
    cols = torch.arange(spec.cols, dtype=torch.int64, device=device)
    step = max(1, chunk_elems // max(1, spec.cols))
    for a in range(r0, r1, step):
        b = min(r1, a + step)
        out[a - r0:b - r0] = _gen_block(spec, a, b, cols, device)
    return out


def gen_columns(spec: MatSpec, cols, rows: Optional[tuple] = None,
                chunk_elems: int = 1 << 20) -> torch.Tensor:
    """Columns ``cols`` of ``spec`` for rows [r0, r1), on the CPU: shape [r1-r0, len(cols)]."""
    r0, r1 = rows if rows is not None else (0, spec.rows)
    cols_t = torch.as_tensor(np.asarray(cols, dtype=np.int64))
    out = torch.empty((r1 - r0, cols_t.numel()), dtype=spec.dtype)
    step = max(1, chunk_elems // max(1, cols_t.numel()))
    for a in range(r0, r1, step):
        b = min(r1, a + step)
        out[a - r0:b - r0] = _gen_block(spec, a, b, cols_t, "cpu")
    return out


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw uint16 bit patterns of a bfloat16 CPU tensor (numpy view, no conversion)."""
    assert t.dtype == torch.bfloat16
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


# --------------------------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LayerSpec:
    """One linear layer's calibration problem: W [d_out x d_in], X [N x d_in], G [N x d_out]."""
    name: str
    d_out: int
    d_in: int
    n_tokens: int
    bits: int
    group: int
    damp: float
    x: MatSpec
    g: MatSpec
    w: MatSpec
    seed: int
    x_key: str  # layers with the same x_key share one X (and one H_X)


def _rng(seed: int, tag: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *(ord(c) for c in tag)])))


def _x_spec(kind: str, seed: int, tag: str, n: int, d: int, dtype) -> MatSpec:
    rng = _rng(seed, tag + ":cols")
    scale = np.ones(d, dtype=np.float32)
    if kind == "normal_x20":  # 4 outlier channels x20
        idx = rng.choice(d, 4, replace=False)
        scale[idx] = 20.0
        return MatSpec(seed, tag, n, d, ("normal",), None, scale, dtype)
    if kind == "normal_t3":  # 1% of channels Student-t(3)
        k = int(round(0.01 * d))
        sel = np.zeros(d, dtype=np.int64)
        sel[rng.choice(d, k, replace=False)] = 1
        return MatSpec(seed, tag, n, d, ("normal", "t3"), sel, scale, dtype)
    if kind == "laplace":
        return MatSpec(seed, tag, n, d, ("laplace",), None, scale, dtype)
    if kind == "normal_x50":  # 0.5% of channels x50
        k = int(round(0.005 * d))
        scale[rng.choice(d, k, replace=False)] = 50.0
        return MatSpec(seed, tag, n, d, ("normal",), None, scale, dtype)
    raise ValueError(kind)


def _g_spec(sigma: float, seed: int, tag: str, n: int, d: int, dtype) -> MatSpec:
    rng = _rng(seed, tag + ":cols")
    xi = rng.standard_normal(d)
    scale = np.exp(sigma * xi).astype(np.float32)  # per-output-channel log-normal(0, sigma)
    return MatSpec(seed, tag, n, d, ("normal",), None, scale, dtype)


def _w_spec(std: float, seed: int, tag: str, d_out: int, d_in: int, dtype) -> MatSpec:
    scale = np.full(d_in, std, dtype=np.float32)
    return MatSpec(seed, tag, d_out, d_in, ("normal",), None, scale, dtype)


def _layer(name, d_out, d_in, n, bits, seed, xkind, gsig, wstd, dtype, x_key=None, x_seed=None):
    xs = x_seed if x_seed is not None else seed
    xk = x_key or f"{name}:X"
    return LayerSpec(
        name=name, d_out=d_out, d_in=d_in, n_tokens=n, bits=bits, group=128, damp=0.01,
        x=_x_spec(xkind, xs, xk, n, d_in, dtype),
        g=_g_spec(gsig, seed, f"{name}:G", n, d_out, dtype),
        w=_w_spec(wstd, seed, f"{name}:W", d_out, d_in, dtype),
        seed=seed, x_key=xk,
    )


N_CAL = 128 * 2048  # calibration tokens: 128 sequences x 2048 (experimental setup)


def workload(k: int, n_tokens: Optional[int] = None) -> LayerSpec:
    """Single-layer workloads 1-4. ``n_tokens`` overrides N."""
    bf = torch.bfloat16
    if k == 1:
        return _layer("tiny256", 256, 256, n_tokens or 2048, 4, 0, "normal_x20", 1.0, 0.02,
                      torch.float32)
    if k == 2:
        return _layer("l3_8b_q_proj", 4096, 4096, n_tokens or N_CAL, 4, 1, "normal_t3", 1.5,
                      0.02, bf)
    if k == 3:
        return _layer("l3_8b_down_proj", 4096, 14336, n_tokens or N_CAL, 2, 2, "laplace", 1.5,
                      0.02, bf)
    if k == 4:
        return _layer("l3_70b_up_proj", 28672, 8192, n_tokens or N_CAL, 2, 3, "normal_x50",
                      2.0, 0.015, bf)
    raise ValueError(k)


WORKLOADS = (1, 2, 3, 4)

BLOCK_SHAPES = (  # LLaMA-3-8B decoder block: (name, d_out, d_in, shared-X key)
    ("q_proj", 4096, 4096, "attn_in"),
    ("k_proj", 1024, 4096, "attn_in"),
    ("v_proj", 1024, 4096, "attn_in"),
    ("o_proj", 4096, 4096, "attn_out"),
    ("gate_proj", 14336, 4096, "mlp_in"),
    ("up_proj", 14336, 4096, "mlp_in"),
    ("down_proj", 4096, 14336, "mlp_act"),
)


def block_layers(n_tokens: Optional[int] = None, seed: int = 4, shrink: int = 1) -> list[LayerSpec]:
    """Workload 5: the 7 linears of one LLaMA-3-8B block. q/k/v share one X, gate/up share one
    X; bits are assigned later by the sensitivity-driven allocation. ``shrink`` divides every
    dimension (16 keeps d_in a multiple of 128 and 14336 / 16 = 896 = 28 * 32 of the 28 * 2^k
    form), for block runs the float64 oracle can repeat in seconds."""
    n = n_tokens or N_CAL
    out = []
    for li, (name, d_out, d_in, xkey) in enumerate(BLOCK_SHAPES):
        d_out, d_in = d_out // shrink, d_in // shrink
        lseed = int(np.random.SeedSequence([seed, li]).generate_state(1)[0])
        xkind = "laplace" if xkey == "mlp_act" else "normal_t3"
        out.append(_layer(name, d_out, d_in, n, 3, lseed, xkind, 1.5, 0.02, torch.bfloat16,
                          x_key=f"blk:{xkey}", x_seed=seed))
    return out


# --------------------------------------------------------------------------------------------
# input drift (the drift-corrected objective: dX = X~ - X, full-precision minus quantised input)
# --------------------------------------------------------------------------------------------
DRIFT_SIGMA = 1.0 / 16   # noise part, relative to each input channel's scale
DRIFT_SHRINK = 0.0625    # signal part: the quantised model's input is the full one shrunk by 1/16


def drift_noise_spec(spec: LayerSpec) -> MatSpec:
    """The noise part Z of the synthetic drift: normal, X's per-channel scales times 1/16, fp32."""
    xs = spec.x
    return MatSpec(xs.seed, xs.tag + ":drift", xs.rows, xs.cols, ("normal",), None,
                   (xs.col_scale * np.float32(DRIFT_SIGMA)).astype(np.float32), torch.float32)


def _drift(Z: torch.Tensor, X: torch.Tensor, dtype) -> torch.Tensor:
    # one exact scaling by a power of two, one IEEE subtraction, one rounding: identical bytes on
    # CPU and GPU
    return (Z - X.float() * DRIFT_SHRINK).to(dtype)


def gen_drift(spec: LayerSpec, device="cpu", X: Optional[torch.Tensor] = None,
              rows: Optional[tuple] = None) -> torch.Tensor:
    """dX = Z - X / 16 in X's dtype: a stand-in for the gap between the full-precision and the
    quantised model's inputs, part noise and part a shrink of the signal (so that dX^T X has a
    systematic component). ``X`` may pass the already generated rows of the layer's input."""
    Z = gen_matrix(drift_noise_spec(spec), device, rows)
    if X is None:
        X = gen_matrix(spec.x, device, rows)
    return _drift(Z, X, spec.x.dtype)


def gen_drift_columns(spec: LayerSpec, cols, rows: Optional[tuple] = None) -> torch.Tensor:
    """Columns ``cols`` of gen_drift(spec) for rows [r0, r1), on the CPU."""
    return _drift(gen_columns(drift_noise_spec(spec), cols, rows), gen_columns(spec.x, cols, rows),
                  spec.x.dtype)


# --------------------------------------------------------------------------------------------
# rotation parameters (random signs and the 28 x 28 orthogonal factor are inputs of the method)
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass
class Rot:
    """Randomised-Hadamard parameters of one side: signs in {+1,-1} and, when d = 28 * 2^k,
    a 28 x 28 orthogonal factor (float32, row-major) on the slow index."""
    d: int
    sign: np.ndarray  # int8 [d]
    q28: Optional[np.ndarray]  # float32 [28, 28] or None
    q28_f64: Optional[np.ndarray]  # the same draw before rounding to float32


def rot_dims_ok(d: int) -> bool:
    if d > 0 and d & (d - 1) == 0:
        return True
    return d % 28 == 0 and (d // 28) & (d // 28 - 1) == 0 and d // 28 > 0


def rotation_params(d: int, seed: int, tag: str) -> Rot:
    if not rot_dims_ok(d):
        raise ValueError(f"dimension {d} is neither 2^k nor 28*2^k")
    rng = _rng(seed, tag + ":rot")
    sign = np.where(rng.integers(0, 2, size=d) == 0, 1, -1).astype(np.int8)
    q = q32 = None
    if d & (d - 1) != 0:
        a = rng.standard_normal((28, 28))
        qm, r = np.linalg.qr(a)
        q = qm * np.sign(np.diag(r))[None, :]  # Haar-distributed orthogonal
        q32 = q.astype(np.float32)
    return Rot(d, sign, q32, q)


def layer_inputs(spec: LayerSpec, device="cpu"):
    """(X, G, W) tensors of ``spec`` on ``device`` plus the two rotation draws."""
    X = gen_matrix(spec.x, device)
    G = gen_matrix(spec.g, device)
    W = gen_matrix(spec.w, device)
    return X, G, W


def layer_rotations(spec: LayerSpec) -> tuple[Rot, Rot]:
    return (rotation_params(spec.d_in, spec.seed, spec.name + ":in"),
            rotation_params(spec.d_out, spec.seed, spec.name + ":out"))


def small_spec(d_out: int, d_in: int, n: int, bits: int = 4, seed: int = 11,
               dtype=torch.bfloat16, xkind: str = "normal_t3", gsig: float = 1.5,
               wstd: float = 0.02, name: str = "small") -> LayerSpec:
    """A small layer with the same value recipe as the full workloads (for parity tests)."""
    return _layer(name, d_out, d_in, n, bits, seed, xkind, gsig, wstd, dtype)


def param_count(specs) -> list[int]:
    return [s.d_out * s.d_in for s in specs]
