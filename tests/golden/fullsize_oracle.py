#!/usr/bin/env python3
"""Float64 oracle outputs of the full-size workloads (N = 262144 tokens), for the end-to-end
GPU parity tests.

Computed on the host from the seeded generator (``synth``) with ``oracle/`` only: nothing here
reads a GPU result. The outputs are cached as ``tests/golden/fullsize/<name>.npz`` (git-ignored:
tens of MB) together with a hash of every input to the computation (the generator's source, the
source of each oracle function used, this file); a cache whose hash differs is stale and is
recomputed.

Workloads (the same specs bench.py and the tests use):

* ``q_proj``: LLaMA-3-8B q_proj, W 4096 x 4096, 4-bit. The whole layer: H_X, H_G, traces
  before and after BiIP, the factor, the blocked sweep of every row, the revert and the
  original-space K-FAC loss (eq. kron_obj, reading R15). Stored: all codes, both trace triples,
  the loss, s_X, s_G and sampled rows of U.
* ``down_proj`` (W 4096 x 14336, 2-bit, d_in = 28 * 512) and ``up_proj_70b`` (W 28672 x 8192,
  2-bit, d_out = 28 * 1024): the full H_X, diag(H_G) (S_G needs only the diagonal, eq. rescale),
  the rotated H_X, its factor, and the sweep of 48 sampled rows of W'' = U W' V^T, which are
  independent of each other given the factor (Alg. 2). Stored: the rows, their codes, the trace
  triples, s_X, s_G and sampled rows of U.
* ``block``: the seven linears of a LLaMA-3-8B block. Scores s = tr(H_X'') tr(H_G'') from the
  full H_X per shared input and diag(H_G) per layer, the exhaustive allocation (reading R14),
  then per layer the factor and 48 sampled rows of codes at the allocated width.

Usage: python tests/golden/fullsize_oracle.py [name ...]   (default: all; about 30 minutes on
8 host cores, most of it generating the inputs and the float64 covariances)
"""
from __future__ import annotations

import hashlib
import inspect
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
import synth  # noqa: E402

CACHE = os.path.join(HERE, "fullsize")
NAMES = ("q_proj", "down_proj", "up_proj_70b", "block")
WORKLOAD = {"q_proj": 2, "down_proj": 3, "up_proj_70b": 4}
N_ROWS = 48          # sampled rows of the sweep
N_U_ROWS = 8         # sampled rows of the factor
CHUNK = 8192         # tokens per generated chunk
ORACLE_FUNCS = (O.widen_bf16, O.as_f64, O.covariance, O.covariance_diag, O.traces,
                O.rescale_factors, O.hadamard, O.rht_matrix, O.rht_rows, O.biip_forward,
                O.biip_forward_rows, O.biip_revert, O.damp, O.inverse_cholesky_factor,
                O.group_params, O.quantize, O.obs_blocked, O.kfac_loss, O.allocate_bits)


def recipe_hash() -> str:
    h = hashlib.sha256()
    with open(os.path.join(ROOT, "synth", "__init__.py"), "rb") as f:
        h.update(f.read())
    for fn in ORACLE_FUNCS:
        h.update(inspect.getsource(fn).encode())
    with open(os.path.abspath(__file__), "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:24]


def sample_rows(d_out: int, seed: int) -> np.ndarray:
    """48 sorted row indices, including the first and the last row."""
    r = np.random.default_rng(seed)
    mid = r.choice(np.arange(1, d_out - 1), N_ROWS - 2, replace=False)
    return np.sort(np.concatenate([[0, d_out - 1], mid])).astype(np.int64)


def _view(t) -> np.ndarray:
    return synth.bf16_bits(t) if str(t.dtype) == "torch.bfloat16" else t.numpy()


def _rot(rot: synth.Rot):
    """(sign, q28) as the GPU path receives them: the float32-rounded 28 x 28 factor."""
    return rot.sign.astype(np.float64), (None if rot.q28 is None else rot.q28.astype(np.float64))


def _log(msg: str):
    print(f"[fullsize-oracle] {time.strftime('%H:%M:%S')} {msg}", flush=True)


def covariance_stream(mspec, full: bool = True) -> np.ndarray:
    """H = A^T A (or its diagonal) of a generated [N x d] matrix, chunk by chunk."""
    acc = None
    for t0 in range(0, mspec.rows, CHUNK):
        blk = _view(synth.gen_matrix(mspec, "cpu", rows=(t0, min(mspec.rows, t0 + CHUNK))))
        part = O.covariance(blk) if full else O.covariance_diag(blk)
        acc = part if acc is None else acc + part
    return acc


def _u_rows(U: np.ndarray, seed: int):
    d = U.shape[0]
    r = np.random.default_rng(seed + 1000)
    rows = np.sort(np.concatenate([[0, d - 1], r.choice(np.arange(1, d - 1), N_U_ROWS - 2,
                                                        replace=False)]))
    return rows.astype(np.int64), U[rows].astype(np.float32)


def whole_layer(spec) -> dict:
    ri, ro = (_rot(r) for r in synth.layer_rotations(spec))
    _log(f"{spec.name}: H_X")
    hx = covariance_stream(spec.x)
    _log(f"{spec.name}: H_G")
    hg = covariance_stream(spec.g)
    w0 = O.as_f64(_view(synth.gen_matrix(spec.w, "cpu")))
    tr_pre = O.traces(hx, hg)
    _log(f"{spec.name}: BiIP, factor, sweep")
    b = O.biip_forward(w0, hx, hg, ri, ro)
    tr_post = O.traces(b["HX"], b["HG"])
    U = O.inverse_cholesky_factor(O.damp(b["HX"], spec.damp))
    q = O.obs_blocked(b["W"], U, spec.bits, spec.group, 128)
    W_hat = O.biip_revert(q["w_hat"], b["sx"], b["sg"], b["V"], b["U"])
    loss = O.kfac_loss(w0 - W_hat, hx, hg)
    urows, uvals = _u_rows(U, spec.seed)
    return {"codes": q["codes"].astype(np.uint8), "tr_pre": np.array(tr_pre),
            "tr_post": np.array(tr_post), "loss": np.array(loss), "sx": b["sx"], "sg": b["sg"],
            "u_rows": urows, "u_vals": uvals}


def sampled_layer(spec, hx=None, bits=None) -> dict:
    """Sampled rows of the solve. ``hx`` may pass the layer's raw H_X (shared inputs)."""
    ri, ro = (_rot(r) for r in synth.layer_rotations(spec))
    if hx is None:
        _log(f"{spec.name}: H_X (d = {spec.d_in})")
        hx = covariance_stream(spec.x)
    _log(f"{spec.name}: diag(H_G) (d = {spec.d_out})")
    hgd = covariance_stream(spec.g, full=False)
    w0 = O.as_f64(_view(synth.gen_matrix(spec.w, "cpu")))
    rows = sample_rows(spec.d_out, spec.seed)
    _log(f"{spec.name}: BiIP of H_X and of the sampled rows, factor, sweep")
    b = O.biip_forward_rows(w0, hx, hgd, ri, ro, rows)
    U = O.inverse_cholesky_factor(O.damp(b["HX"], spec.damp))
    q = O.obs_blocked(b["W_rows"], U, bits or spec.bits, spec.group, 128)
    urows, uvals = _u_rows(U, spec.seed)
    tr_pre = (float(np.trace(hx)), float(np.sum(hgd)), float(np.trace(hx)) * float(np.sum(hgd)))
    return {"rows": rows, "codes": q["codes"].astype(np.uint8), "tr_pre": np.array(tr_pre),
            "tr_post": np.array(b["traces"]), "sx": b["sx"], "sg": b["sg"], "u_rows": urows,
            "u_vals": uvals}


def block(choices=(2, 3, 4), avg_bits: float = 3.0) -> dict:
    specs = synth.block_layers()
    hx = {}
    for sp in specs:
        if sp.x_key not in hx:
            _log(f"block: H_X of {sp.x_key} (d = {sp.d_in})")
            hx[sp.x_key] = covariance_stream(sp.x)
    parts, rows_all = [], []
    for sp in specs:
        _log(f"block {sp.name}: diag(H_G) (d = {sp.d_out}), BiIP")
        hgd = covariance_stream(sp.g, full=False)
        w0 = O.as_f64(_view(synth.gen_matrix(sp.w, "cpu")))
        ri, ro = (_rot(r) for r in synth.layer_rotations(sp))
        rows = sample_rows(sp.d_out, sp.seed)
        parts.append(O.biip_forward_rows(w0, hx[sp.x_key], hgd, ri, ro, rows))
        rows_all.append(rows)
    scores = [p["traces"][2] for p in parts]   # post-BiIP tr(H_X'') tr(H_G'') (Sec. 4.3)
    weights = [sp.d_out * sp.d_in for sp in specs]
    bits, obj = O.allocate_bits(scores, weights, choices, avg_bits)
    _log(f"block: scores {scores}, bits {bits}")
    out = {"scores": np.array(scores), "bits": np.array(bits), "objective": np.array(obj)}
    for sp, b, rows, nb in zip(specs, parts, rows_all, bits):
        _log(f"block {sp.name}: factor, sweep of {len(rows)} rows at {nb} bits")
        U = O.inverse_cholesky_factor(O.damp(b["HX"], sp.damp))
        q = O.obs_blocked(b["W_rows"], U, int(nb), sp.group, 128)
        out[f"{sp.name}:rows"] = rows
        out[f"{sp.name}:codes"] = q["codes"].astype(np.uint8)
        out[f"{sp.name}:tr_post"] = np.array(b["traces"])
        b["HX"] = None
    return out


def compute(name: str) -> dict:
    if name == "q_proj":
        return whole_layer(synth.workload(WORKLOAD[name]))
    if name in ("down_proj", "up_proj_70b"):
        return sampled_layer(synth.workload(WORKLOAD[name]))
    if name == "block":
        return block()
    raise ValueError(name)


def path(name: str) -> str:
    return os.path.join(CACHE, f"{name}.npz")


def load(name: str):
    """The cached outputs of ``name``, or None when missing or computed from another recipe."""
    p = path(name)
    if not os.path.exists(p):
        return None
    with np.load(p, allow_pickle=False) as z:
        if str(z["recipe"]) != recipe_hash():
            return None
        return {k: z[k] for k in z.files if k != "recipe"}


def build(name: str) -> dict:
    t0 = time.time()
    out = compute(name)
    os.makedirs(CACHE, exist_ok=True)
    tmp = path(name) + ".tmp.npz"
    np.savez_compressed(tmp, recipe=np.array(recipe_hash()), **out)
    os.replace(tmp, path(name))
    _log(f"{name}: done in {time.time() - t0:.0f} s -> {path(name)}")
    return out


if __name__ == "__main__":
    import torch
    torch.set_num_threads(len(os.sched_getaffinity(0)))
    todo = sys.argv[1:] or list(NAMES)
    for nm in todo:
        if load(nm) is not None:
            _log(f"{nm}: cache is current")
            continue
        build(nm)
