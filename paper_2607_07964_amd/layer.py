"""Per-layer and per-block drivers: the KronQ hot path as a sequence of libkronq calls.

One layer (Alg. 1 then Alg. 2):
  H_X = X^T X, H_G = G^T G  ->  traces (pre)  ->  BiIP (rescale + both rotations)
  ->  traces (post: the sensitivity score)  ->  damping + inverse-Cholesky factor
  ->  lazy-block OBS sweep with group quantisation.
With the input drift dX (the paper's default KronQ+GPTAQ) also D = dX^T X, its input-side BiIP,
the correction P = alpha ((D U^T) . M_U) U after the factor, and the drift-corrected sweep.
All calls are enqueued on the current stream; nothing here synchronises except ``check()``.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

from . import kronq as K


@dataclasses.dataclass
class RotParams:
    """Device copies of one side's randomised-Hadamard draw."""
    sign: torch.Tensor  # int8 [d]
    q28: Optional[torch.Tensor]  # fp32 [28, 28] or None

    @staticmethod
    def to_device(sign, q28, device) -> "RotParams":
        s = torch.as_tensor(sign, dtype=torch.int8).to(device)
        q = None if q28 is None else torch.as_tensor(q28, dtype=torch.float32).contiguous().to(device)
        return RotParams(s, q)


@dataclasses.dataclass
class LayerState:
    """Device buffers of one layer's solve (allocated once, reused across calls)."""
    d_out: int
    d_in: int
    n_tokens: int
    HX: torch.Tensor
    HG: torch.Tensor
    W: torch.Tensor  # fp32 working copy (rotated, then dequantised)
    U: torch.Tensor
    codes: torch.Tensor
    scales: torch.Tensor
    zeros: torch.Tensor
    sx: torch.Tensor
    sg: torch.Tensor
    hgd: torch.Tensor  # diag(H_G) from G (the S_G rescaling without waiting for H_G)
    tr_pre: torch.Tensor
    tr_post: torch.Tensor
    info: torch.Tensor
    ws_cov_x: torch.Tensor
    ws_cov_g: torch.Tensor
    ws_diag: torch.Tensor
    ws_rot: torch.Tensor
    ws_chol: torch.Tensor
    ws_obs: torch.Tensor
    err: Optional[torch.Tensor] = None
    group: int = 128
    D: Optional[torch.Tensor] = None       # drift statistic dX^T X (then transformed)
    P: Optional[torch.Tensor] = None       # drift correction
    ws_cross: Optional[torch.Tensor] = None
    ws_rdrift: Optional[torch.Tensor] = None
    ws_gptaq: Optional[torch.Tensor] = None
    side: Optional[torch.cuda.Stream] = None
    ev: tuple = ()

    @staticmethod
    def allocate(d_out: int, d_in: int, n_tokens: int, device, keep_err: bool = False,
                 x_dtype=torch.bfloat16, g_dtype=torch.bfloat16,
                 cov_ws: bool = True, group: int = 128, drift: bool = False) -> "LayerState":
        """``cov_ws=False`` leaves the covariance workspaces out (a caller that shares one);
        ``group`` is the quantisation group (d_in: per-channel); ``drift`` adds the buffers of
        the drift correction."""
        f32 = dict(dtype=torch.float32, device=device)

        def ws(op, a, b, n, dt=torch.bfloat16):
            if op in (K.OP_COV, K.OP_CROSS) and (dt != torch.bfloat16 or not cov_ws):
                return torch.empty(256, dtype=torch.uint8, device=device)
            return K.workspace(op, a, b, n, device)

        return LayerState(
            d_out=d_out, d_in=d_in, n_tokens=n_tokens,
            HX=torch.empty(d_in, d_in, **f32), HG=torch.empty(d_out, d_out, **f32),
            W=torch.empty(d_out, d_in, **f32), U=torch.empty(d_in, d_in, **f32),
            codes=torch.empty(d_out, d_in, dtype=torch.uint8, device=device),
            scales=torch.empty(d_out, d_in // group, **f32),
            zeros=torch.empty(d_out, d_in // group, **f32),
            sx=torch.empty(d_in, **f32), sg=torch.empty(d_out, **f32),
            hgd=torch.empty(d_out, **f32),
            tr_pre=torch.empty(3, dtype=torch.float64, device=device),
            tr_post=torch.empty(3, dtype=torch.float64, device=device),
            info=torch.empty(1, dtype=torch.int32, device=device),
            ws_cov_x=ws(K.OP_COV, 0, d_in, n_tokens, x_dtype),
            ws_cov_g=ws(K.OP_COV, 0, d_out, n_tokens, g_dtype),
            ws_diag=K.workspace(K.OP_COV_DIAG, 0, d_out, n_tokens, device),
            ws_rot=ws(K.OP_ROTATE, d_out, d_in, 0), ws_chol=ws(K.OP_CHOL, 0, d_in, 0),
            ws_obs=ws(K.OP_OBS_DRIFT if drift else K.OP_OBS, d_out, d_in, 0),
            err=torch.empty(d_out, d_in, **f32) if keep_err else None,
            group=group,
            D=torch.empty(d_in, d_in, **f32) if drift else None,
            P=torch.empty(d_in, d_in, **f32) if drift else None,
            ws_cross=ws(K.OP_CROSS, 0, d_in, n_tokens, x_dtype) if drift else None,
            ws_rdrift=ws(K.OP_ROTATE_DRIFT, 0, d_in, 0) if drift else None,
            ws_gptaq=ws(K.OP_GPTAQ, 0, d_in, 0) if drift else None,
            side=torch.cuda.Stream(device=device),  # default priority
            ev=tuple(torch.cuda.Event() for _ in range(5)),
        )


def covariances(st: LayerState, X: torch.Tensor, G: torch.Tensor, skip_x: bool = False):
    """Steps a1/a2: H_X = X^T X (unless shared and already computed) and H_G = G^T G."""
    if not skip_x:
        K.kronq_accumulate_cov(X, st.HX, 1.0, 0.0, st.ws_cov_x)
    K.kronq_accumulate_cov(G, st.HG, 1.0, 0.0, st.ws_cov_g)


def biip(st: LayerState, W0: torch.Tensor, rin: RotParams, rout: RotParams, flags: int = K.BIIP):
    """Steps a3-a5: pre traces, BiIP, post traces."""
    K.kronq_traces(st.HX, st.HG, st.tr_pre)
    K.kronq_rotate(W0, st.W, st.HX, st.HG, rin.sign, rout.sign, rin.q28, rout.q28, st.sx, st.sg,
                   flags, st.ws_rot)
    K.kronq_traces(st.HX, st.HG, st.tr_post)


def drift_statistic(st: LayerState, dX: torch.Tensor, X: torch.Tensor, max_cus: int = 0):
    """Alg. 1 first line, second half: D = dX^T X (``max_cus`` > 0: on at most that many CUs)."""
    if max_cus > 0:
        K.kronq_accumulate_cross_limited(dX, X, st.D, max_cus, 1.0, 0.0, st.ws_cross)
    else:
        K.kronq_accumulate_cross(dX, X, st.D, 1.0, 0.0, st.ws_cross)


def drift_biip(st: LayerState, rin: RotParams, flags: int = K.BIIP):
    """Alg. 1: D <- V S_X^-1 D S_X^-1 V^T (needs S_X from the forward BiIP)."""
    K.kronq_rotate_drift(st.D, st.sx, rin.sign, rin.q28, flags & (K.RESCALE_IN | K.ROT_IN),
                         st.ws_rdrift)


def sweep(st: LayerState, bits: int, alpha: Optional[float] = None):
    """Step a7/a8: the lazy-block OBS sweep; with ``alpha`` (drift) first P from D and U."""
    if alpha is None:
        K.kronq_obs_quantize_layer(st.W, st.U, bits, st.codes, st.scales, st.zeros, st.err, None,
                                   group=st.group, ws=st.ws_obs)
        return
    K.kronq_gptaq_correction(st.D, st.U, st.P, alpha, st.ws_gptaq)
    K.kronq_obs_quantize_layer_drift(st.W, st.U, st.P, bits, st.codes, st.scales, st.zeros,
                                     st.err, None, group=st.group, ws=st.ws_obs)


def solve(st: LayerState, bits: int, damp: float = 0.01, alpha: Optional[float] = None):
    """Steps a6-a8: damping + inverse-Cholesky factor, then the lazy-block OBS sweep."""
    K.kronq_cholesky_inv(st.HX, st.U, damp, st.info, st.ws_chol)
    sweep(st, bits, alpha)


# Share of the compute units left free beside the H_G covariance in the two-stream schedule, for
# the factorisation's and the sweep's latency-bound kernels (a covariance workgroup holds its CU
# for a whole tile, so uncapped it starves them: the 8B q_proj takes 14.7 ms per layer uncapped,
# 11.5 ms on half the chip). The covariance loses less than the CUs it gives up, its clock
# being power-limited on the full chip: on half the chip the q_proj H_G takes 5.5-6.1 ms instead
# of 4.1 ms. Half the chip where the factorisation is not much shorter than that covariance; an
# eighth where H_G outlasts factorisation and sweep many times over (70B up_proj, d = 28672
# against d = 8192: 238.7 ms per layer on 7/8 of the chip, 242.9 ms on 3/4, 247.7 ms on one
# stream, 262.5 ms uncapped). The estimate uses rough rates: 1.1 PFLOP/s for a covariance,
# 20 TFLOP/s for the factorisation.
FACTOR_SHARE = 0.5
FACTOR_SHARE_SHORT = 0.125
# The drift statistic, first on the second stream (before H_G), holds 13/16 of the chip and
# leaves the rest to the H_X transform and the factorisation's first leaves and products: at
# q_proj with the drift correction, 18.49-18.56 ms per layer on 208 CUs against 18.85-18.93
# on 192 and 224, 19.28-19.33 on 176, 20.73-20.75 on 128 and 19.61-19.70 uncapped.
DRIFT_SHARE = 13.0 / 16.0
# Measured alternatives (q_proj, alternating with this schedule in one run): H_G started
# right after H_X with W transformed on the current stream, 11.58 against 11.40 ms; W on a third
# stream with H_G starting once S_X exists, 11.12 against 11.06 ms; W on the current stream
# with H_G starting once S_X exists, 11.18 against 11.10 ms; diag(H_G) beside the H_X
# covariance slowed that covariance from 3.55 to 4.3 ms; on 64 CUs beside the factorisation it
# took 5.1 ms, starved by H_G. With the drift correction, the drift statistic on the current
# stream before the factorisation: 20.8 against 20.1 ms.


def _cov_cus(device, n_tokens: int, d_out: int, d_in: int) -> int:
    """CUs the H_G covariance may hold beside the factorisation and the sweep."""
    t_cov = float(n_tokens) * d_out * d_out / 1.1e15
    t_factor = (2.0 / 3.0) * float(d_in) ** 3 / 2.0e13
    share = FACTOR_SHARE if t_factor >= 0.25 * t_cov else FACTOR_SHARE_SHORT
    cus = torch.cuda.get_device_properties(device).multi_processor_count
    return max(8, int(cus * (1.0 - share)))


def schedule(st: LayerState, n_tokens: int, overlap: bool = True,
             cov_cus: Optional[int] = None) -> str:
    """The schedule quantize_layer takes for this layer."""
    if not overlap:
        return "one stream"
    if cov_cus is None:
        cov_cus = _cov_cus(st.HG.device, n_tokens, st.d_out, st.d_in)
    return f"two streams, H_G on {cov_cus} CUs" if cov_cus else "two streams, H_G uncapped"


def biip_split(st: LayerState, W0: torch.Tensor, rin: RotParams, rout: RotParams,
               flags: int = K.BIIP):
    """Steps a3-a5 with S_G from ``st.hgd`` (diag(H_G) from G): pre traces, BiIP of W and H_X,
    then of H_G, post traces. The same transforms as the two-stream schedule's split calls."""
    K.kronq_traces(st.HX, st.HG, st.tr_pre)
    K.kronq_rotate(W0, st.W, st.HX, st.hgd, rin.sign, rout.sign, rin.q28, rout.q28, st.sx, st.sg,
                   flags | K.HG_DIAG, st.ws_rot)
    K.kronq_rotate(None, None, None, st.HG, rin.sign, rout.sign, rin.q28, rout.q28, st.sx, st.sg,
                   flags | K.SX_GIVEN | K.SG_GIVEN, st.ws_rot)
    K.kronq_traces(st.HX, st.HG, st.tr_post)


def quantize_layer(st: LayerState, X, G, W0, rin: RotParams, rout: RotParams, bits: int,
                   damp: float = 0.01, flags: int = K.BIIP, skip_x: bool = False,
                   overlap: bool = True, dX: Optional[torch.Tensor] = None, alpha: float = 1.0,
                   cov_cus: Optional[int] = None):
    """The whole hot path of one layer (enqueue only). ``dX`` (with buffers from
    ``allocate(drift=True)``) adds the drift correction with scaling ``alpha``.

    S_G needs only diag(H_G), which one read of G gives (kronq_cov_diag), so W is rescaled and
    rotated without waiting for the H_G covariance, and the sweep never waits for it either.
    With ``overlap`` diag(H_G) and H_X come first, then the work is split over two streams: the
    current stream rotates H_X, transforms W, factors H_X and runs the sweep; the second stream
    takes (the drift statistic and) the H_G covariance on ``cov_cus`` CUs (None: the policy of
    _cov_cus; 0: no cap) as soon as H_X is formed, whose traces and rotation end the layer. The
    current stream waits for the second at the end. The two schedules differ only in how the
    capped H_G covariance splits the tokens into slices (its sums in another order)."""
    drift = dX is not None
    if drift and st.D is None:
        raise ValueError("the drift correction needs LayerState.allocate(..., drift=True)")
    if overlap and cov_cus is None:
        cov_cus = _cov_cus(st.HG.device, G.shape[0], st.d_out, st.d_in)
    if not overlap:
        K.kronq_cov_diag(G, st.hgd, st.ws_diag)
        covariances(st, X, G, skip_x)
        if drift:
            drift_statistic(st, dX, X)
        biip_split(st, W0, rin, rout, flags)
        if drift:
            drift_biip(st, rin, flags)
        solve(st, bits, damp, alpha if drift else None)
        return
    main = torch.cuda.current_stream(st.HX.device)
    _, ev_sx, ev_w, ev_d, ev_g = st.ev
    # diag(H_G) first and alone (0.3 ms at q_proj): beside the compute-bound H_X covariance it
    # took 0.7 ms and slowed that covariance by more than its own time alone
    K.kronq_cov_diag(G, st.hgd, st.ws_diag)
    if not skip_x:
        K.kronq_accumulate_cov(X, st.HX, 1.0, 0.0, st.ws_cov_x)
    # (before the side stream starts: the traces kernel rewrites all three slots)
    K.kronq_traces(st.HX, None, st.tr_pre)
    # the side stream starts once H_X is formed (it needs nothing of H_X): its work is
    # enqueued before the factorisation's ~160 launches, so that it is dispatched right away
    # rather than after the host has issued them
    ev_sx.record(main)
    with torch.cuda.stream(st.side):
        st.side.wait_event(ev_sx)
        if drift:  # the drift statistic first: the correction P waits for it
            cus_all = torch.cuda.get_device_properties(st.D.device).multi_processor_count
            drift_statistic(st, dX, X, max(8, int(cus_all * DRIFT_SHARE)))
            ev_d.record(st.side)
        # the H_G covariance leaves part of the chip to the factorisation's and the sweep's
        # latency-bound kernels (a covariance workgroup holds its CU for a whole tile)
        K.kronq_accumulate_cov_limited(G, st.HG, cov_cus, 1.0, 0.0, st.ws_cov_g)
        K.kronq_traces(None, st.HG, st.tr_pre)
    K.kronq_rotate(W0, None, st.HX, None, rin.sign, None, rin.q28, None, st.sx, st.sg,
                   flags | K.HX_ONLY, st.ws_rot)
    K.kronq_traces(st.HX, None, st.tr_post)
    # W's transform on this stream, beside the H_G covariance, which ends the layer
    K.kronq_rotate(W0, st.W, None, st.hgd, rin.sign, rout.sign, rin.q28, rout.q28, st.sx,
                   st.sg, flags | K.SX_GIVEN | K.HG_DIAG, st.ws_rot)
    ev_w.record(main)
    with torch.cuda.stream(st.side):
        # the H_G transform uses S_G from W's transform, and the same rotation workspace (the
        # event is recorded above, before this wait is enqueued)
        st.side.wait_event(ev_w)
        K.kronq_rotate(None, None, None, st.HG, rin.sign, rout.sign, rin.q28, rout.q28, st.sx,
                       st.sg, flags | K.SX_GIVEN | K.SG_GIVEN, st.ws_rot)
        K.kronq_traces(None, st.HG, st.tr_post)
        ev_g.record(st.side)
    K.kronq_cholesky_inv(st.HX, st.U, damp, st.info, st.ws_chol)
    if drift:
        main.wait_event(ev_d)
        drift_biip(st, rin, flags)
        K.kronq_gptaq_correction(st.D, st.U, st.P, alpha, st.ws_gptaq)
    if drift:
        K.kronq_obs_quantize_layer_drift(st.W, st.U, st.P, bits, st.codes, st.scales, st.zeros,
                                         st.err, None, group=st.group, ws=st.ws_obs)
    else:
        K.kronq_obs_quantize_layer(st.W, st.U, bits, st.codes, st.scales, st.zeros, st.err, None,
                                   group=st.group, ws=st.ws_obs)
    main.wait_event(ev_g)


def check(st: LayerState):
    """Synchronise and raise if the factorisation met a non-positive pivot."""
    info = int(st.info.item())
    if info != 0:
        raise K.KronqError(-3, "kronq_cholesky_inv", f"pivot of column {info} is not positive")


def revert(st: LayerState, rin: RotParams, rout: RotParams, out: Optional[torch.Tensor] = None,
           flags: int = K.BIIP, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Original-space dequantised weights: S_G^-1 U^T W_hat' V S_X^-1 (Alg. 2, last line)."""
    if out is None:
        out = torch.empty_like(st.W)
    K.kronq_rotate(st.W, out, None, None, rin.sign, rout.sign, rin.q28, rout.q28, st.sx, st.sg,
                   flags | K.INVERSE, ws if ws is not None else st.ws_rot)
    return out


@dataclasses.dataclass
class BlockResult:
    """Outcome of ``quantize_block``: per-layer states (codes, scales, ...) and the allocation."""
    names: list
    states: list
    scores: list      # post-BiIP tr(H_X) tr(H_G) per layer (Sec. 4.3 sensitivity)
    bits: tuple
    objective: float


def quantize_block(specs, X_by_key: dict, Gs: list, W0s: list, rots: list,
                   avg_bits: float = 3.0, choices=(2, 3, 4), flags: int = K.BIIP,
                   keep_err: bool = False) -> BlockResult:
    """The layers of one decoder block with sensitivity-driven bit allocation (Sec. 4.3).

    1. One raw covariance per distinct input (q/k/v share one X, gate/up another); each layer
       takes a copy, since BiIP rescales H_X with that layer's own S_X. Then per layer: H_G,
       BiIP and the post-BiIP traces.
    2. Bits from the exhaustive allocation over the layers' scores s = tr(H_X) tr(H_G) under the
       parameter-weighted average budget (host side; needs the traces, so it synchronises).
    3. Per layer: damping + inverse-Cholesky factor and the OBS sweep at the allocated width.
    ``X_by_key`` maps each spec's ``x_key`` to its X; ``rots`` holds (RotParams in, out) pairs."""
    dev = Gs[0].device
    n = specs[0].n_tokens
    d_max = max(max(sp.d_in, sp.d_out) for sp in specs)
    ws_cov = K.workspace(K.OP_COV, 0, d_max, n, dev)  # shared: the calls are stream-ordered
    raw = {}
    for sp in specs:
        if sp.x_key not in raw:
            H = torch.empty(sp.d_in, sp.d_in, dtype=torch.float32, device=dev)
            K.kronq_accumulate_cov(X_by_key[sp.x_key], H, 1.0, 0.0, ws_cov)
            raw[sp.x_key] = H
    states = []
    for sp, G, W0, (rin, rout) in zip(specs, Gs, W0s, rots):
        st = LayerState.allocate(sp.d_out, sp.d_in, n, dev, keep_err=keep_err, cov_ws=False)
        st.HX.copy_(raw[sp.x_key])
        K.kronq_accumulate_cov(G, st.HG, 1.0, 0.0, ws_cov)
        biip(st, W0, rin, rout, flags)
        states.append(st)
    del raw
    scores = [float(v) for v in torch.stack([st.tr_post[2] for st in states]).cpu()]
    weights = [sp.d_out * sp.d_in for sp in specs]
    bits, obj = K.kronq_allocate_bits(scores, weights, choices, avg_bits)
    for sp, st, b in zip(specs, states, bits):
        solve(st, int(b), sp.damp)
    return BlockResult([sp.name for sp in specs], states, scores, tuple(bits), obj)
