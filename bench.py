#!/usr/bin/env python3
"""Seconds per layer of the KronQ hot path on one MI355X.

One step = the whole per-layer path on one batch of synthetic calibration data already
resident in HBM: H_X = X^T X, H_G = G^T G, traces, BiIP (rescale + both randomised Hadamard
rotations of W, H_X, H_G), traces, damping + inverse-Cholesky factor, lazy-block OBS sweep with
group quantisation. Default workload: the LLaMA-3-8B q_proj shape, W 4096 x 4096, 262144 tokens
(128 x 2048), 4-bit, group 128. --drift adds the drift correction (KronQ+GPTAQ: D = dX^T X, its
BiIP, P and the drift-corrected sweep); --group sets the quantisation group (0: per-channel).
--online times the inference side instead: one decode matvec of the quantised layer with the
rotations applied online (kronq_online_matvec), against a dense bf16 GEMV of the same shape.
--diagnostics times the diagnostics of the incoherence processing on the layer instead: mu(W) and
the row/column norm variation for the original, input-side-processed and BiIP-processed weights,
mu(H_X) and mu(H_G) before and after BiIP from Jacobi eigendecompositions, and the expected-loss
factors of Prop. 2 with the rescale-exponent sweep.

The JSON line carries
  * roofline: the covariance syrk (the dominant kernel; with --drift the drift statistic's
    kernel, 2 N d_in^2 flops per launch) timed by libkronq's hipEvent profiler on its own stream
    inside the timed region, algorithmic flops N d (d + 1) per launch, against the 2.5 PFLOP/s
    dense bf16 MFMA peak; HBM traffic from the committed rocprofv3 counter summary when it was
    taken on the current kernel source;
  * shared_covariance: when the two-stream schedule runs the H_G covariance on part of the chip
    beside the factorisation (a separately named launch of the same kernel), its time and its
    fraction of the peak of the CUs it held; the roofline then covers the whole-chip H_X launch;
  * cpu_baseline: the float64 oracle on this host's cores on a bounded sample (the covariances
    on the first --cpu-tokens tokens, scaled linearly to N; every other step at full size).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "seconds per layer quantised (cov+rotate+OBS) at 8B/70B shapes; % MFMA peak"
PEAK_BF16_TFLOPS = 2500.0
# fp32 FMAs on the vector units without packed instructions: 256 CUs x 4 SIMDs x 16 lanes x
# 2 flops x 2.4 GHz
PEAK_FP32_VALU = 78.6
PEAK_FP32_MFMA = 157.3  # dense fp32 matrix-core peak
PEAK_HBM_GBS = 8000.0
def traffic_file(kernel: str, workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"{kernel.replace('_mfma', '')}_{workload}_traffic.json")
WORKLOADS = {"q_proj": 2, "down_proj": 3, "up_proj_70b": 4}


def cov_source_hash() -> str:
    with open(os.path.join(ROOT, "paper_2607_07964_amd", "csrc", "cov.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic(kernel: str, workload: str):
    """HBM bytes per launch from the rocprofv3 FETCH_SIZE/WRITE_SIZE summary of this kernel on
    this workload (or None)."""
    path = traffic_file(kernel, workload)
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("cov_source_sha256_16") != cov_source_hash():
        return None  # counters were taken on another version of the kernel
    return float(t["bytes_per_launch"])


def cpu_baseline(spec, rot_in, rot_out, n_sample: int, X_dev, G_dev, W_dev, dX_dev=None,
                 alpha: float = 1.0, group: int = 128):
    import numpy as np
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))

    def view(t):
        t = t.cpu()
        return synth.bf16_bits(t) if str(t.dtype) == "torch.bfloat16" else t.numpy()

    Xs, Gs, W = view(X_dev[:n_sample]), view(G_dev[:n_sample]), view(W_dev)
    t0 = time.perf_counter()
    hx = O.covariance(Xs)
    hg = O.covariance(Gs)
    D = None if dX_dev is None else O.cross_covariance(view(dX_dev[:n_sample]), Xs)
    t_cov = time.perf_counter() - t0
    t1 = time.perf_counter()
    O.traces(hx, hg)
    b = O.biip_forward(W, hx, hg, (rot_in.sign, rot_in.q28), (rot_out.sign, rot_out.q28), D=D)
    O.traces(b["HX"], b["HG"])
    U = O.inverse_cholesky_factor(O.damp(b["HX"], spec.damp))
    P = None if D is None else O.gptaq_correction(b["D"], U, alpha)
    O.obs_blocked(b["W"], U, spec.bits, group, 128, P=P)
    t_rest = time.perf_counter() - t1
    scale = spec.n_tokens / n_sample
    return {
        "value": round(t_cov * scale + t_rest, 3), "unit": "s/layer", "cores": int(cores),
        "kind": "oracle", "blas": blas_vendor(),
        "sample": (f"float64 oracle: covariances{' and drift statistic' if D is not None else ''} "
                   f"on the first {n_sample} of {spec.n_tokens} tokens "
                   f"({t_cov:.2f} s, scaled x{scale:g}); traces, BiIP with dense rotations, "
                   f"factor{', P' if D is not None else ''} and blocked OBS sweep at full size "
                   f"({t_rest:.2f} s)"),
    }


def cpu_baseline_online(codes, scales, zeros, group, sx, sg, rot_in, rot_out, x):
    """The float64 oracle's decode matvec: dequantise the codes, then x -> V S_X^-1 x -> W_hat' .
    -> S_G^-1 U^T . with dense V and U (built once, outside the timing)."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))
    c, s, z = codes.cpu().numpy(), scales.cpu().numpy(), zeros.cpu().numpy()
    sx64, sg64 = sx.cpu().double().numpy(), sg.cpu().double().numpy()
    x64 = x.float().cpu().double().numpy().T
    V = O.rht_matrix(c.shape[1], rot_in.sign, rot_in.q28)
    U = O.rht_matrix(c.shape[0], rot_out.sign, rot_out.q28)
    reps = 3 if c.size <= 1 << 26 else 1  # about 2 s and 6 s per call at 4096^2 and 28672 x 8192
    t0 = time.perf_counter()
    for _ in range(reps):
        O.online_matvec(O.dequantize(c, s, z, group), sx64, sg64, V, U, x64)
    t = (time.perf_counter() - t0) / reps
    return {"value": round(t * 1e6, 1), "unit": "us", "cores": int(cores), "kind": "oracle",
            "sample": f"float64 oracle: dequantisation and the online matvec with dense V and U "
                      f"at full size, batch 1, mean of {reps} calls ({t * reps:.2f} s)"}


def online_bench(args, spec, dev) -> int:
    """Decode matvec of a quantised layer (online rotations + packed-code GEMV), batch 1."""
    import torch

    import synth
    from paper_2607_07964_amd import kronq as K
    from paper_2607_07964_amd import layer as L

    d_out, d_in, bits = spec.d_out, spec.d_in, spec.bits
    group = args.group if args.group > 0 else d_in
    g = torch.Generator(device=dev)
    g.manual_seed(spec.seed)
    codes = torch.randint(0, 2 ** bits, (d_out, d_in), generator=g, device=dev, dtype=torch.uint8)
    scales = torch.rand(d_out, d_in // group, generator=g, device=dev) * 0.01 + 0.005
    zeros = torch.randint(0, 2 ** bits, (d_out, d_in // group), generator=g,
                          device=dev).float()
    ri = synth.rotation_params(d_in, spec.seed, spec.name + ":in")
    ro = synth.rotation_params(d_out, spec.seed, spec.name + ":out")
    rin = L.RotParams.to_device(ri.sign, ri.q28, dev)
    rout = L.RotParams.to_device(ro.sign, ro.q28, dev)
    sx = torch.rand(d_in, generator=g, device=dev) + 0.5
    sg = torch.rand(d_out, generator=g, device=dev) + 0.5
    mul_in = K.kronq_online_factors(sx, rin.sign, d_in)
    mul_out = K.kronq_online_factors(sg, rout.sign, d_out)
    packed = K.kronq_pack_codes(codes, bits)
    x = torch.randn(1, d_in, generator=g, device=dev).to(torch.bfloat16)
    y = torch.empty(1, d_out, device=dev)
    ws = K.workspace(K.OP_ONLINE, d_out, d_in, 1, dev)
    Wd = torch.randn(d_out, d_in, generator=g, device=dev).to(torch.bfloat16)  # dense baseline

    def step():
        K.kronq_online_matvec(packed, scales, zeros, bits, group, d_in, mul_in, mul_out, rin.q28,
                              rout.q28, x, y, ws=ws)

    def timed(fn, n):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    reps = max(args.steps, 1) * 100
    warm = max(args.warmup, 1) * 20
    for _ in range(warm):
        step()
    K.kronq_profile_only("online_gemv")
    K.kronq_profile_reset()
    K.kronq_profile_enable(True)
    timed(step, reps)
    K.kronq_profile_enable(False)
    g_ms, g_n = K.kronq_profile_read("online_gemv")
    gemv_ms = g_ms / max(g_n, 1)
    ms = timed(step, reps)  # without the profiler's events around the GEMV
    for _ in range(warm):
        torch.nn.functional.linear(x, Wd)
    dense_ms = timed(lambda: torch.nn.functional.linear(x, Wd), reps)
    # algorithmic HBM bytes of the GEMV kernel: packed codes, scales and zeros, x' and y'
    gbytes = d_out * d_in * bits / 8 + 2 * 4 * d_out * (d_in // group) + 4 * d_in + 4 * d_out
    achieved = gbytes / (gemv_ms * 1e-3) / 1e9
    int_path = bits in (2, 4)  # the GEMV on integer dot products; 3- and 8-bit codes use fp32
    gemv_kernel = "online_gemv_p" if int_path else "online_gemv"  # one vector: persistent
    print(f"[bench] online matvec {ms * 1e3:.2f} us (GEMV kernel {gemv_ms * 1e3:.2f} us), "
          f"dense bf16 GEMV {dense_ms * 1e3:.2f} us", file=sys.stderr, flush=True)
    out = {
        "metric": "microseconds per decode matvec of a quantised layer (online rotations + "
                  "packed-code GEMV, batch 1)",
        "value": round(ms * 1e3, 3), "unit": "us", "n_gpus": 1, "steps": reps, "warmup": warm,
        "ms_per_step": round(ms, 6), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": (f"u{bits} codes, i8 dot products (21-bit fixed-point "
                                        f"activations) with fp32 combine" if int_path else
                                        f"u{bits} codes, fp32 arithmetic"), "data": "synthetic",
        "config": {"workload": f"{spec.name} W {d_out}x{d_in}, {bits}-bit, group {group}, "
                               f"decode batch 1", "d_out": d_out, "d_in": d_in, "bits": bits,
                   "group": group, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": 8000.0,
                     "unit": "GB/s", "frac": round(achieved / 8000.0, 4), "traffic": None,
                     "kernel": gemv_kernel,
                     "launches": g_n,
                     "avg_launch_ms": round(gemv_ms, 6)},
        "dense_bf16_gemv_us": round(dense_ms * 1e3, 3),
        "speedup_vs_dense_bf16": round(dense_ms / ms, 3),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_online(codes, scales, zeros, group, sx, sg, ri, ro, x)
    print(json.dumps(out), flush=True)
    return 0


def diag_bench(args, spec, dev) -> int:
    """The layer's incoherence diagnostics (Sec. 2.3, Fig. 2, Prop. 2) on resident statistics."""
    import torch

    import synth
    from paper_2607_07964_amd import kronq as K
    from paper_2607_07964_amd import layer as L

    d_out, d_in = spec.d_out, spec.d_in
    print(f"[bench] diagnostics setup {spec.name}: W {d_out}x{d_in}, N={spec.n_tokens}",
          file=sys.stderr, flush=True)
    X = synth.gen_matrix(spec.x, dev)
    G = synth.gen_matrix(spec.g, dev)
    W0 = synth.gen_matrix(spec.w, dev)
    ri = synth.rotation_params(d_in, spec.seed, spec.name + ":in")
    ro = synth.rotation_params(d_out, spec.seed, spec.name + ":out")
    rin = L.RotParams.to_device(ri.sign, ri.q28, dev)
    rout = L.RotParams.to_device(ro.sign, ro.q28, dev)
    st = L.LayerState.allocate(d_out, d_in, spec.n_tokens, dev)
    L.covariances(st, X, G)
    del X, G
    HX0, HG0 = st.HX.clone(), st.HG.clone()
    W_in = torch.empty(d_out, d_in, device=dev)  # input-side processing only (Fig. 2b middle)
    sx, sg = torch.empty(d_in, device=dev), torch.empty(d_out, device=dev)
    K.kronq_rotate(W0, W_in, st.HX.clone(), None, rin.sign, None, rin.q28, None, sx, sg,
                   K.RESCALE_IN | K.ROT_IN, st.ws_rot)
    L.biip(st, W0, rin, rout)
    HX1, HG1 = st.HX.clone(), st.HG.clone()
    K.kronq_cholesky_inv(st.HX, st.U, spec.damp, st.info, st.ws_chol)  # st.HX: damped H~
    L.check(st)
    alphas = (0.0, 0.125, 0.25, 0.375, 0.5)
    dmax = max(d_in, d_out)
    ws_e = K.workspace(K.OP_EIGH, 0, dmax, 0, dev)
    ws_s = K.workspace(K.OP_STATS, max(d_out, dmax), max(d_in, dmax), 0, dev)
    ws_p = K.workspace(K.OP_PROXY, d_out, d_in, 0, dev)
    Qs = {d: torch.empty(d, d, device=dev) for d in {d_in, d_out}}
    ev = {d: torch.empty(d, device=dev) for d in {d_in, d_out}}
    stats = {k: torch.empty(5, dtype=torch.float64, device=dev)
             for k in ("W0", "W_in", "W_biip", "HX0", "HG0", "HX1", "HG1")}
    offs = {k: torch.empty(1, dtype=torch.float64, device=dev) for k in ("HX0", "HG0", "HX1", "HG1")}
    proxy = torch.empty(6 + len(alphas), dtype=torch.float64, device=dev)
    hs = {"HX0": HX0, "HG0": HG0, "HX1": HX1, "HG1": HG1}
    torch.cuda.synchronize()

    def step():
        for k, M in (("W0", W0), ("W_in", W_in), ("W_biip", st.W)):
            K.kronq_matrix_stats(M, stats[k], ws_s)
        for k, H in hs.items():
            d = H.shape[0]
            K.kronq_eigh(H, args.sweeps, ev[d], Qs[d], offs[k], ws_e)
            K.kronq_matrix_stats(Qs[d], stats[k], ws_s)
        K.kronq_proxy_loss_factors(HG0, W0, st.HX, st.U, alphas, proxy, ws_p)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    dom = "diag_bjac_apply"
    K.kronq_profile_only(dom)
    K.kronq_profile_reset()
    K.kronq_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    K.kronq_profile_enable(False)
    dom_ms, dom_n = K.kronq_profile_read(dom)
    ms = (t1 - t0) * 1e3 / max(args.steps, 1)
    avg_ms = dom_ms / max(dom_n, 1)
    # algorithmic flops of one block-Jacobi round (order N, N/64 block pairs): Z_y^T A_tile Z_x
    # for every (N/64)^2 tile of A (2 x 2 x 64^3) and V_tile Z_x for every (N/64)^2 tile of V
    # (2 x 64^3), averaged over the launches of the four eigendecompositions (two of order
    # d_in, two of order d_out)
    def round_flops(d):
        t = -(-d // 64)
        return t * t * 6.0 * 64 ** 3
    flops = (round_flops(d_in) + round_flops(d_out)) / 2
    achieved = flops / (avg_ms * 1e-3) / 1e12
    st_np = {k: v.cpu().tolist() for k, v in stats.items()}
    pr = proxy.cpu().tolist()
    diag = {
        "mu_W": {k: round(st_np[k][2], 4) for k in ("W0", "W_in", "W_biip")},
        "cv_in": {k: round(st_np[k][3], 4) for k in ("W0", "W_in", "W_biip")},
        "cv_out": {k: round(st_np[k][4], 4) for k in ("W0", "W_in", "W_biip")},
        "mu_H_over_sqrt_d": {k: round(st_np[k][0], 4) for k in hs},  # max |Q_ij|
        "eigh_offdiag_rel": {k: float(f"{v.item():.3g}") for k, v in offs.items()},
        "proxy_factors": {"nearest": pr[0], "gptq": pr[1], "kronq": pr[2], "rho": pr[3]},
        "rescale_sweep": {str(a): pr[6 + i] / pr[1] for i, a in enumerate(alphas)},
    }
    print(f"[bench] diagnostics pass {ms:.1f} ms; " + json.dumps(diag), file=sys.stderr, flush=True)
    out = {
        "metric": "seconds per layer diagnostic pass (mu(W), CV_in/CV_out for three weight "
                  "states, mu(H_X), mu(H_G) before/after BiIP by Jacobi eigendecomposition, "
                  "expected-loss factors)",
        "value": round(ms / 1e3, 4), "unit": "s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None,
        "dtype": "fp32 (rotations), fp64 (sums)", "data": "synthetic",
        "config": {"workload": f"{spec.name} W {d_out}x{d_in}, N={spec.n_tokens}, "
                               f"{args.sweeps} Jacobi sweeps", "d_out": d_out, "d_in": d_in,
                   "sweeps": args.sweeps, "parallelism": "single GPU"},
        "roofline": {"bound": "alu", "achieved": round(achieved, 2), "peak": PEAK_FP32_VALU,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_VALU, 4),
                     "traffic": None, "kernel": dom, "launches": dom_n,
                     "avg_launch_ms": round(avg_ms, 5)},
        "diagnostics": diag,
    }
    if not args.no_cpu_baseline:
        import numpy as np

        import oracle as O
        try:
            from threadpoolctl import threadpool_info
            cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        except Exception:  # pragma: no cover
            cores = len(os.sched_getaffinity(0))
        print("[bench] timing the float64 oracle's diagnostics on the host", file=sys.stderr,
              flush=True)
        w0 = synth.bf16_bits(W0.cpu()) if W0.dtype == torch.bfloat16 else W0.cpu().numpy()
        mats = [w0, W_in.cpu().numpy(), st.W.cpu().numpy()]
        hcpu = [h.cpu().numpy() for h in hs.values()]
        hg0, hd, u = HG0.cpu().numpy(), st.HX.cpu().numpy(), st.U.cpu().numpy()
        t0 = time.perf_counter()
        for M in mats:
            O.incoherence(M)
            O.norm_cv(M)
        for H in hcpu:
            O.hessian_incoherence(H)
        f = O.proxy_loss_factors(hg0, w0, hd, u)
        for a in alphas:
            O.rescale_objective(np.diag(hg0), np.sum(O.as_f64(w0) ** 2, axis=1), a)
        t = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(t, 3), "unit": "s", "cores": int(cores),
                               "kind": "oracle",
                               "sample": "float64 oracle: the whole diagnostic pass at full size "
                                         "(LAPACK eigh for the four eigendecompositions)"}
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="q_proj")
    ap.add_argument("--cpu-tokens", type=int, default=16384)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--breakdown", action="store_true",
                    help="add the per-kernel times of the profiled single-stream step")
    ap.add_argument("--no-70b", action="store_true",
                    help="leave out the 70B up_proj entry timed after the main workload")
    ap.add_argument("--steps-70b", type=int, default=3, help="timed steps of the 70B entry")
    ap.add_argument("--serial", action="store_true",
                    help="time the single-stream schedule instead of the two-stream one")
    ap.add_argument("--cov-cus", type=int, default=-1,
                    help="CUs of the H_G covariance in the two-stream schedule (0: no cap; "
                         "default: the library's policy)")
    ap.add_argument("--drift", action="store_true",
                    help="the drift-corrected path (KronQ+GPTAQ) with synthetic input drift")
    ap.add_argument("--alpha", type=float, default=1.0, help="drift correction scaling")
    ap.add_argument("--group", type=int, default=128,
                    help="quantisation group (a multiple of 128 dividing d_in; 0: per-channel)")
    ap.add_argument("--online", action="store_true",
                    help="time the inference-side decode matvec of the quantised layer instead")
    ap.add_argument("--diagnostics", action="store_true",
                    help="time the incoherence diagnostics of the layer instead")
    ap.add_argument("--sweeps", type=int, default=12, help="Jacobi sweeps (--diagnostics)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run 3 plain 1 GiB device copies (reference for counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the layer solve has no multi-GPU path; "
              "--gpus above 1 is not supported.", file=sys.stderr)
        return 2

    import torch

    import synth
    from paper_2607_07964_amd import kronq as K
    from paper_2607_07964_amd import layer as L

    K.load()
    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        print("[bench] calibration copies done: 3 x 1 GiB", file=sys.stderr, flush=True)
    spec = synth.workload(WORKLOADS[args.workload])
    if args.online:
        return online_bench(args, spec, dev)
    if args.diagnostics:
        return diag_bench(args, spec, dev)
    out = layer_bench(args, spec, dev, args.steps, args.warmup, args.cpu_tokens)
    if args.workload != "up_proj_70b" and not args.no_70b and not args.drift:
        # the 70B-shaped layer in the same run: a few timed steps with its own roofline and a
        # bounded oracle sample
        spec70 = synth.workload(WORKLOADS["up_proj_70b"])
        torch.cuda.empty_cache()
        out["up_proj_70b"] = layer_bench(args, spec70, dev, args.steps_70b, 1, 1024,
                                         brief=True)
    print(json.dumps(out), flush=True)
    return 0


# Stages of the layer (SURVEY-style rows a1-a8) by kernel-name prefix, for the profiled
# breakdown; the first matching prefix wins.
STAGES = (
    ("cov_diag", ("cov_diag_",)),
    ("covariances", ("syrk_", "cov_scale")),
    ("drift_statistic", ("cross_",)),
    ("traces", ("traces",)),
    ("biip", ("rot_", "fwht_", "mix28_")),
    ("factor", ("chol_", "trtri_")),
    ("gptaq", ("gptaq_", "obs_split_p")),
    ("obs_sweep", ("obs_sweep", "obs_group_params")),
    ("obs_update", ("obs_trailing_update", "obs_split_u")),
)


def stage_of(kernel: str) -> str:
    for name, prefixes in STAGES:
        if any(kernel.startswith(p) for p in prefixes):
            return name
    return "other"


def stage_work(spec, drift: bool) -> dict:
    """Algorithmic work per layer of each stage and the roofline it is held to: (amount, unit,
    peak). Covariances N d (d + 1) flops each on bf16 MFMA; diag(H_G) one read of G; BiIP
    2 passes x (read + write) x 4 B over W, H_X, H_G (the ideal is one pass); factor d^3 / 3 +
    d^3 / 3 fp32 flops; sweep 9 B per weight; trailing update d_out d_in (d_in - 1) flops (bf16
    MFMA, the algorithmic count of the fp32-accurate product)."""
    n, do, di = float(spec.n_tokens), float(spec.d_out), float(spec.d_in)
    w = {
        "cov_diag": (2.0 * n * do, "B", PEAK_HBM_GBS * 1e9),
        "covariances": (n * di * (di + 1) + n * do * (do + 1), "flop", PEAK_BF16_TFLOPS * 1e12),
        "biip": (2 * 2 * 4.0 * (do * di + di * di + do * do), "B", PEAK_HBM_GBS * 1e9),
        "factor": (2.0 * di ** 3 / 3.0, "flop", PEAK_FP32_MFMA * 1e12),
        "obs_sweep": (9.0 * do * di, "B", PEAK_HBM_GBS * 1e9),
        "obs_update": (do * di * (di - 1), "flop", PEAK_BF16_TFLOPS * 1e12),
    }
    if drift:
        w["drift_statistic"] = (2.0 * n * di * di, "flop", PEAK_BF16_TFLOPS * 1e12)
        w["gptaq"] = (2.0 * di ** 3 / 3.0, "flop", PEAK_FP32_MFMA * 1e12)
    return w


def blas_vendor() -> str:
    import numpy as np
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        return f"{b.get('name')} {b.get('version')}"
    except Exception:  # pragma: no cover
        return "unknown"


def cpu_baseline_70b(spec, rot_in, rot_out, n_sample: int, X_dev, G_dev, W_dev,
                     row_sample: int = 512, panel: int = 1024):
    """The float64 oracle on a bounded sample of the 70B-shaped layer, each part scaled
    linearly to the full layer: covariances of X and G on the first ``n_sample`` tokens (x N /
    n_sample); the dense rotation of H_G timed on a ``panel``-column slice of both products
    (x d_out / panel); the rotation of H_X, the factor, at full size; the blocked sweep of
    ``row_sample`` rows of the rotated W (x d_out / row_sample)."""
    import numpy as np
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))

    def view(t):
        t = t.cpu()
        return synth.bf16_bits(t) if str(t.dtype) == "torch.bfloat16" else t.numpy()

    Xs, Gs, W = view(X_dev[:n_sample]), view(G_dev[:n_sample]), O.as_f64(view(W_dev))
    ri = (rot_in.sign, rot_in.q28)
    ro = (rot_out.sign, rot_out.q28)
    t0 = time.perf_counter()
    hx = O.covariance(Xs)
    hg = O.covariance(Gs)
    t_cov = time.perf_counter() - t0
    rows = np.arange(row_sample)
    t1 = time.perf_counter()
    O.traces(hx, hg)
    b = O.biip_forward_rows(W, hx, np.diag(hg), ri, ro, rows)
    U = O.inverse_cholesky_factor(O.damp(b["HX"], spec.damp))
    t_mid = time.perf_counter() - t1
    t2 = time.perf_counter()
    O.obs_blocked(b["W_rows"], U, spec.bits, 128, 128)
    t_sweep = time.perf_counter() - t2
    # U H_G' U^T on a panel of columns: (U (H_G' Ut[:, panel])) with the dense U
    Ud = O.rht_matrix(spec.d_out, *ro)
    hg1 = hg / np.outer(b["sg"], b["sg"])
    t3 = time.perf_counter()
    Ud @ (hg1 @ Ud[:panel].T)
    t_rot = time.perf_counter() - t3
    n_scale, r_scale, p_scale = spec.n_tokens / n_sample, spec.d_out / row_sample, \
        spec.d_out / panel
    total = t_cov * n_scale + t_mid + t_sweep * r_scale + t_rot * p_scale
    return {
        "value": round(total, 3), "unit": "s/layer", "cores": int(cores), "kind": "oracle",
        "blas": blas_vendor(),
        "sample": (f"float64 oracle, each part scaled linearly: covariances of X and G on the "
                   f"first {n_sample} of {spec.n_tokens} tokens ({t_cov:.2f} s, x{n_scale:g}); "
                   f"BiIP of H_X with dense V, factor and traces at full size ({t_mid:.2f} s); "
                   f"dense U H_G U^T on {panel} of {spec.d_out} columns ({t_rot:.2f} s, "
                   f"x{p_scale:g}); blocked sweep of {row_sample} of {spec.d_out} rows "
                   f"({t_sweep:.2f} s, x{r_scale:g})"),
    }


def measured_peaks(X, dev) -> dict:
    """The chip's measured ceilings next to the data-sheet figures: the bf16 MFMA rate of a
    register-resident loop (kronq_probe_mfma_bf16) on the workload's own input values (the clock
    is power-limited under MFMA load, and the limit depends on the data), and a plain 1 GiB
    device copy (read + write bytes)."""
    import torch
    from paper_2607_07964_amd import kronq as K
    out = {}
    data = X.reshape(-1)[:4096].contiguous()
    chk = torch.empty(2048, device=dev)
    iters = 20000
    K.kronq_probe_mfma_bf16(data, 200, chk)  # warm-up
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = None
    for _ in range(3):
        e0.record()
        wgs = K.kronq_probe_mfma_bf16(data, iters, chk)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    tf = wgs * 4.0 * iters * 8 * 32768 / (best * 1e-3) / 1e12
    out["bf16_mfma_tflops"] = round(tf, 1)
    out["bf16_mfma_frac_of_spec"] = round(tf / PEAK_BF16_TFLOPS, 4)
    out["bf16_mfma_data"] = "the first 4096 bf16 values of X"
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 5 * 2 * src.numel() * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    out["hbm_copy_gbs"] = round(gbs, 1)
    out["hbm_copy_frac_of_spec"] = round(gbs / PEAK_HBM_GBS, 4)
    del src, dst
    return out


def layer_bench(args, spec, dev, steps: int, warmup: int, cpu_tokens: int,
                brief: bool = False) -> dict:
    """Seconds per layer of one workload: ``warmup`` untimed steps, ``steps`` timed steps
    (HIP events per step on the issuing stream, and the host clock around all of them), the
    covariance launches timed by libkronq's profiler inside the timed region, then one profiled
    single-stream step for the per-stage breakdown, then the oracle's bounded sample."""
    import torch

    import synth
    from paper_2607_07964_amd import kronq as K
    from paper_2607_07964_amd import layer as L

    print(f"[bench] generating {spec.name}: W {spec.d_out}x{spec.d_in}, N={spec.n_tokens}",
          file=sys.stderr, flush=True)
    X = synth.gen_matrix(spec.x, dev)
    G = synth.gen_matrix(spec.g, dev)
    W0 = synth.gen_matrix(spec.w, dev)
    dX = synth.gen_drift(spec, dev, X=X) if args.drift else None
    ri = synth.rotation_params(spec.d_in, spec.seed, spec.name + ":in")
    ro = synth.rotation_params(spec.d_out, spec.seed, spec.name + ":out")
    rin = L.RotParams.to_device(ri.sign, ri.q28, dev)
    rout = L.RotParams.to_device(ro.sign, ro.q28, dev)
    group = args.group if args.group > 0 else spec.d_in
    st = L.LayerState.allocate(spec.d_out, spec.d_in, spec.n_tokens, dev, x_dtype=X.dtype,
                               g_dtype=G.dtype, group=group, drift=args.drift)
    dominant = "cross_bf16_mfma" if args.drift else "syrk_bf16_mfma"
    torch.cuda.synchronize()

    cov_cus = None if args.cov_cus < 0 else args.cov_cus

    def step(overlap=not args.serial):
        L.quantize_layer(st, X, G, W0, rin, rout, spec.bits, spec.damp, overlap=overlap, dX=dX,
                         alpha=args.alpha, cov_cus=cov_cus)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    L.check(st)
    print(f"[bench] {spec.name}: warmup done ({warmup} steps)", file=sys.stderr, flush=True)

    SHARED = "syrk_bf16_mfma_shared"  # the H_G covariance on part of the chip (two streams)
    K.kronq_profile_only(f"{dominant},{SHARED}")
    K.kronq_profile_reset()
    K.kronq_profile_enable(True)
    main = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(main)
    for i in range(steps):
        step()
        evs[i + 1].record(main)  # the step ends with the issuing stream waiting for the other
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    K.kronq_profile_enable(False)
    dom_ms, dom_n = K.kronq_profile_read(dominant)
    sh_ms, sh_n = K.kronq_profile_read(SHARED)
    L.check(st)
    ms_step = (t1 - t0) * 1e3 / steps
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    med = sorted(per_step)[steps // 2] if steps % 2 else \
        0.5 * sum(sorted(per_step)[steps // 2 - 1:steps // 2 + 1])
    print(f"[bench] {spec.name}: timed {steps} steps: {ms_step:.3f} ms/step "
          f"(median {med:.3f})", file=sys.stderr, flush=True)
    # the chip's measured ceilings, after the timed steps: the register-resident MFMA loop runs
    # the chip at its power limit, which left the first timed step after it slower
    peaks = None if brief else measured_peaks(X, dev)

    # dominant kernel roofline: algorithmic flops N d (d + 1) per covariance launch (averaged
    # over the covariances run on the whole chip: both, or H_X alone when H_G ran beside the
    # factorisation on part of the chip), 2 N d_in^2 for the drift statistic
    fl_x = float(spec.n_tokens) * spec.d_in * (spec.d_in + 1)
    fl_g = float(spec.n_tokens) * spec.d_out * (spec.d_out + 1)
    if args.drift:
        flops = 2.0 * spec.n_tokens * spec.d_in * spec.d_in
    else:
        flops = fl_x if sh_n else (fl_x + fl_g) / 2
    avg_ms = dom_ms / max(dom_n, 1)
    achieved = flops / (avg_ms * 1e-3) / 1e12
    wl_key = next((k for k, v in WORKLOADS.items() if synth.workload(v).name == spec.name),
                  spec.name)
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic(dominant, wl_key), "kernel": dominant, "launches": dom_n,
            "avg_launch_ms": round(avg_ms, 4)}
    if args.drift:
        # the drift statistic holds part of the chip (layer.DRIFT_SHARE) beside the solver
        ncu = torch.cuda.get_device_properties(dev).multi_processor_count
        held = max(8, int(ncu * L.DRIFT_SHARE)) // 8 * 8
        roof["held_cus"] = held
        roof["frac_of_its_cus"] = round(achieved / (PEAK_BF16_TFLOPS * held / ncu), 4)
    shared = None
    if sh_n:
        cus = cov_cus if cov_cus is not None else L._cov_cus(dev, spec.n_tokens, spec.d_out,
                                                              spec.d_in)
        sh_avg = sh_ms / sh_n
        sh_tf = fl_g / (sh_avg * 1e-3) / 1e12
        ncu = torch.cuda.get_device_properties(dev).multi_processor_count
        part_peak = PEAK_BF16_TFLOPS * cus / ncu
        shared = {"kernel": SHARED, "cus": cus, "launches": sh_n, "avg_launch_ms": round(sh_avg, 4),
                  "achieved": round(sh_tf, 2), "frac_of_chip": round(sh_tf / PEAK_BF16_TFLOPS, 4),
                  "peak_of_its_cus": round(part_peak, 1),
                  "frac_of_its_cus": round(sh_tf / part_peak, 4)}

    # per-stage breakdown: one profiled single-stream step (every launch bracketed by events)
    K.kronq_profile_only(None)
    K.kronq_profile_reset()
    K.kronq_profile_enable(True)
    step(overlap=False)
    torch.cuda.synchronize()
    K.kronq_profile_enable(False)
    kern = {}
    for k in K.kronq_profile_names():
        ms, n = K.kronq_profile_read(k)
        if n:
            kern[k] = {"ms": round(ms, 4), "launches": n}
    K.kronq_profile_reset()
    work = stage_work(spec, bool(args.drift))
    stages = {}
    for k, v in kern.items():
        sname = stage_of(k)
        stages.setdefault(sname, 0.0)
        stages[sname] += v["ms"]
    bound_ms = 0.0
    stage_out = {}
    for sname, ms in stages.items():
        ent = {"ms": round(ms, 4)}
        if sname in work:
            amount, unit, peak = work[sname]
            b_ms = amount / peak * 1e3
            if sname != "cov_diag":  # diag(H_G) is part of H_G's work: read early, not extra
                bound_ms += b_ms
            rate = amount / (ms * 1e-3)
            ent.update({"bound_ms": round(b_ms, 4), "frac": round(b_ms / ms, 4),
                        ("TFLOP/s" if unit == "flop" else "GB/s"):
                            round(rate / (1e12 if unit == "flop" else 1e9), 2)})
        stage_out[sname] = ent
    if peaks is not None:
        roof["frac_of_measured_peak"] = round(achieved / peaks["bf16_mfma_tflops"], 4)
    roof["layer_bound_ms"] = round(bound_ms, 4)
    roof["layer_frac"] = round(bound_ms / med, 4)
    print(f"[bench] {spec.name}: stages (one single-stream step) " + json.dumps(stage_out),
          file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        print(f"[bench] {spec.name}: timing the float64 oracle on the host (bounded sample)",
              file=sys.stderr, flush=True)
        if spec.d_out > 16384:
            cpu = cpu_baseline_70b(spec, ri, ro, min(cpu_tokens, spec.n_tokens), X, G, W0)
        else:
            cpu = cpu_baseline(spec, ri, ro, min(cpu_tokens, spec.n_tokens), X, G, W0, dX,
                               args.alpha, group)
    sched = L.schedule(st, spec.n_tokens, not args.serial, cov_cus)
    del X, G, W0, dX, st

    out = {
        "metric": METRIC, "value": round(ms_step / 1e3, 6), "unit": "s/layer", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_step, 4),
        "ms_median": round(med, 4), "step_ms": [round(x, 4) for x in per_step],
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 (covariances, MFMA) + fp32 (rotations, factor, OBS)", "data": "synthetic",
        "config": {"workload": f"{spec.name} W {spec.d_out}x{spec.d_in}, N={spec.n_tokens} tokens, "
                               f"{spec.bits}-bit, group {group}"
                               + (f", drift correction (alpha {args.alpha:g})" if args.drift else ""),
                   "d_out": spec.d_out, "d_in": spec.d_in, "n_tokens": spec.n_tokens,
                   "bits": spec.bits, "group": group, "block": 128, "damp": spec.damp,
                   "drift": bool(args.drift),
                   "parallelism": "single GPU",
                   "schedule": sched},
        "roofline": roof, "cpu_baseline": cpu,
    }
    if shared is not None:
        out["shared_covariance"] = shared
    out["stages_single_stream"] = stage_out
    if peaks is not None:
        out["measured_peaks"] = peaks
    if args.breakdown:
        out["kernels_ms"] = kern
    if brief:
        for k in ("metric", "n_gpus", "higher_is_better", "scaling", "vs_baseline", "dtype",
                  "data"):
            out.pop(k, None)
    return out


if __name__ == "__main__":
    sys.exit(main())
