"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import sys

import numpy as np
import torch

import synth

DEV = "cuda:0"


def note(msg: str):
    """Name the case before a GPU step (flushed, so it survives a crash)."""
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def rel_frob(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def oracle_view(t_cpu: torch.Tensor) -> np.ndarray:
    """Generator output (CPU tensor) in the form the oracle reads: bf16 bit patterns or floats."""
    if t_cpu.dtype == torch.bfloat16:
        return synth.bf16_bits(t_cpu)
    return t_cpu.numpy()


def rot_device(rot: synth.Rot):
    from paper_2607_07964_amd.layer import RotParams
    return RotParams.to_device(rot.sign, rot.q28, DEV)


def rot_oracle(rot: synth.Rot):
    """(sign, q28) exactly as the GPU receives them (the fp32-rounded 28 x 28 factor)."""
    return rot.sign.astype(np.float64), (None if rot.q28 is None else rot.q28.astype(np.float64))
