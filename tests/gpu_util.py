"""Helpers shared by the GPU parity tests: upload seeded bf16 inputs, run the
HIP path through the C ABI, and compare with the float64 oracle."""

from __future__ import annotations

import numpy as np

from paper_2608_07524_amd import inputs as I

# Tolerances (derivations in oracle/tolerances.py).
from oracle.tolerances import BF16_U, GRAD_TOL, LSE_TOL, O_TOL  # noqa: F401


def to_device(torch, bits: np.ndarray, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def to_bits(t) -> np.ndarray:
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def grad_err(got_bits: np.ndarray, ref: np.ndarray) -> float:
    got = I.bf16_to_f64(got_bits)
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))


def max_abs(got_bits: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(I.bf16_to_f64(got_bits) - ref)))


def o_excess(got_bits: np.ndarray, ref: np.ndarray) -> float:
    """Largest |O_gpu - O_ref| beyond the bf16 store rounding of O_ref
    (compared with O_TOL)."""
    got = I.bf16_to_f64(got_bits)
    return float(np.max(np.abs(got - ref) - BF16_U * np.abs(ref)))
