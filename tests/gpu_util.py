"""Helpers for the GPU parity tests: device tensors from the seeded inputs, the ring
driver through the C ABI, and comparisons at the stated tolerances."""
from __future__ import annotations

import numpy as np
import torch

from paper_2609_34318_amd import inputs

# Tolerances for bf16 inputs with fp32 accumulation.
TOL_O = 1e-2        # max |dO| over finite elements of the merged O (fp32 and its bf16 cast)
TOL_LSE = 1e-3      # max |dLSE| over finite entries; -inf must match exactly
TOL_GRAD = 2e-2     # relative L2 of dQ, dK, dV


def dev_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def f32(bits: np.ndarray) -> np.ndarray:
    return inputs.bf16_bits_to_f32(bits)


def assert_lse_close(got: np.ndarray, ref: np.ndarray, tol=TOL_LSE, what="LSE"):
    got = np.asarray(got, dtype=np.float64)
    ninf_g, ninf_r = np.isneginf(got), np.isneginf(ref)
    assert np.array_equal(ninf_g, ninf_r), f"{what}: -inf pattern differs at {np.argwhere(ninf_g != ninf_r)[:5]}"
    assert np.isfinite(got[~ninf_g]).all(), f"{what}: non-finite values"
    err = np.abs(got[~ninf_g] - ref[~ninf_r]).max(initial=0.0)
    assert err <= tol, f"{what}: max |err| {err:.3e} > {tol}"
    return err


def assert_o_close(got: np.ndarray, ref: np.ndarray, tol=TOL_O, what="O"):
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    err = np.abs(got - ref).max(initial=0.0)
    assert err <= tol, f"{what}: max |err| {err:.3e} > {tol}"
    return err


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def worst_head_rel_l2(got, ref):
    """Largest per-head relative L2 of [rows, heads, dim] tensors (None for other shapes)."""
    got, ref = np.asarray(got, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    if got.ndim != 3 or got.shape != ref.shape:
        return None
    worst = 0.0
    for h in range(got.shape[1]):
        n = np.linalg.norm(ref[:, h])
        if n > 0:
            worst = max(worst, np.linalg.norm(got[:, h] - ref[:, h]) / n)
    return worst


def assert_grad_close(got, ref, tol=TOL_GRAD, what="grad"):
    """Relative L2 over the whole tensor (all heads) within tol; the message also names the
    worst head's relative L2."""
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    e = rel_l2(got, ref)
    assert e <= tol, f"{what}: relative L2 {e:.3e} > {tol} (worst head {worst_head_rel_l2(got, ref)})"
    return e
