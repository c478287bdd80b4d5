"""Helpers for the GPU parity tests: put seeded workloads into device pools,
run the C-ABI calls, bring results back as raw bf16 bit patterns, and
compare against the oracle."""

import numpy as np
import pytest

from paper_2606_16135_amd.torch_pool import DevicePool, from_u16, new_active, to_u16  # noqa: F401

ATOL = 2e-2
RTOL = 1e-2
# Relative L2 bound: bf16 rounding of the output (<= 2^-9 relative per
# element) plus bf16 rounding of the probabilities before the PV product
# (<= 2^-9 relative per weight, averaging out over the keys).
REL_L2 = 1e-2


def torch_mod():
    import torch
    return torch


def require_gpu():
    torch = torch_mod()
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_16135_amd import swiftcache as sc
    sc.load()
    return sc


def bits_to_f64(a, dtype="bf16"):
    from oracle.attention import bits_to_f64 as conv
    return conv(a, dtype)


def compare_attention(gpu_bits, ref, what="", dtype="bf16"):
    """Element-wise |gpu - ref| <= ATOL + RTOL |ref| on every element, no NaN,
    and relative L2 below REL_L2.  Returns the error statistics."""
    g = bits_to_f64(gpu_bits, dtype)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    err = np.abs(g - ref)
    bound = ATOL + RTOL * np.abs(ref)
    bad = err > bound
    rel_l2 = float(np.linalg.norm(g - ref) / max(np.linalg.norm(ref), 1e-30))
    stats = dict(max_abs=float(err.max()) if err.size else 0.0, rel_l2=rel_l2, n_bad=int(bad.sum()))
    assert not bad.any(), f"{what}: {stats}"
    assert rel_l2 <= REL_L2, f"{what}: {stats}"
    return stats
