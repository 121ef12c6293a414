"""Shared helpers of the GPU parity tests."""

import sys

import numpy as np
import torch

# Tolerances: fp32 inputs, relative L2 <= 1e-5 per output tensor; bf16 inputs,
# max-abs <= 2e-2 and relative L2 <= 1e-2 (both must hold).
FP32_REL_L2 = 1e-5
BF16_MAX_ABS = 2e-2
BF16_REL_L2 = 1e-2


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def f64(t: torch.Tensor) -> np.ndarray:
    """Exact host copy of a device tensor's values (bf16 -> float64 is exact)."""
    return t.detach().to("cpu").to(torch.float64).numpy()


def errors(got: np.ndarray, ref: np.ndarray):
    err = got - ref
    return float(np.max(np.abs(err))), float(np.linalg.norm(err) / np.linalg.norm(ref))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even to bfloat16 (via torch), back to float64."""
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def assert_close(got, ref, in_dtype, what="", out_bf16=False):
    """Parity check at the stated tolerance.  A bf16 output is compared with
    the reference rounded to bf16 the same way (the output type's own rounding
    is not an error of the computation)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if out_bf16:
        ref = round_bf16(ref)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    max_abs, rel = errors(got, ref)
    log(f"  {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e}")
    if in_dtype == torch.float32:
        assert rel <= FP32_REL_L2, (what, rel)
    else:
        assert max_abs <= BF16_MAX_ABS and rel <= BF16_REL_L2, (what, max_abs, rel)


def f64_dev(t: torch.Tensor) -> np.ndarray:
    """Like f64, with the (exact) widening done on the device before the copy:
    faster for the multi-GB tensors of the full-size workloads."""
    return t.detach().to(torch.float64).to("cpu").numpy()


def assert_units_close(got, ref, what=""):
    """bf16 parity for every unit separately: got, ref are [units..., d] arrays;
    each unit's last-axis vector must meet max-abs and relative L2 on its own."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    g2, r2 = got.reshape(-1, got.shape[-1]), ref.reshape(-1, ref.shape[-1])
    max_abs = np.max(np.abs(g2 - r2), axis=1)
    rel = np.linalg.norm(g2 - r2, axis=1) / np.linalg.norm(r2, axis=1)
    worst = int(np.argmax(rel))
    log(f"  {what}: {g2.shape[0]} units, worst max_abs={max_abs.max():.3e} "
        f"worst rel_l2={rel.max():.3e} (unit {np.unravel_index(worst, got.shape[:-1])})")
    assert max_abs.max() <= BF16_MAX_ABS and rel.max() <= BF16_REL_L2, (what, max_abs.max(), rel.max())
