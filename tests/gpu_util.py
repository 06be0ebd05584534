"""Helpers for the GPU parity tests: move seeded bit patterns to the device and compare the HIP
path's fp32 results with the oracle's fp64 ones."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synthetic as syn

REL_TOL = 4e-3     # |y - y_ref| <= REL_TOL * sum_k |x_k W_kn| + ABS_TOL (the stated acceptance)
ABS_TOL = 1e-6


def dev16(bits: np.ndarray, dt: int) -> torch.Tensor:
    """uint16 bit patterns -> a bf16/fp16 device tensor holding exactly those bits."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()
    return t.view(torch.bfloat16 if dt == syn.BF16 else torch.float16)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def assert_parity(y_gpu, y_ref: np.ndarray, abs_ref: np.ndarray, integer: bool = False, what: str = ""):
    y = (y_gpu.detach().cpu().numpy() if isinstance(y_gpu, torch.Tensor) else np.asarray(y_gpu))
    y = y.astype(np.float64)
    assert y.shape == y_ref.shape, (y.shape, y_ref.shape)
    if integer:
        bad = np.argwhere(y != y_ref)
        assert bad.size == 0, f"{what}: {len(bad)} integer results differ, first at {bad[0]}: " \
                              f"{y[tuple(bad[0])]} vs {y_ref[tuple(bad[0])]}"
        return
    err = np.abs(y - y_ref)
    bound = REL_TOL * abs_ref + ABS_TOL
    ok = err <= bound
    if not ok.all():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{what}: {np.count_nonzero(~ok)} of {ok.size} outside tolerance; "
                             f"worst at {i}: gpu {y[i]!r} ref {y_ref[i]!r} bound {bound[i]!r}")
    return float(np.max(err / bound))
