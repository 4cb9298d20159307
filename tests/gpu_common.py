"""Shared helpers of the GPU parity tests: host arrays -> device tensors, and
the comparison rules (tolerances from the target: losses 1e-5 relative in
fp32 and 2e-2 relative with bf16 joiner inputs; gradients 1e-4 absolute in
fp32, 2e-2 * max|reference| with bf16 joiner inputs; dW and db, whose
magnitude grows with the number of rows, 1e-4 * max(1, max|reference|))."""
from __future__ import annotations

import sys

import numpy as np
import torch

import paper_2206_13236_amd as P

DEV = torch.device("cuda")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def dev_joiner(a, bf16: bool):
    t = dev_f32(a)
    return t.to(torch.bfloat16) if bf16 else t


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def make_dev_batch(b, blank=None) -> P.Batch:
    return P.Batch(dev_i32(b.t_len), dev_i32(b.u_len), dev_i32(b.symbols), b.T, b.U,
                   b.wl.blank if blank is None else blank)


def assert_close(name, got, ref, atol=0.0, rtol=0.0, mask=None):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} vs {ref.shape}"
    if mask is not None:
        got = np.where(mask, got, 0.0)
        ref = np.where(mask, ref, 0.0)
    both_inf = np.isinf(got) & np.isinf(ref) & (np.sign(got) == np.sign(ref))
    with np.errstate(invalid="ignore"):
        diff = np.where(both_inf, 0.0, np.abs(got - ref))
    tol = atol + rtol * np.where(np.isinf(ref), 0.0, np.abs(ref))
    bad = ~(diff <= tol)
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(bad, diff - tol, -np.inf)), got.shape)
        raise AssertionError(
            f"{name}: {int(bad.sum())}/{bad.size} elements out of tolerance (atol={atol}, rtol={rtol}); "
            f"worst at {i}: got {got[i]!r} ref {ref[i]!r}; max abs diff {np.nanmax(diff):.3e}")


def grad_atol(ref, bf16: bool, param: bool = False) -> float:
    m = float(np.max(np.abs(ref))) if np.size(ref) else 0.0
    if bf16:
        return 2e-2 * max(m, 1e-6)
    return 1e-4 * max(1.0, m) if param else 1e-4


def loss_rtol(bf16: bool) -> float:
    return 2e-2 if bf16 else 1e-5
