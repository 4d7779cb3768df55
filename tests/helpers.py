"""Shared helpers of the GPU parity tests (no arithmetic of the method here)."""

import numpy as np
import torch

# Tolerances of the parity bar, as max|gpu - ref| / max|ref| per tensor:
# bf16 activations 2e-2, gradients 5e-2.
TOL_ACT = 2e-2
TOL_GRAD = 5e-2


def f64(t):
    """Tensor (any device, any float dtype) -> numpy float64."""
    return t.detach().to("cpu", torch.float64).numpy()


def max_rel(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    scale = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (scale if scale > 0 else 1.0))


def cuda(t):
    return t.to("cuda")


def announce(msg):
    """Print (and flush) what the next GPU step runs, so a failure is named."""
    print(f"[gpu-case] {msg}", flush=True)


GUARD = 4096  # elements of guard band after every output


def guarded(shape, dtype):
    """An output tensor followed by a guard band filled with a sentinel."""
    n = int(np.prod(shape))
    buf = torch.empty(n + GUARD, dtype=dtype, device="cuda")
    if dtype == torch.bfloat16:
        buf.view(torch.int16).fill_(0x7FA5)  # a NaN payload no kernel writes
    else:
        buf.view(torch.int32).fill_(0x7FC0DEAD)
    return buf[:n].view(shape), buf


def guard_intact(buf, n):
    tail = buf[n:]
    if buf.dtype == torch.bfloat16:
        return bool((tail.view(torch.int16) == 0x7FA5).all())
    return bool((tail.view(torch.int32) == 0x7FC0DEAD).all())


def exact_equal(got, want):
    g = f64(got)
    return bool(np.array_equal(g, want)), float(np.abs(g - want).max())
