"""Helpers shared by the GPU parity tests (seeded inputs to the device, error
metrics).  Holds no arithmetic of the method."""
import numpy as np
import torch

import ld_inputs as inp

DEV = "cuda:0"
# bf16 path against the float64 oracle: normwise max relative error per
# tensor, ||gpu - ref||_inf / ||ref||_inf <= 2e-2.
TOL_BF16 = 2e-2
# fp32 path: float32 storage and accumulation against float64.
TOL_F32 = 1e-4


def tol(dtype):
    return TOL_BF16 if dtype == "bf16" else TOL_F32


def to_dev(t):
    return t.to(DEV)


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def rel(got, want):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    den = np.max(np.abs(want))
    num = np.max(np.abs(got - want))
    if den == 0:
        return num
    return num / den


def layer_weights_dev(sh, layer, gain_jitter=False):
    w = inp.layer_weights(sh, layer, gain_jitter=gain_jitter)
    return {k: v.to(DEV) for k, v in w.items()}, {k: inp.f64(v) for k, v in w.items()}


def zero_grads(sh):
    shapes = inp.weight_shapes(sh)
    return {k: torch.zeros(s, dtype=torch.float32, device=DEV) for k, s in shapes.items()}
