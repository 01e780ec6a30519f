"""Shared helpers of the GPU parity tests: error metric, input plumbing.

The error metric (for every output tensor) is
    rel_err(x, ref) = max |x - ref| / max |ref|
taken over the whole tensor: elementwise relative error is meaningless where
outputs are near zero.  Bars: 1e-5 for float32 inputs, 2e-2 for 16-bit inputs
with float32 accumulation.
"""
import numpy as np
import torch

TOL = {"fp32": 1e-5, "bf16": 2e-2, "fp16": 2e-2}
TORCH_DT = {"fp32": torch.float32, "bf16": torch.bfloat16, "fp16": torch.float16}


def rel_err(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    denom = np.abs(ref).max()
    if denom == 0.0:
        return float(np.abs(x).max())
    return float(np.abs(x - ref).max() / denom)


def f64(t: torch.Tensor) -> np.ndarray:
    """Exact widening of a (CPU or GPU) tensor to a float64 numpy array."""
    return t.detach().to("cpu", torch.float64).numpy()


def to_gpu(inputs: dict) -> dict:
    return {k: v.to("cuda") for k, v in inputs.items()}
