"""Helpers shared by the GPU parity tests: host copies for the oracle and the
error measures the tolerances are stated in."""
import numpy as np
import torch


def host(t: torch.Tensor) -> np.ndarray:
    """Oracle-ready host copy: float32 as float32, bf16 as raw uint16 bits."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def as_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().to(torch.float64).numpy()


def rowwise_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per output row (last axis = head_dim): max|got - ref| / max|ref|."""
    num = np.abs(got - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    return num / np.maximum(den, 1e-30)


def say(*a):
    print(*a, flush=True)
