"""Helpers for the GPU tests: device, tolerance metrics, case logging."""
import sys

import numpy as np
import torch

# Tolerances of the fused product (relative Frobenius error against the float64
# oracle): float32 inputs, and bfloat16 inputs with the bfloat16 distance contraction.
TOL_F32 = 1e-5
TOL_BF16 = 2e-3


def device():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU test run without a visible GPU")
    return torch.device("cuda:0")


def case(msg: str) -> None:
    """Name the case before touching the GPU (flushed, survives a crash)."""
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def to_dev(x: np.ndarray, dev) -> torch.Tensor:
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16).copy()).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def to_np(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().double().numpy()
