"""Shared helpers for the GPU parity tests (test code only)."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")


def device():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device (run with -m 'not gpu' on a CPU host)")
    return torch.device("cuda:0")


def say(msg: str) -> None:
    """Name the case on stdout before a GPU step, so a lost box still tells it."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dtype) -> "torch.Tensor":
    """float32 numpy -> device tensor of dtype (bf16 values must already be
    bf16-representable so the conversion is exact)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device=device(), dtype=dtype).contiguous()


def to_host64(t) -> np.ndarray:
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def normwise(y: np.ndarray, ref: np.ndarray) -> float:
    """max |y - ref| / max |ref| (the layer tolerance of the method)."""
    scale = float(np.max(np.abs(ref)))
    if scale == 0.0:
        return float(np.max(np.abs(y)))
    return float(np.max(np.abs(y - ref))) / scale


F32_LAYER_TOL = 1e-5
BF16_LAYER_TOL = 2e-2
F32_BASIS_TOL = 1e-6
PU_TOL = 1e-5
