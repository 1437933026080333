"""Helpers shared by the GPU tests (not a test module)."""

import numpy as np
import pytest
import torch

BF16_TOL = 1e-2   # max-abs error, bf16 inputs with float32 accumulation
F32_TOL = 1e-5    # max-abs error, float32 mode


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")


def to64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def cpu_normal(shape, seed, dtype):
    g = torch.Generator().manual_seed(int(seed))
    return torch.randn(shape, generator=g, dtype=torch.float32).to(dtype)


def say(*parts):
    print("[case]", *parts, flush=True)
