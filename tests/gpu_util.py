"""Helpers shared by the GPU tests: device buffers through torch (plumbing only)
and tolerance rules derived from the arithmetic of each kernel."""

import numpy as np

F16_REL = 2.0 ** -11      # f16 keeps 11 significant bits: rounding error <= 2^-11 relative


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


def stream():
    torch = torch_cuda()
    return torch.cuda.current_stream().cuda_stream


def report(title, **kv):
    print(title, " ".join(f"{k}={v}" for k, v in kv.items()), flush=True)
