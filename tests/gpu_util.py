"""Helpers shared by the GPU parity tests: move generator bits to the device
and back as raw bit patterns (no arithmetic on either side)."""

import sys

import numpy as np


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(x, dtype):
    """Raw generator array -> CUDA tensor of the same bits."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.cuda()


def bits(t):
    """CUDA tensor -> numpy array of its raw bits."""
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy().view(np.uint32)
    return t.numpy()


def raw_bits(x, dtype):
    x = np.ascontiguousarray(x)
    return x.view(np.uint16) if dtype == "bf16" else x.astype(np.float32).view(np.uint32)


def score_tol(dtype):
    return 2e-3 if dtype == "bf16" else 1e-5
