"""Shared helpers of the GPU tests (inputs and host copies only)."""
import numpy as np
import torch


def host_bytes(t):
    """The tensor's bytes as a host numpy uint8 array (through torch, outside
    the library)."""
    if t.numel() == 0:
        return np.zeros(0, dtype=np.uint8)
    return t.detach().contiguous().cpu().reshape(-1).view(torch.uint8).numpy().copy()


def random_byte_fragments(sizes, seed, device="cuda"):
    rng = np.random.default_rng(seed)
    host = [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]
    dev = [torch.from_numpy(h.copy()).to(device) for h in host]
    return dev, host


def garbage_fill(tensors, value=0x5A):
    for t in tensors:
        if t.numel():
            t.view(-1).view(torch.uint8).fill_(value) if t.dtype != torch.uint8 else t.fill_(value)
