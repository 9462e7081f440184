"""Test-side plumbing: storage tensors as numpy arrays the oracle accepts."""
import numpy as np
import torch


def storage_np(t: torch.Tensor) -> np.ndarray:
    """bf16 tensors as uint16 bit arrays, float32 tensors as float32 arrays (CPU copies)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dtype_name(t: torch.Tensor) -> str:
    return "bf16" if t.dtype == torch.bfloat16 else "f32"
