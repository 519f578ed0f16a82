"""Helpers shared by the tests (no arithmetic of the method)."""
import numpy as np
import torch


def stored_np(t: torch.Tensor) -> np.ndarray:
    """Host numpy view of a tensor's stored elements (same bytes, same element size)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float8_e4m3fn:
        return t.view(torch.uint8).numpy()
    return t.numpy()


def np_or_none(t):
    return None if t is None else t.detach().cpu().numpy()
