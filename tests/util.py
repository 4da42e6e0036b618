"""Small helpers shared by the tests (no method arithmetic)."""
import numpy as np
import torch


def bits(t: torch.Tensor) -> np.ndarray:
    """fp16/bf16 tensor -> uint16 bit patterns (host copy)."""
    assert t.dtype in (torch.float16, torch.bfloat16)
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)


def dname(t: torch.Tensor) -> str:
    return "fp16" if t.dtype == torch.float16 else "bf16"
