"""Small helpers shared by the tests (no method arithmetic)."""
import numpy as np
import torch


def bits(t: torch.Tensor) -> np.ndarray:
    """fp16/bf16 tensor -> uint16 bit patterns (host copy)."""
    assert t.dtype in (torch.float16, torch.bfloat16)
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)


def dname(t: torch.Tensor) -> str:
    return "fp16" if t.dtype == torch.float16 else "bf16"


def stream_classes(before, after, n, k, sink=0, recent=0):
    """Which way the streamed selection found this step's threshold, per row,
    from its caller-owned state (uint32 [B, R, 8]) before and after the call:
    None when the previous step's bound was not used (first step, reset step,
    a budget above the bound's count, fewer tokens, other pins), else the
    distance in first-digit bins (top 12 bits of the order key) from the
    bound's bin to the new threshold's: 0 to 3 lie in the window whose
    second digits the update counts, 4 and more above it (a walk of the
    update's pairs), and a negative distance means fewer than k keys reached
    the bound (S changed outside the calls: the first digit is counted again
    over the row)."""
    b = np.asarray(before, dtype=np.int64).reshape(-1, 8) & 0xFFFFFFFF
    a = np.asarray(after, dtype=np.int64).reshape(-1, 8) & 0xFFFFFFFF
    out = []
    for pb, pa in zip(b, a):
        nopins = sink == 0 and recent == 0
        used = (pb[3] == 1 and k <= pb[1] and n >= pb[2] and pb[4] == sink and pb[5] == recent
                and (n == pb[2] or nopins))
        out.append(int((pa[0] >> 20) - (pb[0] >> 20)) if used else None)
    return out
