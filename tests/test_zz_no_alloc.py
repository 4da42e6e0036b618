"""hill_step_noalloc (include/hill.h): the decode step with the library's
fixed device scratch instead of a caller's workspace, for callers that cannot
allocate.  Its results equal hill_step's bit for bit (the same kernels over
the same arithmetic; only the scratch address differs), call after call on
the shared buffer -- here a 32K-token step and then a smaller one, so the
second call runs over what the first left in the buffer.  A step larger than
the buffer is refused before anything is enqueued."""
import ctypes
import sys

import numpy as np
import pytest
import torch

from paper_2602_18750_amd import workloads as W


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def H():
    import paper_2602_18750_amd as H
    return H


def test_noalloc_rejects_steps_beyond_the_buffer():
    """Host-side checks, before any device call: a 131K-token batch-4 step
    needs more than the fixed buffer; a bad budget is an argument error."""
    lib = H().load_library()
    s_shape = torch.empty((4, 1, 131072), dtype=torch.float32)    # shapes and strides only
    d = H().make_desc(None, None, None, s_shape, shape=(4, 32, 8, 128), dtype=torch.bfloat16)
    need = H().workspace_bytes(d, 6553)
    assert need > H().hill.NOALLOC_SCRATCH_BYTES
    FAKE = 0x10000
    rc = lib.hill_step_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 6553, FAKE, FAKE, None)
    assert rc == 3 and b"fixed device buffer" in lib.hill_last_error()     # HILL_ERR_WORKSPACE
    rc = lib.hill_step_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 0, FAKE, FAKE, None)
    assert rc == 1                                                           # HILL_ERR_INVALID_ARG (k_sel)


@pytest.mark.gpu
def test_noalloc_step_equals_hill_step_on_consecutive_calls():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = "cuda:0"
    cases = [  # B, Hq, Hkv, n, k, steps: the second call is smaller than the first
        (1, 32, 8, 32768, 3276, 2),
        (2, 16, 4, 3000, 300, 1),
    ]
    for B, Hq, Hkv, n, k, steps in cases:
        say("noalloc step", B, Hq, Hkv, n, k)
        x = W.make_random(B, Hq, Hkv, 128, n, "bf16", steps=steps, seed=n + k)
        q, kk, v = x.q.to(dev), x.k.to(dev), x.v.to(dev)
        s_a = H().new_importance(B, 1, n, dev)
        s_b = H().new_importance(B, 1, n, dev)
        for t in range(steps):
            i_a, o_a = H().hill_step(q[t], kk, v, s_a, k)
            i_b, o_b = H().hill_step_noalloc(q[t], kk, v, s_b, k)
            torch.cuda.synchronize()
            assert torch.equal(s_a, s_b), "S differs (n %d, step %d)" % (n, t)
            assert torch.equal(i_a, i_b), "indices differ (n %d, step %d)" % (n, t)
            assert torch.equal(o_a, o_b), "outputs differ (n %d, step %d)" % (n, t)
            idx = i_b.cpu().numpy()
            assert np.all(np.diff(idx, axis=-1) > 0) and idx.min() >= 0 and idx.max() < n
