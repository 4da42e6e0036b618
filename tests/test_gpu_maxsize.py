"""GPU parity at the largest context the library accepts (n_tokens =
2,097,152, include/hill.h): one sequence, GQA 2/1, bf16, a 1% budget.  Rows
this long take the separate softmax-statistics launch, 4096 selection chunks
and 8192 update workgroups, so 32-bit index arithmetic anywhere on the path
would show here.  Two steps through hill_step against the oracle (S, the
selection, the outputs), and the same steps through the streamed selection
(a reset step, then a streamed one) bit for bit against hill_step."""
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs, check_scores, check_selection, raw_abs_update
from util import bits

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
N_MAX = 1 << 21


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_18750_amd as H
    H.load_library()
    yield


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def test_step_at_the_maximum_context():
    import paper_2602_18750_amd as H
    say("max context: generating inputs on the GPU")
    x = W.make_random(1, 2, 1, 128, N_MAX, "bf16", steps=2, seed=2024, device=DEV)
    k_sel = H.budget_k(N_MAX, 0.01)
    s_a = H.new_importance(1, 1, N_MAX, DEV)
    s_b = H.new_importance(1, 1, N_MAX, DEV)
    state = H.new_stream_state(1, 1, DEV)
    qc, kc, vc = bits(x.q.cpu()), bits(x.k.cpu()), bits(x.v.cpu())
    s_ref = np.zeros((1, 1, N_MAX))
    for t in range(2):
        say("max context: step", t)
        i_a, o_a = H.hill_step(x.q[t], x.k, x.v, s_a, k_sel)
        i_b, o_b = H.hill_step(x.q[t], x.k, x.v, s_b, k_sel, stream_state=state, stream_reset=t == 0)
        torch.cuda.synchronize()
        assert torch.equal(s_a, s_b) and torch.equal(i_a, i_b) and torch.equal(o_a, o_b), "step %d" % t
        s_ref, idx_ref, out_ref = O.step(qc[t], kc, vc, s_ref, k_sel, "bf16", "attn", "token")
        idx_g = i_a.cpu().numpy()
        check_scores(s_a.cpu().numpy(), s_ref, "max step %d S" % t)
        check_selection(idx_g, s_ref, k_sel, "max step %d sel" % t)
        own = O.sparse_attn(qc[t], kc, vc, idx_g, "bf16", "token")
        check_outputs(o_a.cpu().numpy(), own, "max step %d out" % t)


@pytest.mark.parametrize("nbits", [8, 4])
def test_sketch_step_at_the_maximum_context(nbits):
    """The same length scored on the int8 / int4 sketch (GQA 8/2: the int4
    scan runs on the matrix cores): the sketch written by the library equals
    the oracle's, and S and the selection of one step match the oracle's on
    that sketch."""
    import math
    import paper_2602_18750_amd as H
    say("max context sketch", nbits)
    x = W.make_random(1, 8, 2, 128, N_MAX, "bf16", steps=1, seed=4048 + nbits, device=DEV)
    k_sel = H.budget_k(N_MAX, 0.01)
    sk = H.sketch_keys(x.k, bits=nbits)
    qc, kc, vc = bits(x.q.cpu()), bits(x.k.cpu()), bits(x.v.cpu())
    k8, ek = O.sketch(kc, "bf16", bits=nbits)
    s = H.new_importance(1, 1, N_MAX, DEV)
    idx, out = H.hill_step(x.q[0], x.k, x.v, s, k_sel, sketch=sk)
    torch.cuda.synchronize()
    assert np.array_equal(sk.exps.cpu().numpy()[:, :, :N_MAX], ek)
    q8, eq = O.sketch(qc[0], "bf16")
    s_ref = O.update(O.logits_i8(q8, eq, k8, ek), np.zeros((1, 1, N_MAX)), 2, "attn", "token", 1 / math.sqrt(128))
    check_scores(s.cpu().numpy(), s_ref, "max sketch%d S" % nbits)
    check_selection(idx.cpu().numpy(), s_ref, k_sel, "max sketch%d sel" % nbits)


@pytest.mark.parametrize("mode,gran", [("raw", "kvhead"), ("attn", "kvhead"), ("raw", "token")])
def test_long_context_modes(mode, gran):
    """A 262,144-token context in the other score modes and granularities
    (RAW sums, one row per KV head), one step against the oracle."""
    import paper_2602_18750_amd as H
    n = 1 << 18
    say("long context", mode, gran)
    x = W.make_random(1, 8, 2, 128, n, "fp16", steps=1, seed=77 + len(mode) + len(gran), device=DEV)
    k_sel = H.budget_k(n, 0.05)
    R = 1 if gran == "token" else 2
    s = H.new_importance(1, R, n, DEV)
    idx, out = H.hill_step(x.q[0], x.k, x.v, s, k_sel, mode=mode, granularity=gran)
    torch.cuda.synchronize()
    qc, kc, vc = bits(x.q.cpu()), bits(x.k.cpu()), bits(x.v.cpu())
    s_ref, _, _ = O.step(qc[0], kc, vc, np.zeros((1, R, n)), k_sel, "fp16", mode, gran)
    a_ref = raw_abs_update(np.zeros((1, R, n)), qc[0], kc, "fp16", 2, gran) if mode == "raw" else None
    check_scores(s.cpu().numpy(), s_ref, "long %s %s S" % (mode, gran), abs_sum=a_ref)
    idx_g = idx.cpu().numpy()
    check_selection(idx_g, s_ref, k_sel, "long %s %s sel" % (mode, gran))
    own = O.sparse_attn(qc[0], kc, vc, idx_g, "fp16", gran)
    check_outputs(out.cpu().numpy(), own, "long %s %s out" % (mode, gran))
