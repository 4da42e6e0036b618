"""GPU checks of the streamed selection (hill_step_streamed; Sec. 4.2 HIE's
running threshold): identical results to hill_step on identical inputs, step
after step, including the cases where the bound must not be used (first
step, a larger budget, a longer context with pins), heavy ties, and parity
with the oracle at full size."""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs, check_scores, check_selection
from util import bits, dname

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_18750_amd as H
    H.load_library()
    yield


def H():
    import paper_2602_18750_amd as H
    return H


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _pair_run(x, schedule, gran="token", sink=0, recent=0, resets=0, mutate=None):
    """hill_step and hill_step_streamed side by side on copies of the same S;
    schedule: list of (n_tokens, k_sel) per step, the first `resets` of them
    reset steps (HILL_STREAM_RESET); mutate: {step: f}, f(S) applied in place
    to both copies of S before that step (a change outside the calls).
    Asserts bit-identical S, indices and outputs and a valid state after
    every step, and that the indices are the oracle's top-k of the GPU's own
    S (with the pins; equal keys to the lower token index, R7).  Returns the
    streamed state."""
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    B, Hkv, ncap = k.shape[0], k.shape[1], k.shape[2]
    R = 1 if gran == "token" else Hkv
    s_a = H().new_importance(B, R, ncap, DEV)
    s_b = H().new_importance(B, R, ncap, DEV)
    state = H().new_stream_state(B, R, DEV)
    for t, (n, ks) in enumerate(schedule):
        if mutate and t in mutate:
            mutate[t](s_a)
            mutate[t](s_b)
        i_a, o_a = H().hill_step(q[t], k, v, s_a, ks, granularity=gran, n_tokens=n, n_sink=sink, n_recent=recent)
        i_b, o_b = H().hill_step(q[t], k, v, s_b, ks, granularity=gran, n_tokens=n, n_sink=sink, n_recent=recent,
                                 stream_state=state, stream_reset=t < resets)
        torch.cuda.synchronize()
        assert torch.equal(s_a, s_b), "step %d: S differs" % t
        assert torch.equal(i_a, i_b), "step %d: indices differ" % t
        assert torch.equal(o_a, o_b), "step %d: outputs differ" % t
        sv = s_b.cpu().numpy()[..., :n].astype(np.float64).reshape(-1, n)
        ref = O.topk_pinned(sv, ks, sink, recent) if (sink or recent) else O.topk(sv, ks)
        assert np.array_equal(i_b.cpu().numpy(), ref.reshape(i_b.shape)), \
            "step %d: not the top-k of the step's own S" % t
        _check_state(state, s_b, n, ks, sink, recent)
    return state


def _check_state(state, s, n, k, sink, recent):
    """The state written by the last step: valid, this n, the pins, and the
    number of tokens whose first radix digit (top 12 bits of the order key;
    pinned tokens take the largest key) reaches the threshold's: at least k."""
    st = state.cpu().numpy().view(np.uint32)
    sv = s.cpu().numpy()[..., :n]
    key = sv.view(np.uint32) | np.uint32(0x80000000)   # S >= 0: order key of a non-negative float
    j = np.arange(n)
    key[..., (j < sink) | (j >= n - recent)] = 0xFFFFFFFF
    digit = (key >> 20).astype(np.int64)
    thr = (st[..., 0] >> 20).astype(np.int64)
    count = (digit >= thr[..., None]).sum(-1)
    assert (st[..., 3] == 1).all() and (st[..., 2] == n).all()
    assert (st[..., 4] == sink).all() and (st[..., 5] == recent).all()
    assert (st[..., 1] == count).all() and (count >= k).all()


STREAM_CASES = [
    # B, Hq, Hkv, n, dtype, gran, steps, k, sink, recent
    (1, 32, 8, 8192 + 77, "bf16", "token", 6, 819, 0, 0),
    (2, 8, 2, 3000, "fp16", "kvhead", 5, 300, 0, 0),
    (1, 32, 32, 4096, "fp16", "token", 4, 819, 0, 0),
    (2, 16, 4, 5000, "bf16", "token", 5, 500, 4, 64),
    (1, 4, 4, 129, "bf16", "token", 4, 13, 0, 0),
]


@pytest.mark.parametrize("B,Hq,Hkv,n,dt,gran,steps,k,sink,recent", STREAM_CASES)
def test_streamed_equals_plain_step(B, Hq, Hkv, n, dt, gran, steps, k, sink, recent):
    say("streamed vs plain", B, Hq, Hkv, n, dt, gran, steps, k, sink, recent)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=steps, seed=n + Hq + k)
    _pair_run(x, [(n, k)] * steps, gran, sink, recent)


def test_streamed_bound_changes():
    """Budget up (bound dropped), budget down (bound kept), context growth
    without pins (bound kept) and with pins (bound dropped)."""
    x = W.make_random(1, 16, 4, 128, 6000, "bf16", steps=8, seed=99)
    say("streamed bound changes, no pins")
    _pair_run(x, [(5000, 500), (5000, 700), (5000, 400), (5200, 400), (5600, 420), (6000, 400), (6000, 400),
                  (6000, 600)])
    say("streamed bound changes, pins")
    _pair_run(x, [(5000, 500), (5100, 500), (5100, 500), (5300, 520), (5300, 300), (6000, 300), (6000, 300),
                  (6000, 300)], sink=3, recent=40)


@pytest.mark.parametrize("factor", [0.25, 4.0, 0.0])
def test_streamed_after_outside_change_of_s(factor):
    """S scaled (or cleared) between streamed calls without a reset: scaled
    down or cleared, fewer than k keys reach the bound's first digit and the
    selection counts that digit again over the whole row; scaled up, the k-th
    key stays in the counted bins.  Either way the results equal hill_step's,
    and the bound written afterwards is valid again."""
    x = W.make_random(1, 16, 4, 128, 5000, "bf16", steps=6, seed=61)
    say("streamed after S *= %g outside the calls" % factor)
    _pair_run(x, [(5000, 500)] * 6, resets=1, mutate={3: lambda s: s.mul_(factor)})


def test_streamed_heavy_ties():
    """Keys drawn from 40 distinct rows: equal S values across thousands of
    tokens, so the threshold needs all three digits and the tie ranks."""
    x = W.make_random(1, 8, 2, 128, 4096, "bf16", steps=4, seed=5)
    g = torch.Generator().manual_seed(3)
    pick = torch.randint(0, 40, (4096,), generator=g)
    x.k[:, :, :, :] = x.k[:, :, pick, :].clone()
    say("streamed heavy ties")
    _pair_run(x, [(4096, 1000), (4096, 1000), (4096, 2047), (4096, 2047)])


def test_heavy_ties_over_more_than_256_chunks():
    """The same over 140,000 tokens (274 selection chunks, so the walks over
    the chunks' candidate lists take two groups of 256) with the threshold
    inside a tie group spread over all chunks: both paths' indices equal the
    oracle's top-k of the step's own S, lower index first among equal keys."""
    n = 140000
    x = W.make_random(1, 8, 2, 128, n, "bf16", steps=3, seed=17)
    g = torch.Generator().manual_seed(4)
    pick = torch.randint(0, 60, (n,), generator=g)
    x.k[:, :, :, :] = x.k[:, :, pick, :].clone()
    say("heavy ties, 140000 tokens")
    _pair_run(x, [(n, 40000), (n, 40000), (n, 70001)])


def test_streamed_workload3_full_size_matches_oracle():
    w = W.WORKLOADS[3].replace(steps=3)
    say("streamed workload 3 layer 0, 3 steps")
    x = W.make_layer(w, 0)
    dt = dname(x.k)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    s = H().new_importance(1, 1, w.n_tokens, DEV)
    state = H().new_stream_state(1, 1, DEV)
    s_ref = np.zeros((1, 1, w.n_tokens))
    for t in range(w.steps):
        idx, out = H().hill_step(q[t], k, v, s, w.k_sel, stream_state=state)
        s_ref = O.update(O.logits(bits(x.q[t]), bits(x.k), dt), s_ref, w.n_kv_heads, "attn", "token",
                         1 / math.sqrt(128))
        torch.cuda.synchronize()
        idx_g = idx.cpu().numpy()
        check_scores(s.cpu().numpy(), s_ref, "stream step %d S" % t)
        check_selection(idx_g, s_ref, w.k_sel, "stream step %d sel" % t)
        out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, "token")
        check_outputs(out.cpu().numpy(), out_own, "stream step %d out" % t)


@pytest.mark.parametrize("nbits", [8, 4])
def test_streamed_sketch_equals_plain_sketch_step(nbits):
    """Scoring on the int8 / int4 sketch with the streamed selection gives the
    same S, indices and outputs as with the refine-based one."""
    x = W.make_random(1, 32, 8, 128, 6000, "bf16", steps=5, seed=31 + nbits)
    say("streamed sketch", nbits)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    sk = H().sketch_keys(k, bits=nbits)
    s_a = H().new_importance(1, 1, 6000, DEV)
    s_b = H().new_importance(1, 1, 6000, DEV)
    state = H().new_stream_state(1, 1, DEV)
    for t in range(5):
        i_a, o_a = H().hill_step(q[t], k, v, s_a, 600, sketch=sk)
        i_b, o_b = H().hill_step(q[t], k, v, s_b, 600, sketch=sk, stream_state=state)
        torch.cuda.synchronize()
        assert torch.equal(s_a, s_b) and torch.equal(i_a, i_b) and torch.equal(o_a, o_b), "step %d" % t


def test_stepcall_rejects_a_host_or_strided_state():
    """Device inputs with a stream state on the host, or one that is not
    contiguous: ValueError from StepCall's constructor, before any launch."""
    x = W.make_random(1, 8, 2, 128, 1000, "bf16", steps=1, seed=3)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    s = H().new_importance(1, 1, 1000, DEV)
    with pytest.raises(ValueError, match="GPU tensors only"):
        H().StepCall(q[0], k, v, s, 100, stream_state=H().new_stream_state(1, 1, DEV).cpu())
    strided = torch.zeros((1, 1, 16), dtype=torch.int32, device=DEV)[:, :, ::2]
    with pytest.raises(ValueError, match="contiguous"):
        H().StepCall(q[0], k, v, s, 100, stream_state=strided)
    torch.cuda.synchronize()
    assert not s.any(), "a rejected StepCall must not have launched anything"


def test_streamed_growing_context_keeps_the_bound():
    """n grows by one token per step and k = floor(0.1 n) grows with it (the
    decode loop's case): results equal hill_step's, and after the first steps
    the state keeps a valid bound (its count covers the next k)."""
    x = W.make_random(1, 16, 4, 128, 4200, "bf16", steps=40, seed=8)
    sched = [(4000 + 5 * t, O.budget_k(4000 + 5 * t, 0.1)) for t in range(40)]
    say("streamed growing context")
    _pair_run(x, sched)


@pytest.mark.parametrize("sink,recent", [(0, 0), (4, 64)])
def test_streamed_reset_steps(sink, recent):
    """HILL_STREAM_RESET steps select through the refine pass and write a
    fresh bound (the same state a streamed step writes); the streamed steps
    after them use it.  Identical results to hill_step throughout, also when
    a reset follows streamed steps."""
    x = W.make_random(2, 16, 4, 128, 5000, "bf16", steps=7, seed=123 + sink)
    say("streamed reset steps", sink, recent)
    sched = [(4800, 480), (4800, 480), (4900, 490), (4900, 490), (5000, 500), (5000, 500), (5000, 520)]
    _pair_run(x, sched, sink=sink, recent=recent, resets=2)
    # a later reset (k grew past the bound's count, or the caller changed S): a fresh start from any state
    x2 = W.make_random(2, 16, 4, 128, 5000, "bf16", steps=3, seed=321 + sink)
    _pair_run(x2, [(5000, 500), (5000, 2000), (5000, 500)], sink=sink, recent=recent, resets=1)


def test_streamed_several_kv_heads_per_workgroup():
    """Workload 4's shape (B 4, n 131072, GQA 32/8): the select+attend kernel
    takes four KV heads per workgroup there; the streamed steps (a reset step,
    then streamed ones, including a growing budget) equal hill_step's."""
    n = 131072
    x = W.make_random(4, 32, 8, 128, n, "bf16", steps=4, seed=404, device=DEV)
    say("streamed, several KV heads per workgroup")
    _pair_run(x, [(n, 6553), (n, 6553), (n, 6600), (n, 6553)], resets=1)


def test_stage_events_stamp_the_stages_that_run():
    """hill_step_events (include/hill.h): a streamed step stamps the scan,
    update, select and merge stages (each interval non-negative, in launch
    order) and leaves the refine stage's events as they were; a reset step
    stamps refine too.  The events are torch's, created by a first record."""
    stages = H().hill.STAGES
    x = W.make_random(1, 32, 8, 128, 5000, "bf16", steps=2, seed=17)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    s = H().new_importance(1, 1, 5000, DEV)
    state = H().new_stream_state(1, 1, DEV)
    stream = torch.cuda.current_stream()
    for t, reset in ((0, True), (1, False)):
        start = [torch.cuda.Event(enable_timing=True) for _ in stages]
        stop = [torch.cuda.Event(enable_timing=True) for _ in stages]
        for a, b in zip(start, stop):
            a.record(stream)
            b.record(stream)
        torch.cuda.synchronize()
        before = [a.elapsed_time(b) for a, b in zip(start, stop)]
        ev = H().HillStepEvents.of([e.cuda_event for e in start], [e.cuda_event for e in stop])
        H().hill_step(q[t], k, v, s, 500, stream_state=state, stream_reset=reset, events=ev)
        torch.cuda.synchronize()
        ran = ["scan", "update"] + (["refine"] if reset else []) + ["select", "merge"]
        prev_stop = None
        for i, name in enumerate(stages):
            dur = start[i].elapsed_time(stop[i])
            if name in ran:
                assert dur >= 0.0, (name, dur)
                if prev_stop is not None:
                    assert prev_stop.elapsed_time(start[i]) >= 0.0, name
                prev_stop = stop[i]
            else:
                assert dur == before[i], "stage %s did not run but its events moved" % name
