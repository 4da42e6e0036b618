"""GPU parity over seeded random configurations: batch, head layout (MHA to
G = 8 GQA), ragged context lengths, budgets from one token to the whole row,
fp16 / bf16, ATTN / RAW scores and token / KV-head rows, a few carried steps
each.  Every step of hill_step is checked against the oracle (S, the
selection band, the attention over the GPU's own index set) and its indices
against the oracle's top-k of the GPU's own S (equal keys to the lower token
index); ATTN cases also run the streamed step on a copy of S, which must give
the same S, indices and outputs bit for bit.  A second set draws scoring on
the int8 / int4 key sketches and pinned sink / recent tokens, a third group
sizes of 3 to 16 query heads per KV head (uneven passes of the matrix-core
scans) on the 16-bit keys or the int8 sketch."""
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs, check_scores, check_selection, raw_abs_update, raw_abs_update_logits
from util import bits

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
N_CASES = 120


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


def _case(i):
    """Configuration i, drawn from its own seeded generator (the same on every run)."""
    g = np.random.default_rng(7919 * (i + 1))
    B = int(g.integers(1, 4))
    Hkv = int(g.choice([1, 2, 4, 8]))
    G = int(g.choice([1, 2, 4, 8]))
    if Hkv * G > 64:
        G = 64 // Hkv
    n = int(g.choice([int(g.integers(1, 64)), int(g.integers(64, 4096)), int(g.integers(4096, 20000))]))
    k = int(np.clip(int(g.choice([1, max(1, n // 20), max(1, n // 10), max(1, n // 3), n])), 1, n))
    dt = str(g.choice(["fp16", "bf16"]))
    mode = str(g.choice(["attn", "attn", "raw"]))
    gran = str(g.choice(["token", "kvhead"]))
    steps = int(g.integers(2, 4))
    return B, Hkv * G, Hkv, n, k, dt, mode, gran, steps


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_configuration_matches_oracle(i):
    B, Hq, Hkv, n, k, dt, mode, gran, steps = _case(i)
    where = "case %d (B %d, Hq %d, Hkv %d, n %d, k %d, %s, %s, %s)" % (i, B, Hq, Hkv, n, k, dt, mode, gran)
    say(where)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=steps, seed=1000 + i)
    q, kk, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    R = 1 if gran == "token" else Hkv
    streamed = mode == "attn"
    s = H().new_importance(B, R, n, DEV)
    s2 = H().new_importance(B, R, n, DEV) if streamed else None
    state = H().new_stream_state(B, R, DEV) if streamed else None
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    for t in range(steps):
        idx, out = H().hill_step(q[t], kk, v, s, k, mode=mode, granularity=gran)
        if streamed:
            idx2, out2 = H().hill_step(q[t], kk, v, s2, k, mode=mode, granularity=gran, stream_state=state,
                                       stream_reset=t == 0)
        s_ref, idx_ref, out_ref = O.step(bits(x.q[t]), bits(x.k), bits(x.v), s_ref, k, dt, mode, gran)
        if a_ref is not None:
            a_ref = raw_abs_update(a_ref, bits(x.q[t]), bits(x.k), dt, Hkv, gran)
        torch.cuda.synchronize()
        sv = s.cpu().numpy()
        idx_g = idx.cpu().numpy()
        check_scores(sv, s_ref, "%s step %d S" % (where, t), abs_sum=a_ref)
        check_selection(idx_g, s_ref, k, "%s step %d sel" % (where, t))
        own = O.topk(sv.astype(np.float64).reshape(-1, n), k).reshape(idx_g.shape)
        assert np.array_equal(idx_g, own), "%s step %d: not the top-k of the step's own S" % (where, t)
        out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, gran)
        check_outputs(out.cpu().numpy(), out_own, "%s step %d out" % (where, t))
        if streamed:
            assert torch.equal(s, s2), "%s step %d: streamed S differs" % (where, t)
            assert torch.equal(idx, idx2), "%s step %d: streamed indices differ" % (where, t)
            assert torch.equal(out, out2), "%s step %d: streamed outputs differ" % (where, t)


N_CASES_SKETCH_PINS = 60


def _case_sketch_pins(i):
    """Configuration i of the second set: scoring on the 16-bit keys or on an
    int8 / int4 sketch, with or without pinned sink and recent tokens (the
    budget raised to hold them)."""
    g = np.random.default_rng(104729 * (i + 1))
    B = int(g.integers(1, 3))
    Hkv = int(g.choice([1, 2, 4, 8]))
    G = int(g.choice([1, 2, 4, 8]))
    if Hkv * G > 64:
        G = 64 // Hkv
    n = int(g.integers(2, 12000))
    k = int(np.clip(int(g.choice([1, max(1, n // 20), max(1, n // 10), max(1, n // 3)])), 1, n))
    dt = str(g.choice(["fp16", "bf16"]))
    nbits = int(g.choice([0, 8, 4]))
    mode = str(g.choice(["attn", "attn", "raw"]))
    gran = str(g.choice(["token", "kvhead"]))
    sink = int(g.choice([0, 0, 4, 64]))
    recent = int(g.choice([0, 0, 32, 256]))
    lo = min(sink, n)
    hi = max(lo, n - min(recent, n))
    k = max(k, lo + n - hi)
    steps = int(g.integers(2, 4))
    return B, Hkv * G, Hkv, n, k, dt, nbits, mode, gran, sink, recent, steps


@pytest.mark.parametrize("i", range(N_CASES_SKETCH_PINS))
def test_random_sketch_and_pins_match_oracle(i):
    B, Hq, Hkv, n, k, dt, nbits, mode, gran, sink, recent, steps = _case_sketch_pins(i)
    where = "sketch/pins case %d (B %d, Hq %d, Hkv %d, n %d, k %d, %s, keys %s, %s, %s, pins %d/%d)" % (
        i, B, Hq, Hkv, n, k, dt, nbits or 16, mode, gran, sink, recent)
    say(where)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=steps, seed=5000 + i)
    q, kk, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    sk = H().sketch_keys(kk, bits=nbits) if nbits else None
    k8, ek = O.sketch(bits(x.k), dt, bits=nbits) if nbits else (None, None)
    R = 1 if gran == "token" else Hkv
    streamed = mode == "attn"
    s = H().new_importance(B, R, n, DEV)
    s2 = H().new_importance(B, R, n, DEV) if streamed else None
    state = H().new_stream_state(B, R, DEV) if streamed else None
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    scale = 1.0 / np.sqrt(128.0)
    for t in range(steps):
        idx, out = H().hill_step(q[t], kk, v, s, k, mode=mode, granularity=gran, sketch=sk, n_sink=sink,
                                 n_recent=recent)
        if streamed:
            idx2, out2 = H().hill_step(q[t], kk, v, s2, k, mode=mode, granularity=gran, sketch=sk, n_sink=sink,
                                       n_recent=recent, stream_state=state, stream_reset=t == 0)
        if nbits:
            q8, eq = O.sketch(bits(x.q[t]), dt)
            lg = O.logits_i8(q8, eq, k8, ek)
            if a_ref is not None:
                a_ref = raw_abs_update_logits(a_ref, lg, Hkv, gran)
        else:
            lg = O.logits(bits(x.q[t]), bits(x.k), dt)
            if a_ref is not None:
                a_ref = raw_abs_update(a_ref, bits(x.q[t]), bits(x.k), dt, Hkv, gran)
        s_ref = O.update(lg, s_ref, Hkv, mode, gran, scale)
        torch.cuda.synchronize()
        sv = s.cpu().numpy()
        idx_g = idx.cpu().numpy()
        check_scores(sv, s_ref, "%s step %d S" % (where, t), abs_sum=a_ref)
        flat = sv.astype(np.float64).reshape(-1, n)
        own = O.topk_pinned(flat, k, sink, recent) if (sink or recent) else O.topk(flat, k)
        assert np.array_equal(idx_g, own.reshape(idx_g.shape)), "%s step %d: not the top-k of the step's own S" % (
            where, t)
        out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, gran)
        check_outputs(out.cpu().numpy(), out_own, "%s step %d out" % (where, t))
        if streamed:
            assert torch.equal(s, s2), "%s step %d: streamed S differs" % (where, t)
            assert torch.equal(idx, idx2), "%s step %d: streamed indices differ" % (where, t)
            assert torch.equal(out, out2), "%s step %d: streamed outputs differ" % (where, t)


N_CASES_GROUPS = 40


def _case_groups(i):
    """Configuration i of the third set: group sizes that are not powers of two
    or exceed one pass of the matrix-core scan (3 to 16 query heads per KV
    head), scored on the 16-bit keys or the int8 sketch."""
    g = np.random.default_rng(15485863 * (i + 1))
    B = int(g.integers(1, 3))
    Hkv = int(g.choice([1, 2, 3]))
    G = int(g.choice([3, 4, 5, 6, 7, 12, 16]))
    n = int(g.integers(1, 9000))
    k = int(np.clip(int(g.choice([1, max(1, n // 20), max(1, n // 10), max(1, n // 3), n])), 1, n))
    dt = str(g.choice(["fp16", "bf16"]))
    nbits = int(g.choice([0, 0, 8]))
    mode = str(g.choice(["attn", "attn", "raw"]))
    gran = str(g.choice(["token", "kvhead"]))
    steps = int(g.integers(2, 4))
    return B, Hkv * G, Hkv, n, k, dt, nbits, mode, gran, steps


@pytest.mark.parametrize("i", range(N_CASES_GROUPS))
def test_random_group_sizes_match_oracle(i):
    B, Hq, Hkv, n, k, dt, nbits, mode, gran, steps = _case_groups(i)
    where = "group case %d (B %d, Hq %d, Hkv %d, n %d, k %d, %s, keys %s, %s, %s)" % (
        i, B, Hq, Hkv, n, k, dt, nbits or 16, mode, gran)
    say(where)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=steps, seed=9000 + i)
    q, kk, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    sk = H().sketch_keys(kk, bits=nbits) if nbits else None
    k8, ek = O.sketch(bits(x.k), dt, bits=nbits) if nbits else (None, None)
    R = 1 if gran == "token" else Hkv
    streamed = mode == "attn"
    s = H().new_importance(B, R, n, DEV)
    s2 = H().new_importance(B, R, n, DEV) if streamed else None
    state = H().new_stream_state(B, R, DEV) if streamed else None
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    scale = 1.0 / np.sqrt(128.0)
    for t in range(steps):
        idx, out = H().hill_step(q[t], kk, v, s, k, mode=mode, granularity=gran, sketch=sk)
        if streamed:
            idx2, out2 = H().hill_step(q[t], kk, v, s2, k, mode=mode, granularity=gran, sketch=sk, stream_state=state,
                                       stream_reset=t == 0)
        if nbits:
            q8, eq = O.sketch(bits(x.q[t]), dt)
            lg = O.logits_i8(q8, eq, k8, ek)
            if a_ref is not None:
                a_ref = raw_abs_update_logits(a_ref, lg, Hkv, gran)
        else:
            lg = O.logits(bits(x.q[t]), bits(x.k), dt)
            if a_ref is not None:
                a_ref = raw_abs_update(a_ref, bits(x.q[t]), bits(x.k), dt, Hkv, gran)
        s_ref = O.update(lg, s_ref, Hkv, mode, gran, scale)
        torch.cuda.synchronize()
        sv = s.cpu().numpy()
        idx_g = idx.cpu().numpy()
        check_scores(sv, s_ref, "%s step %d S" % (where, t), abs_sum=a_ref)
        check_selection(idx_g, s_ref, k, "%s step %d sel" % (where, t))
        own = O.topk(sv.astype(np.float64).reshape(-1, n), k).reshape(idx_g.shape)
        assert np.array_equal(idx_g, own), "%s step %d: not the top-k of the step's own S" % (where, t)
        out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, gran)
        check_outputs(out.cpu().numpy(), out_own, "%s step %d out" % (where, t))
        if streamed:
            assert torch.equal(s, s2), "%s step %d: streamed S differs" % (where, t)
            assert torch.equal(idx, idx2), "%s step %d: streamed indices differ" % (where, t)
            assert torch.equal(out, out2), "%s step %d: streamed outputs differ" % (where, t)
