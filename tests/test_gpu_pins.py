"""GPU parity of selection with pinned tokens (attention sinks at the start
of the context, the recent window at its end; hill_desc n_sink / n_recent)
against the oracle's topk_pinned: bit-exact on identical input, and through
whole decode steps with the usual score / selection / output criteria."""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs, check_scores, check_selection, raw_abs_update
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


def _rows(kind, rows, n, seed):
    g = np.random.default_rng(seed)
    if kind == "grid":
        return (g.integers(-6, 7, (rows, n)) / 4.0).astype(np.float32)
    if kind == "equal":
        return np.full((rows, n), 0.125, dtype=np.float32)
    if kind == "lognormal":
        return np.exp(g.standard_normal((rows, n)) - 8).astype(np.float32)
    if kind == "nan":
        a = g.standard_normal((rows, n)).astype(np.float32)
        a[:, ::7] = np.nan
        a[:, 5::13] = np.inf
        return a
    raise ValueError(kind)


PIN_TOPK_CASES = [
    # kind, rows, n, k, n_sink, n_recent
    ("lognormal", 1, 32768, 3276, 4, 64),
    ("grid", 2, 4097, 819, 16, 400),
    ("equal", 2, 5000, 100, 10, 90),          # k equals the pinned count
    ("grid", 1, 1000, 1000, 600, 600),        # overlapping windows: everything pinned
    ("nan", 2, 2000, 300, 7, 0),              # NaN / +inf around the pins
    ("lognormal", 3, 777, 50, 0, 49),
    ("lognormal", 4, 131072, 6553, 4, 1024),
]


@pytest.mark.parametrize("kind,rows,n,k,sink,recent", PIN_TOPK_CASES)
def test_pinned_topk_is_exact(kind, rows, n, k, sink, recent):
    say("pinned topk", kind, rows, n, k, sink, recent)
    a = _rows(kind, rows, n, seed=n + sink)
    s = H().new_importance(rows, 1, n, DEV)
    s[:, 0, :] = torch.from_numpy(a).to(DEV)
    idx, val = H().hill_topk(s, k, with_values=True, n_sink=sink, n_recent=recent)
    torch.cuda.synchronize()
    ref = O.topk_pinned(a.astype(np.float64), k, sink, recent)
    assert np.array_equal(idx.cpu().numpy()[:, 0, :], ref)
    want = np.take_along_axis(a, ref, axis=1)
    assert np.array_equal(val.cpu().numpy()[:, 0, :].view(np.uint32), want.view(np.uint32))


def test_pinned_topk_kvhead_rows():
    B, Hkv, n, k = 2, 4, 1500, 200
    a = _rows("grid", B * Hkv, n, seed=9).reshape(B, Hkv, n)
    s = H().new_importance(B, Hkv, n, DEV)
    s.copy_(torch.from_numpy(a))
    idx = H().hill_topk(s, k, granularity="kvhead", n_sink=3, n_recent=30)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), O.topk_pinned(a.astype(np.float64), k, 3, 30))


def _check_pinned_selection(idx_g, s_ref, k, sink, recent, where):
    n = s_ref.shape[-1]
    lo = min(sink, n)
    hi = max(lo, n - min(recent, n))
    pinned = np.r_[np.arange(lo), np.arange(hi, n)]
    rows = idx_g.reshape(-1, k)
    mid = []
    for r in rows:
        assert np.all(np.diff(r) > 0), where
        assert np.isin(pinned, r).all(), where + ": a pinned token is missing"
        mid.append(r[(r >= lo) & (r < hi)] - lo)
    mid = np.stack(mid).reshape(idx_g.shape[:-1] + (k - len(pinned),))
    if k > len(pinned):
        check_selection(mid, s_ref[..., lo:hi], k - len(pinned), where)


@pytest.mark.parametrize("mode,gran,sketch", [("attn", "token", False), ("raw", "token", False),
                                              ("attn", "kvhead", False), ("attn", "token", True)])
def test_step_with_pins_matches_oracle(mode, gran, sketch):
    w = W.WORKLOADS[3].replace(n_tokens=8192 + 77, steps=3, layers=1)
    say("pinned step", mode, gran, sketch, w.n_tokens)
    x = W.make_layer(w, 0)
    dt = dname(x.k)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    k_sel = O.budget_k(w.n_tokens, w.budget)
    sink, recent = 4, 256
    R = 1 if gran == "token" else w.n_kv_heads
    s = H().new_importance(w.batch, R, w.n_tokens, DEV)
    s_ref = np.zeros((w.batch, R, w.n_tokens))
    a_ref = np.zeros((w.batch, R, w.n_tokens)) if mode == "raw" else None
    sk = H().sketch_keys(k) if sketch else None
    k8, ek = O.sketch(bits(x.k), dt) if sketch else (None, None)
    for t in range(w.steps):
        idx, out = H().hill_step(q[t], k, v, s, k_sel, mode=mode, granularity=gran, n_sink=sink,
                                 n_recent=recent, sketch=sk)
        if sketch:
            q8, eq = O.sketch(bits(x.q[t]), dt)
            l = O.logits_i8(q8, eq, k8, ek)
        else:
            l = O.logits(bits(x.q[t]), bits(x.k), dt)
        s_ref = O.update(l, s_ref, w.n_kv_heads, mode, gran, 1 / math.sqrt(128))
        if a_ref is not None:
            a_ref = raw_abs_update(a_ref, bits(x.q[t]), bits(x.k), dt, w.n_kv_heads, gran)
        torch.cuda.synchronize()
        idx_g = idx.cpu().numpy()
        check_scores(s.cpu().numpy(), s_ref, "step %d S" % t, abs_sum=a_ref)
        _check_pinned_selection(idx_g, s_ref, k_sel, sink, recent, "step %d sel" % t)
        out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, gran)
        check_outputs(out.cpu().numpy(), out_own, "step %d out" % t)
