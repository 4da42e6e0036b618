"""GPU parity of the regimes the benchmark times, against the oracle.

* The 32K-context Llama-3-8B-shaped decode exactly as bench.py drives it:
  StepCall over a shared workspace on the current stream, three reset steps
  (HILL_STREAM_RESET), then streamed steps, S carried over all 64 decode
  steps, on layers 0 and 31.  S, the selection and the outputs are compared
  with the oracle after every step, and the way each streamed step found its
  threshold (same first-digit bin as the bound, a window bin above it, or
  above the window) is read from the state.
* The 131K-context AR(1) workload: 16 decode steps through StepCall
  (streamed) and hill_step side by side, both against the oracle, with the
  per-step overlap of consecutive selections, |I_t & I_(t-1)| / k.
* Every cell of the 27-cell sweep, one decode step, rows 0 and B-1 against
  the oracle (batch rows are independent).

Importance carried over decode steps and eviction at every step follow
Sec. 4.1 and Sec. 3.1; parity criteria are those of tests/parity.py."""
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs, check_scores, check_selection
from util import bits, dname, stream_classes

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


def _check_step(x, t, s, idx, out, s_ref, idx_ref, out_ref, k_sel, where):
    dt = dname(x.k)
    idx_g = idx.cpu().numpy()
    check_scores(s.cpu().numpy(), s_ref, "%s S" % where)
    check_selection(idx_g, s_ref, k_sel, "%s sel" % where)
    own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, "token")
    check_outputs(out.cpu().numpy(), own, "%s out" % where)
    if np.array_equal(idx_g, idx_ref):
        check_outputs(out.cpu().numpy(), out_ref, "%s out(direct)" % where)
    return idx_g


def _stepcall_run(x, k_sched, where, resets=3):
    """StepCall as bench.py builds it, over len(k_sched) steps (k_sched: the
    budget per step; a change rebuilds the call with the same state, as a
    caller would), against the oracle.  Returns the per-step classes of the
    streamed threshold search (tests/util.py stream_classes)."""
    B, n = x.k.shape[0], x.k.shape[2]
    dt = dname(x.k)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    s = H().new_importance(B, 1, n, DEV)
    state = H().new_stream_state(B, 1, DEV)
    stream = torch.cuda.current_stream()
    ws = H().workspace(H().make_desc(q[0], k, v, s), max(k_sched), DEV)
    call, call_k = None, None
    s_ref = np.zeros((B, 1, n))
    qb, kb, vb = bits(x.q), bits(x.k), bits(x.v)
    classes = []
    for t, k_sel in enumerate(k_sched):
        if k_sel != call_k:
            call = H().StepCall(q[0], k, v, s, k_sel, ws=ws, stream=stream, stream_state=state,
                                stream_reset_calls=max(0, resets - t))
            call_k = k_sel
        before = state.cpu().numpy().copy()
        call(q[t].data_ptr())
        s_ref, idx_ref, out_ref = O.step(qb[t], kb, vb, s_ref, k_sel, dt)
        torch.cuda.synchronize()
        after = state.cpu().numpy()
        cls = stream_classes(before, after, n, k_sel) if t >= resets else [None] * B
        classes.append(cls)
        _check_step(x, t, s, call.idx, call.out, s_ref, idx_ref, out_ref, k_sel, "%s step %d" % (where, t))
    return classes


@pytest.mark.parametrize("layer", [0, 31])
def test_workload3_benchmark_regime(layer):
    """All 64 carried decode steps of one layer, as the benchmark runs them."""
    w = W.WORKLOADS[3]
    say("workload 3 layer %d: 3 reset steps, then 61 streamed steps (StepCall)" % layer)
    x = W.make_layer(w, layer)
    classes = [c[0] for c in _stepcall_run(x, [w.k_sel] * w.steps, "w3 L%d" % layer)]
    streamed = classes[3:]
    say("workload 3 layer %d threshold bin moves per streamed step: %s" % (layer, streamed))
    assert all(c is not None and c >= 0 for c in streamed), "a streamed step ran without its bound"
    assert any(c == 0 for c in streamed), "no step kept the bound's first-digit bin"
    # the selection loads the second-digit bins of the bound's bin and the next one with its
    # opening loads, and those of the window's two further bins on demand: all three paths run
    assert any(c == 1 for c in streamed), "no step moved to the next first-digit bin"
    assert any(c in (2, 3) for c in streamed), "no step moved two or three bins within the window"


def test_workload3_threshold_above_the_window():
    """A budget cut in mid-sequence (3276 -> 400 tokens; the bound stays
    valid since k only shrank) moves the threshold far above the bound's
    bin: the selection walks the update's pairs of the class above the
    window.  Against the oracle at every step."""
    w = W.WORKLOADS[3]
    x = W.make_layer(w.replace(steps=10), 0)
    sched = [w.k_sel] * 6 + [400] * 4
    classes = [c[0] for c in _stepcall_run(x, sched, "w3 cut")]
    say("budget cut: bin moves %s" % classes[3:])
    assert classes[6] is not None and classes[6] >= 4, classes


def test_workload4_ar1_steps_streamed_and_plain():
    """131K tokens, B 4, 16 AR(1) decode steps: StepCall with the streamed
    selection (three reset steps) and hill_step on separate copies of S,
    bit-identical to each other and matching the oracle at every step; the
    overlap of consecutive selections (temporal locality, Sec. 4.2) is
    reported for both."""
    w = W.WORKLOADS[4]
    say("workload 4: 16 AR(1) steps, streamed and plain")
    xg = W.make_layer(w, 0, device=DEV)
    x = W.LayerInputs(q=xg.q.cpu(), k=xg.k.cpu(), v=xg.v.cpu(), heavy=None)
    q, k, v = xg.q, xg.k, xg.v
    B, n, k_sel = w.batch, w.n_tokens, w.k_sel
    s_a = H().new_importance(B, 1, n, DEV)
    s_b = H().new_importance(B, 1, n, DEV)
    state = H().new_stream_state(B, 1, DEV)
    call = H().StepCall(q[0], k, v, s_b, k_sel, stream_state=state)
    qb, kb, vb = bits(x.q), bits(x.k), bits(x.v)
    s_ref = np.zeros((B, 1, n))
    prev, prev_ref, overlap, overlap_ref = None, None, [], []
    for t in range(w.steps):
        i_a, o_a = H().hill_step(q[t], k, v, s_a, k_sel)
        call(q[t].data_ptr())
        s_ref, idx_ref, out_ref = O.step(qb[t], kb, vb, s_ref, k_sel, "bf16")
        torch.cuda.synchronize()
        assert torch.equal(s_a, s_b) and torch.equal(i_a, call.idx) and torch.equal(o_a, call.out), "step %d" % t
        idx_g = _check_step(x, t, s_a, i_a, o_a, s_ref, idx_ref, out_ref, k_sel, "w4 step %d" % t)
        if prev is not None:
            overlap.append(np.mean([len(np.intersect1d(idx_g[b, 0], prev[b, 0])) / k_sel for b in range(B)]))
            overlap_ref.append(np.mean([len(np.intersect1d(idx_ref[b, 0], prev_ref[b, 0])) / k_sel
                                        for b in range(B)]))
        prev, prev_ref = idx_g, idx_ref
    say("workload 4 overlap |I_t & I_t-1| / k per step (GPU): %s" % " ".join("%.4f" % o for o in overlap))
    say("workload 4 overlap per step (oracle):            %s" % " ".join("%.4f" % o for o in overlap_ref))
    assert np.allclose(overlap, overlap_ref, atol=2e-3)


_SWEEP = W.sweep_workloads()
_SHAPES = sorted({(c.batch, c.n_tokens) for c in _SWEEP})


@pytest.mark.parametrize("batch,n", _SHAPES)
def test_sweep_cells_all(batch, n):
    """The three budgets of one (B, n) of the sweep, one decode step each
    from S = 0 (through StepCall as the sweep benchmark runs it), rows 0 and
    B-1 against the oracle."""
    cells = [c for c in _SWEEP if (c.batch, c.n_tokens) == (batch, n)]
    x = W.make_layer(cells[0], 0, device=DEV, seed=5000 + _SHAPES.index((batch, n)))
    for w in cells:
        say("sweep", w.name)
        s = H().new_importance(w.batch, 1, w.n_tokens, DEV)
        call = H().StepCall(x.q[0], x.k, x.v, s, w.k_sel)
        call(x.q[0].data_ptr())
        torch.cuda.synchronize()
        for b in sorted({0, w.batch - 1}):
            xb = W.LayerInputs(q=x.q[:, b:b + 1].cpu(), k=x.k[b:b + 1].cpu(), v=x.v[b:b + 1].cpu(), heavy=None)
            s_ref, idx_ref, out_ref = O.step(bits(xb.q[0]), bits(xb.k), bits(xb.v), np.zeros((1, 1, w.n_tokens)),
                                             w.k_sel, "bf16")
            _check_step(xb, 0, s[b:b + 1], call.idx[b:b + 1], call.out[b:b + 1], s_ref, idx_ref, out_ref, w.k_sel,
                        "%s b%d" % (w.name, b))
        del call, s
    del x
    torch.cuda.empty_cache()
