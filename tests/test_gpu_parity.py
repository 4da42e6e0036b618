"""GPU parity: libhill (through its C ABI) against the CPU oracle on seeded
synthetic inputs.  Runs only on an MI355X with the library built."""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs, check_scores, check_selection, raw_abs_update, raw_abs_update_logits
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


def gpu_inputs(x):
    return x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)


def R_of(gran, Hkv):
    return 1 if gran == "token" else Hkv


# ------------------------------------------------------------------ scoring --

SCORE_CASES = [
    # B, Hq, Hkv, n, dtype, mode, gran
    (1, 32, 32, 4096, "fp16", "attn", "token"),
    (2, 8, 2, 1000, "bf16", "attn", "kvhead"),
    (1, 4, 4, 129, "fp16", "raw", "token"),
    (2, 8, 2, 1, "bf16", "attn", "token"),
    (1, 32, 1, 777, "bf16", "raw", "token"),
    (3, 6, 2, 300, "fp16", "attn", "kvhead"),
    (1, 16, 2, 5000, "bf16", "raw", "kvhead"),
    (1, 32, 8, 2049, "bf16", "attn", "token"),
    (2, 32, 8, 3000, "bf16", "raw", "token"),
    (1, 64, 2, 640, "fp16", "attn", "token"),
    # head counts that do not divide the update's 256 threads; a row just past
    # the length whose softmax partials the update reduces itself
    (1, 6, 3, 2000, "fp16", "attn", "token"),
    (1, 32, 8, 32768 + 129, "bf16", "attn", "token"),
    # the head-count limits: 256 query heads, 128 per KV head
    (1, 256, 2, 700, "bf16", "attn", "token"),
    (1, 256, 256, 300, "fp16", "raw", "kvhead"),
    # matrix-core scan (ATTN, G >= 4) with group sizes that leave query columns
    # empty (G = 5, 7) or take a second pass of 8 heads (G = 12), ragged lengths
    (2, 10, 2, 1001, "bf16", "attn", "token"),
    (1, 7, 1, 35, "bf16", "attn", "token"),
    (1, 12, 1, 333, "fp16", "attn", "kvhead"),
]


@pytest.mark.parametrize("B,Hq,Hkv,n,dt,mode,gran", SCORE_CASES)
def test_score_matches_oracle_over_steps(B, Hq, Hkv, n, dt, mode, gran):
    say("score case", B, Hq, Hkv, n, dt, mode, gran)
    T = 3
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=T, seed=n + 7 * Hq)
    q, k, v = gpu_inputs(x)
    R = R_of(gran, Hkv)
    s = H().new_importance(B, R, n, DEV)
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    for t in range(T):
        H().hill_score(q[t], k, s, mode=mode, granularity=gran)
        l = O.logits(bits(x.q[t]), bits(x.k), dt)
        s_ref = O.update(l, s_ref, Hkv, mode, gran, 1 / math.sqrt(128))
        if a_ref is not None:
            a_ref = raw_abs_update(a_ref, bits(x.q[t]), bits(x.k), dt, Hkv, gran)
        torch.cuda.synchronize()
        check_scores(s.cpu().numpy(), s_ref, "step %d" % t, abs_sum=a_ref)


# -------------------------------------------------------------------- top-k --

def _rows(kind, rows, n, seed):
    g = np.random.default_rng(seed)
    if kind == "normal":
        return g.standard_normal((rows, n)).astype(np.float32)
    if kind == "grid":          # heavy ties
        return (g.integers(-6, 7, (rows, n)) / 4.0).astype(np.float32)
    if kind == "equal":
        return np.full((rows, n), 0.125, dtype=np.float32)
    if kind == "signed":        # +-0, negatives, tiny and huge magnitudes
        a = g.choice(np.array([0.0, -0.0, -1.0, 1e-30, -1e-30, 3e38, -3e38, 2.5], dtype=np.float32),
                     size=(rows, n))
        return a.astype(np.float32)
    if kind == "nan":
        a = g.standard_normal((rows, n)).astype(np.float32)
        a[:, ::7] = np.nan
        a[:, 3::11] = -np.inf
        return a
    if kind == "lognormal":     # the shape of summed attention weights
        return np.exp(g.standard_normal((rows, n)) - 8).astype(np.float32)
    raise ValueError(kind)


TOPK_CASES = [
    ("normal", 1, 1, 1), ("normal", 2, 3, 2), ("normal", 1, 100, 37), ("grid", 3, 4096, 819),
    ("grid", 2, 4097, 4097), ("equal", 2, 5000, 17), ("signed", 2, 3000, 1500), ("nan", 2, 2000, 1999),
    ("lognormal", 1, 32768, 3276), ("lognormal", 4, 131072, 6553), ("grid", 1, 65536, 13107),
    ("normal", 8, 8192, 1), ("lognormal", 16, 9000, 450), ("nan", 1, 300, 300),
]


@pytest.mark.parametrize("kind,rows,n,k", TOPK_CASES)
@pytest.mark.parametrize("values", [False, True])
def test_topk_is_exact_on_identical_input(kind, rows, n, k, values):
    say("topk case", kind, rows, n, k, values)
    a = _rows(kind, rows, n, seed=n + rows)
    s = H().new_importance(rows, 1, n, DEV)
    s[:, 0, :] = torch.from_numpy(a).to(DEV)
    res = H().hill_topk(s, k, granularity="token", with_values=values)
    idx, val = res if values else (res, None)
    torch.cuda.synchronize()
    ref = O.topk(a.astype(np.float64), k)
    assert np.array_equal(idx.cpu().numpy()[:, 0, :], ref)
    if values:
        got = val.cpu().numpy()[:, 0, :]
        want = np.take_along_axis(a, ref, axis=1)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_topk_kvhead_rows():
    B, Hkv, n, k = 3, 4, 1500, 200
    a = _rows("grid", B * Hkv, n, seed=5).reshape(B, Hkv, n)
    s = H().new_importance(B, Hkv, n, DEV)
    s.copy_(torch.from_numpy(a))
    idx = H().hill_topk(s, k, granularity="kvhead")
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), O.topk(a.astype(np.float64), k))


# ---------------------------------------------------------------- attention --

ATTN_CASES = [
    # B, Hq, Hkv, n, k, dtype, gran
    (1, 32, 32, 4096, 819, "fp16", "token"),
    (2, 32, 8, 3000, 300, "bf16", "token"),
    (2, 8, 2, 500, 1, "bf16", "kvhead"),
    (1, 8, 8, 64, 64, "fp16", "token"),
    (1, 32, 1, 1000, 77, "fp16", "token"),
    (3, 6, 3, 333, 100, "bf16", "kvhead"),
    (1, 16, 2, 7000, 5000, "bf16", "token"),
]


@pytest.mark.parametrize("B,Hq,Hkv,n,k,dt,gran", ATTN_CASES)
def test_gather_attn_matches_oracle(B, Hq, Hkv, n, k, dt, gran):
    say("attn case", B, Hq, Hkv, n, k, dt, gran)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, seed=k + n)
    q, kk, v = gpu_inputs(x)
    R = R_of(gran, Hkv)
    g = np.random.default_rng(k)
    idx = np.stack([np.stack([g.permutation(n)[:k] for _ in range(R)]) for _ in range(B)]).astype(np.int32)
    out = H().hill_gather_attn(q[0], kk, v, torch.from_numpy(idx).to(DEV), granularity=gran)
    torch.cuda.synchronize()
    ref = O.sparse_attn(bits(x.q[0]), bits(x.k), bits(x.v), idx, dt, gran)
    check_outputs(out.cpu().numpy(), ref, "attn")


def test_single_token_attention_returns_value_rows():
    B, Hq, Hkv, n = 2, 8, 2, 100
    x = W.make_random(B, Hq, Hkv, 128, n, "bf16", seed=3)
    q, k, v = gpu_inputs(x)
    idx = torch.tensor([[[13]], [[99]]], dtype=torch.int32, device=DEV)
    out = H().hill_gather_attn(q[0], k, v, idx)
    torch.cuda.synchronize()
    want = torch.stack([x.v[0, :, 13].float().repeat_interleave(4, 0), x.v[1, :, 99].float().repeat_interleave(4, 0)])
    assert torch.equal(out.cpu(), want)


# --------------------------------------------------------------- full steps --

def run_steps(x, k_sel, mode, gran, steps, check_every=1, where=""):
    """hill_step over `steps` queries vs the oracle; returns final GPU (S, idx, out)."""
    B, Hkv, n = x.k.shape[0], x.k.shape[1], x.k.shape[2]
    dt = dname(x.k)
    q, k, v = gpu_inputs(x)
    R = R_of(gran, Hkv)
    s = H().new_importance(B, R, n, DEV)
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    for t in range(steps):
        idx, out = H().hill_step(q[t], k, v, s, k_sel, mode=mode, granularity=gran)
        s_ref, idx_ref, out_ref = O.step(bits(x.q[t]), bits(x.k), bits(x.v), s_ref, k_sel, dt, mode, gran)
        if a_ref is not None:
            a_ref = raw_abs_update(a_ref, bits(x.q[t]), bits(x.k), dt, Hkv, gran)
        if t % check_every == 0 or t == steps - 1:
            torch.cuda.synchronize()
            idx_g = idx.cpu().numpy()
            check_scores(s.cpu().numpy(), s_ref, "%s step %d S" % (where, t), abs_sum=a_ref)
            check_selection(idx_g, s_ref, k_sel, "%s step %d sel" % (where, t))
            out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, gran)
            check_outputs(out.cpu().numpy(), out_own, "%s step %d out" % (where, t))
            if np.array_equal(idx_g, idx_ref):
                check_outputs(out.cpu().numpy(), out_ref, "%s step %d out(direct)" % (where, t))
    return s, idx, out


@pytest.mark.parametrize("B,Hq,Hkv,n,k,dt,gran", [(2, 10, 2, 1001, 100, "bf16", "token"),
                                                   (1, 12, 1, 333, 40, "fp16", "kvhead"),
                                                   (1, 7, 1, 35, 9, "bf16", "token")])
def test_step_with_uneven_group_sizes(B, Hq, Hkv, n, k, dt, gran):
    """hill_step where the matrix-core scan leaves query columns empty (G = 5,
    7) or takes two passes (G = 12); the select+attend kernel then takes the
    scan's logits of those heads."""
    say("uneven group", B, Hq, Hkv, n, k, dt, gran)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=3, seed=n + Hq)
    run_steps(x, k, "attn", gran, 3, where="G %d" % (Hq // Hkv))


@pytest.mark.parametrize("mode,gran", [("attn", "token"), ("attn", "kvhead"), ("raw", "token"),
                                       ("raw", "kvhead")])
def test_step_config1_full_size(mode, gran):
    w = W.WORKLOADS[1]
    say("config 1", mode, gran)
    x = W.make_layer(w, 0)
    run_steps(x, w.k_sel, mode, gran, 1, where="cfg1")


def test_step_config2_layers_full_size():
    w = W.WORKLOADS[2]
    for layer in (0, 31):
        say("config 2 layer", layer)
        x = W.make_layer(w, layer)
        s, idx, _ = run_steps(x, w.k_sel, "attn", "token", 1, where="cfg2 L%d" % layer)
        idx = idx.cpu().numpy()
        recall = np.mean([np.isin(x.heavy[b].numpy(), idx[b, 0]).mean() for b in range(w.batch)])
        say("config 2 layer %d heavy-hitter recall %.3f" % (layer, recall))


def test_step_config3_multistep_full_size():
    w = W.WORKLOADS[3]
    say("config 3 layer 0, 6 steps")
    x = W.make_layer(w.replace(steps=6), 0)
    run_steps(x, w.k_sel, "attn", "token", 6, where="cfg3")


def test_step_config4_full_size():
    w = W.WORKLOADS[4]
    say("config 4, 2 steps")
    x = W.make_layer(w.replace(steps=2), 0, device=DEV)
    x = W.LayerInputs(q=x.q.cpu(), k=x.k.cpu(), v=x.v.cpu(), heavy=None)
    run_steps(x, w.k_sel, "attn", "token", 2, where="cfg4")


@pytest.mark.parametrize("cell", [0, 4, 8, 13, 21, 26])
def test_step_sweep_cells_sampled(cell):
    """Sweep cells at full size; batch rows are independent, so the oracle checks two of them.
    Cell 21 (32 x 32K tokens) reduces its softmax partials in the separate
    statistics launch because of the batch (the update would re-read 256 MiB
    of them), cell 26 (64K tokens) because of the row length."""
    w = W.sweep_workloads()[cell]
    say("sweep", w.name)
    x = W.make_layer(w, 0, device=DEV, seed=5000 + cell)
    q, k, v = x.q, x.k, x.v
    s = H().new_importance(w.batch, 1, w.n_tokens, DEV)
    idx, out = H().hill_step(q[0], k, v, s, w.k_sel)
    torch.cuda.synchronize()
    for b in sorted({0, w.batch - 1}):
        xb = W.LayerInputs(q=q[:, b:b + 1].cpu(), k=k[b:b + 1].cpu(), v=v[b:b + 1].cpu(), heavy=None)
        s_ref, idx_ref, out_ref = O.step(bits(xb.q[0]), bits(xb.k), bits(xb.v), np.zeros((1, 1, w.n_tokens)),
                                         w.k_sel, "bf16")
        check_scores(s[b:b + 1].cpu().numpy(), s_ref, "sweep b%d" % b)
        idx_b = idx[b:b + 1].cpu().numpy()
        check_selection(idx_b, s_ref, w.k_sel, "sweep b%d" % b)
        own = O.sparse_attn(bits(xb.q[0]), bits(xb.k), bits(xb.v), idx_b, "bf16", "token")
        check_outputs(out[b:b + 1].cpu().numpy(), own, "sweep b%d" % b)


# ---------------------------------------------------------- layout / state --

def test_strided_cache_query_and_scores():
    """K/V are views into a larger cache (Ncap > n), q a strided view, S padded rows."""
    B, Hq, Hkv, n, ncap, kk = 2, 8, 2, 900, 1024, 90
    x = W.make_random(B, Hq, Hkv, 128, n, "bf16", steps=2, seed=21)
    kc = torch.zeros(B, Hkv, ncap, 128, dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros(B, Hkv, ncap, 128, dtype=torch.bfloat16, device=DEV)
    kc[:, :, :n] = x.k.to(DEV)
    vc[:, :, :n] = x.v.to(DEV)
    qbig = torch.zeros(2, B, Hq, 256, dtype=torch.bfloat16, device=DEV)
    qbig[:, :, :, 64:192] = x.q.to(DEV)
    q = qbig[:, :, :, 64:192]
    s = H().new_importance(B, 1, ncap + 12, DEV)
    s_ref = np.zeros((B, 1, n))
    for t in range(2):
        idx, out = H().hill_step(q[t], kc, vc, s, kk, n_tokens=n)
        s_ref, idx_ref, out_ref = O.step(bits(x.q[t]), bits(x.k), bits(x.v), s_ref, kk, "bf16")
        torch.cuda.synchronize()
        check_scores(s[:, :, :n].cpu().numpy(), s_ref, "strided S")
        assert float(s[:, :, n:].abs().max()) == 0.0        # untouched beyond n
        check_selection(idx.cpu().numpy(), s_ref, kk, "strided sel")
        own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx.cpu().numpy(), "bf16", "token")
        check_outputs(out.cpu().numpy(), own, "strided out")


def test_append_one_token_per_step():
    """The context grows by one token per step; new tokens enter with S = 0."""
    B, Hq, Hkv, n0, T, kk = 1, 32, 8, 2000, 4, 200
    x = W.make_random(B, Hq, Hkv, 128, n0 + T, "bf16", steps=T, seed=31)
    q, k, v = gpu_inputs(x)
    s = H().new_importance(B, 1, n0 + T, DEV)
    s_ref = np.zeros((B, 1, n0 + T))
    for t in range(T):
        n = n0 + t + 1
        idx, out = H().hill_step(q[t], k, v, s, kk, n_tokens=n)
        sr, _, _ = O.step(bits(x.q[t]), bits(x.k[:, :, :n]), bits(x.v[:, :, :n]), s_ref[:, :, :n], kk, "bf16")
        s_ref[:, :, :n] = sr
        torch.cuda.synchronize()
        check_scores(s[:, :, :n].cpu().numpy(), sr, "append S")
        check_selection(idx.cpu().numpy(), sr, kk, "append sel")


def test_step_is_deterministic_and_resumable():
    w = W.WORKLOADS[3]
    x = W.make_layer(w.replace(steps=4, n_tokens=8192), 0)
    q, k, v = gpu_inputs(x)

    def run(s, ts):
        res = None
        for t in ts:
            res = H().hill_step(q[t], k, v, s, 819)
        torch.cuda.synchronize()
        return res

    s1 = H().new_importance(1, 1, 8192, DEV)
    i1, o1 = run(s1, range(4))
    s2 = H().new_importance(1, 1, 8192, DEV)
    run(s2, range(2))
    saved = s2.cpu().clone()
    s3 = H().new_importance(1, 1, 8192, DEV)
    s3.copy_(saved)
    i3, o3 = run(s3, range(2, 4))
    assert torch.equal(s1.cpu(), s3.cpu())
    assert torch.equal(i1.cpu(), i3.cpu())
    assert torch.equal(o1.cpu(), o3.cpu())
    s4 = H().new_importance(1, 1, 8192, DEV)
    i4, o4 = run(s4, range(4))
    assert torch.equal(s1.cpu(), s4.cpu()) and torch.equal(i1.cpu(), i4.cpu()) and torch.equal(o1.cpu(), o4.cpu())


@pytest.mark.parametrize("mode,gran", [("attn", "token"), ("raw", "kvhead")])
def test_step_graph_replays_match_eager(mode, gran):
    """hill_step captured in a HIP graph: every replay (with eager work and
    synchronisation between replays) equals the eager call sequence bit for
    bit -- the library enqueues kernels only, no memsets or allocations."""
    B, Hq, Hkv, n, kk = 2, 32, 8, 5000, 500
    say("graph replay", mode, gran)
    x = W.make_random(B, Hq, Hkv, 128, n, "bf16", steps=1, seed=4242)
    q, k, v = gpu_inputs(x)
    R = R_of(gran, Hkv)
    s_e = H().new_importance(B, R, n, DEV)
    eager = []
    for _ in range(4):
        i, o = H().hill_step(q[0], k, v, s_e, kk, mode=mode, granularity=gran)
        torch.cuda.synchronize()
        eager.append((i.cpu().clone(), o.cpu().clone(), s_e.cpu().clone()))
    cs = torch.cuda.Stream()
    s_g = H().new_importance(B, R, n, DEV)
    call = H().StepCall(q[0], k, v, s_g, kk, mode=mode, granularity=gran, stream=cs)
    qp = q[0].data_ptr()
    with torch.cuda.stream(cs):          # one-time host initialisation outside the capture
        call(qp)
    torch.cuda.synchronize()
    s_g.zero_()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cs):
        call(qp)
    torch.cuda.synchronize()
    assert torch.count_nonzero(s_g).item() == 0   # capturing executed nothing
    junk = torch.randn(256, 256, device=DEV)
    for r in range(4):
        g.replay()
        torch.cuda.synchronize()
        got = (call.idx.cpu(), call.out.cpu(), s_g.cpu())
        for a, e, name in zip(got, eager[r], ("idx", "out", "S")):
            assert torch.equal(a, e), "replay %d: %s differs from the eager call" % (r, name)
        junk = torch.mm(junk, junk.t().contiguous()) / 256.0   # eager work between replays
        torch.cuda.synchronize()


@pytest.mark.parametrize("mode,gran", [("attn", "token"), ("raw", "kvhead"), ("raw", "token")])
def test_step_equals_score_topk_attn_in_sequence(mode, gran):
    B, Hq, Hkv, n, kk = 2, 32, 8, 3000, 300
    x = W.make_random(B, Hq, Hkv, 128, n, "bf16", seed=41)
    q, k, v = gpu_inputs(x)
    R = R_of(gran, Hkv)
    s1 = H().new_importance(B, R, n, DEV)
    i1, o1 = H().hill_step(q[0], k, v, s1, kk, mode=mode, granularity=gran)
    s2 = H().new_importance(B, R, n, DEV)
    H().hill_score(q[0], k, s2, mode=mode, granularity=gran)
    i2 = H().hill_topk(s2, kk, granularity=gran, n_kv_heads=Hkv)
    o2 = H().hill_gather_attn(q[0], k, v, i2, granularity=gran)
    torch.cuda.synchronize()
    assert torch.equal(s1.cpu(), s2.cpu())
    assert torch.equal(i1.cpu(), i2.cpu())
    # hill_step attends per 512-token chunk with the scan's logits (ATTN),
    # hill_gather_attn per split of the index list with its own q.k: same
    # value, different fp32 summation order
    o1, o2 = o1.cpu().double(), o2.cpu().double()
    assert ((o1 - o2).abs().amax(-1) <= 1e-5 * o2.abs().amax(-1)).all()


@pytest.mark.parametrize("gran", ["token", "kvhead"])
def test_full_budget_equals_dense_attention(gran):
    B, Hq, Hkv, n = 1, 32, 8, 1000
    x = W.make_random(B, Hq, Hkv, 128, n, "fp16", seed=51)
    q, k, v = gpu_inputs(x)
    s = H().new_importance(B, R_of(gran, Hkv), n, DEV)
    idx, out = H().hill_step(q[0], k, v, s, n, granularity=gran)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy()[0, 0], np.arange(n))
    qd = x.q[0].double().unsqueeze(2)
    kd = x.k.double().repeat_interleave(4, 1)
    vd = x.v.double().repeat_interleave(4, 1)
    dense = torch.nn.functional.scaled_dot_product_attention(qd, kd, vd).squeeze(2).numpy()
    check_outputs(out.cpu().numpy(), dense, "dense")


def test_errors_raise_and_enqueue_nothing():
    x = W.make_random(1, 8, 2, 128, 100, "fp16", seed=1)
    q, k, v = gpu_inputs(x)
    s = H().new_importance(1, 1, 100, DEV)
    with pytest.raises(H().HillError):
        H().hill_step(q[0], k, v, s, 101)
    torch.cuda.synchronize()
    assert float(s.abs().max()) == 0.0


# ----------------------------------------------- asymmetric-precision sketch --

def _sketch_ref(x_k, dt, nbits=8):
    codes, exps = O.sketch(bits(x_k), dt, bits=nbits)
    return codes, exps


def _unpack4(packed):
    """Codes of the library's int4 layout (include/hill.h): each group of 8
    codes c0..c7 is one 4-byte word whose byte i is (c_i + 8) | (c_{i+4} + 8) << 4."""
    b = packed.view(np.uint8).astype(np.int16)
    lo, hi = (b & 15) - 8, (b >> 4) - 8                      # [..., 64]
    lo = lo.reshape(b.shape[:-1] + (16, 4))
    hi = hi.reshape(b.shape[:-1] + (16, 4))
    return np.concatenate([lo, hi], axis=-1).reshape(b.shape[:-1] + (128,)).astype(np.int8)


def _codes_of(sk):
    c = sk.codes.cpu().numpy()
    return c if sk.bits == 8 else _unpack4(c)


@pytest.mark.parametrize("nbits", [8, 4])
@pytest.mark.parametrize("dt,B,Hkv,n,t0,t1", [
    ("bf16", 1, 8, 4096, 0, 4096), ("fp16", 2, 4, 777, 0, 777), ("bf16", 2, 2, 1000, 123, 517),
    ("bf16", 1, 1, 5, 4, 5),
])
def test_sketch_keys_bit_exact(dt, B, Hkv, n, t0, t1, nbits):
    say("sketch keys", nbits, dt, B, Hkv, n, t0, t1)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float16
    g = torch.Generator().manual_seed(n + t0)
    k = torch.randn(B, Hkv, n, 128, generator=g) * torch.exp(torch.randn(1, Hkv, 1, 128, generator=g))
    k[:, :, ::97] = 0.0                                   # all-zero rows
    k[:, :, 1::89] *= 1e-30                               # tiny rows (exponent clamp)
    k[:, :, 2::53, :5] = 0.5                              # ties at half a code step in some rows
    k = k.to(tdt)
    sk = H().sketch_keys(k.to(DEV), token_begin=t0, token_end=t1, bits=nbits)
    torch.cuda.synchronize()
    codes, exps = _sketch_ref(k, dt, nbits)
    got_c, got_e = _codes_of(sk), sk.exps.cpu().numpy()
    assert np.array_equal(got_c[:, :, t0:t1], codes[:, :, t0:t1])
    assert np.array_equal(got_e[:, :, t0:t1], exps[:, :, t0:t1])
    raw = sk.codes.cpu().numpy()
    assert not raw[:, :, :t0].any() and not raw[:, :, t1:].any()              # untouched outside the range
    assert (got_e[:, :, :t0] == -128).all() and (got_e[:, :, t1:] == -128).all()


SKETCH_SCORE_CASES = [
    # B, Hq, Hkv, n, dtype, mode, gran
    (1, 32, 8, 4096, "bf16", "attn", "token"),
    (2, 8, 2, 1001, "fp16", "attn", "kvhead"),
    (1, 32, 32, 777, "fp16", "raw", "token"),
    (2, 16, 4, 2049, "bf16", "raw", "kvhead"),
    # the int8 matrix-core scan with empty query columns or two passes, ragged lengths
    (2, 10, 2, 1001, "fp16", "attn", "token"),
    (1, 12, 1, 333, "bf16", "attn", "kvhead"),
]


@pytest.mark.parametrize("nbits", [8, 4])
@pytest.mark.parametrize("B,Hq,Hkv,n,dt,mode,gran", SKETCH_SCORE_CASES)
def test_score_on_sketch_matches_oracle(B, Hq, Hkv, n, dt, mode, gran, nbits):
    say("sketch score", nbits, B, Hq, Hkv, n, dt, mode, gran)
    T = 2
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=T, seed=n + 3 * Hq)
    q, k, v = gpu_inputs(x)
    sk = H().sketch_keys(k, bits=nbits)
    k8, ek = _sketch_ref(x.k, dt, nbits)
    R = R_of(gran, Hkv)
    s = H().new_importance(B, R, n, DEV)
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    for t in range(T):
        H().hill_score(q[t], None, s, mode=mode, granularity=gran, sketch=sk)
        q8, eq = O.sketch(bits(x.q[t]), dt)
        l8 = O.logits_i8(q8, eq, k8, ek)
        s_ref = O.update(l8, s_ref, Hkv, mode, gran, 1 / math.sqrt(128))
        if a_ref is not None:
            a_ref = raw_abs_update_logits(a_ref, l8, Hkv, gran)
        torch.cuda.synchronize()
        check_scores(s.cpu().numpy(), s_ref, "sketch step %d" % t, abs_sum=a_ref)


@pytest.mark.parametrize("nbits", [8, 4])
@pytest.mark.parametrize("B,nh,n,dt", [(1, 16, 1000, "bf16"), (2, 8, 4099, "fp16")])
def test_sketch_logits_bit_exact(B, nh, n, dt, nbits):
    """A sketch logit is an integer dot product (at most 128 * 127 * 127 < 2^24
    in magnitude) times a power of two, so in fp32 it is exact.  RAW, KV-head
    rows of one head each, one step from S = 0: S is the logit itself, and the
    GPU's must equal the oracle's exact value bit for bit."""
    say("sketch logits exact", nbits, B, nh, n, dt)
    x = W.make_random(B, nh, nh, 128, n, dt, steps=1, seed=4242 + n)
    q, k, v = gpu_inputs(x)
    sk = H().sketch_keys(k, bits=nbits)
    k8, ek = _sketch_ref(x.k, dt, nbits)
    q8, eq = O.sketch(bits(x.q[0]), dt)
    ref = O.logits_i8(q8, eq, k8, ek).astype(np.float32)   # exact in fp64, hence in fp32
    s = H().new_importance(B, nh, n, DEV)
    H().hill_score(q[0], None, s, mode="raw", granularity="kvhead", sketch=sk)
    torch.cuda.synchronize()
    got = s.cpu().numpy()[:, :, :n]
    assert np.array_equal(got, ref.reshape(B, nh, n))


@pytest.mark.parametrize("nbits", [8, 4])
@pytest.mark.parametrize("B,Hq,Hkv,n,dt", [(1, 32, 8, 1000, "bf16"), (2, 8, 8, 4099, "fp16"), (1, 32, 2, 37, "bf16"),
                                           (1, 32, 1, 515, "fp16"), (3, 6, 2, 300, "bf16")])
def test_sketch_attn_logits_bit_exact(B, Hq, Hkv, n, dt, nbits):
    """ATTN scoring on the sketch (int4 with G >= 4 on the matrix cores, the
    rest on the vector units): the logits it leaves at the start of the
    workspace ([B, Hq, ld] fp32, ld = n rounded up to 4: the library's
    workspace layout) must equal the oracle's exact sketch logits bit for bit,
    for group sizes 4, 1, 16, 32 (two passes of 16 heads) and 3, and for
    ragged n."""
    say("sketch ATTN logits exact", nbits, B, Hq, Hkv, n, dt)
    x = W.make_random(B, Hq, Hkv, 128, n, dt, steps=1, seed=5151 + n + Hq)
    q, k, v = gpu_inputs(x)
    sk = H().sketch_keys(k, bits=nbits)
    k8, ek = _sketch_ref(x.k, dt, nbits)
    q8, eq = O.sketch(bits(x.q[0]), dt)
    ref = O.logits_i8(q8, eq, k8, ek).astype(np.float32)   # [B, Hq, n], exact
    s = H().new_importance(B, 1, n, DEV)
    desc = H().make_desc(q[0], k, None, s)
    ws = H().workspace(desc, 1, DEV)
    ws.fill_(0xFF)                                           # NaN pattern: every logit must be written
    H().hill_score(q[0], None, s, mode="attn", granularity="token", sketch=sk, ws=ws)
    torch.cuda.synchronize()
    ld = (n + 3) // 4 * 4
    got = ws[:B * Hq * ld * 4].view(torch.float32).cpu().numpy().reshape(B, Hq, ld)[:, :, :n]
    assert np.array_equal(got, ref.reshape(B, Hq, n))


def _run_sketch_steps(x, k_sel, mode, gran, steps, where, nbits=8):
    B, Hkv, n = x.k.shape[0], x.k.shape[1], x.k.shape[2]
    dt = dname(x.k)
    q, k, v = gpu_inputs(x)
    sk = H().sketch_keys(k, bits=nbits)
    k8, ek = _sketch_ref(x.k, dt, nbits)
    R = R_of(gran, Hkv)
    s = H().new_importance(B, R, n, DEV)
    s_ref = np.zeros((B, R, n))
    a_ref = np.zeros((B, R, n)) if mode == "raw" else None
    for t in range(steps):
        idx, out = H().hill_step(q[t], k, v, s, k_sel, mode=mode, granularity=gran, sketch=sk)
        q8, eq = O.sketch(bits(x.q[t]), dt)
        l8 = O.logits_i8(q8, eq, k8, ek)
        s_ref = O.update(l8, s_ref, Hkv, mode, gran, 1 / math.sqrt(128))
        if a_ref is not None:
            a_ref = raw_abs_update_logits(a_ref, l8, Hkv, gran)
        torch.cuda.synchronize()
        idx_g = idx.cpu().numpy()
        check_scores(s.cpu().numpy(), s_ref, "%s step %d S" % (where, t), abs_sum=a_ref)
        check_selection(idx_g, s_ref, k_sel, "%s step %d sel" % (where, t))
        # attention reads the 16-bit K and V of the selected tokens
        out_own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), idx_g, dt, gran)
        check_outputs(out.cpu().numpy(), out_own, "%s step %d out" % (where, t))


@pytest.mark.parametrize("nbits", [8, 4])
@pytest.mark.parametrize("mode,gran", [("attn", "token"), ("attn", "kvhead"), ("raw", "token")])
def test_step_on_sketch_matches_oracle(mode, gran, nbits):
    x = W.make_random(2, 32, 8, 128, 3000, "bf16", steps=3, seed=77)
    _run_sketch_steps(x, 300, mode, gran, 3, "sketch%d %s/%s" % (nbits, mode, gran), nbits)


@pytest.mark.parametrize("nbits", [8, 4])
def test_step_on_sketch_config3_full_size(nbits):
    w = W.WORKLOADS[3]
    say("sketch config 3 layer 0, 2 steps", nbits)
    x = W.make_layer(w.replace(steps=2), 0)
    _run_sketch_steps(x, w.k_sel, "attn", "token", 2, "sketch%d cfg3" % nbits, nbits)


@pytest.mark.parametrize("Hq,Hkv,n,k,dt,gran", [(256, 2, 700, 70, "bf16", "token"), (256, 256, 300, 30, "fp16", "kvhead"),
                                               (128, 1, 1000, 100, "bf16", "token")])
def test_step_at_head_count_limits(Hq, Hkv, n, k, dt, gran):
    """256 query heads, or 128 per KV head: the update reduces one head per
    thread, the fused attention walks 16 chunks of 8 heads (or 256 KV heads),
    and the scan passes over the group 16 times."""
    say("head-count limits", Hq, Hkv, n, k, dt, gran)
    x = W.make_random(1, Hq, Hkv, 128, n, dt, steps=2, seed=Hq + Hkv + n)
    run_steps(x, k, "attn", gran, 2, where="heads %d/%d" % (Hq, Hkv))


@pytest.mark.parametrize("nbits", [8, 4])
def test_sketch_step_at_the_group_limit(nbits):
    """128 query heads per KV head on the sketch: the int4 scan's matrix-core
    form takes the group in 8 passes of 16 heads."""
    x = W.make_random(1, 128, 1, 128, 1000, "bf16", steps=2, seed=99 + nbits)
    _run_sketch_steps(x, 100, "attn", "token", 2, "group limit sketch%d" % nbits, nbits)
