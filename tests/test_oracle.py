"""Pins for the CPU oracle (run without a GPU).

Each test checks the oracle against something other than itself: a library
routine (torch / numpy), a closed form, an invariant the paper's definitions
imply, or brute force on tiny inputs.  The oracle is the yard-stick of the GPU
parity tests, so every function here is chosen so that a plausible slip in
it (a dropped term, a wrong sign, a wrong GQA index, a transposed operand,
a wrong scale, an off-by-one in selection) fails at least one test.
"""
import itertools
import math

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from util import bits, dname



# ---------------------------------------------------------------- decoding --

@pytest.mark.parametrize("tdt", [torch.float16, torch.bfloat16])
def test_decode16_exhaustive_matches_torch(tdt):
    """All 65536 bit patterns widen exactly as torch's .double() does."""
    pats = np.arange(65536, dtype=np.uint16)
    ref = torch.from_numpy(pats.view(np.int16).copy()).view(tdt).double().numpy()
    got = O.decode16(pats, "fp16" if tdt == torch.float16 else "bf16")
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


# ------------------------------------------------------------------ logits --

def _dense_logits_library(x):
    """q.K^T via torch.matmul with KV heads repeated per GQA group."""
    q = x.q[0].double()                      # [B,Hq,D]
    k = x.k.double()                         # [B,Hkv,n,D]
    G = q.shape[1] // k.shape[1]
    kr = k.repeat_interleave(G, dim=1)       # [B,Hq,n,D]
    return torch.matmul(kr, q.unsqueeze(-1)).squeeze(-1).numpy()


@pytest.mark.parametrize("B,Hq,Hkv,D,n,dt", [
    (1, 4, 4, 8, 5, "fp16"), (2, 8, 2, 16, 33, "bf16"), (1, 32, 1, 128, 7, "fp16"),
    (3, 6, 3, 4, 11, "bf16"),
])
def test_logits_match_library_matmul(B, Hq, Hkv, D, n, dt):
    x = W.make_random(B, Hq, Hkv, D, n, dt, seed=B * 100 + n)
    got = O.logits(bits(x.q[0]), bits(x.k), dt)
    ref = _dense_logits_library(x)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-12)


def test_logits_one_hot_keys_closed_form():
    """K rows equal to unit vectors e_i make l[h,j] = q[h, i_j] exactly."""
    B, Hq, Hkv, D, n = 1, 4, 2, 8, 8
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=3)
    k = torch.zeros(B, Hkv, n, D, dtype=torch.float16)
    for g in range(Hkv):
        for j in range(n):
            k[0, g, j, (j + 3 * g) % D] = 1.0
    l = O.logits(bits(x.q[0]), bits(k), "fp16")
    q = x.q[0].double().numpy()
    for h in range(Hq):
        g = h // (Hq // Hkv)
        for j in range(n):
            assert l[0, h, j] == q[0, h, (j + 3 * g) % D]


def test_logits_gqa_mapping_is_contiguous_groups():
    """kv(h) = h // G, not h % G: the two differ and the oracle follows the first."""
    B, Hq, Hkv, D, n = 1, 8, 2, 16, 9
    x = W.make_random(B, Hq, Hkv, D, n, "bf16", seed=5)
    got = O.logits(bits(x.q[0]), bits(x.k), "bf16")
    q, k = x.q[0].double().numpy(), x.k.double().numpy()
    G = Hq // Hkv
    right = np.stack([k[0, h // G] @ q[0, h] for h in range(Hq)])
    wrong = np.stack([k[0, h % Hkv] @ q[0, h] for h in range(Hq)])
    np.testing.assert_allclose(got[0], right, rtol=1e-13, atol=1e-12)
    assert not np.allclose(got[0], wrong)


# ----------------------------------------------------------------- weights --

@pytest.mark.parametrize("gran", ["token", "kvhead"])
@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (8, 1)])
def test_attn_update_matches_torch_softmax(gran, Hq, Hkv):
    B, D, n = 2, 16, 29
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=Hq * 10 + Hkv)
    l = O.logits(bits(x.q[0]), bits(x.k), "fp16")
    R = 1 if gran == "token" else Hkv
    S0 = np.random.default_rng(0).random((B, R, n))
    s = 1 / math.sqrt(D)
    got = O.update(l, S0, Hkv, "attn", gran, s)
    w = torch.softmax(torch.from_numpy(l) * s, dim=-1).numpy()     # [B,Hq,n]
    if gran == "token":
        ref = S0 + w.sum(axis=1, keepdims=True)
    else:
        ref = S0 + w.reshape(B, Hkv, Hq // Hkv, n).sum(axis=2)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("gran", ["token", "kvhead"])
def test_attn_update_column_mass_invariant(gran):
    """Each head's weights sum to one, so one step adds |heads(r)| to each row's total."""
    B, Hq, Hkv, D, n = 2, 32, 8, 128, 300
    x = W.make_random(B, Hq, Hkv, D, n, "bf16", seed=9, keys="outlier")
    l = O.logits(bits(x.q[0]), bits(x.k), "bf16")
    R = 1 if gran == "token" else Hkv
    S0 = np.zeros((B, R, n))
    S1 = O.update(l, S0, Hkv, "attn", gran, 1 / math.sqrt(128))
    per_row = Hq if gran == "token" else Hq // Hkv
    np.testing.assert_allclose(S1.sum(axis=-1), per_row, rtol=1e-12)
    assert (S1 > 0).all()


def test_attn_scale_is_inverse_sqrt_d():
    """A scale of 1/sqrt(D) (Eq. 1) gives softmax(l/sqrt(D)); 1/D or 1 give something else."""
    B, Hq, Hkv, D, n = 1, 2, 2, 64, 17
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=2)
    l = O.logits(bits(x.q[0]), bits(x.k), "fp16")
    S = O.update(l, np.zeros((B, Hkv, n)), Hkv, "attn", "kvhead", 1 / 8.0)
    for h in range(Hq):
        e = np.exp(l[0, h] / 8.0 - (l[0, h] / 8.0).max())
        np.testing.assert_allclose(S[0, h], e / e.sum(), rtol=1e-12)
        e2 = np.exp(l[0, h] / 64.0 - (l[0, h] / 64.0).max())
        assert not np.allclose(S[0, h], e2 / e2.sum())


def test_raw_update_linearity_closed_form():
    """RAW: S_T - S_0 = sum_{h in r} (sum_t q_{t,h}) . K_{kv(h)}^T (linear in q)."""
    B, Hq, Hkv, D, n, T = 2, 8, 2, 32, 19, 4
    x = W.make_random(B, Hq, Hkv, D, n, "bf16", steps=T, seed=4)
    S = np.zeros((B, Hkv, n))
    for t in range(T):
        l = O.logits(bits(x.q[t]), bits(x.k), "bf16")
        S = O.update(l, S, Hkv, "raw", "kvhead", 1 / math.sqrt(D))
    qs = x.q.double().sum(dim=0)                          # [B,Hq,D]
    k = x.k.double()
    G = Hq // Hkv
    ref = torch.einsum("bgjd,bgd->bgj", k, qs.view(B, Hkv, G, D).sum(dim=2)).numpy()
    np.testing.assert_allclose(S, ref, rtol=1e-11, atol=1e-10)


def test_multistep_is_sum_of_independent_steps():
    """The per-step softmax runs over all tokens, so S_T = sum_t (one-step S from zero)."""
    B, Hq, Hkv, D, n, T = 1, 8, 2, 16, 40, 5
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", steps=T, seed=6)
    S = np.zeros((B, 1, n))
    acc = np.zeros((B, 1, n))
    for t in range(T):
        S, idx, out = O.step(bits(x.q[t]), bits(x.k), bits(x.v), S, 7, "fp16")
        l = O.logits(bits(x.q[t]), bits(x.k), "fp16")
        acc += O.update(l, np.zeros((B, 1, n)), Hkv, "attn", "token", 1 / 4.0)
    np.testing.assert_allclose(S, acc, rtol=1e-12)


def test_raw_and_attn_select_the_same_tokens_for_one_mha_head_one_step():
    """Softmax is monotone: for one head, one step, from S=0, ranking is unchanged (Sec. 4.4)."""
    B, Hq, Hkv, D, n = 2, 4, 4, 64, 200
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=8)
    S0 = np.zeros((B, Hkv, n))
    _, ia, _ = O.step(bits(x.q[0]), bits(x.k), bits(x.v), S0, 37, "fp16", "attn", "kvhead")
    _, ir, _ = O.step(bits(x.q[0]), bits(x.k), bits(x.v), S0, 37, "fp16", "raw", "kvhead")
    assert np.array_equal(ia, ir)


def test_raw_and_attn_rank_differently_when_heads_are_summed():
    """Summed over heads the monotonicity argument breaks: token mode RAW != ATTN in general."""
    B, Hq, Hkv, D, n = 1, 32, 8, 128, 512
    x = W.make_random(B, Hq, Hkv, D, n, "bf16", seed=11, keys="outlier")
    S0 = np.zeros((B, 1, n))
    _, ia, _ = O.step(bits(x.q[0]), bits(x.k), bits(x.v), S0, 51, "bf16", "attn", "token")
    _, ir, _ = O.step(bits(x.q[0]), bits(x.k), bits(x.v), S0, 51, "bf16", "raw", "token")
    assert not np.array_equal(ia, ir)


# -------------------------------------------------------------------- top-k --

def _brute_topk(S, k):
    """numpy lexsort: primary key -S (NaN last), secondary token index."""
    out = []
    for row in S.reshape(-1, S.shape[-1]):
        n = row.size
        key = np.where(np.isnan(row), np.inf, -row)
        key = np.where(key == 0.0, 0.0, key)                      # -0 ties +0
        order = np.lexsort((np.arange(n), key))
        out.append(np.sort(order[:k]))
    return np.array(out, dtype=np.int32).reshape(S.shape[:-1] + (k,))


@settings(max_examples=150, deadline=None)
@given(st.data())
def test_topk_matches_full_sort_on_tie_heavy_rows(data):
    rows = data.draw(st.integers(1, 4))
    n = data.draw(st.integers(1, 300))
    k = data.draw(st.integers(1, n))
    grid = data.draw(st.sampled_from([2, 5, 17, 1000]))
    vals = data.draw(st.lists(st.integers(-grid, grid), min_size=rows * n, max_size=rows * n))
    S = np.array(vals, dtype=np.float64).reshape(rows, n) / 7.0
    assert np.array_equal(O.topk(S, k), _brute_topk(S, k))


def test_topk_special_cases():
    rng = np.random.default_rng(1)
    S = rng.standard_normal((3, 101))
    # k = 1 is argmax with the first occurrence winning
    S[1, 10] = S[1, 70] = S[1].max() + 1
    got = O.topk(S, 1)[:, 0]
    assert np.array_equal(got, np.argmax(S, axis=1))
    assert got[1] == 10
    # k = n is every index
    assert np.array_equal(O.topk(S, 101), np.tile(np.arange(101), (3, 1)))
    # all equal -> the lowest k indices
    assert np.array_equal(O.topk(np.full((2, 50), 0.25), 13), np.tile(np.arange(13), (2, 1)))
    # -0.0 and +0.0 tie: the lower index wins regardless of sign
    z = np.array([[1.0, -0.0, 0.0, -1.0, -0.0]])
    assert np.array_equal(O.topk(z, 2), [[0, 1]])
    assert np.array_equal(O.topk(z, 4), [[0, 1, 2, 4]])
    # NaN ranks below everything, -inf above NaN
    w = np.array([[np.nan, -np.inf, 3.0, np.nan, np.inf]])
    assert np.array_equal(O.topk(w, 3), [[1, 2, 4]])
    # output is ascending by token index
    big = rng.standard_normal((1, 1000))
    t = O.topk(big, 100)[0]
    assert np.all(np.diff(t) > 0)
    assert set(t) == set(np.argsort(-big[0])[:100])


def test_topk_off_by_one_is_caught():
    """The k-th largest is in, the (k+1)-th is out."""
    S = np.arange(20, dtype=np.float64)[None, ::-1].copy()      # 19..0
    got = O.topk(S, 5)[0]
    assert np.array_equal(got, [0, 1, 2, 3, 4])


# ---------------------------------------------------------------- attention --

def _sdpa_dense(x, scale=None):
    q = x.q[0].double().unsqueeze(2)                          # [B,Hq,1,D]
    G = x.q.shape[2] // x.k.shape[1]
    k = x.k.double().repeat_interleave(G, dim=1)
    v = x.v.double().repeat_interleave(G, dim=1)
    return torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale).squeeze(2).numpy()


@pytest.mark.parametrize("gran", ["token", "kvhead"])
@pytest.mark.parametrize("B,Hq,Hkv,D,n,dt", [(1, 4, 4, 32, 23, "fp16"), (2, 8, 2, 64, 50, "bf16"),
                                            (1, 32, 8, 128, 64, "bf16")])
def test_full_budget_reproduces_dense_sdpa(gran, B, Hq, Hkv, D, n, dt):
    x = W.make_random(B, Hq, Hkv, D, n, dt, seed=n)
    R = 1 if gran == "token" else Hkv
    _, idx, out = O.step(bits(x.q[0]), bits(x.k), bits(x.v), np.zeros((B, R, n)), n, dt, "attn", gran)
    assert np.array_equal(idx, np.tile(np.arange(n), (B, R, 1)))
    np.testing.assert_allclose(out, _sdpa_dense(x), rtol=1e-12, atol=1e-13)


def test_single_token_budget_returns_that_value_row():
    B, Hq, Hkv, D, n = 2, 8, 2, 16, 30
    x = W.make_random(B, Hq, Hkv, D, n, "bf16", seed=12)
    idx = np.array([[[7]], [[29]]], dtype=np.int32)
    out = O.sparse_attn(bits(x.q[0]), bits(x.k), bits(x.v), idx, "bf16", "token")
    v = x.v.double().numpy()
    for b in range(B):
        for h in range(Hq):
            assert np.array_equal(out[b, h], v[b, h // 4, idx[b, 0, 0]])


def test_sparse_attention_matches_library_on_subset_and_is_order_free():
    """Attention over I equals SDPA on the gathered rows, for any order of I."""
    B, Hq, Hkv, D, n = 1, 8, 2, 32, 60
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=13)
    I = np.array([3, 5, 11, 12, 40, 59], dtype=np.int32)
    out = O.sparse_attn(bits(x.q[0]), bits(x.k), bits(x.v), I[None, None], "fp16", "token")
    perm = O.sparse_attn(bits(x.q[0]), bits(x.k), bits(x.v), I[::-1].copy()[None, None], "fp16", "token")
    np.testing.assert_allclose(out, perm, rtol=1e-13, atol=1e-14)
    sub = W.LayerInputs(q=x.q, k=x.k[:, :, I], v=x.v[:, :, I], heavy=None)
    np.testing.assert_allclose(out, _sdpa_dense(sub), rtol=1e-12, atol=1e-13)


def test_kvhead_mode_attends_each_group_over_its_own_set():
    B, Hq, Hkv, D, n = 1, 4, 2, 16, 20
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=14)
    idx = np.array([[[0, 1, 2], [17, 18, 19]]], dtype=np.int32)
    out = O.sparse_attn(bits(x.q[0]), bits(x.k), bits(x.v), idx, "fp16", "kvhead")
    for g, I in enumerate(idx[0]):
        sub = W.LayerInputs(q=x.q[:, :, 2 * g:2 * g + 2], k=x.k[:, g:g + 1, I], v=x.v[:, g:g + 1, I],
                            heavy=None)
        np.testing.assert_allclose(out[:, 2 * g:2 * g + 2], _sdpa_dense(sub), rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------- workflow --

def test_step_orders_update_before_selection():
    """Selection uses S after this step's update (Sec. 4.1 workflow steps 5 then 6)."""
    B, Hq, Hkv, D, n = 1, 4, 4, 16, 50
    x = W.make_random(B, Hq, Hkv, D, n, "fp16", seed=15)
    S0 = np.zeros((B, 1, n))
    S1, idx, _ = O.step(bits(x.q[0]), bits(x.k), bits(x.v), S0, 10, "fp16")
    assert np.array_equal(idx, O.topk(S1, 10))


def test_budget_rounding():
    assert O.budget_k(4096, 0.20) == 819
    assert O.budget_k(32768, 0.10) == 3276
    assert O.budget_k(131072, 0.05) == 6553
    assert O.budget_k(65536, 0.20) == 13107
    assert O.budget_k(3, 0.05) == 1
    for n, a in itertools.product([8192, 32768, 65536], [0.05, 0.10, 0.20]):
        assert O.budget_k(n, a) == W.budget_tokens(n, a)


# ------------------------------------------ asymmetric-precision scoring --
# Sec. 4.4 (asymmetric precision): int8 casts of keys and query for scoring
# only.  The pins check the sketch against the bounds the power-of-two
# rounding rule implies and against the fp64 logits where the cast is exact.

def _decoded(t):
    return t.detach().double().numpy()


@pytest.mark.parametrize("dt", ["bf16", "fp16"])
def test_sketch_rounding_bound_range_and_minimal_exponent(dt):
    g = torch.Generator().manual_seed(11)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float16
    x = torch.randn(64, 128, generator=g)
    x = x * torch.exp(torch.randn(1, 128, generator=g))          # per-channel outliers
    x = x * torch.logspace(-3, 3, 64).unsqueeze(1)               # rows of very different size
    x = x.to(tdt)
    codes, exps = O.sketch(bits(x), dt)
    xd = _decoded(x)
    amax = np.abs(xd).max(axis=1)
    e = exps.astype(np.float64)
    step = np.exp2(e)[:, None]
    assert np.all(np.abs(xd - codes * step) <= step / 2)         # round to nearest
    assert np.all(np.abs(codes) <= 127)
    assert np.all(amax * np.exp2(-e) <= 127)                     # e large enough ...
    assert np.all(amax * np.exp2(-(e - 1)) > 127)                # ... and the smallest such
    assert np.all(np.abs(codes).max(axis=1) >= 64)               # half the code range at least


def test_sketch_ties_to_even_zero_and_tiny_rows():
    s = 8.0   # 2^3
    row = [127 * s, 2.5 * s, 3.5 * s, -2.5 * s, 0.5 * s, -0.5 * s, 1.5 * s, -1.5 * s] + [0.0] * 120
    zero = [0.0] * 128
    tiny = [2.0 ** -130] + [0.0] * 127                           # bf16 subnormal: exponent clamped
    x = torch.tensor([row, zero, tiny], dtype=torch.float32).to(torch.bfloat16)
    codes, exps = O.sketch(bits(x), "bf16")
    assert exps.tolist() == [3, -128, -128]
    assert codes[0, :8].tolist() == [127, 2, 4, -2, 0, 0, 2, -2]
    assert not codes[1].any() and not codes[2].any()


@pytest.mark.parametrize("B,Hq,Hkv,n", [(1, 4, 4, 9), (2, 8, 2, 17), (1, 32, 8, 5)])
def test_sketch_logits_exact_when_the_cast_is_lossless(B, Hq, Hkv, n):
    """Integers in [-127, 127] times 2^s with a row maximum of 127 * 2^s are
    cast without loss, so the sketch logits equal the fp64 logits exactly
    (including the GQA head mapping)."""
    g = np.random.default_rng(B * 31 + n)

    def rows(shape):
        v = g.integers(-127, 128, size=shape + (128,)).astype(np.float64)
        v[..., 0] = 127.0
        return v * np.exp2(g.integers(-6, 7, size=shape + (1,)))

    q = torch.from_numpy(rows((B, Hq))).to(torch.bfloat16)
    k = torch.from_numpy(rows((B, Hkv, n))).to(torch.bfloat16)
    q8, eq = O.sketch(bits(q), "bf16")
    k8, ek = O.sketch(bits(k), "bf16")
    l8 = O.logits_i8(q8, eq, k8, ek)
    l = O.logits(bits(q), bits(k), "bf16")
    assert np.array_equal(l8, l)


def test_sketch_logits_error_bound():
    """|l8 - l| <= sum_i |q_i| dk + |k_i| dq + dq dk with d = half a code step."""
    x = W.make_random(1, 8, 2, 128, 300, "bf16", seed=5)
    q8, eq = O.sketch(bits(x.q[0]), "bf16")
    k8, ek = O.sketch(bits(x.k), "bf16")
    l8 = O.logits_i8(q8, eq, k8, ek)
    l = O.logits(bits(x.q[0]), bits(x.k), "bf16")
    qd, kd = _decoded(x.q[0]), _decoded(x.k)                     # [1,8,128], [1,2,300,128]
    dq = np.exp2(eq.astype(np.float64) - 1)                      # [1,8]
    dk = np.exp2(ek.astype(np.float64) - 1)                      # [1,2,300]
    for h in range(8):
        g = h // 4
        bound = (np.abs(qd[0, h]).sum() * dk[0, g] + np.abs(kd[0, g]).sum(axis=1) * dq[0, h]
                 + 128 * dq[0, h] * dk[0, g])
        assert np.all(np.abs(l8[0, h] - l[0, h]) <= bound * (1 + 1e-12))


@pytest.mark.parametrize("wid,floor", [(3, 0.93), (1, 0.98)])
def test_sketch_selection_recall_vs_full_precision(wid, floor):
    """Quality statistic, not exactness: the top-alpha sets selected on sketch
    scores overlap the full-precision sets (4 steps, S carried).  Per-token
    scales lose most on the per-channel outlier keys of workload 3."""
    w = W.WORKLOADS[wid].replace(n_tokens=4096, steps=4, layers=1)
    x = W.make_layer(w, 0)
    k8, ek = O.sketch(bits(x.k), w.dtype)
    S = np.zeros((w.batch, 1, w.n_tokens))
    S8 = np.zeros_like(S)
    k = O.budget_k(w.n_tokens, w.budget)
    for t in range(w.steps):
        q8, eq = O.sketch(bits(x.q[t]), w.dtype)
        S = O.update(O.logits(bits(x.q[t]), bits(x.k), w.dtype), S, w.n_kv_heads, "attn", "token",
                     O.default_scale(128))
        S8 = O.update(O.logits_i8(q8, eq, k8, ek), S8, w.n_kv_heads, "attn", "token", O.default_scale(128))
        for b in range(w.batch):
            ov = len(np.intersect1d(O.topk(S[b:b + 1], k), O.topk(S8[b:b + 1], k))) / k
            assert ov >= floor, (t, b, ov)


# ------------------------------------------- BKP hot/cold pools (Sec. 4.2) --

def _bkp(hits, hot, idx, n, w, c):
    h = np.array(hits, dtype=np.uint16)[None, None]
    o = np.array(hot, dtype=bool)[None, None]
    i = np.array(idx, dtype=np.int64).reshape(1, 1, -1)
    h2, o2, pr, de = O.bkp_update(h, o, i, n, w, c)
    return h2[0, 0], o2[0, 0], list(pr[0][0]), list(de[0][0])


def test_bkp_worked_cases():
    # N=10, window W=2 (tokens 8, 9), capacity 5: three frequency slots.
    # Hits after the step: token 2 -> 4, token 4 -> 1; non-recent ranking 0 (5), 2 (4), 3 (3).
    h, o, pr, de = _bkp([5, 0, 3, 3, 0, 1, 0, 0, 9, 9], [1, 0, 0, 1, 0, 0, 0, 0, 1, 1], [2, 4], 10, 2, 5)
    assert list(h) == [5, 0, 4, 3, 1, 1, 0, 0, 9, 9]
    assert list(np.nonzero(o)[0]) == [0, 2, 3, 8, 9] and pr == [2] and de == []
    # Full pool: token 6 reaches 4 hits and displaces token 3 (3 hits), the lowest-ranked hot one.
    h, o, pr, de = _bkp([5, 0, 4, 3, 1, 1, 3, 0, 9, 9], [1, 0, 1, 1, 0, 0, 0, 0, 1, 1], [6], 10, 2, 5)
    assert list(np.nonzero(o)[0]) == [0, 2, 6, 8, 9] and pr == [6] and de == [3]
    # Equal hits: the incumbent keeps its slot even though the cold token has the lower index.
    h, o, pr, de = _bkp([0, 2, 2, 0], [0, 0, 1, 0], [1], 4, 0, 1)
    assert list(h) == [0, 3, 2, 0] and pr == [1] and de == [2]          # 3 > 2: strict, promoted
    h, o, pr, de = _bkp([0, 2, 3, 0], [0, 0, 1, 0], [1], 4, 0, 1)
    assert list(h) == [0, 3, 3, 0] and pr == [] and de == []            # tie: incumbent stays
    # The window moves as the context grows: token 5 enters it, token 3 leaves and must compete.
    h, o, pr, de = _bkp([1, 0, 0, 0, 9, 0, 7, 7], [1, 0, 0, 1, 1, 0, 0, 0], [], 6, 2, 3)
    assert list(np.nonzero(o[:6])[0]) == [0, 4, 5] and pr == [5] and de == [3]
    assert list(h) == [1, 0, 0, 0, 9, 0, 7, 7] and list(o[6:]) == [False, False]   # beyond n untouched
    # Saturation of the 2-byte table.
    h, o, pr, de = _bkp([65535, 65534, 0], [0, 0, 0], [0, 1], 3, 0, 2)
    assert list(h) == [65535, 65535, 0] and pr == [0, 1]


def _rank_key(h, old, j):
    return (int(h[j]), bool(old[j]), -j)   # larger is better


@settings(max_examples=200, deadline=None)
@given(st.integers(1, 40), st.data())
def test_bkp_invariants(n, data):
    cap_n = n + data.draw(st.integers(0, 3))
    w = data.draw(st.integers(0, n + 2))
    c = data.draw(st.integers(w, n + 5))
    hits = np.array(data.draw(st.lists(st.integers(0, 65535) | st.integers(0, 4), min_size=cap_n, max_size=cap_n)))
    old = np.array(data.draw(st.lists(st.booleans(), min_size=cap_n, max_size=cap_n)))
    k = data.draw(st.integers(0, n))
    idx = np.sort(np.array(data.draw(st.permutations(list(range(n))))[:k], dtype=np.int64))
    h2, o2, pr, de = _bkp(hits, old, idx, n, w, c)
    sel = np.zeros(n, dtype=bool)
    sel[idx] = True
    assert np.array_equal(h2[:n], np.minimum(hits[:n] + sel, 65535))
    assert np.array_equal(h2[n:], hits[n:]) and np.array_equal(o2[n:], old[n:])
    W_ = min(w, n)
    assert o2[n - W_:n].all()                                         # recent tokens are hot
    assert o2[:n].sum() == min(c, n)                                  # the pool is full (or holds all)
    prs, des = set(pr), set(de)
    assert not prs & des and all(not old[j] for j in prs) and all(old[j] for j in des)
    assert set(np.nonzero(o2[:n])[0]) == (set(np.nonzero(old[:n])[0]) | prs) - des
    assert pr == sorted(pr) and de == sorted(de)
    rest = range(n - W_)
    hot_keys = [_rank_key(h2, old, j) for j in rest if o2[j]]
    cold_keys = [_rank_key(h2, old, j) for j in rest if not o2[j]]
    if hot_keys and cold_keys:
        assert min(hot_keys) > max(cold_keys)                         # every hot token outranks every cold one


def test_bkp_brute_force_by_enumeration():
    """On tiny rows, the frequency slots are the one subset of the non-recent
    tokens whose every member outranks every non-member; enumerate them all."""
    rng = np.random.default_rng(5)
    for _ in range(300):
        n = int(rng.integers(1, 9))
        w = int(rng.integers(0, n + 1))
        c = int(rng.integers(w, n + 2))
        hits = rng.integers(0, 3, n)
        old = rng.random(n) < 0.5
        h2, o2, _, _ = _bkp(hits, old, [], n, w, c)
        rest = list(range(n - w))
        F = max(0, min(c, n) - w)
        good = [set(s) for s in itertools.combinations(rest, F)
                if all(_rank_key(hits, old, a) > _rank_key(hits, old, b) for a in s for b in rest if b not in s)]
        assert len(good) == 1
        assert set(j for j in rest if o2[j]) == good[0]


def test_bkp_suppresses_ping_pong():
    """Two tokens selected alternately with one frequency slot: with the
    incumbent winning ties, the slot changes hands once, not every step."""
    n, moves = 6, 0
    hits = np.zeros(n, dtype=np.uint16)
    hot = np.zeros(n, dtype=bool)
    for t in range(20):
        sel = [1] if t % 2 == 0 else [0]
        hits, hot, pr, de = _bkp(hits, hot, sel, n, 0, 1)
        moves += len(pr)
    assert moves == 1 and hot[1] and not hot[0]


def test_bkp_recurring_sink_stays_hot():
    """A token selected at every step (an attention sink, Sec. 4.2 insight
    two) enters the pool within a few steps and is never demoted, while the
    other selected tokens change."""
    rng = np.random.default_rng(1)
    n, sink = 200, 17
    hits = np.zeros(n, dtype=np.uint16)
    hot = np.zeros(n, dtype=bool)
    first = None
    for t in range(40):
        others = rng.choice(np.setdiff1d(np.arange(n - 20), [sink]), 19, replace=False)
        sel = np.sort(np.append(others, sink))
        hits, hot, pr, de = _bkp(hits, hot, sel, n, 20, 30)
        if hot[sink] and first is None:
            first = t
        if first is not None:
            assert hot[sink] and sink not in de
    assert first is not None and first <= 2


# ------------------------------------------------- pinned selection (sinks, recent) --

def test_pinned_selection_without_pins_is_the_plain_top_k():
    rng = np.random.default_rng(3)
    S = rng.integers(0, 5, (4, 300)).astype(np.float64)
    assert np.array_equal(O.topk_pinned(S, 40), O.topk(S, 40))


@settings(max_examples=200, deadline=None)
@given(st.integers(1, 60), st.data())
def test_pinned_selection_by_brute_force(n, data):
    sink = data.draw(st.integers(0, n + 2))
    recent = data.draw(st.integers(0, n + 2))
    npin = min(n, min(sink, n) + min(recent, n))
    k = data.draw(st.integers(max(1, npin), n)) if npin <= n else n
    S = np.array(data.draw(st.lists(st.integers(-3, 3), min_size=n, max_size=n)), dtype=np.float64) / 2
    got = O.topk_pinned(S[None], k, sink, recent)[0]
    assert len(got) == k and np.all(np.diff(got) > 0)
    pinned = set(range(min(sink, n))) | set(range(n - min(recent, n), n))
    assert pinned <= set(got.tolist())
    free = [j for j in range(n) if j not in pinned]
    # the free slots hold the largest S among the unpinned tokens, ties to the lower index
    want = sorted(free, key=lambda j: (-S[j], j))[:k - len(pinned)]
    assert set(got.tolist()) - pinned == set(want)


def test_pinned_selection_cases():
    S = np.array([[9.0, 1, 8, 7, 0, 6, 5, 4]])
    assert list(O.topk_pinned(S, 4, 1, 2)[0]) == [0, 2, 6, 7]     # sink 0, recent 6-7, best free: 2 (8)
    assert list(O.topk_pinned(S, 3, 1, 2)[0]) == [0, 6, 7]        # k equals the pinned count
    assert list(O.topk_pinned(S, 8, 6, 6)[0]) == list(range(8))   # overlapping windows pin everything
    assert list(O.topk_pinned(S, 3, 0, 1)[0]) == [0, 2, 7]
    with pytest.raises(ValueError):
        O.topk_pinned(S, 2, 1, 2)


# --------------------------------------- APP capacity split (Sec. 4.3, Eqs. 2-4) --

def _eq4(f_c, f_s, b_c, b_s, a):
    """Eq. 4 as printed: beta = B_c f_c (B_s + alpha f_s) / (B_s f_s (B_c + alpha f_c))."""
    return b_c * f_c * (b_s + a * f_s) / (b_s * f_s * (b_c + a * f_c))


def _sec54(f_c, f_s, b_c, b_s, a):
    """The optimum quoted with the sensitivity analysis (Sec. 5.4)."""
    return f_c * (b_s * b_c + a * b_c * f_s + a * b_s * f_s) / (b_s * f_s * (b_c + a * f_c))


@settings(max_examples=200, deadline=None)
@given(st.floats(1e8, 1e11), st.floats(1e8, 1e11), st.floats(1e8, 1e11), st.floats(1e8, 1e11), st.floats(0, 1))
def test_app_balance_is_eq4(f_c, f_s, b_c, b_s, a):
    beta, mc, ms, tc, ts, capped = O.app_split(f_c, f_s, b_c, b_s, a, a, 1.0)
    assert not capped
    assert math.isclose(beta, _eq4(f_c, f_s, b_c, b_s, a), rel_tol=1e-9)
    assert math.isclose(tc, ts, rel_tol=1e-9) and math.isclose(mc + ms, 1.0)


def test_app_limits_and_bound():
    # scoring alone (nothing retained): the split follows the scoring throughputs
    beta = O.app_split(8e9, 2e9, 1e9, 1e9, 0.0, 0.0, 1.0)[0]
    assert math.isclose(beta, 4.0, rel_tol=1e-9)
    # scoring free (f -> inf): the split follows the transfer bandwidths
    beta = O.app_split(1e30, 1e30, 32e9, 8e9, 0.2, 0.2, 1.0)[0]
    assert math.isclose(beta, 4.0, rel_tol=1e-6)
    # identical pools split evenly
    assert math.isclose(O.app_split(5e9, 5e9, 7e9, 7e9, 0.3, 0.3, 2.0)[1], 1.0, rel_tol=1e-9)
    # the host-memory bound (Eq. 3) clips M_c, leaving the cold path the slower one
    beta, mc, ms, tc, ts, capped = O.app_split(10e9, 2e9, 25e9, 6e9, 0.2, 0.2, 100.0, m0=50.0)
    assert capped and mc == 50.0 and ms == 50.0 and beta == 1.0 and ts > tc
    # a larger retained fraction in the hot pool (the skew correction) moves bytes to the cold pool
    assert O.app_split(10e9, 2e9, 25e9, 6e9, 0.3, 0.1, 1.0)[1] < O.app_split(10e9, 2e9, 25e9, 6e9, 0.2, 0.2, 1.0)[1]


def test_app_sec54_variant_differs_by_one_term():
    """The optimum quoted in Sec. 5.4 is Eq. 4 plus alpha f_c / (B_c + alpha f_c);
    the balance of Eq. 2 gives Eq. 4 (the reading taken)."""
    for f_c, f_s, b_c, b_s, a in [(10e9, 2e9, 25e9, 6e9, 0.2), (3e9, 3e9, 8e9, 2e9, 0.1)]:
        assert math.isclose(_sec54(f_c, f_s, b_c, b_s, a) - _eq4(f_c, f_s, b_c, b_s, a),
                            a * f_c / (b_c + a * f_c), rel_tol=1e-9)
        beta = O.app_split(f_c, f_s, b_c, b_s, a, a, 1.0)[0]
        assert not math.isclose(beta, _sec54(f_c, f_s, b_c, b_s, a), rel_tol=1e-3)


# ------------------------------------------------------- int4 key sketch (Sec. 4.4) --

@pytest.mark.parametrize("dt", ["bf16", "fp16"])
def test_sketch4_rounding_bound_range_and_minimal_exponent(dt):
    g = torch.Generator().manual_seed(12)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float16
    x = torch.randn(64, 128, generator=g) * torch.exp(torch.randn(1, 128, generator=g))
    x = (x * torch.logspace(-3, 3, 64).unsqueeze(1)).to(tdt)
    codes, exps = O.sketch(bits(x), dt, bits=4)
    xd = _decoded(x)
    amax = np.abs(xd).max(axis=1)
    e = exps.astype(np.float64)
    step = np.exp2(e)[:, None]
    assert np.all(np.abs(xd - codes * step) <= step / 2)
    assert np.all(np.abs(codes) <= 7)
    assert np.all(amax * np.exp2(-e) <= 7)
    assert np.all(amax * np.exp2(-(e - 1)) > 7)
    assert np.all(np.abs(codes).max(axis=1) >= 4)


def test_sketch4_ties_to_even_and_zero_rows():
    s = 8.0
    row = [7 * s, 2.5 * s, 3.5 * s, -2.5 * s, 0.5 * s, -0.5 * s, 1.5 * s, -1.5 * s] + [0.0] * 120
    over = [7.5 * s] + [6.5 * s] + [0.0] * 126                   # 7.5 needs the next exponent
    x = torch.tensor([row, [0.0] * 128, over], dtype=torch.float32).to(torch.bfloat16)
    codes, exps = O.sketch(bits(x), "bf16", bits=4)
    assert exps.tolist() == [3, -128, 4]
    assert codes[0, :8].tolist() == [7, 2, 4, -2, 0, 0, 2, -2]
    assert not codes[1].any()
    assert codes[2, :2].tolist() == [4, 3]                       # 3.75 -> 4, 3.25 -> 3


@pytest.mark.parametrize("B,Hq,Hkv,n", [(1, 4, 4, 9), (2, 8, 2, 17)])
def test_sketch4_logits_exact_when_the_cast_is_lossless(B, Hq, Hkv, n):
    """Keys on the int4 grid (integers in [-7, 7] times 2^s, row maximum 7 * 2^s)
    and queries on the int8 grid are cast without loss: the asymmetric-precision
    logits equal the fp64 logits exactly."""
    g = np.random.default_rng(B * 37 + n)

    def rows(shape, qmax):
        v = g.integers(-qmax, qmax + 1, size=shape + (128,)).astype(np.float64)
        v[..., 0] = qmax
        return v * np.exp2(g.integers(-6, 7, size=shape + (1,)))

    q = torch.from_numpy(rows((B, Hq), 127)).to(torch.bfloat16)
    k = torch.from_numpy(rows((B, Hkv, n), 7)).to(torch.bfloat16)
    q8, eq = O.sketch(bits(q), "bf16")
    k4, ek = O.sketch(bits(k), "bf16", bits=4)
    assert np.array_equal(O.logits_i8(q8, eq, k4, ek), O.logits(bits(q), bits(k), "bf16"))


def test_sketch4_logits_error_bound():
    x = W.make_random(1, 8, 2, 128, 300, "bf16", seed=6)
    q8, eq = O.sketch(bits(x.q[0]), "bf16")
    k4, ek = O.sketch(bits(x.k), "bf16", bits=4)
    l4 = O.logits_i8(q8, eq, k4, ek)
    l = O.logits(bits(x.q[0]), bits(x.k), "bf16")
    qd, kd = _decoded(x.q[0]), _decoded(x.k)
    dq = np.exp2(eq.astype(np.float64) - 1)
    dk = np.exp2(ek.astype(np.float64) - 1)
    for h in range(8):
        g = h // 4
        bound = (np.abs(qd[0, h]).sum() * dk[0, g] + np.abs(kd[0, g]).sum(axis=1) * dq[0, h]
                 + 128 * dq[0, h] * dk[0, g])
        assert np.all(np.abs(l4[0, h] - l[0, h]) <= bound * (1 + 1e-12))


@pytest.mark.parametrize("wid,floor", [(3, 0.55), (1, 0.85)])
def test_sketch4_selection_recall_vs_full_precision(wid, floor):
    """Quality statistic: int4 keys (int8 queries) keep most of the 16-bit
    selection on plain keys and lose more on per-channel outliers, which a
    per-token scale with 7 levels cannot follow (workload 3)."""
    w = W.WORKLOADS[wid].replace(n_tokens=4096, steps=4, layers=1)
    x = W.make_layer(w, 0)
    k4, ek = O.sketch(bits(x.k), w.dtype, bits=4)
    S = np.zeros((w.batch, 1, w.n_tokens))
    S4 = np.zeros_like(S)
    k = O.budget_k(w.n_tokens, w.budget)
    for t in range(w.steps):
        q8, eq = O.sketch(bits(x.q[t]), w.dtype)
        S = O.update(O.logits(bits(x.q[t]), bits(x.k), w.dtype), S, w.n_kv_heads, "attn", "token",
                     O.default_scale(128))
        S4 = O.update(O.logits_i8(q8, eq, k4, ek), S4, w.n_kv_heads, "attn", "token", O.default_scale(128))
        for b in range(w.batch):
            assert len(np.intersect1d(O.topk(S[b:b + 1], k), O.topk(S4[b:b + 1], k))) / k >= floor


# ------------------------------------- tier migration (Sec. 4.2 BKP (3)) --

def _tier(loc, pr, de, n_prev, n, cap):
    l2, mv = O.tier_apply(np.array(loc)[None, None], [[np.array(pr)]], [[np.array(de)]], n_prev, n, cap)
    return list(l2[0, 0]), mv[0][0]


def test_tier_apply_worked_cases():
    # pool of 3 slots holding tokens 0 and 1 (n_prev 2); the context grows to 4 and the pass
    # promotes 2 and 3 and demotes 0: token 2 takes 0's slot, token 3 the first unused slot (2)
    loc, mv = _tier([0, 1, -1, -1], [2, 3], [0], 2, 4, 3)
    assert loc == [-1, 1, 0, 2]
    assert sorted(mv) == [(0, 0, -1), (2, 0, 1), (3, 2, 1)]
    # full pool, equal volume each way: slots pass in list order
    loc, mv = _tier([2, -1, 0, -1, 1, -1], [1, 3], [0, 4], 6, 6, 3)
    assert loc == [-1, 2, 0, 1, -1, -1]
    # nothing moves
    loc, mv = _tier([0, -1, 1], [], [], 3, 3, 2)
    assert loc == [0, -1, 1] and mv == []
    # filling an empty pool
    loc, mv = _tier([-1, -1, -1, -1], [0, 2, 3], [], 0, 4, 3)
    assert loc == [0, -1, 1, 2]


def test_tier_apply_rejects_inconsistent_lists():
    with pytest.raises(ValueError):
        _tier([0, 1, -1, -1], [2], [0], 2, 4, 3)          # the pool must grow by one
    with pytest.raises(ValueError):
        _tier([0, 1, -1, -1], [1, 2], [0], 2, 4, 3)       # 1 is hot already
    with pytest.raises(ValueError):
        _tier([0, 1, -1, -1], [2, 3], [3], 2, 4, 3)       # 3 is cold


@settings(max_examples=60, deadline=None)
@given(data=st.data())
def test_tier_apply_follows_the_pool_over_passes(data):
    """Many BKP passes with random selections and a growing context: after
    every migration the tokens with a slot are exactly the pool's hot set,
    the slots in use are exactly 0 .. min(capacity, N) - 1 with no slot
    shared, and a token keeps its slot while it stays hot."""
    n0 = data.draw(st.integers(1, 30))
    cap = data.draw(st.integers(1, 25))
    w = data.draw(st.integers(0, cap))
    steps = data.draw(st.integers(1, 6))
    ncap = n0 + 3 * steps
    hits = np.zeros((1, 1, ncap), dtype=np.uint16)
    hot = np.zeros((1, 1, ncap), dtype=bool)
    loc = np.full((1, 1, ncap), -1, dtype=np.int64)
    n_prev = 0
    n = n0
    for _ in range(steps):
        k = data.draw(st.integers(0, n))
        idx = np.sort(np.array(data.draw(st.permutations(list(range(n))))[:k], dtype=np.int64)).reshape(1, 1, -1)
        hits, hot2, pr, de = O.bkp_update(hits, hot, idx, n, w, cap)
        loc2, _ = O.tier_apply(loc, pr, de, n_prev, n, cap)
        assert np.array_equal(loc2[0, 0, :n] >= 0, hot2[0, 0, :n])
        slots = loc2[0, 0][loc2[0, 0] >= 0]
        assert sorted(slots.tolist()) == list(range(min(cap, n)))
        stay = hot[0, 0, :n] & hot2[0, 0, :n]
        assert np.array_equal(loc2[0, 0, :n][stay], loc[0, 0, :n][stay])
        loc, hot, n_prev = loc2, hot2, n
        n = min(ncap, n + data.draw(st.integers(0, 3)))
