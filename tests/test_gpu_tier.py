"""GPU checks of the tiered KV cache (include/hill.h): the hot pool in HBM,
the cold pool in pinned host memory that the kernels read and write in place,
rows moved between them by hill_tier_apply after each BKP pass (Sec. 4.2 BKP
(1)-(3)), and decode steps whose attention reads each selected row from the
pool that holds it.

* The slot table after every migration equals the oracle's tier_apply on the
  same lists, bit for bit, and every row sits where the table says, with the
  token's original values.
* Tiered steps (a BKP pass and a migration after each) give the same S,
  indices and outputs as hill_step_sketch over a cache holding every row in
  HBM, bit for bit, and outputs matching the oracle's attention on the
  selected set.
* Lists that do not fit the pool leave it untouched and raise the status."""
import sys

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2602_18750_amd import workloads as W
from parity import check_outputs
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


def _lists(promote, demote, counts):
    c = counts.cpu().numpy()
    p, d = promote.cpu().numpy(), demote.cpu().numpy()
    B, R = c.shape[0], c.shape[1]
    return ([[p[b, r, :c[b, r, 0]] for r in range(R)] for b in range(B)],
            [[d[b, r, :c[b, r, 1]] for r in range(R)] for b in range(B)])


def _check_placement(cache, k, v, n, where):
    """Every token's K and V rows sit where the slot table says: a hot token's
    in its slot of the hot pool, a cold token's at its position in the cold
    pool (rows of hot tokens in the cold pool are stale and not looked at)."""
    loc = cache.loc.cpu().numpy()[:, :, :n]
    kh, vh = cache.k_hot.cpu(), cache.v_hot.cpu()
    kc, vc = cache.k_cold, cache.v_cold
    kk, vv = k.cpu(), v.cpu()
    B, Hkv = kk.shape[0], kk.shape[1]
    for b in range(B):
        for g in range(Hkv):
            r = 0 if cache.R == 1 else g
            hot = np.nonzero(loc[b, r] >= 0)[0]
            cold = np.nonzero(loc[b, r] < 0)[0]
            slots = torch.from_numpy(loc[b, r, hot].astype(np.int64))
            hot_t = torch.from_numpy(hot.astype(np.int64))
            cold_t = torch.from_numpy(cold.astype(np.int64))
            assert torch.equal(kh[b, g, slots], kk[b, g, hot_t]), "%s: hot K rows (b %d, g %d)" % (where, b, g)
            assert torch.equal(vh[b, g, slots], vv[b, g, hot_t]), "%s: hot V rows (b %d, g %d)" % (where, b, g)
            assert torch.equal(kc[b, g, cold_t], kk[b, g, cold_t]), "%s: cold K rows (b %d, g %d)" % (where, b, g)
            assert torch.equal(vc[b, g, cold_t], vv[b, g, cold_t]), "%s: cold V rows (b %d, g %d)" % (where, b, g)


@pytest.mark.parametrize("gran", ["token", "kvhead"])
def test_migrations_follow_the_oracle(gran):
    """Random selections over a growing context, a BKP pass and a migration
    after each: the slot table equals the oracle's, the rows are in place."""
    B, Hkv, ncap, cap, win = 2, 4, 2400, 500, 64
    say("tier migrations", gran)
    x = W.make_random(B, 4 * Hkv, Hkv, 128, ncap, "bf16", steps=1, seed=606)
    k, v = x.k.to(DEV), x.v.to(DEV)
    cache = H().TieredCache(k, v, cap, granularity=gran, n_cap=ncap)
    R = cache.R
    bstate = H().BkpState(B, R, ncap, DEV)
    g = np.random.default_rng(7)
    loc_ref = np.full((B, R, ncap), -1, dtype=np.int64)
    n_prev = 0
    for t, n in enumerate([300, 700, 700, 1500, 1500, 2000, 2400, 2400]):
        kk = int(g.integers(1, 200))
        idx = np.stack([np.stack([np.sort(g.permutation(n)[:kk]) for _ in range(R)]) for _ in range(B)]).astype(np.int32)
        promote, demote, counts = H().bkp_update(bstate, torch.from_numpy(idx).to(DEV), n_tokens=n, n_recent=win,
                                                 capacity=cap)
        H().hill_tier_apply(cache, promote, demote, counts, n_tokens=n)
        torch.cuda.synchronize()
        pr, de = _lists(promote, demote, counts)
        loc_ref, _ = O.tier_apply(loc_ref, pr, de, n_prev, n, cap)
        n_prev = n
        assert int(cache.status.item()) == 0, "pass %d: status %d" % (t, cache.status.item())
        assert np.array_equal(cache.loc.cpu().numpy(), loc_ref), "pass %d: slot table" % t
        _check_placement(cache, k, v, n, "pass %d" % t)


def test_inconsistent_lists_leave_the_pool_untouched():
    B, Hkv, n, cap = 1, 2, 1000, 200
    x = W.make_random(B, 8, Hkv, 128, n, "bf16", steps=1, seed=11)
    k, v = x.k.to(DEV), x.v.to(DEV)
    cache = H().TieredCache(k, v, cap)
    bstate = H().BkpState(B, 1, n, DEV)
    idx = torch.arange(0, 100, dtype=torch.int32, device=DEV).view(1, 1, 100)
    promote, demote, counts = H().bkp_update(bstate, idx, n_tokens=n, n_recent=50, capacity=cap)
    cache.n_prev = 50     # wrong: the pool was empty, so this pass does not take it from 50 rows to 200
    loc0 = cache.loc.clone()
    H().hill_tier_apply(cache, promote, demote, counts, n_tokens=n)
    torch.cuda.synchronize()
    assert int(cache.status.item()) & 1
    assert torch.equal(cache.loc, loc0)
    cache.status.zero_()
    cache.n_prev = 0
    H().hill_tier_apply(cache, promote, demote, counts, n_tokens=n)
    torch.cuda.synchronize()
    assert int(cache.status.item()) == 0 and int((cache.loc >= 0).sum()) == cap
    _check_placement(cache, k, v, n, "after the retry")


@pytest.mark.parametrize("gran,streamed,nbits", [("token", True, 8), ("token", False, 8), ("kvhead", False, 8),
                                                 ("token", True, 4)])
def test_tiered_steps_equal_the_all_hbm_sketch_step(gran, streamed, nbits):
    """Decode steps over the tiered cache, with a BKP pass (window k, pool 2k)
    and a migration after each, against hill_step_sketch over the whole cache
    in HBM: identical S, indices and outputs; outputs against the oracle's
    attention over the selected set."""
    B, Hq, Hkv, n, k_sel, T = 2, 32, 8, 6000, 600, 6
    say("tiered steps", gran, streamed, nbits)
    x = W.make_random(B, Hq, Hkv, 128, n, "bf16", steps=T, seed=909 + nbits)
    q, k, v = x.q.to(DEV), x.k.to(DEV), x.v.to(DEV)
    cache = H().TieredCache(k, v, 2 * k_sel, granularity=gran, bits=nbits)
    R = cache.R
    bstate = H().BkpState(B, R, n, DEV)
    s_a = H().new_importance(B, R, n, DEV)
    s_b = H().new_importance(B, R, n, DEV)
    st_a = H().new_stream_state(B, R, DEV) if streamed else None
    st_b = H().new_stream_state(B, R, DEV) if streamed else None
    for t in range(T):
        i_a, o_a = H().hill_step(q[t], k, v, s_a, k_sel, granularity=gran, sketch=cache.sketch, stream_state=st_a,
                                 stream_reset=streamed and t == 0)
        i_b, o_b = H().hill_step_tiered(q[t], cache, s_b, k_sel, n_tokens=n, stream_state=st_b,
                                        stream_reset=streamed and t == 0)
        torch.cuda.synchronize()
        assert torch.equal(s_a, s_b), "step %d: S" % t
        assert torch.equal(i_a, i_b), "step %d: indices" % t
        assert torch.equal(o_a, o_b), "step %d: outputs" % t
        hot_frac = float((torch.gather(cache.loc.long(), 2, i_b.long()) >= 0).float().mean())
        own = O.sparse_attn(bits(x.q[t]), bits(x.k), bits(x.v), i_b.cpu().numpy(), "bf16", gran)
        check_outputs(o_b.cpu().numpy(), own, "tiered step %d" % t)
        promote, demote, counts = H().bkp_update(bstate, i_b, n_tokens=n, n_recent=k_sel, capacity=2 * k_sel)
        H().hill_tier_apply(cache, promote, demote, counts, n_tokens=n)
        torch.cuda.synchronize()
        assert int(cache.status.item()) == 0
        say("  step %d: %.3f of the selected rows were in the hot pool" % (t, hot_frac))
    _check_placement(cache, k, v, n, "end")


def test_tiered_steps_at_the_32k_workload():
    """The Llama-3-8B-shaped 32K layer (GQA 32/8, bf16, outlier keys, k 3276)
    with a hot pool of 2k tokens: eight streamed tiered steps (three reset
    steps first) equal the all-HBM sketch step bit for bit."""
    w = W.WORKLOADS[3].replace(steps=8)
    say("tiered steps, 32K workload")
    x = W.make_layer(w, 0, device=DEV)
    q, k, v = x.q, x.k, x.v
    cache = H().TieredCache(k, v, 2 * w.k_sel)
    bstate = H().BkpState(1, 1, w.n_tokens, DEV)
    s_a = H().new_importance(1, 1, w.n_tokens, DEV)
    s_b = H().new_importance(1, 1, w.n_tokens, DEV)
    st_a, st_b = H().new_stream_state(1, 1, DEV), H().new_stream_state(1, 1, DEV)
    for t in range(w.steps):
        i_a, o_a = H().hill_step(q[t], k, v, s_a, w.k_sel, sketch=cache.sketch, stream_state=st_a, stream_reset=t < 3)
        i_b, o_b = H().hill_step_tiered(q[t], cache, s_b, w.k_sel, n_tokens=w.n_tokens, stream_state=st_b,
                                        stream_reset=t < 3)
        promote, demote, counts = H().bkp_update(bstate, i_b, n_tokens=w.n_tokens, n_recent=w.k_sel,
                                                 capacity=2 * w.k_sel)
        H().hill_tier_apply(cache, promote, demote, counts, n_tokens=w.n_tokens)
        torch.cuda.synchronize()
        assert torch.equal(s_a, s_b) and torch.equal(i_a, i_b) and torch.equal(o_a, o_b), "step %d" % t
        assert int(cache.status.item()) == 0
    _check_placement(cache, k, v, w.n_tokens, "32K end")
