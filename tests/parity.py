"""Comparison rules between the GPU path and the CPU oracle.

* Importance S: |S_gpu - S_ref| <= 2e-3 |S_ref| + floor, the relative
  criterion of the target statement (fp16/bf16 inputs, fp32 accumulation on
  the GPU, fp64 in the oracle).  The floor only covers what a relative bound
  cannot: 1e-7 max_j |S_ref[row]| for weights that underflow fp32 (ATTN), and
  for RAW scores, whose sums of signed logits cancel, 2^-18 times the same sum
  taken over |q_i k_i| (the fp32 rounding of a sum is relative to the sum of
  the magnitudes of its terms; 2^-18 is 64 units of fp32 roundoff).
* Selection: with tau the oracle's k-th largest S of the row and a band of
  1e-3 max(|tau|, 1e-5 max|S_ref|), every token above the band is selected,
  none below it is; the GPU row holds k distinct in-range indices, ascending.
  Outside the band the match is exact.
* Attention output: compared with the oracle's attention over the GPU's own
  index set (so near-tie swaps do not fail it): per (b, h),
  max_i |o - o_ref| <= 2e-3 max_i |o_ref|.
* Exact selection: on identical fp32 S input, GPU and oracle index sets are
  equal bit for bit.
"""
import os

import numpy as np

S_RTOL = 2e-3
S_FLOOR = 1e-7          # underflow floor, relative to the row's largest |S|
RAW_FLOOR = 2.0 ** -18  # cancellation floor of RAW sums, relative to their sum of |q_i k_i|
SEL_BAND = 1e-3
S_BAND_FLOOR = 1e-5     # the selection band's floor near tau = 0 (RAW rows), relative to max |S|
OUT_TOL = 2e-3

# (test id, where, worst relative error of the tokens judged by the relative
# criterion, tokens judged, tokens under the floor) per check_scores call
SCORE_RECORD = []


def abs_bits(x):
    """|x| of fp16/bf16 bit patterns (the sign bit cleared), exactly."""
    return np.asarray(x, dtype=np.uint16) & np.uint16(0x7FFF)


def raw_abs_update(acc, q_bits, k_bits, dtype, n_kv_heads, granularity):
    """acc plus this step's RAW accumulation over |q_i k_i|: the oracle's own
    logits and row sums, taken on the magnitudes of the 16-bit inputs."""
    from oracle import oracle as O
    l = O.logits(abs_bits(q_bits), abs_bits(k_bits), dtype)
    return O.update(l, acc, n_kv_heads, "raw", granularity, 1.0)


def raw_abs_update_logits(acc, l, n_kv_heads, granularity):
    """The same over exact logits (sketch scores: each logit is exact, only
    the row sums round): acc plus the row sums of |l|."""
    from oracle import oracle as O
    return O.update(np.abs(l), acc, n_kv_heads, "raw", granularity, 1.0)


def check_scores(s_gpu, s_ref, where="", abs_sum=None):
    """abs_sum: for RAW scores, the same accumulation over |q_i k_i| (see the
    module docstring); None for ATTN."""
    s_gpu = np.asarray(s_gpu, dtype=np.float64)
    s_ref = np.asarray(s_ref, dtype=np.float64)
    assert s_gpu.shape == s_ref.shape, (s_gpu.shape, s_ref.shape)
    floor = S_FLOOR * np.abs(s_ref).max(axis=-1, keepdims=True)
    if abs_sum is not None:
        floor = floor + RAW_FLOOR * np.asarray(abs_sum, dtype=np.float64)
    err = np.abs(s_gpu - s_ref)
    rel = S_RTOL * np.abs(s_ref)
    bad = err > rel + floor
    judged = rel > floor
    worst = float((err[judged] / np.abs(s_ref[judged])).max()) if judged.any() else 0.0
    SCORE_RECORD.append((os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], where, worst,
                         int(judged.sum()), int((~judged).sum())))
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError("%s: %d score mismatches; first at %s: gpu %r ref %r" %
                             (where, int(bad.sum()), tuple(i), s_gpu[tuple(i)], s_ref[tuple(i)]))


def check_selection(idx_gpu, s_ref, k, where=""):
    idx_gpu = np.asarray(idx_gpu)
    s_ref = np.asarray(s_ref, dtype=np.float64)
    rows = s_ref.reshape(-1, s_ref.shape[-1])
    sel = idx_gpu.reshape(-1, idx_gpu.shape[-1])
    n = rows.shape[1]
    assert sel.shape == (rows.shape[0], k), (sel.shape, k)
    for r in range(rows.shape[0]):
        row, got = rows[r], sel[r]
        assert np.all(np.diff(got) > 0), "%s row %d: indices not strictly ascending" % (where, r)
        assert got[0] >= 0 and got[-1] < n, "%s row %d: index out of range" % (where, r)
        tau = np.sort(row)[::-1][k - 1]
        band = SEL_BAND * max(abs(tau), S_BAND_FLOOR * np.abs(row).max())
        chosen = np.zeros(n, dtype=bool)
        chosen[got] = True
        must = row > tau + band
        mustnot = row < tau - band
        assert not (must & ~chosen).any(), "%s row %d: %d clear winners missed" % (
            where, r, int((must & ~chosen).sum()))
        assert not (mustnot & chosen).any(), "%s row %d: %d clear losers selected" % (
            where, r, int((mustnot & chosen).sum()))


def check_outputs(out_gpu, out_ref, where=""):
    out_gpu = np.asarray(out_gpu, dtype=np.float64)
    out_ref = np.asarray(out_ref, dtype=np.float64)
    assert out_gpu.shape == out_ref.shape
    scale = np.abs(out_ref).max(axis=-1, keepdims=True)
    err = np.abs(out_gpu - out_ref).max(axis=-1, keepdims=True)
    bad = err > OUT_TOL * scale
    if bad.any():
        i = np.argwhere(bad[..., 0])[0]
        raise AssertionError("%s: %d heads off; first %s: max err %g vs scale %g" %
                             (where, int(bad.sum()), tuple(i), float(err[tuple(i)][0]),
                              float(scale[tuple(i)][0])))
