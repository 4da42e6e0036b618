"""Comparison rules between the GPU path and the CPU oracle.

* Importance S: |S_gpu - S_ref| <= 2e-3 |S_ref| + 1e-5 max_j |S_ref[row]|
  (fp16/bf16 inputs, fp32 accumulation on the GPU, fp64 in the oracle).
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
import numpy as np

S_RTOL = 2e-3
S_FLOOR = 1e-5
SEL_BAND = 1e-3
OUT_TOL = 2e-3


def check_scores(s_gpu, s_ref, where=""):
    s_gpu = np.asarray(s_gpu, dtype=np.float64)
    s_ref = np.asarray(s_ref, dtype=np.float64)
    assert s_gpu.shape == s_ref.shape, (s_gpu.shape, s_ref.shape)
    floor = S_FLOOR * np.abs(s_ref).max(axis=-1, keepdims=True)
    err = np.abs(s_gpu - s_ref)
    bad = err > S_RTOL * np.abs(s_ref) + floor
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
        band = SEL_BAND * max(abs(tau), S_FLOOR * np.abs(row).max())
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
