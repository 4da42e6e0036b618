"""Compiler resource report of the HIP kernels (no GPU needed): no kernel may
use scratch memory.  A private array that the compiler cannot keep in
registers (an indexed pick, an array captured by reference) moves the whole
per-lane state to scratch and costs the scan a factor of two, silently."""
import os

import pytest


@pytest.fixture(scope="module")
def report():
    from paper_2602_18750_amd import _build
    if not os.path.exists(_build.RESOURCES) or not os.path.exists(_build.LIB):
        _build.build()
    rows = [l.rstrip("\n").split("\t") for l in open(_build.RESOURCES) if l.strip()]
    return rows


def test_every_kernel_is_reported(report):
    names = " ".join(r[1] for r in report)
    for k in ("score_tiles_kernel", "update_attn_kernel", "topk_refine_kernel", "topk_emit_kernel",
              "merge_write_kernel", "sketch_keys_kernel", "bkp_rank_kernel", "calib_read_kernel"):
        assert k in names, k


def test_no_kernel_uses_scratch(report):
    bad = [(r[0], r[1], r[3]) for r in report if r[3] != "scratch=0"]
    assert not bad, bad
