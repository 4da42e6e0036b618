"""C-ABI checks that need no GPU: the library loads, exports every function
include/hill.h declares, and every argument error is reported by its status
code before anything is enqueued.

No call here is valid as a whole, so no kernel is ever launched: each case
breaks exactly one rule, and the pointers are fake (never dereferenced,
because validation fails first)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hill.h")


@pytest.fixture(scope="module")
def H():
    import paper_2602_18750_amd as H
    if not os.path.exists(H.hill.LIB_PATH):
        from paper_2602_18750_amd import _build
        _build.build()
    H.load_library()
    return H


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hill_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    fns = declared_functions()
    for f in ("hill_score", "hill_topk", "hill_gather_attn", "hill_step", "hill_workspace_bytes",
              "hill_status_str", "hill_abi_version", "hill_last_error"):
        assert f in fns


def test_library_exports_every_declared_symbol(H):
    lib = H.load_library()
    for f in declared_functions():
        assert hasattr(lib, f), f
    assert sorted(H.hill.EXPORTS) == declared_functions()


def test_library_exports_nothing_else(H):
    """Built with hidden visibility: the dynamic symbol table holds the C
    entry points of include/hill.h and no internal (C++) function."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    H.load_library()
    lib_path = H.hill.LIB_PATH
    out = subprocess.run([nm, "-D", "--defined-only", lib_path], capture_output=True, text=True, check=True).stdout
    funcs = sorted(ln.split()[-1] for ln in out.splitlines() if len(ln.split()) == 3 and ln.split()[1] == "T")
    assert funcs == declared_functions()


def test_abi_version_and_status_strings(H):
    lib = H.load_library()
    want = int(re.search(r"#define HILL_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert lib.hill_abi_version() == want == H.hill.ABI_VERSION
    assert lib.hill_status_str(0) == b"HILL_OK"
    assert lib.hill_status_str(3) == b"HILL_ERR_WORKSPACE"
    assert lib.hill_status_str(99) == b"HILL_ERR_UNKNOWN"


def test_desc_layout_matches_header(H):
    # 10 x 4-byte fields, then 10 x int64 strides, then the two pinning counts
    assert ctypes.sizeof(H.HillDesc) == 40 + 80 + 8
    assert H.HillDesc.q_stride_b.offset == 40
    assert H.HillDesc.n_sink.offset == 120 and H.HillDesc.n_recent.offset == 124


FAKE = 0x10000          # 16-byte aligned, never dereferenced


def base_desc(H, B=2, Hq=8, Hkv=2, D=128, n=1000, mode=0, gran=0, dtype=1):
    d = H.HillDesc()
    d.struct_size = ctypes.sizeof(d)
    d.batch, d.n_q_heads, d.n_kv_heads, d.head_dim, d.n_tokens = B, Hq, Hkv, D, n
    d.dtype, d.score_mode, d.granularity, d.sm_scale = dtype, mode, gran, 0.0
    d.q_stride_b, d.q_stride_h = Hq * D, D
    d.k_stride_b, d.k_stride_h, d.k_stride_n = Hkv * n * D, n * D, D
    d.v_stride_b, d.v_stride_h, d.v_stride_n = Hkv * n * D, n * D, D
    R = 1 if gran == 0 else Hkv
    sr = (n + 3) // 4 * 4
    d.s_stride_r, d.s_stride_b = sr, R * sr
    return d


def ws_need(H, d, k):
    lib = H.load_library()
    out = ctypes.c_size_t()
    assert lib.hill_workspace_bytes(ctypes.byref(d), k, ctypes.byref(out)) == 0
    return out.value


def call_step(H, d, k=10, q=FAKE, kp=FAKE, v=FAKE, s=FAKE, idx=FAKE, out=FAKE, ws=FAKE, ws_bytes=None):
    lib = H.load_library()
    if ws_bytes is None:
        ws_bytes = ws_need(H, d, k)
    return lib.hill_step(ctypes.byref(d), q, kp, v, s, k, idx, out, ws, ws_bytes, None)


INVALID, UNSUPPORTED, WORKSPACE = 1, 2, 3


@pytest.mark.parametrize("field,value,code", [
    ("struct_size", 12, INVALID),
    ("batch", 0, INVALID),
    ("n_q_heads", 7, INVALID),          # not a multiple of n_kv_heads=2
    ("n_kv_heads", 0, INVALID),
    ("n_tokens", 0, INVALID),
    ("head_dim", 64, UNSUPPORTED),
    ("dtype", 2, UNSUPPORTED),
    ("score_mode", 5, INVALID),
    ("granularity", -1, INVALID),
    ("k_stride_n", 100, INVALID),       # not a multiple of 8
    ("v_stride_n", 64, INVALID),        # < head_dim
    ("q_stride_h", 4, INVALID),
    ("s_stride_r", 999, INVALID),       # < n_tokens
    ("s_stride_r", 1002, INVALID),      # not a multiple of 4
    ("s_stride_b", 1001, INVALID),      # not a multiple of 4
])
def test_descriptor_errors(H, field, value, code):
    d = base_desc(H)
    setattr(d, field, value)
    lib = H.load_library()
    st = call_step(H, d, ws_bytes=1 << 40)
    assert st == code, (field, lib.hill_last_error())
    assert lib.hill_last_error() != b""


def test_overlapping_importance_rows(H):
    d = base_desc(H, gran=1)            # R = 2 rows per sequence
    d.s_stride_b = d.s_stride_r         # second row of b would alias b+1
    assert call_step(H, d, ws_bytes=1 << 40) == INVALID


def test_sm_scale_must_be_finite(H):
    d = base_desc(H)
    d.sm_scale = float("nan")
    assert call_step(H, d, ws_bytes=1 << 40) == INVALID


@pytest.mark.parametrize("ksel", [0, -3, 1001])
def test_budget_out_of_range(H, ksel):
    d = base_desc(H)
    assert call_step(H, d, k=ksel, ws_bytes=1 << 40) == INVALID


@pytest.mark.parametrize("which", ["q", "kp", "v", "s", "idx", "out", "ws"])
def test_null_pointers(H, which):
    d = base_desc(H)
    assert call_step(H, d, **{which: None}) == INVALID


@pytest.mark.parametrize("which", ["q", "kp", "v", "s", "out", "ws"])
def test_misaligned_pointers(H, which):
    d = base_desc(H)
    assert call_step(H, d, **{which: FAKE + 8}) == INVALID


def test_workspace_too_small(H):
    d = base_desc(H)
    need = ws_need(H, d, 10)
    assert call_step(H, d, ws_bytes=need - 1) == WORKSPACE


def test_entry_points_validate_independently(H):
    lib = H.load_library()
    d = base_desc(H)
    need = ws_need(H, d, 10)
    assert lib.hill_score(ctypes.byref(d), FAKE, None, FAKE, FAKE, need, None) == INVALID
    assert lib.hill_topk(ctypes.byref(d), FAKE, 0, FAKE, None, FAKE, need, None) == INVALID
    assert lib.hill_topk(ctypes.byref(d), FAKE, 5, FAKE + 2, None, FAKE, need, None) == INVALID
    assert lib.hill_topk(ctypes.byref(d), FAKE, 5, FAKE, None, FAKE, 16, None) == WORKSPACE
    assert lib.hill_gather_attn(ctypes.byref(d), FAKE, FAKE, FAKE, None, 5, FAKE, FAKE, need, None) == INVALID
    assert lib.hill_gather_attn(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 5, FAKE + 4, FAKE, need, None) == INVALID
    assert lib.hill_workspace_bytes(None, 1, None) == INVALID


def test_workspace_sizes_are_pure_functions_of_shape(H):
    # 32K-token Llama-3-8B-shaped layer: logits dominate (32 heads x 32768 x 4 B)
    d = base_desc(H, B=1, Hq=32, Hkv=8, n=32768)
    a = ws_need(H, d, 3276)
    assert a == ws_need(H, d, 3276)
    assert a >= 32 * 32768 * 4
    # RAW with one row per KV head needs no logits buffer
    d_raw = base_desc(H, B=1, Hq=32, Hkv=8, n=32768, mode=1, gran=1)
    assert ws_need(H, d_raw, 3276) < a


# ------------------------------------------------------------- key sketch --

def test_sketch_entry_points_validate(H):
    lib = H.load_library()
    d = base_desc(H)                     # n = 1000
    need = ws_need(H, d, 10)
    ok_cap = 1000
    for bits in (8, 4):
        # sketch_keys: pointers, capacity, token range
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, None, FAKE, ok_cap, bits, 0, 10, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, None, ok_cap, bits, 0, 10, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE + 8, FAKE, ok_cap, bits, 0, 10, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE + 2, ok_cap, bits, 0, 10, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE, 996, bits, 0, 10, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE, 1002, bits, 0, 10, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE, ok_cap, bits, 5, 4, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE, ok_cap, bits, -1, 4, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE, ok_cap, bits, 0, 1001, None) == INVALID
        assert lib.hill_sketch_keys(ctypes.byref(d), None, FAKE, FAKE, ok_cap, bits, 0, 10, None) == INVALID
        # score / step on the sketch
        assert lib.hill_score_sketch(ctypes.byref(d), FAKE, None, FAKE, ok_cap, bits, FAKE, FAKE, need,
                                     None) == INVALID
        assert lib.hill_score_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, 996, bits, FAKE, FAKE, need, None) == INVALID
        assert lib.hill_score_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, ok_cap, bits, FAKE, FAKE, 16,
                                     None) == WORKSPACE
        assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, ok_cap, bits, FAKE, None, 0, 10,
                                    FAKE, FAKE, FAKE, need, None, None) == INVALID
        assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 1002, bits, FAKE, None, 0, 10,
                                    FAKE, FAKE, FAKE, need, None, None) == INVALID
        assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, ok_cap, bits, FAKE, None, 0, 0,
                                    FAKE, FAKE, FAKE, need, None, None) == INVALID
        # a streamed state must be 16-byte aligned, and needs ATTN scores
        assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, ok_cap, bits, FAKE, FAKE + 4, 0, 10,
                                    FAKE, FAKE, FAKE, need, None, None) == INVALID
        d.score_mode = 1
        assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, ok_cap, bits, FAKE, FAKE, 0, 10,
                                    FAKE, FAKE, FAKE, need, None, None) == UNSUPPORTED
        d.score_mode = 0
    # only 8 and 4 bits exist
    for bits in (0, 2, 6, 16):
        assert lib.hill_sketch_keys(ctypes.byref(d), FAKE, FAKE, FAKE, ok_cap, bits, 0, 10, None) == INVALID
        assert lib.hill_score_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, ok_cap, bits, FAKE, FAKE, need,
                                     None) == INVALID
        assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, ok_cap, bits, FAKE, None, 0, 10,
                                    FAKE, FAKE, FAKE, need, None, None) == INVALID
    assert b"bits" in lib.hill_last_error()


def test_head_count_limits(H):
    d = base_desc(H, Hq=512, Hkv=2)
    assert call_step(H, d, ws_bytes=1 << 40) == UNSUPPORTED
    d = base_desc(H, Hq=256, Hkv=1)      # 256 heads per KV head
    assert call_step(H, d, ws_bytes=1 << 40) == UNSUPPORTED


def test_calib_read_is_a_separate_library(H):
    """The benchmark's roofline calibration read lives in libhill_calib.so,
    outside libhill's ABI; it validates its arguments before launching."""
    from paper_2602_18750_amd import _build
    assert not hasattr(H.load_library(), "hill_calib_read")
    lib = ctypes.CDLL(_build.CALIB_LIB)
    fn = lib.hill_calib_read
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    assert fn(None, 1024, 4, FAKE, None) == 1
    assert fn(FAKE + 8, 1024, 4, FAKE, None) == 1     # misaligned buffer
    assert fn(FAKE, 1024, 4, None, None) == 1          # no sink
    assert fn(FAKE, 1000, 4, FAKE, None) == 1          # not a multiple of 16
    assert fn(FAKE, 0, 4, FAKE, None) == 1
    assert fn(FAKE, 1024, 0, FAKE, None) == 1
    assert fn(FAKE, 1024, 65537, FAKE, None) == 1


def test_step_events_layout_matches_header(H):
    text = open(HEADER).read()
    stages = re.findall(r"HILL_STAGE_([A-Z]+) = (\d+)", text)
    assert [n.lower() for n, _ in stages] == list(H.hill.STAGES)
    assert [int(v) for _, v in stages] == list(range(len(stages)))
    assert int(re.search(r"HILL_STAGES = (\d+)", text).group(1)) == len(H.hill.STAGES)
    assert ctypes.sizeof(H.HillStepEvents) == 2 * len(H.hill.STAGES) * ctypes.sizeof(ctypes.c_void_p)


def _bkp_desc(H, **kw):
    f = dict(batch=2, rows=3, n_tokens=1000, n_recent=10, capacity=100, stride_b=3 * 1000, stride_r=1000)
    f.update(kw)
    return H.BkpDesc(ctypes.sizeof(H.BkpDesc), f["batch"], f["rows"], f["n_tokens"], f["n_recent"],
                     f["capacity"], f["stride_b"], f["stride_r"])


def test_bkp_desc_layout_matches_header(H):
    text = open(HEADER).read()
    body = re.search(r"typedef struct hill_bkp_desc \{(.*?)\} hill_bkp_desc;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = re.findall(r"\b(\w+);", body)
    assert names == [f[0] for f in H.BkpDesc._fields_]
    assert ctypes.sizeof(H.BkpDesc) == 40


@pytest.mark.parametrize("field,value,code", [
    ("batch", 0, INVALID), ("rows", 0, INVALID), ("n_tokens", 0, INVALID), ("n_recent", -1, INVALID),
    ("capacity", 5, INVALID), ("stride_r", 999, INVALID), ("stride_b", 2999, INVALID),
    ("n_tokens", (1 << 21) + 1, UNSUPPORTED), ("batch", 30000, UNSUPPORTED),
])
def test_bkp_descriptor_errors(H, field, value, code):
    lib = H.load_library()
    kw = {field: value}
    if field == "n_tokens" and value > 1000:
        kw.update(stride_r=value, stride_b=3 * value)
    d = _bkp_desc(H, **kw)
    need = ctypes.c_size_t()
    assert lib.hill_bkp_workspace_bytes(ctypes.byref(d), ctypes.byref(need)) == code
    assert lib.hill_bkp_update(ctypes.byref(d), FAKE, 10, FAKE, FAKE, FAKE, FAKE, 10, FAKE, FAKE, 1 << 40,
                               None) == code
    assert lib.hill_last_error() != b""


def test_bkp_arguments_validate(H):
    lib = H.load_library()
    d = _bkp_desc(H)
    need = ctypes.c_size_t()
    assert lib.hill_bkp_workspace_bytes(ctypes.byref(d), ctypes.byref(need)) == 0 and need.value > 0
    ok = dict(idx=FAKE, k=10, hits=FAKE, hot=FAKE, pro=FAKE, dem=FAKE, cap=10, cnt=FAKE, ws=FAKE, wsb=need.value)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.hill_bkp_update(ctypes.byref(d), a["idx"], a["k"], a["hits"], a["hot"], a["pro"], a["dem"],
                                   a["cap"], a["cnt"], a["ws"], a["wsb"], None)

    assert call(k=-1) == INVALID and call(k=1001) == INVALID
    assert call(idx=None) == INVALID and call(idx=FAKE + 2) == INVALID
    assert call(hits=None) == INVALID and call(hits=FAKE + 1) == INVALID
    assert call(hot=None) == INVALID
    assert call(cap=-1) == INVALID and call(pro=None) == INVALID and call(dem=FAKE + 2) == INVALID
    assert call(cnt=None) == INVALID and call(cnt=FAKE + 1) == INVALID
    assert call(ws=None) == INVALID and call(ws=FAKE + 8) == INVALID
    assert call(wsb=need.value - 1) == WORKSPACE
    # the workspace size is a pure function of the descriptor
    need2 = ctypes.c_size_t()
    lib.hill_bkp_workspace_bytes(ctypes.byref(_bkp_desc(H)), ctypes.byref(need2))
    assert need2.value == need.value


def test_desc_field_names_match_header(H):
    text = open(HEADER).read()
    body = re.search(r"typedef struct hill_desc \{(.*?)\} hill_desc;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = []
    for decl in body.split(";"):
        decl = decl.strip()
        if decl:
            names += [x.strip() for x in decl.split(None, 1)[1].split(",")]
    assert names == [f[0] for f in H.HillDesc._fields_]


def test_pinned_tokens_need_room_in_the_budget(H):
    lib = H.load_library()
    d = base_desc(H)                     # n = 1000
    need = ws_need(H, d, 10)
    d.n_sink = -1
    assert lib.hill_topk(ctypes.byref(d), FAKE, 10, FAKE, None, FAKE, need, None) == INVALID
    d.n_sink, d.n_recent = 4, 7          # 11 pinned tokens
    assert lib.hill_topk(ctypes.byref(d), FAKE, 10, FAKE, None, FAKE, need, None) == INVALID
    assert b"pinned" in lib.hill_last_error()
    assert lib.hill_step(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 10, FAKE, FAKE, FAKE, need, None) == INVALID
    d.n_sink, d.n_recent = 600, 600      # the windows overlap: all 1000 tokens are pinned
    assert lib.hill_topk(ctypes.byref(d), FAKE, 999, FAKE, None, FAKE, 1 << 40, None) == INVALID
    # attention over a given list does not select: pins do not constrain it
    d.n_sink, d.n_recent = 4, 7
    assert lib.hill_gather_attn(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 10, FAKE, FAKE, 16, None) == WORKSPACE


def test_streamed_step_validates(H):
    lib = H.load_library()
    d = base_desc(H)
    need = ws_need(H, d, 10)
    args = lambda state, flags=0: (ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, state, flags, 10, FAKE, FAKE, FAKE, need,
                                   None, None)
    assert lib.hill_step_streamed(*args(None)) == INVALID
    assert lib.hill_step_streamed(*args(FAKE + 4)) == INVALID                 # not 16-byte aligned
    d.score_mode = 1                                                           # RAW: S can shrink
    assert lib.hill_step_streamed(*args(FAKE)) == UNSUPPORTED
    d.score_mode = 0
    assert lib.hill_step_streamed(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0, FAKE, FAKE, FAKE, need, None,
                                  None) == INVALID                            # k_sel
    assert lib.hill_step_streamed(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 0, 10, FAKE, FAKE, FAKE, 16, None,
                                  None) == WORKSPACE
    assert lib.hill_step_streamed(None, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 10, FAKE, FAKE, FAKE, need, None,
                                  None) == INVALID
    # flags: only HILL_STREAM_RESET exists; the reset step validates like the others
    assert lib.hill_step_streamed(*args(FAKE, 2)) == INVALID
    assert b"flags" in lib.hill_last_error()
    assert lib.hill_step_streamed(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 1, 10, FAKE, FAKE, FAKE, 16, None,
                                  None) == WORKSPACE
    assert lib.hill_step_sketch(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 1000, 8, FAKE, None, 1, 10,
                                FAKE, FAKE, FAKE, need, None, None) == INVALID   # flags without a state


def _tier_desc(H, **kw):
    f = dict(capacity=100, n_cap=1000, reserved=0, hot_stride_b=2 * 100 * 128, hot_stride_h=100 * 128,
             hot_stride_n=128)
    f.update(kw)
    return H.TierDesc(ctypes.sizeof(H.TierDesc), f["capacity"], f["n_cap"], f["reserved"], f["hot_stride_b"],
                      f["hot_stride_h"], f["hot_stride_n"])


def test_tier_desc_layout_matches_header(H):
    text = open(HEADER).read()
    body = re.search(r"typedef struct hill_tier_desc \{(.*?)\} hill_tier_desc;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = []
    for decl in body.split(";"):
        decl = decl.strip()
        if decl:
            names += [x.strip() for x in decl.split(None, 1)[1].split(",")]
    assert names == [f[0] for f in H.TierDesc._fields_]
    assert ctypes.sizeof(H.TierDesc) == 40


@pytest.mark.parametrize("field,value", [("capacity", 0), ("n_cap", 999), ("n_cap", 998), ("reserved", 1),
                                         ("hot_stride_n", 64), ("hot_stride_h", 12)])
def test_tier_arguments_validate(H, field, value):
    """Descriptor errors of the tiered entry points come back before any
    device query or launch (n_tokens 1000 here)."""
    lib = H.load_library()
    d = base_desc(H)
    t = _tier_desc(H, **{field: value})
    rc = lib.hill_tier_apply(ctypes.byref(d), ctypes.byref(t), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 100, FAKE, 0,
                             FAKE, None)
    assert rc == INVALID
    rc = lib.hill_step_tiered(ctypes.byref(d), ctypes.byref(t), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1000,
                              8, FAKE, None, 0, 10, FAKE, FAKE, FAKE, 1 << 40, None, None)
    assert rc == INVALID


def test_tier_apply_checks_its_lists_and_context(H):
    lib = H.load_library()
    d = base_desc(H)
    t = _tier_desc(H)
    args = lambda list_cap=100, n_prev=0, status=FAKE: (ctypes.byref(d), ctypes.byref(t), FAKE, FAKE, FAKE, FAKE, FAKE,
                                                        FAKE, FAKE, list_cap, FAKE, n_prev, status, None)
    assert lib.hill_tier_apply(*args(list_cap=0)) == INVALID
    assert lib.hill_tier_apply(*args(status=None)) == INVALID
    assert lib.hill_tier_apply(*args(n_prev=1001)) == INVALID       # more than n_tokens
    assert lib.hill_tier_apply(*args(n_prev=-1)) == INVALID
    assert lib.hill_tier_apply(None, ctypes.byref(t), *args()[2:]) == INVALID
    assert lib.hill_tier_apply(ctypes.byref(d), None, *args()[2:]) == INVALID
    # fake pointers pass the shape checks and are then refused as memory the GPU cannot reach
    assert lib.hill_tier_apply(*args()) == INVALID
    assert b"reach" in lib.hill_last_error()
    # a tiered step scores on the sketch
    assert lib.hill_step_tiered(ctypes.byref(d), ctypes.byref(t), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 1000,
                                8, FAKE, None, 0, 10, FAKE, FAKE, FAKE, 1 << 40, None, None) == INVALID


def test_stepcall_rejects_host_tensors(H):
    """StepCall checks where its tensors live before anything reaches the
    library: host tensors raise ValueError in the constructor (a host pointer
    taken for a device one would fault the GPU at the first launch)."""
    import torch
    q = torch.zeros((1, 4, 128), dtype=torch.bfloat16)
    k = torch.zeros((1, 2, 64, 128), dtype=torch.bfloat16)
    s = torch.zeros((1, 1, 64))
    with pytest.raises(ValueError, match="GPU tensors only"):
        H.StepCall(q, k, k, s, 8)
    with pytest.raises(ValueError, match="GPU tensors only"):
        H.StepCall(q, k, k, s, 8, stream_state=torch.zeros((1, 1, 8), dtype=torch.int32))
