"""Python binding of libhill (ctypes).  Argument marshalling only: every step
of the path runs in the library's HIP kernels; torch supplies device memory
and the current stream.

The functions mirror the C-ABI entry points of ``include/hill.h``:

    hill_score(q, k, s, ...)                    S += column sums of this step's weights
    hill_topk(s, k_sel, ...)         -> idx[, val]
    hill_gather_attn(q, k, v, idx, ...) -> out
    hill_step(q, k, v, s, k_sel, ...)  -> (idx, out)
    sketch_keys(k, ...)              -> Sketch (int8 codes + exponents, Sec. 4.4)
    hill_score / hill_step(..., sketch=...)   score on the int8 sketch

Shapes: q [B, Hq, D]; k, v [B, Hkv, Ncap, D] (any strides with D contiguous);
s [B, R, >= n] fp32 with R = 1 (granularity "token") or Hkv ("kvhead");
idx [B, R, k_sel] int32; out [B, Hq, D] fp32.
"""
from __future__ import annotations

import ctypes
import math
import os
import threading
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("HILL_LIBRARY") or os.path.join(_PKG, "libhill.so")

HILL_OK = 0
STATUS = {0: "HILL_OK", 1: "HILL_ERR_INVALID_ARG", 2: "HILL_ERR_UNSUPPORTED", 3: "HILL_ERR_WORKSPACE",
          4: "HILL_ERR_HIP"}
DTYPES = {torch.float16: 0, torch.bfloat16: 1}
MODES = {"attn": 0, "raw": 1}
GRANS = {"token": 0, "kvhead": 1}

ABI_VERSION = 6   # HILL_ABI_VERSION of include/hill.h that this binding's structures follow
EXPORTS = ("hill_abi_version", "hill_status_str", "hill_last_error", "hill_workspace_bytes", "hill_score",
           "hill_topk", "hill_gather_attn", "hill_step", "hill_step_profiled", "hill_sketch_keys",
           "hill_score_sketch", "hill_step_sketch", "hill_bkp_workspace_bytes",
           "hill_bkp_update", "hill_app_balance", "hill_step_streamed", "hill_step_noalloc", "hill_tier_apply",
           "hill_step_tiered")


class HillError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (STATUS.get(status, status), msg))
        self.status = status


class HillDesc(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("n_tokens", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("score_mode", ctypes.c_int32),
        ("granularity", ctypes.c_int32),
        ("sm_scale", ctypes.c_float),
        ("q_stride_b", ctypes.c_int64),
        ("q_stride_h", ctypes.c_int64),
        ("k_stride_b", ctypes.c_int64),
        ("k_stride_h", ctypes.c_int64),
        ("k_stride_n", ctypes.c_int64),
        ("v_stride_b", ctypes.c_int64),
        ("v_stride_h", ctypes.c_int64),
        ("v_stride_n", ctypes.c_int64),
        ("s_stride_b", ctypes.c_int64),
        ("s_stride_r", ctypes.c_int64),
        ("n_sink", ctypes.c_int32),
        ("n_recent", ctypes.c_int32),
    ]


# Stages of a decode step (include/hill.h HILL_STAGE_*), in launch order.
STAGES = ("scan", "stats", "update", "refine", "select", "merge")


class HillStepEvents(ctypes.Structure):
    """Kernel timestamps of a decode step (hill_step_profiled and the streamed
    and sketch steps): hipEvent_t handles or None, per stage, stamped by the
    start and the end of that stage's launch."""
    _fields_ = [("start", ctypes.c_void_p * len(STAGES)), ("stop", ctypes.c_void_p * len(STAGES))]

    @classmethod
    def of(cls, starts, stops):
        """From two sequences of len(STAGES) event handles (ints or None)."""
        ev = cls()
        for i in range(len(STAGES)):
            ev.start[i] = starts[i]
            ev.stop[i] = stops[i]
        return ev


class BkpDesc(ctypes.Structure):
    """hill_bkp_desc (include/hill.h)."""
    _fields_ = [("struct_size", ctypes.c_uint32), ("batch", ctypes.c_int32), ("rows", ctypes.c_int32),
                ("n_tokens", ctypes.c_int32), ("n_recent", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("stride_b", ctypes.c_int64), ("stride_r", ctypes.c_int64)]


class TierDesc(ctypes.Structure):
    """hill_tier_desc (include/hill.h)."""
    _fields_ = [("struct_size", ctypes.c_uint32), ("capacity", ctypes.c_int32), ("n_cap", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("hot_stride_b", ctypes.c_int64), ("hot_stride_h", ctypes.c_int64),
                ("hot_stride_n", ctypes.c_int64)]


class AppParams(ctypes.Structure):
    """hill_app_params (include/hill.h)."""
    _fields_ = [(n, ctypes.c_double) for n in ("f_c", "f_s", "b_c", "b_s", "alpha_c", "alpha_s", "m", "m0")]


class AppPlan(ctypes.Structure):
    """hill_app_plan (include/hill.h)."""
    _fields_ = [(n, ctypes.c_double) for n in ("beta", "m_c", "m_s", "t_c", "t_s")] + [("capped", ctypes.c_int32)]


_lock = threading.Lock()
_lib = None


def load_library(path: str = LIB_PATH):
    """Load libhill.so (built in-tree by ``__graft_entry__.build()``).  Raises if absent:
    there is no fallback implementation."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(path):
            raise RuntimeError("libhill.so is not built (%s); run __graft_entry__.build()" % path)
        lib = ctypes.CDLL(path)
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        D = ctypes.POINTER(HillDesc)
        lib.hill_abi_version.argtypes = []
        lib.hill_abi_version.restype = ctypes.c_int
        lib.hill_status_str.argtypes = [ctypes.c_int]
        lib.hill_status_str.restype = ctypes.c_char_p
        lib.hill_last_error.argtypes = []
        lib.hill_last_error.restype = ctypes.c_char_p
        lib.hill_workspace_bytes.argtypes = [D, I32, ctypes.POINTER(SZ)]
        lib.hill_workspace_bytes.restype = ctypes.c_int
        lib.hill_score.argtypes = [D, P, P, P, P, SZ, P]
        lib.hill_score.restype = ctypes.c_int
        lib.hill_topk.argtypes = [D, P, I32, P, P, P, SZ, P]
        lib.hill_topk.restype = ctypes.c_int
        lib.hill_gather_attn.argtypes = [D, P, P, P, P, I32, P, P, SZ, P]
        lib.hill_gather_attn.restype = ctypes.c_int
        lib.hill_step.argtypes = [D, P, P, P, P, I32, P, P, P, SZ, P]
        lib.hill_step.restype = ctypes.c_int
        lib.hill_step_profiled.argtypes = [D, P, P, P, P, I32, P, P, P, SZ, P, ctypes.POINTER(HillStepEvents)]
        lib.hill_step_profiled.restype = ctypes.c_int
        I64 = ctypes.c_int64
        lib.hill_sketch_keys.argtypes = [D, P, P, P, I64, I32, I32, I32, P]
        lib.hill_sketch_keys.restype = ctypes.c_int
        lib.hill_score_sketch.argtypes = [D, P, P, P, I64, I32, P, P, SZ, P]
        lib.hill_score_sketch.restype = ctypes.c_int
        U32 = ctypes.c_uint32
        lib.hill_step_sketch.argtypes = [D, P, P, P, P, P, I64, I32, P, P, U32, I32, P, P, P, SZ, P,
                                         ctypes.POINTER(HillStepEvents)]
        lib.hill_step_sketch.restype = ctypes.c_int
        lib.hill_bkp_workspace_bytes.argtypes = [ctypes.POINTER(BkpDesc), ctypes.POINTER(SZ)]
        lib.hill_bkp_workspace_bytes.restype = ctypes.c_int
        lib.hill_bkp_update.argtypes = [ctypes.POINTER(BkpDesc), P, I32, P, P, P, P, I32, P, P, SZ, P]
        lib.hill_bkp_update.restype = ctypes.c_int
        lib.hill_step_streamed.argtypes = [D, P, P, P, P, P, U32, I32, P, P, P, SZ, P,
                                           ctypes.POINTER(HillStepEvents)]
        lib.hill_step_streamed.restype = ctypes.c_int
        lib.hill_step_noalloc.argtypes = [D, P, P, P, P, I32, P, P, P]
        lib.hill_step_noalloc.restype = ctypes.c_int
        T = ctypes.POINTER(TierDesc)
        lib.hill_tier_apply.argtypes = [D, T, P, P, P, P, P, P, P, I32, P, I32, P, P]
        lib.hill_tier_apply.restype = ctypes.c_int
        lib.hill_step_tiered.argtypes = [D, T, P, P, P, P, P, P, P, P, I64, I32, P, P, U32, I32, P, P, P, SZ, P,
                                         ctypes.POINTER(HillStepEvents)]
        lib.hill_step_tiered.restype = ctypes.c_int
        lib.hill_app_balance.argtypes = [ctypes.POINTER(AppParams), ctypes.POINTER(AppPlan)]
        lib.hill_app_balance.restype = ctypes.c_int
        if lib.hill_abi_version() != ABI_VERSION:
            raise RuntimeError("libhill.so has ABI version %d, this binding needs %d; rebuild it"
                               % (lib.hill_abi_version(), ABI_VERSION))
        _lib = lib
        return lib


def _check(status: int):
    if status != HILL_OK:
        raise HillError(status, _lib.hill_last_error().decode())


def budget_k(n: int, budget: float) -> int:
    """Token budget: floor(budget * n), at least 1 and at most n."""
    return max(1, min(n, int(math.floor(budget * n + 1e-9))))


def make_desc(q: Optional[torch.Tensor], k: Optional[torch.Tensor], v: Optional[torch.Tensor],
              s: Optional[torch.Tensor], *, mode: str = "attn", granularity: str = "token",
              n_tokens: Optional[int] = None, sm_scale: float = 0.0,
              shape: Optional[Tuple[int, int, int, int]] = None, dtype=None, n_sink: int = 0,
              n_recent: int = 0) -> HillDesc:
    """Descriptor from tensors.  ``shape`` = (B, Hq, Hkv, D) stands in when q/k are absent.
    ``n_sink`` / ``n_recent``: tokens at the start / end of the context that
    every selection keeps."""
    d = HillDesc()
    d.struct_size = ctypes.sizeof(HillDesc)
    if q is not None:
        B, Hq, D = q.shape
    else:
        B, Hq, _, D = shape
    if k is not None:
        _, Hkv, ncap, _ = k.shape
    else:
        Hkv = shape[2]
        ncap = s.shape[-1]
    n = ncap if n_tokens is None else int(n_tokens)
    d.batch, d.n_q_heads, d.n_kv_heads, d.head_dim, d.n_tokens = B, Hq, Hkv, D, n
    tdt = dtype if dtype is not None else (q.dtype if q is not None else k.dtype)
    d.dtype = DTYPES.get(tdt, -1)
    d.score_mode = MODES[mode]
    d.granularity = GRANS[granularity]
    d.sm_scale = float(sm_scale)
    d.n_sink, d.n_recent = int(n_sink), int(n_recent)
    if q is not None:
        d.q_stride_b, d.q_stride_h = q.stride(0), q.stride(1)
        _require_unit_last(q, "q")
    else:
        d.q_stride_b, d.q_stride_h = Hq * D, D
    if k is not None:
        d.k_stride_b, d.k_stride_h, d.k_stride_n = k.stride(0), k.stride(1), k.stride(2)
        _require_unit_last(k, "k")
    else:
        d.k_stride_b, d.k_stride_h, d.k_stride_n = Hkv * n * D, n * D, D
    if v is not None:
        d.v_stride_b, d.v_stride_h, d.v_stride_n = v.stride(0), v.stride(1), v.stride(2)
        _require_unit_last(v, "v")
    else:
        d.v_stride_b, d.v_stride_h, d.v_stride_n = d.k_stride_b, d.k_stride_h, d.k_stride_n
    if s is not None:
        d.s_stride_b, d.s_stride_r = s.stride(0), s.stride(1)
        if s.stride(2) != 1:
            raise ValueError("s must have a contiguous token axis")
    return d


def _require_unit_last(t: torch.Tensor, name: str):
    if t.stride(-1) != 1:
        raise ValueError("%s must have a contiguous last (head_dim) axis" % name)


def workspace_bytes(desc: HillDesc, k_sel: int) -> int:
    lib = load_library()
    out = ctypes.c_size_t(0)
    _check(lib.hill_workspace_bytes(ctypes.byref(desc), int(k_sel), ctypes.byref(out)))
    return int(out.value)


_ws_cache = {}


def workspace(desc: HillDesc, k_sel: int, device) -> torch.Tensor:
    """A cached per-device workspace, grown on demand.  Calls that share it must be
    ordered on one stream; pass ``ws=`` explicitly otherwise."""
    need = max(workspace_bytes(desc, k_sel), 256)
    dev = torch.device(device)
    buf = _ws_cache.get(dev)
    if buf is None or buf.numel() < need:
        buf = torch.empty(need, dtype=torch.uint8, device=dev)
        _ws_cache[dev] = buf
    return buf


def _stream_ptr(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _device_check(*ts):
    for t in ts:
        if t is not None and t.device.type != "cuda":
            raise ValueError("libhill works on GPU tensors only (got %s)" % t.device)


class Sketch:
    """Scoring sketch of a key cache (Sec. 4.4 asymmetric precision): codes
    [B, Hkv, cap, 128] int8 (bits 8) or [B, Hkv, cap, 64] packed int4 bytes
    (bits 4), and one exponent per row [B, Hkv, cap] int8."""

    def __init__(self, codes: torch.Tensor, exps: torch.Tensor, bits: int = 8):
        self.codes, self.exps, self.bits = codes, exps, int(bits)
        self.cap = codes.shape[2]


def new_sketch(B: int, Hkv: int, cap: int, device, bits: int = 8) -> Sketch:
    if bits not in (8, 4):
        raise ValueError("bits must be 8 or 4")
    cap = (cap + 3) // 4 * 4
    return Sketch(torch.zeros((B, Hkv, cap, 128 * bits // 8), dtype=torch.int8, device=device),
                  torch.full((B, Hkv, cap), -128, dtype=torch.int8, device=device), bits)


def sketch_keys(k, sketch: Optional[Sketch] = None, *, token_begin=0, token_end=None, n_tokens=None,
                stream=None, bits: int = 8) -> Sketch:
    """Write the sketch of key rows [token_begin, token_end) (default: all)."""
    lib = load_library()
    _device_check(k)
    B, Hkv, ncap, D = k.shape
    if sketch is None:
        sketch = new_sketch(B, Hkv, ncap, k.device, bits)
    n = ncap if n_tokens is None else int(n_tokens)
    t1 = n if token_end is None else int(token_end)
    desc = make_desc(None, k, None, None, n_tokens=n, shape=(B, Hkv, Hkv, D), dtype=k.dtype)
    _check(lib.hill_sketch_keys(ctypes.byref(desc), _ptr(k), _ptr(sketch.codes), _ptr(sketch.exps), sketch.cap,
                                sketch.bits, int(token_begin), t1, _stream_ptr(stream)))
    return sketch


def hill_score(q, k, s, *, mode="attn", granularity="token", n_tokens=None, sm_scale=0.0, ws=None,
               stream=None, sketch: Optional[Sketch] = None):
    """S += column-wise sum over this step's weights (in place).  With
    ``sketch`` the scores come from the int8 sketch (k may then be None)."""
    lib = load_library()
    _device_check(q, k, s)
    if sketch is not None and k is None:
        B, Hkv, cap, D = sketch.codes.shape
        desc = make_desc(q, None, None, s, mode=mode, granularity=granularity,
                         n_tokens=s.shape[-1] if n_tokens is None else n_tokens, sm_scale=sm_scale,
                         shape=(B, q.shape[1], Hkv, D))
    else:
        desc = make_desc(q, k, None, s, mode=mode, granularity=granularity, n_tokens=n_tokens, sm_scale=sm_scale)
    if ws is None:
        ws = workspace(desc, 1, q.device)
    if sketch is None:
        _check(lib.hill_score(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(s), _ptr(ws), ws.numel(),
                              _stream_ptr(stream)))
    else:
        _check(lib.hill_score_sketch(ctypes.byref(desc), _ptr(q), _ptr(sketch.codes), _ptr(sketch.exps),
                                     sketch.cap, sketch.bits, _ptr(s), _ptr(ws), ws.numel(), _stream_ptr(stream)))
    return s


def hill_topk(s, k_sel, *, granularity="token", n_tokens=None, n_kv_heads=None, with_values=False,
              idx_out=None, val_out=None, ws=None, stream=None, n_sink=0, n_recent=0):
    """Indices [B, R, k_sel] (int32, ascending) of the k_sel largest S per row
    (the first n_sink and last n_recent tokens always among them)."""
    lib = load_library()
    _device_check(s)
    B, R, _ = s.shape
    hkv = n_kv_heads if n_kv_heads is not None else R
    desc = make_desc(None, None, None, s, granularity=granularity, n_tokens=n_tokens,
                     shape=(B, hkv, hkv, 128), dtype=torch.float16, n_sink=n_sink, n_recent=n_recent)
    if idx_out is None:
        idx_out = torch.empty((B, R, k_sel), dtype=torch.int32, device=s.device)
    if with_values and val_out is None:
        val_out = torch.empty((B, R, k_sel), dtype=torch.float32, device=s.device)
    if ws is None:
        ws = workspace(desc, k_sel, s.device)
    _check(lib.hill_topk(ctypes.byref(desc), _ptr(s), int(k_sel), _ptr(idx_out), _ptr(val_out), _ptr(ws),
                         ws.numel(), _stream_ptr(stream)))
    return (idx_out, val_out) if with_values else idx_out


def hill_gather_attn(q, k, v, idx, *, granularity="token", n_tokens=None, sm_scale=0.0, out=None, ws=None,
                     stream=None):
    """Attention over the selected tokens; out [B, Hq, D] fp32."""
    lib = load_library()
    _device_check(q, k, v, idx)
    k_sel = idx.shape[-1]
    desc = make_desc(q, k, v, None, granularity=granularity, n_tokens=n_tokens, sm_scale=sm_scale)
    if not idx.is_contiguous() or idx.dtype != torch.int32:
        raise ValueError("idx must be a contiguous int32 tensor")
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = workspace(desc, k_sel, q.device)
    _check(lib.hill_gather_attn(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(idx), int(k_sel),
                                _ptr(out), _ptr(ws), ws.numel(), _stream_ptr(stream)))
    return out


HILL_STREAM_RESET = 1   # include/hill.h: select through the refine pass and write a fresh bound


def new_stream_state(B: int, R: int, device) -> torch.Tensor:
    """Zeroed state of the streamed selection for one S buffer ([B, R] rows)."""
    return torch.zeros((B, R, 8), dtype=torch.int32, device=device)


def hill_step(q, k, v, s, k_sel=None, *, budget=None, mode="attn", granularity="token", n_tokens=None,
              sm_scale=0.0, idx_out=None, out=None, ws=None, stream=None, events=None,
              sketch: Optional[Sketch] = None, n_sink=0, n_recent=0, stream_state=None, stream_reset=False):
    """One decode step: S update, top-k on the new S, attention.  Returns (idx, out).
    ``n_sink`` / ``n_recent``: pinned tokens every selection keeps.
    ``stream_state``: streamed selection (hill_step_streamed) with this state
    (from new_stream_state, kept with S across steps); ``stream_reset``: this
    step selects through the refine pass and writes a fresh bound
    (HILL_STREAM_RESET: the first steps of a sequence).

    ``events``: optional HillStepEvents; then hill_step_profiled records them.
    ``sketch``: score on the int8 / int4 sketch (hill_step_sketch)."""
    lib = load_library()
    _device_check(q, k, v, s, ws)
    if sketch is not None:
        _device_check(sketch.codes, sketch.exps)
    desc = make_desc(q, k, v, s, mode=mode, granularity=granularity, n_tokens=n_tokens, sm_scale=sm_scale,
                     n_sink=n_sink, n_recent=n_recent)
    if k_sel is None:
        if budget is None:
            raise ValueError("give k_sel or budget")
        k_sel = budget_k(desc.n_tokens, budget)
    B, R = s.shape[0], s.shape[1]
    if idx_out is None:
        idx_out = torch.empty((B, R, k_sel), dtype=torch.int32, device=s.device)
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = workspace(desc, k_sel, q.device)
    if stream_state is not None:
        _device_check(stream_state)
        if stream_state.dtype != torch.int32 or stream_state.numel() < B * R * 8 or not stream_state.is_contiguous():
            raise ValueError("stream_state must be a contiguous int32 [B, R, 8] tensor")
    elif stream_reset:
        raise ValueError("stream_reset needs a stream_state")
    flags = HILL_STREAM_RESET if stream_reset else 0
    if sketch is not None:
        _check(lib.hill_step_sketch(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(sketch.codes),
                                    _ptr(sketch.exps), sketch.cap, sketch.bits, _ptr(s), _ptr(stream_state), flags,
                                    int(k_sel), _ptr(idx_out), _ptr(out), _ptr(ws), ws.numel(), _stream_ptr(stream),
                                    None if events is None else ctypes.byref(events)))
    elif stream_state is not None:
        _check(lib.hill_step_streamed(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(s), _ptr(stream_state),
                                      flags, int(k_sel), _ptr(idx_out), _ptr(out), _ptr(ws), ws.numel(),
                                      _stream_ptr(stream), None if events is None else ctypes.byref(events)))
    elif events is None:
        _check(lib.hill_step(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(s), int(k_sel), _ptr(idx_out),
                             _ptr(out), _ptr(ws), ws.numel(), _stream_ptr(stream)))
    else:
        _check(lib.hill_step_profiled(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(s), int(k_sel),
                                      _ptr(idx_out), _ptr(out), _ptr(ws), ws.numel(), _stream_ptr(stream),
                                      ctypes.byref(events)))
    return idx_out, out


NOALLOC_SCRATCH_BYTES = 32 << 20   # HILL_NOALLOC_SCRATCH_BYTES of include/hill.h


def hill_step_noalloc(q, k, v, s, k_sel, *, mode="attn", granularity="token", n_tokens=None, sm_scale=0.0,
                      idx_out=None, out=None, stream=None, n_sink=0, n_recent=0):
    """hill_step with the library's fixed device scratch instead of a
    workspace (hill_step_noalloc, for callers that cannot allocate; steps up
    to NOALLOC_SCRATCH_BYTES of workspace).  Returns (idx, out)."""
    lib = load_library()
    _device_check(q, k, v, s, idx_out, out)
    desc = make_desc(q, k, v, s, mode=mode, granularity=granularity, n_tokens=n_tokens, sm_scale=sm_scale,
                     n_sink=n_sink, n_recent=n_recent)
    B, R = s.shape[0], s.shape[1]
    if idx_out is None:
        idx_out = torch.empty((B, R, k_sel), dtype=torch.int32, device=s.device)
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check(lib.hill_step_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(s), int(k_sel), _ptr(idx_out),
                                 _ptr(out), _stream_ptr(stream)))
    return idx_out, out


def new_importance(B: int, R: int, n_cap: int, device) -> torch.Tensor:
    """Zeroed fp32 importance buffer [B, R, n_cap] whose row stride is a multiple of 4."""
    pad = (n_cap + 3) // 4 * 4
    return torch.zeros((B, R, pad), dtype=torch.float32, device=device)[:, :, :n_cap]


class BkpState:
    """Per-token state of the Bidirectional KV Cache Pools for [B, R, n_cap]
    tokens: the 2-byte hit table (held as int16, read as uint16 bit
    patterns) and one pool byte per token (1 = hot)."""

    def __init__(self, B: int, R: int, n_cap: int, device):
        self.hits = torch.zeros((B, R, n_cap), dtype=torch.int16, device=device)
        self.hot = torch.zeros((B, R, n_cap), dtype=torch.uint8, device=device)


def bkp_desc(state: BkpState, n_tokens: int, n_recent: int, capacity: int) -> BkpDesc:
    B, R, n_cap = state.hits.shape
    if state.hits.stride() != state.hot.stride() or state.hits.stride(2) != 1:
        raise ValueError("hits and hot need the same strides with tokens contiguous")
    return BkpDesc(ctypes.sizeof(BkpDesc), B, R, int(n_tokens), int(n_recent), int(capacity),
                   state.hits.stride(0), state.hits.stride(1))


def bkp_update(state: BkpState, idx, *, n_tokens: int, n_recent: int, capacity: int, list_cap=None, ws=None,
               stream=None):
    """One BKP pass after a decoding step (Sec. 4.2): hits of the selected
    tokens ``idx`` ([B, R, k] int32, or None) go up by one, the pool is
    rebuilt from the recent window and the most-hit tokens; returns
    (promote, demote, counts) device tensors ([B, R, list_cap] int32 each,
    only the first counts[..., 0] / counts[..., 1] entries meaningful)."""
    lib = load_library()
    _device_check(state.hits, state.hot)
    B, R, _ = state.hits.shape
    d = bkp_desc(state, n_tokens, n_recent, capacity)
    if list_cap is None:
        list_cap = min(int(capacity), int(n_tokens))
    dev = state.hits.device
    if ws is None:
        need = ctypes.c_size_t(0)
        _check(lib.hill_bkp_workspace_bytes(ctypes.byref(d), ctypes.byref(need)))
        ws = torch.empty(max(int(need.value), 256), dtype=torch.uint8, device=dev)
    k = 0 if idx is None else int(idx.shape[-1])
    if idx is not None:
        _device_check(idx)
        if idx.dtype != torch.int32 or tuple(idx.shape) != (B, R, k) or not idx.is_contiguous():
            raise ValueError("idx must be a contiguous int32 [B, R, k] tensor")
    promote = torch.empty((B, R, max(list_cap, 1)), dtype=torch.int32, device=dev)
    demote = torch.empty_like(promote)
    counts = torch.empty((B, R, 2), dtype=torch.int32, device=dev)
    _check(lib.hill_bkp_update(ctypes.byref(d), _ptr(idx) if idx is not None else None, k, _ptr(state.hits),
                               _ptr(state.hot), _ptr(promote), _ptr(demote), int(list_cap), _ptr(counts), _ptr(ws),
                               ws.numel(), _stream_ptr(stream)))
    return promote[..., :list_cap], demote[..., :list_cap], counts


class BkpCall:
    """hill_bkp_update with its buffers allocated and arguments marshalled
    once, for per-step loops (only the index pointer changes per call)."""

    def __init__(self, state: BkpState, k_sel: int, *, n_tokens: int, n_recent: int, capacity: int,
                 list_cap=None, stream=None):
        lib = load_library()
        _device_check(state.hits, state.hot)
        B, R, _ = state.hits.shape
        self.desc = bkp_desc(state, n_tokens, n_recent, capacity)
        self.list_cap = min(int(capacity), int(n_tokens)) if list_cap is None else int(list_cap)
        dev = state.hits.device
        need = ctypes.c_size_t(0)
        _check(lib.hill_bkp_workspace_bytes(ctypes.byref(self.desc), ctypes.byref(need)))
        self.ws = torch.empty(max(int(need.value), 256), dtype=torch.uint8, device=dev)
        self.promote = torch.empty((B, R, max(self.list_cap, 1)), dtype=torch.int32, device=dev)
        self.demote = torch.empty_like(self.promote)
        self.counts = torch.empty((B, R, 2), dtype=torch.int32, device=dev)
        P = ctypes.c_void_p
        self._fn = lib.hill_bkp_update
        self._k = ctypes.c_int32(int(k_sel))
        self._post = (P(state.hits.data_ptr()), P(state.hot.data_ptr()), P(self.promote.data_ptr()),
                      P(self.demote.data_ptr()), ctypes.c_int32(self.list_cap), P(self.counts.data_ptr()),
                      P(self.ws.data_ptr()), ctypes.c_size_t(self.ws.numel()), P(_stream_ptr(stream)))
        self._keep = state

    def __call__(self, idx_ptr: int):
        _check(self._fn(ctypes.byref(self.desc), ctypes.c_void_p(idx_ptr), self._k, *self._post))


class TieredCache:
    """One layer's K/V split between a hot pool in HBM (``capacity`` slot rows
    per row (b, r)) and a cold pool in pinned host memory that the GPU reads
    and writes in place (rows by token position), each token's rows in
    exactly one of them, plus the key sketch of every token in HBM that the
    step scores on (include/hill.h, tiered KV cache).  Starts with every row
    in the cold pool (loc = -1).  ``granularity``: "token" (all KV heads of a
    token share a slot) or "kvhead"."""

    def __init__(self, k, v, capacity: int, *, granularity="token", bits=8, n_cap=None, stream=None):
        _device_check(k, v)
        B, Hkv, n, D = k.shape
        self.granularity = granularity
        self.R = 1 if granularity == "token" else Hkv
        self.capacity = int(capacity)
        self.n_cap = ((n if n_cap is None else int(n_cap)) + 3) // 4 * 4
        dev = k.device
        self.k_cold = torch.empty((B, Hkv, self.n_cap, D), dtype=k.dtype, pin_memory=True)
        self.v_cold = torch.empty((B, Hkv, self.n_cap, D), dtype=v.dtype, pin_memory=True)
        if not (self.k_cold.is_pinned() and self.v_cold.is_pinned()):
            raise RuntimeError("the cold pool could not be allocated as pinned host memory")
        self.k_cold[:, :, :n].copy_(k)
        self.v_cold[:, :, :n].copy_(v)
        self.k_hot = torch.zeros((B, Hkv, self.capacity, D), dtype=k.dtype, device=dev)
        self.v_hot = torch.zeros((B, Hkv, self.capacity, D), dtype=v.dtype, device=dev)
        self.loc = torch.full((B, self.R, self.n_cap), -1, dtype=torch.int32, device=dev)
        self.sketch = sketch_keys(k, bits=bits, stream=stream)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.n_prev = 0   # context of the last migration (the pool holds min(capacity, n_prev) rows)
        self.desc = TierDesc(ctypes.sizeof(TierDesc), self.capacity, self.n_cap, 0, self.k_hot.stride(0),
                             self.k_hot.stride(1), self.k_hot.stride(2))

    def step_desc(self, q, s, n_tokens, **kw) -> HillDesc:
        return make_desc(q, self.k_cold, self.v_cold, s, granularity=self.granularity, n_tokens=n_tokens, **kw)


def hill_tier_apply(cache: TieredCache, promote, demote, counts, *, n_tokens: int, stream=None):
    """Moves the rows that a BKP pass over ``n_tokens`` tokens decided
    (hill_bkp_update's promote / demote / counts) between the pools and
    updates the slot table; records n_tokens as the pool's context."""
    lib = load_library()
    _device_check(promote, demote, counts)
    q0 = torch.empty((cache.k_hot.shape[0], cache.k_hot.shape[1], cache.k_hot.shape[3]), dtype=cache.k_hot.dtype,
                     device="meta")
    desc = make_desc(q0, cache.k_cold, cache.v_cold, None, granularity=cache.granularity, n_tokens=n_tokens)
    if not (promote.is_contiguous() and demote.is_contiguous() and counts.is_contiguous()):
        raise ValueError("promote, demote and counts must be contiguous")
    _check(lib.hill_tier_apply(ctypes.byref(desc), ctypes.byref(cache.desc), _ptr(cache.k_hot), _ptr(cache.v_hot),
                               _ptr(cache.k_cold), _ptr(cache.v_cold), _ptr(cache.loc), _ptr(promote), _ptr(demote),
                               int(promote.shape[-1]), _ptr(counts), int(cache.n_prev), _ptr(cache.status),
                               _stream_ptr(stream)))
    cache.n_prev = int(n_tokens)


def hill_step_tiered(q, cache: TieredCache, s, k_sel, *, n_tokens=None, mode="attn", sm_scale=0.0, idx_out=None,
                     out=None, ws=None, stream=None, events=None, stream_state=None, stream_reset=False):
    """hill_step_sketch over a tiered cache (scores on the cache's sketch, K
    and V of the selected tokens from whichever pool holds them).  Returns
    (idx, out)."""
    lib = load_library()
    _device_check(q, s, ws, stream_state)
    n = cache.n_cap if n_tokens is None else int(n_tokens)
    desc = cache.step_desc(q, s, n, mode=mode, sm_scale=sm_scale)
    B, R = s.shape[0], s.shape[1]
    if idx_out is None:
        idx_out = torch.empty((B, R, k_sel), dtype=torch.int32, device=s.device)
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = workspace(desc, k_sel, q.device)
    if stream_state is not None and (stream_state.dtype != torch.int32 or not stream_state.is_contiguous()):
        raise ValueError("stream_state must be a contiguous int32 [B, R, 8] tensor")
    flags = HILL_STREAM_RESET if stream_reset else 0
    sk = cache.sketch
    _check(lib.hill_step_tiered(ctypes.byref(desc), ctypes.byref(cache.desc), _ptr(q), _ptr(cache.k_hot),
                                _ptr(cache.v_hot), _ptr(cache.k_cold), _ptr(cache.v_cold), _ptr(cache.loc),
                                _ptr(sk.codes), _ptr(sk.exps), sk.cap, sk.bits, _ptr(s), _ptr(stream_state), flags,
                                int(k_sel), _ptr(idx_out), _ptr(out), _ptr(ws), ws.numel(), _stream_ptr(stream),
                                None if events is None else ctypes.byref(events)))
    return idx_out, out


class TierStepCall:
    """hill_step_tiered with its arguments marshalled once, for per-step loops
    (only the query pointer changes); the first ``stream_reset_calls`` calls
    are reset steps of the streamed selection when a state is given."""

    def __init__(self, q, cache: TieredCache, s, k_sel, *, n_tokens=None, ws=None, stream=None, stream_state=None,
                 stream_reset_calls=3):
        lib = load_library()
        _device_check(q, s, ws, stream_state)
        n = cache.n_cap if n_tokens is None else int(n_tokens)
        self.desc = cache.step_desc(q, s, n)
        B, R = s.shape[0], s.shape[1]
        self.k_sel = int(k_sel)
        self.idx = torch.empty((B, R, self.k_sel), dtype=torch.int32, device=s.device)
        self.out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        self.ws = ws if ws is not None else workspace(self.desc, self.k_sel, q.device)
        P = ctypes.c_void_p
        sk = cache.sketch
        self._fn = lib.hill_step_tiered
        self._resets_left = int(stream_reset_calls) if stream_state is not None else 0

        def args(flags):
            return (ctypes.byref(self.desc), ctypes.byref(cache.desc)), \
                   (P(cache.k_hot.data_ptr()), P(cache.v_hot.data_ptr()), P(cache.k_cold.data_ptr()),
                    P(cache.v_cold.data_ptr()), P(cache.loc.data_ptr()), P(sk.codes.data_ptr()),
                    P(sk.exps.data_ptr()), ctypes.c_int64(sk.cap), ctypes.c_int32(sk.bits), P(s.data_ptr()),
                    P(stream_state.data_ptr() if stream_state is not None else None), ctypes.c_uint32(flags),
                    ctypes.c_int32(self.k_sel), P(self.idx.data_ptr()), P(self.out.data_ptr()),
                    P(self.ws.data_ptr()), ctypes.c_size_t(self.ws.numel()), P(_stream_ptr(stream)))
        self._pre, self._post = args(0)
        self._post_reset = args(HILL_STREAM_RESET)[1]
        self._keep = (cache, s, stream_state)

    def __call__(self, q_ptr: int, events=None):
        post = self._post
        if self._resets_left > 0:
            self._resets_left -= 1
            post = self._post_reset
        st = self._fn(*self._pre, ctypes.c_void_p(q_ptr), *post, None if events is None else ctypes.byref(events))
        if st != HILL_OK:
            _check(st)


class TierApplyCall:
    """hill_tier_apply marshalled once for a cache and a BkpCall's lists (the
    context stays n_tokens from the second call on)."""

    def __init__(self, cache: TieredCache, bkp: "BkpCall", *, n_tokens: int, stream=None):
        lib = load_library()
        q0 = torch.empty((cache.k_hot.shape[0], cache.k_hot.shape[1], cache.k_hot.shape[3]), dtype=cache.k_hot.dtype,
                         device="meta")
        self.desc = make_desc(q0, cache.k_cold, cache.v_cold, None, granularity=cache.granularity, n_tokens=n_tokens)
        P = ctypes.c_void_p
        self._fn = lib.hill_tier_apply
        self._cache, self._n = cache, int(n_tokens)
        self._args = (ctypes.byref(self.desc), ctypes.byref(cache.desc), P(cache.k_hot.data_ptr()),
                      P(cache.v_hot.data_ptr()), P(cache.k_cold.data_ptr()), P(cache.v_cold.data_ptr()),
                      P(cache.loc.data_ptr()), P(bkp.promote.data_ptr()), P(bkp.demote.data_ptr()),
                      ctypes.c_int32(bkp.promote.shape[-1]), P(bkp.counts.data_ptr()))
        self._post = (P(cache.status.data_ptr()), P(_stream_ptr(stream)))
        self._keep = bkp

    def __call__(self):
        _check(self._fn(*self._args, ctypes.c_int32(self._cache.n_prev), *self._post))
        self._cache.n_prev = self._n


def app_balance(*, f_c, f_s, b_c, b_s, alpha=None, alpha_c=None, alpha_s=None, m=1.0, m0=0.0) -> dict:
    """Capacity split of the Adaptive Prefetch-based Pipeline (Sec. 4.3, Eqs.
    2-4), computed by the library (host only).  ``alpha`` sets both retained
    fractions; ``alpha_c`` / ``alpha_s`` give skew-corrected ones."""
    lib = load_library()
    ac = alpha if alpha_c is None else alpha_c
    as_ = alpha if alpha_s is None else alpha_s
    if ac is None or as_ is None:
        raise ValueError("give alpha, or alpha_c and alpha_s")
    p = AppParams(f_c, f_s, b_c, b_s, ac, as_, m, m0)
    out = AppPlan()
    _check(lib.hill_app_balance(ctypes.byref(p), ctypes.byref(out)))
    return {f[0]: getattr(out, f[0]) for f in AppPlan._fields_}


class StepCall:
    """hill_step with its arguments marshalled once, for hot loops that call it
    repeatedly on the same buffers (only the query pointer changes per call).
    With ``stream_state``, the first ``stream_reset_calls`` calls are reset
    steps (HILL_STREAM_RESET), the later ones streamed."""

    def __init__(self, q, k, v, s, k_sel, *, mode="attn", granularity="token", n_tokens=None, sm_scale=0.0,
                 ws=None, stream=None, sketch: Optional[Sketch] = None, n_sink=0, n_recent=0, stream_state=None,
                 stream_reset_calls=3):
        lib = load_library()
        _device_check(q, k, v, s, ws, stream_state)
        if sketch is not None:
            _device_check(sketch.codes, sketch.exps)
            if not (sketch.codes.is_contiguous() and sketch.exps.is_contiguous()):
                raise ValueError("sketch codes and exponents must be contiguous")
        self.desc = make_desc(q, k, v, s, mode=mode, granularity=granularity, n_tokens=n_tokens,
                              sm_scale=sm_scale, n_sink=n_sink, n_recent=n_recent)
        B, R = s.shape[0], s.shape[1]
        self.k_sel = int(k_sel)
        self.idx = torch.empty((B, R, self.k_sel), dtype=torch.int32, device=s.device)
        self.out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        self.ws = ws if ws is not None else workspace(self.desc, self.k_sel, q.device)
        P = ctypes.c_void_p
        self._pre = (ctypes.byref(self.desc),)
        if stream_state is not None and (stream_state.dtype != torch.int32 or stream_state.numel() < B * R * 8
                                         or not stream_state.is_contiguous()):
            raise ValueError("stream_state must be a contiguous int32 [B, R, 8] tensor")
        state_ptr = P(stream_state.data_ptr() if stream_state is not None else None)
        self._resets_left = int(stream_reset_calls) if stream_state is not None else 0
        self._post_reset = None
        if sketch is not None:
            self._fn = None
            self._fn_ev = lib.hill_step_sketch   # events and state may be NULL

            def post(flags):
                return (P(k.data_ptr()), P(v.data_ptr()), P(sketch.codes.data_ptr()), P(sketch.exps.data_ptr()),
                        ctypes.c_int64(sketch.cap), ctypes.c_int32(sketch.bits), P(s.data_ptr()), state_ptr,
                        ctypes.c_uint32(flags), ctypes.c_int32(self.k_sel), P(self.idx.data_ptr()),
                        P(self.out.data_ptr()), P(self.ws.data_ptr()), ctypes.c_size_t(self.ws.numel()),
                        P(_stream_ptr(stream)))
            self._post = post(0)
            if stream_state is not None:
                self._post_reset = post(HILL_STREAM_RESET)
        elif stream_state is not None:
            self._fn = None
            self._fn_ev = lib.hill_step_streamed   # events may be NULL

            def post(flags):
                return (P(k.data_ptr()), P(v.data_ptr()), P(s.data_ptr()), state_ptr, ctypes.c_uint32(flags),
                        ctypes.c_int32(self.k_sel), P(self.idx.data_ptr()), P(self.out.data_ptr()),
                        P(self.ws.data_ptr()), ctypes.c_size_t(self.ws.numel()), P(_stream_ptr(stream)))
            self._post = post(0)
            self._post_reset = post(HILL_STREAM_RESET)
        else:
            self._fn = lib.hill_step
            self._fn_ev = lib.hill_step_profiled
            self._post = (P(k.data_ptr()), P(v.data_ptr()), P(s.data_ptr()), ctypes.c_int32(self.k_sel),
                          P(self.idx.data_ptr()), P(self.out.data_ptr()), P(self.ws.data_ptr()),
                          ctypes.c_size_t(self.ws.numel()), P(_stream_ptr(stream)))
        self._keep = (k, v, s, sketch, stream_state)

    def __call__(self, q_ptr: int, events=None):
        if self._fn is None:
            post = self._post
            if self._resets_left > 0:
                self._resets_left -= 1
                post = self._post_reset
            st = self._fn_ev(*self._pre, ctypes.c_void_p(q_ptr), *post,
                             None if events is None else ctypes.byref(events))
        elif events is None:
            st = self._fn(*self._pre, ctypes.c_void_p(q_ptr), *self._post)
        else:
            st = self._fn_ev(*self._pre, ctypes.c_void_p(q_ptr), *self._post, ctypes.byref(events))
        if st != HILL_OK:
            _check(st)
