"""CPU oracle for HillInfer's per-decode-step token-importance path.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this module.  It shares no
code with the GPU library (``paper_2602_18750_amd``) and never imports it.

This is a thin ctypes/numpy wrapper around ``hill_oracle.c`` (plain C, fp64
accumulation over exactly widened fp16/bf16 inputs).  Every function follows
one definition of the paper (arxiv 2602.18750):

* :func:`logits`      -- the raw inner product q.K^T (Sec. 4.4 "Algorithmic
                         Simplification"; Sec. 2.1 Eq. 1 for the product).
* :func:`update`      -- per-step attention weights softmax(q.K^T / sqrt(d))
                         (Eq. 1) or raw logits (Sec. 4.4), summed column-wise
                         into the cumulative importance S (Sec. 4.1).
* :func:`topk`        -- the top-alpha selection (Sec. 3.1, Sec. 4.2 HIE),
                         brute force by full sort, ties to the lower index;
                         :func:`topk_pinned` keeps sink and recent tokens.
* :func:`sparse_attn` -- Eq. 1 restricted to the selected tokens (Sec. 4.1,
                         workflow step 6).
* :func:`step`        -- the three in the workflow's order.
* :func:`sketch`, :func:`logits_i8` -- the int8 key/query casts and the
                         integer logits of asymmetric-precision scoring
                         (Sec. 4.4).
* :func:`bkp_update`  -- the hit-rate table and the hot/cold pool policy of
                         the Bidirectional KV Cache Pools (Sec. 4.2 HKM,
                         BKP (1)-(3)), plain numpy on integers.
* :func:`tier_apply`  -- the migration of rows between the hot and the cold
                         pool that a BKP pass decides (Sec. 4.2 BKP (3)).
* :func:`app_split`   -- the Adaptive Prefetch-based Pipeline's capacity
                         split (Sec. 4.3): Eq. 2's balance solved by
                         bisection, with the host-memory bound Eq. 3.

16-bit inputs are passed as ``numpy.uint16`` bit patterns; the oracle decodes
them itself (:func:`decode16`).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hill_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libhill_oracle.so")
# the same source built with AddressSanitizer and UBSan (clang), for CPU test
# runs that preload the sanitizer runtime; selected by HILL_ORACLE_LIB
SAN_LIB_PATH = os.path.join(_HERE, "libhill_oracle_san.so")
CLANG = os.environ.get("HILL_CLANG", "/opt/rocm/llvm/bin/clang")

F16, BF16 = 0, 1
ATTN, RAW = 0, 1
TOKEN, KVHEAD = 0, 1

_DTYPES = {"fp16": F16, "f16": F16, "float16": F16, "bf16": BF16, "bfloat16": BF16}
_MODES = {"attn": ATTN, "raw": RAW}
_GRANS = {"token": TOKEN, "kvhead": KVHEAD}

_lock = threading.Lock()
_lib = None


def build(force: bool = False, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math); with
    ``sanitize``, the sanitizer variant instead: clang, -O1, AddressSanitizer
    and UBSan with no recovery (any finding aborts), single-threaded."""
    out = SAN_LIB_PATH if sanitize else _LIB_PATH
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        tmp = out + ".tmp%d" % os.getpid()
        if sanitize:
            cmd = [CLANG, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                   "-fno-sanitize-recover=all", "-Wno-unknown-pragmas", "-fPIC", "-shared", "-std=c11",
                   "-D_POSIX_C_SOURCE=200809L", "-o", tmp, _SRC, "-lm"]
        else:
            cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                   "-D_POSIX_C_SOURCE=200809L", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        path = os.environ.get("HILL_ORACLE_LIB")
        if path is None:
            path = build()
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        I = ctypes.c_int
        I64 = ctypes.c_int64
        Dd = ctypes.c_double
        lib.hor_decode16.argtypes = [P, I64, I, P]
        lib.hor_decode16.restype = None
        lib.hor_num_threads.argtypes = []
        lib.hor_num_threads.restype = I
        lib.hor_logits.argtypes = [I, I, I, I, I, I, P, P, P]
        lib.hor_logits.restype = I
        lib.hor_update.argtypes = [I, I, I, I, I, I, Dd, P, P]
        lib.hor_update.restype = I
        lib.hor_topk.argtypes = [I64, I, I, P, P]
        lib.hor_topk.restype = I
        lib.hor_sparse_attn.argtypes = [I, I, I, I, I, I, I, Dd, P, P, P, I, P, P]
        lib.hor_sparse_attn.restype = I
        lib.hor_step.argtypes = [I, I, I, I, I, I, I, I, Dd, P, P, P, P, P, I, P, P, P]
        lib.hor_step.restype = I
        lib.hor_sketch.argtypes = [I64, I, I, I, P, P, P]
        lib.hor_sketch.restype = I
        lib.hor_logits_i8.argtypes = [I, I, I, I, I, P, P, P, P, P]
        lib.hor_logits_i8.restype = I
        _lib = lib
        return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("16-bit inputs must be passed as uint16 bit patterns")
    return a


def _code(table, key):
    if isinstance(key, int):
        return key
    return table[key.lower()]


def num_threads() -> int:
    return int(_load().hor_num_threads())


def default_scale(D: int) -> float:
    """1/sqrt(d), the scale of Eq. 1."""
    return 1.0 / float(np.sqrt(D))


def decode16(bits, dtype) -> np.ndarray:
    """Widen fp16/bf16 bit patterns to float64 exactly."""
    lib = _load()
    bits = _u16(bits)
    out = np.empty(bits.shape, dtype=np.float64)
    lib.hor_decode16(_ptr(bits), bits.size, _code(_DTYPES, dtype), _ptr(out))
    return out


def logits(q, k, dtype) -> np.ndarray:
    """l[b,h,j] = q[b,h,:] . K[b,h//G,j,:] in float64.  q [B,Hq,D], K [B,Hkv,n,D]."""
    lib = _load()
    q, k = _u16(q), _u16(k)
    B, Hq, D = q.shape
    Bk, Hkv, n, Dk = k.shape
    assert Bk == B and Dk == D
    out = np.empty((B, Hq, n), dtype=np.float64)
    rc = lib.hor_logits(B, Hq, Hkv, D, n, _code(_DTYPES, dtype), _ptr(q), _ptr(k), _ptr(out))
    if rc:
        raise ValueError("hor_logits failed (%d)" % rc)
    return out


def sketch(x, dtype, bits: int = 8):
    """Scoring sketch of the last axis of x (16-bit patterns, D = last
    dimension): (codes int8 of x's shape, exponents int8 of x.shape[:-1]);
    codes in [-127, 127] (bits 8) or [-7, 7] (bits 4).  Sec. 4.4 asymmetric
    precision, with the power-of-two per-row scale reading."""
    lib = _load()
    x = _u16(x)
    D = x.shape[-1]
    rows = x.size // D
    qmax = {8: 127, 4: 7}[bits]
    codes = np.empty(x.shape, dtype=np.int8)
    exps = np.empty(x.shape[:-1], dtype=np.int8)
    rc = lib.hor_sketch(rows, D, _code(_DTYPES, dtype), qmax, _ptr(x), _ptr(codes), _ptr(exps))
    if rc:
        raise ValueError("hor_sketch failed (%d)" % rc)
    return codes, exps


def logits_i8(q8, eq, k8, ek) -> np.ndarray:
    """Sketch logits: exact integer q8.k8 scaled by 2^(eq + ek), float64 (k8:
    int8 or int4 key codes, held one per int8).
    q8 [B,Hq,D], eq [B,Hq], k8 [B,Hkv,n,D], ek [B,Hkv,n]."""
    lib = _load()
    q8, k8 = np.ascontiguousarray(q8, dtype=np.int8), np.ascontiguousarray(k8, dtype=np.int8)
    eq, ek = np.ascontiguousarray(eq, dtype=np.int8), np.ascontiguousarray(ek, dtype=np.int8)
    B, Hq, D = q8.shape
    Bk, Hkv, n, Dk = k8.shape
    assert Bk == B and Dk == D and eq.shape == (B, Hq) and ek.shape == (B, Hkv, n)
    out = np.empty((B, Hq, n), dtype=np.float64)
    rc = lib.hor_logits_i8(B, Hq, Hkv, D, n, _ptr(q8), _ptr(eq), _ptr(k8), _ptr(ek), _ptr(out))
    if rc:
        raise ValueError("hor_logits_i8 failed (%d)" % rc)
    return out


def update(l, S, n_kv_heads: int, mode="attn", granularity="token", scale=None) -> np.ndarray:
    """Return S + column-wise sum of this step's weights (a new array)."""
    lib = _load()
    l = np.ascontiguousarray(l, dtype=np.float64)
    B, Hq, n = l.shape
    S = np.array(S, dtype=np.float64, copy=True, order="C")
    gran = _code(_GRANS, granularity)
    R = 1 if gran == TOKEN else n_kv_heads
    assert S.shape == (B, R, n), (S.shape, (B, R, n))
    if scale is None:
        raise ValueError("scale is required (1/sqrt(D) for Eq. 1)")
    rc = lib.hor_update(B, Hq, n_kv_heads, n, _code(_MODES, mode), gran, float(scale), _ptr(l), _ptr(S))
    if rc:
        raise ValueError("hor_update failed (%d)" % rc)
    return S


def topk(S, k: int) -> np.ndarray:
    """k largest per row of S [..., n]; ties to the lower index; ascending."""
    lib = _load()
    S = np.ascontiguousarray(S, dtype=np.float64)
    n = S.shape[-1]
    rows = int(np.prod(S.shape[:-1])) if S.ndim > 1 else 1
    out = np.empty(S.shape[:-1] + (k,), dtype=np.int32)
    rc = lib.hor_topk(rows, n, int(k), _ptr(S), _ptr(out))
    if rc:
        raise ValueError("hor_topk failed (%d)" % rc)
    return out


def topk_pinned(S, k: int, n_sink: int = 0, n_recent: int = 0) -> np.ndarray:
    """Selection that always keeps pinned tokens: the first min(n_sink, n) and
    the last min(n_recent, n) of each row (attention sinks and the recent
    window that Sec. 4.2's locality and hit-rate observations single out);
    the other k - |pinned| slots take the largest S among the tokens between
    the two windows (plain top-k there, ties to the lower index).  Returns
    ascending indices [..., k]."""
    S = np.asarray(S, dtype=np.float64)
    n = S.shape[-1]
    lo = min(int(n_sink), n)
    hi = max(lo, n - min(int(n_recent), n))
    pinned = np.concatenate([np.arange(lo), np.arange(hi, n)]).astype(np.int64)
    free = int(k) - len(pinned)
    if free < 0:
        raise ValueError("k smaller than the pinned tokens")
    rows = S.reshape(-1, n)
    out = np.empty((rows.shape[0], int(k)), dtype=np.int32)
    for i, row in enumerate(rows):
        pick = topk(row[lo:hi][None], free)[0].astype(np.int64) + lo if free else np.empty(0, np.int64)
        out[i] = np.sort(np.concatenate([pinned, pick]))
    return out.reshape(S.shape[:-1] + (int(k),))


def sparse_attn(q, k, v, idx, dtype, granularity="token", scale=None) -> np.ndarray:
    """Eq. 1 over the selected tokens; out [B,Hq,D] float64."""
    lib = _load()
    q, k, v = _u16(q), _u16(k), _u16(v)
    B, Hq, D = q.shape
    _, Hkv, n, _ = k.shape
    assert v.shape == k.shape
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    kk = idx.shape[-1]
    gran = _code(_GRANS, granularity)
    R = 1 if gran == TOKEN else Hkv
    assert idx.shape == (B, R, kk), (idx.shape, (B, R, kk))
    if scale is None:
        scale = default_scale(D)
    out = np.empty((B, Hq, D), dtype=np.float64)
    rc = lib.hor_sparse_attn(B, Hq, Hkv, D, n, _code(_DTYPES, dtype), gran, float(scale),
                             _ptr(q), _ptr(k), _ptr(v), kk, _ptr(idx), _ptr(out))
    if rc:
        raise ValueError("hor_sparse_attn failed (%d)" % rc)
    return out


def step(q, k, v, S, k_sel: int, dtype, mode="attn", granularity="token", scale=None,
         return_times: bool = False):
    """One decode step: update S with q, select k on the new S, attend.

    Returns (S_new, idx, out[, (t_score, t_select, t_attn)])."""
    lib = _load()
    q, k, v = _u16(q), _u16(k), _u16(v)
    B, Hq, D = q.shape
    _, Hkv, n, _ = k.shape
    gran = _code(_GRANS, granularity)
    R = 1 if gran == TOKEN else Hkv
    S = np.array(S, dtype=np.float64, copy=True, order="C")
    assert S.shape == (B, R, n)
    if scale is None:
        scale = default_scale(D)
    l = np.empty((B, Hq, n), dtype=np.float64)
    idx = np.empty((B, R, k_sel), dtype=np.int32)
    out = np.empty((B, Hq, D), dtype=np.float64)
    t = np.zeros(3, dtype=np.float64)
    rc = lib.hor_step(B, Hq, Hkv, D, n, _code(_DTYPES, dtype), _code(_MODES, mode), gran,
                      float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(S), _ptr(l), int(k_sel),
                      _ptr(idx), _ptr(out), _ptr(t))
    if rc:
        raise ValueError("hor_step failed (%d)" % rc)
    if return_times:
        return S, idx, out, tuple(float(x) for x in t)
    return S, idx, out


def budget_k(n: int, alpha: float) -> int:
    """Token budget k = floor(alpha * n), clamped to [1, n] (top-alpha percent, Sec. 3.1)."""
    import math
    return max(1, min(n, int(math.floor(alpha * n + 1e-9))))


HIT_MAX = 65535   # the hit-rate table holds 2 bytes per token (Sec. 5.4 overhead analysis)


def bkp_update(hits, hot, idx, n_tokens: int, n_recent: int, capacity: int):
    """One maintenance pass of the Bidirectional KV Cache Pools after a
    decoding step (Sec. 4.2 BKP), per row (b, r) of a [B, R, Ncap] table:

    1. frequency tracking: every token of this step's selected set ``idx``
       ([B, R, k]) gains one hit, saturating at 65535 (a 2-byte table);
    2. temporal pinning: the ``n_recent`` most recent tokens of the first
       ``n_tokens`` (all of them if fewer) are hot;
    3. the remaining ``min(capacity, n_tokens) - n_recent`` hot slots go to
       the other tokens with the most hits; a token already hot wins a tie in
       hits (a cold token is promoted only when it strictly exceeds the
       lowest-ranked hot token), then the lower token index wins;
    4. promotions are tokens hot now and cold before, demotions the reverse,
       each in ascending token order.

    ``hits`` uint16 and ``hot`` bool/uint8 of shape [B, R, >= n_tokens].
    Returns (hits, hot, promote, demote): updated copies and two nested lists
    [B][R] of int arrays.  Positions at and beyond n_tokens are left as they
    are."""
    hits = np.array(hits, dtype=np.int64, copy=True)
    hot_old = np.array(hot, dtype=bool, copy=True)
    idx = np.asarray(idx, dtype=np.int64)
    B, R = hits.shape[0], hits.shape[1]
    N = int(n_tokens)
    W = min(int(n_recent), N)
    F = max(0, min(int(capacity), N) - W)
    hot_new = hot_old.copy()
    promote = [[None] * R for _ in range(B)]
    demote = [[None] * R for _ in range(B)]
    for b in range(B):
        for r in range(R):
            h = hits[b, r]
            for j in idx[b, r]:                                  # step 1
                h[j] = min(h[j] + 1, HIT_MAX)
            new = np.zeros(N, dtype=bool)
            new[N - W:] = True                                   # step 2
            rest = np.arange(N - W)
            old = hot_old[b, r, :N]
            # step 3: order by hits (more first), incumbency (hot first), index
            order = rest[np.lexsort((rest, ~old[rest], -h[rest]))]
            new[order[:F]] = True
            promote[b][r] = np.nonzero(new & ~old)[0]            # step 4
            demote[b][r] = np.nonzero(old & ~new)[0]
            hot_new[b, r, :N] = new
    return hits.astype(np.uint16), hot_new, promote, demote


def tier_apply(loc, promote, demote, n_prev: int, n_tokens: int, capacity: int):
    """The migration of one BKP pass between the two tiers (Sec. 4.2 BKP (3):
    promoted tokens move up to the hot pool, demoted ones down to the cold
    pool, an equal volume each way once the pool is full; the pools are
    exclusive, so a token's K/V row lives in exactly one of them).

    loc: int [B, R, >= n_tokens], the hot-pool slot of each token or -1 for
    the cold pool, as it stood after the previous pass over n_prev tokens
    (the pool then held min(capacity, n_prev) tokens in slots
    0 .. min(capacity, n_prev) - 1).  promote, demote: nested lists [B][R]
    of ascending token arrays (bkp_update's).

    Slot rule (a layout of this library; the paper places rows in pools but
    fixes no slot order): the slot of the i-th demoted token passes to the
    i-th promoted token; promoted tokens beyond the demoted ones take the
    slots never used before, in order, from min(capacity, n_prev).  A pass
    must leave min(capacity, n_tokens) tokens hot, so #promote - #demote must
    equal min(capacity, n_tokens) - min(capacity, n_prev) (else ValueError).

    Returns the new loc (a copy) and the moves [B][R] as lists of
    (token, slot, direction), direction +1 up (cold -> hot slot) and -1 down
    (hot slot -> cold)."""
    loc = np.array(loc, dtype=np.int64, copy=True)
    B, R = loc.shape[0], loc.shape[1]
    used_prev = min(int(capacity), int(n_prev))
    used_now = min(int(capacity), int(n_tokens))
    moves = [[None] * R for _ in range(B)]
    for b in range(B):
        for r in range(R):
            pr = [int(j) for j in promote[b][r]]
            de = [int(j) for j in demote[b][r]]
            if len(pr) - len(de) != used_now - used_prev:
                raise ValueError("row (%d, %d): %d promotions and %d demotions do not take the pool from %d to %d"
                                 % (b, r, len(pr), len(de), used_prev, used_now))
            mv = []
            for i, j in enumerate(de):
                slot = int(loc[b, r, j])
                if slot < 0:
                    raise ValueError("demoted token %d is not in the hot pool" % j)
                mv.append((j, slot, -1))
            for i, j in enumerate(pr):
                if loc[b, r, j] >= 0:
                    raise ValueError("promoted token %d is already in the hot pool" % j)
                slot = mv[i][1] if i < len(de) else used_prev + (i - len(de))
                mv.append((j, slot, +1))
            for j, slot, d in mv:
                loc[b, r, j] = slot if d > 0 else -1
            moves[b][r] = mv
    return loc, moves


def app_split(f_c, f_s, b_c, b_s, alpha_c, alpha_s, m, m0=0.0, iters=200):
    """Sec. 4.3: choose M_c (the rest, M_s = M - M_c, in the cold pool) so
    that the two parallel paths of Eq. 2 take equal time, each path being its
    scoring time plus moving its retained fraction,
        T_c(M_c) = M_c / f_c + alpha_c M_c / b_c,  T_s(M_s) = M_s / f_s + alpha_s M_s / b_s,
    subject to M_c <= m0 (Eq. 3; m0 <= 0: no bound).  T_c - T_s grows with
    M_c, so the balance point is found by bisection on [0, M]; the bound then
    clips it.  Returns (beta, M_c, M_s, T_c, T_s, capped)."""
    def t_c(x):
        return x / f_c + alpha_c * x / b_c

    def t_s(x):
        return x / f_s + alpha_s * x / b_s

    lo, hi = 0.0, float(m)
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if t_c(mid) < t_s(m - mid):
            lo = mid
        else:
            hi = mid
    mc = 0.5 * (lo + hi)
    capped = m0 > 0 and mc > m0
    if capped:
        mc = float(m0)
    ms = m - mc
    beta = mc / ms if ms > 0 else float("inf")
    return beta, mc, ms, t_c(mc), t_s(ms), capped
