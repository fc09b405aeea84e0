"""fp64 CPU oracle for MagicDec's verify/draft attention and the LSE merge.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library never links, loads or calls it, and it shares no code with it.

The arithmetic lives in ``oracle.c`` (plain C, double precision, direct
two-pass softmax); this module only marshals numpy arrays into it.  What it
computes, with the paper passages it follows, is stated at the top of
``oracle.c``.
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16 = 0, 1
VERIFY, DRAFT, INDEXED = 0, 1, 2

_lib = None


def open_library(path):
    """Bind a build of oracle.c at ``path`` (tests also bind deliberately broken builds)."""
    lib = ctypes.CDLL(path)
    i32, i64, dbl, vp = ctypes.c_int, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    lib.oracle_attention.restype = i32
    lib.oracle_attention.argtypes = [i32, i32, i32, i32, i32, i32, i32, dbl,
                                     vp, vp, vp, i64, i64, i64, i32, vp, i32, vp,
                                     i32, i32, vp, vp, vp, i32, i32]
    lib.oracle_merge_lse.restype = i32
    lib.oracle_merge_lse.argtypes = [i32, i64, i32, vp, vp, vp, vp]
    lib.oracle_snapkv_votes.restype = i32
    lib.oracle_snapkv_votes.argtypes = [i32, i32, i32, i32, i32, i32, dbl, vp, vp, i64, i64, i64,
                                        i32, vp, i32, vp, i32, i32, vp]
    lib.oracle_snapkv_select.restype = i32
    lib.oracle_snapkv_select.argtypes = [i32, vp, i32, vp, i32, i32, vp, vp]
    lib.oracle_attention_indexed.restype = i32
    lib.oracle_attention_indexed.argtypes = [i32, i32, i32, i32, i32, i32, dbl, vp, vp, vp, i64,
                                             i64, i64, i32, vp, i32, vp, vp, vp, i32, vp, vp,
                                             vp, i32, i32]
    return lib


def default_threads():
    """Worker threads for the oracle: the CPUs this process may run on, at most
    16 (one GPU's share of the cores on a shared GPU host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = open_library(_build.LIB)
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _raw(x):
    """Host array -> (contiguous array, dtype code).  bf16 travels as uint16 bits."""
    x = np.ascontiguousarray(x)
    if x.dtype == np.float32:
        return x, F32
    if x.dtype == np.uint16:
        return x, BF16
    raise TypeError(f"oracle inputs must be float32 or uint16 (bf16 bits), got {x.dtype}")


def attention(mode, q, k, v, kv_lens, *, n_sink=0, window=1, scale=None, page_table=None,
              want_probs=False, probs_len=None, nthreads=None, lib=None):
    """Reference attention in fp64.

    q: [B, q_len, Hq, d]; k, v: contiguous [B, S_alloc, Hkv, d] or, with
    ``page_table`` [B, max_pages] int32, paged [P, page_size, Hkv, d].
    float32 arrays, or uint16 arrays holding bf16 bit patterns.
    Returns (o [B, q_len, Hq, d] f64, lse [B, q_len, Hq] f64[, probs]).
    """
    lib = lib or _load()
    q, dt = _raw(q)
    k, dtk = _raw(k)
    v, dtv = _raw(v)
    if not (dt == dtk == dtv):
        raise TypeError("q, k and v must share a dtype")
    B, q_len, Hq, d = q.shape
    Hkv = k.shape[2]
    kv_lens = np.ascontiguousarray(kv_lens, dtype=np.int32)
    page_size, max_pages, pt = 0, 0, None
    if page_table is not None:
        pt = np.ascontiguousarray(page_table, dtype=np.int32)
        page_size, max_pages = k.shape[1], pt.shape[1]
    s_blk, s_tok, s_head = k.shape[1] * Hkv * d, Hkv * d, d
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    o = np.zeros((B, q_len, Hq, d), dtype=np.float64)
    lse = np.zeros((B, q_len, Hq), dtype=np.float64)
    probs = None
    if want_probs:
        probs_len = int(probs_len if probs_len is not None else (kv_lens.max() if B else 0))
        probs = np.zeros((B, q_len, Hq, probs_len), dtype=np.float64)
    if nthreads is None:
        nthreads = default_threads()
    rc = lib.oracle_attention(mode, B, q_len, Hq, Hkv, d, dt, float(scale), _ptr(q), _ptr(k),
                              _ptr(v), s_blk, s_tok, s_head, page_size, _ptr(pt), max_pages,
                              _ptr(kv_lens), n_sink, window, _ptr(o), _ptr(lse), _ptr(probs),
                              int(probs_len or 0), int(nthreads))
    if rc != 0:
        raise ValueError("oracle_attention rejected its arguments")
    return (o, lse, probs) if want_probs else (o, lse)


def indexed(q, k, v, kv_lens, idx, idx_len, *, scale=None, page_table=None, want_probs=False,
            probs_len=None, nthreads=None, lib=None):
    """Draft attention over a listed static cache (fp64).

    idx [B, Hkv, idx_stride] int32 prompt positions (any order, unique); only
    the first idx_len[b] entries of sequence b count and only positions in
    [0, S_b - q_len); the q_len speculated positions are always included,
    causally.  Other arguments as attention()."""
    lib = lib or _load()
    q, dt = _raw(q)
    k, dtk = _raw(k)
    v, dtv = _raw(v)
    if not (dt == dtk == dtv):
        raise TypeError("q, k and v must share a dtype")
    B, q_len, Hq, d = q.shape
    Hkv = k.shape[2]
    kv_lens = np.ascontiguousarray(kv_lens, dtype=np.int32)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    idx_len = np.ascontiguousarray(idx_len, dtype=np.int32)
    if idx.ndim != 3 or idx.shape[:2] != (B, Hkv) or idx_len.shape != (B,):
        raise ValueError("idx must be [B, Hkv, stride] and idx_len [B]")
    page_size, max_pages, pt = 0, 0, None
    if page_table is not None:
        pt = np.ascontiguousarray(page_table, dtype=np.int32)
        page_size, max_pages = k.shape[1], pt.shape[1]
    s_blk, s_tok, s_head = k.shape[1] * Hkv * d, Hkv * d, d
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    o = np.zeros((B, q_len, Hq, d), dtype=np.float64)
    lse = np.zeros((B, q_len, Hq), dtype=np.float64)
    probs = None
    if want_probs:
        probs_len = int(probs_len if probs_len is not None else (kv_lens.max() if B else 0))
        probs = np.zeros((B, q_len, Hq, probs_len), dtype=np.float64)
    if nthreads is None:
        nthreads = default_threads()
    rc = lib.oracle_attention_indexed(B, q_len, Hq, Hkv, d, dt, float(scale), _ptr(q), _ptr(k),
                                      _ptr(v), s_blk, s_tok, s_head, page_size, _ptr(pt),
                                      max_pages, _ptr(kv_lens), _ptr(idx), _ptr(idx_len),
                                      idx.shape[2], _ptr(o), _ptr(lse), _ptr(probs),
                                      int(probs_len or 0), int(nthreads))
    if rc != 0:
        raise ValueError("oracle_attention_indexed rejected its arguments")
    return (o, lse, probs) if want_probs else (o, lse)


def snapkv_votes(q_obs, k, kv_lens, *, pool=5, stride=None, scale=None, page_table=None,
                 lib=None):
    """Pooled observation-window votes per (sequence, kv head), fp64.
    q_obs [B, n_obs, Hq, d]; k as attention(); kv_lens = prompt lengths.
    Returns [B, Hkv, stride] (stride defaults to max(S_b) - n_obs)."""
    lib = lib or _load()
    q_obs, dt = _raw(q_obs)
    k, dtk = _raw(k)
    if dt != dtk:
        raise TypeError("q_obs and k must share a dtype")
    B, n_obs, Hq, d = q_obs.shape
    Hkv = k.shape[2]
    kv_lens = np.ascontiguousarray(kv_lens, dtype=np.int32)
    if stride is None:
        stride = max(1, int(kv_lens.max()) - n_obs) if B else 1
    page_size, max_pages, pt = 0, 0, None
    if page_table is not None:
        pt = np.ascontiguousarray(page_table, dtype=np.int32)
        page_size, max_pages = k.shape[1], pt.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((B, Hkv, stride), dtype=np.float64)
    rc = lib.oracle_snapkv_votes(B, n_obs, Hq, Hkv, d, dt, float(scale), _ptr(q_obs), _ptr(k),
                                 k.shape[1] * Hkv * d, Hkv * d, d, page_size, _ptr(pt), max_pages,
                                 _ptr(kv_lens), pool, stride, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_snapkv_votes rejected its arguments")
    return out


def snapkv_select(vals, lens, n_obs, budget, lib=None):
    """Ascending kept positions per row: top (budget - n_obs) prefix positions by
    value (ties: smaller position), then the observation window.
    vals [rows, stride] (float64), lens [rows] -> (idx [rows, budget] int32, counts [rows])."""
    lib = lib or _load()
    vals = np.ascontiguousarray(vals, dtype=np.float64)
    rows, stride = vals.shape
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    idx = np.full((rows, budget), -1, dtype=np.int32)
    counts = np.zeros(rows, dtype=np.int32)
    rc = lib.oracle_snapkv_select(rows, _ptr(vals), stride, _ptr(lens), n_obs, budget, _ptr(idx),
                                  _ptr(counts))
    if rc != 0:
        raise ValueError("oracle_snapkv_select rejected its arguments")
    return idx, counts


def verify(q, k, v, kv_lens, **kw):
    return attention(VERIFY, q, k, v, kv_lens, **kw)


def draft(q, k, v, kv_lens, n_sink, window, **kw):
    return attention(DRAFT, q, k, v, kv_lens, n_sink=n_sink, window=window, **kw)


def merge_lse(o_parts, lse_parts, lib=None):
    """o_parts [n_parts, n_rows, d], lse_parts [n_parts, n_rows] -> (o, lse) in fp64."""
    lib = lib or _load()
    o_parts = np.ascontiguousarray(o_parts, dtype=np.float64)
    lse_parts = np.ascontiguousarray(lse_parts, dtype=np.float64)
    n_parts, n_rows, d = o_parts.shape
    o = np.zeros((n_rows, d), dtype=np.float64)
    lse = np.zeros((n_rows,), dtype=np.float64)
    rc = lib.oracle_merge_lse(n_parts, n_rows, d, _ptr(o_parts), _ptr(lse_parts), _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle_merge_lse rejected its arguments")
    return o, lse


def bf16_bits_to_f64(bits):
    """Exact widening of bf16 bit patterns (uint16) to float64, for tests."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)
