"""MI355X (gfx950) verify/draft decode attention for MagicDec-style speculative decoding.

A thin ctypes binding over ``libmagicdec.so`` (C ABI in ``include/magicdec.h``):
argument marshalling only.  Every step of the attention runs in the library's
HIP kernels; PyTorch only supplies device memory and the stream.  There is no
CPU fallback: if the library is missing, every call raises.

    md_verify_attn(q, k, v, kv_lens, ...)          -> (o, lse)
    md_draft_attn(q, k, v, kv_lens, n_sink, window, ...) -> (o, lse)
    md_draft_attn_indexed(q, k, v, kv_lens, idx, idx_len, ...) -> (o, lse)
    md_merge_lse(o_parts, lse_parts, ...)         -> (o, lse)
    md_workspace_bytes(...)                       -> int
    md_kv_append(k, v, k_new, v_new, pos0, ...)   -> lens_out
    md_greedy_accept(logits, draft, ...)          -> (accepted, tokens, target)
    md_kv_commit(lens, accepted, q_len, ...)      (in place)
    md_streaming_list(prompt_lens, Hkv, n_sink, window) -> (idx, idx_len)
    md_kv_gather(dst_k, dst_v, src_k, src_v, idx, idx_len, src_lens, ...) -> dst_lens
    md_sd_expected_tokens / md_sd_latency_ratio / md_sd_best_gamma /
    md_sd_alpha_from_omega                        (host-only cost model, Eq. 1-4)

Shapes: q/o [B, L, Hq, d] (L = gamma + 1); k/v contiguous [B, S_alloc, Hkv, d]
or, with ``page_table`` [B, max_pages] int32, paged [P, page_size, Hkv, d];
kv_lens [B] int32 counting the L speculated tokens; lse [B, L, Hq] fp32.
"""
from __future__ import annotations

import ctypes
import functools
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmagicdec.so")

MD_OK, MD_ERR_INVALID_ARG, MD_ERR_UNSUPPORTED, MD_ERR_WORKSPACE, MD_ERR_HIP = range(5)
MD_F32, MD_BF16 = 0, 1
MD_MODE_VERIFY, MD_MODE_DRAFT, MD_MODE_DRAFT_INDEXED = 0, 1, 2
MD_ERRW_SHORT_LEN, MD_ERRW_LONG_LEN, MD_ERRW_BAD_PAGE = 1, 2, 4

EXPORTED = ["md_verify_attn", "md_draft_attn", "md_draft_attn_indexed", "md_merge_lse",
            "md_workspace_bytes", "md_workspace_bytes_indexed", "md_snapkv_votes",
            "md_snapkv_workspace_bytes", "md_snapkv_select", "md_kv_append",
            "md_greedy_accept", "md_greedy_accept_workspace_bytes", "md_kv_commit",
            "md_streaming_list", "md_kv_gather", "md_sd_expected_tokens", "md_sd_latency_ratio",
            "md_sd_best_gamma", "md_sd_alpha_from_omega",
            "md_status_str", "md_last_hip_error", "md_attn_args_size",
            "md_attn_noalloc",
            "md_bench_stream_read", "md_bench_evict", "md_bench_copy", "md_bench_fill",
            "md_bench_attn_stamps"]
MD_NOALLOC_SCRATCH_BYTES = 33 << 20


class MdAttnArgs(ctypes.Structure):
    """Mirror of ``md_attn_args`` (checked against md_attn_args_size())."""
    _fields_ = [
        ("num_seqs", ctypes.c_int32), ("q_len", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("sm_scale", ctypes.c_float),
        ("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("kv_stride_blk", ctypes.c_int64), ("kv_stride_tok", ctypes.c_int64),
        ("kv_stride_head", ctypes.c_int64),
        ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int64), ("page_table", ctypes.c_void_p),
        ("kv_lens", ctypes.c_void_p), ("max_kv_len", ctypes.c_int32),
        ("o", ctypes.c_void_p), ("lse", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
        ("err_word", ctypes.c_void_p),
    ]


class MdSnapkvArgs(ctypes.Structure):
    """Mirror of ``md_snapkv_args``."""
    _fields_ = [
        ("num_seqs", ctypes.c_int32), ("n_obs", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("sm_scale", ctypes.c_float),
        ("q_obs", ctypes.c_void_p), ("k", ctypes.c_void_p),
        ("kv_stride_blk", ctypes.c_int64), ("kv_stride_tok", ctypes.c_int64),
        ("kv_stride_head", ctypes.c_int64),
        ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int64), ("page_table", ctypes.c_void_p),
        ("prompt_lens", ctypes.c_void_p), ("max_prompt_len", ctypes.c_int32),
        ("votes", ctypes.c_void_p), ("votes_stride", ctypes.c_int32),
        ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
    ]


class MdKvCache(ctypes.Structure):
    """Mirror of ``md_kv_cache``."""
    _fields_ = [
        ("num_seqs", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("kv_stride_blk", ctypes.c_int64), ("kv_stride_tok", ctypes.c_int64),
        ("kv_stride_head", ctypes.c_int64),
        ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int64), ("page_table", ctypes.c_void_p),
        ("capacity", ctypes.c_int32),
    ]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libmagicdec.so.  torch is imported first so the library binds to the
    HIP runtime torch already loaded (same soname), not a second copy."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (shares its HIP runtime with the library)
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with __graft_entry__.build() "
            "(python -m paper_2408_11049_amd.build); there is no fallback path")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    args_p = ctypes.POINTER(MdAttnArgs)
    lib.md_verify_attn.argtypes = [args_p, vp]
    lib.md_verify_attn.restype = ctypes.c_int
    lib.md_draft_attn.argtypes = [args_p, i32, i32, vp]
    lib.md_draft_attn.restype = ctypes.c_int
    lib.md_draft_attn_indexed.argtypes = [args_p, vp, vp, i32, vp]
    lib.md_draft_attn_indexed.restype = ctypes.c_int
    lib.md_attn_noalloc.argtypes = [args_p, i32, i32, i32, vp]
    lib.md_attn_noalloc.restype = ctypes.c_int
    lib.md_workspace_bytes_indexed.argtypes = [args_p, i32]
    lib.md_workspace_bytes_indexed.restype = sz
    sk_p = ctypes.POINTER(MdSnapkvArgs)
    lib.md_snapkv_votes.argtypes = [sk_p, vp]
    lib.md_snapkv_votes.restype = ctypes.c_int
    lib.md_snapkv_workspace_bytes.argtypes = [sk_p]
    lib.md_snapkv_workspace_bytes.restype = sz
    lib.md_snapkv_select.argtypes = [i32, i32, vp, i32, vp, i32, i32, i32, vp, vp, vp]
    lib.md_snapkv_select.restype = ctypes.c_int
    lib.md_kv_append.argtypes = [ctypes.POINTER(MdKvCache), i32, vp, vp, vp, vp, vp]
    lib.md_kv_append.restype = ctypes.c_int
    lib.md_greedy_accept.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.md_greedy_accept.restype = ctypes.c_int
    lib.md_greedy_accept_workspace_bytes.argtypes = [i32, i32, i32]
    lib.md_greedy_accept_workspace_bytes.restype = sz
    lib.md_kv_commit.argtypes = [i32, i32, vp, vp, i32, vp, i32, i32, i32, vp]
    lib.md_kv_commit.restype = ctypes.c_int
    lib.md_streaming_list.argtypes = [i32, i32, vp, i32, i32, vp, vp, vp]
    lib.md_streaming_list.restype = ctypes.c_int
    lib.md_kv_gather.argtypes = [ctypes.POINTER(MdKvCache), ctypes.POINTER(MdKvCache), vp, i32,
                                 vp, vp, vp, vp]
    lib.md_kv_gather.restype = ctypes.c_int
    f64 = ctypes.c_double
    lib.md_sd_expected_tokens.argtypes = [i32, f64]
    lib.md_sd_expected_tokens.restype = f64
    lib.md_sd_latency_ratio.argtypes = [i32, f64, f64, f64, f64, f64]
    lib.md_sd_latency_ratio.restype = f64
    lib.md_sd_best_gamma.argtypes = [i32, f64, f64, f64, f64, vp, vp, vp]
    lib.md_sd_best_gamma.restype = ctypes.c_int
    lib.md_sd_alpha_from_omega.argtypes = [i32, f64]
    lib.md_sd_alpha_from_omega.restype = f64
    lib.md_merge_lse.argtypes = [i32, i64, i32, i32, vp, vp, vp, vp, vp]
    lib.md_merge_lse.restype = ctypes.c_int
    lib.md_workspace_bytes.argtypes = [args_p, i32, i32, i32]
    lib.md_workspace_bytes.restype = sz
    lib.md_status_str.argtypes = [ctypes.c_int]
    lib.md_status_str.restype = ctypes.c_char_p
    lib.md_last_hip_error.argtypes = []
    lib.md_last_hip_error.restype = ctypes.c_char_p
    lib.md_attn_args_size.argtypes = []
    lib.md_attn_args_size.restype = sz
    lib.md_bench_stream_read.argtypes = [vp, sz, vp, vp]
    lib.md_bench_stream_read.restype = ctypes.c_int
    lib.md_bench_evict.argtypes = [vp, sz, vp, vp]
    lib.md_bench_evict.restype = ctypes.c_int
    lib.md_bench_copy.argtypes = [vp, vp, sz, vp]
    lib.md_bench_copy.restype = ctypes.c_int
    lib.md_bench_fill.argtypes = [vp, sz, ctypes.c_uint32, vp]
    lib.md_bench_fill.restype = ctypes.c_int
    lib.md_bench_attn_stamps.argtypes = [args_p, i32, i32, i32, vp, i64, ctypes.POINTER(i64), vp]
    lib.md_bench_attn_stamps.restype = ctypes.c_int
    if lib.md_attn_args_size() != ctypes.sizeof(MdAttnArgs):
        raise RuntimeError("md_attn_args layout mismatch between the binding and the library")
    _lib = lib
    return lib


def _check(status: int):
    if status == MD_OK:
        return
    lib = load_library()
    msg = lib.md_status_str(status).decode()
    if status == MD_ERR_HIP:
        raise RuntimeError(f"magicdec: {msg}: {lib.md_last_hip_error().decode()}")
    raise ValueError(f"magicdec: {msg} (status {status})")


def _stream_scoped(fn):
    """Run a binding call with its `stream` (when given) as torch's current
    stream, so every tensor the binding allocates for the call (outputs,
    workspace) belongs to the stream the call's kernels run on: the caching
    allocator then never hands such a block to other work before those
    kernels are done, even when the binding drops it on return."""
    @functools.wraps(fn)
    def wrapped(*args, stream=None, **kw):
        if stream is None:
            return fn(*args, stream=None, **kw)
        import torch
        with torch.cuda.stream(stream):
            return fn(*args, stream=stream, **kw)
    return wrapped


def _stream_handle(t, stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(t.device)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _on_gpu(ref, **tensors):
    """Every tensor a call hands to the kernels must live on ref's GPU: a host
    or other-device address would reach them as a wild pointer, which the
    library (it sees plain pointers) cannot tell from a good one."""
    if not ref.is_cuda:
        raise ValueError(f"tensors must be on a GPU, not {ref.device}")
    for name, t in tensors.items():
        if t is not None and t.device != ref.device:
            raise ValueError(f"{name} is on {t.device}; the call runs on {ref.device}")


def _ints(name, t, n):
    """A device int32 vector the kernels read (or write) n entries of."""
    import torch
    if t.dtype != torch.int32 or not t.is_contiguous() or t.numel() < n:
        raise ValueError(f"{name} must be contiguous int32 with at least {n} entries")


def _torch():
    import torch
    return torch


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return MD_F32
    if t.dtype == torch.bfloat16:
        return MD_BF16
    raise ValueError(f"unsupported dtype {t.dtype}; q/k/v must be float32 or bfloat16")


def make_args(q, k, v, kv_lens, *, max_kv_len: Optional[int] = None, page_table=None,
              sm_scale: float = 0.0, out=None, lse=None, workspace=None,
              err_word=None) -> MdAttnArgs:
    """Fill md_attn_args from tensors (no data is read or moved)."""
    if q.dim() != 4 or k.dim() != 4 or v.dim() != 4:
        raise ValueError("q, k, v must be 4-D")
    B, L, Hq, d = q.shape
    paged = page_table is not None
    _on_gpu(q, k=k, v=v, kv_lens=kv_lens, page_table=page_table, out=out, lse=lse,
            workspace=workspace, err_word=err_word)
    if k.shape != v.shape or k.stride() != v.stride():
        raise ValueError("k and v must share shape and strides")
    if k.shape[3] != d:
        raise ValueError("k/v head_dim must equal q's")
    _ints("kv_lens", kv_lens, B)
    if out is not None and (out.shape != q.shape or out.dtype != q.dtype):
        raise ValueError("o must have q's shape and dtype")
    if lse is not None and (lse.dtype != _torch().float32 or not lse.is_contiguous()
                            or lse.numel() < B * L * Hq):
        raise ValueError("lse must be contiguous float32 [B, L, Hq]")
    if paged and page_table.dim() == 2 and page_table.shape[0] < B:
        raise ValueError("page_table must have a row per sequence")
    if k.stride(3) != 1:
        raise ValueError("the head_dim axis of k/v must be unit-stride")
    if not q.is_contiguous() or (out is not None and not out.is_contiguous()):
        raise ValueError("q and o must be contiguous [B, L, Hq, d]")
    if max_kv_len is None:  # a bound that needs no device sync
        max_kv_len = page_table.shape[1] * k.shape[1] if paged else k.shape[1]
    if B > 0 and not paged and k.shape[1] < max_kv_len:
        raise ValueError("contiguous k/v must hold max_kv_len tokens per sequence")
    if B > 0 and not paged and k.shape[0] < B:
        raise ValueError("contiguous k/v must hold B sequences")
    a = MdAttnArgs()
    a.num_seqs, a.q_len, a.num_q_heads, a.num_kv_heads, a.head_dim = B, L, Hq, k.shape[2], d
    a.dtype = _dtype_code(q)
    if _dtype_code(k) != a.dtype or _dtype_code(v) != a.dtype:
        raise ValueError("q, k, v must share a dtype")
    a.sm_scale = float(sm_scale)
    a.q, a.k, a.v = q.data_ptr(), k.data_ptr(), v.data_ptr()
    a.kv_stride_blk, a.kv_stride_tok, a.kv_stride_head = k.stride(0), k.stride(1), k.stride(2)
    if paged:
        import torch
        if page_table.dtype != torch.int32 or not page_table.is_contiguous():
            raise ValueError("page_table must be contiguous int32 [B, max_pages]")
        a.page_size, a.max_pages_per_seq = k.shape[1], page_table.shape[1]
        a.num_pages = k.shape[0]
        a.page_table = page_table.data_ptr()
    a.kv_lens = kv_lens.data_ptr()
    a.max_kv_len = int(max_kv_len)
    a.o = out.data_ptr() if out is not None else None
    a.lse = lse.data_ptr() if lse is not None else None
    if workspace is not None:
        a.workspace, a.workspace_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    if err_word is not None:
        import torch
        if err_word.dtype != torch.int32 or err_word.numel() < 1:
            raise ValueError("err_word must be a device int32 tensor")
        a.err_word = err_word.data_ptr()
    return a


def md_workspace_bytes(q, k, v, kv_lens, *, mode=MD_MODE_VERIFY, n_sink=0, window=1, **kw) -> int:
    lib = load_library()
    a = make_args(q, k, v, kv_lens, **kw)
    return int(lib.md_workspace_bytes(ctypes.byref(a), mode, n_sink, window))


@_stream_scoped
def _attention(mode, q, k, v, kv_lens, n_sink, window, *, max_kv_len=None, page_table=None,
               sm_scale=0.0, out=None, lse=None, return_lse=True, workspace=None, stream=None,
               idx=None, idx_len=None, err_word=None):
    import torch
    lib = load_library()
    if kv_lens.dtype != torch.int32:
        raise ValueError("kv_lens must be int32")
    if out is None:
        out = torch.empty_like(q)
    if lse is None and return_lse:
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    a = make_args(q, k, v, kv_lens, max_kv_len=max_kv_len, page_table=page_table,
                  sm_scale=sm_scale, out=out, lse=lse, err_word=err_word)
    if mode == MD_MODE_DRAFT_INDEXED:
        need = int(lib.md_workspace_bytes_indexed(ctypes.byref(a), idx.shape[2]))
    else:
        need = int(lib.md_workspace_bytes(ctypes.byref(a), mode, n_sink, window))
    if need and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    _on_gpu(q, workspace=workspace, idx=idx, idx_len=idx_len)
    if idx_len is not None:
        _ints("idx_len", idx_len, q.shape[0])
    if workspace is not None:
        a.workspace = workspace.data_ptr()
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    s = _stream_handle(q, stream)
    if mode == MD_MODE_VERIFY:
        st = lib.md_verify_attn(ctypes.byref(a), s)
    elif mode == MD_MODE_DRAFT:
        st = lib.md_draft_attn(ctypes.byref(a), int(n_sink), int(window), s)
    else:
        st = lib.md_draft_attn_indexed(ctypes.byref(a), _ptr(idx), _ptr(idx_len), idx.shape[2], s)
    _check(st)
    return out, lse


@_stream_scoped
def md_attn_noalloc(mode, q, k, v, kv_lens, n_sink=0, window=1, *, max_kv_len=None,
                    page_table=None, sm_scale=0.0, out=None, lse=None, stream=None):
    """md_verify_attn (mode 0) or md_draft_attn (mode 1) through the entry
    point that allocates nothing on the device: the library's static scratch
    stands in for the workspace (see include/magicdec.h).  `out` and `lse`
    are the caller's; passing both makes the call allocation-free on the
    torch side too."""
    import torch
    lib = load_library()
    if kv_lens.dtype != torch.int32:
        raise ValueError("kv_lens must be int32")
    if out is None:
        out = torch.empty_like(q)
    a = make_args(q, k, v, kv_lens, max_kv_len=max_kv_len, page_table=page_table,
                  sm_scale=sm_scale, out=out, lse=lse)
    _check(lib.md_attn_noalloc(ctypes.byref(a), int(mode), int(n_sink), int(window),
                               _stream_handle(q, stream)))
    return out, lse


def md_verify_attn(q, k, v, kv_lens, **kw):
    """Verification attention over the full cache (see include/magicdec.h)."""
    return _attention(MD_MODE_VERIFY, q, k, v, kv_lens, 0, 1, **kw)


def md_draft_attn(q, k, v, kv_lens, n_sink, window, **kw):
    """StreamingLLM-style sparse draft attention (see include/magicdec.h)."""
    return _attention(MD_MODE_DRAFT, q, k, v, kv_lens, n_sink, window, **kw)


def md_draft_attn_indexed(q, k, v, kv_lens, idx, idx_len, **kw):
    """Draft attention over a listed (SnapKV-style) static cache.

    idx [B, Hkv, stride] int32 prompt positions (unique), idx_len [B] int32
    (see include/magicdec.h)."""
    import torch
    if idx.dtype != torch.int32 or idx_len.dtype != torch.int32:
        raise ValueError("idx and idx_len must be int32")
    if idx.dim() != 3 or not idx.is_contiguous() or idx.shape[:2] != (q.shape[0], k.shape[2]):
        raise ValueError("idx must be contiguous [B, Hkv, stride]")
    return _attention(MD_MODE_DRAFT_INDEXED, q, k, v, kv_lens, 0, 1, idx=idx, idx_len=idx_len, **kw)


def md_bench_attn_stamps(mode, q, k, v, kv_lens, n_sink=0, window=1, *, max_kv_len=None,
                         page_table=None, out=None, workspace=None, stream=None):
    """Measurement: md_verify_attn (mode 0) or md_draft_attn (mode 1) with
    every workgroup recording four wall-clock stamps (start, first tile done,
    main loop done, end).  Returns (o, stamps int64 [workgroups, 4]) -- raw
    readings of the GPU's constant-rate clock (include/magicdec_bench.h)."""
    import torch
    lib = load_library()
    if out is None:
        out = torch.empty_like(q)
    a = make_args(q, k, v, kv_lens, max_kv_len=max_kv_len, page_table=page_table, out=out)
    need = int(lib.md_workspace_bytes(ctypes.byref(a), mode, n_sink, window))
    if need and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if workspace is not None:
        _on_gpu(q, workspace=workspace)
        a.workspace, a.workspace_bytes = workspace.data_ptr(), workspace.numel()
    n = ctypes.c_int64(0)
    s = _stream_handle(q, stream)
    st = lib.md_bench_attn_stamps(ctypes.byref(a), mode, n_sink, window, None, 0, ctypes.byref(n), s)
    if st != MD_ERR_INVALID_ARG or n.value < 0:
        _check(st)
    stamps = torch.zeros((max(n.value, 1), 4), dtype=torch.int64, device=q.device)
    _check(lib.md_bench_attn_stamps(ctypes.byref(a), mode, n_sink, window,
                                    ctypes.c_void_p(stamps.data_ptr()), stamps.numel(),
                                    ctypes.byref(n), s))
    return out, stamps[: n.value]


def make_snapkv_args(q_obs, k, prompt_lens, *, max_prompt_len=None, page_table=None,
                     sm_scale=0.0, votes=None, workspace=None) -> MdSnapkvArgs:
    """Fill md_snapkv_args from tensors (no data is read or moved); votes may
    be None to size the workspace only."""
    import torch
    B, n_obs, Hq, d = q_obs.shape
    paged = page_table is not None
    _on_gpu(q_obs, k=k, prompt_lens=prompt_lens, page_table=page_table, votes=votes,
            workspace=workspace)
    if k.stride(3) != 1 or not q_obs.is_contiguous():
        raise ValueError("q_obs must be contiguous and k unit-stride in head_dim")
    if k.dim() != 4 or k.shape[3] != d:
        raise ValueError("k must be 4-D with q_obs's head_dim")
    _ints("prompt_lens", prompt_lens, B)
    if votes is not None and (votes.dtype != torch.float32 or not votes.is_contiguous()
                              or votes.dim() != 3 or votes.shape[:2] != (B, k.shape[2])):
        raise ValueError("votes must be contiguous float32 [B, Hkv, stride]")
    if max_prompt_len is None:
        max_prompt_len = page_table.shape[1] * k.shape[1] if paged else k.shape[1]
    if B > 0 and not paged and k.shape[1] < max_prompt_len:
        raise ValueError("contiguous k must hold max_prompt_len tokens per sequence")
    a = MdSnapkvArgs()
    a.num_seqs, a.n_obs, a.num_q_heads, a.num_kv_heads, a.head_dim = B, n_obs, Hq, k.shape[2], d
    a.dtype = _dtype_code(q_obs)
    if _dtype_code(k) != a.dtype:
        raise ValueError("q_obs and k must share a dtype")
    a.sm_scale = float(sm_scale)
    a.q_obs, a.k = q_obs.data_ptr(), k.data_ptr()
    a.kv_stride_blk, a.kv_stride_tok, a.kv_stride_head = k.stride(0), k.stride(1), k.stride(2)
    if paged:
        a.page_size, a.max_pages_per_seq = k.shape[1], page_table.shape[1]
        a.num_pages = k.shape[0]
        a.page_table = page_table.data_ptr()
    a.prompt_lens = prompt_lens.data_ptr()
    a.max_prompt_len = int(max_prompt_len)
    a.votes_stride = max(1, int(max_prompt_len) - n_obs)
    if votes is not None:
        a.votes, a.votes_stride = votes.data_ptr(), votes.shape[-1]
    if workspace is not None:
        a.workspace, a.workspace_bytes = workspace.data_ptr(), workspace.numel()
    return a


def md_snapkv_workspace_bytes(q_obs, k, prompt_lens, **kw) -> int:
    """Workspace bytes md_snapkv_votes needs for these tensors."""
    return int(load_library().md_snapkv_workspace_bytes(
        ctypes.byref(make_snapkv_args(q_obs, k, prompt_lens, **kw))))


@_stream_scoped
def md_snapkv_votes(q_obs, k, prompt_lens, *, max_prompt_len=None, page_table=None,
                    sm_scale=0.0, votes=None, workspace=None, stream=None):
    """Raw SnapKV votes [B, Hkv, stride] fp32 of every prefix position
    (q_obs [B, n_obs, Hq, d]; k contiguous or paged; see include/magicdec.h)."""
    import torch
    lib = load_library()
    kw = dict(max_prompt_len=max_prompt_len, page_table=page_table, sm_scale=sm_scale)
    if votes is None:
        stride = make_snapkv_args(q_obs, k, prompt_lens, **kw).votes_stride
        votes = torch.zeros((q_obs.shape[0], k.shape[2], stride), dtype=torch.float32,
                            device=q_obs.device)
    if workspace is None:
        need = md_snapkv_workspace_bytes(q_obs, k, prompt_lens, **kw)
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q_obs.device)
    a = make_snapkv_args(q_obs, k, prompt_lens, votes=votes, workspace=workspace, **kw)
    _check(lib.md_snapkv_votes(ctypes.byref(a), _stream_handle(q_obs, stream)))
    return votes


@_stream_scoped
def md_snapkv_select(votes, prompt_lens, n_obs, budget, *, pool=5, idx=None, idx_len=None,
                     stream=None):
    """Pool the votes [B, Hkv, stride] and keep budget positions per (sequence,
    kv head): returns (idx [B, Hkv, budget] int32 ascending, idx_len [B] int32)."""
    import torch
    lib = load_library()
    B, Hkv, stride = votes.shape
    if votes.dtype != torch.float32 or not votes.is_contiguous():
        raise ValueError("votes must be contiguous float32 [B, Hkv, stride]")
    _on_gpu(votes, prompt_lens=prompt_lens, idx=idx, idx_len=idx_len)
    _ints("prompt_lens", prompt_lens, B)
    if idx is not None and (idx.dtype != torch.int32 or not idx.is_contiguous()
                            or idx.shape[:2] != (B, Hkv) or idx.shape[2] < budget):
        raise ValueError("idx must be contiguous int32 [B, Hkv, >= budget]")
    if idx_len is not None:
        _ints("idx_len", idx_len, B)
    if idx is None:
        idx = torch.full((B, Hkv, budget), -1, dtype=torch.int32, device=votes.device)
    if idx_len is None:
        idx_len = torch.zeros((B,), dtype=torch.int32, device=votes.device)
    _check(lib.md_snapkv_select(B, Hkv, _ptr(votes), stride, _ptr(prompt_lens), n_obs, pool,
                                budget, _ptr(idx), _ptr(idx_len), _stream_handle(votes, stream)))
    return idx, idx_len


@_stream_scoped
def md_merge_lse(o_parts, lse_parts, *, out_dtype=None, out=None, lse=None, stream=None):
    """o_parts [n_parts, n_rows, d] fp32, lse_parts [n_parts, n_rows] fp32 -> (o, lse)."""
    import torch
    lib = load_library()
    n_parts, n_rows, d = o_parts.shape
    if o_parts.dtype != torch.float32 or lse_parts.dtype != torch.float32:
        raise ValueError("o_parts and lse_parts must be float32")
    if not o_parts.is_contiguous() or not lse_parts.is_contiguous():
        raise ValueError("o_parts and lse_parts must be contiguous")
    _on_gpu(o_parts, lse_parts=lse_parts, out=out, lse=lse)
    if tuple(lse_parts.shape) != (n_parts, n_rows):
        raise ValueError("lse_parts must be [n_parts, n_rows]")
    if out is not None and (tuple(out.shape) != (n_rows, d) or not out.is_contiguous()):
        raise ValueError("out must be contiguous [n_rows, d]")
    if lse is not None and (lse.dtype != torch.float32 or lse.numel() < n_rows):
        raise ValueError("lse must be float32 [n_rows]")
    if out is None:
        out = torch.empty((n_rows, d), dtype=out_dtype or torch.float32, device=o_parts.device)
    if lse is None:
        lse = torch.empty((n_rows,), dtype=torch.float32, device=o_parts.device)
    code = _dtype_code(out)
    st = lib.md_merge_lse(n_parts, n_rows, d, code, _ptr(o_parts), _ptr(lse_parts), _ptr(out),
                          _ptr(lse), _stream_handle(o_parts, stream))
    _check(st)
    return out, lse


def make_kv_cache(k, v, *, num_seqs=None, page_table=None) -> MdKvCache:
    """Fill md_kv_cache from the cache tensors: contiguous [B, S_alloc, Hkv, d]
    or, with page_table [B, max_pages] int32, paged [P, page_size, Hkv, d]."""
    import torch
    if k.dim() != 4 or k.shape != v.shape or k.stride() != v.stride() or k.stride(3) != 1:
        raise ValueError("k and v must be 4-D with equal shapes and strides, head_dim unit-stride")
    _on_gpu(k, v=v, page_table=page_table)
    c = MdKvCache()
    paged = page_table is not None
    c.num_seqs = int(num_seqs if num_seqs is not None else
                     (page_table.shape[0] if paged else k.shape[0]))
    c.num_kv_heads, c.head_dim = k.shape[2], k.shape[3]
    c.dtype = _dtype_code(k)
    if _dtype_code(v) != c.dtype:
        raise ValueError("k and v must share a dtype")
    c.k, c.v = k.data_ptr(), v.data_ptr()
    c.kv_stride_blk, c.kv_stride_tok, c.kv_stride_head = k.stride(0), k.stride(1), k.stride(2)
    if paged:
        if page_table.dtype != torch.int32 or not page_table.is_contiguous():
            raise ValueError("page_table must be contiguous int32 [B, max_pages]")
        if page_table.dim() != 2 or page_table.shape[0] < c.num_seqs:
            raise ValueError("page_table must have a row per sequence")
        c.page_size, c.max_pages_per_seq = k.shape[1], page_table.shape[1]
        c.num_pages = k.shape[0]
        c.page_table = page_table.data_ptr()
    else:
        if c.num_seqs > k.shape[0]:
            raise ValueError("contiguous k/v must hold num_seqs sequences")
        c.capacity = k.shape[1]
    return c


@_stream_scoped
def md_kv_append(k, v, k_new, v_new, pos0, *, page_table=None, lens_out=None, stream=None):
    """Write k_new/v_new [B, n_new, Hkv, d] at positions pos0[b] + i of the cache
    (in place).  Returns lens_out [B] int32 = pos0 + n_new."""
    import torch
    lib = load_library()
    B, n_new = k_new.shape[:2]
    if k_new.shape != v_new.shape or not k_new.is_contiguous() or not v_new.is_contiguous():
        raise ValueError("k_new and v_new must be contiguous [B, n_new, Hkv, d] of equal shape")
    if k_new.dtype != k.dtype or v_new.dtype != v.dtype:
        raise ValueError("appended rows must have the cache dtype")
    c = make_kv_cache(k, v, num_seqs=B, page_table=page_table)
    if B and (k_new.shape[2] != c.num_kv_heads or k_new.shape[3] != c.head_dim):
        raise ValueError("appended rows must have the cache's heads and head_dim")
    _on_gpu(k, k_new=k_new, v_new=v_new, pos0=pos0, lens_out=lens_out)
    _ints("pos0", pos0, B)
    if lens_out is None:
        lens_out = torch.empty((B,), dtype=torch.int32, device=k.device)
    _ints("lens_out", lens_out, B)
    _check(lib.md_kv_append(ctypes.byref(c), n_new, _ptr(k_new), _ptr(v_new), _ptr(pos0),
                            _ptr(lens_out), _stream_handle(k, stream)))
    return lens_out


@_stream_scoped
def md_greedy_accept(logits, draft, *, accepted=None, tokens=None, target=None,
                     want_target=True, workspace=None, stream=None):
    """logits [B, gamma + 1, vocab] float32/bfloat16, draft [B, gamma] int32 ->
    (accepted [B], tokens [B, gamma + 1], target [B, gamma + 1] or None), int32."""
    import torch
    lib = load_library()
    B, L, vocab = logits.shape
    if not logits.is_contiguous():
        raise ValueError("logits must be contiguous [B, gamma + 1, vocab]")
    if draft.shape != (B, L - 1) or draft.dtype != torch.int32 or not draft.is_contiguous():
        raise ValueError("draft must be contiguous int32 [B, gamma]")
    _on_gpu(logits, draft=draft, accepted=accepted, tokens=tokens, target=target,
            workspace=workspace)
    if accepted is not None:
        _ints("accepted", accepted, B)
    for name, t_ in (("tokens", tokens), ("target", target)):
        if t_ is not None:
            _ints(name, t_, B * L)
    dev = logits.device
    if accepted is None:
        accepted = torch.empty((B,), dtype=torch.int32, device=dev)
    if tokens is None:
        tokens = torch.empty((B, L), dtype=torch.int32, device=dev)
    if target is None and want_target:
        target = torch.empty((B, L), dtype=torch.int32, device=dev)
    if workspace is None:
        nbytes = lib.md_greedy_accept_workspace_bytes(B, L - 1, vocab)
        workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    _check(lib.md_greedy_accept(B, L - 1, vocab, _dtype_code(logits), _ptr(logits),
                                _ptr(draft) if L > 1 else None, _ptr(accepted), _ptr(tokens),
                                _ptr(target), _ptr(workspace),
                                workspace.numel() * workspace.element_size(),
                                _stream_handle(logits, stream)))
    return accepted, tokens, target


@_stream_scoped
def md_kv_commit(lens, accepted, q_len, *, idx=None, ring_start=0, ring_len=None, stream=None):
    """lens [B] int32 in place: C -> C + accepted + 1; with idx [B, Hkv, stride]
    the kept positions also enter each list's ring [ring_start, ring_start + ring_len)."""
    lib = load_library()
    B = lens.shape[0]
    Hkv, stride = (idx.shape[1], idx.shape[2]) if idx is not None else (0, 0)
    _on_gpu(lens, accepted=accepted, idx=idx)
    _ints("lens", lens, B)
    _ints("accepted", accepted, B)
    if idx is not None and (not idx.is_contiguous() or idx.dtype != lens.dtype or idx.shape[0] < B):
        raise ValueError("idx must be contiguous int32 [B, Hkv, stride]")
    if ring_len is None:
        ring_len = stride - ring_start
    _check(lib.md_kv_commit(B, q_len, _ptr(lens), _ptr(accepted), Hkv, _ptr(idx), stride,
                            ring_start, ring_len, _stream_handle(lens, stream)))
    return lens


@_stream_scoped
def md_streaming_list(prompt_lens, num_kv_heads, n_sink, window, *, idx=None, idx_len=None,
                      stream=None):
    """Sink-plus-window draft lists [B, Hkv, n_sink + window] and idx_len [B]."""
    import torch
    lib = load_library()
    B = prompt_lens.shape[0]
    dev = prompt_lens.device
    _on_gpu(prompt_lens, idx=idx, idx_len=idx_len)
    _ints("prompt_lens", prompt_lens, B)
    if idx is None:
        idx = torch.empty((B, num_kv_heads, n_sink + window), dtype=torch.int32, device=dev)
    if idx_len is None:
        idx_len = torch.empty((B,), dtype=torch.int32, device=dev)
    _ints("idx", idx, B * num_kv_heads * (n_sink + window))
    _ints("idx_len", idx_len, B)
    _check(lib.md_streaming_list(B, num_kv_heads, _ptr(prompt_lens), n_sink, window, _ptr(idx),
                                 _ptr(idx_len), _stream_handle(prompt_lens, stream)))
    return idx, idx_len


@_stream_scoped
def md_kv_gather(dst_k, dst_v, src_k, src_v, idx, idx_len, src_lens, *, dst_page_table=None,
                 src_page_table=None, dst_lens=None, stream=None):
    """Gather each (sequence, kv head)'s listed rows idx [B, Hkv, stride] of the
    src cache into rows 0.. of the dst cache (in place), zeros for entries
    outside [0, src_lens[b]).  Returns dst_lens [B] int32 = min(idx_len, stride)."""
    import torch
    lib = load_library()
    B, Hkv, stride = idx.shape
    if idx.dtype != torch.int32 or not idx.is_contiguous():
        raise ValueError("idx must be contiguous int32 [B, Hkv, stride]")
    _on_gpu(idx, dst_k=dst_k, dst_v=dst_v, src_k=src_k, src_v=src_v, idx_len=idx_len,
            src_lens=src_lens, dst_page_table=dst_page_table, src_page_table=src_page_table,
            dst_lens=dst_lens)
    _ints("idx_len", idx_len, B)
    _ints("src_lens", src_lens, B)
    dst = make_kv_cache(dst_k, dst_v, num_seqs=B, page_table=dst_page_table)
    src = make_kv_cache(src_k, src_v, num_seqs=B, page_table=src_page_table)
    if dst_lens is None:
        dst_lens = torch.empty((B,), dtype=torch.int32, device=idx.device)
    _ints("dst_lens", dst_lens, B)
    _check(lib.md_kv_gather(ctypes.byref(dst), ctypes.byref(src), _ptr(idx), stride,
                            _ptr(idx_len), _ptr(src_lens), _ptr(dst_lens),
                            _stream_handle(idx, stream)))
    return dst_lens


def md_sd_expected_tokens(gamma: int, alpha: float) -> float:
    """Eq. 1: expected tokens per verification (NaN for invalid arguments)."""
    return load_library().md_sd_expected_tokens(int(gamma), float(alpha))


def md_sd_latency_ratio(gamma, alpha, t_target, t_draft, t_verify, t_select=0.0) -> float:
    """Eq. 2 with Eq. 3's draft time: T_Avg^SD / T_T."""
    return load_library().md_sd_latency_ratio(int(gamma), float(alpha), float(t_target),
                                              float(t_draft), float(t_select), float(t_verify))


def md_sd_best_gamma(alpha, t_target, t_draft, t_verify_by_gamma, t_select=0.0):
    """Eq. 4 over gamma = 1 .. len(t_verify_by_gamma); t_verify_by_gamma[g-1] = T_V(g).
    Returns (gamma, ratio)."""
    n = len(t_verify_by_gamma)
    arr = (ctypes.c_double * max(n, 1))(*[float(x) for x in t_verify_by_gamma])
    g = ctypes.c_int32()
    r = ctypes.c_double()
    _check(load_library().md_sd_best_gamma(n, float(alpha), float(t_target), float(t_draft),
                                           float(t_select), ctypes.cast(arr, ctypes.c_void_p),
                                           ctypes.byref(g), ctypes.byref(r)))
    return g.value, r.value


def md_sd_alpha_from_omega(gamma: int, omega: float) -> float:
    """The acceptance rate implied by a measured Omega (inverse of Eq. 1)."""
    return load_library().md_sd_alpha_from_omega(int(gamma), float(omega))


# Short aliases.
verify_attn = md_verify_attn
draft_attn = md_draft_attn
draft_attn_indexed = md_draft_attn_indexed
merge_lse = md_merge_lse
workspace_bytes = md_workspace_bytes
kv_append = md_kv_append
greedy_accept = md_greedy_accept
kv_commit = md_kv_commit
streaming_list = md_streaming_list
kv_gather = md_kv_gather
