"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
(via the binding) and the fp64 oracle on the same seeded inputs, compare."""
import math
import sys

import numpy as np
import torch

import oracle
import paper_2408_11049_amd as md
from paper_2408_11049_amd import workloads as wl

# Max-abs tolerances on O (and lse) against the fp64 oracle.
TOL = {"f32": 1e-5, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True, file=sys.stderr)


def run_gpu(mode, c, n_sink=0, window=1, max_kv_len=None, poison=True):
    """One library call on the case's device tensors; O pre-filled with NaN so
    an unwritten row cannot pass."""
    out = torch.full_like(c["q"], float("nan")) if poison else None
    lse = torch.full(c["q"].shape[:3], float("nan"), dtype=torch.float32, device=c["q"].device)
    kw = dict(max_kv_len=max_kv_len or c["max_kv_len"], page_table=c["page_table"], out=out, lse=lse)
    if mode == oracle.VERIFY:
        o, l = md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], **kw)
    else:
        o, l = md.md_draft_attn(c["q"], c["k"], c["v"], c["kv_lens"], n_sink, window, **kw)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64)


def run_gpu_indexed(c, budget, seed):
    idx, n = wl.index_lists(c["B"], c["Hkv"], c["kv_lens_np"], c["q"].shape[1], budget, seed)
    out = torch.full_like(c["q"], float("nan"))
    lse = torch.full(c["q"].shape[:3], float("nan"), dtype=torch.float32, device=c["q"].device)
    o, l = md.md_draft_attn_indexed(c["q"], c["k"], c["v"], c["kv_lens"],
                                    torch.from_numpy(idx).to(c["q"].device),
                                    torch.from_numpy(n).to(c["q"].device),
                                    max_kv_len=c["max_kv_len"], page_table=c["page_table"],
                                    out=out, lse=lse)
    torch.cuda.synchronize()
    return (o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64), idx, n)


def run_oracle(mode, c, n_sink=0, window=1):
    q, k, v = wl.to_host_bits(c["q"]), wl.to_host_bits(c["k"]), wl.to_host_bits(c["v"])
    return oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=n_sink, window=window,
                            page_table=c["page_table_np"])


def compare(got_o, got_l, ref_o, ref_l, dtype, what):
    tol = TOL[dtype]
    assert not np.isnan(got_o).any(), f"{what}: NaN in O (unwritten row or over-read)"
    assert not np.isnan(got_l).any(), f"{what}: NaN in lse"
    err = float(np.max(np.abs(got_o - ref_o))) if got_o.size else 0.0
    # lse: both sides -inf on empty rows; compare finite entries.
    fin = np.isfinite(ref_l)
    assert np.array_equal(fin, np.isfinite(got_l)), f"{what}: lse finiteness differs"
    lerr = float(np.max(np.abs(got_l[fin] - ref_l[fin]))) if fin.any() else 0.0
    say(f"  {what}: max|dO| = {err:.3e}  max|dlse| = {lerr:.3e}  (tol {tol:g})")
    assert err <= tol, f"{what}: max abs O error {err:.3e} > {tol:g}"
    assert lerr <= tol, f"{what}: max abs lse error {lerr:.3e} > {tol:g}"
    return err, lerr

