"""The C ABI promises thread-safe, re-entrant calls on independent streams:
two host threads drive verify and the listed draft on two streams at the
same time, over shared read-only caches, and each result equals the same
call made alone (bit for bit: the kernels are deterministic)."""
import threading

import numpy as np
import pytest
import torch

import paper_2408_11049_amd as md
from gpu_util import say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_two_threads_two_streams():
    B, L, Hq, Hkv, d = 16, 5, 32, 8, 128
    lens = np.full(B, 8192)
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype="bf16", page_size=16,
                     seed=51, device=DEV, nan_pad=False)
    idx, n = wl.index_lists(B, Hkv, lens, L, 1024, 51)
    idx_t, n_t = torch.from_numpy(idx).to(DEV), torch.from_numpy(n).to(DEV)
    kw = dict(max_kv_len=8192, page_table=c["page_table"])

    def verify(stream, out, lse):
        md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], out=out, lse=lse, stream=stream, **kw)

    def draft(stream, out, lse):
        md.md_draft_attn_indexed(c["q"], c["k"], c["v"], c["kv_lens"], idx_t, n_t, out=out, lse=lse,
                                 stream=stream, **kw)

    def buffers():
        return torch.empty_like(c["q"]), torch.empty(c["q"].shape[:3], dtype=torch.float32, device=DEV)

    ref_v, ref_d = buffers(), buffers()
    verify(torch.cuda.current_stream(), *ref_v)
    draft(torch.cuda.current_stream(), *ref_d)
    torch.cuda.synchronize()
    for rep in range(3):
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        got_v, got_d = buffers(), buffers()
        torch.cuda.synchronize()
        errors = []

        def run(fn, stream, bufs):
            try:
                for _ in range(4):
                    fn(stream, *bufs)
                stream.synchronize()
            except Exception as e:  # surfaced below
                errors.append(e)

        t1 = threading.Thread(target=run, args=(verify, s1, got_v))
        t2 = threading.Thread(target=run, args=(draft, s2, got_d))
        t1.start(); t2.start(); t1.join(); t2.join()
        torch.cuda.synchronize()
        assert not errors, errors
        for a, b in zip(got_v + got_d, ref_v + ref_d):
            assert torch.equal(a, b), f"round {rep}: a concurrent result differs"
        say(f"  round {rep}: concurrent verify and listed draft match the serial results")
