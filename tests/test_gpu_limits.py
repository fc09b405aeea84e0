"""One sequence longer than any workload: 2^21 + 17 tokens of Llama-3.1-8B
heads (bf16), so that element offsets inside a single sequence's K and V
pass 2^32 bytes (contiguous: the sequence block is 4 GiB per tensor; paged:
page ids pass 2^17) and the range is cut into the most chunks a verify plan
makes for eight kv heads.  Verify, draft and the one-token draft against the
fp64 oracle on two kv heads (0 and 7), each computed from that head's slice
of Q, K and V."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import compare, run_gpu, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("page", [0, 16], ids=["contiguous", "paged16"])
def test_single_sequence_past_4gib(page):
    S, L, Hq, Hkv, d, n_sink, window = (1 << 21) + 17, 5, 32, 8, 128, 64, 1984
    G = Hq // Hkv
    say(f"[limits] one sequence of {S} tokens, page {page}")
    c = wl.make_case(B=1, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=[S], dtype="bf16",
                     page_size=page, seed=97, device=DEV)
    try:
        runs = []
        for mode, q_len in [(oracle.VERIFY, L), (oracle.DRAFT, L), (oracle.DRAFT, 1)]:
            cc = c if q_len == L else dict(c, q=c["q"][:, :1].contiguous())
            go, gl = run_gpu(mode, cc, n_sink, window)
            runs.append((mode, cc, go, gl))
        for hk in (0, Hkv - 1):
            k = wl.to_host_bits(c["k"][:, :, hk:hk + 1].contiguous())
            v = wl.to_host_bits(c["v"][:, :, hk:hk + 1].contiguous())
            for mode, cc, go, gl in runs:
                q = wl.to_host_bits(cc["q"][:, :, hk * G:(hk + 1) * G].contiguous())
                ro, rl = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=n_sink,
                                          window=window, page_table=c["page_table_np"])
                name = f"{['verify', 'draft'][mode]} q_len={q.shape[1]} kv head {hk}"
                compare(go[:, :, hk * G:(hk + 1) * G], gl[:, :, hk * G:(hk + 1) * G], ro, rl,
                        "bf16", name)
    finally:
        del c
        torch.cuda.empty_cache()
