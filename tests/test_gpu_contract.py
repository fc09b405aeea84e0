"""The optional error word of md_attn_args: device-side contract violations
(a length below q_len or above max_kv_len, a page id outside the pool for a
position the call reads) are reported as bits, while memory stays in bounds
and every other output is still written.  Each violation is set up on the host
in the inputs; no kernel is made to fault."""
import numpy as np
import pytest
import torch

import paper_2408_11049_amd as md
from gpu_util import say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
B, L, Hq, Hkv, d, PS = 4, 4, 8, 2, 128, 16
LENS = [300, 77, 1030, 512]


def _case(page_size=PS, seed=5):
    return wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=LENS, dtype="bf16",
                        page_size=page_size, seed=seed, device=DEV, nan_pad=False)


def _calls(c, kv_lens, err, max_kv_len):
    """verify, draft and listed draft with the error word; returns the outputs."""
    kw = dict(max_kv_len=max_kv_len, page_table=c["page_table"], err_word=err)
    outs = [md.md_verify_attn(c["q"], c["k"], c["v"], kv_lens, **kw),
            md.md_draft_attn(c["q"], c["k"], c["v"], kv_lens, 4, 64, **kw)]
    idx, n = wl.index_lists(B, Hkv, np.array(LENS), L, 40, 3)
    outs.append(md.md_draft_attn_indexed(c["q"], c["k"], c["v"], kv_lens,
                                         torch.from_numpy(idx).to(DEV),
                                         torch.from_numpy(n).to(DEV), **kw))
    torch.cuda.synchronize()
    return outs


@pytest.mark.parametrize("page_size", [0, PS], ids=["contiguous", "paged16"])
def test_clean_inputs_leave_the_word_alone(page_size):
    say(f"[contract] clean, page_size={page_size}")
    c = _case(page_size)
    err = torch.tensor([8], dtype=torch.int32, device=DEV)  # a bit the library never sets
    outs = _calls(c, c["kv_lens"], err, c["max_kv_len"])
    assert err.item() == 8, "no violation, yet a bit was set (or the word was cleared)"
    for o, lse in outs:
        assert torch.isfinite(o.float()).all() and torch.isfinite(lse).all()


def test_short_and_long_lengths_are_reported():
    """Contiguous cache of max_kv_len rows per sequence: a length above the host
    bound is clamped to it, so every read stays in the sequence's block."""
    say("[contract] kv_lens below q_len and above max_kv_len")
    c = _case(page_size=0)
    max_kv = c["max_kv_len"]
    lens = c["kv_lens"].clone()
    lens[1] = L - 1            # shorter than the speculated tokens
    lens[0] = max_kv + 9       # above the host bound
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    outs = _calls(c, lens, err, max_kv)
    bits = err.item()
    assert bits & md.MD_ERRW_SHORT_LEN and bits & md.MD_ERRW_LONG_LEN, bits
    assert not bits & md.MD_ERRW_BAD_PAGE, bits
    for o, _ in outs:  # every row written; memory stayed in bounds
        assert not torch.isnan(o.float()).any()


@pytest.mark.parametrize("bad", [-1, 10 ** 6], ids=["negative", "past_pool"])
def test_bad_page_ids_are_reported(bad):
    say(f"[contract] page id {bad} inside a sequence's range")
    c = _case()
    pt = c["page_table"].clone()
    pt[2, 5] = bad  # sequence 2 (1030 tokens) reads page 5
    cc = dict(c)
    cc["page_table"] = pt
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    kw = dict(max_kv_len=c["max_kv_len"], page_table=pt, err_word=err)
    md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], **kw)
    torch.cuda.synchronize()
    assert err.item() == md.MD_ERRW_BAD_PAGE, err.item()
    # A page no call reads (past every length) may hold anything.
    pt2 = c["page_table"].clone()
    tail = (LENS[1] + PS - 1) // PS  # first page past sequence 1's length
    if tail < pt2.shape[1]:
        pt2[1, tail] = bad
    err2 = torch.zeros(1, dtype=torch.int32, device=DEV)
    md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], max_kv_len=c["max_kv_len"],
                      page_table=pt2, err_word=err2)
    torch.cuda.synchronize()
    assert err2.item() == 0, err2.item()


def test_listed_draft_checks_usable_entries_only():
    """A list entry that is unusable (-1) is skipped, not reported; a usable
    entry on a bad page is."""
    say("[contract] listed draft pages")
    c = _case()
    idx, n = wl.index_lists(B, Hkv, np.array(LENS), L, 40, 3)
    idx[0, 1, 3] = -1
    pt = c["page_table"].clone()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    kw = dict(max_kv_len=c["max_kv_len"], page_table=pt, err_word=err)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    md.md_draft_attn_indexed(c["q"], c["k"], c["v"], c["kv_lens"], t(idx), t(n), **kw)
    torch.cuda.synchronize()
    assert err.item() == 0, err.item()
    p = int(idx[2, 0, 7])  # a usable entry of sequence 2, kv head 0
    pt[2, p // PS] = -1
    md.md_draft_attn_indexed(c["q"], c["k"], c["v"], c["kv_lens"], t(idx), t(n), **kw)
    torch.cuda.synchronize()
    assert err.item() == md.MD_ERRW_BAD_PAGE, err.item()
