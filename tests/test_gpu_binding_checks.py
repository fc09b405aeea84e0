"""The binding refuses, before any launch, tensors the library could only see
as wild pointers: a host or other-device tensor where a device one is
expected, K/V narrower than Q, and vectors shorter than the batch.  Each call
below raises ValueError; the device is then still healthy (a final call runs)."""
import pytest
import torch

import paper_2408_11049_amd as md
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case():
    return wl.make_case(B=2, q_len=4, Hq=8, Hkv=2, d=128, kv_lens=[100, 37], dtype="bf16",
                        page_size=16, seed=5, device=DEV)


def test_attention_inputs():
    c = _case()
    kw = dict(max_kv_len=c["max_kv_len"], page_table=c["page_table"])
    with pytest.raises(ValueError, match="kv_lens is on cpu"):
        md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"].cpu(), **kw)
    with pytest.raises(ValueError, match="page_table is on cpu"):
        md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], max_kv_len=c["max_kv_len"],
                          page_table=c["page_table"].cpu())
    with pytest.raises(ValueError, match="on a GPU"):
        md.md_verify_attn(c["q"].cpu(), c["k"], c["v"], c["kv_lens"], **kw)
    with pytest.raises(ValueError, match="head_dim"):
        md.md_verify_attn(c["q"][..., :64].contiguous(), c["k"], c["v"], c["kv_lens"], **kw)
    with pytest.raises(ValueError, match="kv_lens must be"):
        md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"][:1], **kw)
    with pytest.raises(ValueError, match="lse must be"):
        md.md_draft_attn(c["q"], c["k"], c["v"], c["kv_lens"], 4, 16,
                         lse=torch.empty(2, 4, 8, dtype=torch.bfloat16, device=DEV), **kw)
    with pytest.raises(ValueError, match="o must have"):
        md.md_draft_attn(c["q"], c["k"], c["v"], c["kv_lens"], 4, 16,
                         out=torch.empty(2, 4, 8, 64, dtype=torch.bfloat16, device=DEV), **kw)
    idx, n = wl.index_lists(2, 2, c["kv_lens_np"], 4, 20, 3)
    with pytest.raises(ValueError, match="idx_len is on cpu"):
        md.md_draft_attn_indexed(c["q"], c["k"], c["v"], c["kv_lens"],
                                 torch.from_numpy(idx).to(DEV), torch.from_numpy(n), **kw)
    o, _ = md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], **kw)
    torch.cuda.synchronize()
    assert torch.isfinite(o.float()).all()


def test_step_inputs():
    c = _case()
    k_new, v_new = wl.new_kv_rows(2, 4, 2, 128, "bf16", seed=6, device=DEV)
    pos0 = torch.tensor([96, 33], dtype=torch.int32, device=DEV)
    with pytest.raises(ValueError, match="pos0 is on cpu"):
        md.md_kv_append(c["k"], c["v"], k_new, v_new, pos0.cpu(), page_table=c["page_table"])
    with pytest.raises(ValueError, match="k_new is on cpu"):
        md.md_kv_append(c["k"], c["v"], k_new.cpu(), v_new, pos0, page_table=c["page_table"])
    logits, draft, _, _ = wl.step_logits(2, 3, 1000, "f32", seed=7, device=DEV)
    with pytest.raises(ValueError, match="draft is on cpu"):
        md.md_greedy_accept(logits, draft.cpu())
    acc, _, _ = md.md_greedy_accept(logits, draft)
    lens = pos0.clone()
    with pytest.raises(ValueError, match="accepted is on cpu"):
        md.md_kv_commit(lens, acc.cpu(), 4)
    with pytest.raises(ValueError, match="accepted must be"):
        md.md_kv_commit(lens, acc[:1], 4)
    with pytest.raises(ValueError, match="on a GPU"):
        md.md_streaming_list(pos0.cpu(), 2, 4, 16)
    idx, n = md.md_streaming_list(pos0, 2, 4, 16)
    dk = torch.zeros((2, 24, 2, 128), dtype=torch.bfloat16, device=DEV)
    dv = torch.zeros_like(dk)
    with pytest.raises(ValueError, match="src_lens is on cpu"):
        md.md_kv_gather(dk, dv, c["k"], c["v"], idx, n, pos0.cpu(), src_page_table=c["page_table"])
    md.md_kv_commit(lens, acc, 4)
    torch.cuda.synchronize()


def test_snapkv_and_merge_inputs():
    c = _case()
    q_obs = c["q"][:, :4].contiguous()
    with pytest.raises(ValueError, match="prompt_lens is on cpu"):
        md.md_snapkv_votes(q_obs, c["k"], c["kv_lens"].cpu(), max_prompt_len=c["max_kv_len"],
                           page_table=c["page_table"])
    votes = md.md_snapkv_votes(q_obs, c["k"], c["kv_lens"], max_prompt_len=c["max_kv_len"],
                               page_table=c["page_table"])
    with pytest.raises(ValueError, match="prompt_lens is on cpu"):
        md.md_snapkv_select(votes, c["kv_lens"].cpu(), 4, 16)
    parts = torch.zeros((2, 8, 128), device=DEV)
    with pytest.raises(ValueError, match="lse_parts is on cpu"):
        md.md_merge_lse(parts, torch.zeros((2, 8)))
    with pytest.raises(ValueError, match="lse_parts must be"):
        md.md_merge_lse(parts, torch.zeros((2, 7), device=DEV))
    torch.cuda.synchronize()
