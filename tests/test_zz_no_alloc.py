"""md_attn_noalloc, the entry point that allocates nothing: its output against
md_verify_attn's and md_draft_attn's (same kernels, same plans, so bit for
bit) and against the fp64 oracle, on two calls in a row, the second with a
smaller input.  Both calls split their ranges, so both use the library's
static scratch; the second reuses what the first left there."""
import numpy as np
import pytest
import torch

import oracle
import paper_2408_11049_amd as md
from gpu_util import compare, run_oracle, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(B, L, Hq, Hkv, lens, page, seed):
    return wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=128, kv_lens=lens, dtype="bf16",
                        page_size=page, seed=seed, device=DEV,
                        S_alloc=None if page else max(lens) + 7)


def _buffers(c):
    out = torch.full_like(c["q"], float("nan"))
    lse = torch.full(c["q"].shape[:3], float("nan"), dtype=torch.float32, device=DEV)
    return out, lse


def _kw(c):
    return dict(max_kv_len=c["max_kv_len"], page_table=c["page_table"])


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("mode,n_sink,window", [(oracle.VERIFY, 0, 1), (oracle.DRAFT, 16, 3000)],
                         ids=["verify", "draft"])
def test_noalloc_matches_workspace_entry(mode, n_sink, window):
    big = _case(2, 4, 16, 2, [30000, 21000], 16, 401)
    small = _case(1, 5, 8, 2, [6000], 0, 402)
    for c in (big, small):
        need = md.md_workspace_bytes(c["q"], c["k"], c["v"], c["kv_lens"], mode=mode,
                                     n_sink=n_sink, window=window, **_kw(c))
        assert 0 < need <= md.MD_NOALLOC_SCRATCH_BYTES, need  # a split plan, in the scratch
    # The entry point without allocation, twice in a row on one stream.
    got = [_buffers(big), _buffers(small)]
    torch.cuda.synchronize()
    mem0 = torch.cuda.memory_allocated(DEV)
    say(f"[no-alloc] mode {mode}: large call then small call")
    for c, (o, l) in zip((big, small), got):
        md.md_attn_noalloc(mode, c["q"], c["k"], c["v"], c["kv_lens"], n_sink, window, out=o,
                           lse=l, **_kw(c))
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated(DEV) == mem0
    # The existing entry points with their own workspaces.
    for c, (o, l) in zip((big, small), got):
        ro, rl = _buffers(c)
        if mode == oracle.VERIFY:
            md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], out=ro, lse=rl, **_kw(c))
        else:
            md.md_draft_attn(c["q"], c["k"], c["v"], c["kv_lens"], n_sink, window, out=ro,
                             lse=rl, **_kw(c))
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), ro.view(torch.int16)), "O differs from the workspace entry"
        assert torch.equal(l, rl), "lse differs from the workspace entry"
        compare(_f64(o), l.cpu().numpy().astype(np.float64),
                *run_oracle(mode, c, n_sink, window), "bf16", f"no-alloc mode {mode} B={c['B']}")


def test_noalloc_single_pass_and_refusals():
    """A plan that needs no workspace runs too; a bad mode is refused."""
    c = _case(64, 1, 8, 4, [300 + 7 * i for i in range(64)], 16, 403)
    assert md.md_workspace_bytes(c["q"], c["k"], c["v"], c["kv_lens"], **_kw(c)) == 0
    o, l = _buffers(c)
    md.md_attn_noalloc(oracle.VERIFY, c["q"], c["k"], c["v"], c["kv_lens"], out=o, lse=l, **_kw(c))
    torch.cuda.synchronize()
    compare(_f64(o), l.cpu().numpy().astype(np.float64), *run_oracle(oracle.VERIFY, c), "bf16",
            "no-alloc single pass")
    with pytest.raises(ValueError):
        md.md_attn_noalloc(md.MD_MODE_DRAFT_INDEXED, c["q"], c["k"], c["v"], c["kv_lens"],
                           out=o, lse=l, **_kw(c))


def _check_units(c, o, l, units, what):
    """Sampled (sequence, kv head) units against the fp64 oracle, one at a time."""
    G = c["Hq"] // c["Hkv"]
    for b, hk in units:
        q, k, v, S = wl.gather_unit(c, b, hk)
        ro, rl = oracle.attention(oracle.VERIFY, q, k, v, S)
        compare(_f64(o[b: b + 1, :, hk * G: (hk + 1) * G]),
                l[b: b + 1, :, hk * G: (hk + 1) * G].cpu().numpy().astype(np.float64), ro, rl,
                "bf16", f"{what} unit ({b},{hk})")


def test_noalloc_balanced_verify(monkeypatch):
    """Two balanced verify calls in a row (64 ragged sequences x 8 kv heads =
    256 head pairs, lengths past 4096: the plan that streams equal shares of
    all groups and merges the groups its ranges cut), the second smaller:
    bit for bit against md_verify_attn, and sampled units against the oracle."""
    monkeypatch.delenv("MD_BALANCED", raising=False)
    big = _case(64, 4, 32, 8, [4096 + (i * 613) % 3000 for i in range(64)], 16, 404)
    small = _case(64, 1, 32, 8, [4096 + (i * 211) % 900 for i in range(64)], 0, 405)
    for c in (big, small):
        need = md.md_workspace_bytes(c["q"], c["k"], c["v"], c["kv_lens"], **_kw(c))
        assert 0 < need <= md.MD_NOALLOC_SCRATCH_BYTES, need  # the balanced plan, in the scratch
    got = [_buffers(big), _buffers(small)]
    torch.cuda.synchronize()
    mem0 = torch.cuda.memory_allocated(DEV)
    say("[no-alloc] balanced verify: large call then small call")
    for c, (o, l) in zip((big, small), got):
        md.md_attn_noalloc(oracle.VERIFY, c["q"], c["k"], c["v"], c["kv_lens"], out=o, lse=l,
                           **_kw(c))
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated(DEV) == mem0
    for c, (o, l), name in zip((big, small), got, ("large", "small")):
        ro, rl = _buffers(c)
        md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], out=ro, lse=rl, **_kw(c))
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), ro.view(torch.int16)), f"{name}: O differs"
        assert torch.equal(l, rl), f"{name}: lse differs"
        _check_units(c, o, l, [(0, 0), (17, 5), (40, 2), (63, 7)], f"no-alloc balanced {name}")
