"""The split-KV merge done inside the attention launch (MD_FUSED_MERGE = 1):
when a unit's range is cut into chunks, the last workgroup of each head group
to finish merges the chunks' partials by log-sum-exp (the split-KV identity,
paper Sec. 2).  Its arrival counters live in the caller's workspace and carry
a per-call tag, so the workspace needs no clearing: these tests hand the
kernels workspaces full of garbage (including values shaped like counters of
other calls), reuse one workspace across calls of different plans, and check
every result against the fp64 oracle -- for the fused merge and for the
default second launch alike."""
import numpy as np
import pytest
import torch

import oracle
import paper_2408_11049_amd as md
from gpu_util import TOL, compare, run_oracle, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(B, L, Hq, Hkv, lens, page, seed):
    return wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=128, kv_lens=lens, dtype="bf16",
                        page_size=page, seed=seed, device=DEV,
                        S_alloc=None if page else max(lens) + 5)


def _call(mode, c, ws, n_sink=0, window=1):
    out = torch.full_like(c["q"], float("nan"))
    lse = torch.full(c["q"].shape[:3], float("nan"), dtype=torch.float32, device=DEV)
    kw = dict(max_kv_len=c["max_kv_len"], page_table=c["page_table"], out=out, lse=lse,
              workspace=ws)
    if mode == oracle.VERIFY:
        md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], **kw)
    else:
        md.md_draft_attn(c["q"], c["k"], c["v"], c["kv_lens"], n_sink, window, **kw)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def _need(mode, c, n_sink=0, window=1):
    return md.md_workspace_bytes(c["q"], c["k"], c["v"], c["kv_lens"], mode=mode, n_sink=n_sink,
                                 window=window, max_kv_len=c["max_kv_len"],
                                 page_table=c["page_table"])


@pytest.fixture(params=["fused", "launch"])
def merge(request, monkeypatch):
    monkeypatch.delenv("MD_FUSED_MERGE", raising=False)
    if request.param == "fused":
        monkeypatch.setenv("MD_FUSED_MERGE", "1")
    return request.param


@pytest.mark.parametrize("fill", ["ones", "random", "foreign_tags"])
def test_garbage_workspace(fill, merge):
    """A split verify and a split draft over a workspace that starts as
    garbage: all bits set, random bytes, or counters tagged by other calls
    with arrival counts just below the chunk count."""
    c = _case(1, 4, 8, 2, [20000], 16, 301)
    for mode, n_sink, window in ((oracle.VERIFY, 0, 1), (oracle.DRAFT, 16, 4000)):
        need = _need(mode, c, n_sink, window)
        assert need > 0, "the case must split its range"
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)
        if fill == "ones":
            ws.fill_(0xFF)
        elif fill == "random":
            g = torch.Generator(device=DEV)
            g.manual_seed(5)
            ws.copy_(torch.randint(0, 256, (need,), generator=g, device=DEV, dtype=torch.uint8))
        else:
            # (tag << 16) | arrivals, with tags no call of this process uses
            words = ws[: need // 8 * 8].view(torch.int64)
            i = torch.arange(words.numel(), device=DEV, dtype=torch.int64)
            words.copy_(((0x7FFF0000 + i) << 16) + i % 7)
        say(f"[split-merge] {merge} {fill} mode {mode} workspace {need} B")
        got = _call(mode, c, ws, n_sink, window)
        compare(*got, *run_oracle(mode, c, n_sink, window), "bf16", f"{fill} mode {mode}")


def test_one_workspace_across_plans(merge):
    """One workspace, sized for the largest, serves calls whose plans differ
    in groups and chunks, in an interleaved order, twice over."""
    cases = [
        (oracle.VERIFY, _case(1, 4, 8, 2, [20000], 16, 311), 0, 1),
        (oracle.VERIFY, _case(2, 5, 16, 2, [9000, 3000], 0, 312), 0, 1),
        (oracle.DRAFT, _case(1, 4, 8, 2, [20000], 16, 311), 16, 4000),
        (oracle.DRAFT, _case(3, 1, 8, 2, [6000, 7000, 2500], 0, 313), 4, 2000),
    ]
    needs = [_need(m, c, s, w) for m, c, s, w in cases]
    assert all(n > 0 for n in needs)
    ws = torch.empty(max(needs), dtype=torch.uint8, device=DEV)
    refs = [run_oracle(m, c, s, w) for m, c, s, w in cases]
    for rep in range(2):
        for i, (m, c, s, w) in enumerate(cases):
            say(f"[split-merge] {merge} reuse pass {rep} case {i}")
            compare(*_call(m, c, ws, s, w), *refs[i], "bf16", f"reuse {rep}/{i}")


def test_fused_matches_separate_merge(monkeypatch):
    """The in-launch merge (MD_FUSED_MERGE = 1) and the separate merge launch
    agree with the oracle and with each other to within rounding."""
    c = _case(2, 5, 32, 8, [30000, 17000], 16, 321)
    ref = run_oracle(oracle.VERIFY, c)
    monkeypatch.setenv("MD_FUSED_MERGE", "1")
    fused = _call(oracle.VERIFY, c, None)
    monkeypatch.delenv("MD_FUSED_MERGE")
    sep = _call(oracle.VERIFY, c, None)
    compare(*fused, *ref, "bf16", "fused")
    compare(*sep, *ref, "bf16", "separate")
    d = float(np.max(np.abs(fused[0] - sep[0])))
    say(f"  fused vs separate: max|dO| = {d:.3e}")
    assert d <= TOL["bf16"] / 4
