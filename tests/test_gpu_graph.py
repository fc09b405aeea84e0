"""A whole speculative step captured once in a HIP graph and replayed: the
library launches on the caller's stream and allocates nothing, so append ->
verify -> listed draft (or a draft over a gathered cache) -> greedy
acceptance -> commit records as one graph.
Each replay starts from a restored state and must match the same step run
eagerly, bit for bit (the kernels are deterministic), with eager work and
synchronisation between replays."""
import numpy as np
import pytest
import torch

import paper_2408_11049_amd as md
from gpu_util import say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_speculative_step_graph_replays_match_eager():
    B, Hq, Hkv, d, gamma, vocab, ps = 8, 32, 8, 128, 4, 32000, 16
    L = gamma + 1
    n_sink, window, budget = 16, 240, 512
    C0 = np.array([3000, 1777, 4096, 999, 2500, 3333, 64, 4000])
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=C0 + 4 * L, dtype="bf16",
                     page_size=ps, seed=31, device=DEV, nan_pad=False)
    max_kv = int(C0.max()) + 4 * L
    # State the step reads and writes, with a snapshot to restore before each run.
    state = dict(k=c["k"], v=c["v"], lens=torch.tensor(C0, dtype=torch.int32, device=DEV))
    idx0, n0 = wl.index_lists(B, Hkv, C0 + L, L, budget, 5)
    lists = torch.full((B, Hkv, budget + 64), -1, dtype=torch.int32, device=DEV)
    lists[:, :, :budget] = torch.from_numpy(idx0).to(DEV)
    state["idx"] = lists
    idx_len = torch.full((B,), budget + 64, dtype=torch.int32, device=DEV)
    snap = {k: t.clone() for k, t in state.items()}
    # Inputs and outputs, allocated once (nothing allocates inside the step).
    q = c["q"]
    k_new, v_new = wl.new_kv_rows(B, L, Hkv, d, "bf16", seed=32, device=DEV)
    logits, draft, _, _ = wl.step_logits(B, gamma, vocab, "f32", seed=33, device=DEV, ties=3)
    kv_lens = torch.empty(B, dtype=torch.int32, device=DEV)
    o_v, l_v = torch.empty_like(q), torch.empty(q.shape[:3], dtype=torch.float32, device=DEV)
    o_d, l_d = torch.empty_like(q), torch.empty(q.shape[:3], dtype=torch.float32, device=DEV)
    acc = torch.empty(B, dtype=torch.int32, device=DEV)
    tok = torch.empty((B, L), dtype=torch.int32, device=DEV)
    lib = md.load_library()
    ws_acc = torch.empty(lib.md_greedy_accept_workspace_bytes(B, gamma, vocab), dtype=torch.uint8,
                         device=DEV)
    kw = dict(max_kv_len=max_kv, page_table=c["page_table"])
    ws_v = md.md_workspace_bytes(q, state["k"], state["v"], kv_lens, mode=md.MD_MODE_VERIFY, **kw)
    ws_i = lib.md_workspace_bytes_indexed(
        md.ctypes.byref(md.make_args(q, state["k"], state["v"], kv_lens, **kw)), budget + 64)
    ws_v = torch.empty(max(ws_v, 256), dtype=torch.uint8, device=DEV)
    ws_i = torch.empty(max(int(ws_i), 256), dtype=torch.uint8, device=DEV)

    def step():
        md.md_kv_append(state["k"], state["v"], k_new, v_new, state["lens"],
                        page_table=c["page_table"], lens_out=kv_lens)
        md.md_verify_attn(q, state["k"], state["v"], kv_lens, out=o_v, lse=l_v, workspace=ws_v, **kw)
        md.md_draft_attn_indexed(q, state["k"], state["v"], kv_lens, state["idx"], idx_len,
                                 out=o_d, lse=l_d, workspace=ws_i, **kw)
        md.md_greedy_accept(logits, draft, accepted=acc, tokens=tok, want_target=False,
                            workspace=ws_acc)
        md.md_kv_commit(state["lens"], acc, L, idx=state["idx"], ring_start=budget, ring_len=64)

    def restore():
        for k_, t in state.items():
            t.copy_(snap[k_])

    def results():
        return [x.clone() for x in (o_v, l_v, o_d, l_d, acc, tok, state["lens"], state["idx"],
                                    state["k"], state["v"])]

    restore()
    step()  # eager reference (also warms every kernel up before capture)
    torch.cuda.synchronize()
    ref = results()
    restore()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        restore()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = results()
        for i, (a, b) in enumerate(zip(got, ref)):
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager step"
        # eager work between replays
        step_sum = float(got[0].float().abs().sum())
        say(f"  replay {rep}: matches the eager step (|O_verify| sum {step_sum:.1f})")


def test_gathered_draft_step_graph_replays_match_eager():
    """The same step with the draft over a gathered cache (md_kv_gather once,
    outside the graph): the step's rows are appended to both caches, the draft
    is verify attention over the gathered cache, and both lengths commit."""
    B, Hq, Hkv, d, gamma, vocab, ps, budget = 8, 32, 8, 128, 4, 32000, 16, 512
    L = gamma + 1
    C0 = np.array([3000, 1777, 4096, 999, 2500, 3333, 600, 4000])
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=C0 + L, dtype="bf16",
                     page_size=ps, seed=41, device=DEV, nan_pad=False)
    kw = dict(max_kv_len=int(C0.max()) + L, page_table=c["page_table"])
    idx, n = wl.index_lists(B, Hkv, C0 + L, L, budget, 6)
    dk = torch.zeros((B, budget + L, Hkv, d), dtype=torch.bfloat16, device=DEV)
    dv = torch.zeros_like(dk)
    lens = torch.tensor(C0, dtype=torch.int32, device=DEV)
    dlens = md.md_kv_gather(dk, dv, c["k"], c["v"], torch.from_numpy(idx).to(DEV),
                            torch.from_numpy(n).to(DEV), lens, src_page_table=c["page_table"])
    state = dict(k=c["k"], v=c["v"], lens=lens, dk=dk, dv=dv, dlens=dlens)
    snap = {k_: t.clone() for k_, t in state.items()}
    q = c["q"]
    k_new, v_new = wl.new_kv_rows(B, L, Hkv, d, "bf16", seed=42, device=DEV)
    logits, draft, _, _ = wl.step_logits(B, gamma, vocab, "f32", seed=43, device=DEV)
    kv_lens, d_kv_lens = (torch.empty(B, dtype=torch.int32, device=DEV) for _ in range(2))
    o_v, l_v = torch.empty_like(q), torch.empty(q.shape[:3], dtype=torch.float32, device=DEV)
    o_d, l_d = torch.empty_like(q), torch.empty(q.shape[:3], dtype=torch.float32, device=DEV)
    acc = torch.empty(B, dtype=torch.int32, device=DEV)
    tok = torch.empty((B, L), dtype=torch.int32, device=DEV)
    lib = md.load_library()
    ws_acc = torch.empty(lib.md_greedy_accept_workspace_bytes(B, gamma, vocab), dtype=torch.uint8,
                         device=DEV)
    kw_d = dict(max_kv_len=budget + L)

    def ws(k, v, lens_, **kw_):
        nb = md.md_workspace_bytes(q, k, v, lens_, mode=md.MD_MODE_VERIFY, **kw_)
        return torch.empty(max(nb, 256), dtype=torch.uint8, device=DEV)

    ws_v, ws_d = ws(c["k"], c["v"], kv_lens, **kw), ws(dk, dv, d_kv_lens, **kw_d)

    def step():
        md.md_kv_append(state["k"], state["v"], k_new, v_new, state["lens"],
                        page_table=c["page_table"], lens_out=kv_lens)
        md.md_kv_append(state["dk"], state["dv"], k_new, v_new, state["dlens"], lens_out=d_kv_lens)
        md.md_verify_attn(q, state["k"], state["v"], kv_lens, out=o_v, lse=l_v, workspace=ws_v, **kw)
        md.md_verify_attn(q, state["dk"], state["dv"], d_kv_lens, out=o_d, lse=l_d, workspace=ws_d,
                          **kw_d)
        md.md_greedy_accept(logits, draft, accepted=acc, tokens=tok, want_target=False,
                            workspace=ws_acc)
        md.md_kv_commit(state["lens"], acc, L)
        md.md_kv_commit(state["dlens"], acc, L)

    def restore():
        for k_, t in state.items():
            t.copy_(snap[k_])

    def results():
        return [x.clone() for x in (o_v, l_v, o_d, l_d, acc, tok)] + \
               [t.clone() for t in state.values()]

    restore()
    step()
    torch.cuda.synchronize()
    ref = results()
    restore()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        restore()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = results()
        for i, (a, b) in enumerate(zip(got, ref)):
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager step"
        say(f"  gathered replay {rep}: matches the eager step ({float(got[2].float().abs().sum()):.1f})")
