"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.

Small cases are compared element by element over the whole output; they span
several 32-token tiles with ragged tails, every row-tile count (G*L from 4 to
64), both head dims and dtypes, contiguous and paged caches (page sizes 1 to
64), single-pass and split-KV (merged) launches, and the degenerate cases
(S = q_len, S = 1, q_len = 1, a window covering the cache, more sinks than
tokens).  The full-size workloads run in the launch configuration the bench
times and are checked on sampled (sequence, kv head) units the oracle
computes one by one, plus properties that hold at any size.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2408_11049_amd as md
from gpu_util import compare, run_gpu, run_gpu_indexed, run_oracle, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

# name, B, q_len, Hq, Hkv, d, kv_lens, dtype, page_size, n_sink, window
SMALL = [
    ("cfg_tiny_f32", 2, 4, 4, 1, 64, [256, 256], "f32", 0, 4, 32),
    ("bf16_d128_g4_ragged", 3, 4, 8, 2, 128, [300, 77, 1030], "bf16", 0, 4, 64),
    ("bf16_d64_paged16", 4, 3, 6, 3, 64, [129, 16, 17, 500], "bf16", 16, 2, 30),
    ("f32_d128", 2, 2, 4, 2, 128, [95, 160], "f32", 0, 1, 7),
    ("f32_d64_paged8", 2, 5, 8, 2, 64, [70, 33], "f32", 8, 3, 10),
    ("bf16_rows40", 2, 5, 16, 2, 128, [700, 450], "bf16", 0, 64, 200),
    ("bf16_rows64", 1, 16, 4, 1, 64, [300], "bf16", 0, 8, 40),
    ("bf16_rows12", 3, 3, 8, 2, 128, [64, 65, 63], "bf16", 0, 16, 20),
    ("bf16_q1_mha", 3, 1, 8, 8, 128, [1, 50, 33], "bf16", 0, 4, 8),
    ("f32_min_len", 2, 4, 4, 2, 64, [4, 5], "f32", 0, 1, 1),
    ("bf16_split_kv", 2, 4, 8, 1, 128, [5000, 3100], "bf16", 0, 16, 496),
    ("f32_split_kv_paged", 1, 3, 4, 1, 64, [4500], "f32", 16, 4, 100),
    ("bf16_window_covers", 2, 4, 4, 2, 128, [40, 60], "bf16", 0, 10, 100),
    ("bf16_sinks_exceed", 2, 2, 4, 2, 64, [30, 50], "bf16", 0, 64, 8),
    ("bf16_page1", 2, 3, 4, 2, 64, [37, 20], "bf16", 1, 2, 9),
    ("bf16_page64", 2, 3, 4, 2, 128, [300, 129], "bf16", 64, 2, 40),
    ("f32_rows40_split", 1, 5, 8, 1, 128, [2600], "f32", 0, 16, 100),
    ("bf16_hkv4_split_paged", 2, 5, 16, 4, 128, [4000, 2500], "bf16", 16, 16, 496),
    # 64 head pairs split into 4 chunks of >= 4096 tokens: pairs with a merge
    ("bf16_head_pairs_split4_paged", 16, 4, 16, 8, 64,
     [17000, 16500, 16900, 16400, 16800, 17000, 16600, 16950,
      16700, 16850, 16450, 16999, 16550, 16650, 16750, 16890], "bf16", 16, 16, 240),
    # one past the longest-first batch limit: head pairs, no ranking
    ("bf16_b257_pairs_no_lpt", 257, 4, 32, 8, 128, [100 + (i * 37) % 300 for i in range(257)],
     "bf16", 16, 16, 64),
    # serving-sized batch of short requests: 8192 head pairs, far more workgroups than CUs
    ("bf16_b2048_short_paged", 2048, 2, 8, 8, 64, [16 + (i * 53) % 600 for i in range(2048)],
     "bf16", 16, 4, 64),
    # one long sequence: 8 units split into 32 chunks of 4096, merged
    ("bf16_b1_s128k_32chunks", 1, 5, 32, 8, 128, [131072], "bf16", 0, 64, 1984),
]


@pytest.mark.parametrize("case", SMALL, ids=[s[0] for s in SMALL])
@pytest.mark.parametrize("mode", [oracle.VERIFY, oracle.DRAFT], ids=["verify", "draft"])
def test_small_against_oracle(case, mode):
    name, B, L, Hq, Hkv, d, lens, dtype, ps, n_sink, window = case
    say(f"[parity] {name} mode={mode} B={B} L={L} Hq={Hq} Hkv={Hkv} d={d} lens={lens} "
        f"{dtype} page={ps} sink={n_sink} window={window}")
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype=dtype, page_size=ps,
                     seed=zlib.crc32(name.encode()) % 1000, device=DEV,
                     S_alloc=None if ps else max(lens) + 5)  # NaN padding after every sequence
    go, gl = run_gpu(mode, c, n_sink, window)
    ro, rl = run_oracle(mode, c, n_sink, window)
    compare(go, gl, ro, rl, dtype, f"{name}/{'verify' if mode == 0 else 'draft'}")


# name, B, q_len, Hq, Hkv, d, kv_lens, dtype, page_size, budget, stride
INDEXED = [
    ("idx_bf16_d128_paged", 3, 4, 8, 2, 128, [900, 300, 1500], "bf16", 16, 257, 300),
    ("idx_bf16_rows20_contig", 2, 5, 8, 2, 128, [700, 2100], "bf16", 0, 400, 512),
    ("idx_f32_d64", 2, 3, 4, 1, 64, [200, 90], "f32", 0, 50, 64),
    ("idx_bf16_split", 1, 4, 8, 1, 128, [9000], "bf16", 16, 2049, 2049),
    ("idx_bf16_rows40", 2, 5, 16, 2, 128, [600, 1200], "bf16", 0, 129, 160),
    ("idx_bf16_budget_zero", 2, 4, 4, 2, 64, [50, 80], "bf16", 0, 0, 8),
    ("idx_bf16_page1_q1", 2, 1, 4, 4, 64, [70, 33], "bf16", 1, 20, 24),
]


def _lists(rng, B, Hkv, lens, q_len, budget, stride, junk=True):
    """Unique prompt positions per (b, kv head), shuffled; per-sequence budgets;
    entries past idx_len hold positions that must be ignored."""
    idx = np.zeros((B, Hkv, stride), np.int32)
    n = np.zeros(B, np.int32)
    for b in range(B):
        pool = lens[b] - q_len
        n[b] = min(budget - (b % 2) * (budget // 3), pool, stride)  # heterogeneous budgets
        for h in range(Hkv):
            idx[b, h, : n[b]] = rng.choice(pool, size=n[b], replace=False)
            if junk:
                idx[b, h, n[b]:] = rng.integers(-5, lens[b] + 5, size=stride - n[b])
    return idx, n


@pytest.mark.parametrize("case", INDEXED, ids=[s[0] for s in INDEXED])
def test_indexed_against_oracle(case):
    import paper_2408_11049_amd as md
    name, B, L, Hq, Hkv, d, lens, dtype, ps, budget, stride = case
    say(f"[parity] {name} indexed B={B} L={L} Hq={Hq} Hkv={Hkv} d={d} lens={lens} {dtype} "
        f"page={ps} budget={budget} stride={stride}")
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype=dtype, page_size=ps,
                     seed=zlib.crc32(name.encode()) % 1000, device=DEV,
                     S_alloc=None if ps else max(lens) + 5)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    idx, n = _lists(rng, B, Hkv, lens, L, budget, stride)
    # Unlisted prompt keys are poisoned: a correct kernel never reads them.
    listed = [[set(int(x) for x in idx[b, h, : n[b]]) for h in range(Hkv)] for b in range(B)]
    out = torch.full_like(c["q"], float("nan"))
    lse = torch.full(c["q"].shape[:3], float("nan"), device=DEV)
    o, l = md.md_draft_attn_indexed(c["q"], c["k"], c["v"], c["kv_lens"],
                                    torch.from_numpy(idx).to(DEV), torch.from_numpy(n).to(DEV),
                                    max_kv_len=c["max_kv_len"], page_table=c["page_table"],
                                    out=out, lse=lse)
    torch.cuda.synchronize()
    go, gl = o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64)
    q, k, v = wl.to_host_bits(c["q"]), wl.to_host_bits(c["k"]), wl.to_host_bits(c["v"])
    ro, rl = oracle.indexed(q, k, v, c["kv_lens_np"], idx, n, page_table=c["page_table_np"])
    compare(go, gl, ro, rl, dtype, f"{name}/indexed")
    # Poison every unlisted prompt key on the device and run again: identical bits.
    if ps == 0:
        k2, v2 = c["k"].clone(), c["v"].clone()
        for b in range(B):
            for h in range(Hkv):
                drop = [j for j in range(lens[b] - L) if j not in listed[b][h]]
                if drop:
                    dj = torch.tensor(drop, device=DEV)
                    k2[b, dj, h] = float("nan")
                    v2[b, dj, h] = float("nan")
        o2, l2 = md.md_draft_attn_indexed(c["q"], k2, v2, c["kv_lens"],
                                          torch.from_numpy(idx).to(DEV),
                                          torch.from_numpy(n).to(DEV), max_kv_len=c["max_kv_len"])
        torch.cuda.synchronize()
        assert torch.equal(o2, o) and torch.equal(l2, l), "an unlisted key was read"


@pytest.mark.parametrize("B,Hkv,Hq", [(64, 8, 8), (65, 8, 8), (256, 2, 8), (128, 8, 8)],
                         ids=["b64_hkv8", "b65_hkv8", "b256_hkv2", "b128_hkv8"])
@pytest.mark.parametrize("lo", [600, 5800], ids=["ragged", "even"])
def test_longest_first_dispatch(lo, B, Hkv, Hq):
    """A verify launch that takes units longest first (one chunk per unit,
    enough head pairs to fill the device, lengths up to 6000, a paged cache):
    whole output against the oracle, NaN padding included.  With lengths
    600..6000 and at most one pair per compute unit (B = 64, 65; 256 with two
    kv heads) each workgroup serves one kv head; with 5800..6000 (every length
    within 1/16 of the mean), or with two pairs per compute unit (B = 128,
    eight kv heads) and ragged lengths, the kernel pairs the heads and the
    workgroups past the pairs return without work -- including an odd batch
    (65) and two kv heads per sequence (one pair each)."""
    L, d = 4, 64
    rng = np.random.default_rng(64 + B + Hkv)
    lens = rng.integers(lo, 6001, size=B)
    lens[rng.integers(B)] = 6000
    say(f"[parity] longest-first verify: B={B} Hkv={Hkv} lens {lens.min()}..{lens.max()}")
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype="bf16", page_size=16,
                     seed=64, device=DEV)
    go, gl = run_gpu(oracle.VERIFY, c)
    ro, rl = run_oracle(oracle.VERIFY, c)
    compare(go, gl, ro, rl, "bf16", "longest-first/verify")


def test_empty_batch():
    c = wl.make_case(B=0, q_len=4, Hq=8, Hkv=2, d=128, kv_lens=[], dtype="bf16", device=DEV)
    import paper_2408_11049_amd as md
    o, l = md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], max_kv_len=4)
    o, l = md.md_draft_attn(c["q"], c["k"], c["v"], c["kv_lens"], 4, 8, max_kv_len=4)
    torch.cuda.synchronize()
    assert o.shape == (0, 4, 8, 128)


FULL = ["tiny_f32", "llama8b_b32_s8k", "llama8b_b64_ragged_paged", "llama8b_b64_s32k_paged",
        "llama8b_b256_s8k_koutlier", "llama70b_b16_s128k"]


@pytest.mark.parametrize("name", FULL)
def test_full_size(name):
    """Every output element of every workload at its full size, in the launch
    configuration the bench times: verify and draft at q_len = gamma + 1, the
    one-token draft, and the listed draft over 2049 seeded prompt positions,
    each against the fp64 oracle over the whole batch."""
    w = wl.WORKLOADS[name]
    say(f"[full] {name}: B={w.B} Hq={w.Hq} Hkv={w.Hkv} d={w.d} S={w.S or (w.S_lo, w.S_hi)} "
        f"L={w.q_len} sinks={w.n_sink} window={w.window} page={w.page_size}")
    c = wl.make_workload(w, device=DEV)
    try:
        k, v = wl.to_host_bits(c["k"]), wl.to_host_bits(c["v"])
        pt = c["page_table_np"]
        for mode, L in [(oracle.VERIFY, w.q_len), (oracle.DRAFT, w.q_len), (oracle.DRAFT, 1),
                        (oracle.INDEXED, w.q_len)]:
            cc = c
            if L != w.q_len:  # the real one-token draft step
                cc = dict(c)
                cc["q"] = c["q"][:, :1].contiguous()
                cc["q_len"] = 1
            if mode == oracle.INDEXED:  # SnapKV-sized budget (2049) of random prompt positions
                go, gl, idx, n = run_gpu_indexed(cc, budget=2049, seed=w.seed_base)
            else:
                go, gl = run_gpu(mode, cc, w.n_sink, w.window)
            q = wl.to_host_bits(cc["q"])
            if mode == oracle.INDEXED:
                ro, rl = oracle.indexed(q, k, v, c["kv_lens_np"], idx, n, page_table=pt)
            else:
                ro, rl = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=w.n_sink,
                                          window=w.window, page_table=pt)
            say(f"  {['verify', 'draft', 'listed draft'][mode]} q_len={L}: whole output compared")
            compare(go, gl, ro, rl, w.dtype, f"{name}/{['verify', 'draft', 'indexed'][mode]}/L={L}")
    finally:
        del c
        torch.cuda.empty_cache()


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged16"])
def test_head_major_layout(paged):
    """The cache given head-major ([.., kv head, token, d] under the same
    [blk, tok, head, d] view, through its strides): verify, draft and the
    listed draft against the oracle on a token-major copy of the same values,
    and an append into it lands where the strides say."""
    B, L, Hq, Hkv, d, ps = 3, 4, 8, 2, 128, 16
    lens = np.array([300, 77, 1030])
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype="bf16",
                     page_size=ps if paged else 0, seed=41, device=DEV, nan_pad=False,
                     S_alloc=None if paged else 1040)
    # Head-major storage holding the same logical values.
    k_hm = c["k"].permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    v_hm = c["v"].permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    assert k_hm.stride(2) == k_hm.shape[1] * d and k_hm.stride(1) == d
    say(f"[parity] head-major {'paged' if paged else 'contiguous'}: strides {k_hm.stride()}")
    kw = dict(max_kv_len=c["max_kv_len"], page_table=c["page_table"])
    q, kh, vh = wl.to_host_bits(c["q"]), wl.to_host_bits(c["k"]), wl.to_host_bits(c["v"])
    pt = c["page_table_np"]
    o, l = md.md_verify_attn(c["q"], k_hm, v_hm, c["kv_lens"], **kw)
    torch.cuda.synchronize()
    ro, rl = oracle.verify(q, kh, vh, c["kv_lens_np"], page_table=pt)
    compare(o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64), ro, rl,
            "bf16", "head-major/verify")
    o, l = md.md_draft_attn(c["q"], k_hm, v_hm, c["kv_lens"], 4, 64, **kw)
    torch.cuda.synchronize()
    ro, rl = oracle.draft(q, kh, vh, c["kv_lens_np"], 4, 64, page_table=pt)
    compare(o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64), ro, rl,
            "bf16", "head-major/draft")
    idx, n = wl.index_lists(B, Hkv, lens, L, 100, 41)
    o, l = md.md_draft_attn_indexed(c["q"], k_hm, v_hm, c["kv_lens"], torch.from_numpy(idx).to(DEV),
                                    torch.from_numpy(n).to(DEV), **kw)
    torch.cuda.synchronize()
    ro, rl = oracle.indexed(q, kh, vh, c["kv_lens_np"], idx, n, page_table=pt)
    compare(o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64), ro, rl,
            "bf16", "head-major/listed draft")
    # Append two tokens after position 10 of every sequence, through the strides.
    k_new, v_new = wl.new_kv_rows(B, 2, Hkv, d, "bf16", seed=42, device=DEV)
    pos0 = torch.full((B,), 10, dtype=torch.int32, device=DEV)
    md.md_kv_append(k_hm, v_hm, k_new, v_new, pos0, page_table=c["page_table"])
    torch.cuda.synchronize()
    for b in range(B):
        for i in range(2):
            j = 10 + i
            blk, tok = (int(pt[b, j // ps]), j % ps) if paged else (b, j)
            assert torch.equal(k_hm[blk, tok], k_new[b, i]) and torch.equal(v_hm[blk, tok], v_new[b, i])
