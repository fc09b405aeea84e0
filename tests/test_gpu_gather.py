"""GPU parity of md_kv_gather (a static selection gathered into a draft cache of
its own, Sec. 4.2) against the oracle (oracle/sdstep.py kv_gather): values
move unchanged, so every case is bit-exact.  Then the draft it serves: verify
attention over the gathered cache, with the step's rows appended to both
caches, against the listed draft over the full cache and the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import oracle.sdstep as sd
import paper_2408_11049_amd as md
from gpu_util import compare, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def bits(t):
    """Exact bit patterns (uint16 for bf16, uint32 for fp32), so NaN fill compares."""
    h = wl.to_host_bits(t)
    return h.view(np.uint32) if h.dtype == np.float32 else h


def _dst_cache(B, rows, Hkv, d, dtype, page_size, seed):
    """A draft cache of `rows` positions per sequence, NaN-filled, contiguous
    or paged over a shuffled pool (with spare pages)."""
    tdt = wl.torch_dtype(dtype)
    if page_size == 0:
        shape, pt = (B, rows, Hkv, d), None
    else:
        npg = -(-rows // page_size)
        P = B * npg + 3
        perm = np.random.default_rng(seed).permutation(P)
        pt = perm[: B * npg].reshape(B, npg).astype(np.int32)
        shape = (P, page_size, Hkv, d)
    k = torch.full(shape, float("nan"), dtype=tdt, device=DEV)
    v = torch.full(shape, float("nan"), dtype=tdt, device=DEV)
    return k, v, pt


def _lists(rng, B, Hkv, src_lens, stride, n):
    """Listed positions with unusable entries mixed in: -1, past src_lens."""
    idx = np.full((B, Hkv, stride), -1, np.int32)
    for b in range(B):
        for h in range(Hkv):
            m = min(stride, max(0, int(n[b])))
            pos = rng.integers(0, max(1, int(src_lens[b])), size=m)
            bad = rng.random(m) < 0.1
            pos[bad] = rng.choice([-1, -5, int(src_lens[b]), int(src_lens[b]) + 7], size=bad.sum())
            idx[b, h, :m] = pos
    return idx


# name, B, Hkv, d, dtype, src lens, src page, dst page, stride, idx_len
GATHER = [
    ("contig_to_contig_bf16", 3, 2, 128, "bf16", [300, 77, 1030], 0, 0, 64, [64, 20, 100]),
    ("paged_to_contig_bf16", 4, 8, 128, "bf16", [129, 16, 500, 2000], 16, 0, 40, [40, 0, 33, -3]),
    ("contig_to_paged_f32_d64", 2, 4, 64, "f32", [90, 200], 0, 8, 50, [50, 17]),
    ("paged_to_paged_bf16", 3, 8, 128, "bf16", [1000, 64, 333], 16, 16, 257, [257, 64, 300]),
    ("paged1_to_paged4_f32", 2, 1, 64, "f32", [37, 20], 1, 4, 9, [9, 5]),
    # shapes that are not powers of two (12 vectors per row, 3 or 6 kv heads)
    ("contig_to_paged_bf16_h3_d96", 2, 3, 96, "bf16", [200, 150], 0, 8, 30, [30, 12]),
    ("paged_to_contig_f32_h6", 2, 6, 64, "f32", [100, 64], 16, 0, 20, [20, 7]),
]


@pytest.mark.parametrize("case", GATHER, ids=[c[0] for c in GATHER])
def test_gather_matches_oracle(case):
    name, B, Hkv, d, dtype, lens, sps, dps, stride, idx_len = case
    say(f"[kv gather] {name}")
    rng = np.random.default_rng(len(name))
    src = wl.make_case(B=B, q_len=1, Hq=Hkv, Hkv=Hkv, d=d, kv_lens=lens, dtype=dtype,
                       page_size=sps, seed=len(name), device=DEV)
    src_lens = np.array(lens, np.int32)
    idx = _lists(rng, B, Hkv, src_lens, stride, idx_len)
    dk, dv, dpt = _dst_cache(B, stride, Hkv, d, dtype, dps, seed=len(name) + 1)
    dk0, dv0 = bits(dk), bits(dv)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)
    out = md.md_kv_gather(dk, dv, src["k"], src["v"], t(idx), t(idx_len), t(src_lens),
                          dst_page_table=None if dpt is None else t(dpt),
                          src_page_table=src["page_table"])
    torch.cuda.synchronize()
    kw = dict(src_page_size=sps, src_page_table=src["page_table_np"], dst_page_size=dps,
              dst_page_table=dpt)
    kref, n = sd.kv_gather(dk0, bits(src["k"]), idx, idx_len, src_lens, **kw)
    vref, _ = sd.kv_gather(dv0, bits(src["v"]), idx, idx_len, src_lens, **kw)
    assert out.cpu().tolist() == n.tolist()
    assert np.array_equal(bits(dk), kref), "K draft cache differs from the oracle"
    assert np.array_equal(bits(dv), vref), "V draft cache differs from the oracle"


def test_gather_refuses_a_short_destination():
    """A contiguous draft cache of 10 rows cannot take lists of 16: the call
    is refused before any launch (a silent drop would leave dst_lens counting
    rows that were never written), and the destination is untouched."""
    say("[kv gather] destination shorter than the lists")
    B, Hkv, d, stride, cap = 3, 2, 128, 16, 10
    src = wl.make_case(B=B, q_len=1, Hq=Hkv, Hkv=Hkv, d=d, kv_lens=[50, 60, 70], dtype="bf16",
                       seed=3, device=DEV)
    idx = np.stack([np.stack([np.arange(stride) * 3 + h for h in range(Hkv)])] * B).astype(np.int32)
    dk, dv, _ = _dst_cache(B, cap, Hkv, d, "bf16", 0, seed=4)
    before = bits(dk).copy()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)
    with pytest.raises(ValueError):
        md.md_kv_gather(dk, dv, src["k"], src["v"], t(idx), t([stride] * B), t([50, 60, 70]))
    torch.cuda.synchronize()
    assert np.array_equal(bits(dk), before)


# name, B, L, Hq, Hkv, d, committed lens, dtype, src page, dst page, budget
DRAFTS = [
    ("bf16_paged_to_contig", 4, 4, 32, 8, 128, [3000, 1500, 700, 5000], "bf16", 16, 0, 257),
    ("bf16_contig_to_paged_ragged_budget", 3, 5, 16, 2, 128, [2100, 900, 4000], "bf16", 0, 16, 1024),
    ("f32_d64_q1", 2, 1, 8, 2, 64, [600, 300], "f32", 0, 0, 129),
]


@pytest.mark.parametrize("case", DRAFTS, ids=[c[0] for c in DRAFTS])
def test_gathered_draft_matches_listed_draft(case):
    """Gather at prefill, append the step's rows to both caches, then: verify
    attention over the draft cache == the listed draft over the full cache ==
    the oracle's listed draft, to the dtype's tolerance."""
    name, B, L, Hq, Hkv, d, C, dtype, sps, dps, budget = case
    say(f"[gathered draft] {name}")
    C = np.array(C, np.int32)
    S = C + L
    full = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=S, dtype=dtype,
                        page_size=sps, seed=len(name), device=DEV)
    idx, n = wl.index_lists(B, Hkv, S, L, budget, seed=len(name))
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)
    idx_t, n_t, C_t = t(idx), t(n), t(C)
    dk, dv, dpt = _dst_cache(B, budget + L + 3, Hkv, d, dtype, dps, seed=len(name) + 2)
    dpt_t = None if dpt is None else t(dpt)
    dlen = md.md_kv_gather(dk, dv, full["k"], full["v"], idx_t, n_t, C_t, dst_page_table=dpt_t,
                           src_page_table=full["page_table"])
    # The step's rows go to both caches, as the verifier's K/V would.
    k_new, v_new = wl.new_kv_rows(B, L, Hkv, d, dtype, seed=len(name) + 3, device=DEV)
    md.md_kv_append(full["k"], full["v"], k_new, v_new, C_t, page_table=full["page_table"])
    dlens = md.md_kv_append(dk, dv, k_new, v_new, dlen, page_table=dpt_t)
    go, gl = md.md_verify_attn(full["q"], dk, dv, dlens, max_kv_len=budget + L, page_table=dpt_t)
    lo, ll = md.md_draft_attn_indexed(full["q"], full["k"], full["v"], t(S), idx_t, n_t,
                                      max_kv_len=int(S.max()), page_table=full["page_table"])
    torch.cuda.synchronize()
    host = wl.to_host_bits
    ro, rl = oracle.indexed(host(full["q"]), host(full["k"]), host(full["v"]), S, idx, n,
                            page_table=full["page_table_np"])
    f64 = lambda x: x.float().cpu().numpy().astype(np.float64)
    compare(f64(go), f64(gl), ro, rl, dtype, f"{name}: draft over the gathered cache")
    compare(f64(lo), f64(ll), ro, rl, dtype, f"{name}: listed draft")


def test_gather_bench_shape_sampled():
    """The bench shape (B = 64 prompts of 32768 tokens, 16-token pages, Hkv 8,
    d 128, budget 2049) into a contiguous draft cache: sampled rows against
    the source rows they name, bit for bit, and the lengths."""
    w = wl.WORKLOADS["llama8b_b64_s32k_paged"]
    say(f"[kv gather] {w.name} budget 2049")
    c = wl.make_workload(w, device=DEV, nan_pad=False)
    C = c["kv_lens_np"] - w.q_len
    idx, n = wl.index_lists(w.B, w.Hkv, c["kv_lens_np"], w.q_len, 2049, w.seed_base)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)
    dk, dv, _ = _dst_cache(w.B, 2049 + w.q_len, w.Hkv, w.d, "bf16", 0, seed=9)
    out = md.md_kv_gather(dk, dv, c["k"], c["v"], t(idx), t(n), t(C),
                          src_page_table=c["page_table"])
    torch.cuda.synchronize()
    assert out.cpu().tolist() == n.tolist()
    rng = np.random.default_rng(10)
    pt = c["page_table_np"]
    for _ in range(400):
        b, h = int(rng.integers(w.B)), int(rng.integers(w.Hkv))
        j = int(rng.integers(n[b]))
        p = int(idx[b, h, j])
        blk, tok = pt[b, p // w.page_size], p % w.page_size
        assert torch.equal(dk[b, j, h], c["k"][blk, tok, h]), (b, h, j)
        assert torch.equal(dv[b, j, h], c["v"][blk, tok, h]), (b, h, j)
