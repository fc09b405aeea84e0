"""GPU parity of the balanced verify: every workgroup streams an equal share
of all head groups' key tiles, and the groups its range boundaries cut are
merged by log-sum-exp (the split-KV identity, Sec. 2) inside the launch.

Each case checks first that the plan is the balanced one (it needs a
workspace, which the longest-first plan of the same call does not), then
compares the output with the fp64 oracle on sampled (sequence, kv head)
units -- each computed alone from the unit's own keys -- and, over every
element, with the longest-first launch of the same call (a different
decomposition: both within the dtype's tolerance of each other).  The cases
cover every compiled balanced instance (one, two and three row tiles of
bf16, both head dims, fp32), the smallest batch, a forced plan over tiny
ragged groups whose tile stream is shorter than the grid, and 16 seeded
random problems (batch, heads, head dim, q_len, lengths from below one tile
to a few thousand, paged or contiguous) forced onto the balanced plan.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2408_11049_amd as md
from gpu_util import TOL, compare, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

# name, B, q_len, Hq, Hkv, d, kv_lens, dtype, page_size, forced
CASES = [
    ("bf16_rows40_three_tiles_paged", 64, 5, 64, 8, 128,
     [4096 + (i * 397) % 2400 for i in range(64)], "bf16", 16, False),
    ("bf16_rows12_d64", 80, 3, 32, 8, 64, [4096 + (i * 211) % 3000 for i in range(80)], "bf16",
     0, False),
    ("bf16_rows4_q1", 64, 1, 32, 8, 128, [4096 + (i * 977) % 5000 for i in range(64)], "bf16",
     16, False),
    ("f32_rows16", 64, 8, 16, 8, 64, [4096 + (i * 131) % 700 for i in range(64)], "f32", 0,
     False),
    ("bf16_two_sequences", 2, 4, 256, 256, 64, [4100, 9000], "bf16", 0, False),
    ("bf16_forced_tiny_groups", 256, 2, 8, 2, 128, [2 + (i * 53) % 300 for i in range(256)],
     "bf16", 16, True),
]


def _kw(c):
    return dict(max_kv_len=c["max_kv_len"], page_table=c["page_table"])


def _run(c):
    o = torch.full_like(c["q"], float("nan"))
    lse = torch.full(c["q"].shape[:3], float("nan"), dtype=torch.float32, device=DEV)
    md.md_verify_attn(c["q"], c["k"], c["v"], c["kv_lens"], out=o, lse=lse, **_kw(c))
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_balanced_verify(case, monkeypatch):
    name, B, L, Hq, Hkv, d, lens, dtype, page, forced = case
    say(f"[balanced] {name}")
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype=dtype, page_size=page,
                     seed=zlib.crc32(name.encode()) % 1000, device=DEV,
                     S_alloc=None if page else max(lens) + 5)
    monkeypatch.setenv("MD_BALANCED", "1")
    assert md.md_workspace_bytes(c["q"], c["k"], c["v"], c["kv_lens"], **_kw(c)) == 0
    ref_o, ref_l = _run(c)  # longest first, one pass
    if forced:
        monkeypatch.setenv("MD_BALANCED", "2")
    else:
        monkeypatch.delenv("MD_BALANCED", raising=False)
    assert md.md_workspace_bytes(c["q"], c["k"], c["v"], c["kv_lens"], **_kw(c)) > 0, \
        "the call did not plan the balanced verify"
    got_o, got_l = _run(c)
    assert not np.isnan(got_o).any() and not np.isnan(got_l).any(), "unwritten output"
    tol = TOL[dtype]
    err_o = float(np.max(np.abs(got_o - ref_o)))
    err_l = float(np.max(np.abs(got_l - ref_l)))
    say(f"  {name}: against longest first max |dO| {err_o:.2e}  |dlse| {err_l:.2e}")
    assert err_o <= 2 * tol and err_l <= 2 * tol
    G = Hq // Hkv
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    units = [(0, 0), (B - 1, Hkv - 1)] + [(int(rng.integers(B)), int(rng.integers(Hkv)))
                                          for _ in range(4)]
    for b, hk in units:
        q, k, v, S = wl.gather_unit(c, b, hk)
        ro, rl = oracle.attention(oracle.VERIFY, q, k, v, S)
        compare(got_o[b: b + 1, :, hk * G: (hk + 1) * G], got_l[b: b + 1, :, hk * G: (hk + 1) * G],
                ro, rl, dtype, f"{name} unit ({b},{hk})")


def _random_case(seed):
    """A seeded problem whose head groups fill the device (at least 512 units
    of 8 or 16 kv heads), with lengths from below one tile to a few thousand."""
    rng = np.random.default_rng(1000 + seed)
    Hkv = int(rng.choice([8, 16]))
    B = int(rng.integers(512 // Hkv, 256 + 1))
    G = int(rng.choice([1, 2, 4, 8]))
    L = int(rng.integers(1, min(16, 48 // G) + 1))  # q_len <= 16, at most three row tiles
    d = int(rng.choice([64, 128]))
    lo = L
    lens = [int(x) for x in rng.integers(lo, int(rng.choice([40, 700, 2500])) + lo + 1, size=B)]
    page = int(rng.choice([0, 16]))
    return (f"random{seed}", B, L, G * Hkv, Hkv, d, lens, "bf16", page, True)


@pytest.mark.parametrize("seed", range(16))
def test_balanced_verify_random(seed, monkeypatch):
    test_balanced_verify(_random_case(seed), monkeypatch)
