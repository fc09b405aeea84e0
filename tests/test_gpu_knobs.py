"""Every tuning override the library reads from the environment, against the
fp64 oracle: MD_PREFETCH_DEPTH (a second tile in flight: its own kernel
instances), MD_OCCUPANCY (instances compiled for one or two waves per SIMD),
MD_LPT (longest-first dispatch off, or on wherever a plan allows it),
MD_HEADS_PER_WG (one head or a head pair per workgroup), MD_FUSED_MERGE
(split ranges merged by each head group's last workgroup instead of a second
launch), MD_SLOTS_SCALE (plans for two or four workgroups per compute unit:
more and shorter chunks), MD_BALANCED and MD_BAL_WG_PER_CU (the balanced
verify off, or forced wherever allowed, with one or two workgroups per
compute unit) and MD_WAVES (eight waves per workgroup wherever the wide
instances exist).  The overrides are
read on every call, so one process sweeps them all; each setting runs the
same shapes: one to four 16-row tiles, both head dims, the streaming and
listed drafts, a split range with its merge and a longest-first batch."""
import functools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import compare, run_gpu, run_gpu_indexed, run_oracle, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

SETTINGS = [
    {}, {"MD_PREFETCH_DEPTH": "2"}, {"MD_PREFETCH_DEPTH": "3"}, {"MD_OCCUPANCY": "1"},
    {"MD_OCCUPANCY": "2"}, {"MD_LPT": "1"}, {"MD_LPT": "2"}, {"MD_HEADS_PER_WG": "1"},
    {"MD_HEADS_PER_WG": "2"}, {"MD_FUSED_MERGE": "1"}, {"MD_SLOTS_SCALE": "2"},
    {"MD_SLOTS_SCALE": "4"}, {"MD_BALANCED": "1"}, {"MD_BALANCED": "2"},
    {"MD_BALANCED": "2", "MD_BAL_WG_PER_CU": "2"}, {"MD_WAVES": "8"},
]
KNOBS = ["MD_PREFETCH_DEPTH", "MD_OCCUPANCY", "MD_LPT", "MD_HEADS_PER_WG", "MD_FUSED_MERGE",
         "MD_SLOTS_SCALE", "MD_BALANCED", "MD_BAL_WG_PER_CU", "MD_WAVES"]

# name, mode, B, L, Hq, Hkv, d, lens, page, n_sink, window, budget
CASES = [
    ("verify_rows20", oracle.VERIFY, 3, 5, 8, 2, 128, [300, 77, 1030], 16, 0, 1, 0),
    ("draft_rows20", oracle.DRAFT, 3, 5, 8, 2, 128, [300, 77, 1030], 16, 4, 64, 0),
    ("listed_rows20", oracle.INDEXED, 3, 5, 8, 2, 128, [300, 77, 1030], 16, 0, 1, 200),
    ("verify_rows16", oracle.VERIFY, 2, 4, 8, 2, 128, [513, 64], 0, 0, 1, 0),
    ("draft_rows40", oracle.DRAFT, 2, 5, 16, 2, 128, [700, 450], 0, 16, 200, 0),
    ("draft_rows20_d64", oracle.DRAFT, 3, 5, 16, 4, 64, [1500, 333, 2100], 16, 8, 900, 0),
    ("verify_rows40", oracle.VERIFY, 2, 5, 16, 2, 128, [700, 450], 16, 0, 1, 0),
    ("verify_rows64", oracle.VERIFY, 1, 16, 4, 1, 64, [300], 0, 0, 1, 0),
    ("verify_split", oracle.VERIFY, 1, 4, 8, 2, 128, [5000], 16, 0, 1, 0),
    ("verify_b64_ragged", oracle.VERIFY, 64, 4, 8, 8, 64,
     [600 + (i * 977) % 5400 for i in range(64)], 16, 0, 1, 0),
    ("verify_b64_short", oracle.VERIFY, 64, 4, 8, 8, 64,
     [100 + (i * 37) % 900 for i in range(64)], 16, 0, 1, 0),
]


@functools.lru_cache(maxsize=None)
def _case(i):
    name, mode, B, L, Hq, Hkv, d, lens, page, n_sink, window, budget = CASES[i]
    c = wl.make_case(B=B, q_len=L, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype="bf16",
                     page_size=page, seed=81 + i, device=DEV,
                     S_alloc=None if page else max(lens) + 3)
    if mode == oracle.INDEXED:
        ref = None  # the oracle runs on the lists the GPU call draws
    else:
        ref = run_oracle(mode, c, n_sink, window)
    return c, ref


@pytest.mark.parametrize("ci", range(len(CASES)), ids=[c[0] for c in CASES])
@pytest.mark.parametrize("setting", SETTINGS,
                         ids=["default"] + ["+".join("%s=%s" % kv for kv in s.items())
                                            for s in SETTINGS[1:]])
def test_setting_against_oracle(setting, ci, monkeypatch):
    for k in KNOBS:
        monkeypatch.delenv(k, raising=False)
    for k, v in setting.items():
        monkeypatch.setenv(k, v)
    name, mode, B, L, Hq, Hkv, d, lens, page, n_sink, window, budget = CASES[ci]
    say(f"[knobs] {setting or 'default'} {name}")
    c, ref = _case(ci)
    if mode == oracle.INDEXED:
        go, gl, idx, n = run_gpu_indexed(c, budget=budget, seed=90)
        q, k, v = wl.to_host_bits(c["q"]), wl.to_host_bits(c["k"]), wl.to_host_bits(c["v"])
        ro, rl = oracle.indexed(q, k, v, c["kv_lens_np"], idx, n, page_table=c["page_table_np"])
    else:
        go, gl = run_gpu(mode, c, n_sink, window)
        ro, rl = ref
    compare(go, gl, ro, rl, "bf16", f"{name} {setting or 'default'}")
