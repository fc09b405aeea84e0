"""GPU parity of the SnapKV-style selection (md_snapkv_votes, md_snapkv_select)
against the fp64 oracle.

- votes: element-wise against oracle_snapkv_votes with pool = 1 (raw votes);
- selection: bit-exact against oracle_snapkv_select on seeded small-integer
  votes, for which 5-tap pooling is exact in fp32 and fp64 alike, so both
  sides order (and tie) the same values;
- end to end: the GPU's kept set is valid under the oracle's fp64 pooled votes
  (no unkept prefix position outvotes a kept one beyond the fp32 error), the
  window is kept, positions ascend, counts match.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2408_11049_amd as md
from gpu_util import say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

# name, B, n_obs, Hq, Hkv, d, prompt lens, dtype, page_size
VOTES = [
    ("bf16_g4_obs32_paged", 2, 32, 8, 2, 128, [900, 2600], "bf16", 16),
    ("bf16_g8_obs32", 2, 32, 16, 2, 128, [700, 1500], "bf16", 0),
    ("f32_g2_obs8_d64", 2, 8, 4, 2, 64, [100, 45], "f32", 0),
    ("bf16_g1_obs32_long", 1, 32, 2, 2, 128, [6000], "bf16", 16),
    ("bf16_short_prompts", 3, 16, 4, 1, 64, [16, 17, 40], "bf16", 0),
    # the eight-wave instances (65-256 rows) in each address form: rows of a
    # wave in one page, pages smaller than a wave's rows, contiguous
    ("f32_g4_obs32_d64_paged", 2, 32, 8, 2, 64, [1500, 700], "f32", 16),
    ("bf16_g8_obs32_d64_paged4", 2, 32, 16, 2, 64, [1100, 2000], "bf16", 4),
    ("f32_g8_obs32_d128", 1, 32, 8, 1, 128, [1300], "f32", 0),
    ("bf16_g4_obs32_paged2", 1, 32, 8, 2, 128, [777], "bf16", 2),
    ("bf16_g3_obs29_ragged", 3, 29, 6, 2, 128, [29, 95, 3001], "bf16", 16),
]


def _case(name, B, n_obs, Hq, Hkv, d, lens, dtype, ps):
    return wl.make_case(B=B, q_len=n_obs, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens, dtype=dtype,
                        page_size=ps, seed=zlib.crc32(name.encode()) % 1000, device=DEV,
                        S_alloc=None if ps else max(lens) + 3)


@pytest.mark.parametrize("case", VOTES, ids=[c[0] for c in VOTES])
def test_votes_against_oracle(case):
    name, B, n_obs, Hq, Hkv, d, lens, dtype, ps = case
    say(f"[snapkv votes] {name}")
    c = _case(*case)
    votes = md.md_snapkv_votes(c["q"], c["k"], c["kv_lens"], max_prompt_len=c["max_kv_len"],
                               page_table=c["page_table"])
    torch.cuda.synchronize()
    got = votes.cpu().numpy().astype(np.float64)
    ref = oracle.snapkv_votes(wl.to_host_bits(c["q"]), wl.to_host_bits(c["k"]), c["kv_lens_np"],
                              pool=1, stride=votes.shape[2], page_table=c["page_table_np"])
    worst = 0.0
    for b, S in enumerate(lens):
        n = S - n_obs
        err = np.abs(got[b, :, :n] - ref[b, :, :n])
        bound = 1e-5 + 1e-4 * np.abs(ref[b, :, :n])
        worst = max(worst, float(np.max(err / bound)) if n > 0 else 0.0)
        assert np.all(err <= bound), f"{name} b={b}: max err {err.max():.3e}"
    say(f"  {name}: max err / bound = {worst:.3f}")


def _random_votes_case(seed):
    """A seeded problem across the votes kernels' paths: 16-256 rows (four or
    eight waves, one to four row tiles), both head dims and dtypes, pages
    from 1 token (per-lane addresses) to 64 or a contiguous cache, prompts
    from the bare window to a few thousand tokens (partial tiles, chunk
    edges, the masked window tiles)."""
    rng = np.random.default_rng(5000 + seed)
    combos = [(1, 8), (2, 16), (2, 32), (4, 16), (4, 29), (4, 32), (8, 16), (8, 29), (8, 32),
              (16, 16)]  # (G, n_obs): 8 to 256 rows
    G, n_obs = combos[int(rng.integers(len(combos)))]
    Hkv = int(rng.choice([1, 2]))
    d = int(rng.choice([64, 128]))
    dtype = str(rng.choice(["bf16", "bf16", "f32"]))
    page = int(rng.choice([0, 1, 2, 4, 16, 64]))
    B = int(rng.integers(1, 4))
    lens = [int(x) for x in rng.integers(n_obs, n_obs + int(rng.choice([60, 900, 4000])), size=B)]
    return (f"random{seed}", B, n_obs, G * Hkv, Hkv, d, lens, dtype, page)


@pytest.mark.parametrize("seed", range(16))
def test_votes_random(seed):
    test_votes_against_oracle(_random_votes_case(seed))


# rows, stride, n_obs, budget, pool, prompt lens (per sequence), Hkv
SELECT = [
    (3, 500, 32, 64, 5, [532, 300, 40], 2),
    (2, 4000, 32, 2049, 5, [4032, 3000], 4),
    (2, 300, 8, 40, 1, [308, 100], 1),
    (1, 70, 32, 64, 5, [32], 2),           # prompt == window: nothing to select
    (2, 1000, 32, 33, 3, [1032, 900], 2),  # one prefix position kept
    (2, 40000, 32, 2049, 5, [40032, 20000], 2),  # rows longer than the register instance
    (2, 2000, 16, 600, 7, [2016, 1500], 2),      # the widest pooling of the register instance
    (1, 900, 8, 400, 9, [908], 2),               # wider pooling: the global instance
    (2, 5000, 32, 3000, 5, [4999, 3001], 2, 1),  # all votes 0: every key ties
    (3, 1001, 16, 300, 5, [1017, 800, 499], 2),  # rows not 16-byte aligned: scalar copies
]


@pytest.mark.parametrize("case", SELECT, ids=[f"sel{i}" for i in range(len(SELECT))])
def test_select_exact(case):
    _, stride, n_obs, budget, pool, lens, Hkv = case[:7]
    hi = case[7] if len(case) > 7 else 40
    B = len(lens)
    rng = np.random.default_rng(stride * 7 + budget)
    # Small integers (heavy ties): 5-tap sums are exact, so pooled order is the
    # same in fp32 (GPU) and fp64 (oracle).
    vals = rng.integers(0, hi, size=(B, Hkv, stride)).astype(np.float32)
    idx, cnt = md.md_snapkv_select(torch.from_numpy(vals).to(DEV),
                                   torch.tensor(lens, dtype=torch.int32, device=DEV), n_obs,
                                   budget, pool=pool)
    torch.cuda.synchronize()
    idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
    pooled = np.zeros((B * Hkv, stride))
    for r in range(B * Hkv):
        n = max(lens[r // Hkv] - n_obs, 0)
        v = vals.reshape(B * Hkv, stride)[r, :n].astype(np.float64)
        pad = np.concatenate([np.zeros(pool // 2), v, np.zeros(pool // 2)])
        pooled[r, :n] = np.convolve(pad, np.ones(pool), mode="valid")[:n] / pool if n else 0
    ridx, rcnt = oracle.snapkv_select(pooled, np.repeat(np.array(lens, np.int32), Hkv), n_obs,
                                      budget)
    for r in range(B * Hkv):
        b = r // Hkv
        assert cnt[b] == rcnt[r], (r, cnt[b], rcnt[r])
        assert np.array_equal(idx.reshape(B * Hkv, budget)[r, : cnt[b]], ridx[r, : rcnt[r]]), r


# (sequence, kv head) units sampled from the 64 x 8 of the full prompt shape.
FULL_UNITS = [(0, 0), (5, 3), (13, 7), (22, 1), (37, 5), (44, 2), (51, 6), (63, 4)]


def test_full_prompt_shape_votes_and_selection():
    """Full prompt shape (Llama-3.1-8B heads, B = 64 prompts of S = 32768 in
    16-token pages, 32 observation queries, budget 2049: the paper's SnapKV
    setting, Sec. 4.4 and 5.2), on 8 sampled (sequence, kv head) units:
    raw votes element-wise against the oracle's (pool 1) to
    1e-5 + 1e-4 |oracle|, and the GPU's kept set valid under the oracle's
    pooled (pool 5) votes -- window kept, positions ascending, no dropped
    prefix position outvoting a kept one beyond the fp32 error."""
    w = wl.WORKLOADS["llama8b_b64_s32k_paged"]
    n_obs, budget = 32, 2049
    c = wl.make_case(B=w.B, q_len=n_obs, Hq=w.Hq, Hkv=w.Hkv, d=w.d, kv_lens=wl.kv_lengths(w),
                     dtype=w.dtype, page_size=w.page_size, seed=w.seed_base, device=DEV)
    votes = md.md_snapkv_votes(c["q"], c["k"], c["kv_lens"], max_prompt_len=c["max_kv_len"],
                               page_table=c["page_table"])
    idx, cnt = md.md_snapkv_select(votes, c["kv_lens"], n_obs, budget, pool=5)
    torch.cuda.synchronize()
    votes_h, idx, cnt = votes.cpu().numpy().astype(np.float64), idx.cpu().numpy(), cnt.cpu().numpy()
    assert np.all(cnt == budget)
    G = w.Hq // w.Hkv
    for b, hk in FULL_UNITS:
        q, k, _, S = wl.gather_unit(c, b, hk)
        n = int(S[0]) - n_obs
        raw = oracle.snapkv_votes(q, k, S, pool=1)[0, 0]
        err = np.abs(votes_h[b, hk, :n] - raw[:n])
        bound = 1e-5 + 1e-4 * np.abs(raw[:n])
        assert np.all(err <= bound), f"unit ({b},{hk}): vote error {err.max():.3e}"
        pooled = oracle.snapkv_votes(q, k, S, pool=5)[0, 0]
        kept = idx[b, hk]
        assert np.all(np.diff(kept) > 0) and np.array_equal(kept[-n_obs:], np.arange(n, n + n_obs))
        pre = kept[:-n_obs]
        mask = np.ones(n, bool)
        mask[pre] = False
        lo, hi = pooled[pre].min(), pooled[mask].max()
        say(f"  unit ({b},{hk}): votes max err / bound {float(np.max(err / bound)):.3f}; "
            f"min kept pooled {lo:.6e}  max dropped {hi:.6e}  (G*n_obs = {G * n_obs})")
        assert lo >= hi - 1e-4 * max(abs(hi), 1e-6), "a dropped position outvotes a kept one"
