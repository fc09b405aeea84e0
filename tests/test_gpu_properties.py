"""GPU properties that need no oracle (they hold at any size), and the
public md_merge_lse against the oracle's merge."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2408_11049_amd as md
from gpu_util import TOL, run_gpu, say
from paper_2408_11049_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(**kw):
    base = dict(B=2, q_len=4, Hq=8, Hkv=2, d=128, kv_lens=[200, 333], dtype="bf16", seed=21,
                device=DEV)
    base.update(kw)
    return wl.make_case(**base)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("mode", [0, 1])
def test_constant_v_gives_constant_o(dtype, mode):
    """V == 1 everywhere visible: every softmax row sums to one, so O == 1."""
    c = _case(dtype=dtype, kv_lens=[1500, 97], S_alloc=1500)
    c["v"].fill_(1.0)
    go, gl = run_gpu(mode, c, 4, 50)
    err = float(np.max(np.abs(go - 1.0)))
    say(f"  constant V ({dtype}, mode {mode}): max|O-1| = {err:.3e}")
    assert err <= (1e-6 if dtype == "f32" else 0.0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_single_key_returns_v(dtype):
    """S_b = 1 and q_len = 1: O is V[b, 0] exactly."""
    c = _case(dtype=dtype, q_len=1, kv_lens=[1, 1, 1], B=3)
    for mode in (0, 1):
        go, gl = run_gpu(mode, c, 1, 1)
        want = c["v"][:, 0].float().cpu().numpy().repeat(4, axis=1)  # kv head h // 4
        assert np.array_equal(go[:, 0], want)


def test_causal_rows_ignore_later_tokens():
    """Changing K/V after position p_i leaves row i bit-for-bit unchanged."""
    S, L = 900, 5
    c = _case(q_len=L, kv_lens=[S, S])
    o0, l0 = run_gpu(0, c)
    for i in range(L - 1):
        p = S - L + i
        c2 = dict(c)
        c2["k"] = c["k"].clone()
        c2["v"] = c["v"].clone()
        c2["k"][:, p + 1:S] += 1.5
        c2["v"][:, p + 1:S] -= 0.75
        o1, l1 = run_gpu(0, c2)
        assert np.array_equal(o1[:, : i + 1], o0[:, : i + 1]), f"row {i} changed"
        assert np.array_equal(l1[:, : i + 1], l0[:, : i + 1])
        assert not np.array_equal(o1[:, i + 1], o0[:, i + 1])


def test_draft_never_reads_evicted_tokens():
    """Draft: NaN in every token outside sinks and windows changes nothing."""
    S, L, n_sink, W = 3000, 4, 16, 200
    c = _case(q_len=L, kv_lens=[S, S - 7])
    o0, l0 = run_gpu(1, c, n_sink, W)
    c2 = dict(c)
    c2["k"], c2["v"] = c["k"].clone(), c["v"].clone()
    for b, Sb in enumerate([S, S - 7]):
        lo = Sb - L - W + 1
        c2["k"][b, n_sink:lo] = float("nan")
        c2["v"][b, n_sink:lo] = float("nan")
    o1, l1 = run_gpu(1, c2, n_sink, W)
    assert np.array_equal(o0, o1) and np.array_equal(l0, l1)


def test_paged_equals_contiguous_bitwise():
    """The same logical cache, paged through a shuffled table, gives identical bits."""
    lens = [700, 129, 1025]
    cp = _case(kv_lens=lens, B=3, page_size=16)
    pt = cp["page_table_np"]
    S_alloc = max(lens)
    kc = torch.zeros((3, S_alloc, 2, 128), dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    for b, S in enumerate(lens):
        npg = math.ceil(S / 16)
        pages = torch.as_tensor(pt[b, :npg], dtype=torch.int64, device=DEV)
        kc[b, :S] = cp["k"].index_select(0, pages).reshape(npg * 16, 2, 128)[:S]
        vc[b, :S] = cp["v"].index_select(0, pages).reshape(npg * 16, 2, 128)[:S]
    cc = dict(cp, k=kc, v=vc, page_table=None, page_table_np=None, page_size=0)
    for mode in (0, 1):
        op, lp = run_gpu(mode, cp, 4, 100)
        oc, lc = run_gpu(mode, cc, 4, 100)
        assert np.array_equal(op, oc) and np.array_equal(lp, lc)


def test_batch_permutation_equivariance():
    """Permuting the sequences permutes the outputs (bit for bit)."""
    c = _case(kv_lens=[100, 2000, 640, 31], B=4, S_alloc=2000)
    perm = [2, 0, 3, 1]
    cp = dict(c, q=c["q"][perm].contiguous(), k=c["k"][perm].contiguous(),
              v=c["v"][perm].contiguous(), kv_lens=c["kv_lens"][perm].contiguous(),
              kv_lens_np=c["kv_lens_np"][perm])
    for mode in (0, 1):
        o, l = run_gpu(mode, c, 8, 64)
        op, lp = run_gpu(mode, cp, 8, 64)
        assert np.array_equal(op, o[perm]) and np.array_equal(lp, l[perm])


@pytest.mark.parametrize("n_parts", [7, 150], ids=["7_parts", "150_parts"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_merge_lse_against_oracle(d, out_dtype, n_parts):
    """md_merge_lse == oracle merge, with empty (-inf) parts holding NaN O and
    rows where every part is empty; 150 parts take each lane of the row's
    wave through the part list more than once."""
    rng = np.random.default_rng(d + n_parts)
    n_rows = 333
    o_parts = rng.standard_normal((n_parts, n_rows, d)).astype(np.float32)
    lse_parts = (rng.standard_normal((n_parts, n_rows)) * 4).astype(np.float32)
    empty = rng.random((n_parts, n_rows)) < 0.3
    empty[:, :5] = True  # five rows with nothing at all
    lse_parts[empty] = -np.inf
    o_parts[empty] = np.nan
    o, l = md.md_merge_lse(torch.from_numpy(o_parts).to(DEV), torch.from_numpy(lse_parts).to(DEV),
                           out_dtype=out_dtype)
    torch.cuda.synchronize()
    ro, rl = oracle.merge_lse(o_parts.astype(np.float64), lse_parts.astype(np.float64))
    go = o.float().cpu().numpy()
    gl = l.cpu().numpy()
    tol = 1e-5 if out_dtype == torch.float32 else 2e-2
    assert not np.isnan(go).any()
    assert np.max(np.abs(go - ro)) <= tol
    fin = np.isfinite(rl)
    assert np.array_equal(fin, np.isfinite(gl))
    assert np.all(gl[~fin] == -np.inf) and np.all(go[:5] == 0)
    assert np.max(np.abs(gl[fin] - rl[fin])) <= 1e-5
