"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each ``pin_*`` takes an optional oracle library handle (``lib=None`` is the
real build) and raises AssertionError on a mismatch.  ``test_oracle_pins.py``
runs them on the real oracle; ``test_oracle_mutants.py`` runs them on builds
of ``oracle.c`` with a planted mistake and requires every mutant to fail at
least one pin.

What each pin rests on:
  sdpa_*      torch's scaled_dot_product_attention in float64, with torch's own
              bottom-right causal bias (``causal_lower_right``): a library
              routine for the verify definition (Sec. 3.1, gamma+1 positions
              verified against the full cache).
  draft_*     the same library routine on an explicitly sliced StreamingLLM
              cache, sinks K[0:n_sink] plus the window K[p-W+1 : p+1]
              (Sec. 5.1 setup; Eq. 3 budget K = n_sink + W).
  mp_*        50-digit mpmath evaluation of the softmax on tiny inputs.
  closed forms: single key, all keys equal, rows summing to one.
  invariances: causality, draft key set, GQA == repeated-KV MHA, paging.
  merge_*     attention over disjoint key sets (library SDPA + logsumexp)
              merged by the oracle equals attention over the union (the
              split-KV identity behind Flash-Decoding, Sec. 2).
"""
import math

import mpmath
import numpy as np
import torch
import torch.nn.functional as F
from torch.nn.attention.bias import causal_lower_right

import oracle
from paper_2408_11049_amd import workloads as wl

TOL = 1e-12


def f64(x):
    return oracle.bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, np.float64)


def host_case(**kw):
    c = wl.make_case(device="cpu", **kw)
    return c, wl.to_host_bits(c["q"]), wl.to_host_bits(c["k"]), wl.to_host_bits(c["v"])


def sdpa_rows(q, k, v, scale, mask):
    """q [H, Lq, d], k/v [H, Lk, d] float64 tensors; mask bool [Lq, Lk] or a torch bias."""
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)
    s = (q @ k.transpose(-1, -2)) * scale
    if hasattr(mask, "_materialize"):  # torch's CausalBias is a Tensor subclass
        mask = mask._materialize()
    lse = torch.logsumexp(s.masked_fill(~mask, float("-inf")), dim=-1)
    return o, lse


def sdpa_verify(q, k, v, kv_lens, scale):
    """Library reference for verify, contiguous float64 arrays."""
    B, q_len, Hq, d = q.shape
    G = Hq // k.shape[2]
    o = np.zeros(q.shape)
    lse = np.zeros(q.shape[:3])
    for b in range(B):
        S = int(kv_lens[b])
        qt = torch.from_numpy(q[b]).permute(1, 0, 2)
        kt = torch.from_numpy(k[b, :S]).permute(1, 0, 2).repeat_interleave(G, 0)
        vt = torch.from_numpy(v[b, :S]).permute(1, 0, 2).repeat_interleave(G, 0)
        ot, lt = sdpa_rows(qt, kt, vt, scale, causal_lower_right(q_len, S))
        o[b] = ot.permute(1, 0, 2).numpy()
        lse[b] = lt.T.numpy()
    return o, lse


def sdpa_draft(q, k, v, kv_lens, n_sink, window, scale):
    """Library reference for the StreamingLLM draft: each query row attends,
    unmasked, to its explicitly sliced cache [K[0:n_sink] ; K[p-W+1 : p+1]]."""
    B, q_len, Hq, d = q.shape
    G = Hq // k.shape[2]
    o = np.zeros(q.shape)
    lse = np.zeros(q.shape[:3])
    for b in range(B):
        S = int(kv_lens[b])
        for i in range(q_len):
            p = S - q_len + i
            w0 = max(0, p - window + 1)
            sinks = list(range(0, min(n_sink, w0)))
            idx = sinks + list(range(w0, p + 1))
            qt = torch.from_numpy(q[b, i]).unsqueeze(1)                       # [Hq, 1, d]
            kt = torch.from_numpy(k[b, idx]).permute(1, 0, 2).repeat_interleave(G, 0)
            vt = torch.from_numpy(v[b, idx]).permute(1, 0, 2).repeat_interleave(G, 0)
            ot, lt = sdpa_rows(qt, kt, vt, scale, torch.ones(1, len(idx), dtype=torch.bool))
            o[b, i] = ot[:, 0].numpy()
            lse[b, i] = lt[:, 0].numpy()
    return o, lse


def close(a, b, tol=TOL, what=""):
    err = float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) if np.size(a) else 0.0
    assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.1e}"


# ----------------------------------------------------------------------------- verify

def pin_sdpa_verify(lib=None):
    """Verify == library SDPA with bottom-right causal bias; GQA, ragged lengths, both dtypes."""
    for dtype, d, Hq, Hkv, q_len, lens in [("f32", 64, 4, 1, 4, [37, 5]),
                                             ("bf16", 32, 6, 2, 3, [9, 16, 3]),
                                             ("bf16", 16, 2, 2, 1, [1, 7])]:
        c, q, k, v = host_case(B=len(lens), q_len=q_len, Hq=Hq, Hkv=Hkv, d=d, kv_lens=lens,
                               dtype=dtype, seed=11, S_alloc=max(lens) + 3)
        scale = 1.0 / math.sqrt(d)
        o, lse = oracle.verify(q, k, v, c["kv_lens_np"], lib=lib)
        ro, rl = sdpa_verify(f64(q), f64(k), f64(v), c["kv_lens_np"], scale)
        close(o, ro, what=f"verify O {dtype}")
        close(lse, rl, what=f"verify lse {dtype}")


def pin_sdpa_verify_scale(lib=None):
    """An explicit softmax scale is applied to the scores (not the default 1/sqrt(d))."""
    c, q, k, v = host_case(B=1, q_len=2, Hq=2, Hkv=1, d=16, kv_lens=[11], dtype="f32", seed=3)
    o, lse = oracle.verify(q, k, v, c["kv_lens_np"], scale=0.37, lib=lib)
    ro, rl = sdpa_verify(f64(q), f64(k), f64(v), c["kv_lens_np"], 0.37)
    close(o, ro, what="scaled O")
    close(lse, rl, what="scaled lse")


def pin_mpmath(lib=None):
    """50-digit brute force of one tiny verify row set and one draft row set."""
    mpmath.mp.dps = 50
    c, q, k, v = host_case(B=1, q_len=3, Hq=2, Hkv=1, d=4, kv_lens=[9], dtype="f32", seed=5)
    Q, K, V = f64(q), f64(k), f64(v)
    scale = mpmath.mpf(1) / mpmath.sqrt(4)
    for mode, n_sink, W in [(oracle.VERIFY, 0, 1), (oracle.DRAFT, 2, 3)]:
        o, lse = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=n_sink, window=W, lib=lib)
        for i in range(3):
            p = 9 - 3 + i
            J = [j for j in range(p + 1)
                 if mode == oracle.VERIFY or j < n_sink or j >= p - W + 1]
            for h in range(2):
                s = [scale * mpmath.fsum(mpmath.mpf(Q[0, i, h, c_]) * mpmath.mpf(K[0, j, 0, c_])
                                         for c_ in range(4)) for j in J]
                Z = mpmath.fsum(mpmath.exp(x) for x in s)
                for c_ in range(4):
                    ref = mpmath.fsum(mpmath.exp(x) * mpmath.mpf(V[0, j, 0, c_])
                                      for x, j in zip(s, J)) / Z
                    assert abs(float(ref) - o[0, i, h, c_]) <= TOL, "mpmath O"
                assert abs(float(mpmath.log(Z)) - lse[0, i, h]) <= TOL, "mpmath lse"


def pin_probs_rows_sum_to_one(lib=None):
    """Every explicit softmax row sums to 1 and O is exactly that row applied to V."""
    c, q, k, v = host_case(B=2, q_len=4, Hq=4, Hkv=2, d=16, kv_lens=[12, 30], dtype="bf16", seed=9,
                           S_alloc=30)
    for mode in (oracle.VERIFY, oracle.DRAFT):
        o, lse, P = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=2, window=5,
                                     want_probs=True, probs_len=30, lib=lib)
        close(P.sum(-1), np.ones(P.shape[:3]), tol=1e-13, what="row sums")
        # O is the P-weighted sum of V rows.
        V = f64(v)
        for b in range(2):
            for h in range(4):
                ref = np.einsum("ij,jd->id", P[b, :, h, : c["kv_lens_np"][b]],
                                V[b, : c["kv_lens_np"][b], h // 2])
                close(o[b, :, h], ref, what="O = P V")


def pin_single_key(lib=None):
    """S_b = 1, q_len = 1: the only key has weight 1, so O = V[b, 0] exactly."""
    c, q, k, v = host_case(B=3, q_len=1, Hq=4, Hkv=2, d=8, kv_lens=[1, 1, 1], dtype="bf16", seed=2)
    for mode in (oracle.VERIFY, oracle.DRAFT):
        o, lse = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=1, window=1, lib=lib)
        V = f64(v)
        for h in range(4):
            assert np.array_equal(o[:, 0, h], V[:, 0, h // 2]), "O != V[0]"
        s = np.einsum("bhd,bhd->bh", f64(q)[:, 0], np.repeat(f64(k)[:, 0], 2, axis=1)) / math.sqrt(8)
        close(lse[:, 0], s, tol=1e-14, what="lse = single score")


def pin_equal_keys(lib=None):
    """All keys identical: softmax is uniform over the visible set, so O is the
    mean of the visible V rows and lse = s + ln|J|."""
    B, q_len, S, d = 1, 3, 20, 8
    c, q, k, v = host_case(B=B, q_len=q_len, Hq=1, Hkv=1, d=d, kv_lens=[S], dtype="f32", seed=4)
    k = np.repeat(k[:, :1], S, axis=1).copy()
    V = f64(v)
    for mode, n_sink, W in [(oracle.VERIFY, 0, 1), (oracle.DRAFT, 3, 4)]:
        o, lse = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=n_sink, window=W, lib=lib)
        for i in range(q_len):
            p = S - q_len + i
            if mode == oracle.VERIFY:
                J = np.arange(p + 1)
            else:
                J = np.concatenate([np.arange(n_sink), np.arange(p - W + 1, p + 1)])
            close(o[0, i, 0], V[0, J, 0].mean(axis=0), tol=1e-13, what="uniform mean")
            s = float(f64(q)[0, i, 0] @ f64(k)[0, 0, 0]) / math.sqrt(d)
            close(lse[0, i, 0], s + math.log(len(J)), tol=1e-12, what="uniform lse")


def pin_causal_invariance(lib=None):
    """Changing keys/values after position p_i leaves row i unchanged, and changing them at
    or before p_i does change it (causality among the speculated tokens)."""
    S, q_len = 24, 5
    c, q, k, v = host_case(B=1, q_len=q_len, Hq=2, Hkv=1, d=16, kv_lens=[S], dtype="f32", seed=6)
    o0, l0 = oracle.verify(q, k, v, c["kv_lens_np"], lib=lib)
    for i in range(q_len - 1):
        p = S - q_len + i
        k2, v2 = k.copy(), v.copy()
        k2[0, p + 1:] += 3.0
        v2[0, p + 1:] -= 2.0
        o1, l1 = oracle.verify(q, k2, v2, c["kv_lens_np"], lib=lib)
        assert np.array_equal(o1[0, : i + 1], o0[0, : i + 1]), "row changed by a later token"
        assert np.array_equal(l1[0, : i + 1], l0[0, : i + 1])
        assert not np.allclose(o1[0, i + 1], o0[0, i + 1]), "later row ignores its own token"


def pin_draft_equals_verify_when_budget_covers(lib=None):
    """n_sink + W >= S_b: the draft set is the whole causal prefix."""
    c, q, k, v = host_case(B=2, q_len=4, Hq=4, Hkv=2, d=16, kv_lens=[10, 17], dtype="bf16", seed=8,
                           S_alloc=17)
    ov, lv = oracle.verify(q, k, v, c["kv_lens_np"], lib=lib)
    for n_sink, W in [(0, 17), (5, 12), (17, 1), (20, 30)]:
        od, ld = oracle.draft(q, k, v, c["kv_lens_np"], n_sink, W, lib=lib)
        assert np.array_equal(od, ov) and np.array_equal(ld, lv), (n_sink, W)


def pin_sdpa_draft(lib=None):
    """Draft == library SDPA over the explicitly sliced StreamingLLM cache, per query row."""
    for dtype, lens, q_len, n_sink, W in [("bf16", [40, 23], 4, 4, 8), ("f32", [64], 1, 4, 32),
                                          ("bf16", [19], 3, 0, 5), ("f32", [12], 5, 9, 2)]:
        c, q, k, v = host_case(B=len(lens), q_len=q_len, Hq=4, Hkv=2, d=16, kv_lens=lens,
                               dtype=dtype, seed=13, S_alloc=max(lens))
        o, lse = oracle.draft(q, k, v, c["kv_lens_np"], n_sink, W, lib=lib)
        ro, rl = sdpa_draft(f64(q), f64(k), f64(v), c["kv_lens_np"], n_sink, W, 0.25)
        close(o, ro, what=f"draft O {dtype} {n_sink}+{W}")
        close(lse, rl, what=f"draft lse {dtype} {n_sink}+{W}")


def pin_draft_ignores_evicted(lib=None):
    """Draft: keys outside sinks and window may hold anything, even NaN."""
    S, q_len, n_sink, W = 40, 3, 3, 6
    c, q, k, v = host_case(B=1, q_len=q_len, Hq=2, Hkv=1, d=8, kv_lens=[S], dtype="f32", seed=10)
    o0, l0 = oracle.draft(q, k, v, c["kv_lens_np"], n_sink, W, lib=lib)
    k2, v2 = k.copy(), v.copy()
    lo = S - q_len - W + 1            # first key any row's window reaches
    k2[0, n_sink:lo] = np.nan
    v2[0, n_sink:lo] = np.nan
    o1, l1 = oracle.draft(q, k2, v2, c["kv_lens_np"], n_sink, W, lib=lib)
    assert np.array_equal(o0, o1) and np.array_equal(l0, l1)


def pin_gqa_equals_repeated_mha(lib=None):
    """GQA: query head h reads kv head h // G; repeating K/V G times as MHA is identical."""
    c, q, k, v = host_case(B=2, q_len=2, Hq=6, Hkv=2, d=8, kv_lens=[7, 13], dtype="bf16", seed=12,
                           S_alloc=13)
    o, lse = oracle.verify(q, k, v, c["kv_lens_np"], lib=lib)
    kr = np.repeat(k, 3, axis=2).copy()
    vr = np.repeat(v, 3, axis=2).copy()
    o2, l2 = oracle.verify(q, kr, vr, c["kv_lens_np"], lib=lib)
    assert np.array_equal(o, o2) and np.array_equal(lse, l2)


def pin_paged_equals_contiguous(lib=None):
    """A paged cache holding the same logical tokens gives the same result,
    whatever page order the table uses."""
    lens = [37, 16, 5]
    c, q, k, v = host_case(B=3, q_len=4, Hq=4, Hkv=2, d=16, kv_lens=lens, dtype="bf16", seed=14,
                           page_size=8)
    pt = c["page_table_np"]
    kc = np.zeros((3, 40, 2, 16), dtype=np.uint16)
    vc = np.zeros_like(kc)
    for b, S in enumerate(lens):
        for j in range(S):
            kc[b, j] = k[pt[b, j // 8], j % 8]
            vc[b, j] = v[pt[b, j // 8], j % 8]
    for mode in (oracle.VERIFY, oracle.DRAFT):
        op, lp = oracle.attention(mode, q, k, v, c["kv_lens_np"], n_sink=2, window=6,
                                  page_table=pt, lib=lib)
        oc, lc = oracle.attention(mode, q, kc, vc, c["kv_lens_np"], n_sink=2, window=6, lib=lib)
        assert np.array_equal(op, oc) and np.array_equal(lp, lc)
        # Permute the physical pages and the table with them.
        perm = np.random.default_rng(1).permutation(k.shape[0])
        inv = np.argsort(perm)
        k2, v2 = k[perm].copy(), v[perm].copy()
        pt2 = np.where(pt >= 0, inv[np.maximum(pt, 0)], -1).astype(np.int32)
        o2, l2 = oracle.attention(mode, q, k2, v2, c["kv_lens_np"], n_sink=2, window=6,
                                  page_table=pt2, lib=lib)
        assert np.array_equal(op, o2) and np.array_equal(lp, l2)


def pin_bf16_decode(lib=None):
    """bf16 bit patterns widen exactly: 0x3F80 = 1, 0xC040 = -3, 0x3F81 = 1 + 2^-7, 0x0001 = 2^-133."""
    bits = np.array([0x3F80, 0xC040, 0x3F81, 0x0001], dtype=np.uint16)
    want = np.array([1.0, -3.0, 1.0 + 2.0 ** -7, 2.0 ** -133])
    q = np.full((1, 1, 1, 4), 0x3F80, dtype=np.uint16)
    k = np.full((1, 1, 1, 4), 0x3F80, dtype=np.uint16)
    v = bits.reshape(1, 1, 1, 4)
    o, lse = oracle.verify(q, k, v, np.array([1], np.int32), lib=lib)
    assert np.array_equal(o.reshape(-1), want), o
    assert lse[0, 0, 0] == 4 * 0.5  # score = scale * sum(1*1) = 4 / sqrt(4)


# ----------------------------------------------------------------------------- indexed draft

def _index_lists(rng, B, Hkv, lens, q_len, budget, stride):
    """Seeded unique prompt positions per (b, kv head), shuffled, padded with -7."""
    idx = np.full((B, Hkv, stride), -7, dtype=np.int32)
    n = np.zeros(B, dtype=np.int32)
    for b in range(B):
        pool = lens[b] - q_len
        n[b] = min(budget, pool)
        for h in range(Hkv):
            idx[b, h, : n[b]] = rng.choice(pool, size=n[b], replace=False)
    return idx, n


def pin_indexed_full_list_is_verify(lib=None):
    """Listing every prompt position gives exactly the verify result."""
    lens = [30, 19]
    c, q, k, v = host_case(B=2, q_len=3, Hq=4, Hkv=2, d=16, kv_lens=lens, dtype="bf16", seed=31,
                           S_alloc=30)
    idx = np.full((2, 2, 40), -1, np.int32)
    for b, S in enumerate(lens):
        idx[b, :, : S - 3] = np.arange(S - 3)[::-1]
    o, l = oracle.indexed(q, k, v, c["kv_lens_np"], idx, np.array(lens, np.int32) - 3, lib=lib)
    ov, lv = oracle.verify(q, k, v, c["kv_lens_np"], lib=lib)
    assert np.array_equal(o, ov) and np.array_equal(l, lv)


def pin_indexed_streaming_list_is_draft(lib=None):
    """q_len = 1 and the list [0, n_sink) u [S-W, S-1): exactly the StreamingLLM draft."""
    S, n_sink, W = 50, 4, 9
    c, q, k, v = host_case(B=1, q_len=1, Hq=2, Hkv=1, d=8, kv_lens=[S], dtype="f32", seed=32)
    lst = list(range(n_sink)) + list(range(S - W, S - 1))
    idx = np.array(lst, np.int32).reshape(1, 1, -1)
    o, l = oracle.indexed(q, k, v, c["kv_lens_np"], idx, np.array([len(lst)], np.int32), lib=lib)
    od, ld = oracle.draft(q, k, v, c["kv_lens_np"], n_sink, W, lib=lib)
    assert np.array_equal(o, od) and np.array_equal(l, ld)


def pin_indexed_sdpa(lib=None):
    """Indexed draft == library SDPA over the explicitly gathered keys of each
    row: the sorted listed positions, then the speculated positions up to p."""
    rng = np.random.default_rng(33)
    lens, q_len = [60, 41], 4
    c, q, k, v = host_case(B=2, q_len=q_len, Hq=6, Hkv=2, d=16, kv_lens=lens, dtype="bf16",
                           seed=34, S_alloc=60)
    idx, n = _index_lists(rng, 2, 2, lens, q_len, budget=13, stride=20)
    o, l = oracle.indexed(q, k, v, c["kv_lens_np"], idx, n, lib=lib)
    Q, K, V = f64(q), f64(k), f64(v)
    for b, S in enumerate(lens):
        for i in range(q_len):
            p = S - q_len + i
            for h in range(6):
                hk = h // 3
                keys = sorted(int(x) for x in idx[b, hk, : n[b]]) + list(range(S - q_len, p + 1))
                qt = torch.from_numpy(Q[b, i, h]).reshape(1, 1, -1)
                kt = torch.from_numpy(K[b, keys, hk]).unsqueeze(0)
                vt = torch.from_numpy(V[b, keys, hk]).unsqueeze(0)
                ot, lt = sdpa_rows(qt, kt, vt, 0.25, torch.ones(1, len(keys), dtype=torch.bool))
                close(o[b, i, h], ot[0, 0].numpy(), what="indexed O")
                close(l[b, i, h], lt[0, 0].item(), what="indexed lse")


def pin_indexed_ignores_unlisted_and_padding(lib=None):
    """Unlisted prompt keys may hold NaN; entries past idx_len, negative or at
    or after S - q_len are ignored; list order does not matter."""
    rng = np.random.default_rng(35)
    lens, q_len = [64, 40], 3
    c, q, k, v = host_case(B=2, q_len=q_len, Hq=2, Hkv=1, d=8, kv_lens=lens, dtype="f32", seed=36,
                           S_alloc=64)
    idx, n = _index_lists(rng, 2, 1, lens, q_len, budget=10, stride=16)
    o0, l0 = oracle.indexed(q, k, v, c["kv_lens_np"], idx, n, lib=lib)
    k2, v2 = k.copy(), v.copy()
    for b, S in enumerate(lens):
        listed = set(int(x) for x in idx[b, 0, : n[b]])
        for j in range(S - q_len):
            if j not in listed:
                k2[b, j] = np.nan
                v2[b, j] = np.nan
    idx2 = idx.copy()
    for b in range(2):
        idx2[b, 0, : n[b]] = rng.permutation(idx2[b, 0, : n[b]])
        idx2[b, 0, n[b]:] = [lens[b] - 1, -3, 10 ** 6, 0, 1, 2][: 16 - n[b]] + [0] * max(0, 10 - n[b])
    extra = np.concatenate([idx2, np.array([[[lens[0] - q_len]], [[lens[1]]]], np.int32)], axis=2)
    o1, l1 = oracle.indexed(q, k2, v2, c["kv_lens_np"], extra, n, lib=lib)
    assert np.array_equal(o0, o1) and np.array_equal(l0, l1)


def pin_indexed_empty_list(lib=None):
    """An empty list leaves only the speculated tokens, causally (row 0 sees one key)."""
    c, q, k, v = host_case(B=1, q_len=3, Hq=2, Hkv=1, d=8, kv_lens=[20], dtype="f32", seed=37)
    o, l = oracle.indexed(q, k, v, c["kv_lens_np"], np.zeros((1, 1, 4), np.int32),
                          np.zeros(1, np.int32), lib=lib)
    V = f64(v)
    assert np.array_equal(o[0, 0, 0], V[0, 17, 0])  # p = 17 sees only itself
    assert np.array_equal(o[0, 0, 1], V[0, 17, 0])


# ----------------------------------------------------------------------------- SnapKV selection

def pin_snapkv_votes_library(lib=None):
    """Pooled votes == torch float64: softmax of the observation queries over
    their causal keys (torch's bottom-right causal bias), summed over the
    window's queries and the group's query heads, prefix slice, then
    avg_pool1d(kernel 5, stride 1, padding 2)."""
    lens, n_obs, G = [40, 29], 6, 2
    c, q, k, v = host_case(B=2, q_len=n_obs, Hq=4, Hkv=2, d=16, kv_lens=lens, dtype="bf16",
                           seed=41, S_alloc=40)
    pooled = oracle.snapkv_votes(q, k, c["kv_lens_np"], pool=5, stride=40, lib=lib)
    Q, K = f64(q), f64(k)
    for b, S in enumerate(lens):
        n = S - n_obs
        for hk in range(2):
            vote = torch.zeros(n, dtype=torch.float64)
            for g in range(G):
                h = hk * G + g
                qt = torch.from_numpy(Q[b, :, h])                 # [n_obs, d]
                kt = torch.from_numpy(K[b, :S, hk])               # [S, d]
                s = (qt @ kt.T) * 0.25
                mask = causal_lower_right(n_obs, S)._materialize()
                a = torch.softmax(s.masked_fill(~mask, float("-inf")), dim=-1)
                vote += a[:, :n].sum(0)
            ref = F.avg_pool1d(vote.view(1, 1, -1), kernel_size=5, stride=1, padding=2).view(-1)
            close(pooled[b, hk, :n], ref.numpy(), what="snapkv pooled votes")
            assert np.all(pooled[b, hk, n:] == 0.0)


def pin_snapkv_single_spike(lib=None):
    """A key that takes (nearly) all attention spreads 1/5 of its vote to each of
    its four neighbours and itself: the pooling closed form."""
    n_obs, S, d = 2, 20, 8
    q = np.zeros((1, n_obs, 1, d), np.float32)
    q[..., 0] = 1.0
    k = np.zeros((1, S, 1, d), np.float32)
    k[0, 7, 0, 0] = 400.0           # score 400/sqrt(8): every other weight ~ e^-141
    pooled = oracle.snapkv_votes(q, k, np.array([S], np.int32), pool=5, stride=S, lib=lib)
    want = np.zeros(S)
    want[5:10] = n_obs / 5.0
    close(pooled[0, 0], want, tol=1e-12, what="spike pooling")


def pin_snapkv_select_library(lib=None):
    """Selection == numpy stable argsort of the negated values (ties: smaller
    position), top budget - n_obs, ascending, then the observation window."""
    rng = np.random.default_rng(43)
    rows, stride, n_obs, budget = 5, 300, 8, 40
    vals = np.round(rng.random((rows, stride)), 2)          # many exact ties
    lens = np.array([300, 308, 45, 20, 150], np.int32) + 0
    lens = np.minimum(lens, stride + n_obs)
    idx, cnt = oracle.snapkv_select(vals, lens, n_obs, budget, lib=lib)
    for r in range(rows):
        n = max(0, lens[r] - n_obs)
        keep = min(budget - n_obs, n)
        top = np.sort(np.argsort(-vals[r, :n], kind="stable")[:keep])
        want = np.concatenate([top, np.arange(n, lens[r])]).astype(np.int32)
        assert cnt[r] == len(want) and np.array_equal(idx[r, : cnt[r]], want), r


def pin_snapkv_select_ties_and_short(lib=None):
    """All-equal values keep the first positions; a prompt shorter than the
    budget keeps everything."""
    idx, cnt = oracle.snapkv_select(np.ones((1, 50)), np.array([58], np.int32), 8, 20, lib=lib)
    assert cnt[0] == 20 and np.array_equal(idx[0], np.r_[np.arange(12), np.arange(50, 58)])
    idx, cnt = oracle.snapkv_select(np.ones((1, 50)), np.array([15], np.int32), 8, 20, lib=lib)
    assert cnt[0] == 15 and np.array_equal(idx[0, :15], np.arange(15))


# ----------------------------------------------------------------------------- merge

def pin_merge_partition(lib=None):
    """Attention over disjoint key sets (library SDPA + logsumexp), merged, equals
    attention over their union; empty parts contribute nothing."""
    rng = np.random.default_rng(3)
    H, S, d = 3, 29, 8
    q = torch.from_numpy(rng.standard_normal((H, 2, d)))
    k = torch.from_numpy(rng.standard_normal((H, S, d)))
    v = torch.from_numpy(rng.standard_normal((H, S, d)))
    full_o, full_l = sdpa_rows(q, k, v, 0.3, torch.ones(2, S, dtype=torch.bool))
    for cuts in ([0, 29], [0, 10, 29], [0, 1, 2, 15, 28, 29], [0, 7, 7, 29]):
        parts_o, parts_l = [], []
        for a, b in zip(cuts[:-1], cuts[1:]):
            if b == a:  # an empty part: lse = -inf, O is never read (NaN to prove it)
                parts_o.append(np.full((H * 2, d), np.nan))
                parts_l.append(np.full((H * 2,), -np.inf))
                continue
            po, pl = sdpa_rows(q, k[:, a:b], v[:, a:b], 0.3, torch.ones(2, b - a, dtype=torch.bool))
            parts_o.append(po.reshape(H * 2, d).numpy())
            parts_l.append(pl.reshape(H * 2).numpy())
        o, lse = oracle.merge_lse(np.stack(parts_o), np.stack(parts_l), lib=lib)
        close(o, full_o.reshape(H * 2, d).numpy(), what=f"merge O {cuts}")
        close(lse, full_l.reshape(H * 2).numpy(), what=f"merge lse {cuts}")


def pin_merge_all_empty(lib=None):
    """Every part empty: O = 0 and lse = -inf."""
    o, lse = oracle.merge_lse(np.full((3, 2, 4), np.nan), np.full((3, 2), -np.inf), lib=lib)
    assert np.array_equal(o, np.zeros((2, 4))) and np.all(lse == -np.inf)


def pin_merge_shifted(lib=None):
    """Two copies of one part at lse 0: O unchanged, lse = ln 2 (weights 1/2 each)."""
    o_p = np.random.default_rng(0).standard_normal((1, 5, 4))
    o, lse = oracle.merge_lse(np.concatenate([o_p, o_p]), np.zeros((2, 5)), lib=lib)
    close(o, o_p[0], tol=1e-15, what="equal parts")
    close(lse, np.full(5, math.log(2.0)), tol=1e-15, what="ln 2")


ALL_PINS = [pin_sdpa_verify, pin_sdpa_verify_scale, pin_mpmath, pin_probs_rows_sum_to_one,
            pin_single_key, pin_equal_keys, pin_causal_invariance,
            pin_draft_equals_verify_when_budget_covers, pin_sdpa_draft, pin_draft_ignores_evicted,
            pin_gqa_equals_repeated_mha, pin_paged_equals_contiguous, pin_bf16_decode,
            pin_indexed_full_list_is_verify, pin_indexed_streaming_list_is_draft, pin_indexed_sdpa,
            pin_indexed_ignores_unlisted_and_padding, pin_indexed_empty_list,
            pin_snapkv_votes_library, pin_snapkv_single_spike, pin_snapkv_select_library,
            pin_snapkv_select_ties_and_short,
            pin_merge_partition, pin_merge_all_empty, pin_merge_shifted]
