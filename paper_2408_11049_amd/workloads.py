"""Seeded synthetic workloads for MagicDec's verify/draft attention.

This module draws inputs and nothing else: it holds no attention arithmetic,
so the GPU path and the fp64 oracle can both be fed from it.  Values are
i.i.d. N(0, 1) drawn in fp32 and rounded to the storage dtype, on Llama-3.1
head shapes (the paper's models; Sec. 5), with long-context lengths standing
in for the PG-19 / RULER prompts the paper decodes (Sec. 5.1, 5.2), which are
not used.

Seeds: workload ``base`` uses generator streams ``base*10 + s`` with
s = 0 Q, 1 K, 2 V, 3 lengths, 4 page placement, 5 outlier channels,
6 logits, 7 planted tokens and drafts, 8 appended K/V rows, 9 the bench's
SnapKV observation queries.

Padding that a correct kernel never reads (tokens past kv_lens[b] in a
contiguous cache, slots past the end in a sequence's last page, pages owned by
no sequence) is filled with NaN, so an over-read shows up as NaN output.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

(STREAM_Q, STREAM_K, STREAM_V, STREAM_LEN, STREAM_PAGE, STREAM_OUTLIER, STREAM_LOGITS,
 STREAM_DRAFT, STREAM_NEW_KV) = range(9)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    gamma: int              # speculation length; q_len = gamma + 1
    n_sink: int
    window: int
    dtype: str              # "f32" | "bf16"
    seed_base: int
    S: int = 0              # uniform KV length (every sequence), or 0 if ragged
    S_lo: int = 0           # ragged: S_b uniform integer in [S_lo, S_hi]
    S_hi: int = 0
    page_size: int = 0      # 0 = contiguous [B, S_alloc, Hkv, d]; else [P, page_size, Hkv, d]
    k_outlier_dims: int = 0  # K channels scaled by k_outlier_scale (same dims for all heads/tokens)
    k_outlier_scale: float = 1.0

    @property
    def q_len(self) -> int:
        return self.gamma + 1

    @property
    def max_kv_len(self) -> int:
        return self.S if self.S else self.S_hi

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny_f32", B=2, Hq=4, Hkv=1, d=64, S=256, gamma=3, n_sink=4, window=32,
                 dtype="f32", seed_base=1),
        Workload("llama8b_b32_s8k", B=32, Hq=32, Hkv=8, d=128, S=8192, gamma=3, n_sink=16,
                 window=496, dtype="bf16", seed_base=2),
        Workload("llama8b_b64_ragged_paged", B=64, Hq=32, Hkv=8, d=128, S_lo=16384, S_hi=32768,
                 gamma=4, n_sink=16, window=1008, dtype="bf16", seed_base=3, page_size=16),
        Workload("llama8b_b64_s32k_paged", B=64, Hq=32, Hkv=8, d=128, S=32768, gamma=4,
                 n_sink=16, window=1008, dtype="bf16", seed_base=3, page_size=16),
        Workload("llama8b_b256_s8k_koutlier", B=256, Hq=32, Hkv=8, d=128, S=8192, gamma=2,
                 n_sink=16, window=496, dtype="bf16", seed_base=4, k_outlier_dims=4,
                 k_outlier_scale=8.0),
        Workload("llama70b_b16_s128k", B=16, Hq=64, Hkv=8, d=128, S=131072, gamma=4, n_sink=64,
                 window=1984, dtype="bf16", seed_base=5),
    ]
}


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _randn_into(out: torch.Tensor, g: torch.Generator, slab: int = 1 << 26):
    """Fill ``out`` (any float dtype) with N(0,1) drawn in fp32, slab by slab
    along dim 0 so huge caches never need a full fp32 copy."""
    n0 = out.shape[0]
    per = max(1, slab // max(1, out[0].numel()))
    for s in range(0, n0, per):
        e = min(n0, s + per)
        tmp = torch.randn(out[s:e].shape, generator=g, device=out.device, dtype=torch.float32)
        out[s:e].copy_(tmp)
        del tmp


def torch_dtype(dtype: str):
    return torch.float32 if dtype == "f32" else torch.bfloat16


def kv_lengths(w: Workload) -> np.ndarray:
    """Per-sequence KV lengths (including the q_len speculated tokens)."""
    if w.S:
        return np.full((w.B,), w.S, dtype=np.int32)
    g = _gen(w.seed_base * 10 + STREAM_LEN, "cpu")
    s = torch.randint(w.S_lo, w.S_hi + 1, (w.B,), generator=g, dtype=torch.int64)
    return s.numpy().astype(np.int32)


def outlier_channels(w: Workload) -> np.ndarray:
    g = _gen(w.seed_base * 10 + STREAM_OUTLIER, "cpu")
    return torch.randperm(w.d, generator=g)[: w.k_outlier_dims].numpy()


def make_case(*, B, q_len, Hq, Hkv, d, kv_lens, dtype="bf16", page_size=0, seed=0,
              S_alloc: Optional[int] = None, extra_pages: int = 2, device="cpu",
              k_outlier_dims: int = 0, k_outlier_scale: float = 1.0, outlier_seed=None,
              nan_pad: bool = True):
    """Draw one seeded problem.

    Returns a dict with q [B, q_len, Hq, d], k, v (contiguous [B, S_alloc, Hkv, d]
    or paged [P, page_size, Hkv, d]), kv_lens (int32 tensor), max_kv_len,
    page_table ([B, max_pages] int32 with -1 for unused entries, or None).
    """
    tdt = torch_dtype(dtype)
    kv_lens = np.asarray(kv_lens, dtype=np.int32).reshape(-1)
    assert kv_lens.shape[0] == B
    max_kv_len = int(kv_lens.max()) if B else 0
    q = torch.empty((B, q_len, Hq, d), dtype=tdt, device=device)
    _randn_into(q, _gen(seed * 10 + STREAM_Q, device)) if B else None
    page_table = None
    if page_size == 0:
        S_alloc = max_kv_len if S_alloc is None else S_alloc
        shape = (B, S_alloc, Hkv, d)
    else:
        max_pages = max(1, math.ceil(max_kv_len / page_size))
        n_pages = [math.ceil(int(s) / page_size) for s in kv_lens]
        P = sum(n_pages) + extra_pages
        perm = torch.randperm(P, generator=_gen(seed * 10 + STREAM_PAGE, "cpu")).numpy()
        pt = np.full((B, max_pages), -1, dtype=np.int32)
        off = 0
        for b in range(B):
            pt[b, : n_pages[b]] = perm[off: off + n_pages[b]]
            off += n_pages[b]
        page_table = pt
        shape = (P, page_size, Hkv, d)
    k = torch.empty(shape, dtype=tdt, device=device)
    v = torch.empty(shape, dtype=tdt, device=device)
    if shape[0]:
        _randn_into(k, _gen(seed * 10 + STREAM_K, device))
        _randn_into(v, _gen(seed * 10 + STREAM_V, device))
    if k_outlier_dims:
        g = _gen((outlier_seed if outlier_seed is not None else seed) * 10 + STREAM_OUTLIER, "cpu")
        ch = torch.randperm(d, generator=g)[:k_outlier_dims].tolist()
        k[..., ch] *= k_outlier_scale
    if nan_pad:
        nan = float("nan")
        if page_size == 0:
            for b in range(B):
                if kv_lens[b] < S_alloc:
                    k[b, kv_lens[b]:] = nan
                    v[b, kv_lens[b]:] = nan
        else:
            used = set()
            for b in range(B):
                npg = math.ceil(int(kv_lens[b]) / page_size)
                used.update(int(x) for x in page_table[b, :npg])
                tail = int(kv_lens[b]) - (npg - 1) * page_size
                if npg and tail < page_size:
                    last = int(page_table[b, npg - 1])
                    k[last, tail:] = nan
                    v[last, tail:] = nan
            for p in range(shape[0]):
                if p not in used:
                    k[p] = nan
                    v[p] = nan
    out = dict(q=q, k=k, v=v, kv_lens=torch.from_numpy(kv_lens.copy()).to(device),
               kv_lens_np=kv_lens, max_kv_len=max_kv_len, page_size=page_size,
               page_table=None if page_table is None else torch.from_numpy(page_table).to(device),
               page_table_np=page_table, dtype=dtype, B=B, q_len=q_len, Hq=Hq, Hkv=Hkv, d=d)
    return out


def make_workload(w: Workload, device="cpu", *, q_len: Optional[int] = None, nan_pad=True):
    """Full-size inputs of a named workload (q_len defaults to gamma + 1)."""
    return make_case(B=w.B, q_len=q_len or w.q_len, Hq=w.Hq, Hkv=w.Hkv, d=w.d,
                     kv_lens=kv_lengths(w), dtype=w.dtype, page_size=w.page_size,
                     seed=w.seed_base, device=device, k_outlier_dims=w.k_outlier_dims,
                     k_outlier_scale=w.k_outlier_scale, outlier_seed=w.seed_base,
                     nan_pad=nan_pad, extra_pages=2 if w.page_size else 0)


def index_lists(B, Hkv, lens, q_len, budget, seed):
    """Seeded stand-in for a SnapKV selection: for every (sequence, kv head),
    min(budget, S_b - q_len) distinct prompt positions in ascending order.
    Returns (idx [B, Hkv, budget] int32, idx_len [B] int32)."""
    g = _gen(seed * 10 + STREAM_PAGE + 100, "cpu")
    idx = np.zeros((B, Hkv, max(1, budget)), np.int32)
    n = np.zeros(B, np.int32)
    for b in range(B):
        pool = int(lens[b]) - q_len
        n[b] = max(0, min(budget, pool))
        for h in range(Hkv):
            idx[b, h, : n[b]] = np.sort(torch.randperm(pool, generator=g)[: n[b]].numpy())
    return idx, n


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """Device/host tensor -> numpy array the oracle accepts (float32, or bf16 bit patterns)."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def gather_unit(case: dict, b: int, hk: int):
    """Host copy of one (sequence b, kv head hk) unit as a contiguous
    B=1, Hkv=1 problem: q [1, q_len, G, d], k/v [1, S_b, 1, d], kv_lens [S_b].

    Only indexing (a gather through the page table when paged): the sampled
    full-size parity checks hand this to the oracle one unit at a time."""
    G = case["Hq"] // case["Hkv"]
    S_b = int(case["kv_lens_np"][b])
    q = case["q"][b: b + 1, :, hk * G: (hk + 1) * G, :]
    if case["page_size"] == 0:
        k = case["k"][b: b + 1, :S_b, hk: hk + 1, :]
        v = case["v"][b: b + 1, :S_b, hk: hk + 1, :]
    else:
        ps = case["page_size"]
        npg = math.ceil(S_b / ps)
        pages = torch.as_tensor(case["page_table_np"][b, :npg], dtype=torch.int64,
                                device=case["k"].device)
        k = case["k"].index_select(0, pages)[:, :, hk: hk + 1, :].reshape(1, npg * ps, 1, -1)[:, :S_b]
        v = case["v"].index_select(0, pages)[:, :, hk: hk + 1, :].reshape(1, npg * ps, 1, -1)[:, :S_b]
    return (to_host_bits(q), to_host_bits(k), to_host_bits(v), np.array([S_b], dtype=np.int32))


def new_kv_rows(B, n_new, Hkv, d, dtype="bf16", seed=0, device="cpu"):
    """K and V rows of n_new new tokens per sequence, [B, n_new, Hkv, d], N(0, 1)."""
    g = _gen(seed * 10 + STREAM_NEW_KV, device)
    tdt = torch_dtype(dtype)
    k = torch.randn((B, n_new, Hkv, d), generator=g, device=device).to(tdt)
    v = torch.randn((B, n_new, Hkv, d), generator=g, device=device).to(tdt)
    return k, v


# Planted logit: far above any N(0, 1) draw and exact in bf16.
PLANTED_LOGIT = 64.0


def step_logits(B, gamma, vocab, dtype="f32", seed=0, device="cpu", accept=None, ties=0,
                nan_rows=0, neg_inf_rows=0):
    """Seeded verifier logits and drafts for one greedy-acceptance step.

    logits [B, gamma + 1, vocab]: N(0, 1) with one planted logit PLANTED_LOGIT
    per row, at token planted[b, i] (drawn uniformly).  draft [B, gamma]
    int32 copies planted[b, :a_b] and then differs from the planted token at
    a_b (a_b = accept[b], default uniform in 0..gamma), random after.
    ties: rows (seeded) that also carry PLANTED_LOGIT at a second token;
    nan_rows / neg_inf_rows: rows turned entirely NaN / -inf except for the
    first half, which is NaN (for the -inf rows), so only -inf values remain.
    Returns (logits, draft, planted [B, gamma + 1] int64 numpy, accept numpy)."""
    L = gamma + 1
    g = _gen(seed * 10 + STREAM_LOGITS, device)
    x = torch.randn((B, L, vocab), generator=g, device=device, dtype=torch.float32)
    gd = _gen(seed * 10 + STREAM_DRAFT, "cpu")
    planted = torch.randint(0, vocab, (B, L), generator=gd).numpy()
    if accept is None:
        accept = torch.randint(0, gamma + 1, (B,), generator=gd).numpy()
    accept = np.asarray(accept, dtype=np.int64)
    draft = torch.randint(0, vocab, (B, max(gamma, 1)), generator=gd).numpy()[:, :gamma].copy()
    for b in range(B):
        draft[b, : accept[b]] = planted[b, : accept[b]]
        if accept[b] < gamma:
            draft[b, accept[b]] = (planted[b, accept[b]] + 1) % vocab
    rows = torch.randperm(B * L, generator=gd).numpy()
    tie_rows = rows[:ties]
    nan_r = rows[ties: ties + nan_rows]
    inf_r = rows[ties + nan_rows: ties + nan_rows + neg_inf_rows]
    tie_tok = torch.randint(0, vocab, (max(ties, 1),), generator=gd).numpy()
    bi = torch.arange(B).repeat_interleave(L).numpy()
    ii = torch.arange(L).repeat(B).numpy()
    x[torch.as_tensor(bi), torch.as_tensor(ii), torch.as_tensor(planted.reshape(-1))] = PLANTED_LOGIT
    for n, r in enumerate(tie_rows):
        x[bi[r], ii[r], int(tie_tok[n])] = PLANTED_LOGIT
    for r in nan_r:
        x[bi[r], ii[r]] = float("nan")
    for r in inf_r:
        x[bi[r], ii[r]] = float("-inf")
        x[bi[r], ii[r], : vocab // 2] = float("nan")
    logits = x.to(torch_dtype(dtype))
    return (logits, torch.from_numpy(draft.astype(np.int32)).to(device),
            planted.astype(np.int64), accept)
