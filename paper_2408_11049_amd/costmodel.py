"""The speculative-decoding cost model on MI355X, fed with measured attention
times: the per-layer attention analogue of the paper's speedup analysis
(Sec. 3.1 Eq. 1-2, Sec. 3.2, Sec. 4.1 Eq. 3-4).

For each batch size B and sequence length S, one Llama-3.1-8B layer's decode
attention (Hq = 32, Hkv = 8, d = 128, bf16 K/V) is timed on this GPU, from a
cold cache:

  T_T        verify at q_len = 1 (plain decoding: one token per sequence),
  T_V(g)     verify at q_len = g + 1 (g speculated tokens plus the last one),
  T_D        one-token draft over a StreamingLLM cache of 16 sinks + 496
             window (budget 512, Table 1), over a listed SnapKV-style cache
             of 2049 positions (Sec. 5.2), and over the same 2049 rows
             gathered once into a draft cache of their own (md_kv_gather);
             static selections cost nothing per step (T_select = 0 in Eq. 3).

Those times go through the library's cost model (md_sd_best_gamma, Eq. 4 over
gamma) for a set of acceptance rates, giving the best speculation length, the
attention-only latency ratio T_Avg^SD / T_T and its inverse, the speedup the
attention part of a layer would see.  Attention is the part of the step that
grows with B and S (Sec. 3.2); the projections and MLP a full layer adds are
outside this model, so these are the attention-only analogues of Fig. 2-3,
not end-to-end speedups.  S_inflection is the smallest measured S at which the
best ratio drops below 1.

    python -m paper_2408_11049_amd.costmodel [--quick]

prints one JSON line per (B, S) and a markdown summary.
"""
from __future__ import annotations

import argparse
import json
import sys

LLAMA8B = dict(Hq=32, Hkv=8, d=128, dtype="bf16")
ALPHAS = (0.7, 0.8, 0.9, 0.93)
N_SINK, WINDOW, LISTED = 16, 496, 2049


def _timer(dev, flush, lib, sh):
    import numpy as np
    import torch

    import paper_2408_11049_amd as md

    stream = torch.cuda.current_stream(dev)

    def timed(fn, reps):
        ts = []
        for _ in range(reps + 1):
            md._check(lib.md_bench_fill(md.ctypes.c_void_p(flush.data_ptr()), flush.numel(), 0, sh))
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        return float(np.median(ts[1:]))  # the first call warms the instance up

    return timed


def measure(B, S, max_gamma=8, reps=5, device="cuda:0", seed=7):
    """Times in microseconds: t_target, t_verify[g - 1] for g = 1 .. max_gamma,
    t_draft_streaming, t_draft_listed, t_draft_gathered."""
    import torch

    import paper_2408_11049_amd as md
    from paper_2408_11049_amd import workloads as wl

    dev = torch.device(device)
    lib = md.load_library()
    sh = md.ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    timed = _timer(dev, flush, lib, sh)
    c = wl.make_case(B=B, q_len=max_gamma + 1, kv_lens=[S] * B, seed=seed, device=dev,
                     nan_pad=False, **LLAMA8B)
    k, v, lens = c["k"], c["v"], c["kv_lens"]
    qs = {L: c["q"][:, :L].contiguous() for L in range(1, max_gamma + 2)}
    outs = {L: torch.empty_like(qs[L]) for L in qs}

    def ws(q, mode, **kw):
        n = md.md_workspace_bytes(q, k, v, lens, mode=mode, n_sink=N_SINK, window=WINDOW,
                                  max_kv_len=S)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=dev) if n else None

    wsv = {L: ws(qs[L], md.MD_MODE_VERIFY) for L in qs}
    wsd = ws(qs[1], md.MD_MODE_DRAFT)

    def verify(L):
        return lambda: md.md_verify_attn(qs[L], k, v, lens, out=outs[L], return_lse=False,
                                         workspace=wsv[L], max_kv_len=S)

    t_verify = [timed(verify(g + 1), reps) for g in range(1, max_gamma + 1)]
    t_target = timed(verify(1), reps)
    t_stream = timed(lambda: md.md_draft_attn(qs[1], k, v, lens, N_SINK, WINDOW, out=outs[1],
                                              return_lse=False, workspace=wsd, max_kv_len=S),
                     reps)
    idx_np, n_np = wl.index_lists(B, LLAMA8B["Hkv"], c["kv_lens_np"], 1, LISTED, seed)
    idx, n_t = torch.from_numpy(idx_np).to(dev), torch.from_numpy(n_np).to(dev)
    t_listed = timed(lambda: md.md_draft_attn_indexed(qs[1], k, v, lens, idx, n_t, out=outs[1],
                                                      return_lse=False, max_kv_len=S), reps)
    ck = torch.empty((B, LISTED + 1) + tuple(k.shape[2:]), dtype=k.dtype, device=dev)
    cv = torch.empty_like(ck)
    glen = md.md_kv_gather(ck, cv, k, v, idx, n_t, (lens - 1).contiguous())
    # the drafted token's row, as the draft step appends it
    glen1 = md.md_kv_append(ck, cv, k[:, S - 1:S].contiguous(), v[:, S - 1:S].contiguous(), glen)
    t_gathered = timed(lambda: md.md_verify_attn(qs[1], ck, cv, glen1, out=outs[1],
                                                 return_lse=False, max_kv_len=LISTED + 1), reps)
    del c, k, v, ck, cv, flush
    torch.cuda.empty_cache()
    return dict(B=B, S=S, t_target=t_target, t_verify=t_verify, t_draft_streaming=t_stream,
                t_draft_listed=t_listed, t_draft_gathered=t_gathered)


def analyse(m, alphas=ALPHAS):
    """Best gamma and attention-only ratio (Eq. 4 over gamma, Eq. 2) per draft
    cache and acceptance rate, from the library's cost model."""
    import paper_2408_11049_amd as md

    out = {"tv1_over_tt": m["t_verify"][0] / m["t_target"]}
    for name, td in (("streaming", m["t_draft_streaming"]), ("listed", m["t_draft_listed"]),
                     ("gathered", m["t_draft_gathered"])):
        for a in alphas:
            g, r = md.md_sd_best_gamma(a, m["t_target"], td, m["t_verify"])
            out[f"{name}@{a}"] = {"gamma": g, "ratio": r, "speedup": 1.0 / r}
    return out


def grid(quick=False):
    if quick:
        return [(4, 4096), (16, 16384)]
    Bs = (1, 4, 16, 64, 256)
    Ss = (1024, 4096, 16384, 32768, 65536, 131072)
    return [(B, S) for B in Bs for S in Ss if B * S <= (1 << 22)]


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--max-gamma", type=int, default=8)
    args = ap.parse_args(argv)
    rows = []
    for B, S in grid(args.quick):
        print(f"[costmodel] B={B} S={S}", file=sys.stderr, flush=True)
        m = measure(B, S, max_gamma=args.max_gamma)
        m["model"] = analyse(m)
        rows.append(m)
        print(json.dumps(m), flush=True)
    print("\n| B | S | T_T us | T_V(1)/T_T | T_V(4)/T_T | T_D 512 us | T_D 2049 listed us | "
          "T_D 2049 gathered us | " + " | ".join(f"gathered a={a}: g, x" for a in ALPHAS) + " |")
    print("|" + "---|" * (8 + len(ALPHAS)))
    for m in rows:
        cells = [str(m["B"]), str(m["S"]), f"{m['t_target']:.1f}",
                 f"{m['t_verify'][0] / m['t_target']:.3f}",
                 f"{m['t_verify'][3] / m['t_target']:.3f}" if len(m["t_verify"]) >= 4 else "-",
                 f"{m['t_draft_streaming']:.1f}", f"{m['t_draft_listed']:.1f}",
                 f"{m['t_draft_gathered']:.1f}"]
        for a in ALPHAS:
            e = m["model"][f"gathered@{a}"]
            cells.append(f"{e['gamma']}, {e['speedup']:.2f}")
        print("| " + " | ".join(cells) + " |")
    print("\nS_inflection (smallest measured S with attention-only speedup > 1):")
    for name in ("streaming", "listed", "gathered"):
        for a in ALPHAS:
            parts = []
            for B in sorted({m["B"] for m in rows}):
                s = [m["S"] for m in rows if m["B"] == B and m["model"][f"{name}@{a}"]["ratio"] < 1.0]
                parts.append(f"B={B}: {min(s) if s else '-'}")
            print(f"  {name} a={a}: " + ", ".join(parts))


if __name__ == "__main__":
    main()
