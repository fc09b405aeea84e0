"""bench.py's host side, without a GPU: the one-GPU guard, the algorithmic
byte counts its GB/s and roofline divide by, and the readers of the committed
rocprofv3 summaries (which must describe the kernel source as it stands)."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2408_11049_amd import workloads as wl  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and not r.stdout


# K+V bytes of one call, from the definitions: 2 (K, V) * d * 2 B * Hkv per
# visible token per sequence.  Draft: sinks + window + q_len - 1 tokens.
@pytest.mark.parametrize("name,verify,draft", [
    ("llama8b_b32_s8k", 1_073_741_824, 67_502_080),          # 32 x 8 x (16 + 496 + 3) x 512
    ("llama8b_b64_s32k_paged", 8_589_934_592, 269_484_032),  # 64 x 8 x (16 + 1008 + 4) x 512
    ("llama8b_b256_s8k_koutlier", 8_589_934_592, 538_968_064),  # 256 x 8 x (16 + 496 + 2) x 512
    ("llama70b_b16_s128k", 8_589_934_592, 134_479_872),      # 16 x 8 x (64 + 1984 + 4) x 512
])
def test_algorithmic_bytes(name, verify, draft):
    w = wl.WORKLOADS[name]
    lens = np.full(w.B, w.S)
    assert bench.kv_bytes(w, lens, "verify", w.q_len) == verify
    assert bench.kv_bytes(w, lens, "draft", w.q_len) == draft


def test_short_sequences_read_their_whole_prefix_in_draft_mode():
    w = wl.WORKLOADS["llama8b_b64_s32k_paged"]
    lens = np.array([5, 1000, 1029, 1030])  # up to 16 + 1008 + 4 tokens, then the gap opens
    per_tok = 2 * w.Hkv * w.d * 2
    want = (5 + 1000 + 1028 + 1028) * per_tok
    assert bench.kv_bytes(w, lens, "draft", w.q_len) == want


def test_profile_readers_match_the_kernel_source(monkeypatch):
    """The committed summaries carry the SHA-256 of the kernel sources they were
    taken on; bench.py reports their figures only while it matches."""
    traffic, mfma, trace = bench.read_counters(), bench.read_mfma(), bench.read_trace()
    assert traffic is not None and 8.5e9 < traffic < 8.7e9, "profiles/ are stale: re-profile"
    assert mfma is not None and 0 < mfma["frac"] < 1
    assert trace is not None and 0 < trace["verify_kernel_mean_us"] <= trace["verify_event_mean_us"]
    other = [os.path.join(ROOT, "paper_2408_11049_amd", "csrc", "step.hip")]
    monkeypatch.setattr(bench, "KERNEL_SOURCES", other)
    assert bench.read_counters() is None and bench.read_mfma() is None and bench.read_trace() is None


def _trace_csv(path, names_durs):
    """A kernel-trace CSV in rocprofv3's layout: one row per dispatch."""
    import csv
    with open(path, "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(["Kind", "Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        t = 1000
        for i, (n, d) in enumerate(names_durs):
            wr.writerow(["KERNEL_DISPATCH", i + 1, n, t, t + int(d * 1000)])
            t += int(d * 1000) + 5000


def test_trace_summary_picks_the_timed_calls(tmp_path):
    """S settling verify calls, W warm-up steps, then K timed steps, each verify
    then draft, each after an eviction read: the summary takes attention calls
    S + 2W .. S + 2(W+K)-1 only (a merge dispatch counts with its call),
    whatever runs after them."""
    V, D = "void md::attn_partial_kernel<128, true, 2, true, false, 1, 1>(md::AttnParams)", \
        "void md::attn_partial_kernel<128, true, 2, true, false, 1, 2>(md::AttnParams)"
    M, E = "void md::merge_lse_kernel<128, true>(int, long, float const*)", "md::bench_evict_kernel"
    seq = [(E, 100), (V, 1500)] * 4  # four settling verify calls, untimed
    for step in range(2 + 3):  # W = 2, K = 3
        seq += [(E, 100), (V, 900 if step < 2 else 1000 + step), (E, 100), (D, 50), (M, 4)]
    seq += [(V, 5.0), (D, 7.0)]  # later calls of the same templates are not timed
    csv_path = tmp_path / "t.csv"
    _trace_csv(csv_path, seq)
    line = {"metric": "m", "value": 1, "unit": "GB/s", "steps": 3, "warmup": 2, "ms_per_step": 1,
            "roofline": {"achieved": 1, "frac": 0.5, "algorithmic_bytes_per_launch": 8e9},
            "detail": {"t_verify_us": 1010.0, "t_draft_us": 60.0, "verify_kv_bytes": 8e9,
                       "draft_kv_bytes": 2.7e8, "settle_calls (untimed verify calls)": 4}}
    bj = tmp_path / "b.json"
    bj.write_text("noise\n" + __import__("json").dumps(line) + "\n")
    md_text = bench.summarize_trace(str(csv_path), str(bj), "cmd")
    fields = dict(l.split(": ", 1) for l in md_text.splitlines() if ": " in l and l[0].isalpha()
                  and " " not in l.split(": ", 1)[0])
    assert float(fields["verify_kernel_mean_us"]) == pytest.approx((1002 + 1003 + 1004) / 3)
    assert float(fields["draft_kernel_mean_us"]) == pytest.approx(54.0)  # attention + merge
    assert fields["kernel_source_sha256"] == bench.kernel_source_sha256()
    assert "WARNING" not in md_text


def test_lds_summary_groups_by_kernel(tmp_path):
    """--summarize lds: per-instance means of the LDS counters, the bench's
    timed verify and draft instances named, kernels without LDS traffic and the
    bench helpers left out."""
    import csv
    V, D = "void md::attn_partial_kernel<128, true, 2, true, false, 1, 1, true>(md::AttnParams)", \
        "void md::attn_partial_kernel<128, true, 2, true, false, 1, 2, false>(md::AttnParams)"
    E, C = "md::bench_evict_kernel", "at::native::copy_kernel"
    seq = [(E, 0, 0), (V, 100, 10)] * 2  # two settling verify calls
    for step in range(1 + 2):            # W = 1, K = 2
        seq += [(E, 0, 0), (V, 100, 10), (E, 0, 0), (D, 40, 8), (C, 0, 0)]
    path = tmp_path / "c.csv"
    with open(path, "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (n, active, conflict) in enumerate(seq):
            for ctr in bench.LDS_COUNTERS:
                val = {"SQ_LDS_IDX_ACTIVE": active, "SQ_LDS_BANK_CONFLICT": conflict}.get(ctr, 1.0)
                wr.writerow([i + 1, n, ctr, val if n not in (E, C) else 0.0])
    line = {"metric": "m", "value": 1, "unit": "GB/s", "steps": 2, "warmup": 1,
            "detail": {"settle_calls (untimed verify calls)": 2}}
    bj = tmp_path / "b.json"
    bj.write_text(__import__("json").dumps(line) + "\n")
    text = bench.summarize_lds(str(path), str(bj), "cmd")
    rows = [l for l in text.splitlines() if l.startswith("| ") and "attn_partial" in l]
    assert len(rows) == 2
    v = next(r for r in rows if r.startswith("| verify (bench)"))
    d = next(r for r in rows if r.startswith("| draft (bench)"))
    assert "| 5 |" in v and "| 0.100 |" in v  # 2 settling + 3 step calls, 10 / 100
    assert "| 3 |" in d and "| 0.200 |" in d
    assert "bench_evict" not in text and "copy_kernel" not in text


def test_config_summary_walks_back_from_the_table(tmp_path):
    """--summarize configs: the table is the run's last attention work; per
    configuration one warm call of each kind, its settling verify calls, then
    10 timed calls per kind -- picked by walking back from the end, whatever
    ran before (here a bench-shape step and a stray earlier call)."""
    import json
    names = bench.CONFIGS
    seq = [("void md::attn_partial_kernel<128, true, 2, true, false, 1, 1, true, 4>(x)", 999)] * 7
    cfgs = {}
    for ci, name in enumerate(names):
        kern = {k: f"void md::attn_partial_kernel<{ci}, {ki}>(x)" for ki, k in enumerate(bench.CONFIG_KINDS)}
        settle = 3 + ci
        seq += [(kern[k], 500) for k in bench.CONFIG_KINDS]       # warm
        seq += [(kern["verify"], 700)] * settle                     # settling
        for ki, k in enumerate(bench.CONFIG_KINDS):
            seq += [(kern[k], 100 * (ci + 1) + ki)] * 10
            if k == "draft" and ci == 1:                           # a split plan: merge after each call
                seq = seq[:-10] + sum([[(kern[k], 100 * (ci + 1) + ki),
                                        ("void md::merge_lse_kernel<128, true, true>(x)", 4)]] * 10, [])
        cfgs[name] = {"settle_calls (untimed verify calls first, >= 60 ms)": settle}
        for ki, k in enumerate(bench.CONFIG_KINDS):
            cfgs[name][f"t_{k}_us_p10_p50_p90"] = [1, 100 * (ci + 1) + ki + 5, 1]
            cfgs[name][f"{k}_kv_bytes"] = 1e9
    path = tmp_path / "t.csv"
    _trace_csv(path, seq)
    bj = tmp_path / "b.json"
    bj.write_text(json.dumps({"metric": "m", "value": 1, "unit": "GB/s", "steps": 1, "warmup": 1,
                              "detail": {"configs": cfgs}}) + "\n")
    text = bench.summarize_configs(str(path), str(bj), "cmd")
    rows = [l.split(" | ") for l in text.splitlines() if l.startswith("| ") and "attn_partial" in l]
    assert len(rows) == 4 * len(names)
    for r in rows:
        ci, ki = names.index(r[0][2:]), bench.CONFIG_KINDS.index(r[1])
        want = 100 * (ci + 1) + ki + (4 if (ci == 1 and ki == 2) else 0)
        assert float(r[3]) == pytest.approx(want), r
        assert ("+ merge" in r[2]) == (ci == 1 and ki == 2)


def test_config_counter_summary(tmp_path):
    """--summarize config-counters: FETCH_SIZE and WRITE_SIZE of the table's
    timed calls (attention plus merge), each run picked with its own settling
    counts and scaled by the run's 1 GiB copy."""
    import csv
    import json
    names = bench.CONFIGS

    def run(ctr, settle_extra):
        rows, cfgs, did = [], {}, 0

        def add(name, val):
            nonlocal did
            did += 1
            rows.append([did, name, ctr, val])
        add("md::bench_copy_kernel", (1 << 20) / (2 if ctr == "FETCH_SIZE" else 1))
        for ci, name in enumerate(names):
            kern = {k: f"void md::attn_partial_kernel<{ci}, {ki}>(x)" for ki, k in enumerate(bench.CONFIG_KINDS)}
            settle = 2 + ci + settle_extra
            for k in bench.CONFIG_KINDS:
                add(kern[k], 1.0)
            for _ in range(settle):
                add(kern["verify"], 1.0)
            for k in bench.CONFIG_KINDS:
                for _ in range(10):
                    add(kern[k], 1000.0 * (ci + 1))
                    if ci == 4:
                        add("void md::merge_lse_kernel<128, true, true>(x)", 10.0)
            cfgs[name] = {"settle_calls (untimed verify calls first, >= 60 ms)": settle}
            for k in bench.CONFIG_KINDS:
                cfgs[name][f"{k}_kv_bytes"] = 1024.0 * 1000.0 * (ci + 1)
        path = tmp_path / f"{ctr}.csv"
        with open(path, "w", newline="") as f:
            wr = csv.writer(f)
            wr.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
            wr.writerows(rows)
        bj = tmp_path / f"{ctr}.json"
        bj.write_text(json.dumps({"metric": "m", "value": 1, "unit": "GB/s", "steps": 1, "warmup": 1,
                                  "detail": {"configs": cfgs}}) + "\n")
        return str(path), str(bj)

    fc, fj = run("FETCH_SIZE", 0)
    wc, wj = run("WRITE_SIZE", 3)  # another run settles longer
    text = bench.summarize_config_counters(fc, wc, fj, wj, "cmd")
    rows = [l.split(" | ") for l in text.splitlines() if l.startswith("| ") and "attn_partial" in l]
    assert len(rows) == 4 * len(names)
    for r in rows:
        ci = names.index(r[0][2:])
        extra = 10.0 if ci == 4 else 0.0
        assert float(r[3]) == pytest.approx((1000.0 * (ci + 1) + extra) * 1024 * 2, rel=1e-3)
        assert float(r[4]) == pytest.approx((1000.0 * (ci + 1) + extra) * 1024, rel=1e-3)


def test_prefill_summary(tmp_path):
    """--summarize prefill: trace times and counter bytes of the SnapKV and
    gather kernels, the counters scaled by the run's 1 GiB copy, each read
    compared with its algorithmic bytes from the bench line."""
    import csv
    import json
    P0 = "void md::snapkv_pass_kernel<128, true, 2, true, 0, 64>(md::SnapkvParams)"
    P1 = "void md::snapkv_pass_kernel<128, true, 2, true, 1, 64>(md::SnapkvParams)"
    S, G, C = "void md::snapkv_select_reg_kernel<5>(x)", "void md::kv_gather_pow2_kernel<true, false>(x)", \
        "md::bench_copy_kernel(x)"
    seq = [(C, 0, 0), (P0, 10.0, 2.0), (P1, 10.0, 4.0), (S, 4.0, 1.0), (G, 6.0, 5.0)] * 2
    tr, fe, wr = tmp_path / "t.csv", tmp_path / "f.csv", tmp_path / "w.csv"
    with open(tr, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for i, (n, _, _) in enumerate(seq):
            w.writerow([i + 1, n, 1000 * i, 1000 * i + (2000 if n == P0 else 500)])
    for path, ctr, col in ((fe, "FETCH_SIZE", 1), (wr, "WRITE_SIZE", 2)):
        with open(path, "w", newline="") as f:
            w = csv.writer(f)
            w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
            for i, row in enumerate(seq):
                # the copy reads and writes 1 GiB: FETCH_SIZE reads half of it here
                val = (512.0 * 1024 if col == 1 else 1024.0 * 1024) if row[0] == C else row[col] * 1024
                w.writerow([i + 1, row[0], ctr, val])
    line = {"metric": "m", "value": 1, "unit": "GB/s", "steps": 1, "warmup": 1,
            "detail": {"snapkv_votes_k_bytes (two passes over K)": 2 * 10.0 * 2 ** 20 * 2,
                       "kv_gather_bytes (read + write)": 2 * 6.0 * 2 ** 20 * 2,
                       "t_snapkv_votes_us (prefill, 32 observation queries)": 1.0,
                       "t_snapkv_select_us (pool 5, budget 2049)": 1.0,
                       "t_kv_gather_us (the 2049 listed rows into a draft cache, once per prompt)": 1.0}}
    bj = tmp_path / "b.json"
    bj.write_text(json.dumps(line) + "\n")
    text = bench.summarize_prefill(str(tr), str(fe), str(wr), str(bj), "cmd")
    rows = {r.split("|")[2].strip(): r for r in text.splitlines() if r.startswith("| `")}
    assert set(rows) == {"softmax statistics over K", "votes (K again, votes written)",
                         "pool, radix select, compaction", "listed rows into a draft cache"}
    # scale_fetch = 2: each pass reads 2 x 10 MiB = its algorithmic K bytes exactly
    assert rows["softmax statistics over K"].rstrip(" |").endswith("1.0000")
    assert "| 2.0 |" in rows["softmax statistics over K"]  # 2000 ns per dispatch
    # the selection's algorithmic read is what the votes pass wrote (4 MiB); it reads 8 MiB
    assert rows["pool, radix select, compaction"].rstrip(" |").endswith("2.0000")
    assert "bench_copy" not in text


def test_steps_summary_groups_by_grid(tmp_path):
    """--summarize steps: step kernels grouped by (kernel, grid size), so the
    one-token appends of the engine-shaped steps do not mix with the timed
    (gamma+1)-token append, whose read is compared with its algorithmic bytes."""
    import csv
    import json
    A, M, C = "void md::kv_append_kernel<true>(x)", "void md::argmax_partial_kernel<false, true>(x)", \
        "md::bench_copy_kernel(x)"
    seq = [(C, 1, 0, 0), (A, 81920, 2.0, 1.0), (A, 16384, 0.5, 0.25), (M, 573440, 8.0, 0.0),
           (A, 81920, 2.0, 1.0)]
    tr, fe, wr = tmp_path / "t.csv", tmp_path / "f.csv", tmp_path / "w.csv"
    with open(tr, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Grid_Size_X", "Start_Timestamp", "End_Timestamp"])
        for i, (n, g, _, _) in enumerate(seq):
            w.writerow([i + 1, n, g, 10000 * i, 10000 * i + (4000 if n == M else 1000)])
    for path, ctr, col in ((fe, "FETCH_SIZE", 2), (wr, "WRITE_SIZE", 3)):
        with open(path, "w", newline="") as f:
            w = csv.writer(f)
            w.writerow(["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
            for i, row in enumerate(seq):
                val = (512.0 * 1024 if col == 2 else 1024.0 * 1024) if row[0] == C else row[col] * 1024
                w.writerow([i + 1, row[0], row[1], ctr, val])
    line = {"metric": "m", "value": 1, "unit": "GB/s", "steps": 1, "warmup": 1,
            "detail": {"greedy_accept_logits_bytes": 16.0 * 2 ** 20,
                       "kv_append_bytes (read + write)": 2 * 4.0 * 2 ** 20,
                       "t_kv_append_us (gamma+1 tokens, paged)": 1.0,
                       "t_greedy_accept_us (fp32 logits, vocab 128256)": 1.0,
                       "t_kv_commit_us (lengths + 1024-slot ring)": 1.0}}
    bj = tmp_path / "b.json"
    bj.write_text(json.dumps(line) + "\n")
    text = bench.summarize_steps(str(tr), str(fe), str(wr), str(bj), "cmd")
    rows = [r for r in text.splitlines() if r.startswith("| `")]
    big = next(r for r in rows if "| 81920 |" in r)
    small = next(r for r in rows if "| 16384 |" in r)
    arg = next(r for r in rows if "argmax" in r)
    assert "| 2 |" in big and big.rstrip(" |").endswith("1.0000")  # 2 MiB x 2 = 4 MiB
    assert small.rstrip(" |").endswith("--")
    assert arg.rstrip(" |").endswith("1.0000") and "| 4.00 |" in arg
    assert "bench_copy" not in text


def test_issue_summary(tmp_path):
    """--summarize issue: per-instance means of the SQ issue and wait counters
    for the SnapKV passes and the bench's timed verify and draft; the wait
    shares are ratios to the wave-cycles, instructions are per wave."""
    import csv
    import json
    V = "void md::attn_partial_kernel<128, true, 2, true, false, 1, 1, true, 4>(md::AttnParams)"
    D = "void md::attn_partial_kernel<128, true, 2, true, false, 1, 2, false, 8>(md::AttnParams)"
    P0 = "void md::snapkv_pass_kernel<128, true, 1, true, true, 0, 64, 8>(md::SnapkvParams)"
    C = "md::bench_copy_kernel(x)"
    # counters per kernel: waves, wave-cycles, wait any, wait issue, valu active, valu insts,
    # transcendental, busy, gui active
    ctr = {V: (4, 1000, 380, 80, 250, 4000, 200, 10, 1000),
           D: (8, 1000, 330, 370, 300, 800, 40, 10, 1000),
           P0: (100, 1000, 400, 350, 136, 5000, 700, 10, 1000),
           C: (1, 10, 1, 1, 1, 1, 0, 1, 10)}
    seq = [C, V, D, V, D, P0, P0]
    path = tmp_path / "c.csv"
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, n in enumerate(seq):
            for c, v in zip(bench.ISSUE_COUNTERS, ctr[n]):
                w.writerow([i + 1, n, c, v])
    bj = tmp_path / "b.json"
    bj.write_text(json.dumps({"metric": "m", "value": 1, "unit": "GB/s", "steps": 1, "warmup": 1,
                              "detail": {}}) + "\n")
    text = bench.summarize_issue(str(path), str(bj), "cmd")
    rows = [r for r in text.splitlines() if r.startswith("| ") and not r.startswith("| kernel")]
    assert len(rows) == 3 and "bench_copy" not in text
    by = {("verify" if "verify (bench)" in r else "draft" if "draft (bench)" in r else "pass0"): r
          for r in rows}
    cells = [c.strip() for c in by["pass0"].split("|")[1:-1]]
    assert cells[1:] == ["2", "100", "0.400", "0.350", "0.1", "50", "7"]  # busy: 100 x 136 / 256 / 1000
    assert by["draft"].split("|")[5].strip() == "0.370"
    assert "kernel_source_sha256:" in text and "snapkv_source_sha256:" in text
