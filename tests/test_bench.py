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
    """The committed counter summaries carry the SHA-256 of attn.hip they were
    taken on; bench.py reports traffic and MFMA figures only while it matches."""
    traffic, mfma = bench.read_counters(), bench.read_mfma()
    assert traffic is not None and 8.5e9 < traffic < 8.7e9, "profiles/ are stale: re-profile"
    assert mfma is not None and 0 < mfma["util_pct"] < 100
    other = os.path.join(ROOT, "paper_2408_11049_amd", "csrc", "merge.hip")
    monkeypatch.setattr(bench, "KERNEL_SOURCE", other)
    assert bench.read_counters() is None and bench.read_mfma() is None
