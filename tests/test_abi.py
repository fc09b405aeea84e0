"""C ABI checks that need no GPU: the library loads, exports every symbol the
headers declare, agrees with the binding on the struct layout, and rejects
every malformed argument on the host before any launch.  No compute call is
made here (only calls that return an error before reaching a kernel)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2408_11049_amd as md

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("magicdec.h", "magicdec_bench.h")]


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(md.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return md.load_library()


def declared_functions():
    names = []
    for h in HEADERS:
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(md_[a-z_0-9]+)\s*\(", text, re.M)
    return sorted(set(names))


def test_headers_declare_the_entry_points():
    names = declared_functions()
    for n in ["md_verify_attn", "md_draft_attn", "md_merge_lse", "md_workspace_bytes",
              "md_status_str"]:
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", md.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (md_[a-z_0-9]+)$", out, re.M))
    declared = set(declared_functions())
    assert declared <= exported, f"declared but not exported: {sorted(declared - exported)}"
    assert set(md.EXPORTED) <= exported
    for n in declared:
        assert hasattr(lib, n)


def test_no_oracle_in_the_product_library():
    out = subprocess.run(["nm", "-D", md.LIB_PATH], capture_output=True, text=True).stdout
    assert "oracle" not in out
    deps = subprocess.run(["readelf", "-d", md.LIB_PATH], capture_output=True, text=True).stdout
    assert "liboracle" not in deps


def test_struct_layout_matches(lib):
    assert lib.md_attn_args_size() == ctypes.sizeof(md.MdAttnArgs)


def test_status_strings(lib):
    for s in range(5):
        assert lib.md_status_str(s)
    assert lib.md_status_str(99) == b"unknown status"


FAKE = 0x10000  # aligned, never dereferenced: validation rejects before any launch


def good_args(**over):
    a = md.MdAttnArgs()
    a.num_seqs, a.q_len, a.num_q_heads, a.num_kv_heads, a.head_dim = 4, 4, 8, 2, 128
    a.dtype = md.MD_BF16
    a.q = a.k = a.v = a.o = a.kv_lens = FAKE
    a.kv_stride_head = 128
    a.kv_stride_tok = 2 * 128
    a.kv_stride_blk = 64 * 2 * 128
    a.max_kv_len = 64
    for k, v in over.items():
        setattr(a, k, v)
    return a


BAD = [
    ("q_len 0", dict(q_len=0), md.MD_ERR_INVALID_ARG),
    ("q_len 17", dict(q_len=17), md.MD_ERR_INVALID_ARG),
    ("negative batch", dict(num_seqs=-1), md.MD_ERR_INVALID_ARG),
    ("Hq not multiple of Hkv", dict(num_q_heads=7), md.MD_ERR_INVALID_ARG),
    ("zero kv heads", dict(num_kv_heads=0), md.MD_ERR_INVALID_ARG),
    ("bad dtype", dict(dtype=7), md.MD_ERR_INVALID_ARG),
    ("max_kv_len < q_len", dict(max_kv_len=3), md.MD_ERR_INVALID_ARG),
    ("null q", dict(q=None), md.MD_ERR_INVALID_ARG),
    ("null k", dict(k=None), md.MD_ERR_INVALID_ARG),
    ("null v", dict(v=None), md.MD_ERR_INVALID_ARG),
    ("null o", dict(o=None), md.MD_ERR_INVALID_ARG),
    ("null kv_lens", dict(kv_lens=None), md.MD_ERR_INVALID_ARG),
    ("misaligned q", dict(q=FAKE + 8), md.MD_ERR_INVALID_ARG),
    ("misaligned k", dict(k=FAKE + 2), md.MD_ERR_INVALID_ARG),
    ("misaligned o", dict(o=FAKE + 4), md.MD_ERR_INVALID_ARG),
    ("misaligned error word", dict(err_word=FAKE + 2), md.MD_ERR_INVALID_ARG),
    ("token stride not 16 B", dict(kv_stride_tok=2 * 128 + 4), md.MD_ERR_INVALID_ARG),
    ("head stride overlaps", dict(kv_stride_head=64), md.MD_ERR_INVALID_ARG),
    ("negative stride", dict(kv_stride_blk=-8), md.MD_ERR_INVALID_ARG),
    ("page table without page size", dict(page_table=FAKE), md.MD_ERR_INVALID_ARG),
    ("page size without table", dict(page_size=16, max_pages_per_seq=4, num_pages=8),
     md.MD_ERR_INVALID_ARG),
    ("page size not power of two", dict(page_size=12, max_pages_per_seq=8, num_pages=8,
                                        page_table=FAKE), md.MD_ERR_INVALID_ARG),
    ("page table too narrow", dict(page_size=16, max_pages_per_seq=3, num_pages=8,
                                   page_table=FAKE), md.MD_ERR_INVALID_ARG),
    ("head_dim 96", dict(head_dim=96), md.MD_ERR_UNSUPPORTED),
    ("G*L > 64", dict(num_q_heads=34, num_kv_heads=2), md.MD_ERR_UNSUPPORTED),
    # 32-bit kernel indexing: per-lane row offsets, workgroup and row counts.
    ("token stride over 2^28", dict(kv_stride_tok=(1 << 28) + 8), md.MD_ERR_UNSUPPORTED),
    ("units over 2^31 - 1", dict(num_seqs=1 << 30), md.MD_ERR_UNSUPPORTED),
    ("rows over 4 (2^31 - 1)", dict(num_seqs=1 << 28), md.MD_ERR_UNSUPPORTED),
    ("max_kv_len within 64 of 2^31", dict(max_kv_len=2**31 - 60), md.MD_ERR_UNSUPPORTED),
]


@pytest.mark.parametrize("name,over,want", BAD, ids=[b[0] for b in BAD])
def test_verify_rejects(lib, name, over, want):
    assert lib.md_verify_attn(ctypes.byref(good_args(**over)), None) == want
    assert lib.md_draft_attn(ctypes.byref(good_args(**over)), 4, 16, None) == want
    if want == md.MD_ERR_UNSUPPORTED:  # the workspace queries refuse the same sizes
        a = ctypes.byref(good_args(**over))
        assert lib.md_workspace_bytes(a, md.MD_MODE_VERIFY, 0, 1) == 0
        assert lib.md_workspace_bytes_indexed(a, 64) == 0


def test_window_past_position_limit(lib):
    a = ctypes.byref(good_args())
    assert lib.md_draft_attn(a, 4, 2**31 - 60, None) == md.MD_ERR_UNSUPPORTED
    assert lib.md_draft_attn_indexed(a, FAKE, FAKE, 2**31 - 60, None) == md.MD_ERR_UNSUPPORTED
    assert lib.md_workspace_bytes(a, md.MD_MODE_DRAFT, 4, 2**31 - 60) == 0
    assert lib.md_workspace_bytes_indexed(a, 2**31 - 60) == 0


def test_indexed_rejects(lib):
    a = good_args()
    assert lib.md_draft_attn_indexed(ctypes.byref(a), None, FAKE, 8, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_draft_attn_indexed(ctypes.byref(a), FAKE, None, 8, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_draft_attn_indexed(ctypes.byref(a), FAKE, FAKE, 0, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_draft_attn_indexed(ctypes.byref(a), FAKE + 2, FAKE, 8, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_draft_attn_indexed(ctypes.byref(good_args(q_len=0)), FAKE, FAKE, 8, None) == \
        md.MD_ERR_INVALID_ARG
    assert lib.md_workspace_bytes_indexed(ctypes.byref(a), 0) == 0
    e = good_args(num_seqs=0, q=None, k=None, v=None, o=None, kv_lens=None)
    assert lib.md_draft_attn_indexed(ctypes.byref(e), None, None, 8, None) == md.MD_OK


def test_indexed_workspace_tracks_list_capacity(lib):
    a = good_args(num_seqs=1, num_kv_heads=1, num_q_heads=4, max_kv_len=1 << 17,
                  kv_stride_tok=128, kv_stride_blk=(1 << 17) * 128)
    small = lib.md_workspace_bytes_indexed(ctypes.byref(a), 1000)
    big = lib.md_workspace_bytes_indexed(ctypes.byref(a), 60000)
    assert small == 0 and big > 0


def good_snapkv(**over):
    a = md.MdSnapkvArgs()
    a.num_seqs, a.n_obs, a.num_q_heads, a.num_kv_heads, a.head_dim = 2, 32, 8, 2, 128
    a.dtype = md.MD_BF16
    a.q_obs = a.k = a.prompt_lens = a.votes = FAKE
    a.kv_stride_head, a.kv_stride_tok, a.kv_stride_blk = 128, 256, 100 * 256
    a.max_prompt_len, a.votes_stride = 100, 68
    for k, v in over.items():
        setattr(a, k, v)
    return a


SNAP_BAD = [
    ("n_obs 0", dict(n_obs=0), md.MD_ERR_INVALID_ARG),
    ("stride too small", dict(votes_stride=67), md.MD_ERR_INVALID_ARG),
    ("prompt shorter than window", dict(max_prompt_len=31), md.MD_ERR_INVALID_ARG),
    ("null votes", dict(votes=None), md.MD_ERR_INVALID_ARG),
    ("null q_obs", dict(q_obs=None), md.MD_ERR_INVALID_ARG),
    ("misaligned k", dict(k=FAKE + 4), md.MD_ERR_INVALID_ARG),
    ("rows over 256", dict(n_obs=65, max_prompt_len=200, votes_stride=200), md.MD_ERR_UNSUPPORTED),
    ("head_dim 80", dict(head_dim=80), md.MD_ERR_UNSUPPORTED),
    ("units over 2^31 - 1", dict(num_seqs=1 << 30), md.MD_ERR_UNSUPPORTED),
    ("no workspace", dict(), md.MD_ERR_WORKSPACE),
]


@pytest.mark.parametrize("name,over,want", SNAP_BAD, ids=[b[0] for b in SNAP_BAD])
def test_snapkv_votes_rejects(lib, name, over, want):
    assert lib.md_snapkv_votes(ctypes.byref(good_snapkv(**over)), None) == want


def test_snapkv_workspace_and_select_args(lib):
    assert lib.md_snapkv_workspace_bytes(ctypes.byref(good_snapkv())) > 0
    assert lib.md_snapkv_workspace_bytes(None) == 0
    sel = lib.md_snapkv_select
    assert sel(2, 2, FAKE, 68, FAKE, 32, 4, 64, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG  # even pool
    assert sel(2, 2, FAKE, 68, FAKE, 32, 5, 16, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG  # budget < n_obs
    assert sel(2, 2, None, 68, FAKE, 32, 5, 64, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sel(2, 0, FAKE, 68, FAKE, 32, 5, 64, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sel(0, 2, None, 68, None, 32, 5, 64, None, None, None) == md.MD_OK


def test_null_args(lib):
    assert lib.md_verify_attn(None, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_draft_attn(None, 1, 1, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_workspace_bytes(None, 0, 0, 1) == 0


@pytest.mark.parametrize("n_sink,window", [(-1, 8), (4, 0), (0, -3)])
def test_draft_rejects_budget(lib, n_sink, window):
    assert lib.md_draft_attn(ctypes.byref(good_args()), n_sink, window, None) == md.MD_ERR_INVALID_ARG


def test_empty_batch_is_a_noop(lib):
    a = good_args(num_seqs=0, q=None, k=None, v=None, o=None, kv_lens=None)
    assert lib.md_verify_attn(ctypes.byref(a), None) == md.MD_OK
    assert lib.md_draft_attn(ctypes.byref(a), 4, 8, None) == md.MD_OK


def test_workspace_required_and_checked(lib):
    # Few units and a long cache: the planner splits the range, needing workspace.
    a = good_args(num_seqs=1, num_kv_heads=1, num_q_heads=4, max_kv_len=1 << 16,
                  kv_stride_tok=128, kv_stride_blk=(1 << 16) * 128)
    need = lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1)
    assert need > 0
    assert lib.md_verify_attn(ctypes.byref(a), None) == md.MD_ERR_WORKSPACE
    a.workspace, a.workspace_bytes = FAKE, need - 1
    assert lib.md_verify_attn(ctypes.byref(a), None) == md.MD_ERR_WORKSPACE
    a.workspace, a.workspace_bytes = FAKE + 16, need
    assert lib.md_verify_attn(ctypes.byref(a), None) == md.MD_ERR_WORKSPACE  # not 256-aligned


def test_workspace_zero_when_units_fill_the_device(lib, monkeypatch):
    # 64 sequences x 8 kv heads = 512 units >= two per compute unit: one pass
    # (the balanced verify off; on, it keeps partials of the groups it cuts).
    monkeypatch.setenv("MD_BALANCED", "1")
    a = good_args(num_seqs=64, num_kv_heads=8, num_q_heads=32, q_len=5, max_kv_len=32768)
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == 0
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_DRAFT, 16, 1008) == 0


@pytest.mark.parametrize("B,Hkv,Hq,L,hp,default_on", [
    (64, 8, 32, 5, 2, True),     # 256 head pairs: one per compute unit
    (128, 3, 12, 4, 1, True),    # odd head count: single heads, 384 groups
    (256, 8, 32, 3, 2, False),   # 1024 pairs, four per unit: dispatch balances
    (256, 8, 32, 5, 2, False),
])
def test_balanced_verify_workspace(lib, monkeypatch, B, Hkv, Hq, L, hp, default_on):
    """The balanced verify (the units fill the device, lengths up to 32768,
    at most two head groups per compute unit unless forced): one 8-byte
    counter per head group, then two partial slots per workgroup (its range's
    first and last pieces) of hp * G * L rows; one workgroup per compute unit
    (256 on this host)."""
    a = good_args(num_seqs=B, num_kv_heads=Hkv, num_q_heads=Hq, q_len=L, max_kv_len=32768,
                  kv_stride_tok=Hkv * 128, kv_stride_blk=32768 * Hkv * 128)
    groups, R = B * Hkv // hp, Hq // Hkv * L
    nw = 256
    up = lambda x: (x + 255) // 256 * 256
    want = up(groups * 8) + up(2 * nw * hp * R * 128 * 4) + up(2 * nw * hp * R * 4)
    monkeypatch.delenv("MD_BALANCED", raising=False)
    got = lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1)
    assert got == (want if default_on else 0)
    monkeypatch.setenv("MD_BALANCED", "2")
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == want
    monkeypatch.setenv("MD_BALANCED", "1")
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == 0


@pytest.mark.parametrize("forced", [None, "2"])
def test_balanced_verify_not_beyond_three_row_tiles(lib, monkeypatch, forced):
    """64 query rows per kv head (G = 4, q_len = 16: four row tiles) stay on the
    single-pass plan, forced or not: the balanced instances are compiled only
    up to three row tiles of bf16, where their piece loop does not spill."""
    if forced:
        monkeypatch.setenv("MD_BALANCED", forced)
    else:
        monkeypatch.delenv("MD_BALANCED", raising=False)
    a = good_args(num_seqs=64, num_kv_heads=8, num_q_heads=32, q_len=16, max_kv_len=32768,
                  kv_stride_tok=8 * 128, kv_stride_blk=32768 * 8 * 128)
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == 0
    a.q_len = 12  # 48 rows, three row tiles: balanced
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) > 0


def _split_bytes(n_chunks, n_rows, d, groups):
    """A split plan's workspace: one 8-byte arrival counter per head group,
    then the partial O and lse, each part 256-byte aligned."""
    up = lambda x: (x + 255) // 256 * 256
    return up(groups * 8) + up(n_chunks * n_rows * d * 4) + up(n_chunks * n_rows * 4)


@pytest.mark.parametrize("B,S,hp", [
    (1, 131072, 1),   # pairs would cut 128k tokens into 64 chunks of 2048: one head per group
    (4, 65536, 2),    # 16 pairs x 16 chunks of 4096 tokens: pairs
    (16, 4096, 1),    # 64 pairs x 4 chunks of 1024: one head
    (16, 16384, 2),   # 64 pairs x 4 chunks of 4096: pairs
])
def test_plan_pairs_heads_only_where_they_pay(lib, B, S, hp):
    """The verify split as md_workspace_bytes reveals it (256 compute units on
    this host): the workgroups are B * 8 / hp, and the range is cut into
    ceil(256 / workgroups) chunks, at least 1024 tokens each."""
    a = good_args(num_seqs=B, num_kv_heads=8, num_q_heads=32, q_len=5, max_kv_len=S,
                  kv_stride_tok=8 * 128, kv_stride_blk=S * 8 * 128)
    groups = B * 8 // hp
    n_chunks = min(-(-256 // groups), -(-S // 1024))
    chunk = -(-(-(-S // n_chunks)) // 32) * 32
    n_chunks = -(-S // chunk)
    got = lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1)
    assert got == _split_bytes(n_chunks, B * 5 * 32, 128, groups), (got, n_chunks)


def test_tuning_overrides_are_read_per_call(lib, monkeypatch):
    """MD_HEADS_PER_WG changes the plan of the very next call (B = 16,
    S = 16384: 64 head pairs in 4 chunks of 4096, or 128 single heads in 2
    chunks), and unsetting it restores the default."""
    a = good_args(num_seqs=16, num_kv_heads=8, num_q_heads=32, q_len=5, max_kv_len=16384,
                  kv_stride_tok=8 * 128, kv_stride_blk=16384 * 8 * 128)
    rows = 16 * 5 * 32
    monkeypatch.delenv("MD_HEADS_PER_WG", raising=False)
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == _split_bytes(4, rows, 128, 64)
    monkeypatch.setenv("MD_HEADS_PER_WG", "1")
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == _split_bytes(2, rows, 128, 128)
    monkeypatch.setenv("MD_HEADS_PER_WG", "7")  # out of range: ignored
    assert lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1) == _split_bytes(4, rows, 128, 64)


def test_workspace_draft_smaller_than_verify(lib):
    a = good_args(num_seqs=2, num_kv_heads=1, num_q_heads=8, q_len=4, max_kv_len=1 << 17,
                  kv_stride_tok=128, kv_stride_blk=(1 << 17) * 128)
    wv = lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_VERIFY, 0, 1)
    wd = lib.md_workspace_bytes(ctypes.byref(a), md.MD_MODE_DRAFT, 64, 1984)
    assert 0 <= wd < wv


MERGE_BAD = [
    ("no parts", dict(n_parts=0), md.MD_ERR_INVALID_ARG),
    ("negative rows", dict(n_rows=-1), md.MD_ERR_INVALID_ARG),
    ("bad dtype", dict(dt=3), md.MD_ERR_INVALID_ARG),
    ("head_dim 32", dict(d=32), md.MD_ERR_UNSUPPORTED),
    ("null o_parts", dict(op=None), md.MD_ERR_INVALID_ARG),
    ("null o", dict(o=None), md.MD_ERR_INVALID_ARG),
    ("misaligned lse", dict(lse=FAKE + 4), md.MD_ERR_INVALID_ARG),
    ("rows over 4 (2^31 - 1)", dict(n_rows=4 * 2**31), md.MD_ERR_UNSUPPORTED),
]


@pytest.mark.parametrize("name,over,want", MERGE_BAD, ids=[m[0] for m in MERGE_BAD])
def test_merge_rejects(lib, name, over, want):
    kw = dict(n_parts=2, n_rows=8, d=128, dt=0, op=FAKE, lp=FAKE, o=FAKE, lse=FAKE)
    kw.update(over)
    assert lib.md_merge_lse(kw["n_parts"], kw["n_rows"], kw["d"], kw["dt"], kw["op"], kw["lp"],
                            kw["o"], kw["lse"], None) == want


def test_merge_zero_rows_is_a_noop(lib):
    assert lib.md_merge_lse(3, 0, 64, 0, None, None, None, None, None) == md.MD_OK


def test_bench_helpers_reject_bad_args(lib):
    assert lib.md_bench_stream_read(None, 16, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_bench_stream_read(FAKE, 17, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_bench_copy(FAKE, FAKE + 4, 32, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_bench_fill(FAKE + 8, 32, 0, None) == md.MD_ERR_INVALID_ARG


def good_cache(**over):
    c = md.MdKvCache()
    c.num_seqs, c.num_kv_heads, c.head_dim, c.dtype = 2, 2, 128, md.MD_BF16
    c.k, c.v = FAKE, FAKE + 0x1000
    c.kv_stride_blk, c.kv_stride_tok, c.kv_stride_head = 64 * 2 * 128, 2 * 128, 128
    c.capacity = 64
    for k, v in over.items():
        setattr(c, k, v)
    return c


APPEND_BAD = [
    ("negative n_new", {}, -1),
    ("zero heads", {"num_kv_heads": 0}, 3),
    ("bad dtype", {"dtype": 7}, 3),
    ("row not 16-byte multiple", {"head_dim": 4}, 3),
    ("stride not 16-byte multiple", {"kv_stride_tok": 100}, 3),
    ("zero capacity", {"capacity": 0}, 3),
    ("table without page size", {"page_table": FAKE}, 3),
    ("page size not a power of two", {"page_size": 12, "page_table": FAKE,
                                      "max_pages_per_seq": 4, "num_pages": 8}, 3),
    ("paged without pages", {"page_size": 16, "page_table": FAKE, "max_pages_per_seq": 4,
                             "num_pages": 0}, 3),
    ("misaligned cache", {"k": FAKE + 4}, 3),
    ("null cache", {"v": None}, 3),
]


@pytest.mark.parametrize("name,over,n_new", APPEND_BAD, ids=[b[0] for b in APPEND_BAD])
def test_kv_append_rejects(lib, name, over, n_new):
    c = good_cache(**over)
    st = lib.md_kv_append(ctypes.byref(c), n_new, FAKE, FAKE, FAKE, FAKE + 64, None)
    assert st == md.MD_ERR_INVALID_ARG


def test_kv_append_pointer_rules(lib):
    c = good_cache()
    ap = lib.md_kv_append
    assert ap(None, 3, FAKE, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert ap(ctypes.byref(c), 3, FAKE, FAKE, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG  # lens_out == pos0
    assert ap(ctypes.byref(c), 3, FAKE, FAKE, FAKE, FAKE + 4, None) == md.MD_ERR_INVALID_ARG  # overlap
    assert ap(ctypes.byref(c), 3, FAKE, FAKE, FAKE + 4, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert ap(ctypes.byref(c), 3, FAKE + 8, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert ap(ctypes.byref(c), 3, FAKE, FAKE, None, None, None) == md.MD_ERR_INVALID_ARG
    assert ap(ctypes.byref(c), 3, FAKE, FAKE, FAKE + 2, None, None) == md.MD_ERR_INVALID_ARG
    # nothing to write: no launch, no pointer read
    assert ap(ctypes.byref(c), 0, None, None, None, None, None) == md.MD_OK
    assert ap(ctypes.byref(good_cache(num_seqs=0)), 5, None, None, None, None, None) == md.MD_OK


GATHER_BAD = [
    ("heads differ", {}, {"num_kv_heads": 4}),
    ("head_dim differs", {}, {"head_dim": 64, "kv_stride_head": 64}),
    ("dtype differs", {}, {"dtype": md.MD_F32}),
    ("sequences differ", {}, {"num_seqs": 3}),
    ("bad destination", {"capacity": 0}, {}),
    ("destination shorter than the lists", {"capacity": 15}, {}),
    ("paged destination shorter than the lists",
     {"capacity": 0, "page_size": 4, "page_table": FAKE + 0x2000, "max_pages_per_seq": 3,
      "num_pages": 8}, {}),
    ("bad source", {}, {"kv_stride_tok": 100}),
    ("misaligned destination", {"k": FAKE + 4}, {}),
    ("null source", {}, {"v": None}),
]


@pytest.mark.parametrize("name,dst_over,src_over", GATHER_BAD, ids=[b[0] for b in GATHER_BAD])
def test_kv_gather_rejects(lib, name, dst_over, src_over):
    d, s = good_cache(**dst_over), good_cache(**src_over)
    st = lib.md_kv_gather(ctypes.byref(d), ctypes.byref(s), FAKE, 16, FAKE + 64, FAKE + 128,
                          FAKE + 192, None)
    assert st == md.MD_ERR_INVALID_ARG


def test_kv_gather_pointer_rules(lib):
    d, s = good_cache(), good_cache()
    g = lib.md_kv_gather
    assert g(None, ctypes.byref(s), FAKE, 16, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), None, FAKE, 16, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), ctypes.byref(s), FAKE, 0, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), ctypes.byref(s), None, 16, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), ctypes.byref(s), FAKE, 16, None, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), ctypes.byref(s), FAKE, 16, FAKE, None, None, None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), ctypes.byref(s), FAKE + 2, 16, FAKE, FAKE, None, None) == md.MD_ERR_INVALID_ARG
    # dst_lens overlapping idx_len or src_lens (two sequences: 8 bytes each)
    assert g(ctypes.byref(d), ctypes.byref(s), FAKE, 16, FAKE + 64, FAKE + 128, FAKE + 68,
             None) == md.MD_ERR_INVALID_ARG
    assert g(ctypes.byref(d), ctypes.byref(s), FAKE, 16, FAKE + 64, FAKE + 128, FAKE + 124,
             None) == md.MD_ERR_INVALID_ARG
    # nothing to gather: no launch, no pointer read
    e = good_cache(num_seqs=0)
    assert g(ctypes.byref(e), ctypes.byref(good_cache(num_seqs=0)), None, 16, None, None, None,
             None) == md.MD_OK


def test_greedy_accept_args(lib):
    ga = lib.md_greedy_accept
    ws = lib.md_greedy_accept_workspace_bytes(64, 4, 128256)
    assert ws > 0 and ws % 256 == 0
    assert lib.md_greedy_accept_workspace_bytes(64, -1, 128256) == 0
    assert lib.md_greedy_accept_workspace_bytes(64, 4, 0) == 0
    ok = (64, 4, 128256, md.MD_F32, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws, None)

    def call(**over):
        names = ["B", "n_draft", "vocab", "dtype", "logits", "draft", "accepted", "tokens",
                 "target", "ws", "ws_bytes", "stream"]
        args = dict(zip(names, ok))
        args.update(over)
        return ga(*[args[n] for n in names])

    assert call(n_draft=-1) == md.MD_ERR_INVALID_ARG
    assert call(n_draft=1024) == md.MD_ERR_INVALID_ARG
    assert call(vocab=0) == md.MD_ERR_INVALID_ARG
    assert call(dtype=5) == md.MD_ERR_INVALID_ARG
    assert call(logits=None) == md.MD_ERR_INVALID_ARG
    assert call(logits=FAKE + 4) == md.MD_ERR_INVALID_ARG
    assert call(draft=None) == md.MD_ERR_INVALID_ARG
    assert call(tokens=None) == md.MD_ERR_INVALID_ARG
    assert call(accepted=FAKE + 1) == md.MD_ERR_INVALID_ARG
    assert call(ws=None) == md.MD_ERR_WORKSPACE
    assert call(ws_bytes=ws - 1) == md.MD_ERR_WORKSPACE
    assert call(ws=FAKE + 16) == md.MD_ERR_WORKSPACE
    assert call(B=0, logits=None, draft=None, accepted=None, tokens=None, ws=None) == md.MD_OK


def test_accept_plan_splits_long_rows(lib):
    # Few rows: more chunks per row (more workspace); the workspace stays tiny.
    few = lib.md_greedy_accept_workspace_bytes(1, 4, 128256)
    many = lib.md_greedy_accept_workspace_bytes(256, 4, 128256)
    assert 0 < few <= 2 * 256 * ((5 * 64 * 4 + 255) // 256)
    assert many > 0 and many < 1 << 20


def test_kv_commit_args(lib):
    kc = lib.md_kv_commit
    assert kc(2, 0, FAKE, FAKE, 0, None, 0, 0, 0, None) == md.MD_ERR_INVALID_ARG  # q_len < 1
    assert kc(2, 5, None, FAKE, 0, None, 0, 0, 0, None) == md.MD_ERR_INVALID_ARG
    assert kc(2, 5, FAKE, None, 0, None, 0, 0, 0, None) == md.MD_ERR_INVALID_ARG
    assert kc(2, 5, FAKE, FAKE, 0, FAKE, 64, 0, 64, None) == md.MD_ERR_INVALID_ARG  # no heads
    assert kc(2, 5, FAKE, FAKE, 2, FAKE, 64, 16, 49, None) == md.MD_ERR_INVALID_ARG  # past stride
    assert kc(2, 5, FAKE, FAKE, 2, FAKE, 64, -1, 8, None) == md.MD_ERR_INVALID_ARG
    assert kc(2, 5, FAKE, FAKE, 2, FAKE, 64, 16, 0, None) == md.MD_ERR_INVALID_ARG
    assert kc(0, 5, None, None, 2, None, 0, 0, 0, None) == md.MD_OK


def test_streaming_list_args(lib):
    sl = lib.md_streaming_list
    assert sl(2, 0, FAKE, 4, 8, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sl(2, 2, FAKE, -1, 8, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sl(2, 2, FAKE, 4, 0, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sl(2, 2, None, 4, 8, FAKE, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sl(2, 2, FAKE, 4, 8, FAKE + 2, FAKE, None) == md.MD_ERR_INVALID_ARG
    assert sl(0, 2, None, 4, 8, None, None, None) == md.MD_OK


def test_readme_c_example_compiles():
    """The C example in README.md uses the header's names and types as they
    are (gcc, syntax and type checks only; read from stdin)."""
    text = open(os.path.join(ROOT, "README.md")).read()
    start = text.index("```c") + 4
    snippet = text[start:text.index("```", start)]
    body = snippet.replace('#include "magicdec.h"', "")
    src = ('#include <stdio.h>\n#include <stdint.h>\n#include "magicdec.h"\n'
           "int demo(int B, int gamma, int Hq, int Hkv, int64_t S_alloc, int S_max,\n"
           "         const void* d_q, const void* d_k, const void* d_v, const int32_t* d_kv_lens,\n"
           "         void* d_o, float* d_lse, void* d_ws, void* stream) {\n"
           + body + "\n  return st;\n}\n")
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-fsyntax-only", "-x", "c",
                        "-I", os.path.join(ROOT, "include"), "-"],
                       input=src, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_struct_layouts_match_the_header(tmp_path):
    """Offsets and sizes of every C-ABI struct, as gcc lays them out from the
    header, equal the binding's ctypes mirrors."""
    structs = {"md_attn_args": md.MdAttnArgs, "md_snapkv_args": md.MdSnapkvArgs,
               "md_kv_cache": md.MdKvCache}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "magicdec.h"',
             "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'  printf("{name} size %zu\\n", sizeof({name}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{name} {f} %zu\\n", offsetof({name}, {f}));')
    lines.append("  return 0;\n}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out.splitlines()}
    for name, cls in structs.items():
        assert got[(name, "size")] == ctypes.sizeof(cls), name
        for f, _ in cls._fields_:
            assert got[(name, f)] == getattr(cls, f).offset, (name, f)


def test_noalloc_header_limit_matches_binding():
    text = open(HEADERS[0]).read()
    m = re.search(r"#define MD_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == md.MD_NOALLOC_SCRATCH_BYTES


def test_noalloc_scratch_holds_every_plan():
    """On a 256-compute-unit device (this host's fallback, and MI355X) every
    split plan fits the static scratch: a sweep over batch, heads, query rows
    (up to 64), head dims and lengths up to 2^30, verify and draft."""
    worst = 0
    for B in (1, 2, 3, 5, 8, 16, 31, 64, 127):
        for Hkv, Hq in ((1, 64), (2, 32), (8, 64), (8, 32), (4, 4), (3, 12)):
            for L in (1, 4, 16):
                if (Hq // Hkv) * L > 64:
                    continue
                for d in (64, 128):
                    for S in (4096, 65536, 1 << 20, 1 << 30):
                        a = good_args(num_seqs=B, num_kv_heads=Hkv, num_q_heads=Hq, q_len=L,
                                      head_dim=d, max_kv_len=S, kv_stride_tok=Hkv * d,
                                      kv_stride_head=d, kv_stride_blk=S * Hkv * d)
                        for mode, ns, w in ((0, 0, 1), (1, 64, S // 2)):
                            worst = max(worst, lib_bytes(a, mode, ns, w))
    assert 0 < worst <= md.MD_NOALLOC_SCRATCH_BYTES, worst


def lib_bytes(a, mode, ns, w):
    return md.load_library().md_workspace_bytes(ctypes.byref(a), mode, ns, w)


def test_noalloc_refuses_before_any_hip_call(lib, monkeypatch):
    """Argument errors and a plan larger than the scratch come back before
    the library touches a device (this host has none)."""
    a = good_args(num_seqs=3, num_kv_heads=2, num_q_heads=32, q_len=4, max_kv_len=1 << 21,
                  kv_stride_tok=2 * 128, kv_stride_blk=(1 << 21) * 2 * 128)
    assert lib.md_attn_noalloc(None, 0, 0, 1, None) == md.MD_ERR_INVALID_ARG
    assert lib.md_attn_noalloc(ctypes.byref(a), 2, 0, 1, None) == md.MD_ERR_INVALID_ARG
    # Four workgroups per compute unit (a measurement override) make this plan
    # need more than the scratch: 3 head pairs x 342 chunks x 384 rows.
    monkeypatch.setenv("MD_SLOTS_SCALE", "4")
    need = lib.md_workspace_bytes(ctypes.byref(a), 0, 0, 1)
    assert need > md.MD_NOALLOC_SCRATCH_BYTES
    assert lib.md_attn_noalloc(ctypes.byref(a), 0, 0, 1, None) == md.MD_ERR_WORKSPACE
