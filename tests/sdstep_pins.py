"""Pins of the speculative-step oracle (oracle/sdstep.py) against facts that
do not come from it.

Each ``pin_*`` takes the oracle module (``mod=None`` is the real one) and
raises AssertionError on a mismatch; ``test_oracle_pins.py`` runs them on the
real module and ``test_oracle_mutants.py`` on copies with a planted mistake.

  accept_eq1       Eq. 1: with drafts accepted independently with probability
                   alpha, the exact expectation of accepted + 1 over all 2^gamma
                   match patterns is (1 - alpha^(gamma+1)) / (1 - alpha) and
                   the geometric sum of alpha^k, k = 0..gamma.
  accept_cases     hand-made steps: the leading matching run, the bonus at the
                   first mismatch or after the last draft.
  argmax_*         brute force over each row (first index of the largest value),
                   ties, NaN and -inf rows, bf16 bit patterns.
  append_*         paged == contiguous on the same logical positions, read back
                   through an independent gather; nothing else changes.
  commit/ring_*    C' = C + a + 1; after any sequence of steps the rolling
                   list holds exactly the sinks and the last W committed
                   positions, each once (the StreamingLLM cache, Sec. 5.1).
  gather_*         a hand-worked gather (unusable entries and an over-long
                   idx_len included); paged == contiguous read back through
                   an independent gather; and attention over the gathered
                   cache with the speculated rows appended equals the listed
                   draft over the full cache (the fp64 attention oracles,
                   pinned on their own).
"""
import itertools

import numpy as np

import oracle.sdstep as real


def _m(mod):
    return real if mod is None else mod


def _logits_with_targets(rng, target, V):
    """[B, L, V] float32 logits whose unique row maximum sits at target."""
    B, L = target.shape
    x = rng.standard_normal((B, L, V)).astype(np.float32)
    for b in range(B):
        for i in range(L):
            x[b, i, target[b, i]] = np.abs(x[b, i]).max() + 1.0
    return x


def pin_accept_eq1(mod=None):
    s = _m(mod)
    rng = np.random.default_rng(11)
    V = 8
    for gamma in (1, 2, 3, 5):
        target = rng.integers(0, V, size=(1, gamma + 1))
        logits = _logits_with_targets(rng, target, V)
        for alpha in (0.3, 0.8, 0.93):
            e = 0.0
            for pattern in itertools.product((0, 1), repeat=gamma):
                draft = np.where(np.array(pattern, bool), target[0, :gamma],
                                 (target[0, :gamma] + 1) % V)[None]
                acc, tokens, _ = s.greedy_accept(logits, draft)
                m = sum(pattern)
                e += alpha ** m * (1 - alpha) ** (gamma - m) * (int(acc[0]) + 1)
            closed = (1 - alpha ** (gamma + 1)) / (1 - alpha)
            geometric = sum(alpha ** k for k in range(gamma + 1))
            assert abs(e - closed) < 1e-12, (gamma, alpha, e, closed)
            assert abs(s.expected_tokens(gamma, alpha) - geometric) < 1e-12
        assert s.expected_tokens(gamma, 1.0) == gamma + 1


def pin_accept_cases(mod=None):
    s = _m(mod)
    rng = np.random.default_rng(12)
    V, gamma = 16, 4
    target = np.array([[3, 5, 7, 9, 11], [3, 5, 7, 9, 11], [0, 1, 2, 3, 4], [15, 14, 13, 12, 10]])
    logits = _logits_with_targets(rng, target, V)
    draft = np.array([[3, 5, 7, 9],       # all accepted: bonus after the last draft
                      [4, 5, 7, 9],       # first draft wrong: only the bonus
                      [0, 1, 9, 3],       # a later match after a mismatch does not count
                      [15, 14, 13, 0]])   # mismatch at the last draft
    acc, tokens, tgt = s.greedy_accept(logits, draft)
    assert np.array_equal(tgt, target)
    assert acc.tolist() == [4, 0, 2, 3]
    assert tokens.tolist() == [[3, 5, 7, 9, 11], [3, -1, -1, -1, -1], [0, 1, 2, -1, -1],
                               [15, 14, 13, 12, -1]]


def _first_max(row):
    best, arg = None, 0
    for v_i, v in enumerate(row):
        v = -np.inf if np.isnan(v) else float(v)
        if best is None or v > best:
            best, arg = v, v_i
    return arg


def pin_argmax_brute(mod=None):
    s = _m(mod)
    rng = np.random.default_rng(13)
    x = rng.integers(-3, 4, size=(3, 4, 37)).astype(np.float32)  # heavy ties
    x[0, 1, 5] = np.nan
    x[1, 2, :] = -np.inf
    x[1, 3, :] = np.nan
    x[2, 0, :3] = np.nan
    x[2, 0, 3:] = -np.inf
    x[2, 1, 0] = np.nan
    x[2, 1, 1:] = -2.0
    got = s.target_tokens(x)
    ref = np.array([[_first_max(x[b, i]) for i in range(4)] for b in range(3)])
    assert np.array_equal(got, ref), (got, ref)
    assert got[1, 2] == 0 and got[1, 3] == 0 and got[2, 0] == 0 and got[2, 1] == 1


def pin_argmax_bf16(mod=None):
    s = _m(mod)
    # bf16 bit patterns: 0x3F80 = 1.0, 0x3F81 = 1.0078125, 0xBF80 = -1.0,
    # 0x4000 = 2.0, 0x7F80 = +inf, 0xFF80 = -inf
    bits = np.array([[[0x3F80, 0x3F81, 0xBF80, 0x3F81]],
                     [[0xFF80, 0xBF80, 0x4000, 0x3F80]],
                     [[0x3F80, 0x7F80, 0x4000, 0x7F80]]], dtype=np.uint16)
    assert s.target_tokens(bits).ravel().tolist() == [1, 2, 1]
    assert s.widen(np.array([0x3F81], np.uint16))[0] == 1.0078125


def _gather(cache, b, j, page_size, page_table):
    """Independent logical read: position j of sequence b."""
    if page_size == 0:
        return cache[b, j]
    return cache[page_table[b][j // page_size], j % page_size]


def pin_append_paged_contiguous(mod=None):
    s = _m(mod)
    rng = np.random.default_rng(14)
    B, Hkv, d, ps = 3, 2, 8, 4
    lens = np.array([5, 12, 1])
    n = 3
    S_alloc = 16
    cont = rng.standard_normal((B, S_alloc, Hkv, d)).astype(np.float32)
    pages = rng.permutation(B * (S_alloc // ps)).reshape(B, S_alloc // ps)
    paged = np.zeros((B * S_alloc // ps, ps, Hkv, d), np.float32)
    for b in range(B):
        for j in range(S_alloc):
            paged[pages[b, j // ps], j % ps] = cont[b, j]
    new = rng.standard_normal((B, n, Hkv, d)).astype(np.float32)
    c2 = s.kv_append(cont, new, lens)
    p2 = s.kv_append(paged, new, lens, page_size=ps, page_table=pages)
    for b in range(B):
        for j in range(S_alloc):
            want = new[b, j - lens[b]] if lens[b] <= j < lens[b] + n else cont[b, j]
            assert np.array_equal(_gather(c2, b, j, 0, None), want), (b, j)
            assert np.array_equal(_gather(p2, b, j, ps, pages), want), (b, j)
    # bf16 bit patterns move unchanged
    bits = rng.integers(0, 1 << 16, size=(B, n, Hkv, d), dtype=np.uint16)
    cb = s.kv_append(np.zeros((B, S_alloc, Hkv, d), np.uint16), bits, lens)
    assert np.array_equal(cb[1, 12:15], bits[1])


def pin_commit_lengths(mod=None):
    s = _m(mod)
    assert s.kv_commit([100, 7, 0], [4, 0, 2]).tolist() == [105, 8, 3]


def _ring_contents(idx_row):
    vals = idx_row[idx_row >= 0]
    assert len(np.unique(vals)) == len(vals), "a position listed twice"
    return set(int(v) for v in vals)


def pin_ring_window(mod=None):
    s = _m(mod)
    rng = np.random.default_rng(15)
    for n_sink, W, gamma in [(4, 8, 3), (16, 64, 4), (2, 3, 5), (0, 5, 2)]:
        prompt = np.array([3, n_sink + W + 7, 40, n_sink + 1])
        B, Hkv = len(prompt), 2
        idx = s.streaming_list(prompt, Hkv, n_sink, W)
        C = prompt.copy()
        sinks = np.minimum(prompt, n_sink)  # a prompt shorter than n_sink has fewer sinks
        for step in range(25):
            for b in range(B):
                for h in range(Hkv):
                    want = set(range(sinks[b])) | set(range(max(sinks[b], C[b] - W), C[b]))
                    assert _ring_contents(idx[b, h]) == want, (n_sink, W, step, b, sorted(want))
            acc = rng.integers(0, gamma + 1, size=B)
            idx = s.ring_commit(idx, C, acc, n_sink, W)
            C = s.kv_commit(C, acc)


def pin_gather_by_hand(mod=None):
    s = _m(mod)
    # src[b, t, h, 0] = 100 b + 10 t + h + 1 (no zeros, so a zero row shows).
    src = np.zeros((2, 4, 2, 1), np.float32)
    for b in range(2):
        for t in range(4):
            for h in range(2):
                src[b, t, h, 0] = 100 * b + 10 * t + h + 1
    idx = np.array([[[3, 0, 2], [-1, 2, 5]],
                    [[1, 0, 9], [2, 3, 0]]], np.int32)
    src_lens = [4, 3]
    want = np.full((2, 4, 2, 1), -7.0, np.float32)
    # sequence 0: three entries; -1 and 5 (>= 4) are unusable -> zeros
    want[0, 0, :, 0] = [31, 0]
    want[0, 1, :, 0] = [1, 22]
    want[0, 2, :, 0] = [21, 0]
    # sequence 1: two entries; position 3 is not below src_lens = 3 -> zero
    want[1, 0, :, 0] = [111, 122]
    want[1, 1, :, 0] = [101, 0]
    for idx_len in ([3, 2], [5, 2]):  # idx_len past the stride is clamped
        got, n = s.kv_gather(np.full((2, 4, 2, 1), -7.0, np.float32), src, idx, idx_len, src_lens)
        assert np.array_equal(got, want), (idx_len, got[..., 0])
        assert list(n) == [3, 2], n


def pin_gather_paged_contiguous(mod=None):
    s = _m(mod)
    rng = np.random.default_rng(16)
    B, Hkv, d, ps, S_alloc, D_alloc, stride = 3, 2, 4, 4, 16, 8, 8
    src = rng.standard_normal((B, S_alloc, Hkv, d)).astype(np.float32)
    spages = rng.permutation(B * (S_alloc // ps)).reshape(B, S_alloc // ps)
    src_p = np.zeros((B * S_alloc // ps, ps, Hkv, d), np.float32)
    for b in range(B):
        for j in range(S_alloc):
            src_p[spages[b, j // ps], j % ps] = src[b, j]
    dpages = rng.permutation(B * (D_alloc // ps)).reshape(B, D_alloc // ps)
    idx = rng.integers(-2, S_alloc + 2, size=(B, Hkv, stride)).astype(np.int32)
    idx_len, src_lens = np.array([8, 3, 0]), np.array([16, 9, 5])
    dst = rng.standard_normal((B, D_alloc, Hkv, d)).astype(np.float32)
    dst_p = np.zeros((B * D_alloc // ps, ps, Hkv, d), np.float32)
    for b in range(B):
        for j in range(D_alloc):
            dst_p[dpages[b, j // ps], j % ps] = dst[b, j]
    c2, n = s.kv_gather(dst, src, idx, idx_len, src_lens)
    p2, _ = s.kv_gather(dst_p, src_p, idx, idx_len, src_lens, src_page_size=ps,
                        src_page_table=spages, dst_page_size=ps, dst_page_table=dpages)
    for b in range(B):
        for j in range(D_alloc):
            for h in range(Hkv):
                if j < n[b]:
                    p = idx[b, h, j]
                    want = src[b, p, h] if 0 <= p < src_lens[b] else np.zeros(d, np.float32)
                else:
                    want = dst[b, j, h]
                assert np.array_equal(_gather(c2, b, j, 0, None)[h], want), (b, j, h)
                assert np.array_equal(_gather(p2, b, j, ps, dpages)[h], want), (b, j, h)


def pin_gather_listed_draft_equivalence(mod=None):
    import oracle

    s = _m(mod)
    rng = np.random.default_rng(17)
    B, L, Hq, Hkv, d, S_alloc, stride = 2, 3, 4, 2, 16, 48, 12
    S = np.array([40, 25], np.int32)
    q = rng.standard_normal((B, L, Hq, d)).astype(np.float32)
    k = rng.standard_normal((B, S_alloc, Hkv, d)).astype(np.float32)
    v = rng.standard_normal((B, S_alloc, Hkv, d)).astype(np.float32)
    n = np.array([10, 6], np.int32)
    idx = np.full((B, Hkv, stride), -1, np.int32)
    for b in range(B):
        for h in range(Hkv):
            idx[b, h, : n[b]] = np.sort(rng.choice(S[b] - L, size=n[b], replace=False))
    ro, rl = oracle.indexed(q, k, v, S, idx, n)
    kc, nk = s.kv_gather(np.zeros((B, 16, Hkv, d), np.float32), k, idx, n, S - L)
    vc, _ = s.kv_gather(np.zeros((B, 16, Hkv, d), np.float32), v, idx, n, S - L)
    spec_k = np.stack([k[b, S[b] - L: S[b]] for b in range(B)])
    spec_v = np.stack([v[b, S[b] - L: S[b]] for b in range(B)])
    kc = s.kv_append(kc, spec_k, nk)
    vc = s.kv_append(vc, spec_v, nk)
    go, gl = oracle.attention(oracle.VERIFY, q, kc, vc, (nk + L).astype(np.int32))
    assert np.allclose(go, ro, rtol=0, atol=1e-12), np.max(np.abs(go - ro))
    assert np.allclose(gl, rl, rtol=0, atol=1e-12), np.max(np.abs(gl - rl))


ALL_SDSTEP_PINS = [pin_accept_eq1, pin_accept_cases, pin_argmax_brute, pin_argmax_bf16,
                   pin_append_paged_contiguous, pin_commit_lengths, pin_ring_window,
                   pin_gather_by_hand, pin_gather_paged_contiguous,
                   pin_gather_listed_draft_equivalence]
