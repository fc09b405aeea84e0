"""Oracle for the steps around each verification: greedy acceptance with a
bonus token, writing the verified tokens' K/V into the cache, committing the
accepted length, the rolling list of a StreamingLLM-style draft cache, and
gathering a static selection into a draft cache of its own.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use this module.  It shares no code
with the GPU library.

One speculative step (Sec. 3.1; greedy decoding in Sec. 5.1).  A sequence
holds C committed tokens.  The verifier runs q_len = gamma + 1 tokens,
[t0, d_1 .. d_gamma] (t0 = the last token produced, whose K/V is not cached
yet, then the gamma drafts), and their K/V are written at positions
C .. C + gamma, so the cache length during verification is S = C + q_len.
Under greedy decoding the target's token after input i is the argmax of its
logits at i; draft d_{i+1} is accepted while it equals that token.  With a
drafts accepted, the bonus is the target's token at input a, the K/V of
t0, d_1 .. d_a stay (C' = C + a + 1) and the rest is rolled back.  When each
draft is accepted independently with probability alpha, a + 1 has mean
(1 - alpha^(gamma+1)) / (1 - alpha): Eq. 1.
"""
import numpy as np


def widen(x):
    """float32 values or bf16 bit patterns (uint16) -> float64, exactly."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def expected_tokens(gamma, alpha):
    """Eq. 1: expected tokens per verification, Omega(gamma, alpha)."""
    if alpha == 1.0:
        return float(gamma + 1)
    return (1.0 - alpha ** (gamma + 1)) / (1.0 - alpha)


def target_tokens(logits):
    """logits [..., V] -> the first index of the largest logit; NaN compares
    as -inf, so a row of NaN and -inf gives index 0."""
    x = widen(logits)
    x = np.where(np.isnan(x), -np.inf, x)
    return np.argmax(x, axis=-1).astype(np.int64)


def greedy_accept(logits, draft):
    """logits [B, gamma + 1, V]; draft [B, gamma] token ids.

    Returns (accepted [B], tokens [B, gamma + 1], target [B, gamma + 1]):
    accepted[b] = the length of the leading run of i with
    draft[b, i] == target[b, i]; tokens[b] = the accepted drafts, then the
    bonus target[b, accepted[b]], then -1 padding."""
    target = target_tokens(logits)
    B, L = target.shape
    draft = np.asarray(draft, dtype=np.int64).reshape(B, L - 1)
    accepted = np.zeros(B, dtype=np.int64)
    tokens = np.full((B, L), -1, dtype=np.int64)
    for b in range(B):
        a = 0
        while a < L - 1 and draft[b, a] == target[b, a]:
            a += 1
        accepted[b] = a
        tokens[b, :a] = draft[b, :a]
        tokens[b, a] = target[b, a]
    return accepted, tokens, target


def cache_slot(b, j, page_size, page_table):
    """(block, token) of logical position j of sequence b: the sequence's own
    row when contiguous, else its page from the page table."""
    if not page_size:
        return b, j
    return int(page_table[b, j // page_size]), j % page_size


def kv_append(cache, new, pos0, page_size=0, page_table=None):
    """Write new [B, n, Hkv, d] at positions pos0[b] .. pos0[b] + n - 1 of a
    contiguous [B, S_alloc, Hkv, d] or paged [P, page_size, Hkv, d] cache.
    Values move unchanged (any dtype).  Returns the updated copy."""
    out = np.array(cache, copy=True)
    B, n = new.shape[:2]
    for b in range(B):
        for i in range(n):
            blk, tok = cache_slot(b, int(pos0[b]) + i, page_size, page_table)
            out[blk, tok] = new[b, i]
    return out


def kv_gather(dst, src, idx, idx_len, src_lens, *, src_page_size=0, src_page_table=None,
              dst_page_size=0, dst_page_table=None):
    """A static selection gathered into a draft cache of its own: a static KV
    selection collects its sparse cache once, before generation, so drafting
    then reads it like any cache (Sec. 4.2).  src and dst hold one of K or V,
    as in kv_append.  For every sequence b, kv head h and
    j < n_b = min(idx_len[b], stride) (idx [B, Hkv, stride]), row j of head h
    of dst takes row p = idx[b, h, j] of head h of src if 0 <= p < src_lens[b],
    and zeros otherwise.  Values move unchanged.

    Returns (updated copy of dst, n [B])."""
    out = np.array(dst, copy=True)
    idx = np.asarray(idx)
    B, Hkv, stride = idx.shape
    n = np.clip(np.asarray(idx_len, np.int64), 0, stride)
    for b in range(B):
        for h in range(Hkv):
            for j in range(int(n[b])):
                p = int(idx[b, h, j])
                dblk, dtok = cache_slot(b, j, dst_page_size, dst_page_table)
                if 0 <= p < int(src_lens[b]):
                    sblk, stok = cache_slot(b, p, src_page_size, src_page_table)
                    out[dblk, dtok, h] = src[sblk, stok, h]
                else:
                    out[dblk, dtok, h] = 0
    return out, n


def kv_commit(lens, accepted):
    """Committed lengths after a step: C' = C + accepted + 1."""
    return np.asarray(lens, np.int64) + np.asarray(accepted, np.int64) + 1


def ring_commit(idx, lens, accepted, ring_start, ring_len):
    """Record the kept positions C .. C + a of every sequence in its listed
    draft cache (idx [B, Hkv, stride]): position j goes to slot
    ring_start + j % ring_len of each kv head's list, which holds j - ring_len
    before, so the ring keeps the last ring_len committed positions (a
    rolling window).  Returns the updated copy."""
    idx = np.array(idx, copy=True)
    for b in range(idx.shape[0]):
        C = int(lens[b])
        for j in range(C, C + int(accepted[b]) + 1):
            idx[b, :, ring_start + j % ring_len] = j
    return idx


def streaming_list(prompt_lens, Hkv, n_sink, window):
    """StreamingLLM-style static draft cache built at prefill, as a list
    [B, Hkv, n_sink + window] for listed-cache draft attention: the sinks
    0 .. min(n_sink, C) - 1 in slots 0.., and the last `window` prompt
    positions j >= n_sink in ring slots n_sink + j % window; empty slots hold
    -1.  ring_commit(..., n_sink, window) then rolls the window forward."""
    B = len(prompt_lens)
    idx = np.full((B, Hkv, n_sink + window), -1, dtype=np.int32)
    for b, C in enumerate(prompt_lens):
        C = int(C)
        for j in range(min(n_sink, C)):
            idx[b, :, j] = j
        for j in range(max(n_sink, C - window), C):
            idx[b, :, n_sink + j % window] = j
    return idx
