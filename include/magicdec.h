/*
 * magicdec.h -- C ABI of libmagicdec.so: batched GQA decode attention for
 * speculative decoding with a sparse-KV self-speculative draft (MagicDec,
 * arXiv 2408.11049), on AMD Instinct MI355X (gfx950).
 *
 * The paper's hot path at large batch and long context is attention over the
 * KV cache: its loading cost grows with both batch size and sequence length
 * and dominates the decode step (Sec. 1 insight 1; Sec. 3.2), and verification
 * of gamma+1 speculated tokens shares that loading cost with plain decoding
 * (Sec. 3.2), while the draft reads only a fixed-budget compressed cache
 * (Sec. 4.1, Eq. 3; StreamingLLM-style drafting, Sec. 5.1).
 *
 * Conventions shared by every entry point
 *   - All pointers in md_attn_args are DEVICE pointers except where noted.
 *     The caller owns every buffer; the library allocates nothing per call
 *     and keeps no pointer after it returns.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*;
 *     NULL is the null stream).  Buffers must stay alive and unmodified until
 *     the stream reaches the call.  Nothing synchronises with the host.
 *   - Calls are thread-safe and re-entrant.  The only global state is a
 *     per-device cache of the compute-unit count, a per-process call counter
 *     and, for md_attn_noalloc only, one static scratch buffer per device.
 *     The MD_* tuning overrides (MD_PREFETCH_DEPTH, MD_OCCUPANCY, MD_LPT,
 *     MD_HEADS_PER_WG, MD_FUSED_MERGE, MD_SLOTS_SCALE, MD_BALANCED,
 *     MD_BAL_WG_PER_CU, MD_BAL_NW, MD_WAVES; for measurement) are read from the environment on
 *     every call, md_workspace_bytes included; do not change them while
 *     another thread is inside the library, nor between sizing a workspace
 *     and the call that uses it.
 *   - Errors are return codes (md_status).  Argument errors are detected on
 *     the host before any HIP call, so a failed call has launched nothing.
 *   - Device-side contract violations leave memory in bounds but results
 *     meaningless: kv_lens[b] < q_len yields rows with an empty key set
 *     (O = 0, lse = -inf); kv_lens[b] is clamped to max_kv_len; page ids
 *     outside [0, num_pages) are never dereferenced (the loads of those
 *     tokens are redirected to element 0 of k and v, and the outputs of the
 *     rows that see them are unspecified).  They are reported only to a
 *     caller that passes an error word
 *     (md_attn_args.err_word, for debugging): each attention call then ORs
 *     into it MD_ERRW_SHORT_LEN if some kv_lens[b] < q_len (negative
 *     included), MD_ERRW_LONG_LEN if some kv_lens[b] > max_kv_len, and
 *     MD_ERRW_BAD_PAGE if a position the call reads (below the clamped
 *     length; for a listed draft, a usable list entry or a speculated
 *     position) has a page id outside [0, num_pages).  The library never
 *     clears the word.  The checks read the lengths and the page ids once
 *     more, before the K/V stream; without the word they cost nothing.
 */
#ifndef MAGICDEC_H_
#define MAGICDEC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MD_OK = 0,
  MD_ERR_INVALID_ARG = 1, /* a malformed argument (see each entry point) */
  MD_ERR_UNSUPPORTED = 2, /* valid, but this shape or dtype is not built */
  MD_ERR_WORKSPACE = 3,   /* workspace missing, too small or misaligned */
  MD_ERR_HIP = 4          /* the HIP runtime reported an error on launch */
} md_status;

typedef enum { MD_F32 = 0, MD_BF16 = 1 } md_dtype;

typedef enum { MD_MODE_VERIFY = 0, MD_MODE_DRAFT = 1, MD_MODE_DRAFT_INDEXED = 2 } md_mode;

/* Bits of md_attn_args.err_word (device-side contract checks). */
typedef enum {
  MD_ERRW_SHORT_LEN = 1, /* some kv_lens[b] < q_len */
  MD_ERRW_LONG_LEN = 2,  /* some kv_lens[b] > max_kv_len */
  MD_ERRW_BAD_PAGE = 4   /* a position read has a page id outside [0, num_pages) */
} md_err_bits;

/*
 * One attention call over a batch of B sequences for one layer.
 *
 * Shapes (B = num_seqs, L = q_len = gamma + 1, Hq = num_q_heads,
 * Hkv = num_kv_heads, d = head_dim, G = Hq / Hkv):
 *   q   [B, L, Hq, d]          row-major, contiguous, 16-byte aligned
 *   o   [B, L, Hq, d]          row-major, contiguous, 16-byte aligned, dtype of q
 *   lse [B, L, Hq]             fp32, natural log of the softmax denominator
 *                              (including the max), or NULL
 *   k, v                       element (blk, tok, hk, c) lives at
 *                              blk*kv_stride_blk + tok*kv_stride_tok +
 *                              hk*kv_stride_head + c   (element strides; c unit
 *                              stride; strides multiples of 16 bytes)
 *     contiguous (page_size == 0): blk = sequence b, tok = token j;
 *                              each sequence holds >= max_kv_len tokens.
 *     paged (page_size > 0, a power of two): blk = page_table[b*max_pages_per_seq
 *                              + j/page_size], tok = j % page_size; the pool
 *                              holds num_pages pages.
 *   kv_lens [B] int32          S_b, the number of cached tokens of sequence b,
 *                              INCLUDING the L speculated tokens, whose K/V are
 *                              already written at positions S_b-L .. S_b-1.
 *
 * Query row i of sequence b sits at position p = S_b - L + i and sees
 *   verify: keys j with 0 <= j <= p                   (Sec. 3.1, T_V)
 *   draft : keys j <= p with j < n_sink or j >= p - window + 1
 *           (sink tokens plus the query's own last `window` positions:
 *            a StreamingLLM-style cache of budget n_sink + window, Sec. 5.1)
 * Query head h reads kv head h / G.  Scores are scaled by sm_scale
 * (sm_scale <= 0 selects 1/sqrt(d)); softmax and accumulation are fp32.
 */
typedef struct {
  int32_t num_seqs;     /* B >= 0 (0 is a no-op) */
  int32_t q_len;        /* L in [1, 16] */
  int32_t num_q_heads;  /* Hq >= 1, a multiple of num_kv_heads */
  int32_t num_kv_heads; /* Hkv >= 1; G * L <= 64 */
  int32_t head_dim;     /* d in {64, 128} */
  int32_t dtype;        /* md_dtype of q, k, v, o */
  float sm_scale;       /* <= 0: 1/sqrt(d) */
  const void* q;
  const void* k;
  const void* v;
  int64_t kv_stride_blk;
  int64_t kv_stride_tok;
  int64_t kv_stride_head;
  int32_t page_size;          /* 0 = contiguous, else tokens per page (power of two) */
  int32_t max_pages_per_seq;  /* columns of page_table (paged only) */
  int64_t num_pages;          /* pages in the pool (paged only) */
  const int32_t* page_table;  /* [B, max_pages_per_seq] or NULL when contiguous */
  const int32_t* kv_lens;     /* [B] */
  int32_t max_kv_len;         /* HOST bound on every kv_lens[b]; sizes the grid */
  void* o;
  float* lse;
  void* workspace;            /* device scratch, >= md_workspace_bytes(), 256-byte aligned;
                                 any contents (nothing in it needs clearing) */
  size_t workspace_bytes;
  int32_t* err_word;          /* device int32 or NULL: contract checks (md_err_bits, above) */
} md_attn_args;

/*
 * Verification attention: all L = gamma+1 speculated tokens of every sequence
 * against the full KV cache, causal among themselves (Sec. 3.1-3.2).
 * Errors: MD_ERR_INVALID_ARG for a NULL args/q/k/v/o/kv_lens, a NULL or
 * superfluous page_table, bad sizes, a non power-of-two page size, a table too
 * narrow for max_kv_len, max_kv_len < q_len, misaligned pointers or strides;
 * MD_ERR_UNSUPPORTED for head_dim not in {64,128}, G*L > 64, or sizes past
 * the kernels' 32-bit indexing: max_kv_len (or a draft window or list
 * capacity) > 2^31 - 65, kv_stride_tok > 2^28 elements,
 * num_seqs * num_kv_heads > 2^31 - 1, num_seqs * q_len * num_q_heads >
 * 4 (2^31 - 1); MD_ERR_WORKSPACE when md_workspace_bytes() is nonzero for
 * these arguments and the workspace is missing, smaller or not 256-byte
 * aligned (which calls need one -- split ranges, the balanced verify --
 * depends on the sizes and the device, so size it for every new shape);
 * MD_ERR_HIP.
 */
int md_verify_attn(const md_attn_args* a, void* stream);

/*
 * Draft attention with a StreamingLLM-style sparse cache read in place: the
 * same queries see only the first n_sink tokens and their last `window`
 * positions (budget K = n_sink + window; Sec. 4.1 Eq. 3, Sec. 5.1).
 * n_sink >= 0 and window >= 1, else MD_ERR_INVALID_ARG; other errors as
 * md_verify_attn.
 */
int md_draft_attn(const md_attn_args* a, int32_t n_sink, int32_t window, void* stream);

/*
 * Draft attention over a static compressed cache given as token positions,
 * read in place from the full cache: the SnapKV-style drafting the paper
 * finds best (static KV selection made at prefill, Sec. 4.4; Sec. 5.2, Table
 * 2), with optional per-sequence budgets (Sec. 4.3).  Query row i of
 * sequence b (position p) sees the listed positions of its kv head that lie
 * in [0, S_b - q_len), taken as a set, plus the speculated positions
 * S_b - q_len .. p.
 *   idx      device int32 [B, Hkv, idx_stride]: positions, any order, unique
 *            (a repeated position would be counted twice); entries outside
 *            [0, S_b - q_len) are skipped
 *   idx_len  device int32 [B]: entries of sequence b's lists that count
 *            (clamped to [0, idx_stride])
 *   idx_stride >= 1, host value: list capacity; sizes the grid
 * Errors: MD_ERR_INVALID_ARG for NULL idx/idx_len (with B > 0), idx_stride
 * < 1 or misaligned lists; others as md_verify_attn.
 */
int md_draft_attn_indexed(const md_attn_args* a, const int32_t* idx, const int32_t* idx_len,
                          int32_t idx_stride, void* stream);

/*
 * Log-sum-exp merge of attention computed over disjoint key sets (the
 * split-KV identity of Flash-Decoding, Sec. 2).  Per row r:
 *   lse[r] = ln sum_k exp(lse_parts[k][r]),
 *   o[r]   = sum_k exp(lse_parts[k][r] - lse[r]) * o_parts[k][r]
 * Parts whose lse is -inf are skipped (their o is never read); a row with
 * every part empty gets o = 0, lse = -inf.
 *   o_parts   [n_parts][n_rows][head_dim] fp32 (each part already normalised)
 *   lse_parts [n_parts][n_rows] fp32
 *   o         [n_rows][head_dim] in out_dtype (md_dtype)
 *   lse       [n_rows] fp32 or NULL
 * All device pointers, 16-byte aligned.  Errors: MD_ERR_INVALID_ARG for
 * n_parts < 1, n_rows < 0, NULL or misaligned pointers, a bad dtype;
 * MD_ERR_UNSUPPORTED for head_dim not in {64,128} or n_rows > 4 (2^31 - 1);
 * MD_ERR_HIP.
 */
int md_merge_lse(int32_t n_parts, int64_t n_rows, int32_t head_dim, int32_t out_dtype,
                 const float* o_parts, const float* lse_parts, void* o, float* lse,
                 void* stream);

/*
 * Workspace bytes an attention call with these arguments needs (0 when the
 * call runs as a single pass).  A split-range call keeps there, per head
 * group, an arrival counter tagged with the call, then every chunk's partial
 * O and lse (the split-KV identity, Sec. 2).  A balanced verify (batches of
 * 2..256 long sequences whose head groups number at most two per compute
 * unit: every workgroup streams an equal share of all groups' key tiles, so
 * ragged lengths do not leave units idle) keeps the same counters, then two
 * partial slots per workgroup for the groups its share cuts.  Whatever the
 * buffer held before is never mistaken for this call's state, so it needs no
 * clearing.  mode is MD_MODE_VERIFY or MD_MODE_DRAFT; n_sink and window are
 * used for MD_MODE_DRAFT only.  Pure host arithmetic on the sizes plus the
 * current device's compute-unit count (256 if no device is visible);
 * pointers in `a` are not read.  Returns 0 for malformed arguments too:
 * the attention call itself reports those.
 */
size_t md_workspace_bytes(const md_attn_args* a, int32_t mode, int32_t n_sink, int32_t window);

/* Workspace bytes of md_draft_attn_indexed with lists of capacity idx_stride
 * (same conventions as md_workspace_bytes). */
size_t md_workspace_bytes_indexed(const md_attn_args* a, int32_t idx_stride);

/*
 * md_verify_attn (mode MD_MODE_VERIFY) or md_draft_attn (mode MD_MODE_DRAFT,
 * with n_sink and window as there) without a caller workspace, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  The caller still passes
 * every input and output; a->workspace and a->workspace_bytes are ignored.
 *   - A split-range plan keeps its state (tagged arrival counters, partial O
 *     and lse) in a static device buffer of MD_NOALLOC_SCRATCH_BYTES that the
 *     library holds on each GPU it runs on until the process ends.  That
 *     covers every plan on a device of up to 256 compute units (MI355X); a
 *     plan needing more (md_workspace_bytes > MD_NOALLOC_SCRATCH_BYTES)
 *     returns MD_ERR_WORKSPACE before any launch.
 *   - The call allocates nothing (no hipMalloc, hipFree or allocating
 *     library routine).  Its first call on a device looks up that device's
 *     buffer address once (hipGetSymbolAddress).
 *   - All calls on one GPU share its buffer, which keeps the last call's
 *     contents; nothing in it needs clearing (the counters carry a per-call
 *     tag).  Calls that can overlap in time on one GPU (other streams, other
 *     threads) race on it and give wrong results: serialise them.
 *   - `stream` (NULL: the null stream) must belong to the current device.
 * Errors: as md_verify_attn / md_draft_attn; MD_ERR_INVALID_ARG for another
 * mode or a stream of another device; MD_ERR_WORKSPACE for a plan larger than
 * the buffer; MD_ERR_HIP if the address lookup fails.
 */
#define MD_NOALLOC_SCRATCH_BYTES ((size_t)33 << 20)
int md_attn_noalloc(const md_attn_args* a, int32_t mode, int32_t n_sink, int32_t window,
                    void* stream);

/*
 * SnapKV-style selection of the static draft cache at prefill: the static
 * KV selection the paper finds best (Sec. 4.4; budget 2049 in Sec. 5.2),
 * with its observation window (32 queries) and average pooling (kernel 5).
 * The steps restate the published SnapKV method:
 *   vote(j)   = sum over the n_obs observation queries o (positions
 *               S_b - n_obs + o) and the G query heads of kv head hk of the
 *               softmax weight of key j, each query's softmax running over
 *               the keys at or before its own position;
 *   pooled(j) = mean of vote over j - pool/2 .. j + pool/2, zero outside the
 *               prefix [0, S_b - n_obs);
 *   kept      = the budget - n_obs prefix positions of largest pooled vote
 *               (ties: the smaller position), all of them if fewer, then the
 *               n_obs observation positions; ascending.
 * md_snapkv_votes writes vote(j) (before pooling) for j in [0, S_b - n_obs);
 * md_snapkv_select pools and selects, writing lists md_draft_attn_indexed
 * reads directly.
 */
typedef struct {
  int32_t num_seqs;       /* B >= 0 */
  int32_t n_obs;          /* observation queries, >= 1, G * n_obs <= 256 */
  int32_t num_q_heads, num_kv_heads, head_dim, dtype;  /* as md_attn_args */
  float sm_scale;         /* <= 0: 1/sqrt(d) */
  const void* q_obs;      /* [B, n_obs, Hq, d], contiguous, 16-byte aligned */
  const void* k;          /* as md_attn_args (contiguous or paged) */
  int64_t kv_stride_blk, kv_stride_tok, kv_stride_head;
  int32_t page_size, max_pages_per_seq;
  int64_t num_pages;
  const int32_t* page_table;
  const int32_t* prompt_lens;  /* [B], S_b (the prompt includes the window) */
  int32_t max_prompt_len;      /* host bound on every S_b */
  float* votes;                /* [B, Hkv, votes_stride] fp32 */
  int32_t votes_stride;        /* >= max_prompt_len - n_obs */
  void* workspace;             /* >= md_snapkv_workspace_bytes(), 256-byte aligned */
  size_t workspace_bytes;
} md_snapkv_args;

/* Votes of every (sequence, kv head) prefix position.  Errors:
 * MD_ERR_INVALID_ARG for NULL or misaligned pointers, bad sizes, a votes
 * stride below max_prompt_len - n_obs, max_prompt_len < n_obs;
 * MD_ERR_UNSUPPORTED for head_dim not in {64,128}, G * n_obs > 256 or
 * num_seqs * num_kv_heads > 2^31 - 1; MD_ERR_WORKSPACE; MD_ERR_HIP. */
int md_snapkv_votes(const md_snapkv_args* a, void* stream);
size_t md_snapkv_workspace_bytes(const md_snapkv_args* a);

/*
 * Pool the votes and select, per (sequence, kv head) row r = b * Hkv + hk:
 *   votes   [B * Hkv][votes_stride] fp32 (only [0, S_b - n_obs) is read)
 *   idx     [B * Hkv][budget] int32 out: ascending kept positions
 *   idx_len [B] int32 out: kept count per sequence (min(budget, S_b) when
 *           S_b >= n_obs)
 * pool odd >= 1; budget >= n_obs; S_b is clamped to votes_stride + n_obs.
 * Errors: MD_ERR_INVALID_ARG for bad sizes or NULL/misaligned pointers;
 * MD_ERR_HIP.
 */
int md_snapkv_select(int32_t num_seqs, int32_t num_kv_heads, const float* votes,
                     int32_t votes_stride, const int32_t* prompt_lens, int32_t n_obs,
                     int32_t pool, int32_t budget, int32_t* idx, int32_t* idx_len, void* stream);

/*
 * ---- The speculative step around verification (Sec. 3.1; greedy decoding,
 * Sec. 5.1) ----
 *
 * A sequence holds C committed tokens.  One step runs the verifier on
 * q_len = gamma + 1 tokens [t0, d_1 .. d_gamma] (t0 = the last token produced,
 * then the drafts), whose K/V go to positions C .. C + gamma (md_kv_append),
 * so verification sees S = C + q_len.  Greedy acceptance (md_greedy_accept)
 * keeps the drafts that match the target's argmax up to the first mismatch
 * plus one bonus token; with a drafts accepted the K/V of t0, d_1 .. d_a stay
 * and the cache is committed to C' = C + a + 1 (md_kv_commit), which rolls
 * the rejected positions back.  The expected a + 1 per step is Eq. 1.
 */

/* One layer's KV cache as a write target, addressed as in md_attn_args. */
typedef struct {
  int32_t num_seqs;           /* B >= 0 */
  int32_t num_kv_heads;       /* Hkv >= 1 */
  int32_t head_dim;           /* d >= 1; d * element size a multiple of 16 bytes */
  int32_t dtype;              /* md_dtype of k, v and the appended rows */
  void* k;
  void* v;
  int64_t kv_stride_blk, kv_stride_tok, kv_stride_head;  /* element strides, 16-byte multiples */
  int32_t page_size;          /* 0 = contiguous, else tokens per page (power of two) */
  int32_t max_pages_per_seq;  /* columns of page_table (paged only) */
  int64_t num_pages;          /* pages in the pool (paged only) */
  const int32_t* page_table;  /* device [B, max_pages_per_seq], or NULL when contiguous */
  int32_t capacity;           /* contiguous: tokens each sequence's block holds (>= 1);
                                 paged: ignored (max_pages_per_seq * page_size) */
} md_kv_cache;

/*
 * Write n_new tokens' K and V rows of every sequence into the cache:
 *   k_new, v_new  device [B, n_new, Hkv, d], contiguous, dtype of the cache,
 *                 16-byte aligned
 *   pos0          device int32 [B]: row i of sequence b goes to position
 *                 pos0[b] + i (pages through page_table when paged)
 *   lens_out      device int32 [B] or NULL: set to pos0[b] + n_new; must not
 *                 overlap pos0
 * Positions past the capacity (or the table), and pages outside
 * [0, num_pages), are not written: memory stays in bounds, those rows are
 * lost.  Values move bit for bit.  The caller provides the pages.
 * Errors: MD_ERR_INVALID_ARG for NULL or misaligned pointers, bad sizes,
 * n_new < 0, lens_out overlapping pos0; MD_ERR_HIP.
 */
int md_kv_append(const md_kv_cache* c, int32_t n_new, const void* k_new, const void* v_new,
                 const int32_t* pos0, int32_t* lens_out, void* stream);

/*
 * Greedy acceptance with a bonus token, per sequence b:
 *   target[b][i] = the first index of the largest of logits[b][i][0 .. vocab),
 *                  a NaN logit comparing as -inf (a row of NaN and -inf gives 0);
 *   accepted[b]  = the length of the leading run of i < n_draft with
 *                  draft[b][i] == target[b][i];
 *   tokens[b][i] = draft[b][i] for i < accepted[b], target[b][accepted[b]] (the
 *                  bonus) at i = accepted[b], -1 after.
 *   logits    device [B, n_draft + 1, vocab] in dtype (MD_F32 or MD_BF16), contiguous
 *   draft     device int32 [B, n_draft]
 *   accepted  device int32 [B] out
 *   tokens    device int32 [B, n_draft + 1] out
 *   target    device int32 [B, n_draft + 1] out, or NULL
 *   workspace >= md_greedy_accept_workspace_bytes(), 256-byte aligned
 * The argmax is exact (a comparison), so results are bit-exact in any
 * reduction order.  Errors: MD_ERR_INVALID_ARG for NULL or misaligned
 * pointers, n_draft outside [0, 1023], vocab outside [1, 2^30], a bad dtype;
 * MD_ERR_WORKSPACE; MD_ERR_HIP.
 */
int md_greedy_accept(int32_t num_seqs, int32_t n_draft, int32_t vocab, int32_t dtype,
                     const void* logits, const int32_t* draft, int32_t* accepted,
                     int32_t* tokens, int32_t* target, void* workspace, size_t workspace_bytes,
                     void* stream);

/* Workspace bytes of md_greedy_accept for these sizes on the current device
 * (0 for malformed sizes). */
size_t md_greedy_accept_workspace_bytes(int32_t num_seqs, int32_t n_draft, int32_t vocab);

/*
 * Commit (and roll back) one step:
 *   lens      device int32 [B], in: C (committed before the step); out:
 *             C + a + 1 with a = accepted[b] clamped to [0, q_len - 1]
 *   accepted  device int32 [B]
 * With idx != NULL the kept positions C .. C + a are also recorded in every
 * kv head's listed draft cache (idx [B, Hkv, idx_stride], as read by
 * md_draft_attn_indexed): position j goes to slot ring_start + j % ring_len,
 * which held j - ring_len, so slots [ring_start, ring_start + ring_len) hold
 * the last ring_len committed positions: a rolling window.  Empty ring slots
 * hold -1 (skipped by the attention), and the lists' idx_len must cover the
 * ring.  Positions recorded this way must not also sit in the static part
 * of the list.
 * Errors: MD_ERR_INVALID_ARG for NULL or misaligned pointers, q_len < 1, and,
 * with idx, num_kv_heads < 1, ring_start < 0, ring_len < 1 or
 * ring_start + ring_len > idx_stride; MD_ERR_HIP.
 */
int md_kv_commit(int32_t num_seqs, int32_t q_len, int32_t* lens, const int32_t* accepted,
                 int32_t num_kv_heads, int32_t* idx, int32_t idx_stride, int32_t ring_start,
                 int32_t ring_len, void* stream);

/*
 * The StreamingLLM-style draft cache built at prefill, as lists for
 * md_draft_attn_indexed that md_kv_commit(..., ring_start = n_sink,
 * ring_len = window) then rolls forward (the static sink-plus-window cache
 * the paper drafts with, Sec. 5.1, kept current as tokens are committed):
 *   idx      device int32 [B, Hkv, n_sink + window] out: slots 0 .. n_sink-1
 *            hold the sinks 0 .. min(n_sink, C) - 1, slot n_sink + j % window
 *            holds prompt position j for the last `window` positions
 *            j >= n_sink; other slots -1.  (A prompt shorter than n_sink has
 *            fewer sinks.)
 *   idx_len  device int32 [B] out: n_sink + window
 *   prompt_lens device int32 [B]: C
 * Errors: MD_ERR_INVALID_ARG for NULL or misaligned pointers, num_kv_heads
 * < 1, n_sink < 0, window < 1; MD_ERR_HIP.
 */
int md_streaming_list(int32_t num_seqs, int32_t num_kv_heads, const int32_t* prompt_lens,
                      int32_t n_sink, int32_t window, int32_t* idx, int32_t* idx_len,
                      void* stream);

/*
 * Gather a static selection into a draft cache of its own, once, before
 * generation (Sec. 4.2: a static KV selection collects its sparse cache up
 * front, so drafting pays no search).  A draft step then streams the
 * gathered rows contiguously instead of reading each listed row of the full
 * cache (md_draft_attn_indexed).  For every sequence b, kv head h and
 * j < n_b = min(max(idx_len[b], 0), idx_stride): row j of head h of dst gets
 * the K and V rows of head h at position p = idx[b][h][j] of src when
 * 0 <= p < src_lens[b], and zeros otherwise.
 *   dst, src   caches with equal num_seqs, num_kv_heads, head_dim and dtype
 *              (contiguous or paged, independently); their memory must not
 *              overlap
 *   idx        device int32 [B, Hkv, idx_stride] (md_snapkv_select's lists)
 *   idx_len    device int32 [B]
 *   src_lens   device int32 [B]: how many positions of src are valid
 *   dst_lens   device int32 [B] out, or NULL: set to n_b; must not overlap
 *              idx_len or src_lens
 * Values move bit for bit.  Rows on pages outside [0, num_pages) are not
 * written.
 * Drafting over dst: md_kv_append the step's rows at position dst_lens[b] of
 * dst (as of the full cache), then md_verify_attn over dst with kv_lens =
 * dst_lens + q_len; md_kv_commit then advances dst_lens like the full
 * cache's lengths.  The gathered rows come first and every query sees them,
 * the speculated rows last and causally: md_draft_attn_indexed over
 * (src, idx) for lists of usable entries.  An unusable entry gathers a zero
 * row, which takes part in that attention (score 0, value 0) where
 * md_draft_attn_indexed skips the entry.
 * Errors: MD_ERR_INVALID_ARG for NULL or misaligned pointers, a malformed or
 * mismatched cache, idx_stride < 1, a destination that holds fewer than
 * idx_stride rows per sequence (capacity, or max_pages_per_seq * page_size),
 * dst_lens overlapping idx_len or src_lens; MD_ERR_HIP.
 */
int md_kv_gather(const md_kv_cache* dst, const md_kv_cache* src, const int32_t* idx,
                 int32_t idx_stride, const int32_t* idx_len, const int32_t* src_lens,
                 int32_t* dst_lens, void* stream);

/*
 * ---- Speculative-decoding cost model (Sec. 3.1 Eq. 1-2; Sec. 4.1 Eq. 3-4) ----
 *
 * Host-only arithmetic (no device, no stream), for choosing the speculation
 * length from measured times.  Per decoding step of a batch at one sequence
 * length: t_target = T_T (one token per sequence), t_draft = T_D(B, K) per
 * drafted token with KV budget K, t_select = T_select(B, S, K) per drafted
 * token (0 for static selections), t_verify = T_V(gamma), alpha the draft
 * acceptance rate.  Any consistent time unit.
 *
 * md_sd_expected_tokens: Omega(gamma, alpha) = sum_{k=0..gamma} alpha^k, i.e.
 *   (1 - alpha^(gamma+1)) / (1 - alpha) (Eq. 1), summed so it stays exact to
 *   rounding as alpha -> 1.  NaN for gamma < 0 or alpha outside [0, 1].
 * md_sd_latency_ratio: T_Avg^SD / T_T = (gamma (t_draft + t_select) + t_verify)
 *   / (Omega t_target) (Eq. 2 with Eq. 3's draft time); below 1 means
 *   speculation is faster.  NaN for invalid arguments (negative times,
 *   t_target <= 0).
 * md_sd_best_gamma: Eq. 4 over gamma = 1 .. max_gamma for a fixed budget and
 *   selection: t_verify[g - 1] = T_V(g) (host array); writes the minimising
 *   gamma (ties: the smaller) and its ratio.  MD_ERR_INVALID_ARG for
 *   max_gamma < 1, NULL pointers or invalid times.
 * md_sd_alpha_from_omega: the alpha in [0, 1] with Omega(gamma, alpha) = omega
 *   (to ~1e-15), e.g. the acceptance rate implied by a measured Omega; NaN
 *   outside 1 <= omega <= gamma + 1.
 */
double md_sd_expected_tokens(int32_t gamma, double alpha);
double md_sd_latency_ratio(int32_t gamma, double alpha, double t_target, double t_draft,
                           double t_select, double t_verify);
int md_sd_best_gamma(int32_t max_gamma, double alpha, double t_target, double t_draft,
                     double t_select, const double* t_verify, int32_t* gamma_out,
                     double* ratio_out);
double md_sd_alpha_from_omega(int32_t gamma, double omega);

/* Static description of a status code; never NULL. */
const char* md_status_str(int status);

/* Text of the last MD_ERR_HIP on the calling thread ("" if none). */
const char* md_last_hip_error(void);

/* sizeof(md_attn_args) as compiled into the library, so bindings can check
 * their copy of the struct layout. */
size_t md_attn_args_size(void);

#ifdef __cplusplus
}
#endif

#endif /* MAGICDEC_H_ */
