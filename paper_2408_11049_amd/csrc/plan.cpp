// plan.cpp -- argument validation and the split-KV work decomposition.
// Pure host arithmetic: no HIP call is made here, so every error path can be
// exercised on a machine without a GPU.
#include <limits.h>
#include <stdlib.h>

#include <algorithm>

#include "internal.h"

namespace md {

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Largest visible range of any unit, in tokens.  Verify: the whole cache.
// Draft: sinks plus the union of the L queries' windows, which is
// [S - L - W + 1, S) -- or the whole prefix when that reaches the sinks.
int64_t visible_bound(int64_t max_kv_len, int L, int mode, int64_t n_sink, int64_t window) {
  if (mode == MD_MODE_VERIFY) return max_kv_len;
  if (mode == MD_MODE_DRAFT_INDEXED) return window + L;  // list capacity + speculated tokens
  int64_t lo = max_kv_len - L - window + 1;
  if (lo <= n_sink) return max_kv_len;
  return n_sink + (max_kv_len - lo);
}

}  // namespace

// Sizes that are malformed in themselves.
static int check_attn_shape(const md_attn_args* a) {
  if (a->num_seqs < 0) return MD_ERR_INVALID_ARG;
  if (a->q_len < 1 || a->q_len > 16) return MD_ERR_INVALID_ARG;
  if (a->num_q_heads < 1 || a->num_kv_heads < 1) return MD_ERR_INVALID_ARG;
  if (a->num_q_heads % a->num_kv_heads != 0) return MD_ERR_INVALID_ARG;
  if (a->head_dim < 1) return MD_ERR_INVALID_ARG;
  if (a->max_kv_len < a->q_len) return MD_ERR_INVALID_ARG;
  return MD_OK;
}

int env_knob(const char* name, int lo, int hi) {
  const char* e = getenv(name);
  const int v = e ? atoi(e) : 0;
  return (v >= lo && v <= hi) ? v : 0;
}

int check_attn_sizes(const md_attn_args* a) {
  const int shape = check_attn_shape(a);
  if (shape != MD_OK) return shape;
  if (a->head_dim != 64 && a->head_dim != 128) return MD_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(a->num_q_heads / a->num_kv_heads) * a->q_len > kMaxRows)
    return MD_ERR_UNSUPPORTED;
  if (a->kv_stride_tok > kMaxTokStride) return MD_ERR_UNSUPPORTED;
  if (a->max_kv_len > kMaxPosition) return MD_ERR_UNSUPPORTED;
  // Units (workgroups) and query rows (merge workgroups of four rows) in 32 bits.
  if (static_cast<int64_t>(a->num_seqs) * a->num_kv_heads > INT32_MAX) return MD_ERR_UNSUPPORTED;
  const int64_t rows_per_seq = static_cast<int64_t>(a->q_len) * a->num_q_heads;
  if (a->num_seqs > 4 * static_cast<int64_t>(INT32_MAX) / rows_per_seq) return MD_ERR_UNSUPPORTED;
  return MD_OK;
}

int validate_attn(const md_attn_args* a, int mode, int n_sink, int window) {
  if (!a) return MD_ERR_INVALID_ARG;
  if (mode != MD_MODE_VERIFY && mode != MD_MODE_DRAFT && mode != MD_MODE_DRAFT_INDEXED)
    return MD_ERR_INVALID_ARG;
  if (mode == MD_MODE_DRAFT && (n_sink < 0 || window < 1)) return MD_ERR_INVALID_ARG;
  if (mode == MD_MODE_DRAFT_INDEXED && window < 1) return MD_ERR_INVALID_ARG;
  const int shape = check_attn_shape(a);
  if (shape != MD_OK) return shape;
  if (a->dtype != MD_F32 && a->dtype != MD_BF16) return MD_ERR_INVALID_ARG;
  const bool paged = a->page_size != 0;
  if (a->page_size < 0) return MD_ERR_INVALID_ARG;
  if (paged) {
    if (!is_pow2(a->page_size) || a->max_pages_per_seq < 1 || a->num_pages < 1)
      return MD_ERR_INVALID_ARG;
    if (ceil_div(a->max_kv_len, a->page_size) > a->max_pages_per_seq) return MD_ERR_INVALID_ARG;
    if (a->num_pages > INT32_MAX) return MD_ERR_INVALID_ARG;  // page ids are int32
  }
  if (a->kv_stride_blk < 0 || a->kv_stride_tok < 0 || a->kv_stride_head < 0)
    return MD_ERR_INVALID_ARG;
  // Every malformed argument above is reported before a limit below.
  if (mode != MD_MODE_VERIFY && window > kMaxPosition) return MD_ERR_UNSUPPORTED;
  const int sizes = check_attn_sizes(a);
  if (sizes != MD_OK) return sizes;
  if (a->num_seqs == 0) return MD_OK;  // nothing will be read or written
  const int num_cus = device_cu_count();
  Plan p = make_plan(a, mode, n_sink, window, num_cus);
  if (p.n_chunks > kMaxChunks) return MD_ERR_UNSUPPORTED;  // unreachable below ~16k compute units

  if (!a->q || !a->k || !a->v || !a->o || !a->kv_lens) return MD_ERR_INVALID_ARG;
  if (paged != (a->page_table != nullptr)) return MD_ERR_INVALID_ARG;
  if (!aligned16(a->q) || !aligned16(a->k) || !aligned16(a->v) || !aligned16(a->o))
    return MD_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(a->kv_lens) & 3u) ||
      (a->lse && (reinterpret_cast<uintptr_t>(a->lse) & 3u)) ||
      (paged && (reinterpret_cast<uintptr_t>(a->page_table) & 3u)) ||
      (reinterpret_cast<uintptr_t>(a->err_word) & 3u))
    return MD_ERR_INVALID_ARG;
  // Every token row must start on a 16-byte boundary for the 128-bit loads.
  const int64_t per16 = a->dtype == MD_BF16 ? 8 : 4;
  if (a->kv_stride_blk % per16 || a->kv_stride_tok % per16 || a->kv_stride_head % per16)
    return MD_ERR_INVALID_ARG;
  // A token row must not overlap the next head's row.
  if (a->num_kv_heads > 1 && a->kv_stride_head < a->head_dim) return MD_ERR_INVALID_ARG;

  if (p.workspace_bytes) {
    if (!a->workspace || a->workspace_bytes < p.workspace_bytes) return MD_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(a->workspace) & 255u) return MD_ERR_WORKSPACE;
  }
  return MD_OK;
}

// The range split for n_groups workgroups' worth of units: one chunk each
// when they alone cover every compute unit, else each range is cut just until
// they do, never below kMinChunkTokens tokens per chunk.
static void split_units(int64_t U, int64_t n_groups, int64_t slots, int64_t* n_chunks_out,
                        int64_t* chunk_len_out) {
  int64_t n_chunks = 1;
  if (n_groups > 0 && n_groups < slots) {
    n_chunks = ceil_div(slots, n_groups);
    const int64_t cap = ceil_div(U, kMinChunkTokens);
    if (n_chunks > cap) n_chunks = cap;
    if (n_chunks < 1) n_chunks = 1;
  }
  int64_t chunk_len = ceil_div(ceil_div(U, n_chunks), kTile) * kTile;
  if (chunk_len < kTile) chunk_len = kTile;
  n_chunks = ceil_div(U, chunk_len);
  if (n_chunks < 1) n_chunks = 1;
  *n_chunks_out = n_chunks;
  *chunk_len_out = chunk_len;
}

// Kv heads per workgroup.  In the token-major cache the kv heads of a token
// are adjacent, so a workgroup that serves two heads of a sequence (two waves
// each) reads 2 x 256 B runs of every token row (bf16, d = 128) side by side
// instead of one: on MI355X a load-only model of the verify stream read the
// B = 64, S = 32768 cache at 7.03 TB/s this way against 6.62 TB/s with one
// head per workgroup.  Pairs halve the workgroups, though, so a range that
// must be split to fill the device is cut into twice as many chunks, each
// paying a pipeline fill and its share of the merge.  Measured over verify
// and draft calls of B = 1 .. 64 and S = 2048 .. 131072 (Llama-3.1-8B heads):
// pairs gain 5-13% where they alone fill the device and 2-3% where their
// chunks stay at 4096 tokens or more, and lose up to a third on short split
// ranges (one-token verify at B = 1, S = 4096: 35 us against 26).  So pairs
// are taken in those two cases only.  A listed draft reads a different list
// per head -- no adjacent rows -- and keeps one head per workgroup.
// MD_HEADS_PER_WG (1 or 2) overrides, for measurement.
static int heads_per_workgroup(const md_attn_args* a, int mode, int64_t U, int64_t slots) {
  const int forced = env_knob("MD_HEADS_PER_WG", 1, 2);
  if (a->num_kv_heads % 2) return 1;
  if (forced) return forced;
  if (mode == MD_MODE_DRAFT_INDEXED) return 1;
  const int64_t pairs = static_cast<int64_t>(a->num_seqs) * a->num_kv_heads / 2;
  if (pairs >= slots) return 2;
  int64_t n_chunks, chunk_len;
  split_units(U, pairs, slots, &n_chunks, &chunk_len);
  return chunk_len >= kPairMinChunkTokens ? 2 : 1;
}

Plan make_plan(const md_attn_args* a, int mode, int n_sink, int window, int num_cus) {
  Plan p;
  const int L = a->q_len;
  p.G = a->num_q_heads / a->num_kv_heads;
  p.R = p.G * L;
  p.NT = (p.R + 15) / 16;
  const int64_t U = visible_bound(a->max_kv_len, L, mode, n_sink, window);
  p.U_max = static_cast<int32_t>(U);
  p.n_rows = static_cast<int64_t>(a->num_seqs) * L * a->num_q_heads;
  p.n_units = static_cast<int64_t>(a->num_seqs) * a->num_kv_heads;

  // One workgroup of kWaves waves (one per SIMD) per compute unit is enough
  // to stream at full rate.  When the workgroups alone cover every compute
  // unit, one chunk per unit avoids the merge pass; else each unit's range is
  // split just until they do, never below kMinChunkTokens tokens per chunk.  (Every
  // chunk pays a pipeline fill, a cross-wave merge and a partial write:
  // measured on MI355X, splitting further -- two or four workgroups per
  // compute unit -- was 5-15% slower on long caches and slower still on
  // short draft ranges.)
  // MD_SLOTS_SCALE = 2..4 plans for that many workgroups per compute unit
  // (measurement only).
  const int64_t slots = (num_cus > 0 ? num_cus : 256) * std::max(1, env_knob("MD_SLOTS_SCALE", 2, 4));
  p.hp = heads_per_workgroup(a, mode, U, slots);
  p.n_groups = p.n_units / p.hp;
  int64_t n_chunks, chunk_len;
  split_units(U, p.n_groups, slots, &n_chunks, &chunk_len);
  p.n_chunks = static_cast<int32_t>(n_chunks);
  p.chunk_len = static_cast<int32_t>(chunk_len);
  // Balanced verify: where the units alone fill the device and lengths may
  // differ (the cases longest-first dispatch serves), every workgroup takes
  // an equal share of all head groups' tiles, in pairs of adjacent kv heads
  // when the head count is even.  Only with at most two head groups per
  // compute unit: there the longest sequence sets the makespan of one group
  // per workgroup, while with more groups per unit the hardware dispatcher
  // already evens the load out and the extra pieces only add prologues.
  // MD_BALANCED = 1 / 2 turns it off / on wherever allowed (measurement).
  const int bal_knob = env_knob("MD_BALANCED", 1, 2);
  const int bal_hp =
      (a->num_kv_heads % 2 == 0 && env_knob("MD_HEADS_PER_WG", 1, 2) != 1) ? 2 : 1;
  const int64_t cus = num_cus > 0 ? num_cus : 256;
  if (mode == MD_MODE_VERIFY && p.n_chunks == 1 && a->num_seqs >= 2 &&
      a->num_seqs <= kLptMaxSeqs && bal_knob != 1 && p.NT <= kBalMaxNT(a->dtype == MD_BF16) &&
      (bal_knob == 2 ||
       (a->max_kv_len >= kLptMinLen && p.n_units / bal_hp <= 2 * cus))) {
    const int hp = bal_hp;
    const int64_t groups = p.n_units / hp;
    // One workgroup per compute unit: every range then streams at once.
    // MD_BAL_WG_PER_CU = 2 doubles them, MD_BAL_NW sets their number
    // (measurement).
    const int64_t wpc = std::max(1, env_knob("MD_BAL_WG_PER_CU", 1, 2));
    const int64_t nw_forced = env_knob("MD_BAL_NW", 1, 4096);
    const int64_t nw = nw_forced ? nw_forced : cus * wpc;
    const int64_t tiles = ceil_div(a->max_kv_len, kTile) * (a->num_kv_heads / hp);
    const size_t slots = static_cast<size_t>(2 * nw);  // a first and a last piece per workgroup
    const size_t ctr = align_up(static_cast<size_t>(groups) * 8, 256);
    const size_t po = align_up(slots * hp * p.R * a->head_dim * 4, 256);
    const size_t pl = align_up(slots * hp * p.R * 4, 256);
    if (tiles * a->num_seqs < (int64_t{1} << 30) && ctr + po + pl <= kBalMaxWorkspace) {
      p.bal = true;
      p.hp = hp;
      p.n_groups = groups;
      p.bal_nw = static_cast<int32_t>(nw);
      p.counter_bytes = ctr;
      p.part_o_bytes = po;
      p.part_lse_bytes = pl;
      p.workspace_bytes = ctr + po + pl;
      return p;
    }
  }
  if (p.n_chunks > 1) {
    p.counter_bytes = align_up(static_cast<size_t>(p.n_groups) * 8, 256);
    p.part_o_bytes = align_up(static_cast<size_t>(n_chunks) * p.n_rows * a->head_dim * 4, 256);
    p.part_lse_bytes = align_up(static_cast<size_t>(n_chunks) * p.n_rows * 4, 256);
    p.workspace_bytes = p.counter_bytes + p.part_o_bytes + p.part_lse_bytes;
  }
  return p;
}

namespace {

// Chunks of a range of U keys over n_units units: at least 2 * wg_per_cu
// workgroups per compute unit (two rounds of wg_per_cu resident ones), never
// below kMinChunkTokens per chunk.
void split_range(int64_t U, int64_t n_units, int num_cus, int wg_per_cu, int32_t* n_chunks_out,
                 int32_t* chunk_len_out) {
  const int64_t slots = static_cast<int64_t>(num_cus > 0 ? num_cus : 256) * wg_per_cu;
  int64_t n_chunks = 1;
  if (n_units > 0 && n_units < 2 * slots) {
    n_chunks = ceil_div(2 * slots, n_units);
    const int64_t cap = ceil_div(U, kMinChunkTokens);
    if (n_chunks > cap) n_chunks = cap;
    if (n_chunks < 1) n_chunks = 1;
  }
  int64_t chunk_len = ceil_div(ceil_div(U > 0 ? U : 1, n_chunks), kTile) * kTile;
  n_chunks = ceil_div(U > 0 ? U : 1, chunk_len);
  *n_chunks_out = static_cast<int32_t>(n_chunks);
  *chunk_len_out = static_cast<int32_t>(chunk_len);
}

}  // namespace

int validate_snapkv(const md_snapkv_args* a) {
  if (!a) return MD_ERR_INVALID_ARG;
  if (a->num_seqs < 0 || a->n_obs < 1 || a->num_q_heads < 1 || a->num_kv_heads < 1)
    return MD_ERR_INVALID_ARG;
  if (a->num_q_heads % a->num_kv_heads) return MD_ERR_INVALID_ARG;
  if (a->dtype != MD_F32 && a->dtype != MD_BF16) return MD_ERR_INVALID_ARG;
  if (a->max_prompt_len < a->n_obs) return MD_ERR_INVALID_ARG;
  if (a->votes_stride < 1 || a->votes_stride < a->max_prompt_len - a->n_obs)
    return MD_ERR_INVALID_ARG;
  const bool paged = a->page_size != 0;
  if (a->page_size < 0) return MD_ERR_INVALID_ARG;
  if (paged) {
    if (!is_pow2(a->page_size) || a->max_pages_per_seq < 1 || a->num_pages < 1 ||
        a->num_pages > INT32_MAX)
      return MD_ERR_INVALID_ARG;
    if (ceil_div(a->max_prompt_len, a->page_size) > a->max_pages_per_seq) return MD_ERR_INVALID_ARG;
  }
  if (a->kv_stride_blk < 0 || a->kv_stride_tok < 0 || a->kv_stride_head < 0)
    return MD_ERR_INVALID_ARG;
  if (a->head_dim != 64 && a->head_dim != 128) return MD_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(a->num_q_heads / a->num_kv_heads) * a->n_obs > kSnapkvMaxRows)
    return MD_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(a->num_seqs) * a->num_kv_heads > INT32_MAX) return MD_ERR_UNSUPPORTED;
  if (a->num_seqs == 0) return MD_OK;
  if (!a->q_obs || !a->k || !a->prompt_lens || !a->votes) return MD_ERR_INVALID_ARG;
  if (paged != (a->page_table != nullptr)) return MD_ERR_INVALID_ARG;
  if (!aligned16(a->q_obs) || !aligned16(a->k) || (reinterpret_cast<uintptr_t>(a->votes) & 3u) ||
      (reinterpret_cast<uintptr_t>(a->prompt_lens) & 3u))
    return MD_ERR_INVALID_ARG;
  const int64_t per16 = a->dtype == MD_BF16 ? 8 : 4;
  if (a->kv_stride_blk % per16 || a->kv_stride_tok % per16 || a->kv_stride_head % per16)
    return MD_ERR_INVALID_ARG;
  if (a->num_kv_heads > 1 && a->kv_stride_head < a->head_dim) return MD_ERR_INVALID_ARG;
  const SnapkvPlan pl = make_snapkv_plan(a, device_cu_count());
  if (!a->workspace || a->workspace_bytes < pl.workspace_bytes ||
      (reinterpret_cast<uintptr_t>(a->workspace) & 255u))
    return MD_ERR_WORKSPACE;
  return MD_OK;
}

SnapkvPlan make_snapkv_plan(const md_snapkv_args* a, int num_cus) {
  SnapkvPlan p;
  p.G = a->num_q_heads / a->num_kv_heads;
  p.R = p.G * a->n_obs;
  p.TW = p.R <= 64 ? 1 : (p.R <= 128 ? 2 : 4);
  p.n_units = a->num_seqs * a->num_kv_heads;
  // Above 64 rows both passes take shorter chunks in several rounds of
  // resident workgroups (measured at 128 rows and 512 units: 4096
  // workgroups within 0.5% of 2048 and 2-6% faster than 1024, which leaves
  // part of the last round's slots idle).
  const int wg_per_cu = p.TW == 1 ? 2 : 8;
  split_range(a->max_prompt_len, p.n_units, num_cus, wg_per_cu, &p.n_chunks_stats,
              &p.chunk_len_stats);
  split_range(a->max_prompt_len - a->n_obs, p.n_units, num_cus, wg_per_cu, &p.n_chunks_votes,
              &p.chunk_len_votes);
  p.part_bytes = align_up(static_cast<size_t>(p.n_units) * p.n_chunks_stats * p.R * 4, 256);
  p.lse_bytes = align_up(static_cast<size_t>(p.n_units) * p.R * 4, 256);
  p.workspace_bytes = 2 * p.part_bytes + p.lse_bytes;
  return p;
}

int validate_accept(int32_t num_seqs, int32_t n_draft, int32_t vocab, int32_t dtype) {
  // vocab <= 2^30: a chunk's length, rounded up to 8 elements, stays an int32.
  if (num_seqs < 0 || n_draft < 0 || n_draft + 1 > kAcceptMaxRowsPerSeq || vocab < 1 ||
      vocab > (1 << 30))
    return MD_ERR_INVALID_ARG;
  if (dtype != MD_F32 && dtype != MD_BF16) return MD_ERR_INVALID_ARG;
  const int64_t rows = static_cast<int64_t>(num_seqs) * (n_draft + 1);
  if (rows * 64 > INT32_MAX) return MD_ERR_INVALID_ARG;  // grid bound at the largest split
  return MD_OK;
}

AcceptPlan make_accept_plan(int32_t num_seqs, int32_t n_draft, int32_t vocab, int num_cus) {
  AcceptPlan pl;
  const int64_t rows = static_cast<int64_t>(num_seqs) * (n_draft + 1);
  if (rows <= 0 || vocab < 1) return pl;
  constexpr int64_t kMinChunk = 2048;
  const int64_t L = n_draft + 1;
  int64_t n = (8 * static_cast<int64_t>(num_cus) + rows - 1) / rows;
  n = std::min<int64_t>(n, (vocab + kMinChunk - 1) / kMinChunk);
  n = std::min<int64_t>(n, kAcceptMaxPartialsPerSeq / L);  // the accept pass stages L * n in LDS
  n = std::max<int64_t>(1, std::min<int64_t>(n, 64));
  int64_t len = (vocab + n - 1) / n;
  len = (len + 7) / 8 * 8;
  pl.chunk_len = static_cast<int32_t>(len);
  pl.n_chunks = static_cast<int32_t>((vocab + len - 1) / len);
  pl.part_bytes = align_up(static_cast<size_t>(rows) * pl.n_chunks * 4, 256);
  pl.workspace_bytes = 2 * pl.part_bytes;
  return pl;
}

int validate_kv_cache(const md_kv_cache* c, int32_t n_new) {
  if (!c || n_new < 0) return MD_ERR_INVALID_ARG;
  if (c->num_seqs < 0 || c->num_kv_heads < 1 || c->head_dim < 1) return MD_ERR_INVALID_ARG;
  if (c->dtype != MD_F32 && c->dtype != MD_BF16) return MD_ERR_INVALID_ARG;
  const int64_t es = c->dtype == MD_BF16 ? 2 : 4;
  if ((c->head_dim * es) % 16) return MD_ERR_INVALID_ARG;
  if (c->kv_stride_blk < 0 || c->kv_stride_tok < 0 || c->kv_stride_head < 0 ||
      (c->kv_stride_blk * es) % 16 || (c->kv_stride_tok * es) % 16 || (c->kv_stride_head * es) % 16)
    return MD_ERR_INVALID_ARG;
  if (c->page_size != 0) {
    if (c->page_size < 0 || (c->page_size & (c->page_size - 1)) || !c->page_table ||
        c->max_pages_per_seq < 1 || c->num_pages < 1)
      return MD_ERR_INVALID_ARG;
  } else {
    if (c->page_table || c->capacity < 1) return MD_ERR_INVALID_ARG;
  }
  return MD_OK;
}

}  // namespace md
