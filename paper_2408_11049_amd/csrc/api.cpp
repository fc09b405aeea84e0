// api.cpp -- the C ABI of libmagicdec.so: argument checks, the split-KV plan,
// and the launches on the caller's stream.  No allocation, no host sync.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>

#include <algorithm>
#include <atomic>
#include <string>

#include "internal.h"
#include "kernels.h"
#include "magicdec.h"
#include "magicdec_bench.h"

namespace md {

namespace {

CacheView cache_view(const md_kv_cache* c) {
  CacheView v{};
  v.k = static_cast<unsigned char*>(c->k);
  v.v = static_cast<unsigned char*>(c->v);
  v.s_blk = c->kv_stride_blk;
  v.s_tok = c->kv_stride_tok;
  v.s_head = c->kv_stride_head;
  v.page_table = c->page_table;
  v.page_shift = 0;
  if (c->page_size)
    while ((1 << v.page_shift) < c->page_size) ++v.page_shift;
  v.max_pages = c->max_pages_per_seq;
  v.num_pages = c->num_pages;
  v.capacity = c->capacity;
  return v;
}

bool overlaps(const void* a, const void* b, size_t n) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + n && y < x + n;
}

thread_local std::string g_last_hip_error;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// K/V tiles in flight per wave.  MD_PREFETCH_DEPTH (1..3) overrides the
// default, for tuning sweeps.
int prefetch_depth(int NT, int mode) {
  const int forced = env_knob("MD_PREFETCH_DEPTH", 1, 3);
  (void)NT;
  (void)mode;
  // Measured on MI355X: with K and V both streamed as whole rows, one tile in
  // flight per wave already saturates HBM for every shape; deeper rings
  // only cost registers.
  return forced ? forced : 1;
}

// Waves per SIMD targeted by the kernel instance (MD_OCCUPANCY = 1 or 2
// overrides, for tuning sweeps).  Long verify streams with two row tiles run
// best at one wave per SIMD (more registers, no spills); the short draft
// calls and single-row-tile shapes at two.
int occupancy(int NT, int depth, int mode) {
  const int forced = env_knob("MD_OCCUPANCY", 1, 2);
  if (forced) return forced;
  if (depth != 1 || NT > 2) return 1;
  return (mode == MD_MODE_VERIFY && NT == 2) ? 1 : 2;
}

// Longest-first dispatch pays where units differ in length and each is long:
// single-chunk verify plans of long caches (the ranking costs B compares per
// thread, so small batches only).  MD_LPT = 1 or 2 forces it off (1) or on
// where allowed (2), for A/B measurements.
int longest_first(int mode, int n_chunks, int num_seqs, int max_kv_len) {
  const int forced = env_knob("MD_LPT", 1, 2);
  if (mode != MD_MODE_VERIFY || n_chunks != 1 || num_seqs < 2 || num_seqs > kLptMaxSeqs)
    return 0;
  if (forced) return forced == 2;
  return max_kv_len >= kLptMinLen;
}

}  // namespace

int hip_fail(hipError_t e) {
  g_last_hip_error = hipGetErrorString(e);
  (void)hipGetLastError();  // the launch error is reported here, not to the next call
  return MD_ERR_HIP;
}

namespace {

// A fresh tag per attention call (1 .. 2^48 - 1; a process would need
// centuries of calls to wrap it): it marks the arrival counters of that
// call's split plan (see attn.hip).
unsigned long long next_call_tag() {
  static std::atomic<unsigned long long> seq{0};
  constexpr unsigned long long kMask = (1ull << 48) - 1;
  unsigned long long t = (seq.fetch_add(1, std::memory_order_relaxed) + 1) & kMask;
  while (t == 0) t = (seq.fetch_add(1, std::memory_order_relaxed) + 1) & kMask;
  return t;
}

// Waves per workgroup.  The wide instances (two waves per SIMD in one
// workgroup, each taking half of the unit's tiles) exist for up to two row
// tiles of bf16 outside the listed draft and the balanced verify.  Measured
// on MI355X (same process): drafts whose waves would each take 16 tiles ran
// 3-6% faster wide (one-token drafts at one row tile, (gamma+1)-token drafts
// at two), those at 4-8 tiles per wave 4-5% slower (the merge of eight waves
// and a larger first burst), long verifies within 1% either way at one row
// tile and slower at two; so drafts take them from 16 tiles per wave.
// MD_WAVES = 4 / 8 forces either (measurement).
int waves_per_workgroup(const Plan& pl, int mode, bool bf16) {
  if (!bf16 || pl.NT > 2 || mode == MD_MODE_DRAFT_INDEXED || pl.bal) return kWaves;
  const int forced = env_knob("MD_WAVES", kWaves, kWavesWide);
  if (forced == kWaves || forced == kWavesWide) return forced;
  if (mode != MD_MODE_DRAFT) return kWaves;
  const int64_t range = std::min<int64_t>(pl.U_max, pl.chunk_len);
  const int64_t tiles_per_wave = (range + kTile - 1) / kTile / (kWaves / pl.hp);
  return tiles_per_wave >= 16 ? kWavesWide : kWaves;
}

// Workgroups of an attention launch: a head group per chunk; for a
// longest-first launch that may pair heads, one per unit; for the balanced
// verify, one per range of its tile stream.
int64_t grid_size(const Plan& pl, int lpt) {
  if (pl.bal) return pl.bal_nw;
  return (lpt && pl.hp == 2) ? pl.n_units : pl.n_groups * pl.n_chunks;
}

}  // namespace

int64_t attn_grid_size(const md_attn_args* a, int mode, int n_sink, int window) {
  const Plan pl = make_plan(a, mode, n_sink, window, device_cu_count());
  return grid_size(pl, !pl.bal && longest_first(mode, pl.n_chunks, a->num_seqs, a->max_kv_len));
}

// The attention entry points.  `workspace`/`workspace_bytes` override the
// caller's workspace in `a` (the entry point without allocation passes the
// library's own buffer); `stamps` is the measurement hook (NULL normally).
int run_attention(const md_attn_args* a, int mode, int n_sink, int window, void* stream,
                  const int32_t* idx, const int32_t* idx_len, void* workspace,
                  size_t workspace_bytes, unsigned long long* stamps) {
  md_attn_args local;
  if (a && workspace) {
    local = *a;
    local.workspace = workspace;
    local.workspace_bytes = workspace_bytes;
    a = &local;
  }
  if (a) workspace = a->workspace;
  int st = validate_attn(a, mode, n_sink, window);
  if (st != MD_OK) return st;
  if (a->num_seqs == 0) return MD_OK;
  if (mode == MD_MODE_DRAFT_INDEXED) {
    if (!idx || !idx_len) return MD_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(idx) & 3u) || (reinterpret_cast<uintptr_t>(idx_len) & 3u))
      return MD_ERR_INVALID_ARG;
  }
  const int num_cus = device_cu_count();
  const Plan pl = make_plan(a, mode, n_sink, window, num_cus);
  const bool bf16 = a->dtype == MD_BF16;
  const bool paged = a->page_size != 0;

  AttnParams p{};
  p.q = a->q;
  p.k = a->k;
  p.v = a->v;
  p.s_blk = a->kv_stride_blk;
  p.s_tok = a->kv_stride_tok;
  p.s_head = a->kv_stride_head;
  p.page_table = a->page_table;
  p.page_shift = 0;
  if (paged)
    while ((1 << p.page_shift) < a->page_size) ++p.page_shift;
  p.max_pages = a->max_pages_per_seq;
  p.num_pages = a->num_pages;
  p.kv_lens = a->kv_lens;
  p.max_kv_len = a->max_kv_len;
  p.L = a->q_len;
  p.Hq = a->num_q_heads;
  p.Hkv = a->num_kv_heads;
  p.G = pl.G;
  p.R = pl.R;
  const float scale = a->sm_scale > 0.f ? a->sm_scale : 1.0f / sqrtf(static_cast<float>(a->head_dim));
  p.scale_log2 = scale * 1.44269504088896340736f;
  p.mode = mode;
  p.n_sink = mode == MD_MODE_DRAFT ? n_sink : 0;
  p.window = mode == MD_MODE_DRAFT ? window : 1;
  if (mode == MD_MODE_DRAFT_INDEXED) {
    p.idx = idx;
    p.idx_len = idx_len;
    p.idx_stride = window;
  }
  p.n_chunks = pl.n_chunks;
  p.chunk_len = pl.chunk_len;
  p.num_seqs = a->num_seqs;
  p.lpt = !pl.bal && longest_first(mode, pl.n_chunks, a->num_seqs, a->max_kv_len);
  p.bal = pl.bal;
  p.waves = waves_per_workgroup(pl, mode, bf16);
  p.hp = pl.hp;
  p.err = a->err_word;
  const int64_t n_blocks = grid_size(pl, p.lpt);
  if (p.lpt && pl.hp == 2) {
    // One workgroup per unit; the kernel pairs heads (and idles the surplus
    // half) only when longest-first can still balance the pairs.
    p.hp = 1;
    p.hp_auto = 1;
    p.slots = num_cus > 0 ? num_cus : 256;
  }
  p.o = a->o;
  p.lse = a->lse;
  p.n_rows = pl.n_rows;
  if (pl.n_chunks > 1 || pl.bal) {
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    p.counters = reinterpret_cast<unsigned long long*>(ws);
    p.part_o = reinterpret_cast<float*>(ws + pl.counter_bytes);
    p.part_lse = reinterpret_cast<float*>(ws + pl.counter_bytes + pl.part_o_bytes);
    p.tag = next_call_tag();
    // The chunks merge in a second launch by default.  MD_FUSED_MERGE = 1
    // merges them inside the attention launch instead, in the last workgroup
    // of each head group to finish: measured on MI355X, same process, that
    // was 1-10 us slower per call (the second launch follows the first with
    // no gap on the stream, and the device-scope fences around the arrival
    // counters cost more than the launch saves), so it stays opt-in.  The
    // balanced verify always merges its cut groups inside the launch: only
    // the kernel knows which groups its ranges cut.
    p.merge_launch = !env_knob("MD_FUSED_MERGE", 1, 1);
  }
  p.stamps = stamps;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int depth = prefetch_depth(pl.NT, mode);
  hipError_t e = launch_attn_partial(p, a->head_dim, bf16, pl.NT, paged, depth,
                                     occupancy(pl.NT, depth, mode), n_blocks, s);
  if (e != hipSuccess) return hip_fail(e);
  if (pl.n_chunks > 1 && p.merge_launch) {
    e = launch_merge_lse(pl.n_chunks, pl.n_rows, a->head_dim, bf16, p.part_o, p.part_lse, a->o,
                         a->lse, s, true);
    if (e != hipSuccess) return hip_fail(e);
  }
  return MD_OK;
}

int device_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 256;
  }
  int c = cache[dev].load(std::memory_order_relaxed);
  if (c > 0) return c;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace md

extern "C" {

int md_verify_attn(const md_attn_args* a, void* stream) {
  return md::run_attention(a, MD_MODE_VERIFY, 0, 1, stream, nullptr, nullptr, nullptr, 0,
                           nullptr);
}

int md_draft_attn(const md_attn_args* a, int32_t n_sink, int32_t window, void* stream) {
  return md::run_attention(a, MD_MODE_DRAFT, n_sink, window, stream, nullptr, nullptr, nullptr,
                           0, nullptr);
}

int md_draft_attn_indexed(const md_attn_args* a, const int32_t* idx, const int32_t* idx_len,
                          int32_t idx_stride, void* stream) {
  return md::run_attention(a, MD_MODE_DRAFT_INDEXED, 0, idx_stride, stream, idx, idx_len,
                           nullptr, 0, nullptr);
}

int md_bench_attn_stamps(const md_attn_args* a, int32_t mode, int32_t n_sink, int32_t window,
                         uint64_t* stamps, int64_t stamps_len, int64_t* n_workgroups,
                         void* stream) {
  if (!a || !n_workgroups || (mode != MD_MODE_VERIFY && mode != MD_MODE_DRAFT))
    return MD_ERR_INVALID_ARG;
  const int st = md::validate_attn(a, mode, n_sink, window);
  if (st != MD_OK) return st;
  *n_workgroups = md::attn_grid_size(a, mode, n_sink, window);
  if (!stamps || (reinterpret_cast<uintptr_t>(stamps) & 7u) || stamps_len < 4 * *n_workgroups)
    return MD_ERR_INVALID_ARG;
  return md::run_attention(a, mode, n_sink, window, stream, nullptr, nullptr, nullptr, 0,
                           reinterpret_cast<unsigned long long*>(stamps));
}

int md_merge_lse(int32_t n_parts, int64_t n_rows, int32_t head_dim, int32_t out_dtype,
                 const float* o_parts, const float* lse_parts, void* o, float* lse,
                 void* stream) {
  if (n_parts < 1 || n_rows < 0) return MD_ERR_INVALID_ARG;
  if (out_dtype != MD_F32 && out_dtype != MD_BF16) return MD_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return MD_ERR_UNSUPPORTED;
  if ((n_rows + 3) / 4 > INT32_MAX) return MD_ERR_UNSUPPORTED;  // four rows per workgroup
  if (n_rows == 0) return MD_OK;
  if (!o_parts || !lse_parts || !o) return MD_ERR_INVALID_ARG;
  if (!md::aligned16(o_parts) || !md::aligned16(lse_parts) || !md::aligned16(o) || (lse && !md::aligned16(lse)))
    return MD_ERR_INVALID_ARG;
  hipError_t e = md::launch_merge_lse(n_parts, n_rows, head_dim, out_dtype == MD_BF16, o_parts,
                                      lse_parts, o, lse, static_cast<hipStream_t>(stream), false);
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

size_t md_workspace_bytes(const md_attn_args* a, int32_t mode, int32_t n_sink, int32_t window) {
  if (!a) return 0;
  if (mode != MD_MODE_VERIFY && mode != MD_MODE_DRAFT) return 0;
  if (mode == MD_MODE_DRAFT && (n_sink < 0 || window < 1 || window > md::kMaxPosition)) return 0;
  if (md::check_attn_sizes(a) != MD_OK) return 0;
  return md::make_plan(a, mode, n_sink, window, md::device_cu_count()).workspace_bytes;
}

size_t md_workspace_bytes_indexed(const md_attn_args* a, int32_t idx_stride) {
  if (!a || idx_stride < 1 || idx_stride > md::kMaxPosition) return 0;
  if (md::check_attn_sizes(a) != MD_OK) return 0;
  return md::make_plan(a, MD_MODE_DRAFT_INDEXED, 0, idx_stride, md::device_cu_count())
      .workspace_bytes;
}

int md_snapkv_votes(const md_snapkv_args* a, void* stream) {
  const int st = md::validate_snapkv(a);
  if (st != MD_OK) return st;
  if (a->num_seqs == 0) return MD_OK;
  const md::SnapkvPlan pl = md::make_snapkv_plan(a, md::device_cu_count());
  md::SnapkvParams p{};
  p.q = a->q_obs;
  p.k = a->k;
  p.s_blk = a->kv_stride_blk;
  p.s_tok = a->kv_stride_tok;
  p.s_head = a->kv_stride_head;
  p.page_table = a->page_table;
  p.page_shift = 0;
  if (a->page_size)
    while ((1 << p.page_shift) < a->page_size) ++p.page_shift;
  p.max_pages = a->max_pages_per_seq;
  p.num_pages = a->num_pages;
  p.kv_lens = a->prompt_lens;
  p.max_kv_len = a->max_prompt_len;
  p.n_obs = a->n_obs;
  p.Hq = a->num_q_heads;
  p.Hkv = a->num_kv_heads;
  p.G = pl.G;
  p.R = pl.R;
  const float scale =
      a->sm_scale > 0.f ? a->sm_scale : 1.0f / sqrtf(static_cast<float>(a->head_dim));
  p.scale_log2 = scale * 1.44269504088896340736f;
  p.n_units = pl.n_units;
  p.n_chunks_stats = pl.n_chunks_stats;
  p.chunk_len_stats = pl.chunk_len_stats;
  p.n_chunks_votes = pl.n_chunks_votes;
  p.chunk_len_votes = pl.chunk_len_votes;
  unsigned char* ws = static_cast<unsigned char*>(a->workspace);
  p.part_m = reinterpret_cast<float*>(ws);
  p.part_l = reinterpret_cast<float*>(ws + pl.part_bytes);
  p.lse2 = reinterpret_cast<float*>(ws + 2 * pl.part_bytes);
  p.votes = a->votes;
  p.votes_stride = a->votes_stride;
  const hipError_t e = md::launch_snapkv_votes(p, a->head_dim, a->dtype == MD_BF16, pl.TW,
                                               a->page_size != 0,
                                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

size_t md_snapkv_workspace_bytes(const md_snapkv_args* a) {
  if (!a || a->num_seqs < 0 || a->n_obs < 1 || a->num_q_heads < 1 || a->num_kv_heads < 1 ||
      a->num_q_heads % a->num_kv_heads || a->max_prompt_len < a->n_obs ||
      static_cast<int64_t>(a->num_seqs) * a->num_kv_heads > INT32_MAX)
    return 0;
  return md::make_snapkv_plan(a, md::device_cu_count()).workspace_bytes;
}

int md_snapkv_select(int32_t num_seqs, int32_t num_kv_heads, const float* votes,
                     int32_t votes_stride, const int32_t* prompt_lens, int32_t n_obs,
                     int32_t pool, int32_t budget, int32_t* idx, int32_t* idx_len, void* stream) {
  if (num_seqs < 0 || num_kv_heads < 1 || votes_stride < 1 || n_obs < 0 || pool < 1 ||
      pool % 2 == 0 || budget < n_obs || budget < 1)
    return MD_ERR_INVALID_ARG;
  if (num_seqs == 0) return MD_OK;
  if (!votes || !prompt_lens || !idx || !idx_len) return MD_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(votes) & 3u) || (reinterpret_cast<uintptr_t>(prompt_lens) & 3u) ||
      (reinterpret_cast<uintptr_t>(idx) & 3u) || (reinterpret_cast<uintptr_t>(idx_len) & 3u))
    return MD_ERR_INVALID_ARG;
  if (static_cast<int64_t>(num_seqs) * num_kv_heads > INT32_MAX) return MD_ERR_INVALID_ARG;
  md::SnapkvSelectParams p{};
  p.votes = votes;
  p.stride = votes_stride;
  p.lens = prompt_lens;
  p.rows = num_seqs * num_kv_heads;
  p.rows_per_seq = num_kv_heads;
  p.n_obs = n_obs;
  p.pool = pool;
  p.budget = budget;
  p.idx = idx;
  p.counts = idx_len;
  const hipError_t e = md::launch_snapkv_select(p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_kv_append(const md_kv_cache* c, int32_t n_new, const void* k_new, const void* v_new,
                 const int32_t* pos0, int32_t* lens_out, void* stream) {
  const int st = md::validate_kv_cache(c, n_new);
  if (st != MD_OK) return st;
  if (c->num_seqs == 0 || n_new == 0) return MD_OK;
  if (!c->k || !c->v || !k_new || !v_new || !pos0) return MD_ERR_INVALID_ARG;
  if (!md::aligned16(c->k) || !md::aligned16(c->v) || !md::aligned16(k_new) ||
      !md::aligned16(v_new) || (reinterpret_cast<uintptr_t>(pos0) & 3u) ||
      (reinterpret_cast<uintptr_t>(lens_out) & 3u))
    return MD_ERR_INVALID_ARG;
  if (lens_out) {  // every thread reads pos0[b] while one writes lens_out[b]: no overlap
    const uintptr_t lo = reinterpret_cast<uintptr_t>(lens_out), po = reinterpret_cast<uintptr_t>(pos0);
    const uintptr_t n = static_cast<uintptr_t>(c->num_seqs) * 4;
    if (lo < po + n && po < lo + n) return MD_ERR_INVALID_ARG;
  }
  const int es = c->dtype == MD_BF16 ? 2 : 4;
  md::AppendParams p{};
  p.k_new = static_cast<const unsigned char*>(k_new);
  p.v_new = static_cast<const unsigned char*>(v_new);
  p.k = static_cast<unsigned char*>(c->k);
  p.v = static_cast<unsigned char*>(c->v);
  p.s_blk = c->kv_stride_blk;
  p.s_tok = c->kv_stride_tok;
  p.s_head = c->kv_stride_head;
  p.esize = es;
  p.page_table = c->page_table;
  p.page_shift = 0;
  if (c->page_size)
    while ((1 << p.page_shift) < c->page_size) ++p.page_shift;
  p.max_pages = c->max_pages_per_seq;
  p.num_pages = c->num_pages;
  p.capacity = c->capacity;
  p.pos0 = pos0;
  p.lens_out = lens_out;
  p.B = c->num_seqs;
  p.n_new = n_new;
  p.Hkv = c->num_kv_heads;
  p.row_vecs = c->head_dim * es / 16;
  p.n_items = 2 * static_cast<int64_t>(c->num_seqs) * n_new * c->num_kv_heads * p.row_vecs;
  const hipError_t e = md::launch_kv_append(p, c->page_size != 0, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_kv_gather(const md_kv_cache* dst, const md_kv_cache* src, const int32_t* idx,
                 int32_t idx_stride, const int32_t* idx_len, const int32_t* src_lens,
                 int32_t* dst_lens, void* stream) {
  int st = md::validate_kv_cache(dst, 0);
  if (st != MD_OK) return st;
  st = md::validate_kv_cache(src, 0);
  if (st != MD_OK) return st;
  if (dst->num_seqs != src->num_seqs || dst->num_kv_heads != src->num_kv_heads ||
      dst->head_dim != src->head_dim || dst->dtype != src->dtype || idx_stride < 1)
    return MD_ERR_INVALID_ARG;
  // Every list entry has a destination row: a shorter cache would drop rows
  // while dst_lens still counted them.
  const int64_t dst_rows = dst->page_size
                               ? static_cast<int64_t>(dst->max_pages_per_seq) * dst->page_size
                               : static_cast<int64_t>(dst->capacity);
  if (dst_rows < idx_stride) return MD_ERR_INVALID_ARG;
  if (dst->num_seqs == 0) return MD_OK;
  if (!dst->k || !dst->v || !src->k || !src->v || !idx || !idx_len || !src_lens)
    return MD_ERR_INVALID_ARG;
  if (!md::aligned16(dst->k) || !md::aligned16(dst->v) || !md::aligned16(src->k) ||
      !md::aligned16(src->v) || (reinterpret_cast<uintptr_t>(idx) & 3u) ||
      (reinterpret_cast<uintptr_t>(idx_len) & 3u) || (reinterpret_cast<uintptr_t>(src_lens) & 3u) ||
      (reinterpret_cast<uintptr_t>(dst_lens) & 3u))
    return MD_ERR_INVALID_ARG;
  const size_t nb = static_cast<size_t>(dst->num_seqs) * 4;
  // every thread reads idx_len[b] and src_lens[b] while one writes dst_lens[b]
  if (dst_lens && (md::overlaps(dst_lens, idx_len, nb) || md::overlaps(dst_lens, src_lens, nb)))
    return MD_ERR_INVALID_ARG;
  const int es = dst->dtype == MD_BF16 ? 2 : 4;
  md::GatherParams p{};
  p.dst = md::cache_view(dst);
  p.src = md::cache_view(src);
  p.idx = idx;
  p.idx_stride = idx_stride;
  p.idx_len = idx_len;
  p.src_lens = src_lens;
  p.dst_lens = dst_lens;
  p.B = dst->num_seqs;
  p.Hkv = dst->num_kv_heads;
  p.row_vecs = dst->head_dim * es / 16;
  p.esize = es;
  const double items = 2.0 * p.B * idx_stride * p.Hkv * p.row_vecs;
  if (items > 9.0e18) return MD_ERR_INVALID_ARG;
  p.n_items = 2 * static_cast<int64_t>(p.B) * idx_stride * p.Hkv * p.row_vecs;
  auto log2_exact = [](int32_t x) {
    int s = 0;
    while ((int64_t{1} << s) < x) ++s;
    return (int64_t{1} << s) == x ? s : -1;
  };
  p.vec_shift = log2_exact(p.row_vecs);
  p.head_shift = log2_exact(p.Hkv);
  const hipError_t e = md::launch_kv_gather(p, src->page_size != 0, dst->page_size != 0,
                                            static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

size_t md_greedy_accept_workspace_bytes(int32_t num_seqs, int32_t n_draft, int32_t vocab) {
  if (md::validate_accept(num_seqs, n_draft, vocab, MD_F32) != MD_OK) return 0;
  return md::make_accept_plan(num_seqs, n_draft, vocab, md::device_cu_count()).workspace_bytes;
}

int md_greedy_accept(int32_t num_seqs, int32_t n_draft, int32_t vocab, int32_t dtype,
                     const void* logits, const int32_t* draft, int32_t* accepted,
                     int32_t* tokens, int32_t* target, void* workspace, size_t workspace_bytes,
                     void* stream) {
  const int st = md::validate_accept(num_seqs, n_draft, vocab, dtype);
  if (st != MD_OK) return st;
  if (num_seqs == 0) return MD_OK;
  if (!logits || (n_draft > 0 && !draft) || !accepted || !tokens) return MD_ERR_INVALID_ARG;
  if (!md::aligned16(logits) || (reinterpret_cast<uintptr_t>(draft) & 3u) ||
      (reinterpret_cast<uintptr_t>(accepted) & 3u) || (reinterpret_cast<uintptr_t>(tokens) & 3u) ||
      (reinterpret_cast<uintptr_t>(target) & 3u))
    return MD_ERR_INVALID_ARG;
  const md::AcceptPlan pl = md::make_accept_plan(num_seqs, n_draft, vocab, md::device_cu_count());
  if (!workspace || workspace_bytes < pl.workspace_bytes ||
      (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return MD_ERR_WORKSPACE;
  md::AcceptParams p{};
  p.logits = logits;
  p.vocab = vocab;
  p.n_chunks = pl.n_chunks;
  p.chunk_len = pl.chunk_len;
  p.B = num_seqs;
  p.L = n_draft + 1;
  p.part_val = static_cast<float*>(workspace);
  p.part_idx = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(workspace) + pl.part_bytes);
  p.draft = draft;
  p.accepted = accepted;
  p.tokens = tokens;
  p.target = target;
  const int epv = dtype == MD_BF16 ? 8 : 4;
  const hipError_t e = md::launch_greedy_accept(p, dtype == MD_BF16, vocab % epv == 0,
                                                static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_kv_commit(int32_t num_seqs, int32_t q_len, int32_t* lens, const int32_t* accepted,
                 int32_t num_kv_heads, int32_t* idx, int32_t idx_stride, int32_t ring_start,
                 int32_t ring_len, void* stream) {
  if (num_seqs < 0 || q_len < 1) return MD_ERR_INVALID_ARG;
  if (idx && (num_kv_heads < 1 || idx_stride < 1 || ring_start < 0 || ring_len < 1 ||
              static_cast<int64_t>(ring_start) + ring_len > idx_stride))
    return MD_ERR_INVALID_ARG;
  if (num_seqs == 0) return MD_OK;
  if (!lens || !accepted || (reinterpret_cast<uintptr_t>(lens) & 3u) ||
      (reinterpret_cast<uintptr_t>(accepted) & 3u) || (reinterpret_cast<uintptr_t>(idx) & 3u))
    return MD_ERR_INVALID_ARG;
  const hipError_t e = md::launch_kv_commit(num_seqs, q_len, lens, accepted, num_kv_heads, idx,
                                            idx_stride, ring_start, ring_len,
                                            static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_streaming_list(int32_t num_seqs, int32_t num_kv_heads, const int32_t* prompt_lens,
                      int32_t n_sink, int32_t window, int32_t* idx, int32_t* idx_len,
                      void* stream) {
  if (num_seqs < 0 || num_kv_heads < 1 || n_sink < 0 || window < 1 ||
      static_cast<int64_t>(n_sink) + window > INT32_MAX ||
      static_cast<int64_t>(num_seqs) * num_kv_heads > INT32_MAX)
    return MD_ERR_INVALID_ARG;
  if (num_seqs == 0) return MD_OK;
  if (!prompt_lens || !idx || !idx_len || (reinterpret_cast<uintptr_t>(prompt_lens) & 3u) ||
      (reinterpret_cast<uintptr_t>(idx) & 3u) || (reinterpret_cast<uintptr_t>(idx_len) & 3u))
    return MD_ERR_INVALID_ARG;
  const hipError_t e = md::launch_streaming_list(num_seqs, num_kv_heads, prompt_lens, n_sink,
                                                 window, idx, idx_len,
                                                 static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

const char* md_status_str(int status) {
  switch (status) {
    case MD_OK: return "ok";
    case MD_ERR_INVALID_ARG: return "invalid argument";
    case MD_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case MD_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case MD_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* md_last_hip_error(void) { return md::g_last_hip_error.c_str(); }

size_t md_attn_args_size(void) { return sizeof(md_attn_args); }

int md_bench_stream_read(const void* buf, size_t bytes, float* sink, void* stream) {
  if (!buf || !sink || !md::aligned16(buf) || bytes % 16) return MD_ERR_INVALID_ARG;
  hipError_t e = md::launch_bench_read(buf, bytes, sink, md::device_cu_count() * 2,
                                       static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_bench_evict(const void* buf, size_t bytes, float* sink, void* stream) {
  if (!buf || !sink || !md::aligned16(buf) || bytes % 16) return MD_ERR_INVALID_ARG;
  hipError_t e = md::launch_bench_evict(buf, bytes, sink, md::device_cu_count() * 2,
                                        static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_bench_copy(void* dst, const void* src, size_t bytes, void* stream) {
  if (!dst || !src || !md::aligned16(dst) || !md::aligned16(src) || bytes % 16) return MD_ERR_INVALID_ARG;
  hipError_t e = md::launch_bench_copy(dst, src, bytes, md::device_cu_count() * 8,
                                       static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

int md_bench_fill(void* buf, size_t bytes, uint32_t value, void* stream) {
  if (!buf || !md::aligned16(buf) || bytes % 16) return MD_ERR_INVALID_ARG;
  hipError_t e = md::launch_bench_fill(buf, bytes, value, md::device_cu_count() * 8,
                                       static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MD_OK : md::hip_fail(e);
}

}  // extern "C"
