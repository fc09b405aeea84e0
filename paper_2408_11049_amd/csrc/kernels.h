// kernels.h -- device-side parameter blocks and the launchers of the HIP
// kernels behind the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "magicdec.h"

namespace md {

// Everything one attention launch needs, passed by value as the kernel
// argument.  Strides are in elements; pointers are device pointers.
struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  int64_t s_blk, s_tok, s_head;
  const int32_t* page_table;  // [B, max_pages] (paged instances only)
  int32_t page_shift;         // log2(page_size)
  int32_t max_pages;
  int64_t num_pages;
  const int32_t* kv_lens;
  int32_t max_kv_len;
  int32_t L, Hq, Hkv, G, R;
  float scale_log2;           // softmax scale * log2(e)
  int32_t mode, n_sink, window;
  int32_t n_chunks, chunk_len;
  void* o;                    // final O (single chunk)
  float* lse;                 // final lse or nullptr (single chunk)
  float* part_o;              // [n_chunks][n_rows][d] (several chunks)
  float* part_lse;            // [n_chunks][n_rows]
  // Several chunks: one arrival counter per head group; the last workgroup
  // of a group to finish merges its chunks (see attn.hip).  A counter holds
  // (tag << 16) | arrivals, so a value left by anything but this call reads
  // as zero arrivals; the last arrival resets it to 0.  merge_launch = 1
  // (the default) leaves the merge to a separate launch instead.
  unsigned long long* counters;
  unsigned long long tag;     // per call: nonzero, below 2^48
  int32_t merge_launch;
  // Measurement only (NULL in normal use): per workgroup, four wall-clock
  // stamps (start, first K/V tile staged, main loop done, end).
  unsigned long long* stamps;
  int64_t n_rows;
  int32_t num_seqs;           // B
  int32_t lpt;                // 1: workgroups take sequences longest first (see attn.hip)
  int32_t bal;                // 1: the balanced verify instances (see attn.hip): grid = workgroups
                              // sharing all groups' tiles equally; workgroup w keeps the partials
                              // of its range's first / last piece in slots 2w / 2w + 1
  int32_t hp;                 // kv heads per workgroup (1 or 2; divides Hkv)
  int32_t waves;              // waves per workgroup: kWaves, or kWavesWide (up to two row
                              // tiles of bf16, not listed, not balanced)
  int32_t hp_auto;            // longest-first launch of one workgroup per unit that
                              // pairs heads when the lengths allow (see attn.hip)
  int32_t slots;              // compute units of the device (hp_auto's balance test)
  const int32_t* idx;         // indexed draft: [B, Hkv, idx_stride] prompt positions
  const int32_t* idx_len;     // indexed draft: [B] list lengths
  int32_t idx_stride;
  int32_t* err;               // md_attn_args.err_word, or nullptr
};

// depth: K/V tiles each wave keeps in flight (1..3; bf16 instances).
// occ: waves per SIMD the instance is compiled for (2 only with depth 1 and
// NT <= 2; otherwise 1).
// SnapKV-style selection (prefill): votes passes and the selection.
struct SnapkvParams {
  const void* q;              // observation queries [B, n_obs, Hq, d]
  const void* k;
  int64_t s_blk, s_tok, s_head;
  const int32_t* page_table;
  int32_t page_shift, max_pages;
  int64_t num_pages;
  const int32_t* kv_lens;     // prompt lengths [B]
  int32_t max_kv_len;
  int32_t n_obs, Hq, Hkv, G, R;
  float scale_log2;
  int32_t n_units;
  int32_t n_chunks, chunk_len;              // of the pass being launched
  int32_t n_chunks_stats, chunk_len_stats;  // softmax statistics pass
  int32_t n_chunks_votes, chunk_len_votes;  // votes pass
  float* part_m;              // [units][n_chunks_stats][R]
  float* part_l;
  float* lse2;                // [units][R]
  float* votes;               // [B, Hkv, votes_stride]
  int32_t votes_stride;
};

struct SnapkvSelectParams {
  const float* votes;         // [rows][stride]
  int32_t stride;
  const int32_t* lens;        // prompt lengths [B]
  int32_t rows, rows_per_seq;
  int32_t n_obs, pool, budget;
  int32_t* idx;               // [rows][budget]
  int32_t* counts;            // [B]
};

hipError_t launch_snapkv_votes(const SnapkvParams& p, int head_dim, bool bf16, int TW, bool paged,
                               hipStream_t s);
hipError_t launch_snapkv_select(const SnapkvSelectParams& p, hipStream_t s);

hipError_t launch_attn_partial(const AttnParams& p, int head_dim, bool bf16, int NT, bool paged,
                               int depth, int occ, int64_t n_blocks, hipStream_t s);

// parts_readable: every part's O may be read, empty parts included (the
// library's own split plans); md_merge_lse never reads an empty part's O.
hipError_t launch_merge_lse(int n_parts, int64_t n_rows, int head_dim, bool out_bf16,
                            const float* o_parts, const float* lse_parts, void* o, float* lse,
                            hipStream_t s, bool parts_readable);

// The speculative step around verification.
struct AppendParams {
  const unsigned char* k_new;  // [B, n_new, Hkv, d] bytes
  const unsigned char* v_new;
  unsigned char* k;            // cache base pointers (bytes)
  unsigned char* v;
  int64_t s_blk, s_tok, s_head;  // element strides
  int32_t esize;
  const int32_t* page_table;
  int32_t page_shift, max_pages;
  int64_t num_pages;
  int32_t capacity;            // contiguous: tokens per sequence block
  const int32_t* pos0;
  int32_t* lens_out;
  int32_t B, n_new, Hkv, row_vecs;  // row_vecs = 16-byte vectors per (token, head) row
  int64_t n_items;             // 2 * B * n_new * Hkv * row_vecs
};

// One cache as the gather kernel addresses it (element strides).
struct CacheView {
  unsigned char* k;
  unsigned char* v;
  int64_t s_blk, s_tok, s_head;
  const int32_t* page_table;  // [B, max_pages] (paged)
  int32_t page_shift;
  int32_t max_pages;
  int64_t num_pages;
  int64_t capacity;           // tokens per sequence (contiguous)
};

struct GatherParams {
  CacheView dst, src;
  const int32_t* idx;       // [B, Hkv, idx_stride]
  int32_t idx_stride;
  const int32_t* idx_len;   // [B]
  const int32_t* src_lens;  // [B]
  int32_t* dst_lens;        // [B] or nullptr
  int32_t B, Hkv;
  int32_t row_vecs;         // 16-byte vectors per row (d * element size / 16)
  int32_t esize;
  int64_t n_items;          // 2 (K, V) * B * idx_stride * Hkv * row_vecs
  int32_t vec_shift;        // log2(row_vecs) and log2(Hkv) when both are powers of
  int32_t head_shift;       // two (then one grid row per sequence), else -1
};

struct AcceptParams {
  const void* logits;          // [rows][vocab]
  int32_t vocab, n_chunks, chunk_len;  // chunk_len: elements, a multiple of 8
  int32_t B, L;                // rows = B * L
  float* part_val;             // [rows][n_chunks]
  int32_t* part_idx;
  const int32_t* draft;        // [B, L - 1]
  int32_t* accepted;
  int32_t* tokens;             // [B, L]
  int32_t* target;             // [B, L] or nullptr
};

hipError_t launch_kv_gather(const GatherParams& p, bool src_paged, bool dst_paged, hipStream_t s);
hipError_t launch_kv_append(const AppendParams& p, bool paged, hipStream_t s);
hipError_t launch_greedy_accept(const AcceptParams& p, bool bf16, bool vec, hipStream_t s);
hipError_t launch_kv_commit(int B, int q_len, int32_t* lens, const int32_t* accepted, int Hkv,
                            int32_t* idx, int idx_stride, int ring_start, int ring_len,
                            hipStream_t s);
hipError_t launch_streaming_list(int B, int Hkv, const int32_t* prompt_lens, int n_sink,
                                 int window, int32_t* idx, int32_t* idx_len, hipStream_t s);

// Records a HIP error's text for md_last_hip_error (calling thread) and
// returns MD_ERR_HIP.
int hip_fail(hipError_t e);

hipError_t launch_bench_read(const void* buf, size_t bytes, float* sink, int n_blocks,
                             hipStream_t s);
hipError_t launch_bench_evict(const void* buf, size_t bytes, float* sink, int n_blocks,
                              hipStream_t s);
hipError_t launch_bench_copy(void* dst, const void* src, size_t bytes, int n_blocks,
                             hipStream_t s);
hipError_t launch_bench_fill(void* buf, size_t bytes, uint32_t value, int n_blocks,
                             hipStream_t s);

}  // namespace md
