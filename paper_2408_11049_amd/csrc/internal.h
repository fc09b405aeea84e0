// internal.h -- host-side types shared by the entry points, the planner and
// the kernel launchers of libmagicdec.so.  No HIP types appear here, so the
// validation and planning code compiles and runs without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "magicdec.h"

namespace md {

// Work decomposition of one attention call.
//
// A "unit" is one (sequence b, kv head hk) pair: the G*L query rows that share
// that kv head are packed into 16-row MFMA tiles and stream the unit's K/V
// once.  The unit's visible key range (the whole causal prefix for verify;
// sinks followed by the window for draft, read as one virtual range) is cut
// into n_chunks chunks of chunk_len tokens.  A workgroup of kWaves waves
// (kWavesWide in the wide instances) takes one chunk of hp units of the same
// sequence (hp adjacent kv heads): waves / hp per unit, which interleave
// kTile-token tiles.  With
// n_chunks > 1 the chunks write normalised partial results and a merge pass
// combines them by log-sum-exp (the split-KV decomposition named in the
// paper's Sec. 2).
constexpr int kWaves = 4;
// Waves of the wide instances (up to two row tiles of bf16): two per SIMD.
constexpr int kWavesWide = 8;
constexpr int kTile = 32;            // tokens per wave iteration
constexpr int kMinChunkTokens = 1024;  // every wave gets >= 8 tiles of a chunk
constexpr int kMaxRows = 64;         // G*L bound: at most four 16-row tiles
constexpr int kPairMinChunkTokens = 4096;  // head pairs on split ranges: chunks at least this long
constexpr int kMaxChunks = 65535;    // a split plan's arrival count fits 16 bits
// Longest-first dispatch (single-chunk verify plans): every workgroup ranks
// the sequences by length, so it is kept to small batches of long caches.
constexpr int kLptMaxSeqs = 256;
constexpr int kLptMinLen = 4096;
// The balanced verify (same launches as longest-first) keeps its partial
// results within this much workspace, else longest-first is used: enough
// for one workgroup per compute unit on 256 of them at up to three row tiles
// of head pairs (25.4 MB at 48 rows), and within the static scratch of the
// entry point that allocates nothing.
constexpr size_t kBalMaxWorkspace = size_t{30} << 20;
// Row tiles up to which the balanced verify runs (its instances spill
// registers beyond): three for bf16, two for fp32.
constexpr int kBalMaxNT(bool bf16) { return bf16 ? 3 : 2; }

struct Plan {
  int32_t G = 0;         // Hq / Hkv
  int32_t R = 0;         // G * L query rows per unit
  int32_t NT = 0;        // 16-row tiles per unit
  int32_t U_max = 0;     // bound on any unit's visible range, in tokens
  int32_t n_chunks = 0;
  int32_t chunk_len = 0;
  int64_t n_rows = 0;    // B * L * Hq
  int64_t n_units = 0;   // B * Hkv
  int32_t hp = 1;        // units (adjacent kv heads) per workgroup
  int64_t n_groups = 0;  // n_units / hp; the grid is n_groups * n_chunks
  // Balanced verify: bal_nw workgroups take equal shares of every group's
  // tiles; the workspace holds a counter per group and 2 bal_nw partial
  // slots of hp * R rows.
  bool bal = false;
  int32_t bal_nw = 0;
  // Workspace of a split plan, in this order (each part 256-byte aligned):
  size_t counter_bytes = 0;  // [n_groups] uint64 arrival counters (tagged; never cleared)
  size_t part_o_bytes = 0;   // [n_chunks][n_rows][d] fp32 partial O
  size_t part_lse_bytes = 0; // [n_chunks][n_rows] fp32 partial lse
  size_t workspace_bytes = 0;
};

// Kernel index limits: workgroup, unit and row counts are 32-bit, and a
// full verify tile adds a 32-bit per-lane offset spanning up to 7 token rows,
// so the token stride is bounded.
constexpr int64_t kMaxTokStride = int64_t{1} << 28;  // elements
// Token positions, windows and list capacities stay below this, so that a
// position plus a tile, q_len or the window arithmetic of a unit never wraps.
constexpr int32_t kMaxPosition = INT32_MAX - 64;

// A tuning override from the environment: its value when set within
// [lo, hi], else 0.  Read on every call (well under a microsecond of host
// time), so a process can change it between calls -- the tests sweep every
// setting in one process; changing one while another thread is inside the
// library is not supported (setenv is not thread-safe).
int env_knob(const char* name, int lo, int hi);

// Shape checks shared by the attention calls and their workspace queries:
// MD_OK, MD_ERR_INVALID_ARG (malformed) or MD_ERR_UNSUPPORTED (beyond the
// compiled limits).  Only sizes are read.
int check_attn_sizes(const md_attn_args* a);

// Checks every argument the host can see.  Returns MD_OK or an md_status.
// mode MD_MODE_DRAFT_INDEXED reads `window` as the list capacity idx_stride.
int validate_attn(const md_attn_args* a, int mode, int n_sink, int window);

// The decomposition for these sizes on a device with num_cus compute units.
// Only sizes are read from `a`.  Call after validate_attn succeeded.
// mode MD_MODE_DRAFT_INDEXED reads `window` as the list capacity idx_stride.
Plan make_plan(const md_attn_args* a, int mode, int n_sink, int window, int num_cus);

// SnapKV selection: validation and the chunking of its two passes.
constexpr int kSnapkvMaxRows = 256;  // G * n_obs
struct SnapkvPlan {
  int32_t G = 0, R = 0, TW = 0;
  int32_t n_units = 0;
  int32_t n_chunks_stats = 0, chunk_len_stats = 0;
  int32_t n_chunks_votes = 0, chunk_len_votes = 0;
  size_t part_bytes = 0;   // part_m and part_l each: [units][n_chunks_stats][R] fp32
  size_t lse_bytes = 0;    // [units][R] fp32
  size_t workspace_bytes = 0;
};
int validate_snapkv(const md_snapkv_args* a);
SnapkvPlan make_snapkv_plan(const md_snapkv_args* a, int num_cus);

// Greedy acceptance: rows = B * L logits rows, each cut into n_chunks chunks
// of chunk_len elements (a multiple of 8; every chunk non-empty), one
// workgroup per chunk, enough of them to fill the device.
// The acceptance pass stages one sequence's partials and drafts in LDS.
constexpr int kAcceptMaxRowsPerSeq = 1024;      // n_draft + 1
constexpr int kAcceptMaxPartialsPerSeq = 4096;  // (n_draft + 1) * n_chunks
struct AcceptPlan {
  int32_t n_chunks = 0, chunk_len = 0;
  size_t part_bytes = 0;       // part_val and part_idx each: [rows][n_chunks] 4-byte
  size_t workspace_bytes = 0;
};
int validate_accept(int32_t num_seqs, int32_t n_draft, int32_t vocab, int32_t dtype);
AcceptPlan make_accept_plan(int32_t num_seqs, int32_t n_draft, int32_t vocab, int num_cus);

// The KV-cache write target of md_kv_append.
int validate_kv_cache(const md_kv_cache* c, int32_t n_new);

// Compute units of the current device (cached per device); 256 when no
// device is visible, so sizes stay defined on a host without a GPU.
int device_cu_count();

// The attention calls behind md_verify_attn, md_draft_attn and
// md_draft_attn_indexed (api.cpp).  A non-NULL `workspace` replaces the one
// in `a`; `stamps` (measurement, normally NULL) receives four wall-clock
// stamps per workgroup.
int run_attention(const md_attn_args* a, int mode, int n_sink, int window, void* stream,
                  const int32_t* idx, const int32_t* idx_len, void* workspace,
                  size_t workspace_bytes, unsigned long long* stamps);

// Workgroups the attention launch for these (validated) arguments uses.
int64_t attn_grid_size(const md_attn_args* a, int mode, int n_sink, int window);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace md
