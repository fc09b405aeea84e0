// Host-side checks of the library's argument validation and planning code
// (paper_2408_11049_amd/csrc/plan.cpp), built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_sanitizers.py.  plan.cpp makes no
// HIP call; the compute-unit count comes from the stub below.  The driver
// walks malformed and extreme arguments and a sweep of valid shapes through
// every validator and planner, and checks the plans' invariants; any
// out-of-bounds access, signed overflow or other undefined behaviour aborts.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "internal.h"

namespace md {
int device_cu_count() { return 256; }
}  // namespace md

namespace {

int g_fail = 0;
void check(bool ok, const char* what, long long a = 0, long long b = 0) {
  if (!ok) {
    fprintf(stderr, "FAILED: %s (%lld, %lld)\n", what, a, b);
    ++g_fail;
  }
}

// Aligned stand-ins for device pointers: validation only compares them.
unsigned char* const kFake = reinterpret_cast<unsigned char*>(uintptr_t{1} << 40);

md_attn_args good_args(int B, int L, int Hq, int Hkv, int d, int64_t S, int page) {
  md_attn_args a{};
  a.num_seqs = B;
  a.q_len = L;
  a.num_q_heads = Hq;
  a.num_kv_heads = Hkv;
  a.head_dim = d;
  a.dtype = MD_BF16;
  a.q = a.k = a.v = kFake;
  a.o = kFake + 4096;
  a.kv_lens = reinterpret_cast<const int32_t*>(kFake + 8192);
  a.kv_stride_head = d;
  a.kv_stride_tok = static_cast<int64_t>(Hkv) * d;
  a.max_kv_len = static_cast<int32_t>(S);
  if (page) {
    a.page_size = page;
    a.max_pages_per_seq = static_cast<int32_t>((S + page - 1) / page);
    a.num_pages = static_cast<int64_t>(B) * a.max_pages_per_seq;
    a.page_table = reinterpret_cast<const int32_t*>(kFake + 12288);
    a.kv_stride_blk = static_cast<int64_t>(page) * a.kv_stride_tok;
  } else {
    a.kv_stride_blk = S * a.kv_stride_tok;
  }
  a.workspace = kFake + (uintptr_t{1} << 20);
  a.workspace_bytes = SIZE_MAX / 2;
  return a;
}

int g_bal_plans = 0;

void plan_invariants(const md_attn_args& a, int mode, int n_sink, int window) {
  const md::Plan p = md::make_plan(&a, mode, n_sink, window, 256);
  g_bal_plans += p.bal ? 1 : 0;
  check(p.n_chunks >= 1, "n_chunks >= 1", p.n_chunks);
  check(p.chunk_len >= md::kTile && p.chunk_len % md::kTile == 0, "chunk_len tiles", p.chunk_len);
  check(static_cast<int64_t>(p.n_chunks) * p.chunk_len >= p.U_max, "chunks cover the range",
        p.n_chunks, p.U_max);
  check(p.NT >= 1 && p.NT <= 4, "row tiles", p.NT);
  check(p.hp == 1 || p.hp == 2, "heads per workgroup", p.hp);
  check(p.n_groups * p.hp == p.n_units, "groups x hp = units", p.n_groups, p.n_units);
  if (p.bal) {
    check(mode == MD_MODE_VERIFY && p.n_chunks == 1 && p.bal_nw > 0, "balanced verify plan");
    check(p.NT <= md::kBalMaxNT(a.dtype == MD_BF16), "balanced verify row tiles", p.NT);
    check(p.workspace_bytes <= md::kBalMaxWorkspace, "balanced workspace bound",
          static_cast<long long>(p.workspace_bytes));
  }
  if (p.n_chunks > 1 || p.bal)
    check(p.workspace_bytes >= p.counter_bytes + p.part_o_bytes + p.part_lse_bytes,
          "workspace parts", static_cast<long long>(p.workspace_bytes));
  else
    check(p.workspace_bytes == 0, "single pass needs no workspace");
}

}  // namespace

int main() {
  // ---- malformed attention arguments: every one refused, none crashes
  const int64_t big = INT32_MAX;
  struct Bad {
    int field;
    int64_t value;
  };
  const Bad bads[] = {{0, -1}, {1, 0}, {1, 17}, {2, 0}, {3, 0}, {3, 3}, {4, 0}, {4, 96},
                      {5, 7}, {6, 0}, {6, big}, {7, -16}, {8, 3}, {9, -1}, {9, 0},
                      {10, big}, {11, 1}, {12, 0}};
  for (const Bad& bd : bads) {
    md_attn_args a = good_args(4, 4, 8, 2, 128, 4096, 16);
    switch (bd.field) {
      case 0: a.num_seqs = static_cast<int32_t>(bd.value); break;
      case 1: a.q_len = static_cast<int32_t>(bd.value); break;
      case 2: a.num_q_heads = static_cast<int32_t>(bd.value); break;
      case 3: a.num_kv_heads = static_cast<int32_t>(bd.value); break;
      case 4: a.head_dim = static_cast<int32_t>(bd.value); break;
      case 5: a.dtype = static_cast<int32_t>(bd.value); break;
      case 6: a.max_kv_len = static_cast<int32_t>(bd.value); break;
      case 7: a.kv_stride_tok = bd.value; break;
      case 8: a.page_size = static_cast<int32_t>(bd.value); break;
      case 9: a.max_pages_per_seq = static_cast<int32_t>(bd.value); break;
      case 10: a.num_pages = bd.value * 4; break;
      case 11: a.q = kFake + 1; break;
      case 12: a.workspace_bytes = 0; a.num_seqs = 1; a.num_kv_heads = 1; a.num_q_heads = 4;
               a.max_kv_len = 1 << 20; a.max_pages_per_seq = 1 << 16; break;
    }
    // (A missing workspace only matters to the verify plan here: the draft
    // ranges are short enough for a single pass.)
    for (int mode = 0; mode < (bd.field == 12 ? 1 : 3); ++mode) {
      const int st = md::validate_attn(&a, mode, 4, 64);
      check(st != MD_OK, "malformed argument refused", bd.field, bd.value);
      (void)md::check_attn_sizes(&a);
    }
  }
  check(md::validate_attn(nullptr, 0, 0, 1) == MD_ERR_INVALID_ARG, "null args");

  // ---- extreme but valid sizes: plans stay within their invariants
  const int64_t lens[] = {1, 5, 31, 32, 33, 1023, 1024, 4096, 8192, 32768, 131072, 1 << 20,
                          static_cast<int64_t>(md::kMaxPosition)};
  const int batches[] = {1, 2, 3, 16, 64, 255, 256, 4096, 1 << 16};
  const int heads[][2] = {{4, 1}, {8, 2}, {32, 8}, {64, 8}, {16, 16}, {64, 1}};
  // The sweep runs with the default plan choice, then with the balanced
  // verify forced wherever allowed, and with its range count at the knob's
  // extremes (one range; 4096 ranges).
  const char* const bal_env[][2] = {{nullptr, nullptr}, {"MD_BALANCED", "2"},
                                    {"MD_BAL_NW", "1"}, {"MD_BAL_NW", "4096"}};
  int bal_per_pass[4] = {0, 0, 0, 0};
  for (int pass = 0; pass < 4; ++pass) {
  unsetenv("MD_BALANCED");
  unsetenv("MD_BAL_NW");
  if (bal_env[pass][0]) setenv(bal_env[pass][0], bal_env[pass][1], 1);
  if (pass >= 2) setenv("MD_BALANCED", "2", 1);
  const int bal_before = g_bal_plans;
  for (int64_t S : lens)
    for (int B : batches)
      for (const auto& hh : heads)
        for (int L : {1, 4, 16}) {
          if ((hh[0] / hh[1]) * L > md::kMaxRows || S < L) continue;
          for (int page : {0, 16}) {
            md_attn_args a = good_args(B, L, hh[0], hh[1], 128, S, page);
            if (page && static_cast<int64_t>(B) * a.max_pages_per_seq > INT32_MAX) continue;
            if (md::check_attn_sizes(&a) != MD_OK) continue;
            for (int mode = 0; mode < 3; ++mode) {
              const int window = mode == MD_MODE_VERIFY ? 1 : static_cast<int>(S < 2048 ? S : 2048);
              if (md::validate_attn(&a, mode, 64, window) != MD_OK) continue;
              plan_invariants(a, mode, 64, window);
            }
          }
        }
  bal_per_pass[pass] = g_bal_plans - bal_before;
  }
  unsetenv("MD_BALANCED");
  unsetenv("MD_BAL_NW");
  // Default choice: B = 64 x 8 kv heads at S >= 4096 is balanced; forced,
  // more shapes are.
  check(bal_per_pass[0] > 0, "default sweep reaches balanced plans", bal_per_pass[0]);
  check(bal_per_pass[1] > bal_per_pass[0], "forced sweep reaches more balanced plans",
        bal_per_pass[1], bal_per_pass[0]);
  check(bal_per_pass[2] > 0 && bal_per_pass[3] > 0, "range-count extremes plan",
        bal_per_pass[2], bal_per_pass[3]);
  printf("balanced plans per pass: %d %d %d %d\n", bal_per_pass[0], bal_per_pass[1],
         bal_per_pass[2], bal_per_pass[3]);

  // ---- SnapKV, acceptance and cache validators over edge sizes
  for (int32_t n : {0, 1, 32, 256, INT32_MAX}) {
    md_snapkv_args s{};
    s.num_seqs = 2;
    s.n_obs = n;
    s.num_q_heads = 32;
    s.num_kv_heads = 8;
    s.head_dim = 128;
    s.dtype = MD_BF16;
    s.q_obs = s.k = kFake;
    s.kv_stride_head = 128;
    s.kv_stride_tok = 1024;
    s.kv_stride_blk = 1024 * 40000;
    s.prompt_lens = reinterpret_cast<const int32_t*>(kFake);
    s.max_prompt_len = 40000;
    s.votes = reinterpret_cast<float*>(kFake);
    s.votes_stride = 40000;
    s.workspace = kFake;
    s.workspace_bytes = SIZE_MAX / 2;
    const int st = md::validate_snapkv(&s);
    if (st == MD_OK) {
      const md::SnapkvPlan sp = md::make_snapkv_plan(&s, 256);
      check(sp.n_chunks_stats >= 1 && sp.n_chunks_votes >= 1, "snapkv chunks");
    }
  }
  for (int32_t B : {0, 1, 64, 1 << 20})
    for (int32_t nd : {-1, 0, 4, 1023, 1024})
      for (int32_t vocab : {0, 1, 8, 128256, 1 << 30, (1 << 30) + 1, INT32_MAX}) {
        if (md::validate_accept(B, nd, vocab, MD_F32) != MD_OK) continue;
        const md::AcceptPlan ap = md::make_accept_plan(B, nd, vocab, 256);
        check(B == 0 || (ap.n_chunks >= 1 && static_cast<int64_t>(ap.n_chunks) * ap.chunk_len >= vocab),
              "accept chunks cover the vocabulary", ap.n_chunks, vocab);
      }
  md_kv_cache c{};
  c.num_seqs = 2;
  c.num_kv_heads = 8;
  c.head_dim = 128;
  c.dtype = MD_BF16;
  c.kv_stride_head = 128;
  c.kv_stride_tok = 1024;
  c.kv_stride_blk = 1024 * 64;
  c.capacity = 64;
  check(md::validate_kv_cache(&c, 5) == MD_OK, "good cache");
  check(md::validate_kv_cache(&c, -1) != MD_OK, "negative n_new");
  check(md::validate_kv_cache(nullptr, 0) != MD_OK, "null cache");
  c.kv_stride_tok = 1001;
  check(md::validate_kv_cache(&c, 1) != MD_OK, "misaligned stride");

  if (g_fail) return 1;
  printf("plan driver: ok\n");
  return 0;
}
