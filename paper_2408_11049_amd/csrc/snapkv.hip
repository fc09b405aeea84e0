// snapkv.hip -- SnapKV-style selection of the static draft cache at prefill.
//
// The paper's best drafter keeps a static compressed KV cache chosen by
// SnapKV (static KV selection, Sec. 4.4; best budget 2049, Sec. 5.2), with an
// observation window of 32 queries and average pooling of kernel 5 (the
// footnote of Sec. 4.4).  Per (sequence, kv head):
//   vote(j)   = sum over the observation queries o and the kv head's G query
//               heads h of softmax_j'(scale q_{o,h} . k_j') at j, the softmax
//               running over the keys each query sees (j' <= its position);
//   pooled(j) = mean of vote over j-2 .. j+2 (zero outside the prefix);
//   keep the budget - 32 prefix positions of largest pooled vote plus the
//   32 observation positions, ascending.
//
// Kernels:
//   snapkv_pass_kernel<PASS=0>  per (unit, key chunk): each observation row's
//       running max and sum of exp over the chunk (softmax statistics);
//   snapkv_lse_kernel           merges the chunks into one log2-sum-exp per row;
//   snapkv_pass_kernel<PASS=1>  per (unit, prefix chunk): p = 2^(s - lse) and
//       the per-key sum over all rows: the raw votes;
//   snapkv_select_kernel        per unit: pooled votes, radix select of the
//       top keep, ordered compaction, plus the window.
// In the pass kernels all G*n_obs rows of a unit share each 64-key tile,
// loaded once into LDS as whole 256 B rows; each wave owns one or two 16-row
// MFMA tiles of the rows and computes S = Q K^T on v_mfma_f32_16x16x32_bf16,
// so each lane holds four rows of one key: a key's vote sums inside the lane
// and across the wave's four lane groups, and the softmax statistics of a
// row stay in its lanes until the chunk ends.  A tile costs one barrier: the
// staging buffers and the per-wave vote sums alternate between two slots.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "kernels.h"

namespace md {

namespace {

typedef __bf16 sk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float sk_f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t sk_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSkWaves = 4;      // up to 64 rows, and the votes pass at any row count
constexpr int kSkWavesWide = 8;  // statistics pass, 65-256 rows: eight waves of one or two row tiles
constexpr int kSkTile = 64;  // keys per tile: measured 5% faster than 32 keys, 128 slower

template <int D, bool BF16, int KT = kSkTile, int WV = kSkWaves>
struct SkShape {
  static constexpr int ES = BF16 ? 2 : 4;
  static constexpr int KCB = D * ES / 64;     // 16 B A-operand chunks per lane per 16-key block
  static constexpr int LPT = D * ES / 16;     // lanes per key row
  static constexpr int ROWS_PER_WG_LOAD = WV * 64 / LPT;  // key rows one pass of all waves loads
  static constexpr int NLD = KT / ROWS_PER_WG_LOAD;             // loads per lane per tile
  static constexpr int NB = KT / 16;                             // 16-key MFMA blocks per tile
  static constexpr int KROW = D * ES + 16;    // padded LDS row (odd multiple of 16 B)
};

}  // namespace

// TW: 16-row tiles per wave, WV: waves (rows per workgroup = 16 * TW * WV); KT:
// keys per tile.  The statistics pass runs 65-256 rows as eight waves of one
// or two row tiles (more waves to cover the MFMA, exponential and load
// latencies; the bf16 single-tile instance is held to 80 registers, six
// waves per SIMD).  The votes pass keeps four waves (the whole call 10%
// faster than with eight: half the LDS reads of each tile and of the
// per-wave vote sums).
template <int D, bool BF16, int TW, bool PAGED, bool WA, int PASS, int KT, int WV>
__global__ void __launch_bounds__(WV * 64)
    __attribute__((amdgpu_waves_per_eu(BF16 && WV == 8 && TW == 1 ? 6 : 1)))
snapkv_pass_kernel(const SnapkvParams p) {
  using SH = SkShape<D, BF16, KT, WV>;
  constexpr int NB = SH::NB;
  __shared__ __attribute__((aligned(16))) unsigned char kt[2][KT * SH::KROW];
  __shared__ float red[2][WV][KT];  // PASS 1: per-wave key sums of two tiles

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l16 = lane & 15;
  const int grp = lane >> 4;
  // Chunk-major numbering, as in the attention kernel: workgroups that start
  // together read the same key range of neighbouring kv heads (measured:
  // equal to 1.8% faster than unit-major).
  const int n_unit_grid = static_cast<int>(gridDim.x) / p.n_chunks;
  const int chunk = static_cast<int>(blockIdx.x) / n_unit_grid;
  const int unit = static_cast<int>(blockIdx.x) % n_unit_grid;
  const int hk = unit % p.Hkv;
  const int b = unit / p.Hkv;
  const int S = min(max(p.kv_lens[b], 0), p.max_kv_len);
  const int n_pre = max(S - p.n_obs, 0);
  // PASS 0 covers every key a query sees; PASS 1 only the prefix that is voted on.
  const int U = PASS == 0 ? S : n_pre;
  const int v_begin = chunk * p.chunk_len;
  const int v_end = min(U, v_begin + p.chunk_len);
  const int n_tiles = v_end > v_begin ? (v_end - v_begin + KT - 1) / KT : 0;

  // Rows of this wave's tile t: r = (wave * TW + t) * 16 + i, r = o * G + g.
  // Q is the MFMA A operand (lane l16 loads row i = l16), so the C tile of
  // S = Q K^T gives each lane rows 4 * grp + e (e = item) of key l16.
  sk_u32x4 qreg[TW][SH::KCB];
  int row_pos[TW][4];  // query position of the lane's rows (-1: padding)
  float lse2[TW][4];   // PASS 1: their log2-sum-exp (+inf for padding: p = 0)
  for (int t = 0; t < TW; ++t) {
    const int rq = (wave * TW + t) * 16 + l16;
    for (int cb = 0; cb < SH::KCB; ++cb) qreg[t][cb] = sk_u32x4{0, 0, 0, 0};
    if (rq < p.R) {
      const int o = rq / p.G, g = rq % p.G;
      const unsigned char* qp = static_cast<const unsigned char*>(p.q) +
                                ((static_cast<int64_t>(b) * p.n_obs + o) * p.Hq + hk * p.G + g) *
                                    D * SH::ES;
      for (int cb = 0; cb < SH::KCB; ++cb)
        qreg[t][cb] = *reinterpret_cast<const sk_u32x4*>(qp + cb * 64 + grp * 16);
    }
    for (int e = 0; e < 4; ++e) {
      const int r = (wave * TW + t) * 16 + 4 * grp + e;
      row_pos[t][e] = r < p.R ? S - p.n_obs + r / p.G : -1;
      lse2[t][e] = INFINITY;
      if (PASS == 1 && r < p.R) lse2[t][e] = p.lse2[static_cast<int64_t>(unit) * p.R + r];
    }
  }

  const unsigned char* kbase = static_cast<const unsigned char*>(p.k);
  const int64_t head_off = static_cast<int64_t>(hk) * p.s_head;
  const int32_t* ptab = PAGED ? p.page_table + static_cast<int64_t>(b) * p.max_pages : nullptr;
  const int pmask = (1 << p.page_shift) - 1;

  // Cooperative tile load: thread -> key row (threadIdx / LPT) + n * ROWS_PER_WG_LOAD,
  // 16 B chunk threadIdx % LPT; a wave's lanes cover RPW consecutive rows of
  // each load.  Page ids are read one tile ahead of the K loads that use
  // them, so a tile's loads never wait on a page-table read.
  //  WA (pages of at least RPW rows, or contiguous rows): a wave's RPW rows
  //    lie in one page, so their base address is wave-uniform scalar
  //    arithmetic and each lane adds a fixed 32-bit offset.  Rows past the
  //    range read the range's last key (contiguous) or stay inside the page
  //    of the group's first row; a group wholly past it reads element 0.
  //  !WA: each lane computes its own row address; keys past the range read
  //    element 0.  Keys past the range are masked either way.
  constexpr int RPW = 64 / SH::LPT;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lane_chunk = static_cast<uint32_t>(lane % SH::LPT) * 16;
  const uint32_t lane_row = static_cast<uint32_t>(lane / SH::LPT);
  const uint32_t row_bytes = WA ? static_cast<uint32_t>(p.s_tok * SH::ES) : 0;
  const uint32_t lane_off = lane_row * row_bytes + lane_chunk;

  // Page ids of a tile's loads: per lane (pid[n], !WA), or, with WA, one
  // vector read in which lane n < NLD fetches load n's id (pid[0]), taken
  // out with readlane where the load is issued.
  auto load_pids = [&](int (&pid)[SH::NLD], int tile) {
    if constexpr (PAGED) {
      if constexpr (WA) {
        const int n = lane % SH::NLD;
        const int jw = v_begin + tile * KT + n * SH::ROWS_PER_WG_LOAD + wave_u * RPW;
        const bool ok = tile < n_tiles && jw < v_end;
        const int pg = ptab[ok ? (jw >> p.page_shift) : 0];
        pid[0] = ok ? pg : -1;
      } else {
        for (int n = 0; n < SH::NLD; ++n) {
          const int tt = n * SH::ROWS_PER_WG_LOAD + threadIdx.x / SH::LPT;
          const int j = v_begin + tile * KT + tt;
          const bool ok = tile < n_tiles && j < v_end;
          pid[n] = ptab[ok ? (j >> p.page_shift) : 0];
        }
      }
    }
  };
  auto load_tile = [&](sk_u32x4 (&x)[SH::NLD], int tile, const int (&pid)[SH::NLD]) {
    if (tile >= n_tiles) return;  // past the chunk: nothing to stage
    for (int n = 0; n < SH::NLD; ++n) {
      int64_t off = 0;
      uint32_t voff = lane_chunk;
      if constexpr (WA) {
        const int jw = v_begin + tile * KT + n * SH::ROWS_PER_WG_LOAD + wave_u * RPW;
        voff = lane_off;
        if constexpr (PAGED) {
          const int pg = __builtin_amdgcn_readlane(pid[0], n);
          const bool ok = pg >= 0 && pg < p.num_pages;
          off = ok ? static_cast<int64_t>(pg) * p.s_blk +
                         static_cast<int64_t>(jw & pmask) * p.s_tok + head_off
                   : 0;
          if (!ok) voff = lane_chunk;
        } else {
          const int jc = min(jw, v_end - 1);
          off = static_cast<int64_t>(b) * p.s_blk + static_cast<int64_t>(jc) * p.s_tok + head_off;
          if (jw + RPW > v_end)  // a group that reaches past the range
            voff = min(lane_row, static_cast<uint32_t>(v_end - 1 - jc)) * row_bytes + lane_chunk;
        }
      } else {
        const int tt = n * SH::ROWS_PER_WG_LOAD + threadIdx.x / SH::LPT;
        const int j = v_begin + tile * KT + tt;
        bool ok = j < v_end;
        if (PAGED) {
          ok = ok && pid[n] >= 0 && pid[n] < p.num_pages;
          off = ok ? static_cast<int64_t>(pid[n]) * p.s_blk +
                         static_cast<int64_t>(j & pmask) * p.s_tok + head_off
                   : 0;
        } else {
          off = ok ? static_cast<int64_t>(b) * p.s_blk + static_cast<int64_t>(j) * p.s_tok + head_off
                   : 0;
        }
      }
      x[n] = __builtin_nontemporal_load(
          reinterpret_cast<const sk_u32x4*>(kbase + off * SH::ES + voff));
    }
  };
  auto store_tile = [&](const sk_u32x4 (&x)[SH::NLD], int buf) {
    for (int n = 0; n < SH::NLD; ++n) {
      const int tt = n * SH::ROWS_PER_WG_LOAD + threadIdx.x / SH::LPT;
      *reinterpret_cast<sk_u32x4*>(kt[buf] + tt * SH::KROW + (threadIdx.x % SH::LPT) * 16) = x[n];
    }
  };

  // Row statistics: the running max in the exponent's units (score x scale
  // x log2e, the scale folded into the exponent's fused multiply-add) and
  // the running sum.
  const float c2 = p.scale_log2;
  float mc_run[TW][4], l_run[TW][4];  // running max x scale x log2e, and sum
  for (int t = 0; t < TW; ++t)
    for (int e = 0; e < 4; ++e) {
      mc_run[t][e] = -INFINITY;
      l_run[t][e] = 0.f;
    }

  sk_u32x4 xr[SH::NLD];
  int pids[SH::NLD] = {};
  load_pids(pids, 0);
  load_tile(xr, 0, pids);
  load_pids(pids, 1);
  const int n_full = n_tiles > 0 ? (v_end - v_begin) / KT : 0;  // tiles with every key in range
  // Tiles before n_plain hold only in-range keys that every observation
  // query sees (j < S - n_obs <= its position): no mask.  PASS 1 covers only
  // such keys, up to its partial last tile.
  const int n_plain = PASS == 0 ? min(n_full, max(n_pre - v_begin, 0) / KT) : n_tiles;
  auto reduce_votes = [&](int tile) {  // PASS 1: sum the waves' sums of tile `tile`
    if (threadIdx.x < KT) {
      const int j = v_begin + tile * KT + threadIdx.x;
      if (j < v_end) {
        float sum = 0.f;
        for (int w = 0; w < WV; ++w) sum += red[tile & 1][w][threadIdx.x];
        p.votes[(static_cast<int64_t>(b) * p.Hkv + hk) * p.votes_stride + j] = sum;
      }
    }
  };
  auto body = [&](int tile, auto masked) {
    const int buf = tile & 1;
    store_tile(xr, buf);
    __syncthreads();
    if (PASS == 1 && tile > 0) reduce_votes(tile - 1);
    load_tile(xr, tile + 1, pids);  // next tile in flight while this one is used
    load_pids(pids, tile + 2);
    const int v0 = v_begin + tile * KT;

    // S = Q K^T for this wave's row tiles and the tile's NB 16-key blocks.
    sk_f32x4 sacc[TW][NB];
    for (int tb = 0; tb < NB; ++tb) {
      for (int t = 0; t < TW; ++t) sacc[t][tb] = sk_f32x4{0.f, 0.f, 0.f, 0.f};
      const unsigned char* krow = kt[buf] + (tb * 16 + l16) * SH::KROW + grp * 16;
      for (int cb = 0; cb < SH::KCB; ++cb) {
        const sk_u32x4 kk = *reinterpret_cast<const sk_u32x4*>(krow + cb * 64);
        for (int t = 0; t < TW; ++t) {
          if constexpr (BF16) {
            sacc[t][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(sk_bf16x8, qreg[t][cb]), __builtin_bit_cast(sk_bf16x8, kk),
                sacc[t][tb], 0, 0, 0);
          } else {
            for (int jj = 0; jj < 4; ++jj)
              sacc[t][tb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __uint_as_float(qreg[t][cb][jj]), __uint_as_float(kk[jj]), sacc[t][tb], 0, 0, 0);
          }
        }
      }
    }

    if constexpr (PASS == 0) {
      // Online max and sum of 2^(s * scale * log2e - mc) per row, over this
      // lane's NB keys (one per block), with mc the running max in the
      // exponent's units; the sum is rescaled on every tile (a select on a
      // moved max costs more than the multiply-add it saves).
      for (int t = 0; t < TW; ++t)
        for (int e = 0; e < 4; ++e) {
          float x[NB];
          float mx = -INFINITY;
          for (int tb = 0; tb < NB; ++tb) {
            x[tb] = sacc[t][tb][e];
            if constexpr (decltype(masked)::value) {
              const int j = v0 + tb * 16 + l16;
              if (!(j < v_end && j <= row_pos[t][e])) x[tb] = -INFINITY;
            }
            mx = fmaxf(mx, x[tb]);
          }
          const float mcn = fmaxf(mc_run[t][e], mx * c2);
          // Unmasked tiles come first and give every row a finite max on
          // the first of them; only masked tiles can meet a row with none
          // (then the sums use 0 as reference and the max stays -inf).
          float mcu = mcn;
          if constexpr (decltype(masked)::value) mcu = mcn == -INFINITY ? 0.f : mcn;
          float s = 0.f;
          for (int tb = 0; tb < NB; ++tb) s += __builtin_amdgcn_exp2f(fmaf(x[tb], c2, -mcu));
          l_run[t][e] = fmaf(l_run[t][e], __builtin_amdgcn_exp2f(mc_run[t][e] - mcu), s);
          mc_run[t][e] = mcn;
        }
    } else {
      // p = 2^(s*scale*log2e - lse2) summed over every row, per key: inside
      // the lane over its rows, then over the four row groups of the wave.
      float col[NB];
      for (int tb = 0; tb < NB; ++tb) col[tb] = 0.f;
      for (int t = 0; t < TW; ++t)
        for (int tb = 0; tb < NB; ++tb)
          for (int e = 0; e < 4; ++e)
            col[tb] += __builtin_amdgcn_exp2f(sacc[t][tb][e] * p.scale_log2 - lse2[t][e]);
      for (int tb = 0; tb < NB; ++tb) {
        col[tb] += __shfl_xor(col[tb], 16);
        col[tb] += __shfl_xor(col[tb], 32);
      }
      // Each wave's sums go to this tile's slots; the four waves' sums are
      // added after the next tile's barrier (reduce_votes), so a tile needs
      // one barrier.
      if (grp == 0)
        for (int tb = 0; tb < NB; ++tb) red[buf][wave][tb * 16 + l16] = col[tb];
    }
    // No barrier here: the next tile stages into the other buffer, and this
    // buffer and these sums are rewritten only after the next tile's barrier,
    // which every wave reaches after finishing this tile.
  };
  int tile = 0;
  for (; tile < n_plain; ++tile) body(tile, std::false_type{});
  for (; tile < n_tiles; ++tile) body(tile, std::true_type{});
  if (PASS == 1 && n_tiles > 0) {
    __syncthreads();
    reduce_votes(n_tiles - 1);
  }

  if constexpr (PASS == 0) {
    // Combine each row over the 16 lanes holding its keys, then write (m, l)
    // for this chunk.
    for (int t = 0; t < TW; ++t)
      for (int e = 0; e < 4; ++e) {
        float m = mc_run[t][e], l = l_run[t][e];
        for (int off = 1; off < 16; off <<= 1) {
          const float mo = __shfl_xor(m, off), lo = __shfl_xor(l, off);
          const float mn = fmaxf(m, mo);
          const float m_use = mn == -INFINITY ? 0.f : mn;
          l = l * __builtin_amdgcn_exp2f(m - m_use) + lo * __builtin_amdgcn_exp2f(mo - m_use);
          m = mn;
        }
        const int r = (wave * TW + t) * 16 + 4 * grp + e;
        if (l16 == 0 && r < p.R) {
          const int64_t at = (static_cast<int64_t>(unit) * p.n_chunks + chunk) * p.R + r;
          p.part_m[at] = m;
          p.part_l[at] = l;
        }
      }
  }
}

// lse2[unit][r] = log2 sum over chunks of l_c * 2^(m_c).
__global__ void __launch_bounds__(256) snapkv_lse_kernel(const SnapkvParams p) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(p.n_units) * p.R) return;
  const int64_t unit = i / p.R, r = i % p.R;
  float M = -INFINITY;
  for (int c = 0; c < p.n_chunks; ++c) M = fmaxf(M, p.part_m[(unit * p.n_chunks + c) * p.R + r]);
  float L = 0.f;
  if (M != -INFINITY)
    for (int c = 0; c < p.n_chunks; ++c) {
      const float m = p.part_m[(unit * p.n_chunks + c) * p.R + r];
      if (m != -INFINITY) L += p.part_l[(unit * p.n_chunks + c) * p.R + r] * __builtin_amdgcn_exp2f(m - M);
    }
  p.lse2[i] = L > 0.f ? M + __builtin_amdgcn_logf(L) : INFINITY;
}

// ---------------------------------------------------------------------------
// Selection.  One workgroup per (sequence, kv head) row.

namespace {

// Order-preserving map of a float onto uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t sk_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float sk_pooled(const float* v, int n, int j, int pool) {
  float s = 0.f;
  for (int t = j - pool / 2; t <= j + pool / 2; ++t)
    if (t >= 0 && t < n) s += v[t];
  return s / static_cast<float>(pool);
}

}  // namespace

constexpr int kSelThreads = 512;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelPer = 4;             // global instance: consecutive positions per thread in a step
constexpr int kSelStep = kSelThreads * kSelPer;
constexpr int kSelRegThreads = 1024;   // register instance: threads per workgroup
constexpr int kSelRegWaves = kSelRegThreads / 64;
constexpr int kSelKpt = 33;            // and pooled keys per thread
constexpr int kSelPadW = 2;            // LDS pad words per segment: odd stride 35
constexpr int kSelRegKeys = kSelRegThreads * kSelKpt;  // its longest row: 33792 prefix positions
constexpr int kSelRegHalo = 3;         // and its widest pooling: pool <= 7

// Count every active lane's bin in the wave's histogram h.  Pooled votes of
// similar size share their top key bits, so the early radix passes pile
// onto a few bins: the bin of the lowest uncounted lane goes in with one
// atomic for all lanes that share it, twice (with skewed keys, most likely
// the wave's most common bins), and the remaining lanes add directly.
__device__ __forceinline__ void sk_hist_add(uint32_t* h, bool active, uint32_t bin, int lane) {
  bool mine = active;  // this lane's key is not counted yet
  for (int round = 0; round < 2; ++round) {
    const uint64_t pending = __ballot(mine);
    if (pending == 0) return;  // wave-uniform
    const int leader = __ffsll(static_cast<long long>(pending)) - 1;
    const uint32_t lb = __builtin_amdgcn_readlane(bin, leader);  // leader is wave-uniform
    const bool same = mine && bin == lb;
    const uint64_t n_same = __ballot(same);
    if (lane == leader) atomicAdd(&h[lb], static_cast<uint32_t>(__popcll(n_same)));
    mine = mine && !same;
  }
  if (mine) atomicAdd(&h[bin], 1u);
}

// Exclusive prefix sum of x over a workgroup of WAVES waves (thread order),
// and the total.  Uses wsum[WAVES]; contains two barriers.
template <int WAVES = kSelWaves>
__device__ __forceinline__ uint32_t sk_block_scan(uint32_t x, uint32_t* wsum, uint32_t& total,
                                                  int lane, int w) {
  uint32_t incl = x;
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(incl, off);
    if (lane >= off) incl += o;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  uint32_t before = 0;
  total = 0;
  for (int x2 = 0; x2 < WAVES; ++x2) {
    if (x2 < w) before += wsum[x2];
    total += wsum[x2];
  }
  __syncthreads();
  return before + incl - x;
}

// The keep-th largest key of a row and how many keys exceed it, by radix
// select over 11-, 11- and 10-bit digits, most significant first:
// `key_at(e)` is this thread's e-th key (0 <= e < PER), valid(e) whether it
// is a position of the row; THREADS threads per workgroup.  hist is one
// histogram of kSelBins counters per wave (LDS).  Every thread returns the
// same (tau, above).
constexpr int kSelBins = 2048;
template <int PER, int THREADS, typename KeyAt, typename Valid>
__device__ __forceinline__ void sk_radix_select(KeyAt key_at, Valid valid, int keep,
                                                uint32_t* hist, uint32_t* wsum,
                                                uint32_t* s_prefix, uint32_t* s_above,
                                                uint32_t& tau, uint32_t& above_out) {
  constexpr int kDigitsPerThread = kSelBins / THREADS;
  constexpr int WAVES = THREADS / 64;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  uint32_t prefix = 0, above = 0;
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const uint32_t dmask = pass == 2 ? 0x3ffu : 0x7ffu;
    const uint32_t hi_mask = pass == 0 ? 0u : (pass == 1 ? 0xffe00000u : 0xfffffc00u);
    for (int i = tid; i < WAVES * kSelBins; i += THREADS) hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const uint32_t k = key_at(e);
      const bool act = valid(e) && (k & hi_mask) == (prefix & hi_mask);
      sk_hist_add(hist + w * kSelBins, act, (k >> shift) & dmask, lane);
    }
    __syncthreads();
    // Thread t owns digits kSelBins-1-4t .. kSelBins-4-4t (descending); a scan
    // over the threads finds the digit where the running count reaches keep.
    uint32_t c[kDigitsPerThread];
    uint32_t cnt = 0;
#pragma unroll
    for (int i = 0; i < kDigitsPerThread; ++i) {
      const int d = kSelBins - 1 - (kDigitsPerThread * tid + i);
      c[i] = 0;
      for (int x = 0; x < WAVES; ++x) c[i] += hist[x * kSelBins + d];
      cnt += c[i];
    }
    uint32_t total;
    uint32_t run = above + sk_block_scan<WAVES>(cnt, wsum, total, lane, w);
#pragma unroll
    for (int i = 0; i < kDigitsPerThread; ++i) {
      const uint32_t d = static_cast<uint32_t>(kSelBins - 1 - (kDigitsPerThread * tid + i));
      if (run < static_cast<uint32_t>(keep) && run + c[i] >= static_cast<uint32_t>(keep)) {
        *s_prefix = prefix | (d << shift);
        *s_above = run;
      }
      run += c[i];
    }
    __syncthreads();
    prefix = *s_prefix;
    above = *s_above;
    __syncthreads();
  }
  tau = prefix;
  above_out = above;
}

// Register instance, rows of at most kSelRegKeys prefix positions: 1024
// threads, four waves per SIMD (measured 22% faster than 512 threads with
// twice the keys each).  Thread t owns the contiguous segment [33t, 33t + 33)
// of the row.  The raw votes are copied into LDS with 16-byte global loads,
// position j at word j + 2 (j / 33) (two pad words per segment: an odd stride
// of 35, so the 64 lanes reading the same offset of their segments hit
// distinct banks); each thread pools its segment from its own window of LDS
// in sk_pooled's order and keeps the 33 keys in registers for the radix
// passes and the compaction.  The positions a thread keeps are contiguous in
// its segment, so two block scans give every thread its output offset and
// the row comes out ascending.
__device__ __forceinline__ int sk_pad(int j) { return j + kSelPadW * (j / kSelKpt); }

template <int POOL>
__global__ void __launch_bounds__(kSelRegThreads) snapkv_select_reg_kernel(const SnapkvSelectParams p) {
  // The raw votes, then (the keys in registers) the radix histograms.
  constexpr int kBuf = kSelRegKeys + kSelPadW * kSelRegThreads;
  __shared__ float buf[kBuf];
  static_assert(kSelRegWaves * kSelBins <= kBuf, "histograms fit the buffer");
  __shared__ uint32_t wsum[kSelRegWaves];
  __shared__ uint32_t s_prefix, s_above;

  const int row = blockIdx.x;
  const int b = row / p.rows_per_seq;
  const int S = min(max(p.lens[b], 0), p.stride + p.n_obs);
  const int n = max(S - p.n_obs, 0);  // <= stride <= kSelRegKeys
  const int keep = min(p.budget - p.n_obs, n);
  const float* v = p.votes + static_cast<int64_t>(row) * p.stride;
  int32_t* out = p.idx + static_cast<int64_t>(row) * p.budget;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = tid & 63;
  const int j0 = tid * kSelKpt;  // this thread's segment

  uint32_t key[kSelKpt];
  if (keep > 0) {
    const bool vec = (reinterpret_cast<uintptr_t>(v) & 15u) == 0;
    const int n4 = vec ? n / 4 : 0;
#pragma unroll 4
    for (int i = tid; i < n4; i += kSelRegThreads) {
      const float4 x = reinterpret_cast<const float4*>(v)[i];
      buf[sk_pad(4 * i)] = x.x;
      buf[sk_pad(4 * i + 1)] = x.y;
      buf[sk_pad(4 * i + 2)] = x.z;
      buf[sk_pad(4 * i + 3)] = x.w;
    }
    for (int j = 4 * n4 + tid; j < n; j += kSelRegThreads) buf[sk_pad(j)] = v[j];
    __syncthreads();
    // Raw vote at segment offset o (-POOL/2 <= o < 33 + POOL/2) of this
    // thread's window, +0 outside the prefix; the word index stays inside the
    // buffer.
    const int base = j0 + kSelPadW * tid;  // sk_pad(j0)
    auto raw = [&](int o) -> float {
      const int jj = j0 + o;
      const int seg = o < 0 ? -kSelPadW : (o >= kSelKpt ? kSelPadW : 0);
      const float x = buf[min(max(base + o + seg, 0), kBuf - 1)];  // always inside the buffer
      return (jj >= 0 && jj < n) ? x : 0.f;
    };
    // Taps -POOL/2 .. POOL/2 in order; a tap outside the prefix adds an exact
    // +0 (the running sum starts at +0, so it is never -0), which leaves every
    // sum as sk_pooled forms it.
    constexpr int h = POOL / 2;
#pragma unroll
    for (int e = 0; e < kSelKpt; ++e) {
      float acc = 0.f;
#pragma unroll
      for (int t = -h; t <= h; ++t) acc += raw(e + t);
      key[e] = j0 + e < n ? sk_key(acc / static_cast<float>(POOL)) : 0u;
    }
  } else {
#pragma unroll
    for (int e = 0; e < kSelKpt; ++e) key[e] = 0u;
  }
  __syncthreads();  // every raw read is done: the buffer holds the histograms now

  // Positions past the row hold key 0, the smallest key: with keep <= n they
  // leave the keep-th largest key and the count above it as they are, so the
  // radix passes count every register without a mask (only the ties of the
  // compaction below look at the position).
  uint32_t tau = 0, above = 0;
  if (keep > 0)
    sk_radix_select<kSelKpt, kSelRegThreads>(
        [&](int e) { return key[e]; }, [](int) { return true; }, keep,
        reinterpret_cast<uint32_t*>(buf), wsum, &s_prefix, &s_above, tau, above);
  const uint32_t need_eq = keep > 0 ? static_cast<uint32_t>(keep) - above : 0;

  if (keep > 0) {
    // Keep key > tau, and key == tau while fewer than need_eq of those lie
    // before it; ties go to the smaller position.
    uint32_t n_gt = 0, n_eq = 0;
#pragma unroll
    for (int e = 0; e < kSelKpt; ++e) {
      n_gt += key[e] > tau;  // never a position past the row (key 0)
      n_eq += j0 + e < n && key[e] == tau;
    }
    uint32_t eq_total;
    const uint32_t eq_before = sk_block_scan<kSelRegWaves>(n_eq, wsum, eq_total, lane, w);
    const uint32_t eq_take =
        eq_before >= need_eq ? 0u : (need_eq - eq_before < n_eq ? need_eq - eq_before : n_eq);
    uint32_t take_total;
    uint32_t pos = sk_block_scan<kSelRegWaves>(n_gt + eq_take, wsum, take_total, lane, w);
    uint32_t eq_left = eq_take;
#pragma unroll
    for (int e = 0; e < kSelKpt; ++e) {
      const bool eq = j0 + e < n && key[e] == tau;
      const bool take = key[e] > tau || (eq && eq_left > 0);
      eq_left -= (eq && eq_left > 0) ? 1u : 0u;
      if (take) out[pos++] = j0 + e;
    }
  }
  // The observation window, always kept.
  const int kept = keep > 0 ? keep : 0;
  for (int j = n + tid; j < S; j += kSelRegThreads) out[kept + (j - n)] = j;
  if (tid == 0 && (row % p.rows_per_seq) == 0) p.counts[b] = kept + (S - n);
}

// Global instance, rows longer than kSelRegKeys: every sweep pools from
// global memory (each pooled key is formed in sk_pooled's order, so both
// instances see the same keys), kSelPer * kSelThreads positions per step.
__global__ void __launch_bounds__(kSelThreads) snapkv_select_kernel(const SnapkvSelectParams p) {
  __shared__ uint32_t hist[kSelWaves][256];
  __shared__ uint32_t wsum[kSelWaves];
  __shared__ uint32_t s_prefix, s_above;

  const int row = blockIdx.x;
  const int b = row / p.rows_per_seq;
  const int S = min(max(p.lens[b], 0), p.stride + p.n_obs);
  const int n = max(S - p.n_obs, 0);
  const int keep = min(p.budget - p.n_obs, n);
  const float* v = p.votes + static_cast<int64_t>(row) * p.stride;
  int32_t* out = p.idx + static_cast<int64_t>(row) * p.budget;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = tid & 63;

  auto key_at = [&](int j) -> uint32_t { return sk_key(sk_pooled(v, n, j, p.pool)); };

  // Radix select, most significant byte first: after four passes tau is the
  // key of the keep-th largest pooled vote and `above` keys exceed it.
  uint32_t prefix = 0, above = 0;
  if (keep > 0) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      const uint32_t hi_mask = pass == 0 ? 0u : (0xffffffffu << (32 - 8 * pass));
      for (int i = tid; i < kSelWaves * 256; i += kSelThreads) (&hist[0][0])[i] = 0;
      __syncthreads();
      for (int base = 0; base < n; base += kSelPer * kSelThreads) {
        uint32_t k[kSelPer];  // the keys first, so their reads overlap
#pragma unroll
        for (int e = 0; e < kSelPer; ++e) {
          const int j = base + e * kSelThreads + tid;
          k[e] = j < n ? key_at(j) : 0u;
        }
#pragma unroll
        for (int e = 0; e < kSelPer; ++e) {
          const bool act = base + e * kSelThreads + tid < n && (k[e] & hi_mask) == (prefix & hi_mask);
          sk_hist_add(hist[w], act, (k[e] >> shift) & 255u, lane);
        }
      }
      __syncthreads();
      uint32_t cnt = 0;
      const uint32_t d = 255u - static_cast<uint32_t>(tid);
      if (tid < 256)
        for (int x = 0; x < kSelWaves; ++x) cnt += hist[x][d];
      uint32_t total;
      const uint32_t excl = sk_block_scan(cnt, wsum, total, lane, w);
      if (tid < 256 && above + excl < static_cast<uint32_t>(keep) &&
          above + excl + cnt >= static_cast<uint32_t>(keep)) {
        s_prefix = prefix | (d << shift);
        s_above = above + excl;
      }
      __syncthreads();
      prefix = s_prefix;
      above = s_above;
      __syncthreads();
    }
  }
  const uint32_t tau = prefix;
  const uint32_t need_eq = keep > 0 ? static_cast<uint32_t>(keep) - above : 0;

  // Ordered compaction, kSelStep positions per step, kSelPer consecutive ones
  // per thread: keep key > tau, and key == tau while fewer than need_eq of
  // those were kept before it; positions come out ascending, so ties go to
  // the smaller position.
  uint32_t out_base = 0, eq_base = 0;
  for (int base = 0; base < n && keep > 0; base += kSelStep) {
    const int j0 = base + tid * kSelPer;
    bool gt[kSelPer], eq[kSelPer];
    uint32_t n_eq = 0;
#pragma unroll
    for (int e = 0; e < kSelPer; ++e) {
      const int j = j0 + e;
      const uint32_t k = j < n ? key_at(j) : 0u;
      gt[e] = j < n && k > tau;
      eq[e] = j < n && k == tau;
      n_eq += eq[e];
    }
    uint32_t eq_total;
    uint32_t eq_before = eq_base + sk_block_scan(n_eq, wsum, eq_total, lane, w);
    bool take[kSelPer];
    uint32_t n_take = 0;
#pragma unroll
    for (int e = 0; e < kSelPer; ++e) {
      take[e] = gt[e] || (eq[e] && eq_before < need_eq);
      eq_before += eq[e];
      n_take += take[e];
    }
    uint32_t take_total;
    uint32_t pos = out_base + sk_block_scan(n_take, wsum, take_total, lane, w);
#pragma unroll
    for (int e = 0; e < kSelPer; ++e)
      if (take[e]) out[pos++] = j0 + e;
    out_base += take_total;
    eq_base += eq_total;
  }
  // The observation window, always kept.
  const int kept = keep > 0 ? keep : 0;
  for (int j = n + tid; j < S; j += kSelThreads) out[kept + (j - n)] = j;
  if (tid == 0 && (row % p.rows_per_seq) == 0) p.counts[b] = kept + (S - n);
}

// ---------------------------------------------------------------------------
// Host-side dispatch.

template <int D, bool BF16, int TW, int PASS>
static hipError_t sk_launch_tw(const SnapkvParams& p, bool paged, int64_t blocks, hipStream_t s) {
  // Wave-uniform row addresses where a wave's rows share a page and the
  // lane offsets fit 32 bits.
  using SH = SkShape<D, BF16>;
  constexpr int RPW = 64 / SH::LPT;
  const bool wa = (!paged || (int64_t{1} << p.page_shift) >= RPW) &&
                  p.s_tok >= 0 && p.s_tok * SH::ES * RPW <= (int64_t{1} << 30);
#define MD_SK_LAUNCH(PG, WAV)                                                                 \
  do {                                                                                        \
    if constexpr (TW == 1 || PASS == 1)                                                       \
      hipLaunchKernelGGL((snapkv_pass_kernel<D, BF16, TW, PG, WAV, PASS, kSkTile, kSkWaves>), \
                         dim3(blocks), dim3(kSkWaves * 64), 0, s, p);                         \
    else                                                                                      \
      hipLaunchKernelGGL((snapkv_pass_kernel<D, BF16, TW / 2, PG, WAV, PASS, kSkTile,         \
                                             kSkWavesWide>),                                  \
                         dim3(blocks), dim3(kSkWavesWide * 64), 0, s, p);                     \
  } while (0)
  if (paged) {
    if (wa) MD_SK_LAUNCH(true, true); else MD_SK_LAUNCH(true, false);
  } else {
    if (wa) MD_SK_LAUNCH(false, true); else MD_SK_LAUNCH(false, false);
  }
#undef MD_SK_LAUNCH
  return hipGetLastError();
}

template <int D, bool BF16, int PASS>
static hipError_t sk_launch_d(const SnapkvParams& p, int TW, bool paged, int64_t blocks,
                              hipStream_t s) {
  switch (TW) {
    case 1: return sk_launch_tw<D, BF16, 1, PASS>(p, paged, blocks, s);
    case 2: return sk_launch_tw<D, BF16, 2, PASS>(p, paged, blocks, s);
    case 4: return sk_launch_tw<D, BF16, 4, PASS>(p, paged, blocks, s);
  }
  return hipErrorInvalidValue;
}

template <int PASS>
static hipError_t sk_launch(const SnapkvParams& p, int head_dim, bool bf16, int TW, bool paged,
                            int64_t blocks, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  if (head_dim == 128)
    return bf16 ? sk_launch_d<128, true, PASS>(p, TW, paged, blocks, s)
                : sk_launch_d<128, false, PASS>(p, TW, paged, blocks, s);
  return bf16 ? sk_launch_d<64, true, PASS>(p, TW, paged, blocks, s)
              : sk_launch_d<64, false, PASS>(p, TW, paged, blocks, s);
}

hipError_t launch_snapkv_votes(const SnapkvParams& p, int head_dim, bool bf16, int TW, bool paged,
                               hipStream_t s) {
  SnapkvParams q = p;
  q.chunk_len = p.chunk_len_stats;
  q.n_chunks = p.n_chunks_stats;
  hipError_t e = sk_launch<0>(q, head_dim, bf16, TW, paged,
                              static_cast<int64_t>(p.n_units) * q.n_chunks, s);
  if (e != hipSuccess) return e;
  const int64_t rows = static_cast<int64_t>(p.n_units) * p.R;
  hipLaunchKernelGGL(snapkv_lse_kernel, dim3(static_cast<uint32_t>((rows + 255) / 256)), dim3(256),
                     0, s, q);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  q.chunk_len = p.chunk_len_votes;
  q.n_chunks = p.n_chunks_votes;
  return sk_launch<1>(q, head_dim, bf16, TW, paged,
                      static_cast<int64_t>(p.n_units) * q.n_chunks, s);
}

hipError_t launch_snapkv_select(const SnapkvSelectParams& p, hipStream_t s) {
  if (p.rows <= 0) return hipSuccess;
  const dim3 grid(p.rows), block(kSelThreads), rblock(kSelRegThreads);
  if (p.stride <= kSelRegKeys && p.pool / 2 <= kSelRegHalo) {
    switch (p.pool) {  // odd, checked by the caller
      case 1: hipLaunchKernelGGL(snapkv_select_reg_kernel<1>, grid, rblock, 0, s, p); break;
      case 3: hipLaunchKernelGGL(snapkv_select_reg_kernel<3>, grid, rblock, 0, s, p); break;
      case 5: hipLaunchKernelGGL(snapkv_select_reg_kernel<5>, grid, rblock, 0, s, p); break;
      default: hipLaunchKernelGGL(snapkv_select_reg_kernel<7>, grid, rblock, 0, s, p); break;
    }
  } else {
    hipLaunchKernelGGL(snapkv_select_kernel, grid, block, 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace md
