// attn.hip -- split-KV decode attention for MagicDec's verify and draft calls
// on gfx950 (MI355X).
//
// The paper locates the cost of large-batch long-context decoding in loading
// the KV cache (Sec. 1 insight 1, Sec. 3.2); verification of gamma+1 tokens
// reads the same cache as one decode step, and the StreamingLLM draft reads a
// fixed budget of sink and window tokens (Sec. 4.1 Eq. 3, Sec. 5.1).  The
// kernel therefore streams every visible K/V element of a (sequence, kv head)
// unit from HBM exactly once, for all G*(gamma+1) query rows that share it.
//
// One workgroup = one (unit, chunk); its kWaves waves take interleaved
// 32-token tiles of the chunk and run independent online softmaxes, merged
// through LDS at the end.  Per tile and wave:
//   K  16 B loads straight into the MFMA A-operand layout (8 bf16 channels of
//      one token per lane), Q held as the B operand for the whole chunk:
//      S^T[token, row] = K Q^T on v_mfma_f32_16x16x32_bf16.
//   softmax  each lane owns one query row and 8 of the tile's tokens; the
//      row max needs two cross-lane steps, the row sum is reduced only once
//      at the end.
//   V  16 B coalesced loads (whole 256 B token rows), staged through a
//      wave-private LDS tile and read back transposed as the A operand of
//      O^T[channel, row] += V^T P^T, whose output layout puts each lane's
//      row in the same place as its softmax state (no shuffles to rescale).
// The next tile's K/V (and page ids, two tiles ahead) are in flight while
// the current one is computed.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "kernels.h"

namespace md {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

template <int D, bool BF16>
struct Shape {
  static constexpr int ES = BF16 ? 2 : 4;          // element bytes
  static constexpr int E16 = 16 / ES;              // elements per 16 B
  static constexpr int KCB = D * ES / 64;          // 16 B K loads per lane per 16-token block
  static constexpr int KL = 2 * KCB;               // per tile (two 16-token blocks)
  static constexpr int LPT = D * ES / 16;          // lanes per V token row
  static constexpr int TPI = 64 / LPT;             // V tokens per load instruction
  static constexpr int NV = kTile / TPI;           // V loads per lane per tile
  static constexpr int CB16 = D / 16;              // 16-channel blocks of O
  static constexpr int VROW = D * ES + (BF16 ? 8 : 16);  // padded LDS row (bytes)
  static constexpr int VTILE = kTile * VROW;       // one wave's LDS V tile
};

// Where a virtual token of the unit's visible range lives.
struct UnitGeom {
  int S;           // clamped kv length
  int seg0;        // virtual tokens [0, seg0) are real tokens [0, seg0)
  int seg1_start;  // virtual v >= seg0 is real token v - seg0 + seg1_start
  int v_begin, v_end;
};

__device__ __forceinline__ int real_token(const UnitGeom& u, int v) {
  return v < u.seg0 ? v : v - u.seg0 + u.seg1_start;
}

template <int D, bool BF16, int NT, bool PAGED>
__global__ void __launch_bounds__(kWaves * 64)
attn_partial_kernel(const AttnParams p) {
  using SH = Shape<D, BF16>;
  constexpr int ROWS = NT * 16;
  // LDS: the V tiles during the main loop, then the cross-wave merge buffers.
  constexpr int kMergeO = kWaves * 16 * D * 4;
  constexpr int kMergeStats = 2 * kWaves * ROWS * 4;
  constexpr int kLds = (kWaves * SH::VTILE > kMergeO + kMergeStats) ? kWaves * SH::VTILE
                                                                     : kMergeO + kMergeStats;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLds];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l16 = lane & 15;
  const int grp = lane >> 4;

  const int chunk = blockIdx.x % p.n_chunks;
  const int unit = blockIdx.x / p.n_chunks;
  const int hk = unit % p.Hkv;
  const int b = unit / p.Hkv;
  const int L = p.L;

  // ---- the unit's visible range (a1/a5 of the method's hot path)
  UnitGeom u;
  u.S = min(p.kv_lens[b], p.max_kv_len);
  if (u.S < 0) u.S = 0;
  int U = u.S;
  u.seg0 = u.S;
  u.seg1_start = 0;
  if (p.mode == MD_MODE_DRAFT) {
    int lo = u.S - L - p.window + 1;
    if (lo > p.n_sink) {  // sinks, a gap that is never read, then the windows
      u.seg0 = p.n_sink;
      u.seg1_start = lo;
      U = p.n_sink + (u.S - lo);
    }
  }
  u.v_begin = chunk * p.chunk_len;
  u.v_end = min(U, u.v_begin + p.chunk_len);
  const int n_tiles = u.v_end > u.v_begin ? (u.v_end - u.v_begin + kTile - 1) / kTile : 0;

  // ---- per-lane query rows: row r = rt*16 + l16 is (i = r / G, head hk*G + r % G)
  int row_pos[NT];  // query position p = S - L + i; -1 (sees nothing) for padding rows
  for (int rt = 0; rt < NT; ++rt) {
    int r = rt * 16 + l16;
    row_pos[rt] = r < p.R ? u.S - L + r / p.G : -1;
  }

  // ---- Q as the B operand: lane holds channels cb*(64/ES) + grp*E16 .. +E16 of its row
  u32x4 qreg[NT][SH::KCB];
  for (int rt = 0; rt < NT; ++rt) {
    int r = rt * 16 + l16;
    for (int cb = 0; cb < SH::KCB; ++cb) qreg[rt][cb] = u32x4{0, 0, 0, 0};
    if (r < p.R) {
      int i = r / p.G, h = hk * p.G + r % p.G;
      const unsigned char* qp = static_cast<const unsigned char*>(p.q) +
                                ((static_cast<int64_t>(b) * L + i) * p.Hq + h) * D * SH::ES;
      for (int cb = 0; cb < SH::KCB; ++cb)
        qreg[rt][cb] = *reinterpret_cast<const u32x4*>(qp + cb * 64 + grp * 16);
    }
  }

  const unsigned char* kbase = static_cast<const unsigned char*>(p.k);
  const unsigned char* vbase = static_cast<const unsigned char*>(p.v);
  const int64_t head_off = static_cast<int64_t>(hk) * p.s_head;
  const int32_t* ptab = PAGED ? p.page_table + static_cast<int64_t>(b) * p.max_pages : nullptr;
  const int pmask = (1 << p.page_shift) - 1;

  // Element offset of real token t given its page id (paged) -- or -1 if the
  // page id is outside the pool, so the token is never dereferenced.
  auto tok_offset = [&](int t, int pid) -> int64_t {
    if (PAGED) {
      if (pid < 0 || pid >= p.num_pages) return -1;
      return static_cast<int64_t>(pid) * p.s_blk + static_cast<int64_t>(t & pmask) * p.s_tok +
             head_off;
    }
    return static_cast<int64_t>(b) * p.s_blk + static_cast<int64_t>(t) * p.s_tok + head_off;
  };

  // Page id of the token this lane stands for (lane & 31 of tile `tile`).
  auto load_pid = [&](int tile) -> int {
    if (!PAGED) return 0;
    int v = u.v_begin + tile * kTile + (lane & 31);
    if (tile >= n_tiles || v >= u.v_end) return -1;
    return ptab[real_token(u, v) >> p.page_shift];
  };

  struct TileRegs {
    u32x4 k[SH::KL];
    u32x4 v[SH::NV];
  };

  // Issue the loads of one tile.  tpid: this lane's page id for token lane&31.
  auto load_tile = [&](TileRegs& T, int tile, int tpid) {
    const int v0 = u.v_begin + tile * kTile;
    const bool live = tile < n_tiles;
    // K: lane = token (l16) of block tb, channel group grp of block cb.
    for (int tb = 0; tb < 2; ++tb) {
      int vt = v0 + tb * 16 + l16;
      int pid = PAGED ? __shfl(tpid, tb * 16 + l16) : 0;
      bool ok = live && vt < u.v_end;
      int64_t off = ok ? tok_offset(real_token(u, vt), pid) : -1;
      for (int cb = 0; cb < SH::KCB; ++cb) {
        u32x4 x = u32x4{0, 0, 0, 0};
        if (off >= 0) x = *reinterpret_cast<const u32x4*>(kbase + off * SH::ES + cb * 64 + grp * 16);
        T.k[tb * SH::KCB + cb] = x;
      }
    }
    // V: whole token rows, LPT lanes per token.
    for (int n = 0; n < SH::NV; ++n) {
      int tt = n * SH::TPI + lane / SH::LPT;
      int vt = v0 + tt;
      int pid = PAGED ? __shfl(tpid, tt) : 0;
      bool ok = live && vt < u.v_end;
      int64_t off = ok ? tok_offset(real_token(u, vt), pid) : -1;
      u32x4 x = u32x4{0, 0, 0, 0};
      if (off >= 0)
        x = *reinterpret_cast<const u32x4*>(vbase + off * SH::ES + (lane % SH::LPT) * 16);
      T.v[n] = x;
    }
  };

  // Online softmax state (log2 domain) and the O^T accumulators.
  float m_run[NT], l_run[NT];
  f32x4 acc[NT][SH::CB16];
  for (int rt = 0; rt < NT; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.f;
    for (int c = 0; c < SH::CB16; ++c) acc[rt][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  unsigned char* vt_lds = lds + wave * SH::VTILE;

  TileRegs cur, nxt;
  int tile = wave;
  int pid_cur = load_pid(tile);
  int pid_nxt = load_pid(tile + kWaves);
  if (tile < n_tiles) load_tile(cur, tile, pid_cur);

  for (; tile < n_tiles; tile += kWaves) {
    // Prefetch: page ids two tiles ahead, K/V one tile ahead.
    int pid_nn = load_pid(tile + 2 * kWaves);
    load_tile(nxt, tile + kWaves, pid_nxt);

    const int v0 = u.v_begin + tile * kTile;

    // Stage V rows in this wave's LDS tile (row tt, channels (lane%LPT)*E16..).
    for (int n = 0; n < SH::NV; ++n) {
      int tt = n * SH::TPI + lane / SH::LPT;
      unsigned char* dst = vt_lds + tt * SH::VROW + (lane % SH::LPT) * 16;
      reinterpret_cast<u32x2*>(dst)[0] = u32x2{cur.v[n].x, cur.v[n].y};
      reinterpret_cast<u32x2*>(dst)[1] = u32x2{cur.v[n].z, cur.v[n].w};
    }

    // Real token index and validity of this lane's 8 score slots.
    int tok[2][4];
    bool tvalid[2][4];
    for (int tb = 0; tb < 2; ++tb)
      for (int e = 0; e < 4; ++e) {
        int vt = v0 + tb * 16 + grp * 4 + e;
        tvalid[tb][e] = vt < u.v_end;
        tok[tb][e] = real_token(u, vt);
      }

    // S^T = K Q^T, masked, scaled into the log2 domain.
    float x[NT][2][4];
    for (int tb = 0; tb < 2; ++tb) {
      for (int rt = 0; rt < NT; ++rt) {
        f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int cb = 0; cb < SH::KCB; ++cb) {
          const u32x4 kk = cur.k[tb * SH::KCB + cb];
          const u32x4 qq = qreg[rt][cb];
          if constexpr (BF16) {
            s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kk),
                                                        __builtin_bit_cast(bf16x8, qq), s, 0, 0, 0);
          } else {
            for (int j = 0; j < 4; ++j)
              s = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kk[j]),
                                                        __uint_as_float(qq[j]), s, 0, 0, 0);
          }
        }
        for (int e = 0; e < 4; ++e) {
          const int t = tok[tb][e];
          const int pos = row_pos[rt];
          bool vis = tvalid[tb][e] && t <= pos;
          if (p.mode == MD_MODE_DRAFT) vis = vis && (t < p.n_sink || t >= pos - p.window + 1);
          x[rt][tb][e] = vis ? s[e] * p.scale_log2 : -INFINITY;
        }
      }
    }

    // Online softmax per row: tile max over this lane's 8 slots and the 3
    // other lanes holding the same row (lanes l16 + 16*grp).
    u32x4 pb[NT];    // bf16 P^T B operand (8 slots)
    float pf[NT][2][4];  // fp32 P for the fp32 path
    for (int rt = 0; rt < NT; ++rt) {
      float mx = -INFINITY;
      for (int tb = 0; tb < 2; ++tb)
        for (int e = 0; e < 4; ++e) mx = fmaxf(mx, x[rt][tb][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[rt], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[rt] - m_use);
      m_run[rt] = m_new;
      float psum = 0.f;
      uint32_t h[8];
      for (int tb = 0; tb < 2; ++tb)
        for (int e = 0; e < 4; ++e) {
          float pv = fast_exp2(x[rt][tb][e] - m_use);
          if constexpr (BF16) {
            uint32_t hb = f32_to_bf16(pv);
            h[tb * 4 + e] = hb;
            psum += bf16_to_f32(hb);  // normalise by exactly what multiplies V
          } else {
            pf[rt][tb][e] = pv;
            psum += pv;
          }
        }
      if constexpr (BF16) {
        pb[rt] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                       h[6] | (h[7] << 16)};
      }
      l_run[rt] = l_run[rt] * alpha + psum;
      for (int c = 0; c < SH::CB16; ++c) acc[rt][c] *= alpha;
    }

    // O^T += V^T P^T.  A operand: lane = channel (l16) of block c, slots of
    // group grp = tokens {4grp..4grp+3, 16+4grp..16+4grp+3} as in the scores.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int c = 0; c < SH::CB16; ++c) {
      const int ch = c * 16 + l16;
      if constexpr (BF16) {
        const unsigned char* src = vt_lds + ch * 2;
        uint32_t e[8];
        for (int j = 0; j < 8; ++j) {
          int tt = (j < 4) ? grp * 4 + j : 16 + grp * 4 + (j - 4);
          e[j] = *reinterpret_cast<const uint16_t*>(src + tt * SH::VROW);
        }
        const u32x4 va = u32x4{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                               e[6] | (e[7] << 16)};
        for (int rt = 0; rt < NT; ++rt)
          acc[rt][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, va), __builtin_bit_cast(bf16x8, pb[rt]), acc[rt][c], 0,
              0, 0);
      } else {
        const unsigned char* src = vt_lds + ch * 4;
        for (int tb = 0; tb < 2; ++tb)
          for (int j = 0; j < 4; ++j) {
            float va = *reinterpret_cast<const float*>(src + (tb * 16 + grp * 4 + j) * SH::VROW);
            for (int rt = 0; rt < NT; ++rt)
              acc[rt][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(va, pf[rt][tb][j], acc[rt][c], 0,
                                                                0, 0);
          }
      }
    }
    // The next iteration overwrites this wave's LDS tile: keep the reads first.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    cur = nxt;
    pid_nxt = pid_nn;
  }

  // ---- row sums: add the 4 lanes that share a row
  for (int rt = 0; rt < NT; ++rt) {
    l_run[rt] += __shfl_xor(l_run[rt], 16);
    l_run[rt] += __shfl_xor(l_run[rt], 32);
  }

  // ---- merge the kWaves waves of the workgroup (LDS reused after the loop)
  __syncthreads();
  float* sm_m = reinterpret_cast<float*>(lds + kMergeO);
  float* sm_l = sm_m + kWaves * ROWS;
  float* mo = reinterpret_cast<float*>(lds);
  if (grp == 0) {
    for (int rt = 0; rt < NT; ++rt) {
      sm_m[wave * ROWS + rt * 16 + l16] = m_run[rt];
      sm_l[wave * ROWS + rt * 16 + l16] = l_run[rt];
    }
  }
  __syncthreads();
  // Each wave rescales its own O by 2^(m_w - M) / L_total.
  for (int rt = 0; rt < NT; ++rt) {
    const int r = rt * 16 + l16;
    float M = -INFINITY;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm_m[w * ROWS + r]);
    float Lt = 0.f;
    if (M != -INFINITY)
      for (int w = 0; w < kWaves; ++w) {
        float mw = sm_m[w * ROWS + r];
        if (mw != -INFINITY) Lt += sm_l[w * ROWS + r] * fast_exp2(mw - M);
      }
    float f = 0.f;
    if (m_run[rt] != -INFINITY && Lt > 0.f) f = fast_exp2(m_run[rt] - M) / Lt;
    for (int c = 0; c < SH::CB16; ++c) acc[rt][c] *= f;
  }

  const bool direct = p.n_chunks == 1;
  const int tid = threadIdx.x;
  for (int rt = 0; rt < NT; ++rt) {
    // Wave w writes its scaled O^T rows (lane: row l16, channels c*16+4grp..+3).
    for (int c = 0; c < SH::CB16; ++c)
      *reinterpret_cast<f32x4*>(mo + (wave * 16 + l16) * D + c * 16 + grp * 4) = acc[rt][c];
    __syncthreads();
    // Thread -> (row, 8 channels); sum the waves in a fixed order.
    constexpr int kGroupsPerRow = D / 8;
    const int rr = tid / kGroupsPerRow;
    const int c0 = (tid % kGroupsPerRow) * 8;
    const int r = rt * 16 + rr;
    if (rr < 16 && r < p.R) {
      float o8[8];
      for (int j = 0; j < 8; ++j) o8[j] = 0.f;
      for (int w = 0; w < kWaves; ++w)
        for (int j = 0; j < 8; ++j) o8[j] += mo[(w * 16 + rr) * D + c0 + j];
      const int i = r / p.G, h = hk * p.G + r % p.G;
      const int64_t row_g = (static_cast<int64_t>(b) * L + i) * p.Hq + h;
      float M = -INFINITY, Lt = 0.f;
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm_m[w * ROWS + r]);
      if (M != -INFINITY)
        for (int w = 0; w < kWaves; ++w) {
          float mw = sm_m[w * ROWS + r];
          if (mw != -INFINITY) Lt += sm_l[w * ROWS + r] * fast_exp2(mw - M);
        }
      const float lse = (Lt > 0.f) ? (M + fast_log2(Lt)) * 0.69314718055994530942f : -INFINITY;
      if (direct) {
        if constexpr (BF16) {
          uint32_t hb[8];
          for (int j = 0; j < 8; ++j) hb[j] = f32_to_bf16(o8[j]);
          *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.o) + row_g * D + c0) =
              u32x4{hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16), hb[4] | (hb[5] << 16),
                    hb[6] | (hb[7] << 16)};
        } else {
          float* op = static_cast<float*>(p.o) + row_g * D + c0;
          *reinterpret_cast<f32x4*>(op) = f32x4{o8[0], o8[1], o8[2], o8[3]};
          *reinterpret_cast<f32x4*>(op + 4) = f32x4{o8[4], o8[5], o8[6], o8[7]};
        }
        if (p.lse && c0 == 0) p.lse[row_g] = lse;
      } else {
        float* op = p.part_o + (static_cast<int64_t>(chunk) * p.n_rows + row_g) * D + c0;
        *reinterpret_cast<f32x4*>(op) = f32x4{o8[0], o8[1], o8[2], o8[3]};
        *reinterpret_cast<f32x4*>(op + 4) = f32x4{o8[4], o8[5], o8[6], o8[7]};
        if (c0 == 0) p.part_lse[static_cast<int64_t>(chunk) * p.n_rows + row_g] = lse;
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Host-side dispatch over the compiled instances.

template <int D, bool BF16, int NT>
static hipError_t launch_nt(const AttnParams& p, bool paged, int64_t n_blocks, hipStream_t s) {
  dim3 grid(static_cast<uint32_t>(n_blocks)), block(kWaves * 64);
  if (paged)
    hipLaunchKernelGGL((attn_partial_kernel<D, BF16, NT, true>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((attn_partial_kernel<D, BF16, NT, false>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t launch_d(const AttnParams& p, int NT, bool paged, int64_t n_blocks,
                           hipStream_t s) {
  switch (NT) {
    case 1: return launch_nt<D, BF16, 1>(p, paged, n_blocks, s);
    case 2: return launch_nt<D, BF16, 2>(p, paged, n_blocks, s);
    case 3: return launch_nt<D, BF16, 3>(p, paged, n_blocks, s);
    case 4: return launch_nt<D, BF16, 4>(p, paged, n_blocks, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attn_partial(const AttnParams& p, int head_dim, bool bf16, int NT, bool paged,
                               int64_t n_blocks, hipStream_t s) {
  if (n_blocks <= 0) return hipSuccess;
  if (head_dim == 128)
    return bf16 ? launch_d<128, true>(p, NT, paged, n_blocks, s)
                : launch_d<128, false>(p, NT, paged, n_blocks, s);
  return bf16 ? launch_d<64, true>(p, NT, paged, n_blocks, s)
              : launch_d<64, false>(p, NT, paged, n_blocks, s);
}

}  // namespace md
