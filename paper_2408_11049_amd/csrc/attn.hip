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
// One workgroup = one chunk of hp units (hp adjacent kv heads of a sequence,
// so that the waves of a workgroup read neighbouring runs of each token row);
// the W / hp waves of a unit (W = 4, or 8 in the wide instances of up to
// two row tiles) take interleaved 32-token tiles of the chunk and run
// independent online softmaxes, merged through LDS at the end.
// Per tile and wave:
//   load     K and V as whole token rows (256 B for bf16, d = 128: 16 lanes
//            per row, nontemporal 16 B loads, one address per token), staged
//            through the wave's private LDS tiles.
//   scores   K read back as the MFMA A operand (a token per lane), Q held as
//            the B operand for the whole chunk: S^T[token, row] = K Q^T on
//            v_mfma_f32_16x16x32_bf16.
//   softmax  each lane owns one query row and 8 of the tile's tokens; the
//            row max needs two cross-lane steps, the row sum is reduced only
//            once at the end.
//   values   V read back transposed (ds_read_b64_tr_b16) as the A operand of
//            O^T[channel, row] += V^T P^T, whose output layout puts each
//            lane's row in the same place as its softmax state (no shuffles
//            to rescale).
// The next tile's K/V (and page ids, two tiles ahead) are in flight while
// the current one is computed.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "kernels.h"

namespace md {

// Device-scope release / acquire around a split plan's arrival counter.
#ifndef MD_PARTIAL_RELEASE
// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left at their maxima): this wave's
// stores are complete.
#define MD_PARTIAL_WAVE_DONE() __builtin_amdgcn_s_waitcnt(0x0F70)
#define MD_PARTIAL_RELEASE() __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent")
#define MD_PARTIAL_ACQUIRE() __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent")
#endif

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Two fp32 -> packed bf16, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

template <int D, bool BF16>
struct Shape {
  static constexpr int ES = BF16 ? 2 : 4;          // element bytes
  static constexpr int E16 = 16 / ES;              // elements per 16 B
  static constexpr int KCB = D * ES / 64;          // 16 B A-operand chunks per lane per 16-token block
  static constexpr int LPT = D * ES / 16;          // lanes per token row (16 B each)
  static constexpr int TPI = 64 / LPT;             // token rows per load instruction
  static constexpr int NV = kTile / TPI;           // K (and V) loads per lane per tile
  static constexpr int CB16 = D / 16;              // 16-channel blocks of O
  // Padded LDS rows (bytes).  K: an odd multiple of 16 B, so the 16 rows of
  // one A-operand read hit distinct banks.  V: an odd multiple of 32 B, so
  // the 16-row transposed reads of one channel block spread over all banks.
  static constexpr int KROW = D * ES + 16;
  static constexpr int VROW = D * ES + (BF16 ? 32 : 16);
  static constexpr int KTILE = kTile * KROW;
  static constexpr int VTILE = kTile * VROW;
  static constexpr int WTILE = KTILE + VTILE;      // one wave's LDS staging
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

// Longest-processing-time-first dispatch.  Workgroups start roughly in
// blockIdx order (round-robin over the XCDs), so with ragged lengths the
// units that happen to start last set the finish time.  With p.lpt (one chunk
// per unit, B <= kLptMaxSeqs), workgroup r instead takes the r-th head group
// in the order (length descending, sequence ascending, kv head ascending):
// every workgroup ranks the B clamped lengths in LDS (B compares per thread)
// and picks the sequence of rank r / gps, gps = Hkv / hp head groups per
// sequence.  The order is a bijection, so each unit is still computed once,
// with the same arithmetic.
//
// With p.hp_auto the grid has one workgroup per unit and the kernel chooses
// hp here: head pairs stream faster, but there are half as many of them, and
// each is twice as long -- at one pair per compute unit, too few and too
// coarse for longest-first to even out unequal lengths.  Pairs are taken when
// the longest clamped length is within 1/16 of the mean, or when there are at
// least two pairs per compute unit and the longest pair is no more than a
// compute unit's mean share of the work (the workgroups past the pairs then
// return at once); otherwise one head per workgroup.  Measured on MI355X
// (Llama-3.1-8B heads, lengths uniform in a range): at B = 64 single heads
// beat pairs by 6-33% on ragged lengths; at B = 128 and 256 pairs beat
// single heads by 4-7%.  Returns the head group, or -1 for a workgroup with
// nothing to do.
template <typename P>
__device__ __forceinline__ int lpt_group(const P& p, int r, int* sl, int& hp) {
  const int B = p.num_seqs;
  for (int t = threadIdx.x; t < B; t += static_cast<int>(blockDim.x)) {
    const int s = min(p.kv_lens[t], p.max_kv_len);
    sl[t] = s < 0 ? 0 : s;
  }
  __syncthreads();
  if (p.hp_auto) {
    if (threadIdx.x < 64) {
      int mx = 0;
      long long sum = 0;
      for (int t = threadIdx.x; t < B; t += 64) {
        mx = max(mx, sl[t]);
        sum += sl[t];
      }
      for (int o = 32; o >= 1; o >>= 1) {
        mx = max(mx, __shfl_xor(mx, o));
        sum += __shfl_xor(sum, o);
      }
      if (threadIdx.x == 0) {
        const bool even = 16LL * mx * B <= 17LL * sum;
        const bool many = static_cast<long long>(B) * p.Hkv >= 4LL * p.slots &&
                          2LL * mx * p.slots <= static_cast<long long>(p.Hkv) * sum;
        sl[kLptMaxSeqs + 1] = (even || many) ? 2 : 1;
      }
    }
    __syncthreads();
    hp = sl[kLptMaxSeqs + 1];
  }
  const int gps = p.Hkv / hp;
  if (r >= B * gps) return -1;  // uniform over the workgroup: it returns as a whole
  const int want = r / gps;
  for (int t = threadIdx.x; t < B; t += static_cast<int>(blockDim.x)) {
    const int lt = sl[t];
    int rank = 0;
    for (int j = 0; j < B; ++j) {
      const int lj = sl[j];
      rank += (lj > lt) || (lj == lt && j < t);
    }
    if (rank == want) sl[kLptMaxSeqs] = t;
  }
  __syncthreads();
  const int b = sl[kLptMaxSeqs];
  __syncthreads();  // the LDS is reused by the tiles
  return b * gps + r % gps;
}

// Balanced verify (p.bal).  The tiles of every head group -- group g =
// b * gps + j owns tiles_b = max(1, ceil(S_b / kTile)) of them, groups in
// order -- form one stream of TT tiles, cut into NW ranges of equal length,
// one per workgroup (NW below): every workgroup streams the same number of
// tiles (to within one) whatever the lengths, and keeps the head pairs that
// read a token row's neighbouring runs together.  A group that a range
// boundary cuts is computed in pieces by consecutive workgroups, which merge
// them (the split-KV identity); with NW = min(workgroups, TT) ranges, stream
// tile t belongs to workgroup ((t + 1) NW - 1) / TT, whose range starts at
// w TT / NW.  Only a range's first and last pieces can be cut, so workgroup
// w keeps the partials of its first piece in slot 2w and of its last in
// slot 2w + 1.
struct BalCursor {
  int lo;      // this workgroup's range [lo, hi)
  int t, hi;   // its next stream tile and the end of its range
  int b, j;    // the current group: sequence b, its group j
  int g0, gt;  // the group's first stream tile and its number of tiles
  int TT;      // tiles in the whole stream
  int NW;      // workgroups sharing it: min(grid, TT), so no range is empty
};

template <typename P>
__device__ __forceinline__ int bal_tiles(const P& p, int b) {
  int s = min(p.kv_lens[b], p.max_kv_len);
  s = s < 0 ? 0 : s;
  return max(1, (s + kTile - 1) / kTile);
}

__device__ __forceinline__ int bal_owner(int t, int nw, int tt) {
  return static_cast<int>((static_cast<int64_t>(t + 1) * nw - 1) / tt);
}

// The workgroup's range and its first group; false for an empty range.  sl:
// LDS for kLptMaxSeqs + 1 ints (free again on return).
template <typename P>
__device__ bool bal_start(const P& p, int gps, int* sl, BalCursor& c) {
  const int B = p.num_seqs;  // <= kLptMaxSeqs
  if (threadIdx.x < 64) {    // wave 0: stream tiles per sequence, inclusive scan
    constexpr int kPer = kLptMaxSeqs / 64;
    int v[kPer];
    int local = 0;
    for (int e = 0; e < kPer; ++e) {
      const int bb = static_cast<int>(threadIdx.x) * kPer + e;
      v[e] = bb < B ? bal_tiles(p, bb) * gps : 0;
      local += v[e];
    }
    int incl = local;
    for (int o = 1; o < 64; o <<= 1) {
      const int x = __shfl_up(incl, o);
      if (static_cast<int>(threadIdx.x) >= o) incl += x;
    }
    int run = incl - local;
    for (int e = 0; e < kPer; ++e) {
      run += v[e];
      sl[threadIdx.x * kPer + e] = run;
    }
  }
  __syncthreads();
  const int tt = sl[B - 1];
  // At least one tile per range: a group's pieces then come from consecutive
  // workgroups with no empty one between them (their count is its arrivals).
  const int nw = min(static_cast<int>(gridDim.x), tt);
  if (static_cast<int>(blockIdx.x) >= nw) return false;  // uniform over the workgroup
  const int lo = static_cast<int>(static_cast<int64_t>(blockIdx.x) * tt / nw);
  const int hi = static_cast<int>(static_cast<int64_t>(blockIdx.x + 1) * tt / nw);
  for (int bb = threadIdx.x; bb < B; bb += static_cast<int>(blockDim.x)) {
    const int ex = bb ? sl[bb - 1] : 0;
    if (ex <= lo && lo < sl[bb]) sl[kLptMaxSeqs] = bb;
  }
  __syncthreads();
  const int b = sl[kLptMaxSeqs];
  const int ex = b ? sl[b - 1] : 0;
  __syncthreads();  // the LDS is reused by the tiles
  const int tb = bal_tiles(p, b);
  c.TT = tt;
  c.NW = nw;
  c.lo = lo;
  c.t = lo;
  c.hi = hi;
  c.b = b;
  c.j = (lo - ex) / tb;
  c.g0 = ex + c.j * tb;
  c.gt = tb;
  return true;
}

// Moves to the workgroup's next piece; false when its range is done.
template <typename P>
__device__ __forceinline__ bool bal_next(const P& p, int gps, BalCursor& c) {
  c.t = min(c.hi, c.g0 + c.gt);
  if (c.t >= c.hi) return false;
  c.g0 += c.gt;
  if (++c.j == gps) {
    c.j = 0;
    ++c.b;
    c.gt = bal_tiles(p, c.b);
  }
  return true;
}

// Contract checks for a caller that passes an error word (debug use), ahead
// of the K/V stream; they change no result.  The lengths are checked once per
// sequence (its first head group's first chunk).  Paged: the page id of every
// position this workgroup reads -- one position per page and segment of a
// shared range, checked by the sequence's first head group; every usable
// list entry and speculated position of a listed draft, by the first wave of
// each head.
template <bool PAGED, bool IDX, typename P, typename U>
__device__ void check_contract(const P& p, const U& u, int b, int chunk, bool first_group,
                               bool first_wave, const int32_t* idxrow, int lane) {
  uint32_t bits = 0;
  if (chunk == 0 && first_group && threadIdx.x == 0) {
    const int raw = p.kv_lens[b];
    if (raw < p.L) bits |= MD_ERRW_SHORT_LEN;
    if (raw > p.max_kv_len) bits |= MD_ERRW_LONG_LEN;
  }
  if constexpr (PAGED) {
    const bool mine = IDX ? first_wave : first_group;
    const int start = IDX ? lane : static_cast<int>(threadIdx.x);
    const int step = IDX ? 64 : static_cast<int>(blockDim.x);
    const int pmask = (1 << p.page_shift) - 1;
    if (mine) {
      for (int v = u.v_begin + start; v < u.v_end; v += step) {
        int t;
        if constexpr (IDX) {
          if (v < u.seg0) {
            t = idxrow[v];
            if (t < 0 || t >= u.S - p.L) continue;  // an unusable entry is skipped, not read
          } else {
            t = v - u.seg0 + u.seg1_start;
          }
        } else {
          t = real_token(u, v);
          if (v != u.v_begin && v != u.seg0 && (t & pmask) != 0) continue;  // page already covered
        }
        const int pg = t >> p.page_shift;
        const int pid = pg < p.max_pages ? p.page_table[static_cast<int64_t>(b) * p.max_pages + pg] : -1;
        if (pid < 0 || pid >= p.num_pages) bits |= MD_ERRW_BAD_PAGE;
      }
    }
  }
  if (bits) atomicOr(reinterpret_cast<unsigned int*>(p.err), bits);
}

// The attention kernel.  D: head_dim; BF16: bf16 (else fp32) K/V/Q/O; NT:
// 16-row query tiles per unit; PAGED: K/V through the page table; IDX: the
// visible range is a per-(sequence, kv head) list of prompt positions
// followed by the speculated tokens (the listed draft), else the causal
// prefix (verify) or sinks then windows (draft); P: K/V tiles in flight per
// wave; OCC: waves per SIMD the instance is compiled for; BAL: the balanced
// verify (a workgroup takes an equal share of all groups' tiles, piece by
// piece; its own instances, so the others keep their register budget); W:
// waves per workgroup (kWaves, or kWavesWide: two per SIMD in one workgroup,
// each taking half as many of the unit's tiles).
template <int D, bool BF16, int NT, bool PAGED, bool IDX, int P, int OCC, bool BAL, int W>
__global__ void __launch_bounds__(W * 64) __attribute__((amdgpu_waves_per_eu(OCC)))
attn_partial_kernel(const AttnParams p) {
  using SH = Shape<D, BF16>;
  constexpr int ROWS = NT * 16;
  // LDS: the V tiles during the main loop, then the cross-wave merge buffers.
  // Cross-wave merge rows are padded by 16 B: at D floats a row is a multiple
  // of the 256 B bank period, so the 16 rows a wave stores at once would all
  // start in the same bank (measured: drafts 1-3% faster, outputs identical).
  // Every wave's row tiles are held at once (up to 135 KB at four row tiles).
  constexpr int MROW = D + 4;
  constexpr int kMergeO = W * NT * 16 * MROW * 4;
  constexpr int kMergeStats = 2 * W * ROWS * 4;
  constexpr int kLds = (W * SH::WTILE > kMergeO + kMergeStats) ? W * SH::WTILE
                                                               : kMergeO + kMergeStats;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLds];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l16 = lane & 15;
  const int grp = lane >> 4;
  // Measurement stamps (p.stamps, normally NULL): wall clock of workgroup
  // start, first tile done, main loop done and end, by its first lane.
  auto stamp = [&](int k) {
    if (p.stamps != nullptr && threadIdx.x == 0)
      p.stamps[static_cast<int64_t>(blockIdx.x) * 4 + k] = __builtin_amdgcn_s_memrealtime();
  };
  stamp(0);

  // Workgroups are numbered chunk-major: those that start together take the
  // same chunk of different head groups, so they read neighbouring runs of
  // the same token rows at the same time (measured on MI355X: split verify
  // plans 1-5% faster than group-major; with one chunk the two coincide).
  const int n_grp = static_cast<int>(gridDim.x) / p.n_chunks;
  const int chunk = static_cast<int>(blockIdx.x) / n_grp;
  // The workgroup's head group: hp adjacent kv heads hk0 .. hk0+hp-1 of
  // sequence b.  Wave w serves kv head hk0 + w % hp and is slot w / hp of
  // that head's wph = W / hp waves, which interleave its tiles.
  // Wave-uniform by construction; readfirstlane lets the compiler keep the
  // unit's address arithmetic in scalar registers.
  int hp_sel = p.hp;
  int group_sel = 0;
  BalCursor bc{};
  if constexpr (BAL) {
    if (!bal_start(p, p.Hkv / p.hp, reinterpret_cast<int*>(lds), bc)) return;
  } else if (p.lpt) {
    group_sel = lpt_group(p, static_cast<int>(blockIdx.x), reinterpret_cast<int*>(lds), hp_sel);
    if (group_sel < 0) return;
  } else {
    group_sel = static_cast<int>(blockIdx.x) % n_grp;
  }
  const int hp = __builtin_amdgcn_readfirstlane(hp_sel);
  const int wph = W / hp;
  const int gps = p.Hkv / hp;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int wslot = wave_u / hp;
  const int L = p.L;

  // One pass per piece: a balanced workgroup takes the pieces of its range
  // in turn; every other launch has exactly one.
  for (;;) {
  const int group = __builtin_amdgcn_readfirstlane(BAL ? bc.b * gps + bc.j : group_sel);
  const int b = group / gps;
  const int hk0 = (group % gps) * hp;
  const int hk = hk0 + wave_u % hp;
  // A balanced piece: tiles [lt0, lt1) of its group; whole when it is all of it.
  const int lt0 = __builtin_amdgcn_readfirstlane(bc.t - bc.g0);
  const int lt1 = __builtin_amdgcn_readfirstlane(min(bc.hi, bc.g0 + bc.gt) - bc.g0);
  const bool bal_whole = lt0 == 0 && lt1 == bc.gt;

  // ---- the unit's visible range: the causal prefix, sinks then windows, or the list
  UnitGeom u;
  u.S = __builtin_amdgcn_readfirstlane(min(p.kv_lens[b], p.max_kv_len));
  if (u.S < 0) u.S = 0;
  int U = u.S;
  u.seg0 = u.S;
  u.seg1_start = 0;
  if constexpr (IDX) {
    // The listed prompt positions, then the L speculated tokens.
    const int nb = min(max(p.idx_len[b], 0), p.idx_stride);
    u.seg0 = nb;
    u.seg1_start = u.S - L;
    U = nb + L;
  } else if (p.mode == MD_MODE_DRAFT) {
    int lo = u.S - L - p.window + 1;
    if (lo > p.n_sink) {  // sinks, a gap that is never read, then the windows
      u.seg0 = p.n_sink;
      u.seg1_start = lo;
      U = p.n_sink + (u.S - lo);
    }
  }
  if constexpr (BAL) {
    u.v_begin = lt0 * kTile;
    u.v_end = min(U, lt1 * kTile);
  } else {
    u.v_begin = chunk * p.chunk_len;
    u.v_end = min(U, u.v_begin + p.chunk_len);
  }
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

  // Element offset of real token t given its page id (paged).  A token that
  // must not be read (past the chunk, or a page id outside the pool) is
  // redirected to element 0 of the tensor -- always in bounds.  Past the
  // chunk its value is discarded (the score is masked, the V row zeroed);
  // a page id outside the pool is a caller's contract violation, reported
  // through the error word only, and the rows that see the token get
  // unspecified results.  Loads are therefore never under divergent control
  // flow, which lets the compiler keep every prefetched tile in flight
  // across loop iterations.
  auto tok_offset = [&](int t, int pid, bool& ok) -> int64_t {
    if (PAGED) {
      ok = ok && pid >= 0 && pid < p.num_pages;
      return ok ? static_cast<int64_t>(pid) * p.s_blk +
                      static_cast<int64_t>(t & pmask) * p.s_tok + head_off
                : 0;
    }
    return ok ? static_cast<int64_t>(b) * p.s_blk + static_cast<int64_t>(t) * p.s_tok + head_off
              : 0;
  };

  // Where the token this lane stands for (lane & 31 of tile `tile`) lives:
  // its position (-1 if it must not be read: past the chunk, an unusable list
  // entry) and, paged, its page id.  The list row and the table row always
  // have an entry 0, so every load here is in bounds.
  const int32_t* idxrow =
      IDX ? p.idx + (static_cast<int64_t>(b) * p.Hkv + hk) * p.idx_stride : nullptr;
  struct TokRef {
    int tok;
    int pid;
  };
  auto load_ref = [&](int tile) -> TokRef {
    const int v = u.v_begin + tile * kTile + (lane & 31);
    const bool ok = tile < n_tiles && v < u.v_end;
    int t;
    bool valid = ok;
    if constexpr (IDX) {
      const bool listed = v < u.seg0;
      const int lt = idxrow[(ok && listed) ? v : 0];
      t = listed ? lt : v - u.seg0 + u.seg1_start;
      valid = ok && t >= 0 && (!listed || t < u.S - L);
    } else {
      t = real_token(u, v);
    }
    int pid = 0;
    if constexpr (PAGED) {
      const int raw = ptab[valid ? (t >> p.page_shift) : 0];
      pid = valid ? raw : -1;
    }
    return TokRef{valid ? t : -1, pid};
  };

  struct TileRegs {
    u32x4 k[SH::NV];
    u32x4 v[SH::NV];
    uint32_t ok;  // bit n: token row of load n is real (else V is staged as zeros)
    int tok;      // IDX: position of this lane's tile token (lane & 31), -1 if none
  };

  // 16-byte streaming load: every K/V byte is read exactly once, so the
  // loads carry the nontemporal hint and do not displace reusable lines.
  auto ld16 = [](const unsigned char* ptr) -> u32x4 {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ptr));
  };

  // Issue the loads of one tile.  K and V are read the same way: LPT lanes
  // cover one whole token row (256 B for bf16, d = 128), TPI rows per
  // instruction -- full-row accesses stream markedly faster from HBM than
  // the 64 B-per-row pattern of the MFMA operand layout.  One address per
  // token serves both.  r: where this lane's token (lane & 31) lives.
  // Full verify tiles (every tile of a unit but its last): the TPI tokens of
  // load n are tokens v0 + n*TPI .. of one sequence -- and, with pages of at
  // least TPI tokens, of one page, whose id lane n*TPI holds -- so the row
  // group's address is wave-uniform and each lane adds a fixed 32-bit offset
  // (its row within the group, its 16 B chunk within the row).  The loads
  // then need no per-lane address arithmetic.
  const bool fast_verify =
      !IDX && p.mode == MD_MODE_VERIFY && (!PAGED || (1 << p.page_shift) >= SH::TPI);
  const uint32_t lane_off = static_cast<uint32_t>(
      (lane / SH::LPT) * p.s_tok * SH::ES + (lane % SH::LPT) * 16);
  auto load_tile_full = [&](TileRegs& T, int v0, TokRef r) {
    T.ok = (1u << SH::NV) - 1u;
    T.tok = r.tok;
    for (int n = 0; n < SH::NV; ++n) {
      int64_t base;  // element offset of token v0 + n*TPI in kv head hk (uniform)
      if constexpr (PAGED) {
        const int pid = __builtin_amdgcn_readlane(r.pid, n * SH::TPI);
        const bool pg_ok = pid >= 0 && pid < p.num_pages;
        base = pg_ok ? static_cast<int64_t>(pid) * p.s_blk +
                           static_cast<int64_t>((v0 + n * SH::TPI) & pmask) * p.s_tok + head_off
                     : 0;  // a page outside the pool: element 0, in bounds
        if (!pg_ok) T.ok &= ~(1u << n);
      } else {
        base = static_cast<int64_t>(b) * p.s_blk + static_cast<int64_t>(v0 + n * SH::TPI) * p.s_tok +
               head_off;
      }
      T.k[n] = ld16(kbase + base * SH::ES + lane_off);
      T.v[n] = ld16(vbase + base * SH::ES + lane_off);
    }
  };

  auto load_tile = [&](TileRegs& T, int tile, TokRef r) {
    const int v0 = u.v_begin + tile * kTile;
    const bool live = tile < n_tiles;
    if (fast_verify && live && v0 + kTile <= u.v_end) {
      load_tile_full(T, v0, r);
      return;
    }
    T.ok = 0;
    T.tok = r.tok;
    for (int n = 0; n < SH::NV; ++n) {
      const int tt = n * SH::TPI + lane / SH::LPT;
      const int vt = v0 + tt;
      const int pid = PAGED ? __shfl(r.pid, tt) : 0;
      int t;
      bool ok;
      if constexpr (IDX) {
        t = __shfl(r.tok, tt);
        ok = t >= 0;
      } else {
        t = real_token(u, vt);
        ok = live && vt < u.v_end;
      }
      const int64_t off = tok_offset(t, pid, ok) * SH::ES + (lane % SH::LPT) * 16;
      T.k[n] = ld16(kbase + off);
      T.v[n] = ld16(vbase + off);
      T.ok |= static_cast<uint32_t>(ok) << n;
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

  unsigned char* kt_lds = lds + wave * SH::WTILE;
  unsigned char* vt_lds = kt_lds + SH::KTILE;

  // One tile: K and V rows to LDS, after which the tile's registers are
  // refilled with tile `tile + P*wph` (so P tiles stay in flight through
  // the compute below); then S^T = K Q^T, the online softmax and
  // O^T += V^T P^T, all operands read back from LDS.
  // Per-unit facts for the mask fast path: the smallest and largest query
  // positions of the unit's real rows.
  const int pos_min = u.S - L;
  const int pos_max = u.S - 1;
  constexpr float kLazy = 8.f;  // log2 headroom before the running max must move

  auto process = [&](TileRegs& T, int tile, TokRef& ref_slot) {
    const int v0 = u.v_begin + tile * kTile;
    const int tok_cur = T.tok;
    // Does any key of this tile need masking for any real row?  (Uniform.)
    const bool full = v0 + kTile <= u.v_end;
    bool needs_mask = true;
    if constexpr (IDX) {
      // Listed prompt positions precede every query; only the speculated
      // tokens and unusable entries need the mask.
      needs_mask = !full || v0 + kTile > u.seg0 || __any(tok_cur < 0);
    } else if (full && !(v0 < u.seg0 && v0 + kTile > u.seg0)) {
      const int t0 = real_token(u, v0), t1 = t0 + kTile - 1;
      needs_mask = t1 > pos_min;
      if (p.mode == MD_MODE_DRAFT)
        needs_mask = needs_mask || !(t1 < p.n_sink || t0 >= pos_max - p.window + 1);
    }

    // Stage the K and V rows in this wave's LDS tiles (row tt, 16 B chunk
    // lane%LPT); V rows of tokens that are not real are written as zeros.
    for (int n = 0; n < SH::NV; ++n) {
      const int tt = n * SH::TPI + lane / SH::LPT;
      u32x4 x = T.v[n];
      if (needs_mask) x = ((T.ok >> n) & 1u) ? x : u32x4{0, 0, 0, 0};
      *reinterpret_cast<u32x4*>(kt_lds + tt * SH::KROW + (lane % SH::LPT) * 16) = T.k[n];
      *reinterpret_cast<u32x4*>(vt_lds + tt * SH::VROW + (lane % SH::LPT) * 16) = x;
    }

    // The tile's registers are free: refill them P tiles ahead.  Page ids
    // run P tiles further ahead still, so waiting for one never waits on a
    // K/V load that is not already needed.
    {
      const int ahead = tile + P * wph;
      const TokRef far = load_ref(ahead + P * wph);
      load_tile(T, ahead, ref_slot);
      ref_slot = far;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // S^T = K Q^T.  A operand from LDS: lane = token (l16) of block tb,
    // channel chunk grp of block cb.
    f32x4 sacc[NT][2];
    for (int tb = 0; tb < 2; ++tb) {
      for (int rt = 0; rt < NT; ++rt) sacc[rt][tb] = f32x4{0.f, 0.f, 0.f, 0.f};
      const unsigned char* krow = kt_lds + (tb * 16 + l16) * SH::KROW + grp * 16;
      for (int cb = 0; cb < SH::KCB; ++cb) {
        const u32x4 kk = *reinterpret_cast<const u32x4*>(krow + cb * 64);
        for (int rt = 0; rt < NT; ++rt) {
          const u32x4 qq = qreg[rt][cb];
          if constexpr (BF16) {
            sacc[rt][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, kk), __builtin_bit_cast(bf16x8, qq), sacc[rt][tb], 0, 0, 0);
          } else {
            for (int j = 0; j < 4; ++j)
              sacc[rt][tb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __uint_as_float(kk[j]), __uint_as_float(qq[j]), sacc[rt][tb], 0, 0, 0);
          }
        }
      }
    }

    // Scale into the log2 domain; mask only where some key is not visible.
    float x[NT][2][4];
    if (!needs_mask) {
      for (int rt = 0; rt < NT; ++rt)
        for (int tb = 0; tb < 2; ++tb)
          for (int e = 0; e < 4; ++e) x[rt][tb][e] = sacc[rt][tb][e] * p.scale_log2;
    } else {
      for (int tb = 0; tb < 2; ++tb)
        for (int e = 0; e < 4; ++e) {
          const int vt = v0 + tb * 16 + grp * 4 + e;
          int t;
          bool tv;
          if constexpr (IDX) {
            t = __shfl(tok_cur, tb * 16 + grp * 4 + e);
            tv = t >= 0;
          } else {
            t = real_token(u, vt);
            tv = vt < u.v_end;
          }
          for (int rt = 0; rt < NT; ++rt) {
            const int pos = row_pos[rt];
            bool vis = tv && t <= pos;
            if (!IDX && p.mode == MD_MODE_DRAFT)
              vis = vis && (t < p.n_sink || t >= pos - p.window + 1);
            x[rt][tb][e] = vis ? sacc[rt][tb][e] * p.scale_log2 : -INFINITY;
          }
        }
    }

    // Online softmax per row (lane l16 + 16*grp all hold row l16).  The
    // running max is moved only when some row's tile max exceeds it by more
    // than kLazy, so most tiles skip the rescale; until then P <= 2^kLazy.
    u32x4 pb[NT];        // bf16 P^T B operand (8 slots)
    float pf[NT][2][4];  // fp32 P for the fp32 path
    for (int rt = 0; rt < NT; ++rt) {
      float mx = fmaxf(fmaxf(fmaxf(x[rt][0][0], x[rt][0][1]), fmaxf(x[rt][0][2], x[rt][0][3])),
                       fmaxf(fmaxf(x[rt][1][0], x[rt][1][1]), fmaxf(x[rt][1][2], x[rt][1][3])));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      if (__any(mx > m_run[rt] + kLazy)) {
        const float m_new = fmaxf(m_run[rt], mx);
        const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run[rt] - m_new);
        m_run[rt] = m_new;
        l_run[rt] *= alpha;
        for (int c = 0; c < SH::CB16; ++c) acc[rt][c] *= alpha;
      }
      const float m_use = m_run[rt] == -INFINITY ? 0.f : m_run[rt];
      float pv[8];
      for (int tb = 0; tb < 2; ++tb)
        for (int e = 0; e < 4; ++e) pv[tb * 4 + e] = fast_exp2(x[rt][tb][e] - m_use);
      if constexpr (BF16) {
        const u32x4 h = u32x4{pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                              pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
        pb[rt] = h;
        // Normalise by exactly what multiplies V (the rounded P).
        float psum = 0.f;
        for (int j = 0; j < 4; ++j)
          psum += __uint_as_float(h[j] << 16) + __uint_as_float(h[j] & 0xffff0000u);
        l_run[rt] += psum;
      } else {
        float psum = 0.f;
        for (int tb = 0; tb < 2; ++tb)
          for (int e = 0; e < 4; ++e) {
            pf[rt][tb][e] = pv[tb * 4 + e];
            psum += pv[tb * 4 + e];
          }
        l_run[rt] += psum;
      }
    }

    // O^T += V^T P^T.  A operand: lane = channel (l16) of block c, slots of
    // group grp = tokens {4grp..4grp+3, 16+4grp..16+4grp+3} as in the scores.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int c = 0; c < SH::CB16; ++c) {
      if constexpr (BF16) {
        // Transposed LDS reads: in each 16-lane group, lane k supplies row
        // (4*grp + k/4) and channels c*16 + 4*(k%4) .. +3, and lane i gets
        // channel c*16 + i of those 4 rows -- tokens 4grp..4grp+3, then the
        // same 16 tokens later for slots 4..7.
        const unsigned char* src = vt_lds + (4 * grp + (l16 >> 2)) * SH::VROW +
                                   (c * 16 + 4 * (l16 & 3)) * 2;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(src));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(src + 16 * SH::VROW));
        const bf16x8 va = __builtin_bit_cast(
            bf16x8, u32x4{__builtin_bit_cast(u32x2, lo).x, __builtin_bit_cast(u32x2, lo).y,
                          __builtin_bit_cast(u32x2, hi).x, __builtin_bit_cast(u32x2, hi).y});
        for (int rt = 0; rt < NT; ++rt)
          acc[rt][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              va, __builtin_bit_cast(bf16x8, pb[rt]), acc[rt][c], 0, 0, 0);
      } else {
        const unsigned char* src = vt_lds + (c * 16 + l16) * 4;
        for (int tb = 0; tb < 2; ++tb)
          for (int j = 0; j < 4; ++j) {
            float va = *reinterpret_cast<const float*>(src + (tb * 16 + grp * 4 + j) * SH::VROW);
            for (int rt = 0; rt < NT; ++rt)
              acc[rt][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(va, pf[rt][tb][j], acc[rt][c], 0,
                                                                0, 0);
          }
      }
    }
    // The next tile overwrites this wave's LDS tile: keep the reads first.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  if (p.err)
    check_contract<PAGED, IDX>(p, u, b, BAL ? (lt0 == 0 ? 0 : 1) : chunk, hk0 == 0, wslot == 0,
                               idxrow, lane);

  // Prologue: this wave's first P tiles in flight; the token locations of
  // the P tiles after them.
  TileRegs ring[P];
  TokRef ref_ring[P];
  {
    TokRef ref0[P];
    for (int s = 0; s < P; ++s) ref0[s] = load_ref(wslot + s * wph);
    for (int s = 0; s < P; ++s) ref_ring[s] = load_ref(wslot + (s + P) * wph);
    for (int s = 0; s < P; ++s) load_tile(ring[s], wslot + s * wph, ref0[s]);
  }
  // Every ring slot is processed unconditionally (a tile past the chunk is
  // fully masked: it leaves m, l and O unchanged), so no slot becomes a
  // conditionally-updated loop-carried value that would force a full wait.
  for (int base = wslot; base < n_tiles; base += P * wph) {
#pragma unroll
    for (int s = 0; s < P; ++s) process(ring[s], base + s * wph, ref_ring[s]);
    if (p.stamps != nullptr && base == wslot) stamp(1);
  }
  stamp(2);

  // ---- row sums: add the 4 lanes that share a row
  for (int rt = 0; rt < NT; ++rt) {
    l_run[rt] += __shfl_xor(l_run[rt], 16);
    l_run[rt] += __shfl_xor(l_run[rt], 32);
  }

  // ---- merge the waves of each unit (LDS reused after the loop): wave w
  // holds unit hk0 + w % hp, so unit hs's waves are j * hp + hs, j < wph.
  // One round for every row tile: each wave leaves its running max and sum
  // and its unnormalised O^T in LDS, and after one barrier each thread sums
  // the waves of its (row, 8 channels) in a fixed order, weighting wave w by
  // 2^(m_w - M) / L with M the row's max and L = sum_w l_w 2^(m_w - M).
  __syncthreads();  // every wave is done with its LDS tiles
  float* mo = reinterpret_cast<float*>(lds);
  float* sm_m = reinterpret_cast<float*>(lds + kMergeO);
  float* sm_l = sm_m + W * ROWS;
  if (grp == 0) {
    for (int rt = 0; rt < NT; ++rt) {
      sm_m[wave * ROWS + rt * 16 + l16] = m_run[rt];
      sm_l[wave * ROWS + rt * 16 + l16] = l_run[rt];
    }
  }
  // Wave w's O^T rows (lane: row l16, channels c*16+4grp..+3) of each row tile.
  for (int rt = 0; rt < NT; ++rt)
    for (int c = 0; c < SH::CB16; ++c)
      *reinterpret_cast<f32x4*>(mo + ((wave * NT + rt) * 16 + l16) * MROW + c * 16 + grp * 4) =
          acc[rt][c];
  __syncthreads();

  const bool direct = BAL ? bal_whole : p.n_chunks == 1;
  const int tid = threadIdx.x;
  // Partial results: chunk k of a split plan at row k * n_rows + row_g; piece
  // k of a cut balanced group -- the piece of workgroup w0 + k, its
  // workgroups being w0 .. w1 -- in that workgroup's slot, 2w for its range's
  // first piece (every piece but possibly w0's) and 2w + 1 for its last,
  // rows hs * R + r.
  const int bal_w0 = BAL ? bal_owner(bc.g0, bc.NW, bc.TT) : 0;
  const int bal_w1 = BAL ? bal_owner(bc.g0 + bc.gt - 1, bc.NW, bc.TT) : 0;
  // w0's piece is the first of its range when the range starts with the group.
  const int bal_w0_last =
      BAL ? static_cast<int>(static_cast<int64_t>(bal_w0) * bc.TT / bc.NW != bc.g0) : 0;
  const int n_parts = BAL ? bal_w1 - bal_w0 + 1 : p.n_chunks;
  const int my_part = BAL ? static_cast<int>(blockIdx.x) - bal_w0 : chunk;
  auto part_row = [&](int k, int hs, int r, int64_t row_g) -> int64_t {
    return BAL ? (static_cast<int64_t>(2 * (bal_w0 + k) + (k == 0 ? bal_w0_last : 0)) * hp + hs) *
                         p.R + r
               : static_cast<int64_t>(k) * p.n_rows + row_g;
  };
  // Final O (8 channels from c0 of row row_g, in the input dtype) and lse.
  auto store_out = [&](int64_t row_g, int c0, const float* o8, float lse) {
    if constexpr (BF16) {
      *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(p.o) + row_g * D + c0) =
          u32x4{pack_bf16x2(o8[0], o8[1]), pack_bf16x2(o8[2], o8[3]),
                pack_bf16x2(o8[4], o8[5]), pack_bf16x2(o8[6], o8[7])};
    } else {
      float* op = static_cast<float*>(p.o) + row_g * D + c0;
      *reinterpret_cast<f32x4*>(op) = f32x4{o8[0], o8[1], o8[2], o8[3]};
      *reinterpret_cast<f32x4*>(op + 4) = f32x4{o8[4], o8[5], o8[6], o8[7]};
    }
    if (p.lse && c0 == 0) p.lse[row_g] = lse;
  };
  constexpr int kGroupsPerRow = D / 8;
  const int items_per_unit = p.R * kGroupsPerRow;  // (row, 8 channels)
  for (int item = tid; item < hp * items_per_unit; item += W * 64) {
    const int hs = item / items_per_unit;
    const int r = (item % items_per_unit) / kGroupsPerRow;
    const int c0 = (item % kGroupsPerRow) * 8;
    const int rt = r >> 4, rr = r & 15;
    float M = -INFINITY;
    for (int jw = 0; jw < wph; ++jw) M = fmaxf(M, sm_m[(jw * hp + hs) * ROWS + r]);
    float wgt[W];
    float Lt = 0.f;
    for (int jw = 0; jw < wph; ++jw) {
      const float mw = sm_m[(jw * hp + hs) * ROWS + r];
      wgt[jw] = mw == -INFINITY ? 0.f : fast_exp2(mw - M);
      Lt += sm_l[(jw * hp + hs) * ROWS + r] * wgt[jw];
    }
    const float inv = Lt > 0.f ? 1.f / Lt : 0.f;
    float o8[8];
    for (int j = 0; j < 8; ++j) o8[j] = 0.f;
    for (int jw = 0; jw < wph; ++jw) {
      const float f = wgt[jw] * inv;
      const float* src = mo + (((jw * hp + hs) * NT + rt) * 16 + rr) * MROW + c0;
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(src);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(src + 4);
      for (int j = 0; j < 4; ++j) {
        o8[j] += f * x0[j];
        o8[4 + j] += f * x1[j];
      }
    }
    const int i = r / p.G, h = (hk0 + hs) * p.G + r % p.G;
    const int64_t row_g = (static_cast<int64_t>(b) * L + i) * p.Hq + h;
    const float lse = (Lt > 0.f) ? (M + fast_log2(Lt)) * 0.69314718055994530942f : -INFINITY;
    if (direct) {
      store_out(row_g, c0, o8, lse);
    } else {
      const int64_t prow = part_row(my_part, hs, r, row_g);
      float* op = p.part_o + prow * D + c0;
      *reinterpret_cast<f32x4*>(op) = f32x4{o8[0], o8[1], o8[2], o8[3]};
      *reinterpret_cast<f32x4*>(op + 4) = f32x4{o8[4], o8[5], o8[6], o8[7]};
      if (c0 == 0) p.part_lse[prow] = lse;
    }
  }

  // ---- split range: the last workgroup of the head group to finish merges
  // the chunks' partials by log-sum-exp (the split-KV identity), so no
  // second launch is needed.  Every chunk's workgroup arrives once (an empty
  // chunk with lse = -inf), so the group's n_chunks-th arrival sees every
  // partial.  The counter carries the call's 48-bit tag above its 16-bit
  // arrival count: a value from any other call (or uninitialised memory)
  // counts as zero arrivals, so the workspace needs no clearing; the last
  // arrival resets it to 0.
  if (!direct && (BAL || !p.merge_launch)) {
    // Every wave waits until its partial stores are performed at the L2
    // (vmcnt 0), the barrier lines the waves up, and one device-scope release
    // fence (an L2 write-back on gfx950) then publishes them all before the
    // arrival.  One fence per workgroup instead of one per wave: device-scope
    // fences serialise in the L2, and four per workgroup at the end of a
    // launch cost more than the separate merge launch they replace.
    MD_PARTIAL_WAVE_DONE();
    __syncthreads();
    int* is_last = reinterpret_cast<int*>(lds);
    if (tid == 0) {
      MD_PARTIAL_RELEASE();
      unsigned long long* ctr = p.counters + group;
      unsigned long long cur = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      unsigned long long next;
      do {
        const unsigned long long seen = (cur >> 16) == p.tag ? (cur & 0xffffull) : 0ull;
        next = (p.tag << 16) | (seen + 1);
      } while (!__hip_atomic_compare_exchange_weak(ctr, &cur, next, __ATOMIC_RELAXED,
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      const int last = (next & 0xffffull) == static_cast<unsigned long long>(n_parts);
      if (last) __hip_atomic_store(ctr, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (last) MD_PARTIAL_ACQUIRE();  // the other chunks' partials, as their workgroups left them
      *is_last = last;
    }
    __syncthreads();
    if (*is_last) {
      constexpr float kLog2e = 1.44269504088896340736f;
      constexpr float kLn2 = 0.69314718055994530942f;
      const int items_per_unit = p.R * kGroupsPerRow;
      for (int item = tid; item < hp * items_per_unit; item += W * 64) {
        const int hs = item / items_per_unit;
        const int r = (item % items_per_unit) / kGroupsPerRow;
        const int c0 = (item % kGroupsPerRow) * 8;
        const int i = r / p.G, h = (hk0 + hs) * p.G + r % p.G;
        const int64_t row_g = (static_cast<int64_t>(b) * L + i) * p.Hq + h;
        float mx = -INFINITY;
        for (int k = 0; k < n_parts; ++k) mx = fmaxf(mx, p.part_lse[part_row(k, hs, r, row_g)]);
        float o8[8];
        for (int j = 0; j < 8; ++j) o8[j] = 0.f;
        float lse = -INFINITY;
        if (mx != -INFINITY) {
          float tot = 0.f;
          for (int k = 0; k < n_parts; ++k) {
            const float l = p.part_lse[part_row(k, hs, r, row_g)];
            if (l != -INFINITY) tot += fast_exp2((l - mx) * kLog2e);
          }
          lse = mx + fast_log2(tot) * kLn2;
          for (int k = 0; k < n_parts; ++k) {
            const int64_t prow = part_row(k, hs, r, row_g);
            const float l = p.part_lse[prow];
            if (l == -INFINITY) continue;  // an empty chunk: its O is not read
            const float wk = fast_exp2((l - lse) * kLog2e);
            const float* op = p.part_o + prow * D + c0;
            const f32x4 x0 = *reinterpret_cast<const f32x4*>(op);
            const f32x4 x1 = *reinterpret_cast<const f32x4*>(op + 4);
            for (int j = 0; j < 4; ++j) {
              o8[j] += wk * x0[j];
              o8[4 + j] += wk * x1[j];
            }
          }
        }
        store_out(row_g, c0, o8, lse);
      }
    }
  }
  if constexpr (!BAL) {
    break;
  } else {
    if (!bal_next(p, gps, bc)) break;
  }
  __syncthreads();  // the next piece reuses the LDS
  }  // pieces
  stamp(3);
}

// ---------------------------------------------------------------------------
// Host-side dispatch over the compiled instances.

template <int D, bool BF16, int NT, bool IDX, int P, int OCC, bool BAL = false, int W = kWaves>
static hipError_t launch_p(const AttnParams& p, bool paged, int64_t n_blocks, hipStream_t s) {
  dim3 grid(static_cast<uint32_t>(n_blocks)), block(W * 64);
  if (paged)
    hipLaunchKernelGGL((attn_partial_kernel<D, BF16, NT, true, IDX, P, OCC, BAL, W>), grid, block,
                       0, s, p);
  else
    hipLaunchKernelGGL((attn_partial_kernel<D, BF16, NT, false, IDX, P, OCC, BAL, W>), grid, block,
                       0, s, p);
  return hipGetLastError();
}

// Instances: tiles in flight per wave (depth) x waves per SIMD (occupancy).
// Two waves per SIMD fit the register file with one tile in flight and up to
// two row tiles; a second tile in flight is built for the bf16 range modes
// with up to three row tiles (MD_PREFETCH_DEPTH); everything else runs one
// tile, one wave per SIMD.
template <int D, bool BF16, int NT, bool IDX>
static hipError_t launch_nt(const AttnParams& p, bool paged, int depth, int occ,
                            int64_t n_blocks, hipStream_t s) {
  // The balanced verify: one tile in flight, the verify's default waves per
  // SIMD (two for one row tile of bf16, else one).  Compiled only where its
  // piece loop fits the registers without spilling (bf16 up to three row
  // tiles, fp32 up to two); the planner never chooses it elsewhere.
  if constexpr (!IDX && NT <= kBalMaxNT(BF16)) {
    if (p.bal) {
      (void)depth;
      (void)occ;
      return launch_p<D, BF16, NT, IDX, 1, (BF16 && NT == 1) ? 2 : 1, true>(p, paged, n_blocks, s);
    }
  } else {
    if (p.bal) return hipErrorInvalidValue;
  }
  if constexpr (BF16 && NT <= 2 && !IDX) {
    // Eight waves in one workgroup, two per SIMD (the registers of up to two
    // row tiles allow it, 248 at two): each takes half as many of the unit's
    // tiles.  Their merge buffers fill 140 KB of LDS at two row tiles.
    if (p.waves == kWavesWide)
      return launch_p<D, BF16, NT, IDX, 1, 2, false, kWavesWide>(p, paged, n_blocks, s);
  }
  if (p.waves != kWaves) return hipErrorInvalidValue;
  if constexpr (BF16) {
    if constexpr (!IDX && NT <= 3)
      if (depth >= 2) return launch_p<D, BF16, NT, IDX, 2, 1>(p, paged, n_blocks, s);
    if constexpr (NT <= 2)
      if (occ >= 2) return launch_p<D, BF16, NT, IDX, 1, 2>(p, paged, n_blocks, s);
    return launch_p<D, BF16, NT, IDX, 1, 1>(p, paged, n_blocks, s);
  } else {
    (void)depth;  // fp32 serves small problems: one tile in flight
    (void)occ;
    return launch_p<D, BF16, NT, IDX, 1, 1>(p, paged, n_blocks, s);
  }
}

template <int D, bool BF16, bool IDX>
static hipError_t launch_d(const AttnParams& p, int NT, bool paged, int depth, int occ,
                           int64_t n_blocks, hipStream_t s) {
  switch (NT) {
    case 1: return launch_nt<D, BF16, 1, IDX>(p, paged, depth, occ, n_blocks, s);
    case 2: return launch_nt<D, BF16, 2, IDX>(p, paged, depth, occ, n_blocks, s);
    case 3: return launch_nt<D, BF16, 3, IDX>(p, paged, depth, occ, n_blocks, s);
    case 4: return launch_nt<D, BF16, 4, IDX>(p, paged, depth, occ, n_blocks, s);
  }
  return hipErrorInvalidValue;
}

template <bool IDX>
static hipError_t launch_i(const AttnParams& p, int head_dim, bool bf16, int NT, bool paged,
                           int depth, int occ, int64_t n_blocks, hipStream_t s) {
  if (head_dim == 128)
    return bf16 ? launch_d<128, true, IDX>(p, NT, paged, depth, occ, n_blocks, s)
                : launch_d<128, false, IDX>(p, NT, paged, depth, occ, n_blocks, s);
  return bf16 ? launch_d<64, true, IDX>(p, NT, paged, depth, occ, n_blocks, s)
              : launch_d<64, false, IDX>(p, NT, paged, depth, occ, n_blocks, s);
}

hipError_t launch_attn_partial(const AttnParams& p, int head_dim, bool bf16, int NT, bool paged,
                               int depth, int occ, int64_t n_blocks, hipStream_t s) {
  if (n_blocks <= 0) return hipSuccess;
  if (p.mode == MD_MODE_DRAFT_INDEXED)
    return launch_i<true>(p, head_dim, bf16, NT, paged, depth, occ, n_blocks, s);
  return launch_i<false>(p, head_dim, bf16, NT, paged, depth, occ, n_blocks, s);
}

}  // namespace md
