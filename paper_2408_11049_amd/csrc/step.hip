// step.hip -- the kernels on either side of verification in one speculative
// step (Sec. 3.1; greedy decoding, Sec. 5.1):
//
//   kv_append       writes the gamma+1 verified tokens' K/V rows into the
//                   cache (contiguous or paged), 16 bytes per thread;
//   argmax_partial  first pass of greedy acceptance: each workgroup reduces
//                   one chunk of one logits row to (largest value, first
//                   index);
//   accept          second pass, one wave per sequence: reduces each row's
//                   chunks to the target token, then walks the rows in order
//                   to count the leading matching drafts and emit the bonus;
//   kv_commit       C' = C + a + 1, recording the kept positions in the
//                   rolling ring of a listed draft cache;
//   streaming_list  the sink-plus-window lists a StreamingLLM-style draft
//                   cache starts from at prefill;
//   kv_gather       a static selection's listed rows copied, once, into a
//                   draft cache of its own.
//
// All of them are bound by HBM or by launch latency; none is a contraction.
#include <hip/hip_runtime.h>
#include <limits.h>

#include "kernels.h"

namespace md {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- append --

template <bool PAGED>
__global__ void __launch_bounds__(256) kv_append_kernel(const AppendParams p) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t item = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; item < p.n_items;
       item += stride) {
    int64_t r = item;
    const int c = static_cast<int>(r % p.row_vecs);
    r /= p.row_vecs;
    const int hk = static_cast<int>(r % p.Hkv);
    r /= p.Hkv;
    const int i = static_cast<int>(r % p.n_new);
    r /= p.n_new;
    const int b = static_cast<int>(r % p.B);
    const bool is_v = r >= p.B;

    const int32_t base = p.pos0[b];
    if (!is_v && i == 0 && hk == 0 && c == 0 && p.lens_out) p.lens_out[b] = base + p.n_new;
    const int64_t j = static_cast<int64_t>(base) + i;
    if (j < 0) continue;
    int64_t blk, tok;
    if (PAGED) {
      const int64_t pg = j >> p.page_shift;
      if (pg >= p.max_pages) continue;
      blk = p.page_table[static_cast<int64_t>(b) * p.max_pages + pg];
      if (blk < 0 || blk >= p.num_pages) continue;
      tok = j & ((int64_t{1} << p.page_shift) - 1);
    } else {
      if (j >= p.capacity) continue;
      blk = b;
      tok = j;
    }
    const int64_t src = ((static_cast<int64_t>(b) * p.n_new + i) * p.Hkv + hk) * p.row_vecs + c;
    const int64_t dst = (blk * p.s_blk + tok * p.s_tok + hk * p.s_head) * p.esize + c * 16;
    const uint4 val = reinterpret_cast<const uint4*>(is_v ? p.v_new : p.k_new)[src];
    *reinterpret_cast<uint4*>((is_v ? p.v : p.k) + dst) = val;
  }
}

hipError_t launch_kv_append(const AppendParams& p, bool paged, hipStream_t s) {
  const int64_t want = (p.n_items + 255) / 256;
  const uint32_t blocks = static_cast<uint32_t>(want < (1 << 20) ? want : (1 << 20));
  if (paged)
    hipLaunchKernelGGL(kv_append_kernel<true>, dim3(blocks), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(kv_append_kernel<false>, dim3(blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------- gather --

// Where logical position j of sequence b lives in cache c: (block, token),
// or false when it lies outside the cache (past the capacity or the table,
// or on a page outside the pool).
template <bool PAGED>
__device__ __forceinline__ bool cache_row(const CacheView& c, int b, int64_t j, int64_t& blk,
                                          int64_t& tok) {
  if (j < 0) return false;
  if (PAGED) {
    const int64_t pg = j >> c.page_shift;
    if (pg >= c.max_pages) return false;
    blk = c.page_table[static_cast<int64_t>(b) * c.max_pages + pg];
    if (blk < 0 || blk >= c.num_pages) return false;
    tok = j & ((int64_t{1} << c.page_shift) - 1);
  } else {
    if (j >= c.capacity) return false;
    blk = b;
    tok = j;
  }
  return true;
}

// One 16-byte vector per item, items ordered (vector, kv head, list slot,
// sequence, K/V): the kv heads of one destination row are written side by
// side (one whole token row), each read from its own listed source row.
template <bool SRC_PAGED, bool DST_PAGED>
__global__ void __launch_bounds__(256) kv_gather_kernel(const GatherParams p) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t item = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; item < p.n_items;
       item += stride) {
    int64_t r = item;
    const int c = static_cast<int>(r % p.row_vecs);
    r /= p.row_vecs;
    const int hk = static_cast<int>(r % p.Hkv);
    r /= p.Hkv;
    const int j = static_cast<int>(r % p.idx_stride);
    r /= p.idx_stride;
    const int b = static_cast<int>(r % p.B);
    const bool is_v = r >= p.B;

    const int n = min(max(p.idx_len[b], 0), p.idx_stride);
    if (!is_v && j == 0 && hk == 0 && c == 0 && p.dst_lens) p.dst_lens[b] = n;
    if (j >= n) continue;
    int64_t dblk, dtok;
    if (!cache_row<DST_PAGED>(p.dst, b, j, dblk, dtok)) continue;
    const int32_t pos = p.idx[(static_cast<int64_t>(b) * p.Hkv + hk) * p.idx_stride + j];
    u32x4 val = u32x4{0u, 0u, 0u, 0u};
    int64_t sblk, stok;
    if (pos >= 0 && pos < p.src_lens[b] && cache_row<SRC_PAGED>(p.src, b, pos, sblk, stok)) {
      const int64_t so =
          (sblk * p.src.s_blk + stok * p.src.s_tok + hk * p.src.s_head) * p.esize + c * 16;
      val = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4*>((is_v ? p.src.v : p.src.k) + so));
    }
    const int64_t dof =
        (dblk * p.dst.s_blk + dtok * p.dst.s_tok + hk * p.dst.s_head) * p.esize + c * 16;
    *reinterpret_cast<u32x4*>((is_v ? p.dst.v : p.dst.k) + dof) = val;
  }
}

// The same copy when row_vecs and Hkv are powers of two: grid (items of one
// sequence, sequences, K/V), each sequence's items in the order above, so an
// item's (list slot, kv head, vector) are shifts and masks of its index
// rather than 64-bit divisions, and only the listed rows are visited.  Each
// thread takes four items per iteration and issues their list reads, then
// their row loads, then their stores, so the dependent reads of one item
// (list entry, page id, row) overlap those of the others (measured 22%
// faster than one item at a time).
template <bool SRC_PAGED, bool DST_PAGED>
__global__ void __launch_bounds__(256) kv_gather_pow2_kernel(const GatherParams p) {
  constexpr int U = 4;  // items per thread and iteration: their loads overlap
  const bool is_v = blockIdx.z != 0;
  const int vshift = p.vec_shift, hshift = p.head_shift;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int b = blockIdx.y; b < p.B; b += gridDim.y) {
    const int n = min(max(p.idx_len[b], 0), p.idx_stride);
    if (!is_v && blockIdx.x == 0 && threadIdx.x == 0 && p.dst_lens) p.dst_lens[b] = n;
    const int64_t live = static_cast<int64_t>(n) << (hshift + vshift);
    const int src_len = p.src_lens[b];
    const int32_t* idxb = p.idx + static_cast<int64_t>(b) * p.Hkv * p.idx_stride;
    for (int64_t item0 = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; item0 < live;
         item0 += U * stride) {
      int c[U], hk[U], j[U];
      int32_t pos[U];
      bool in[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t item = item0 + u * stride;
        in[u] = item < live;
        const int64_t it = in[u] ? item : 0;
        c[u] = static_cast<int>(it & ((int64_t{1} << vshift) - 1));
        const int64_t r = it >> vshift;
        hk[u] = static_cast<int>(r & ((int64_t{1} << hshift) - 1));
        j[u] = static_cast<int>(r >> hshift);
        pos[u] = idxb[static_cast<int64_t>(hk[u]) * p.idx_stride + j[u]];
      }
      u32x4 val[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        val[u] = u32x4{0u, 0u, 0u, 0u};
        int64_t sblk, stok;
        if (in[u] && pos[u] >= 0 && pos[u] < src_len &&
            cache_row<SRC_PAGED>(p.src, b, pos[u], sblk, stok)) {
          const int64_t so =
              (sblk * p.src.s_blk + stok * p.src.s_tok + hk[u] * p.src.s_head) * p.esize + c[u] * 16;
          val[u] = __builtin_nontemporal_load(
              reinterpret_cast<const u32x4*>((is_v ? p.src.v : p.src.k) + so));
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        int64_t dblk, dtok;
        if (!in[u] || !cache_row<DST_PAGED>(p.dst, b, j[u], dblk, dtok)) continue;
        const int64_t dof =
            (dblk * p.dst.s_blk + dtok * p.dst.s_tok + hk[u] * p.dst.s_head) * p.esize + c[u] * 16;
        *reinterpret_cast<u32x4*>((is_v ? p.dst.v : p.dst.k) + dof) = val[u];
      }
    }
  }
}

hipError_t launch_kv_gather(const GatherParams& p, bool src_paged, bool dst_paged, hipStream_t s) {
  if (p.vec_shift >= 0 && p.head_shift >= 0) {
    const int64_t per_seq = static_cast<int64_t>(p.idx_stride) << (p.vec_shift + p.head_shift);
    const int64_t want = (per_seq + 4 * 256 - 1) / (4 * 256);  // four items per thread
    const dim3 g(static_cast<uint32_t>(want < 4096 ? want : 4096),
                 static_cast<uint32_t>(p.B < 65535 ? p.B : 65535), 2),
        blk(256);
    if (src_paged && dst_paged)
      hipLaunchKernelGGL((kv_gather_pow2_kernel<true, true>), g, blk, 0, s, p);
    else if (src_paged)
      hipLaunchKernelGGL((kv_gather_pow2_kernel<true, false>), g, blk, 0, s, p);
    else if (dst_paged)
      hipLaunchKernelGGL((kv_gather_pow2_kernel<false, true>), g, blk, 0, s, p);
    else
      hipLaunchKernelGGL((kv_gather_pow2_kernel<false, false>), g, blk, 0, s, p);
    return hipGetLastError();
  }
  const int64_t want = (p.n_items + 255) / 256;
  const uint32_t blocks = static_cast<uint32_t>(want < (1 << 20) ? want : (1 << 20));
  const dim3 g(blocks), blk(256);
  if (src_paged && dst_paged)
    hipLaunchKernelGGL((kv_gather_kernel<true, true>), g, blk, 0, s, p);
  else if (src_paged)
    hipLaunchKernelGGL((kv_gather_kernel<true, false>), g, blk, 0, s, p);
  else if (dst_paged)
    hipLaunchKernelGGL((kv_gather_kernel<false, true>), g, blk, 0, s, p);
  else
    hipLaunchKernelGGL((kv_gather_kernel<false, false>), g, blk, 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------- accept --

// Keep the larger value; between equal values the smaller index.  NaN never
// reaches here (it is read as -inf), so the order is total and any reduction
// order gives the same (value, index).
__device__ __forceinline__ void take(float& bv, int& bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

__device__ __forceinline__ void wave_take(float& bv, int& bi) {
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(bv, off);
    const int oi = __shfl_xor(bi, off);
    take(bv, bi, ov, oi);
  }
}

__device__ __forceinline__ float logit_value(float v) { return v != v ? -INFINITY : v; }

template <bool BF16>
__device__ __forceinline__ float load_logit(const void* base, int64_t e) {
  if (BF16) {
    const uint32_t u = static_cast<const uint16_t*>(base)[e];
    return logit_value(__uint_as_float(u << 16));
  }
  return logit_value(static_cast<const float*>(base)[e]);
}

// Element e of a 16-byte vector of logits, widened to fp32 (bf16 holds two
// per dword, the lower address in the low half).
template <bool BF16>
__device__ __forceinline__ float vec_elem(const u32x4& x, int e) {
  if (BF16) {
    const uint32_t w = x[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  return __uint_as_float(x[e]);
}

// Largest element of the vector; fmaxf drops NaN operands, so NaN counts as
// nothing (an all-NaN vector gives NaN, which loses every comparison).
template <bool BF16>
__device__ __forceinline__ float vec_max(const u32x4& x) {
  constexpr int EPV = BF16 ? 8 : 4;
  float m = vec_elem<BF16>(x, 0);
#pragma unroll
  for (int e = 1; e < EPV; ++e) m = fmaxf(m, vec_elem<BF16>(x, e));
  return m;
}

// One workgroup per (row, chunk); block = row * n_chunks + chunk.  VEC: the
// rows start 16-byte aligned (vocab a multiple of the vector width), so each
// thread streams 16-byte vectors, four in flight.  A thread keeps only the
// first vector holding its largest value (vectors arrive in increasing index
// order, so a strict comparison keeps the earliest) and resolves the index
// inside that vector once at the end: a few VALU operations per element.
template <bool BF16, bool VEC>
__global__ void __launch_bounds__(256) argmax_partial_kernel(const AcceptParams p) {
  constexpr int EPV = BF16 ? 8 : 4;  // elements per 16-byte vector
  constexpr int U = 4;
  const int64_t row = blockIdx.x / p.n_chunks;
  const int chunk = static_cast<int>(blockIdx.x % p.n_chunks);
  const int c0 = chunk * p.chunk_len;
  const int c1 = min(p.vocab, c0 + p.chunk_len);
  const int tid = threadIdx.x;
  float bv = -INFINITY;
  int bi = INT_MAX;
  const unsigned char* rowp =
      static_cast<const unsigned char*>(p.logits) + row * p.vocab * (BF16 ? 2 : 4);
  if (VEC) {
    const u32x4* vp = reinterpret_cast<const u32x4*>(rowp);
    const int v0 = c0 / EPV, v1 = c1 / EPV;
    int bvec = -1;
    u32x4 bw = {0u, 0u, 0u, 0u};
    for (int v = v0 + tid; v < v1; v += 256 * U) {
      u32x4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int vv = v + u * 256;
        // Out-of-range lanes re-read the first vector of the chunk (in bounds)
        // and are discarded below.
        x[u] = __builtin_nontemporal_load(vp + (vv < v1 ? vv : v0));
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int vv = v + u * 256;
        const float m = vec_max<BF16>(x[u]);
        if (vv < v1 && m > bv) {
          bv = m;
          bvec = vv;
          bw = x[u];
        }
      }
    }
    if (bvec >= 0) {
#pragma unroll
      for (int e = EPV - 1; e >= 0; --e)
        if (vec_elem<BF16>(bw, e) == bv) bi = bvec * EPV + e;
    }
  } else {
    for (int e = c0 + tid; e < c1; e += 256) take(bv, bi, load_logit<BF16>(rowp, e), e);
  }
  wave_take(bv, bi);
  __shared__ float sv[4];
  __shared__ int si[4];
  const int wave = tid >> 6;
  if ((tid & 63) == 0) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < 4; ++w) take(bv, bi, sv[w], si[w]);
    p.part_val[blockIdx.x] = bv;
    p.part_idx[blockIdx.x] = bi;
  }
}

// One wave per sequence.  Every chunk partial of the sequence's rows and its
// drafts are staged in LDS in one round of loads; lane i then reduces row i
// to its target token, and a ballot finds the first mismatching draft.
__global__ void __launch_bounds__(64) accept_kernel(const AcceptParams p) {
  __shared__ float s_val[kAcceptMaxPartialsPerSeq];
  __shared__ int s_idx[kAcceptMaxPartialsPerSeq];
  __shared__ int s_tgt[kAcceptMaxRowsPerSeq];
  __shared__ int s_draft[kAcceptMaxRowsPerSeq];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int L = p.L, nc = p.n_chunks, n = L * nc;
  const int64_t base = static_cast<int64_t>(b) * n;  // rows of b are contiguous
  for (int t = lane; t < n; t += 64) {
    s_val[t] = p.part_val[base + t];
    s_idx[t] = p.part_idx[base + t];
  }
  for (int i = lane; i < L - 1; i += 64) s_draft[i] = p.draft[static_cast<int64_t>(b) * (L - 1) + i];
  __syncthreads();
  for (int i = lane; i < L; i += 64) {
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int c = 0; c < nc; ++c) take(bv, bi, s_val[i * nc + c], s_idx[i * nc + c]);
    const int t = bi == INT_MAX ? 0 : bi;
    s_tgt[i] = t;
    if (p.target) p.target[static_cast<int64_t>(b) * L + i] = t;
  }
  __syncthreads();
  // a = the first i < L - 1 whose draft differs from the target (L - 1 if none).
  int a = L - 1;
  for (int i0 = 0; i0 < L - 1; i0 += 64) {
    const int i = i0 + lane;
    const unsigned long long miss = __ballot(i < L - 1 && s_draft[i] != s_tgt[i]);
    if (miss) {
      a = i0 + __ffsll(static_cast<long long>(miss)) - 1;
      break;
    }
  }
  for (int i = lane; i < L; i += 64)
    p.tokens[static_cast<int64_t>(b) * L + i] = i < a ? s_draft[i] : (i == a ? s_tgt[a] : -1);
  if (lane == 0) p.accepted[b] = a;
}

hipError_t launch_greedy_accept(const AcceptParams& p, bool bf16, bool vec, hipStream_t s) {
  const uint32_t blocks = static_cast<uint32_t>(static_cast<int64_t>(p.B) * p.L * p.n_chunks);
  if (bf16) {
    if (vec)
      hipLaunchKernelGGL((argmax_partial_kernel<true, true>), dim3(blocks), dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((argmax_partial_kernel<true, false>), dim3(blocks), dim3(256), 0, s, p);
  } else {
    if (vec)
      hipLaunchKernelGGL((argmax_partial_kernel<false, true>), dim3(blocks), dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((argmax_partial_kernel<false, false>), dim3(blocks), dim3(256), 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_kernel, dim3(p.B), dim3(64), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------- commit --

// One wave per sequence.  Every lane reads lens[b] before the barrier; lane 0
// writes the new length after it.
__global__ void __launch_bounds__(64)
kv_commit_kernel(int q_len, int32_t* __restrict__ lens, const int32_t* __restrict__ accepted,
                 int Hkv, int32_t* __restrict__ idx, int idx_stride, int ring_start,
                 int ring_len) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int C = lens[b];
  int a = accepted[b];
  a = a < 0 ? 0 : (a > q_len - 1 ? q_len - 1 : a);
  if (idx) {
    // Only the last ring_len kept positions survive in the ring.
    const int n_keep = a + 1 < ring_len ? a + 1 : ring_len;
    const int first = C + a + 1 - n_keep;
    for (int t = lane; t < n_keep * Hkv; t += 64) {
      const int j = first + t / Hkv;
      const int hk = t % Hkv;
      if (j < 0) continue;
      idx[(static_cast<int64_t>(b) * Hkv + hk) * idx_stride + ring_start + j % ring_len] = j;
    }
  }
  __syncthreads();
  if (lane == 0) lens[b] = C + a + 1;
}

hipError_t launch_kv_commit(int B, int q_len, int32_t* lens, const int32_t* accepted, int Hkv,
                            int32_t* idx, int idx_stride, int ring_start, int ring_len,
                            hipStream_t s) {
  hipLaunchKernelGGL(kv_commit_kernel, dim3(B), dim3(64), 0, s, q_len, lens, accepted, Hkv, idx,
                     idx_stride, ring_start, ring_len);
  return hipGetLastError();
}

// --------------------------------------------------------- streaming list --

// One workgroup per (sequence, kv head) list.  Ring slot n_sink + r holds the
// one position j in [max(n_sink, C - window), C) with j % window == r.
__global__ void __launch_bounds__(256)
streaming_list_kernel(int Hkv, const int32_t* __restrict__ prompt_lens, int n_sink, int window,
                      int32_t* __restrict__ idx, int32_t* __restrict__ idx_len) {
  const int64_t list = blockIdx.x;
  const int b = static_cast<int>(list / Hkv);
  const int C = prompt_lens[b];
  const int n = n_sink + window;
  const int lo = C - window > n_sink ? C - window : n_sink;
  for (int s = threadIdx.x; s < n; s += 256) {
    int val = -1;
    if (s < n_sink) {
      val = s < C ? s : -1;
    } else if (lo < C) {
      const int r = s - n_sink;
      const int j = lo + ((r - lo % window) % window + window) % window;
      val = j < C ? j : -1;
    }
    idx[list * n + s] = val;
  }
  if (list % Hkv == 0 && threadIdx.x == 0) idx_len[b] = n;
}

hipError_t launch_streaming_list(int B, int Hkv, const int32_t* prompt_lens, int n_sink,
                                 int window, int32_t* idx, int32_t* idx_len, hipStream_t s) {
  hipLaunchKernelGGL(streaming_list_kernel, dim3(static_cast<uint32_t>(int64_t{B} * Hkv)),
                     dim3(256), 0, s, Hkv, prompt_lens, n_sink, window, idx, idx_len);
  return hipGetLastError();
}

}  // namespace md
