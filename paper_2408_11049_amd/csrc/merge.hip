// merge.hip -- log-sum-exp merge of attention partials computed over
// disjoint key sets: the second phase of the split-KV decomposition (the
// Flash-Decoding identity the paper cites in Sec. 2), and the public
// md_merge_lse.
//
// One wave per row.  The part count is small (tens), so each lane first
// scans the lse values for the row maximum and the normaliser, then the wave
// walks the parts in order, each lane owning d/64 channels of the row.  Parts
// with lse = -inf are skipped without reading their O.  When every part's O is
// readable (the library's own split plans, which write every part) and there
// are at most kRegParts parts, each lane instead issues the loads of all lse
// values and of its channels of every part at once and combines them from
// registers: one memory round trip instead of two dependent ones.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace md {

typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t merge_f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

constexpr int kRegParts = 8;

template <int D, bool OUT_BF16, bool REG>
__global__ void __launch_bounds__(256)
merge_lse_kernel(int n_parts, int64_t n_rows, const float* __restrict__ o_parts,
                 const float* __restrict__ lse_parts, void* __restrict__ o,
                 float* __restrict__ lse) {
  constexpr float kLog2e = 1.44269504088896340736f;
  constexpr float kLn2 = 0.69314718055994530942f;
  constexpr int CPL = D / 64;  // channels per lane
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;

  if constexpr (REG) {
    // n_parts <= kRegParts, every part's O readable: all loads first.
    float lv[kRegParts];
    float xo[kRegParts][CPL];
    for (int k = 0; k < kRegParts; ++k) {
      if (k < n_parts) {
        lv[k] = lse_parts[k * n_rows + row];
        const float* src = o_parts + (k * n_rows + row) * D + lane * CPL;
        if constexpr (CPL == 2) {
          const f32x2 x = *reinterpret_cast<const f32x2*>(src);
          xo[k][0] = x.x;
          xo[k][1] = x.y;
        } else {
          xo[k][0] = src[0];
        }
      }
    }
    float mx = -INFINITY;
    for (int k = 0; k < kRegParts; ++k)
      if (k < n_parts) mx = fmaxf(mx, lv[k]);
    float acc[CPL];
    for (int j = 0; j < CPL; ++j) acc[j] = 0.f;
    float lse_r = -INFINITY;
    if (mx != -INFINITY) {
      float tot = 0.f;
      for (int k = 0; k < kRegParts; ++k)
        if (k < n_parts && lv[k] != -INFINITY) tot += __builtin_amdgcn_exp2f((lv[k] - mx) * kLog2e);
      lse_r = mx + __builtin_amdgcn_logf(tot) * kLn2;
      for (int k = 0; k < kRegParts; ++k) {
        // An empty part's O is ignored (never multiplied: it may hold NaN).
        if (k >= n_parts || lv[k] == -INFINITY) continue;
        const float w = __builtin_amdgcn_exp2f((lv[k] - lse_r) * kLog2e);
        for (int j = 0; j < CPL; ++j) acc[j] += w * xo[k][j];
      }
    }
    if constexpr (OUT_BF16) {
      uint16_t* dst = static_cast<uint16_t*>(o) + row * D + lane * CPL;
      if constexpr (CPL == 2)
        *reinterpret_cast<uint32_t*>(dst) =
            merge_f32_to_bf16(acc[0]) | (merge_f32_to_bf16(acc[1]) << 16);
      else
        dst[0] = static_cast<uint16_t>(merge_f32_to_bf16(acc[0]));
    } else {
      float* dst = static_cast<float*>(o) + row * D + lane * CPL;
      for (int j = 0; j < CPL; ++j) dst[j] = acc[j];
    }
    if (lse && lane == 0) lse[row] = lse_r;
    return;
  }

  float mx = -INFINITY;
  for (int k = lane; k < n_parts; k += 64) mx = fmaxf(mx, lse_parts[k * n_rows + row]);
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));

  float acc[CPL];
  for (int j = 0; j < CPL; ++j) acc[j] = 0.f;
  float lse_r = -INFINITY;
  if (mx != -INFINITY) {
    float tot = 0.f;
    for (int k = lane; k < n_parts; k += 64) {
      float l = lse_parts[k * n_rows + row];
      if (l != -INFINITY) tot += __builtin_amdgcn_exp2f((l - mx) * kLog2e);
    }
    for (int off = 32; off > 0; off >>= 1) tot += __shfl_xor(tot, off);
    lse_r = mx + __builtin_amdgcn_logf(tot) * kLn2;
    for (int k = 0; k < n_parts; ++k) {
      const float l = lse_parts[k * n_rows + row];
      if (l == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f((l - lse_r) * kLog2e);
      const float* src = o_parts + (k * n_rows + row) * D + lane * CPL;
      if constexpr (CPL == 2) {
        f32x2 x = *reinterpret_cast<const f32x2*>(src);
        acc[0] += w * x.x;
        acc[1] += w * x.y;
      } else {
        acc[0] += w * src[0];
      }
    }
  }
  if constexpr (OUT_BF16) {
    uint16_t* dst = static_cast<uint16_t*>(o) + row * D + lane * CPL;
    if constexpr (CPL == 2)
      *reinterpret_cast<uint32_t*>(dst) = merge_f32_to_bf16(acc[0]) | (merge_f32_to_bf16(acc[1]) << 16);
    else
      dst[0] = static_cast<uint16_t>(merge_f32_to_bf16(acc[0]));
  } else {
    float* dst = static_cast<float*>(o) + row * D + lane * CPL;
    for (int j = 0; j < CPL; ++j) dst[j] = acc[j];
  }
  if (lse && lane == 0) lse[row] = lse_r;
}

template <int D, bool OUT_BF16>
static void launch_d(bool reg, dim3 grid, dim3 block, hipStream_t s, int n_parts, int64_t n_rows,
                     const float* o_parts, const float* lse_parts, void* o, float* lse) {
  if (reg)
    hipLaunchKernelGGL((merge_lse_kernel<D, OUT_BF16, true>), grid, block, 0, s, n_parts, n_rows,
                       o_parts, lse_parts, o, lse);
  else
    hipLaunchKernelGGL((merge_lse_kernel<D, OUT_BF16, false>), grid, block, 0, s, n_parts,
                       n_rows, o_parts, lse_parts, o, lse);
}

hipError_t launch_merge_lse(int n_parts, int64_t n_rows, int head_dim, bool out_bf16,
                            const float* o_parts, const float* lse_parts, void* o, float* lse,
                            hipStream_t s, bool parts_readable) {
  if (n_rows <= 0) return hipSuccess;
  dim3 grid(static_cast<uint32_t>((n_rows + 3) / 4)), block(256);
  const bool reg = parts_readable && n_parts <= kRegParts;
  if (head_dim == 128) {
    if (out_bf16)
      launch_d<128, true>(reg, grid, block, s, n_parts, n_rows, o_parts, lse_parts, o, lse);
    else
      launch_d<128, false>(reg, grid, block, s, n_parts, n_rows, o_parts, lse_parts, o, lse);
  } else {
    if (out_bf16)
      launch_d<64, true>(reg, grid, block, s, n_parts, n_rows, o_parts, lse_parts, o, lse);
    else
      launch_d<64, false>(reg, grid, block, s, n_parts, n_rows, o_parts, lse_parts, o, lse);
  }
  return hipGetLastError();
}

}  // namespace md
