// Device helpers shared by the gfx950 kernels: MFMA operand wrappers,
// workgroup numbering, score keys, workgroup scans and the threshold search.
#pragma once

#include <hip/hip_ext.h>

#include "ckv_internal.h"

namespace ckv {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kKpWaves = kKpThreads / 64;  // waves per K-pass workgroup

template <int DT>
struct Elt {
  static constexpr int bytes = DT == 2 ? 4 : 2;
};

// acc += A * B over one 16-byte operand chunk per lane. Lane l holds row
// (l % 32) of A and column (l % 32) of B; the two lane halves hold the two
// halves of the chunk's contraction slice, identically for A and B, so the
// result is the dot product over the chunk whatever order the hardware sums in.
template <int DT>
__device__ __forceinline__ f32x16 mfma_chunk(uint4 a, uint4 b, f32x16 c);

template <>
__device__ __forceinline__ f32x16 mfma_chunk<0>(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x16 mfma_chunk<1>(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x16 mfma_chunk<2>(uint4 a, uint4 b, f32x16 c) {
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Row of the 32x32 MFMA result held in accumulator v by lane half h.
__device__ __forceinline__ int acc_row(int v, int h) { return 8 * (v >> 2) + 4 * h + (v & 3); }

// Workgroups are dispatched round-robin over the 8 XCDs; renumber them so that
// each XCD works on one contiguous range of tiles (neighbouring tiles share
// halo rows and K lines in that XCD's L2).
__device__ __forceinline__ int xcd_remap(int b, int n) {
  const int xcd = b & 7, i = b >> 3, per = n >> 3, rem = n & 7;
  return xcd * per + (xcd < rem ? xcd : rem) + i;
}

// Order-preserving integer key of a score (scores are >= 0; -0 ranks as +0).
__device__ __forceinline__ uint32_t score_key(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? 0u : u;
}

// Exclusive prefix sum over the workgroup; also returns the total.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* wsum, uint32_t& total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wv] = x;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    const uint32_t sv = wsum[i];
    before += i < wv ? sv : 0u;
    tot += sv;
  }
  __syncthreads();
  total = tot;
  return before + x - v;
}

// Find, in a histogram of NBINS bins read through `get(bin)`, the bin holding
// the need-th largest key (bins ordered by value, need >= 1 and <= total).
// Each thread owns NBINS/kThreads consecutive bins, walked from the top; the
// reads are unrolled so that they are all in flight at once. Returns (bin,
// keys in higher bins, keys in the bin) in res[0..2] for every thread of the
// workgroup.
template <int NBINS, typename Get>
__device__ __forceinline__ void find_bin(uint32_t need, Get get, uint32_t* wsum, uint32_t* res) {
  static_assert(NBINS % kThreads == 0, "bins per thread");
  constexpr int kPer = NBINS / kThreads;
  const int top = NBINS - 1 - kPer * (int)threadIdx.x;
  uint32_t c[kPer];
  uint32_t local = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    c[i] = get(top - i);
    local += c[i];
  }
  uint32_t tot;
  const uint32_t above = block_excl_scan<kThreads>(local, wsum, tot);
  if (above < need && need <= above + local) {
    uint32_t run = above;
    bool found = false;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (!found && need <= run + c[i]) {
        res[0] = (uint32_t)(top - i);
        res[1] = run;
        res[2] = c[i];
        found = true;
      }
      run += c[i];
    }
  }
  __syncthreads();
}

// Launch kernel(a) on stream st, with its start and end times recorded into
// tm's events when they are given.
template <typename K>
__host__ hipError_t launch(K kernel, int grid, int block, hipStream_t st, const Timing& tm,
                           const LayerArgs& a) {
  if (tm.start || tm.stop)
    hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(block), 0, st, tm.start, tm.stop, 0, a);
  else
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(block), 0, st, a);
  return hipGetLastError();
}

}  // namespace dev
}  // namespace ckv
