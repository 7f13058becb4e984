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
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Pointers read from memory (argument blocks in device memory, LDS tables)
// are generic, and generic (flat) loads count against the LDS wait counter
// too, so every LDS access would also wait for them. Casting a pointer known
// to address global memory lets the compiler issue global loads instead.
#define CKV_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ const CKV_GLOBAL T* to_global(const T* p) {
  return (const CKV_GLOBAL T*)p;
}
template <class T>
__device__ __forceinline__ CKV_GLOBAL T* to_global(T* p) {
  return (CKV_GLOBAL T*)p;
}

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
// tm's events when they are given. The launch's own status is returned (not
// hipGetLastError, which may hold an earlier error of the caller's).
template <typename K, typename A>
__host__ hipError_t launch(K kernel, dim3 grid, int block, hipStream_t st, const Timing& tm,
                           const A& a) {
  void* args[] = {const_cast<A*>(&a)};
  return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, dim3(block), args, 0, st,
                            tm.start, tm.stop, 0);
}
template <typename K, typename A>
__host__ hipError_t launch(K kernel, int grid, int block, hipStream_t st, const Timing& tm,
                           const A& a) {
  return launch(kernel, dim3(grid), block, st, tm, a);
}

constexpr int kPoolPer = 8;  // consecutive scores pooled per thread

// x[i] = row[o0 - HW + i] for i in [0, 8 + 2*HW); inputs outside [0, Ls)
// read as pad. Aligned 16-byte loads when the window lies inside the row
// (o0 - HW is a multiple of 4 and rows start 16-byte aligned).
template <int HW>
__device__ __forceinline__ void pool_inputs(const float* row_p, int64_t o0, int64_t Ls, float pad,
                                            float* x) {
  const CKV_GLOBAL float* row = to_global(row_p);
  constexpr int NX = kPoolPer + 2 * HW;
  const int64_t lo = o0 - HW;
  if (lo >= 0 && lo + NX <= Ls) {
    const CKV_GLOBAL f32x4* src = (const CKV_GLOBAL f32x4*)(row + lo);
#pragma unroll
    for (int v = 0; v < NX / 4; ++v) {
      const f32x4 t = src[v];
      x[4 * v] = t.x;
      x[4 * v + 1] = t.y;
      x[4 * v + 2] = t.z;
      x[4 * v + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const int64_t j = lo + i;
      x[i] = j >= 0 && j < Ls ? row[j] : pad;
    }
  }
}

constexpr int kCopyBatch = 8;  // 16-byte K and V chunks in flight per thread

// Copy n rows of K and V: source token src(i) -> output row dst(i), for i in
// [0, n). Rows whose source or destination is out of range are skipped. The
// loads of a batch are all issued before its stores.
template <int NT, class Src, class Dst>
__device__ __forceinline__ void copy_rows(const LayerArgs& a, const SeqArgs& sq, int g, int64_t n,
                                          Src src, Dst dst) {
  const int nv = a.d * a.elt / 16;  // 8, 16 or 32 chunks per row
  const int nv_log2 = nv == 8 ? 3 : (nv == 16 ? 4 : 5);
  // native vectors (not HIP's uint4 struct) so the batch stays in registers
  const CKV_GLOBAL char* __restrict__ kb =
      to_global(static_cast<const char*>(sq.k)) + (int64_t)g * sq.kv_sh * a.elt;
  const CKV_GLOBAL char* __restrict__ vb =
      to_global(static_cast<const char*>(sq.v)) + (int64_t)g * sq.kv_sh * a.elt;
  CKV_GLOBAL u32x4* __restrict__ ko = to_global(static_cast<u32x4*>(sq.k_out)) + (int64_t)g * sq.n_ret * nv;
  CKV_GLOBAL u32x4* __restrict__ vo = to_global(static_cast<u32x4*>(sq.v_out)) + (int64_t)g * sq.n_ret * nv;
  const int64_t total = n << nv_log2;
  for (int64_t e0 = 0; e0 < total; e0 += (int64_t)NT * kCopyBatch) {
    u32x4 kr[kCopyBatch], vr[kCopyBatch];
    int64_t to[kCopyBatch];
#pragma unroll
    for (int u = 0; u < kCopyBatch; ++u) {
      const int64_t e = e0 + threadIdx.x + (int64_t)u * NT;
      const int64_t i = e >> nv_log2;
      const int c = (int)(e & (nv - 1));
      const int64_t j = e < total ? src(i) : -1;
      const int64_t p = e < total ? dst(i) : -1;
      const bool ok = j >= 0 && j < sq.L && p >= 0 && p < sq.n_ret;
      to[u] = ok ? (p << nv_log2) + c : -1;
      const int64_t jj = ok ? j : 0;  // row 0 is a valid address for skipped lanes
      kr[u] = ((const CKV_GLOBAL u32x4*)(kb + jj * sq.kv_st * a.elt))[c];
      vr[u] = ((const CKV_GLOBAL u32x4*)(vb + jj * sq.kv_st * a.elt))[c];
    }
#pragma unroll
    for (int u = 0; u < kCopyBatch; ++u) {
      if (to[u] >= 0) {
        ko[to[u]] = kr[u];
        vo[to[u]] = vr[u];
      }
    }
  }
}

// Contiguous run: row src0 + i -> output row dst0 + i.
template <int NT>
__device__ __forceinline__ void copy_run(const LayerArgs& a, const SeqArgs& sq, int g, int64_t dst0,
                                         int64_t src0, int64_t n) {
  copy_rows<NT>(a, sq, g, n, [=](int64_t i) { return src0 + i; }, [=](int64_t i) { return dst0 + i; });
}

// Layer l's argument block of a multi-layer launch.
__device__ __forceinline__ const LayerArgs& layer_args(const MultiArgs& m, int l) {
  return *reinterpret_cast<const LayerArgs*>(m.table + (int64_t)l * m.stride);
}

}  // namespace dev
}  // namespace ckv
