// bench_stream.hip -- streaming-read ceiling of the GPU, measured by bench.py
// beside the eviction path (built into bench_stream.so; not part of libckv).
//
// Each kind sweeps a device buffer once with 16-byte loads per lane and keeps
// nothing but a checksum, so its time is the cost of reading the bytes:
//   kind 0  global_load_dwordx4 into registers (default cache policy),
//   kind 1  the same with nontemporal loads,
//   kind 2  global_load_lds_dwordx4 straight into LDS, the route the K passes
//           take: every wave keeps three 4 KB stages of its own in flight in a
//           private four-slot ring and waits for them with partial vmcnt waits.
// Workgroups take 4 KB-per-wave chunks grid-stride, so consecutive waves read
// consecutive chunks. A copy kernel (bench_stream_copy) gives the rate of an
// even read/write mix, the traffic of kernels that write as much as they read.
#include <hip/hip_runtime.h>
#include <stddef.h>

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kLoads = 4;                    // 16-byte loads per lane per stage
constexpr size_t kChunk = kLoads * 64;       // 16-byte units per wave stage (4 KB)
constexpr unsigned kNever = 0x9E3779B9u;     // checksum value that stores the sum

// s_waitcnt: at most n vector-memory operations of this wave outstanding
// (vmcnt in bits 3:0, expcnt and lgkmcnt at their no-wait maxima).
#define WAIT_VM(n) __builtin_amdgcn_s_waitcnt(0xF70 | (n))

template <int KIND>
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ x,
                                                               size_t n16, unsigned* sink) {
  unsigned s = 0;
  if constexpr (KIND < 2) {
    const size_t stride = (size_t)gridDim.x * kThreads;
    size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
      u32x4 a, b, c, d;
      if constexpr (KIND == 1) {
        a = __builtin_nontemporal_load(x + i);
        b = __builtin_nontemporal_load(x + i + stride);
        c = __builtin_nontemporal_load(x + i + 2 * stride);
        d = __builtin_nontemporal_load(x + i + 3 * stride);
      } else {
        a = x[i];
        b = x[i + stride];
        c = x[i + 2 * stride];
        d = x[i + 3 * stride];
      }
      s ^= a.x ^ b.y ^ c.z ^ d.w;
    }
    for (; i < n16; i += stride) s ^= x[i].x;
  } else {
    __shared__ u32x4 ring[kWaves][4][kLoads * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const size_t n_chunks = n16 / kChunk;  // the host passes whole chunks only
    const size_t step = (size_t)gridDim.x * kWaves;
    size_t next = (size_t)blockIdx.x * kWaves + wave;  // next chunk to issue
    int issued = 0;
    auto issue = [&](size_t c) {
      const u32x4* src = x + c * kChunk + lane;
      u32x4* dst = &ring[wave][issued & 3][0];
#pragma unroll
      for (int k = 0; k < kLoads; ++k) __builtin_amdgcn_global_load_lds(src + k * 64, dst + k * 64, 16, 0, 0);
      ++issued;
    };
    for (int k = 0; k < 3 && next < n_chunks; ++k, next += step) issue(next);
    for (int done = 0; done < issued; ++done) {
      if (next < n_chunks) {
        issue(next);
        next += step;
      }
      // stage `done` has landed once at most the later stages' loads remain
      switch (issued - done - 1) {
        case 3: WAIT_VM(12); break;
        case 2: WAIT_VM(8); break;
        case 1: WAIT_VM(4); break;
        default: WAIT_VM(0); break;
      }
      s ^= ring[wave][done & 3][lane].x;
    }
  }
  if (s == kNever) sink[threadIdx.x] = s;
}

// dst[i] = src[i] for n16 16-byte units, grid-stride, four loads in flight
// per lane before their stores.
__global__ __launch_bounds__(kThreads) void stream_copy_kernel(const u32x4* __restrict__ x,
                                                               u32x4* __restrict__ y, size_t n16) {
  const size_t stride = (size_t)gridDim.x * kThreads;
  size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = x[i], b = x[i + stride], c = x[i + 2 * stride], d = x[i + 3 * stride];
    y[i] = a;
    y[i + stride] = b;
    y[i + 2 * stride] = c;
    y[i + 3 * stride] = d;
  }
  for (; i < n16; i += stride) y[i] = x[i];
}

}  // namespace

// Copy `bytes` bytes from src to dst (distinct, 16-byte aligned, bytes a
// multiple of 16) on `grid` workgroups of 256 threads. Returns a hipError_t
// value (0 on success).
extern "C" int bench_stream_copy(const void* src, void* dst, size_t bytes, int grid, void* stream) {
  if (!src || !dst || bytes % 16 || ((size_t)src & 15) || ((size_t)dst & 15) || grid < 1 ||
      grid > 65536)
    return (int)hipErrorInvalidValue;
  const u32x4* x = static_cast<const u32x4*>(src);
  u32x4* y = static_cast<u32x4*>(dst);
  size_t n16 = bytes / 16;
  void* args[] = {(void*)&x, (void*)&y, (void*)&n16};
  return (int)hipLaunchKernel(reinterpret_cast<const void*>(stream_copy_kernel), dim3(grid),
                              dim3(kThreads), args, 0, static_cast<hipStream_t>(stream));
}

// Read `bytes` bytes at src once with read route `kind` on `grid` workgroups
// of 256 threads. sink: 256 unsigned of device memory, written only when a
// checksum happens to equal a fixed value. bytes must be a multiple of 4096,
// src 16-byte aligned. Returns a hipError_t value (0 on success).
extern "C" int bench_stream_read(const void* src, size_t bytes, unsigned* sink, int grid, int kind,
                                 void* stream) {
  if (!src || !sink || bytes % 4096 || ((size_t)src & 15) || grid < 1 || grid > 65536)
    return (int)hipErrorInvalidValue;
  const u32x4* x = static_cast<const u32x4*>(src);
  size_t n16 = bytes / 16;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  void* args[] = {(void*)&x, (void*)&n16, (void*)&sink};
  const void* fn;
  switch (kind) {
    case 0: fn = reinterpret_cast<const void*>(stream_read_kernel<0>); break;
    case 1: fn = reinterpret_cast<const void*>(stream_read_kernel<1>); break;
    case 2: fn = reinterpret_cast<const void*>(stream_read_kernel<2>); break;
    default: return (int)hipErrorInvalidValue;
  }
  return (int)hipLaunchKernel(fn, dim3(grid), dim3(kThreads), args, 0, st);
}
