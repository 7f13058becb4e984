// gfx950 (MI355X) kernels of CompressKV's layer-error profile (arXiv
// 2508.02401, Sec. 3.4, Eq. 6-8): decode attention of T query tokens over a
// full or a compressed KV cache, and the W_O-projected error ratio of every
// decoding step.
//
// decode_kernel: one workgroup per (KV head g, chunk of the cache). The
//   query rows of the group (its G heads x T tokens, head-major) are split
//   into 32-row blocks; each wave keeps one block in registers and walks the
//   chunk's 32-key blocks (waves sharing a query block take alternate key
//   blocks). Per key block: S^T = K Q^T (keys x rows) with fp32 MFMA, an
//   online max and sum per row, P = exp2(S - m), O += P V with fp32 MFMA.
//   Every wave writes its rows' (max, sum, O) as one partial.
// decode_merge_kernel: per (KV head, row): the partials rescaled to the
//   common max and summed, divided by the sum: out[t][h][:].
// project_kernel: Y = W_O X for the 2T columns X = [A_full | A_comp - A_full]
//   with fp32 MFMA, one workgroup per 32 rows of W_O and 32 columns, then the
//   column sums of Y^2 over its rows as one partial.
// error_kernel: the partials summed per column; ratio_t = sqrt(num_t) /
//   (sqrt(den_t) + eps) and e = sum_t ratio_t.
// Everything accumulates in fp32: the ratios compare two attention outputs
// that may differ in their third digit, which plain bf16 products would
// blur. fp32 inputs use fp32 MFMA (32x32x2); 16-bit inputs use 16-bit MFMA
// with the queries and probabilities split into high and low parts.
#include <math.h>

#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

constexpr int kDecThreads = kDecodeThreads;
constexpr int kDecWaves = kDecThreads / 64;

__device__ __forceinline__ f32x16 mfma_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

template <int DT>
__device__ __forceinline__ float elt_load(const void* base, int64_t i) {
  if constexpr (DT == 0) {
    const uint16_t u = static_cast<const CKV_GLOBAL uint16_t*>(to_global(static_cast<const uint16_t*>(base)))[i];
    return __uint_as_float((uint32_t)u << 16);
  } else if constexpr (DT == 1) {
    return (float)static_cast<const CKV_GLOBAL _Float16*>(to_global(static_cast<const _Float16*>(base)))[i];
  } else {
    return to_global(static_cast<const float*>(base))[i];
  }
}

// The 16 / element-bytes elements of a 16-byte piece, in fp32.
template <int DT>
__device__ __forceinline__ void unpack16(const u32x4 u, float* f) {
  if constexpr (DT == 2) {
    f[0] = __uint_as_float(u.x);
    f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z);
    f[3] = __uint_as_float(u.w);
  } else {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (DT == 0) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
      } else {
        f[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] & 0xFFFFu));
        f[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] >> 16));
      }
    }
  }
}

// EPV = 16 / element-bytes consecutive elements at element offset off, in fp32.
template <int DT>
__device__ __forceinline__ void load_row16(const void* base, int64_t off, float* f) {
  unpack16<DT>(*reinterpret_cast<const CKV_GLOBAL u32x4*>(to_global(static_cast<const char*>(base)) +
                                                          off * Elt<DT>::bytes),
               f);
}

// ---------------------------------------------------------------------------
// Decode attention, partials per (KV head, chunk, wave).
// ---------------------------------------------------------------------------
template <int DT, int D>
__global__ __launch_bounds__(kDecThreads) void decode_kernel_f32(const DecodeBatch B) {
  constexpr int KB = 32;      // keys per block
  constexpr int KS = D + 1;   // LDS row stride: lanes reading one column of 32 rows hit 32 banks
  __shared__ float kl[KB * KS];  // K block [key][d], fp32
  __shared__ float vl[KB * KS];  // V block [key][d], fp32
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // this workgroup's prompt (a uniform scan over at most kMaxDecodeSeqs)
  int si = 0;
  while (si + 1 < B.n && (int)blockIdx.x >= B.blk_off[si + 1]) ++si;
  const DecodeArgs& a = B.s[si];
  const int lb = (int)blockIdx.x - B.blk_off[si];
  const int g = lb / a.n_chunks, chunk = lb - g * a.n_chunks;
  const int G = B.H / B.n_kv;
  const int R = G * a.T;                    // query rows of the group
  const int nqb = (R + 31) >> 5;            // their 32-row blocks (<= kDecWaves)
  const int wpq = kDecWaves / (nqb == 3 ? 4 : nqb);  // waves per query block
  const int qb = wave / wpq, sub = wave - qb * wpq;
  const bool active = qb < nqb;
  const int64_t j0 = (int64_t)chunk * a.chunk;
  const int64_t j1 = j0 + a.chunk < a.n ? j0 + a.chunk : a.n;
  const int nkb = (int)((j1 - j0 + KB - 1) / KB);

  // this lane's query row (column of S^T and row of O): r = head-in-group * T + t
  const int r = qb * 32 + l32;
  const bool row_ok = active && r < R;
  float q[D / 2];  // lane half h holds elements 2i + h
  {
    const int hl = row_ok ? r / a.T : 0, t = row_ok ? r - (r / a.T) * a.T : 0;
    const int64_t qoff = (int64_t)t * a.q_st + (int64_t)(g * G + hl) * a.q_sh;
#pragma unroll
    for (int i = 0; i < D / 2; ++i) q[i] = row_ok ? elt_load<DT>(a.q, qoff + 2 * i + h) : 0.f;
  }
  f32x16 o[D / 32];
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb) o[nb] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float alpha = B.alpha;
  const int64_t kv_base = (int64_t)g * a.kv_sh;

  // K and V blocks of 32 keys go through LDS in fp32; each thread loads NLD
  // 16-byte pieces of both per block, and the next block's loads are issued
  // before the current block is reduced, so they overlap its MFMA work
  constexpr int EPV = 16 / Elt<DT>::bytes;              // elements per 16-byte load
  constexpr int NLD = KB * D / EPV / kDecThreads;       // loads per thread per block
  static_assert(NLD >= 1 && KB * D / EPV % kDecThreads == 0, "block loads");
  u32x4 kr[NLD], vr[NLD];
  auto issue = [&](int kb) {
    const int64_t t0 = j0 + (int64_t)kb * KB;
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int e = tid + u * kDecThreads;
      const int key = e / (D / EPV), c = (e - key * (D / EPV)) * EPV;
      const int64_t tok = t0 + key < j1 ? t0 + key : j1 - 1;  // past the chunk: a valid row
      const int64_t off = (kv_base + tok * a.kv_st + c) * Elt<DT>::bytes;
      // each cache row is read once: non-temporal loads
      kr[u] = __builtin_nontemporal_load(reinterpret_cast<const CKV_GLOBAL u32x4*>(to_global(static_cast<const char*>(a.k)) + off));
      vr[u] = __builtin_nontemporal_load(reinterpret_cast<const CKV_GLOBAL u32x4*>(to_global(static_cast<const char*>(a.v)) + off));
    }
  };
  issue(0);
  for (int kb = 0; kb < nkb; ++kb) {
    const int64_t t0 = j0 + (int64_t)kb * KB;
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int e = tid + u * kDecThreads;
      const int key = e / (D / EPV), c = (e - key * (D / EPV)) * EPV;
      const bool in = t0 + key < j1;  // keys past the chunk hold 0
      float kf[EPV], vf[EPV];
      unpack16<DT>(kr[u], kf);
      unpack16<DT>(vr[u], vf);
#pragma unroll
      for (int i = 0; i < EPV; ++i) {
        kl[key * KS + c + i] = in ? kf[i] : 0.f;
        vl[key * KS + c + i] = in ? vf[i] : 0.f;
      }
    }
    __syncthreads();
    if (kb + 1 < nkb) issue(kb + 1);
    if (active && (kb % wpq) == sub) {
      // S^T[key][row]: lane (row l32, half h) receives keys acc_row(v, h)
      f32x16 s = f32x16{};
#pragma unroll
      for (int i = 0; i < D / 2; ++i) s = mfma_f32(kl[l32 * KS + 2 * i + h], q[i], s);
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = acc_row(v, h);
        s[v] = t0 + key < j1 ? s[v] * alpha : -INFINITY;  // exp2 units
        mx = fmaxf(mx, s[v]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32));  // the row's max over both lane halves
      const float m_new = fmaxf(m_run, mx);
      const float resc = m_run == -INFINITY ? 0.f : exp2f(m_run - m_new);
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s[v] = m_new == -INFINITY ? 0.f : exp2f(s[v] - m_new);
        psum += s[v];
      }
      l_run = l_run * resc + psum;
      m_run = m_new;
#pragma unroll
      for (int nb = 0; nb < D / 32; ++nb) {
        // O^T[n][row] += V^T P^T: lane half h supplies key acc_row(v, h), the
        // key of its P value s[v]; the result's column is the lane's own row,
        // so the rescale is the lane's own
        f32x16 acc = o[nb] * resc;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          acc = mfma_f32(vl[acc_row(v, h) * KS + nb * 32 + l32], s[v], acc);
        o[nb] = acc;
      }
    }
    __syncthreads();
  }
  if (!active) return;
  // the partial of this wave: (max, sum) per row, and O rows
  l_run += __shfl_xor(l_run, 32);
  const int slot = chunk * wpq + sub;
  float* part = a.part + (((int64_t)g * a.n_slots + slot) * a.prow + qb * 32) * (D + 2);
  if (h == 0) {
    part[l32 * (D + 2) + D] = m_run;
    part[l32 * (D + 2) + D + 1] = l_run;
  }
  // o[nb][v]: O^T[nb*32 + acc_row(v, h)][row l32]
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) part[l32 * (D + 2) + nb * 32 + acc_row(v, h)] = o[nb][v];
}

// 16-bit inputs (bf16, f16): the same decode with 16-bit MFMA (32x32x16) at
// fp32-level accuracy. K and V are exact in the MFMA type; the queries and
// the probabilities are split into a high part (rounded to the type) and a
// low part (the rounded remainder), and each product is the sum of two MFMAs,
// which leaves a relative error near 2^-16 (bf16) or 2^-22 (f16) instead of
// 2^-8 or 2^-11.
template <int DT>
__device__ __forceinline__ uint32_t to16(float x) {
  if constexpr (DT == 0) {  // round to nearest even
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  } else {
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x);
  }
}
template <int DT>
__device__ __forceinline__ float from16(uint32_t b) {
  if constexpr (DT == 0) return __uint_as_float(b << 16);
  else return (float)__builtin_bit_cast(_Float16, (uint16_t)b);
}
// 8 values -> the high and low 16-bit parts, packed two per word.
template <int DT>
__device__ __forceinline__ void split8(const float* x, uint4& hi, uint4& lo) {
  uint32_t hb[8], lb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    hb[i] = to16<DT>(x[i]);
    lb[i] = to16<DT>(x[i] - from16<DT>(hb[i]));
  }
  hi = make_uint4(hb[0] | hb[1] << 16, hb[2] | hb[3] << 16, hb[4] | hb[5] << 16, hb[6] | hb[7] << 16);
  lo = make_uint4(lb[0] | lb[1] << 16, lb[2] | lb[3] << 16, lb[4] | lb[5] << 16, lb[6] | lb[7] << 16);
}

// Blocks of 64 keys keep the staging registers small enough for two
// workgroups per CU (two waves per SIMD): one workgroup reduces a block while
// the other's loads are in flight.
template <int DT, int D>
__global__ __launch_bounds__(kDecThreads) __attribute__((amdgpu_waves_per_eu(2)))
void decode_kernel_16(const DecodeBatch B) {
  constexpr int SB = 32;              // keys per MFMA tile (a sub-block)
  constexpr int NSB = 2;              // sub-blocks staged per block
  constexpr int KB = SB * NSB;        // keys per block
  constexpr int NC = D / 16;          // 16-element contraction chunks of a row
  constexpr int KROW = D * 2 + 16;    // K and V row bytes in LDS, padded by one 16-byte chunk
  __shared__ __align__(16) unsigned char kl[KB * KROW];  // K block [key][d], raw 16-bit
  __shared__ __align__(16) unsigned char vl[KB * KROW];  // V block [key][d], raw 16-bit
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // this workgroup's prompt (a uniform scan over at most kMaxDecodeSeqs)
  int si = 0;
  while (si + 1 < B.n && (int)blockIdx.x >= B.blk_off[si + 1]) ++si;
  const DecodeArgs& a = B.s[si];
  const int lb = (int)blockIdx.x - B.blk_off[si];
  const int g = lb / a.n_chunks, chunk = lb - g * a.n_chunks;
  const int G = B.H / B.n_kv;
  const int R = G * a.T;
  const int nqb = (R + 31) >> 5;
  const int wpq = kDecWaves / (nqb == 3 ? 4 : nqb);
  const int qb = wave / wpq, sub = wave - qb * wpq;
  const bool active = qb < nqb;
  const int64_t j0 = (int64_t)chunk * a.chunk;
  const int64_t j1 = j0 + a.chunk < a.n ? j0 + a.chunk : a.n;
  const int nkb = (int)((j1 - j0 + KB - 1) / KB);

  // query row r = head-in-group * T + t; lane half h holds elements
  // 16c + 8h .. 16c + 8h + 7 of it, split into high and low parts
  const int r = qb * 32 + l32;
  const bool row_ok = active && r < R;
  uint4 qh[NC], ql[NC];
  {
    const int hl = row_ok ? r / a.T : 0, t = row_ok ? r - (r / a.T) * a.T : 0;
    const int64_t qoff = (int64_t)t * a.q_st + (int64_t)(g * G + hl) * a.q_sh;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float x[8];
      if (row_ok) load_row16<DT>(a.q, qoff + 16 * c + 8 * h, x);
      else
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = 0.f;
      split8<DT>(x, qh[c], ql[c]);
    }
  }
  f32x16 o[D / 32];
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb) o[nb] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float alpha = B.alpha;
  const int64_t kv_base = (int64_t)g * a.kv_sh;

  // every block of KB keys is staged by all threads (16-byte loads, the next
  // block's issued before the current one is reduced); the waves of a query
  // block split its sub-blocks, so every wave works on every block
  constexpr int NLD = KB * D / 8 / kDecThreads;  // 16-byte loads per thread per block
  static_assert(NLD >= 1 && KB * D / 8 % kDecThreads == 0, "block loads");
  u32x4 kr[NLD], vr[NLD];
  auto issue = [&](int kb) {
    const int64_t t0 = j0 + (int64_t)kb * KB;
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int e = tid + u * kDecThreads;
      const int key = e / (D / 8), c = (e - key * (D / 8)) * 8;
      const int64_t tok = t0 + key < j1 ? t0 + key : j1 - 1;  // past the chunk: a valid row
      const int64_t off = (kv_base + tok * a.kv_st + c) * 2;
      // each cache row is read once: non-temporal loads
      kr[u] = __builtin_nontemporal_load(reinterpret_cast<const CKV_GLOBAL u32x4*>(to_global(static_cast<const char*>(a.k)) + off));
      vr[u] = __builtin_nontemporal_load(reinterpret_cast<const CKV_GLOBAL u32x4*>(to_global(static_cast<const char*>(a.v)) + off));
    }
  };
  issue(0);
  for (int kb = 0; kb < nkb; ++kb) {
    const int64_t t0 = j0 + (int64_t)kb * KB;
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int e = tid + u * kDecThreads;
      const int key = e / (D / 8), c = (e - key * (D / 8)) * 8;
      const bool in = t0 + key < j1;  // keys past the chunk hold 0
      const u32x4 kz = in ? kr[u] : u32x4{0u, 0u, 0u, 0u};
      const u32x4 vz = in ? vr[u] : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(kl + key * KROW + c * 2) = kz;
      *reinterpret_cast<u32x4*>(vl + key * KROW + c * 2) = vz;
    }
    __syncthreads();
    if (kb + 1 < nkb) issue(kb + 1);
    for (int sb = sub; active && sb < NSB; sb += wpq) {
      const int64_t ts = t0 + sb * SB;  // first key of the sub-block
      if (ts >= j1) break;
      // S^T[key][row] = K Q^T with Q = high + low parts; lane (row l32, half
      // h) receives keys acc_row(v, h) of the sub-block
      f32x16 s = f32x16{};
      const unsigned char* krow = kl + (sb * SB + l32) * KROW;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const uint4 kc = *reinterpret_cast<const uint4*>(krow + (16 * c + 8 * h) * 2);
        s = mfma_chunk<DT>(kc, qh[c], s);
        s = mfma_chunk<DT>(kc, ql[c], s);
      }
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s[v] = ts + acc_row(v, h) < j1 ? s[v] * alpha : -INFINITY;  // exp2 units
        mx = fmaxf(mx, s[v]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float resc = m_run == -INFINITY ? 0.f : fast_exp2(m_run - m_new);
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s[v] = fast_exp2(s[v] - m_new);
        psum += s[v];
      }
      l_run = l_run * resc + psum;
      m_run = m_new;
      // P^T operands: MFMA step m takes this lane's keys acc_row(8m .. 8m+7, h)
      // = 16m + 4h + (0..3) and 16m + 8 + 4h + (0..3), in that order
      uint4 ph[2], pl[2];
      {
        float p0[8], p1[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          p0[i] = s[i];
          p1[i] = s[8 + i];
        }
        split8<DT>(p0, ph[0], pl[0]);
        split8<DT>(p1, ph[1], pl[1]);
      }
#pragma unroll
      for (int nb = 0; nb < D / 32; ++nb) {
        // O^T[n][row] += V^T P^T: lane (n = nb*32 + l32, half h) supplies V of
        // the same 8 keys, gathered from the row-major tile (the lanes of a
        // half read 32 consecutive elements of one key row)
        f32x16 acc = o[nb] * resc;
        const unsigned char* vcol = vl + (sb * SB) * KROW + (nb * 32 + l32) * 2;
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          uint32_t e[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int key = 16 * m + 8 * (j >> 2) + 4 * h + (j & 3);
            e[j] = *reinterpret_cast<const uint16_t*>(vcol + key * KROW);
          }
          const uint4 va = make_uint4(e[0] | e[1] << 16, e[2] | e[3] << 16, e[4] | e[5] << 16,
                                      e[6] | e[7] << 16);
          acc = mfma_chunk<DT>(va, ph[m], acc);
          acc = mfma_chunk<DT>(va, pl[m], acc);
        }
        o[nb] = acc;
      }
    }
    __syncthreads();
  }
  if (!active) return;
  l_run += __shfl_xor(l_run, 32);
  const int slot = chunk * wpq + sub;
  float* part = a.part + (((int64_t)g * a.n_slots + slot) * a.prow + qb * 32) * (D + 2);
  if (h == 0) {
    part[l32 * (D + 2) + D] = m_run;
    part[l32 * (D + 2) + D + 1] = l_run;
  }
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) part[l32 * (D + 2) + nb * 32 + acc_row(v, h)] = o[nb][v];
}

// out[t][h][c] from the partials of every slot, one thread per (row, c).
template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_merge_kernel(const DecodeBatch B) {
  int si = 0;
  while (si + 1 < B.n && (int)blockIdx.x >= B.mrg_off[si + 1]) ++si;
  const DecodeArgs& a = B.s[si];
  const int G = B.H / B.n_kv;
  const int R = G * a.T;
  const int64_t e = (int64_t)((int)blockIdx.x - B.mrg_off[si]) * kDecThreads + threadIdx.x;
  const int64_t per_g = (int64_t)R * D;
  if (e >= per_g * B.n_kv) return;
  const int g = (int)(e / per_g);
  const int rc = (int)(e - (int64_t)g * per_g);
  const int r = rc / D, c = rc - r * D;
  const int nqb = (R + 31) >> 5;
  const int wpq = kDecWaves / (nqb == 3 ? 4 : nqb);
  const int n_used = a.n_chunks * wpq;
  const CKV_GLOBAL float* base = to_global(a.part) + ((int64_t)g * a.n_slots * a.prow + r) * (D + 2);
  const int64_t stride = (int64_t)a.prow * (D + 2);
  // one pass over the slots, U at a time, with the running maximum: the sums
  // are rescaled whenever a slot's maximum exceeds it
  constexpr int U = 16;  // slots loaded at once
  float m = -INFINITY, l = 0.f, acc = 0.f;
  for (int s0 = 0; s0 < n_used; s0 += U) {
    float ms[U], ls[U], os[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool in = s0 + u < n_used;
      const CKV_GLOBAL float* p = base + (in ? s0 + u : 0) * stride;
      ms[u] = in ? p[D] : -INFINITY;
      ls[u] = p[D + 1];
      os[u] = p[c];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (ms[u] == -INFINITY) continue;  // a slot that saw no key, or past the last
      if (ms[u] > m) {
        const float f = exp2f(m - ms[u]);  // 0 while nothing has been added
        l *= f;
        acc *= f;
        m = ms[u];
      }
      const float f = exp2f(ms[u] - m);
      l += ls[u] * f;
      acc += os[u] * f;
    }
  }
  const int hl = r / a.T, t = r - hl * a.T;
  a.out[((int64_t)t * B.H + g * G + hl) * D + c] = acc / l;
}

// ---------------------------------------------------------------------------
// Projection and error ratios.
// ---------------------------------------------------------------------------
// Workgroup (row block rb, column block cb, K range ks): the 32 x 32 tile of
// Y = W X over the ks-th of n_split K ranges, that range split over the
// workgroup's waves, the waves' sums added in LDS in a fixed order and the
// tile written to part_y. K is taken 16 at a time: lane half h holds
// k0 + 8h .. k0 + 8h + 7 of its W row (one 16-byte load for 2-byte weights)
// and of its X column, and MFMA m pairs k0 + m with k0 + 8 + m. K is a
// multiple of 16 (H * d with d in {64, 128}).
constexpr int kProjThreads = 256;
constexpr int kProjWaves = kProjThreads / 64;

template <int DT>
__global__ __launch_bounds__(kProjThreads) void project_kernel(const ErrorArgs a) {
  __shared__ float red[kProjWaves][32][33];
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6;
  const int rb = blockIdx.x, cb = blockIdx.y, ks = blockIdx.z;
  const int row = rb * 32 + l32, col = cb * 32 + l32;
  const int rrow = row < a.D ? row : a.D - 1;  // rows past D compute a copy, not used
  const int T = a.T;
  const bool full_col = col < T, diff_col = col >= T && col < 2 * T;
  const int tcol = full_col ? col : (diff_col ? col - T : 0);
  const int64_t n16 = a.K / 16;
  const int64_t per_ks = (n16 + a.n_split - 1) / a.n_split;
  const int64_t k0 = ks * per_ks, k1 = k0 + per_ks < n16 ? k0 + per_ks : n16;
  const int64_t per = (k1 - k0 + kProjWaves - 1) / kProjWaves;
  const int64_t b0 = k0 + wave * per, b1 = b0 + per < k1 ? b0 + per : k1;
  const CKV_GLOBAL float* af = to_global(a.a_full) + (int64_t)tcol * a.K;
  const CKV_GLOBAL float* ac = to_global(a.a_comp) + (int64_t)tcol * a.K;
  f32x16 acc = f32x16{};
  // U batches of 16 k per step, all their loads issued before their MFMAs
  constexpr int U = 4;
  for (int64_t b = b0; b < b1; b += U) {
    float w[U][8], x[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool in = b + u < b1;
      const int64_t k = (in ? b + u : b0) * 16 + 8 * h;
      if constexpr (DT == 2) {
        load_row16<2>(a.w, (int64_t)rrow * a.w_stride + k, w[u]);
        load_row16<2>(a.w, (int64_t)rrow * a.w_stride + k + 4, w[u] + 4);
      } else {
        load_row16<DT>(a.w, (int64_t)rrow * a.w_stride + k, w[u]);
      }
      const f32x4 f0 = *reinterpret_cast<const CKV_GLOBAL f32x4*>(af + k);
      const f32x4 f1 = *reinterpret_cast<const CKV_GLOBAL f32x4*>(af + k + 4);
      const f32x4 c0 = *reinterpret_cast<const CKV_GLOBAL f32x4*>(ac + k);
      const f32x4 c1 = *reinterpret_cast<const CKV_GLOBAL f32x4*>(ac + k + 4);
      const float fv[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
      const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
      for (int m = 0; m < 8; ++m)
        x[u][m] = !in ? 0.f : (full_col ? fv[m] : (diff_col ? cv[m] - fv[m] : 0.f));
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < 8; ++m) acc = mfma_f32(w[u][m], x[u][m], acc);
  }
  // acc[v]: row rb*32 + acc_row(v, h), column cb*32 + l32
#pragma unroll
  for (int v = 0; v < 16; ++v) red[wave][acc_row(v, h)][l32] = acc[v];
  __syncthreads();
  float* tile = a.part_y + (((int64_t)ks * gridDim.x + rb) * gridDim.y + cb) * 1024;
  for (int e = tid; e < 1024; e += kProjThreads) {
    const int r = e >> 5, c = e & 31;
    float y = 0.f;
#pragma unroll
    for (int wv = 0; wv < kProjWaves; ++wv) y += red[wv][r][c];
    tile[e] = y;
  }
}

// 16-bit W_O: the columns of X = [A_full | A_comp - A_full] (fp32) split into
// two 16-bit parts in W_O's type, high = X rounded, low = X - high rounded,
// so that the 16-bit MFMA of W_O with high and then low gives W_O X to about
// 16 significant bits (W_O itself is exact in its type). x_hl is
// [2][n_cols][K]; columns from 2T on are zero.
template <int DT>
__global__ __launch_bounds__(kProjThreads) void xsplit_kernel(const ErrorArgs a) {
  const int64_t n = (int64_t)a.n_cols * a.K;
  for (int64_t e = (int64_t)blockIdx.x * kProjThreads + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * kProjThreads) {
    const int col = (int)(e / a.K);
    const int64_t k = e - (int64_t)col * a.K;
    float x = 0.f;
    if (col < a.T) x = a.a_full[(int64_t)col * a.K + k];
    else if (col < 2 * a.T)
      x = a.a_comp[(int64_t)(col - a.T) * a.K + k] - a.a_full[(int64_t)(col - a.T) * a.K + k];
    uint16_t hi, lo;
    if constexpr (DT == 0) {  // bf16, round to nearest even (X is finite)
      auto rne = [](float v) {
        const uint32_t u = __float_as_uint(v);
        return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
      };
      hi = rne(x);
      lo = rne(x - __uint_as_float((uint32_t)hi << 16));
    } else {
      const _Float16 h = (_Float16)x;
      const _Float16 l = (_Float16)(x - (float)h);
      hi = __builtin_bit_cast(uint16_t, h);
      lo = __builtin_bit_cast(uint16_t, l);
    }
    a.x_hl[e] = hi;
    a.x_hl[n + e] = lo;
  }
}

// 16-bit W_O: workgroup (row blocks 4*bx .. 4*bx+3, column block cb, K range
// ks); wave w computes the 32 x 32 tile of row block 4*bx + w over the K
// range with the 32x32x16 MFMA (W_O rows against the high and then the low
// part of X, one accumulator) and writes it to part_y.
//
// Every load of the workgroup is issued at the start, so that the whole
// range is in flight at once: W_O in tiles of 32 rows x 128 k (8 KB, at most
// kProjTiles per wave) into registers with contiguous loads (lane l of load i
// takes 16-byte chunk l % 16 of tile row 4i + l / 16), and the X tiles the
// four waves share (both parts, 32 columns) into LDS by all threads. A tile
// of W_O then goes through the wave's LDS region. In LDS, chunk c of row (or
// column) r sits at position c ^ (r % 16); lane half h of lane l32 reads
// chunk 2j + h of row l32 for the j-th 16-k step of the tile, as its X column
// does.
constexpr int kProjTileK = 128;                                // k per tile
constexpr int kProjTileLoads = 32 * kProjTileK * 2 / 16 / 64;  // 16-byte W_O loads per lane: 8
constexpr int kProjTiles = kProjRangeK / kProjTileK;           // tiles per K range: 2
constexpr int kProjXChunks = kProjTiles * 2 * 32 * (kProjTileK / 8);  // 16-byte X chunks: 2048
constexpr int kProjXLoads = kProjXChunks / kProjThreads;              // per thread: 8

template <int DT>
__global__ __launch_bounds__(kProjThreads) void project16_kernel(const ErrorArgs a) {
  __shared__ uint4 wl[kProjWaves][32 * (kProjTileK / 8)];  // a W_O tile per wave, 8 KB
  __shared__ uint4 xl[kProjXChunks];                        // [tile][part][col][chunk], 32 KB
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6;
  const int n_rb = (a.D + 31) / 32;
  const int rb = blockIdx.x * kProjWaves + wave, cb = blockIdx.y, ks = blockIdx.z;
  const int64_t n16 = a.K / 16;
  const int64_t per_ks = (n16 + a.n_split - 1) / a.n_split;
  const int64_t k0 = ks * per_ks, k1 = k0 + per_ks < n16 ? k0 + per_ks : n16;  // in 16-k steps
  const int n_steps = k1 > k0 ? (int)(k1 - k0) : 0;  // <= kProjTiles * 8 (checked on the host)
  const CKV_GLOBAL uint16_t* w0 = to_global(static_cast<const uint16_t*>(a.w));
  const CKV_GLOBAL uint16_t* x0 = to_global(a.x_hl);
  // this wave's W_O tiles (rows past D or k past the range: zeros)
  u32x4 t[kProjTiles][kProjTileLoads];
#pragma unroll
  for (int tl = 0; tl < kProjTiles; ++tl)
#pragma unroll
    for (int i = 0; i < kProjTileLoads; ++i) {
      const int r = 4 * i + lane / 16, c = lane % 16;
      const int row = rb * 32 + r;
      const bool ok = rb < n_rb && row < a.D && tl * 8 + c / 2 < n_steps;
      const int64_t off =
          ok ? (int64_t)row * a.w_stride + (k0 + tl * 8) * 16 + 8 * c : 0;
      t[tl][i] = ok ? *reinterpret_cast<const CKV_GLOBAL u32x4*>(w0 + off) : u32x4{0u, 0u, 0u, 0u};
    }
  // the shared X tiles: chunk e = ((tile * 2 + part) * 32 + col) * 16 + c
  u32x4 xv[kProjXLoads];
#pragma unroll
  for (int i = 0; i < kProjXLoads; ++i) {
    const int e = i * kProjThreads + tid;
    const int c = e % 16, col = (e / 16) % 32, part = (e / 512) % 2, tl = e / 1024;
    const bool ok = tl * 8 + c / 2 < n_steps;
    const int64_t off = ok ? ((int64_t)part * a.n_cols + cb * 32 + col) * a.K +
                                 (k0 + tl * 8) * 16 + 8 * c
                           : 0;
    xv[i] = ok ? *reinterpret_cast<const CKV_GLOBAL u32x4*>(x0 + off) : u32x4{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int i = 0; i < kProjXLoads; ++i) {
    const int e = i * kProjThreads + tid;
    const int c = e % 16, rc = e / 16;  // rc = (tile * 2 + part) * 32 + col
    xl[rc * 16 + (c ^ (rc & 15))] = make_uint4(xv[i].x, xv[i].y, xv[i].z, xv[i].w);
  }
  __syncthreads();
  if (rb >= n_rb) return;  // after the barrier: these waves only helped load X
  uint4* tile = wl[wave];
  f32x16 acc = f32x16{};
#pragma unroll
  for (int tl = 0; tl < kProjTiles; ++tl) {
    if (tl * 8 >= n_steps) break;
#pragma unroll
    for (int i = 0; i < kProjTileLoads; ++i) {
      const int r = 4 * i + lane / 16, c = lane % 16;
      tile[r * 16 + (c ^ (r & 15))] = make_uint4(t[tl][i].x, t[tl][i].y, t[tl][i].z, t[tl][i].w);
    }
    __builtin_amdgcn_wave_barrier();
    const uint4* xh = xl + (tl * 2 + 0) * 32 * 16;
    const uint4* xlo = xl + (tl * 2 + 1) * 32 * 16;
#pragma unroll
    for (int j = 0; j < kProjTileK / 16; ++j) {
      const int pos = (2 * j + h) ^ (l32 & 15);
      const uint4 wv = tile[l32 * 16 + pos];
      acc = mfma_chunk<DT>(wv, xh[l32 * 16 + pos], acc);
      acc = mfma_chunk<DT>(wv, xlo[l32 * 16 + pos], acc);
    }
    __builtin_amdgcn_wave_barrier();  // the next tile's stores come after these reads
  }
  // acc[v]: row rb*32 + acc_row(v, h), column cb*32 + l32
  float* out = a.part_y + (((int64_t)ks * n_rb + rb) * gridDim.y + cb) * 1024;
#pragma unroll
  for (int v = 0; v < 16; ++v) out[acc_row(v, h) * 32 + l32] = acc[v];
}

// Workgroup (rb, cb): Y = the n_split partial tiles added in order, then
// per column the sum of Y^2 over the tile's rows (rows past D excluded) into
// part[rb][col].
__global__ __launch_bounds__(kProjThreads) void square_kernel(const ErrorArgs a) {
  constexpr int RG = kProjThreads / 32;  // row groups: thread t sums rows t/32, t/32 + RG, ...
  __shared__ float colsum[RG][32];
  const int rb = blockIdx.x, cb = blockIdx.y, nrb = gridDim.x, ncb = gridDim.y;
  const int c = threadIdx.x & 31, rg = threadIdx.x >> 5;
  float sq = 0.f;
  for (int r = rg; r < 32; r += RG) {
    if (rb * 32 + r >= a.D) break;
    // the n_split partials in order, loaded 16 at a time
    float y = 0.f;
    for (int ks0 = 0; ks0 < a.n_split; ks0 += 16) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        v[u] = ks0 + u < a.n_split ? a.part_y[(((int64_t)(ks0 + u) * nrb + rb) * ncb + cb) * 1024 + r * 32 + c]
                                   : 0.f;
#pragma unroll
      for (int u = 0; u < 16; ++u) y += v[u];
    }
    sq += y * y;
  }
  colsum[rg][c] = sq;
  __syncthreads();
  if (threadIdx.x < 32) {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < RG; ++i) t += colsum[i][c];
    const int col = cb * 32 + c;
    if (col < 2 * a.T) a.part[(int64_t)rb * 2 * a.T + col] = t;
  }
}

// One workgroup: num_t and den_t summed over the row blocks (kDecWaves
// threads per step and column kind, each over every kDecWaves-th block, then
// combined in a fixed order), the ratios and their sum in step order.
__global__ __launch_bounds__(kDecThreads) void error_kernel(const ErrorArgs a) {
  constexpr int kSplit = 8;                         // threads per column
  constexpr int kCols = kDecThreads / kSplit;       // columns per round
  __shared__ float part_l[kSplit][kCols];
  __shared__ float col_l[kCols];
  const int n_rb = (a.D + 31) / 32;
  const int j = threadIdx.x % kSplit, cl = threadIdx.x / kSplit;
  float total = 0.f;
  for (int c0 = 0; c0 < 2 * a.T; c0 += kCols) {
    const int col = c0 + cl;
    float acc = 0.f;
    if (col < 2 * a.T) {
      // row blocks j, j + kSplit, ... in that order, kBatch loads in flight
      constexpr int kBatch = 8;
      for (int rb0 = j; rb0 < n_rb; rb0 += kSplit * kBatch) {
        float v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int rb = rb0 + u * kSplit;
          v[u] = rb < n_rb ? a.part[(int64_t)rb * 2 * a.T + col] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) acc += v[u];
      }
    }
    part_l[j][cl] = acc;
    __syncthreads();
    if (threadIdx.x < kCols) {
      float v = 0.f;
#pragma unroll
      for (int i = 0; i < kSplit; ++i) v += part_l[i][threadIdx.x];
      col_l[threadIdx.x] = v;
    }
    __syncthreads();
    // columns c0 .. c0 + kCols - 1 hold den (col < T) or num (col >= T) of
    // their steps; a step's pair lands in the same round when T <= kCols / 2
    if (threadIdx.x == 0) {
      for (int i = 0; i < kCols && c0 + i < 2 * a.T; ++i) part_l[0][i] = col_l[i];
    }
    __syncthreads();
    if (threadIdx.x < kCols && c0 + threadIdx.x < 2 * a.T)
      a.part[(int64_t)n_rb * 2 * a.T + c0 + threadIdx.x] = part_l[0][threadIdx.x];
    __syncthreads();
  }
  // the column sums sit after the row-block partials; ratios in step order
  const float* sums = a.part + (int64_t)n_rb * 2 * a.T;
  if (threadIdx.x == 0) {
    for (int t = 0; t < a.T; ++t) {
      const float r = sqrtf(sums[a.T + t]) / (sqrtf(sums[t]) + a.eps);
      a.ratio[t] = r;
      total += r;
    }
    *a.e = total;
  }
}

template <template <int, int> class KernelOf>
hipError_t launch_dec(int dtype, int d, const DecodeBatch& b, int grid, hipStream_t st) {
  const Timing tm;
  if (dtype == 0) return d == 64 ? launch(KernelOf<0, 64>::fn, grid, kDecThreads, st, tm, b)
                                 : launch(KernelOf<0, 128>::fn, grid, kDecThreads, st, tm, b);
  if (dtype == 1) return d == 64 ? launch(KernelOf<1, 64>::fn, grid, kDecThreads, st, tm, b)
                                 : launch(KernelOf<1, 128>::fn, grid, kDecThreads, st, tm, b);
  return d == 64 ? launch(KernelOf<2, 64>::fn, grid, kDecThreads, st, tm, b)
                 : launch(KernelOf<2, 128>::fn, grid, kDecThreads, st, tm, b);
}

template <int DT, int D>
struct DecodeOf {
  static constexpr auto fn = decode_kernel_16<DT, D>;
};
template <int D>
struct DecodeOf<2, D> {
  static constexpr auto fn = decode_kernel_f32<2, D>;
};

}  // namespace

hipError_t launch_decode(int dtype, const DecodeBatch& b, hipStream_t st) {
  hipError_t e = launch_dec<DecodeOf>(dtype, b.d, b, b.blk_off[b.n], st);
  if (e != hipSuccess) return e;
  const Timing tm;
  return b.d == 64 ? launch(decode_merge_kernel<64>, b.mrg_off[b.n], kDecThreads, st, tm, b)
                   : launch(decode_merge_kernel<128>, b.mrg_off[b.n], kDecThreads, st, tm, b);
}

hipError_t launch_error(int w_dtype, const ErrorArgs& a, hipStream_t st) {
  const Timing tm;
  const int n_rb = (a.D + 31) / 32;
  const dim3 grid(n_rb, (2 * a.T + 31) / 32, a.n_split);
  const dim3 tiles(grid.x, grid.y);
  hipError_t e;
  if (w_dtype == 2) {
    e = launch(project_kernel<2>, grid, kProjThreads, st, tm, a);
  } else {
    // 16-bit W_O: split X once, then one wave per 32 x 32 tile and K range
    const int64_t n = (int64_t)a.n_cols * a.K;
    const int xg = (int)((n + kProjThreads - 1) / kProjThreads);  // one element per thread
    e = w_dtype == 0 ? launch(xsplit_kernel<0>, xg, kProjThreads, st, tm, a)
                     : launch(xsplit_kernel<1>, xg, kProjThreads, st, tm, a);
    if (e != hipSuccess) return e;
    const dim3 g16((n_rb + kProjWaves - 1) / kProjWaves, grid.y, a.n_split);
    e = w_dtype == 0 ? launch(project16_kernel<0>, g16, kProjThreads, st, tm, a)
                     : launch(project16_kernel<1>, g16, kProjThreads, st, tm, a);
  }
  if (e != hipSuccess) return e;
  if ((e = launch(square_kernel, tiles, kProjThreads, st, tm, a)) != hipSuccess) return e;
  return launch(error_kernel, 1, kDecThreads, st, tm, a);
}

}  // namespace ckv
