// gfx950 (MI355X) scoring kernels of CompressKV's prefill-end token selection.
//
// Paper: CompressKV, arXiv 2508.02401, Sec. 3.3 ("Token Selection Driven by
// Semantic Retrieval Heads"). For one KV group g with chosen query heads
// sel(g), window rows i in [0, w) at positions L-w+i:
//   s[h,i,j] = scale * <q[h,i], k[g,j]>               (Eq. 2 logits)
//   p[h,i,j] = softmax over the visible keys j <= L-w+i
//   S[h,j]   = sum_i p[h,i,j]                          (window sum)
//   P[h,j]   = pool_k(S[h,.])[j] on the prefix [0, L-w)
//   A[g,j]   = mean over h in sel(g) of P[h,j]          (head mean)
//
// The exact softmax needs each row's normaliser before the column sums, so
// the logits are formed twice from K:
//   rowstats_kernel  pass 1: per (group, 1024-token chunk) online max and
//                    sum of exp2 for every chosen row, MFMA 32x32 tiles with
//                    tokens as the MFMA rows so each lane reduces its own
//                    registers;
//   lse_kernel       merges the chunk partials into one log2-sum-exp2 per row;
//   score_kernel     pass 2: MFMA tiles with queries as rows, exp2(a*s - lse),
//                    8-row group sums with one cross-half shuffle, per-head
//                    sums in LDS, pooling with a 16-token halo, head mean;
//                    it also accumulates the first-level histogram of the
//                    score keys that the selection starts from.
#include <math.h>

#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

// Stage the chosen heads' window queries of group g into LDS. Row r holds
// head slot r / w8, window row r % w8; padding rows are zero.
template <int EB, int NV, int LDS_ROW>
__device__ __forceinline__ void stage_queries(const LayerArgs& a, const SeqArgs& sq, int sel0,
                                              int n_sel, int nrows, uint4* q_lds) {
  for (int e = threadIdx.x; e < nrows * NV; e += kThreads) {
    const int r = e / NV, c = e - r * NV;
    const int slot = r / a.w8, i = r - slot * a.w8;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (slot < n_sel && i < a.w) {
      const char* src = static_cast<const char*>(sq.q) +
                        ((int64_t)a.sel[sel0 + slot] * sq.q_sh + (int64_t)i * sq.q_sr) * EB;
      val = reinterpret_cast<const uint4*>(src)[c];
    }
    q_lds[r * LDS_ROW + c] = val;
  }
}

// ---------------------------------------------------------------------------
// Pass 1: per-chunk row statistics.
// ---------------------------------------------------------------------------
template <int DT, int D, int MAXQB>
__global__ __launch_bounds__(kThreads) void rowstats_kernel(const LayerArgs a) {
  constexpr int EB = Elt<DT>::bytes;
  constexpr int NV = D * EB / 16;   // 16-byte vectors per row
  constexpr int NC = D * EB / 32;   // operand chunks per lane
  constexpr int LDS_ROW = NV + 1;   // padded row stride (bank spread)
  __shared__ uint4 q_lds[MAXQB * 32 * LDS_ROW];
  __shared__ float2 red[kWaves][MAXQB * 32];

  const int b = xcd_remap(blockIdx.x, gridDim.x);
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_rows) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_rows;
  const int g = local / sq.n_chunks;
  const int chunk = local - g * sq.n_chunks;
  const int sel0 = a.grp_off[g], n_sel = a.grp_off[g + 1] - sel0;
  const int w = a.w, w8 = a.w8;
  const int nqb = (n_sel * w8 + 31) >> 5;
  const int64_t L = sq.L;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const float alpha = a.alpha;

  // the selection state of this group starts from zero in every call; the
  // scoring kernel that accumulates into it runs after this one
  if (chunk == 0 && a.do_hist) {
    for (int i = tid; i < kCtlWords; i += kThreads) sq.ctl[g * kCtlWords + i] = 0u;
    for (int i = tid; i < kHistBins; i += kThreads) sq.hist[(int64_t)g * kHistBins + i] = 0u;
  }

  stage_queries<EB, NV, LDS_ROW>(a, sq, sel0, n_sel, nqb * 32, q_lds);
  __syncthreads();

  uint4 qreg[MAXQB][NC];
#pragma unroll
  for (int qb = 0; qb < MAXQB; ++qb)
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qreg[qb][c] = qb < nqb ? q_lds[(qb * 32 + l32) * LDS_ROW + 2 * c + h]
                             : make_uint4(0u, 0u, 0u, 0u);

  float m_run[MAXQB], z_run[MAXQB];
#pragma unroll
  for (int qb = 0; qb < MAXQB; ++qb) {
    m_run[qb] = -INFINITY;
    z_run[qb] = 0.f;
  }

  const char* kbase = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * EB;
  const int64_t t_begin = (int64_t)chunk * kChunk;
  for (int blk = wave; blk < kChunk / 32; blk += kWaves) {
    const int64_t t0 = t_begin + blk * 32;
    if (t0 >= L) break;
    int64_t t = t0 + l32;
    if (t > L - 1) t = L - 1;
    const uint4* kp = reinterpret_cast<const uint4*>(kbase + t * sq.kv_st * EB) + h;
    uint4 kreg[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) kreg[c] = kp[2 * c];
    // every window row sees every key below L - w
    const bool full = t0 + 32 <= L - w;
#pragma unroll
    for (int qb = 0; qb < MAXQB; ++qb) {
      if (qb >= nqb) break;
      f32x16 acc = {};
#pragma unroll
      for (int c = 0; c < NC; ++c) acc = mfma_chunk<DT>(kreg[c], qreg[qb][c], acc);
      // acc[v]: key t0 + acc_row(v, h), query row qb*32 + l32
      if (!full) {
        const int iw = (qb * 32 + l32) % w8;
        const int64_t last = L - w + iw;  // last key this row sees (>= L for padding)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t tok = t0 + acc_row(v, h);
          if (tok >= L || tok > last) acc[v] = -INFINITY;
        }
      }
      float mx = acc[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) mx = fmaxf(mx, acc[v]);
      const float m_new = fmaxf(m_run[qb], mx);
      const float ms = m_new == -INFINITY ? 0.f : m_new * alpha;
      float z = z_run[qb] * fast_exp2(m_run[qb] * alpha - ms);
#pragma unroll
      for (int v = 0; v < 16; ++v) z += fast_exp2(fmaf(acc[v], alpha, -ms));
      z_run[qb] = z;
      m_run[qb] = m_new;
    }
  }

  // merge the two lane halves (same query row, different keys), then the waves
#pragma unroll
  for (int qb = 0; qb < MAXQB; ++qb) {
    if (qb >= nqb) break;
    const float mo = __shfl_xor(m_run[qb], 32);
    const float zo = __shfl_xor(z_run[qb], 32);
    const float mn = fmaxf(m_run[qb], mo);
    const float msn = mn == -INFINITY ? 0.f : mn * alpha;
    const float z = z_run[qb] * fast_exp2(m_run[qb] * alpha - msn) + zo * fast_exp2(mo * alpha - msn);
    if (h == 0) red[wave][qb * 32 + l32] = make_float2(mn, z);
  }
  __syncthreads();
  if (tid < nqb * 32) {
    float m = -INFINITY;
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) m = fmaxf(m, red[wv][tid].x);
    const float ms = m == -INFINITY ? 0.f : m * alpha;
    float z = 0.f;
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) z += red[wv][tid].y * fast_exp2(red[wv][tid].x * alpha - ms);
    sq.partial[((int64_t)g * sq.n_chunks + chunk) * kMaxRows + tid] = make_float2(m, z);
  }
}

// Merge chunk partials: lse[r] = log2(sum_j exp2(alpha * s_rj)) so that the
// softmax probability is exp2(alpha * s - lse). Padding rows get +inf (p = 0).
__global__ __launch_bounds__(kMaxRows) void lse_kernel(const LayerArgs a) {
  const int s = blockIdx.x / a.n_kv, g = blockIdx.x - s * a.n_kv;
  const SeqArgs& sq = a.seq[s];
  const int r = threadIdx.x;
  const int n_sel = a.grp_off[g + 1] - a.grp_off[g];
  const int slot = r / a.w8, i = r - slot * a.w8;
  float out = INFINITY;
  if (slot < n_sel && i < a.w) {
    const float2* p = sq.partial + (int64_t)g * sq.n_chunks * kMaxRows + r;
    float m = -INFINITY;
    for (int c = 0; c < sq.n_chunks; ++c) m = fmaxf(m, p[(int64_t)c * kMaxRows].x);
    const float ms = m * a.alpha;
    float z = 0.f;
    for (int c = 0; c < sq.n_chunks; ++c) {
      const float2 v = p[(int64_t)c * kMaxRows];
      z += v.y * fast_exp2(v.x * a.alpha - ms);
    }
    out = ms + log2f(z);
  }
  sq.lse[(int64_t)g * kMaxRows + r] = out;
}

// ---------------------------------------------------------------------------
// Pass 2: probabilities, window sums, pooling, head mean.
// ---------------------------------------------------------------------------
template <int DT, int D, int MAXQB>
__global__ __launch_bounds__(kThreads) void score_kernel(const LayerArgs a) {
  constexpr int EB = Elt<DT>::bytes;
  constexpr int NV = D * EB / 16;
  constexpr int NC = D * EB / 32;
  constexpr int LDS_ROW = NV + 1;
  __shared__ uint4 q_lds[MAXQB * 32 * LDS_ROW];
  __shared__ __align__(16) float c_lds[MAXQB * 32];
  __shared__ uint32_t hist_lds[kHistBins];
  extern __shared__ float sh[];  // [max_sel][kTileComp] per-head window sums

  const int b = xcd_remap(blockIdx.x, gridDim.x);
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_score) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_score;
  const int g = local / sq.n_tiles;
  const int tile = local - g * sq.n_tiles;
  const int sel0 = a.grp_off[g], n_sel = a.grp_off[g + 1] - sel0;
  const int w8 = a.w8;
  const int nqb = (n_sel * w8 + 31) >> 5;
  const int64_t Ls = sq.L - a.w;
  const int64_t j0 = (int64_t)tile * kTileOut;
  const int64_t base = j0 - kHalo;  // token of computed column 0
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const float alpha = a.alpha;

  stage_queries<EB, NV, LDS_ROW>(a, sq, sel0, n_sel, nqb * 32, q_lds);
  for (int r = tid; r < nqb * 32; r += kThreads) c_lds[r] = sq.lse[(int64_t)g * kMaxRows + r];
  for (int e = tid; e < n_sel * kTileComp; e += kThreads) sh[e] = 0.f;
  const bool do_hist = a.do_hist && sq.n_keep > 0;
  if (do_hist)
    for (int i = tid; i < kHistBins; i += kThreads) hist_lds[i] = 0u;
  __syncthreads();

  uint4 qreg[MAXQB][NC];
#pragma unroll
  for (int qb = 0; qb < MAXQB; ++qb)
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qreg[qb][c] = qb < nqb ? q_lds[(qb * 32 + l32) * LDS_ROW + 2 * c + h]
                             : make_uint4(0u, 0u, 0u, 0u);

  const char* kbase = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * EB;
  for (int blk = wave; blk < kTileComp / 32; blk += kWaves) {
    const int64_t tb = base + blk * 32;
    if (tb + 32 <= 0 || tb >= Ls) continue;
    int64_t t = tb + l32;
    t = t < 0 ? 0 : (t > Ls - 1 ? Ls - 1 : t);
    const uint4* kp = reinterpret_cast<const uint4*>(kbase + t * sq.kv_st * EB) + h;
    uint4 kreg[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) kreg[c] = kp[2 * c];
#pragma unroll
    for (int qb = 0; qb < MAXQB; ++qb) {
      if (qb >= nqb) break;
      f32x16 acc = {};
#pragma unroll
      for (int c = 0; c < NC; ++c) acc = mfma_chunk<DT>(qreg[qb][c], kreg[c], acc);
      // acc[v]: query row qb*32 + acc_row(v, h), key tb + l32; prefix keys are
      // visible to every window row, so no mask is needed here.
      float gs[4];
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        const float4 cv = *reinterpret_cast<const float4*>(&c_lds[qb * 32 + 8 * a4 + 4 * h]);
        gs[a4] = fast_exp2(fmaf(acc[4 * a4 + 0], alpha, -cv.x)) +
                 fast_exp2(fmaf(acc[4 * a4 + 1], alpha, -cv.y)) +
                 fast_exp2(fmaf(acc[4 * a4 + 2], alpha, -cv.z)) +
                 fast_exp2(fmaf(acc[4 * a4 + 3], alpha, -cv.w));
      }
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) gs[a4] += __shfl_xor(gs[a4], 32);
      // rows qb*32 + 8*a4 .. +7 all belong to head slot (qb*32 + 8*a4) / w8
      if (h == 0) {
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          const int slot = (qb * 32 + 8 * a4) / w8;
          if (slot < n_sel) sh[slot * kTileComp + blk * 32 + l32] += gs[a4];
        }
      }
    }
  }
  __syncthreads();

  const int r = a.kp >> 1;
  const float kpf = (float)a.kp;
  float* out = sq.scores + (int64_t)g * Ls;
  for (int o = tid; o < kTileOut; o += kThreads) {
    const int64_t j = j0 + o;
    if (j >= Ls) break;
    const int lo = (int)(j < r ? -j : -r);
    const int hi = (int)(Ls - 1 - j < r ? Ls - 1 - j : r);
    const int tc = o + kHalo;
    float total = 0.f;
    for (int slot = 0; slot < n_sel; ++slot) {
      const float* row = sh + slot * kTileComp + tc;
      if (a.pool == 0) {
        float acc = 0.f;
        for (int dt = lo; dt <= hi; ++dt) acc += row[dt];
        total += acc / kpf;
      } else {
        float m = row[lo];
        for (int dt = lo + 1; dt <= hi; ++dt) m = fmaxf(m, row[dt]);
        total += m;
      }
    }
    const float score = total / (float)n_sel;
    out[j] = score;
    if (do_hist) atomicAdd(&hist_lds[score_key(score) >> kHistShift], 1u);
  }
  if (!do_hist) return;

  // first-level histogram of this tile's keys into the group's histogram
  __syncthreads();
  uint32_t* ghist = sq.hist + (int64_t)g * kHistBins;
  for (int i = tid; i < kHistBins; i += kThreads) {
    const uint32_t c = hist_lds[i];
    if (c) atomicAdd(&ghist[i], c);
  }
}

template <int DT>
constexpr int maxqb() {
  return DT == 2 ? kMaxRowsF32 / 32 : kMaxRows / 32;
}

}  // namespace

hipError_t launch_rowstats(int dtype, const LayerArgs& a, int grid, hipStream_t st) {
#define CKV_RS(DT, D) hipLaunchKernelGGL((rowstats_kernel<DT, D, maxqb<DT>()>), dim3(grid), dim3(kThreads), 0, st, a)
  if (dtype == 0) { if (a.d == 64) CKV_RS(0, 64); else CKV_RS(0, 128); }
  else if (dtype == 1) { if (a.d == 64) CKV_RS(1, 64); else CKV_RS(1, 128); }
  else { if (a.d == 64) CKV_RS(2, 64); else CKV_RS(2, 128); }
#undef CKV_RS
  return hipGetLastError();
}

hipError_t launch_lse(const LayerArgs& a, int grid, hipStream_t st) {
  hipLaunchKernelGGL(lse_kernel, dim3(grid), dim3(kMaxRows), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_score(int dtype, const LayerArgs& a, int grid, hipStream_t st) {
  const size_t lds = (size_t)a.max_sel * kTileComp * sizeof(float);
#define CKV_SC(DT, D) hipLaunchKernelGGL((score_kernel<DT, D, maxqb<DT>()>), dim3(grid), dim3(kThreads), lds, st, a)
  if (dtype == 0) { if (a.d == 64) CKV_SC(0, 64); else CKV_SC(0, 128); }
  else if (dtype == 1) { if (a.d == 64) CKV_SC(1, 64); else CKV_SC(1, 128); }
  else { if (a.d == 64) CKV_SC(2, 64); else CKV_SC(2, 128); }
#undef CKV_SC
  return hipGetLastError();
}

}  // namespace ckv
