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
//                    sum of exp2 for every chosen row;
//   lse_kernel       merges the chunk partials into one log2-sum-exp2 per row;
//   score_kernel     pass 2: exp2(alpha*s - lse), window sums per head,
//                    pooling with a 16-token halo, head mean, and the
//                    first-level histogram of the score keys that the
//                    selection starts from.
//
// Work decomposition (both passes): a group's chosen rows are padded per head
// to a multiple of 8 and split into 32-row query blocks. Each wave of a
// workgroup owns one query block and keeps its query operand in registers for
// its whole life. K is streamed once per workgroup through a ring of LDS
// slots with direct global-to-LDS loads (global_load_lds_dwordx4): every load
// instruction moves 1 KB of consecutive rows, so HBM sees whole lines, and the
// loads of the next stages stay in flight (explicit partial vmcnt waits and a
// plain s_barrier, since a fenced barrier would drain them). Rows land in LDS
// with their 16-byte chunks XOR-swizzled so that the MFMA-layout reads (lane l
// takes token l % 32) spread over all banks. Logits come from v_mfma 32x32x16.
#include <math.h>

#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

// Waves per query block when a workgroup's 4 waves share nqb blocks.
__device__ __forceinline__ int waves_per_qblock(int nqb) {
  return nqb == 1 ? 4 : (nqb == 2 ? 2 : 1);
}

// This lane's query operand for query block qb, straight from global memory:
// row qb*32 + l32 of the group's padded row space (head slot row / w8, window
// row row % w8); padding rows are zero.
template <int NC, int EB>
__device__ __forceinline__ void load_queries(const LayerArgs& a, const SeqArgs& sq, int sel0,
                                             int n_sel, int qb, int l32, int h, uint4* q) {
  const int row = qb * 32 + l32;
  const int slot = row / a.w8, i = row - slot * a.w8;
  if (slot < n_sel && i < a.w) {
    const uint4* src = reinterpret_cast<const uint4*>(
                           static_cast<const char*>(sq.q) +
                           ((int64_t)a.sel[sel0 + slot] * sq.q_sh + (int64_t)i * sq.q_sr) * EB) +
                       h;
#pragma unroll
    for (int c = 0; c < NC; ++c) q[c] = src[2 * c];
  } else {
#pragma unroll
    for (int c = 0; c < NC; ++c) q[c] = make_uint4(0u, 0u, 0u, 0u);
  }
}

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left at their no-wait maxima).
constexpr int vmcnt_imm(int n) { return 0xF70 | (n & 15) | ((n >> 4) << 14); }

// Staging of K through LDS. A stage is ST = SB / ROWB consecutive tokens (a
// multiple of 32); its LDS image is row-major, ROWB bytes per token, with the
// 16-byte chunk c of token t stored at position c ^ swz(t).
template <int DT, int D, int SB>
struct Stager {
  static constexpr int EB = Elt<DT>::bytes;
  static constexpr int ROWB = D * EB;            // bytes per token row: 128, 256 or 512
  static constexpr int NV = ROWB / 16;           // 16-byte chunks per row
  static constexpr int NC = ROWB / 32;           // MFMA operand chunks per lane
  static constexpr int ST = SB / ROWB;           // tokens per stage
  static constexpr int VEC = SB / 16;            // 16-byte vectors per stage
  static constexpr int PT = VEC / kThreads;      // load instructions per wave per stage
  static constexpr int BLOCKS = ST / 32;
  static_assert(ST % 32 == 0 && VEC % kThreads == 0, "stage shape");

  // Rows of 256 B or more start on the same bank: spread chunks by t % 16.
  // 128-byte rows alternate halves of the banks: spread by (t / 2) % 8.
  __device__ static __forceinline__ int swz(int t) { return ROWB >= 256 ? (t & 15) : ((t >> 1) & 7); }

  // Per-lane part of a stage's loads, the same for every stage: load k of
  // this lane fills LDS vector seg*64 + lane (seg = k*waves + wave) with
  // chunk pos ^ swz(t) of stage token t.
  struct Plan {
    int64_t off[PT];  // byte offset of that chunk from the stage's first row
    int tok[PT];      // t
    int chunk[PT];    // pos ^ swz(t)
  };
  __device__ static __forceinline__ Plan plan(int wave, int64_t kv_st) {
    Plan p;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 0; k < PT; ++k) {
      const int e = (k * kWaves + wave) * 64 + lane;
      const int t = e / NV, pos = e - t * NV;
      p.tok[k] = t;
      p.chunk[k] = pos ^ swz(t);
      p.off[k] = (int64_t)t * kv_st * EB + p.chunk[k] * 16;
    }
    return p;
  }

  // Issue the direct-to-LDS loads of the stage whose first token is t0.
  // Tokens outside [lo, hi] read row lo or hi instead (their results are
  // never used); only stages that cross lo or hi take that slower path.
  __device__ static __forceinline__ void fetch(const char* kbase, int64_t kv_st, int64_t t0,
                                               int64_t lo, int64_t hi, const Plan& p, int wave,
                                               uint4* slot) {
    if (t0 >= lo && t0 + ST - 1 <= hi) {
      const char* sb = kbase + t0 * kv_st * EB;
#pragma unroll
      for (int k = 0; k < PT; ++k)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint4*>(sb + p.off[k]),
                                         slot + (k * kWaves + wave) * 64, 16, 0, 0);
    } else {
#pragma unroll
      for (int k = 0; k < PT; ++k) {
        int64_t tok = t0 + p.tok[k];
        tok = tok < lo ? lo : (tok > hi ? hi : tok);
        const uint4* src = reinterpret_cast<const uint4*>(kbase + tok * kv_st * EB) + p.chunk[k];
        __builtin_amdgcn_global_load_lds(src, slot + (k * kWaves + wave) * 64, 16, 0, 0);
      }
    }
  }

  // Byte offsets, within a block, of this lane's operand chunks (token l32 of
  // the block, halves by h). The swizzle of token bi*32 + l32 equals that of
  // l32, so the offsets are the same for every block.
  __device__ static __forceinline__ void operand_offsets(int l32, int h, int* off) {
#pragma unroll
    for (int c = 0; c < NC; ++c) off[c] = (l32 * NV + ((2 * c + h) ^ swz(l32))) * 16;
  }

  // This lane's operand chunks of block bi.
  __device__ static __forceinline__ void operand(const uint4* slot, int bi, const int* off,
                                                 uint4* kr) {
    const char* blk = reinterpret_cast<const char*>(slot) + bi * 32 * ROWB;
#pragma unroll
    for (int c = 0; c < NC; ++c) kr[c] = *reinterpret_cast<const uint4*>(blk + off[c]);
  }
};

// Stage size: 16 KB (at least one 32-token block): with two blocks per stage
// every wave has a block when a group has 2 query blocks.
template <int DT, int D>
constexpr int stage_bytes() {
  return 32 * D * Elt<DT>::bytes > 16384 ? 32 * D * Elt<DT>::bytes : 16384;
}

// Wait until at most n_after of this wave's later stages are still loading.
template <int PT, int MAXA>
__device__ __forceinline__ void wait_stages(int n_after) {
  static_assert(MAXA <= 2, "ring depth");
  if (MAXA >= 2 && n_after >= 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * PT));
  else if (MAXA >= 1 && n_after >= 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm(PT));
  else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
}

// Stage loop shared by both passes over stages 0..ns-1 (stage k starts at
// token t_first + k*ST, tokens clamped to [lo, hi]) with an NS-slot LDS ring
// (slots are distinct LDS arrays so the compiler can tell the in-flight loads
// from the slot being read). At step k: wait for stage k, barrier (stage k is
// complete and every wave has finished with stage k-1's slot), issue stage
// k+NS-1 into that freed slot, then body(slot, k) reduces stage k.
template <class S, int NS, class Body>
__device__ __forceinline__ void stage_loop(uint4* const* slot, const char* kbase, int64_t kv_st,
                                           int64_t t_first, int ns, int64_t lo, int64_t hi,
                                           int wave, Body body) {
  const typename S::Plan p = S::plan(wave, kv_st);
#pragma unroll
  for (int j = 0; j < NS - 1; ++j)
    if (j < ns) S::fetch(kbase, kv_st, t_first + (int64_t)j * S::ST, lo, hi, p, wave, slot[j]);
  for (int k0 = 0; k0 < ns; k0 += NS) {
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int k = k0 + j;
      if (k < ns) {
        const int left = ns - 1 - k;
        wait_stages<S::PT, NS - 2>(left < NS - 2 ? left : NS - 2);
        __builtin_amdgcn_s_barrier();
        if (k + NS - 1 < ns)
          S::fetch(kbase, kv_st, t_first + (int64_t)(k + NS - 1) * S::ST, lo, hi, p, wave,
                   slot[(j + NS - 1) % NS]);
        body(slot[j], k);
      }
    }
  }
  __syncthreads();
}

// Operand-reading and MFMA part shared by both passes: the wave's blocks of a
// stage are sub, sub + WPQ, ... (NB of them at most); acc[i] receives the
// 32x32 logit tile of block i, queries x keys when KEYS_AS_ROWS is false,
// keys x queries otherwise. has[i] tells whether block i is computed.
template <int DT, class S, int WPQ, bool KEYS_AS_ROWS>
__device__ __forceinline__ void stage_tiles(const uint4* slot, const int* opoff, const uint4* q,
                                            const bool* has, f32x16* acc) {
  constexpr int NB = (S::BLOCKS + WPQ - 1) / WPQ;
  constexpr int NC = S::NC;
  uint4 kr[NB][NC];
#pragma unroll
  for (int i = 0; i < NB; ++i)
    if (has[i]) S::operand(slot, i * WPQ, opoff, kr[i]);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (!has[i]) continue;
    acc[i] = f32x16{};
#pragma unroll
    for (int c = 0; c < NC; ++c)
      acc[i] = KEYS_AS_ROWS ? mfma_chunk<DT>(kr[i][c], q[c], acc[i]) : mfma_chunk<DT>(q[c], kr[i][c], acc[i]);
  }
}

// ---------------------------------------------------------------------------
// Pass 1: per-chunk row statistics.
// ---------------------------------------------------------------------------
template <int DT, int D, int WPQ, class S, int NS>
__device__ __forceinline__ void rowstats_body(const LayerArgs& a, const SeqArgs& sq, int g,
                                              int chunk, int sel0, int n_sel, int nqb,
                                              uint4* const* slots, float2 (*red)[32]) {
  constexpr int NC = S::NC;
  constexpr int NB = (S::BLOCKS + WPQ - 1) / WPQ;
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int qb = wave / WPQ, sub = wave % WPQ;
  const bool active = qb < nqb;
  const int w = a.w, w8 = a.w8;
  const int L = (int)sq.L, Ls = L - w;
  const float alpha = a.alpha;
  const char* kbase = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * S::EB;
  const int t_begin = chunk * kChunk;
  const int n_tok = L - t_begin < kChunk ? L - t_begin : kChunk;
  const int ns = (n_tok + S::ST - 1) / S::ST;
  // this lane's query row (column of the MFMA result) and its last visible key
  const int last = Ls + (qb * 32 + l32) % w8;  // >= L for padding rows

  uint4 q[NC];
  if (active) load_queries<NC, S::EB>(a, sq, sel0, n_sel, qb, l32, h, q);
  int opoff[NC];
  S::operand_offsets(l32, h, opoff);
#pragma unroll
  for (int c = 0; c < NC; ++c) opoff[c] += sub * 32 * S::ROWB;
  float m_run = -INFINITY, z_run = 0.f;

  stage_loop<S, NS>(slots, kbase, sq.kv_st, t_begin, ns, 0, L - 1, wave, [&](const uint4* slot, int k) {
    if (!active) return;
    const int ts = t_begin + k * S::ST + sub * 32;  // token of this wave's first block
    bool has[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) has[i] = sub + i * WPQ < S::BLOCKS && ts + i * WPQ * 32 < L;
    f32x16 acc[NB];
    stage_tiles<DT, S, WPQ, true>(slot, opoff, q, has, acc);
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (!has[i]) continue;
      // acc[i][v]: key t0 + acc_row(v, h) of this lane's query row
      const int t0 = ts + i * WPQ * 32;
      if (t0 + 32 > Ls) {  // keys inside the window: causal mask (a uniform branch)
        const int rel = last - t0;
        const int lim = rel < -1 ? -1 : (rel > 32 ? 32 : rel);
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (acc_row(v, h) > lim) acc[i][v] = -INFINITY;
      }
      float mx = acc[i][0];
#pragma unroll
      for (int v = 1; v < 16; ++v) mx = fmaxf(mx, acc[i][v]);
      const float m_new = fmaxf(m_run, mx);
      const float ms = m_new == -INFINITY ? 0.f : m_new * alpha;
      float z = z_run * fast_exp2(m_run * alpha - ms);
#pragma unroll
      for (int v = 0; v < 16; ++v) z += fast_exp2(fmaf(acc[i][v], alpha, -ms));
      z_run = z;
      m_run = m_new;
    }
  });

  // merge the two lane halves (same query row, different keys), then the
  // waves that share this query block
  {
    const float mo = __shfl_xor(m_run, 32);
    const float zo = __shfl_xor(z_run, 32);
    const float mn = fmaxf(m_run, mo);
    const float msn = mn == -INFINITY ? 0.f : mn * alpha;
    const float z = z_run * fast_exp2(m_run * alpha - msn) + zo * fast_exp2(mo * alpha - msn);
    if (h == 0) red[wave][l32] = make_float2(mn, z);
  }
  __syncthreads();
  if (tid < nqb * 32) {
    const int qq = tid >> 5, r = tid & 31;
    float m = -INFINITY;
#pragma unroll
    for (int sw = 0; sw < WPQ; ++sw) m = fmaxf(m, red[qq * WPQ + sw][r].x);
    const float ms = m == -INFINITY ? 0.f : m * alpha;
    float z = 0.f;
#pragma unroll
    for (int sw = 0; sw < WPQ; ++sw)
      z += red[qq * WPQ + sw][r].y * fast_exp2(red[qq * WPQ + sw][r].x * alpha - ms);
    sq.partial[((int64_t)g * sq.n_chunks + chunk) * kMaxRows + tid] = make_float2(m, z);
  }
}

template <int DT, int D>
__global__ __launch_bounds__(kThreads) void rowstats_kernel(const LayerArgs a) {
  using S = Stager<DT, D, stage_bytes<DT, D>()>;
  constexpr int NS = 4;  // 4-slot ring
  __shared__ uint4 slot0[S::VEC];
  __shared__ uint4 slot1[S::VEC];
  __shared__ uint4 slot2[S::VEC];
  __shared__ uint4 slot3[S::VEC];
  __shared__ float2 red[kWaves][32];
  uint4* const slots[NS] = {slot0, slot1, slot2, slot3};

  const int b = xcd_remap(blockIdx.x, gridDim.x);
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_rows) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_rows;
  const int g = local / sq.n_chunks;
  const int chunk = local - g * sq.n_chunks;
  const int sel0 = a.grp_off[g], n_sel = a.grp_off[g + 1] - sel0;
  const int nqb = (n_sel * a.w8 + 31) >> 5;

  // the selection state of this group starts from zero in every call; the
  // scoring kernel that accumulates into it runs after this one
  if (chunk == 0 && a.do_hist) {
    for (int i = threadIdx.x; i < kCtlWords; i += kThreads) sq.ctl[g * kCtlWords + i] = 0u;
    for (int i = threadIdx.x; i < kHistBins; i += kThreads)
      sq.hist[(int64_t)g * kHistBins + i] = 0u;
  }
  const int wpq = waves_per_qblock(nqb);
  if (wpq == 1) rowstats_body<DT, D, 1, S, NS>(a, sq, g, chunk, sel0, n_sel, nqb, slots, red);
  else if (wpq == 2) rowstats_body<DT, D, 2, S, NS>(a, sq, g, chunk, sel0, n_sel, nqb, slots, red);
  else rowstats_body<DT, D, 4, S, NS>(a, sq, g, chunk, sel0, n_sel, nqb, slots, red);
}

// Merge chunk partials: lse[r] = log2(sum_j exp2(alpha * s_rj)) so that the
// softmax probability is exp2(alpha * s - lse). Padding rows get +inf (p = 0).
// One workgroup per (prompt, group, 32-row block); the 8 lanes of a row merge
// every 8th chunk each, then one lane merges their 8 results.
constexpr int kLseRows = 32;
constexpr int kLseLanes = kThreads / kLseRows;

__device__ __forceinline__ void lse_merge(float& m, float& z, float m2, float z2, float alpha) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;  // both empty
  const float ms = mn * alpha;
  z = z * fast_exp2(m * alpha - ms) + z2 * fast_exp2(m2 * alpha - ms);
  m = mn;
}

__global__ __launch_bounds__(kThreads) void lse_kernel(const LayerArgs a) {
  __shared__ float2 part[kLseLanes][kLseRows];
  constexpr int kBlocks = kMaxRows / kLseRows;
  const int sg = blockIdx.x / kBlocks, rb = blockIdx.x - sg * kBlocks;
  const int s = sg / a.n_kv, g = sg - s * a.n_kv;
  const SeqArgs& sq = a.seq[s];
  const int lr = threadIdx.x % kLseRows, c0 = threadIdx.x / kLseRows;
  const int r = rb * kLseRows + lr;
  const int n_sel = a.grp_off[g + 1] - a.grp_off[g];
  const int slot = r / a.w8, i = r - slot * a.w8;
  const bool valid = slot < n_sel && i < a.w;
  float m = -INFINITY, z = 0.f;
  if (valid) {
    const float2* p = sq.partial + (int64_t)g * sq.n_chunks * kMaxRows + r;
#pragma unroll 8
    for (int c = c0; c < sq.n_chunks; c += kLseLanes) {
      const float2 v = p[(int64_t)c * kMaxRows];
      lse_merge(m, z, v.x, v.y, a.alpha);
    }
  }
  part[c0][lr] = make_float2(m, z);
  __syncthreads();
  if (threadIdx.x < kLseRows) {
    float mm = -INFINITY, zz = 0.f;
#pragma unroll
    for (int c = 0; c < kLseLanes; ++c) lse_merge(mm, zz, part[c][lr].x, part[c][lr].y, a.alpha);
    sq.lse[(int64_t)g * kMaxRows + r] = valid ? mm * a.alpha + log2f(zz) : INFINITY;
  }
}

// ---------------------------------------------------------------------------
// Pass 2: probabilities, window sums, pooling, head mean.
// ---------------------------------------------------------------------------
constexpr int kGroupRows = kMaxRows / 8;  // 8-row groups of one group's rows

template <int DT, int D, int WPQ, class S, int NS>
__device__ __forceinline__ void score_body(const LayerArgs& a, const SeqArgs& sq, int g, int tile,
                                           int sel0, int n_sel, int nqb, uint4* const* slots,
                                           uint4* slot01, float* gsum) {
  constexpr int NC = S::NC;
  constexpr int NB = (S::BLOCKS + WPQ - 1) / WPQ;
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int qb = wave / WPQ, sub = wave % WPQ;
  const bool active = qb < nqb;
  const int w8 = a.w8;
  const int Ls = (int)sq.L - a.w;
  const int j0 = tile * kTileOut;
  const int base = j0 - kHalo;  // token of computed column 0
  const float alpha = a.alpha;
  const char* kbase = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * S::EB;

  // stages overlapping the prefix [0, Ls)
  const int end_tok = base + kTileComp < Ls ? base + kTileComp : Ls;
  const int ns = (end_tok - base + S::ST - 1) / S::ST;

  uint4 q[NC];
  float4 cv[4];  // lse of this lane's 16 result rows qb*32 + 8*a4 + 4*h + e (exp2 units)
  if (active) {
    load_queries<NC, S::EB>(a, sq, sel0, n_sel, qb, l32, h, q);
    const float4* lse4 = reinterpret_cast<const float4*>(sq.lse + (int64_t)g * kMaxRows + qb * 32);
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) cv[a4] = lse4[2 * a4 + h];
  }
  int opoff[NC];
  S::operand_offsets(l32, h, opoff);
#pragma unroll
  for (int c = 0; c < NC; ++c) opoff[c] += sub * 32 * S::ROWB;

  stage_loop<S, NS>(slots, kbase, sq.kv_st, base, ns, 0, Ls - 1, wave, [&](const uint4* slot, int k) {
    if (!active) return;
    const int cs = k * S::ST + sub * 32;  // computed column of this wave's first block
    bool has[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int tb = base + cs + i * WPQ * 32;  // first token of block i
      // blocks wholly before token 0 or at/after Ls are not needed
      has[i] = sub + i * WPQ < S::BLOCKS && tb + 32 > 0 && tb < Ls;
    }
    f32x16 acc[NB];
    stage_tiles<DT, S, WPQ, false>(slot, opoff, q, has, acc);
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (!has[i]) continue;
      // acc[i][v]: query row qb*32 + acc_row(v, h), key at computed column col;
      // prefix keys are visible to every window row, so no mask is needed.
      float gs[4];
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4)
        gs[a4] = fast_exp2(fmaf(acc[i][4 * a4 + 0], alpha, -cv[a4].x)) +
                 fast_exp2(fmaf(acc[i][4 * a4 + 1], alpha, -cv[a4].y)) +
                 fast_exp2(fmaf(acc[i][4 * a4 + 2], alpha, -cv[a4].z)) +
                 fast_exp2(fmaf(acc[i][4 * a4 + 3], alpha, -cv[a4].w));
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) gs[a4] += __shfl_xor(gs[a4], 32);
      // lane half h stores groups a4 = h and h + 2
      const int col = cs + i * WPQ * 32 + l32;
      gsum[(qb * 4 + h) * kTileComp + col] = h ? gs[1] : gs[0];
      gsum[(qb * 4 + 2 + h) * kTileComp + col] = h ? gs[3] : gs[2];
    }
  });

  const bool do_hist = a.do_hist && sq.n_keep > 0;
  uint32_t* hist_lds = reinterpret_cast<uint32_t*>(slot01);  // K stages are no longer read
  if (do_hist)
    for (int i = tid; i < kHistBins; i += kThreads) hist_lds[i] = 0u;
  __syncthreads();

  // head window sums: the head in slot hs owns 8-row groups
  // [hs*w8/8, (hs+1)*w8/8); fold them into the slot's first group row
  const int gph = w8 / 8;
  for (int col = tid; col < kTileComp; col += kThreads) {
    for (int hs = 0; hs < n_sel; ++hs) {
      float acc = gsum[(hs * gph) * kTileComp + col];
      for (int r8 = 1; r8 < gph; ++r8) acc += gsum[(hs * gph + r8) * kTileComp + col];
      gsum[(hs * gph) * kTileComp + col] = acc;
    }
  }
  __syncthreads();

  const int r = a.kp >> 1;
  const float kpf = (float)a.kp;
  float* out = sq.scores + (int64_t)g * Ls;
  for (int o = tid; o < kTileOut; o += kThreads) {
    const int j = j0 + o;
    if (j >= Ls) break;
    const int lo = j < r ? -j : -r;
    const int hi = Ls - 1 - j < r ? Ls - 1 - j : r;
    const int tc = o + kHalo;
    float total = 0.f;
    for (int hs = 0; hs < n_sel; ++hs) {
      const float* row = gsum + (hs * gph) * kTileComp + tc;
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

template <int DT, int D>
__global__ __launch_bounds__(kThreads) void score_kernel(const LayerArgs a) {
  using S = Stager<DT, D, stage_bytes<DT, D>()>;
  constexpr int NS = 3;  // 3-slot ring
  static_assert(kTileComp % S::ST == 0, "tile is whole stages");
  static_assert(2 * S::VEC * 16 >= kHistBins * 4, "histogram reuses two K slots");
  // slots 0 and 1 are adjacent so that the histogram can reuse them as one
  __shared__ uint4 slot01[2 * S::VEC];
  __shared__ uint4 slot2[S::VEC];
  // gsum[r8][col]: sum over the 8 rows of 8-row group r8 of p at computed
  // column col; rows of one head are whole groups, so a head's window sum is a
  // fixed-order sum of its groups
  __shared__ float gsum[kGroupRows * kTileComp];
  uint4* const slots[NS] = {slot01, slot01 + S::VEC, slot2};

  const int b = xcd_remap(blockIdx.x, gridDim.x);
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_score) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_score;
  const int g = local / sq.n_tiles;
  const int tile = local - g * sq.n_tiles;
  const int sel0 = a.grp_off[g], n_sel = a.grp_off[g + 1] - sel0;
  const int nqb = (n_sel * a.w8 + 31) >> 5;
  const int wpq = waves_per_qblock(nqb);
  if (wpq == 1) score_body<DT, D, 1, S, NS>(a, sq, g, tile, sel0, n_sel, nqb, slots, slot01, gsum);
  else if (wpq == 2) score_body<DT, D, 2, S, NS>(a, sq, g, tile, sel0, n_sel, nqb, slots, slot01, gsum);
  else score_body<DT, D, 4, S, NS>(a, sq, g, tile, sel0, n_sel, nqb, slots, slot01, gsum);
}

template <template <int, int> class KernelOf>
hipError_t launch_typed(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  if (dtype == 0) return a.d == 64 ? launch(KernelOf<0, 64>::fn, grid, kThreads, st, tm, a)
                                   : launch(KernelOf<0, 128>::fn, grid, kThreads, st, tm, a);
  if (dtype == 1) return a.d == 64 ? launch(KernelOf<1, 64>::fn, grid, kThreads, st, tm, a)
                                   : launch(KernelOf<1, 128>::fn, grid, kThreads, st, tm, a);
  return a.d == 64 ? launch(KernelOf<2, 64>::fn, grid, kThreads, st, tm, a)
                   : launch(KernelOf<2, 128>::fn, grid, kThreads, st, tm, a);
}

template <int DT, int D>
struct RowStatsOf {
  static constexpr auto fn = rowstats_kernel<DT, D>;
};
template <int DT, int D>
struct ScoreOf {
  static constexpr auto fn = score_kernel<DT, D>;
};

}  // namespace

hipError_t launch_rowstats(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch_typed<RowStatsOf>(dtype, a, grid, st, tm);
}

hipError_t launch_lse(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(lse_kernel, grid * (kMaxRows / kLseRows), kThreads, st, tm, a);
}

hipError_t launch_score(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch_typed<ScoreOf>(dtype, a, grid, st, tm);
}

}  // namespace ckv
