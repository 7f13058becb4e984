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
//   rowstats_kernel  pass 1: online max and sum of exp2 of every chosen row,
//                    one partial per workgroup;
//   score_kernel     pass 2: merges those partials into one log2-sum-exp2
//                    per row, then exp2(alpha*s - lse) summed over each
//                    chosen head's window rows, written per head (S[h,j]);
//   pool_kernel      pooling along the tokens, head mean, scores, and the
//                    first-level histogram of the score keys that the
//                    selection starts from.
//
// Work decomposition of the two K passes: a group's chosen rows are padded
// per head to a multiple of 8 and split into 32-row query blocks; each wave
// keeps one query block's operand in registers for its whole life. K is cut
// into 16 KB stages, and the P workgroups of a group take the stages
// round-robin (workgroup p: stages p, p+P, p+2P, ...), so at any moment the
// whole chip reads one compact window of each K head rather than hundreds of
// scattered streams; this keeps HBM near its streaming rate. Stages go
// through a ring of LDS slots filled by direct global-to-LDS loads
// (global_load_lds_dwordx4): every load instruction moves 1 KB of consecutive
// rows, and the loads of the next stages stay in flight (explicit partial
// vmcnt waits and a plain s_barrier, since a fenced barrier would drain
// them). Rows land in LDS with their 16-byte chunks XOR-swizzled so that the
// MFMA-layout reads (lane l takes token l % 32) spread over all banks. Logits
// come from v_mfma 32x32x16.
#include <math.h>

#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

// Waves per query block when a K-pass workgroup's waves share nqb blocks
// (nqb <= 4; 3 blocks use the 4-block split and leave the last waves idle).
__device__ __forceinline__ int waves_per_qblock(int nqb) {
  return nqb == 1 ? kKpWaves : (nqb == 2 ? kKpWaves / 2 : kKpWaves / 4);
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
// this wave are outstanding and all its LDS operations are done (gfx9
// encoding: vmcnt in bits 3:0 and 15:14, expcnt left at its no-wait maximum,
// lgkmcnt 0). The stage loop's barrier follows this wait: the window-sum
// fold reads LDS rows that other waves wrote in the previous step, so those
// writes must be complete when the barrier releases. The direct-to-LDS key
// loads count in vmcnt only, so this does not drain the key stream.
constexpr int vmcnt_imm(int n) { return 0x070 | (n & 15) | ((n >> 4) << 14); }

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
  static constexpr int PT = VEC / kKpThreads;    // load instructions per wave per stage
  static constexpr int BLOCKS = ST / 32;
  static_assert(ST % 32 == 0 && VEC % kKpThreads == 0, "stage shape");

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
      const int e = (k * kKpWaves + wave) * 64 + lane;
      const int t = e / NV, pos = e - t * NV;
      p.tok[k] = t;
      p.chunk[k] = pos ^ swz(t);
      p.off[k] = (int64_t)t * kv_st * EB + p.chunk[k] * 16;
    }
    return p;
  }

  // Issue the direct-to-LDS loads of the stage whose first token is t0, with
  // cache policy AUX (0, or kLoadNonTemporal). Tokens outside [lo, hi] read
  // row lo or hi instead (their results are never used); only stages that
  // cross lo or hi take that slower path.
  template <int AUX>
  __device__ static __forceinline__ void fetch(const char* kbase, int64_t kv_st, int64_t t0,
                                               int64_t lo, int64_t hi, const Plan& p, int wave,
                                               uint4* slot) {
    if (t0 >= lo && t0 + ST - 1 <= hi) {
      const char* sb = kbase + t0 * kv_st * EB;
#pragma unroll
      for (int k = 0; k < PT; ++k)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint4*>(sb + p.off[k]),
                                         slot + (k * kKpWaves + wave) * 64, 16, 0, AUX);
    } else {
#pragma unroll
      for (int k = 0; k < PT; ++k) {
        int64_t tok = t0 + p.tok[k];
        tok = tok < lo ? lo : (tok > hi ? hi : tok);
        const uint4* src = reinterpret_cast<const uint4*>(kbase + tok * kv_st * EB) + p.chunk[k];
        __builtin_amdgcn_global_load_lds(src, slot + (k * kKpWaves + wave) * 64, 16, 0, AUX);
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

// Cache policy of a load that is the last read of its data (gfx950 `nt`).
constexpr int kLoadNonTemporal = 2;

// Stage size: kStageBytes (at least one 32-token block).
template <int DT, int D>
constexpr int stage_bytes() {
  return stage_tokens(D * Elt<DT>::bytes) * D * Elt<DT>::bytes;
}

// Wait until at most n_after of this wave's later stages are still loading
// (each stage is PT load instructions per wave; n_after <= MAXA).
template <int PT, int MAXA>
__device__ __forceinline__ void wait_stages(int n_after) {
  static_assert(MAXA <= 6 && MAXA * PT <= 63, "vmcnt range");
  if (MAXA >= 6 && n_after >= 6) __builtin_amdgcn_s_waitcnt(vmcnt_imm(6 * PT));
  else if (MAXA >= 5 && n_after >= 5) __builtin_amdgcn_s_waitcnt(vmcnt_imm(5 * PT));
  else if (MAXA >= 4 && n_after >= 4) __builtin_amdgcn_s_waitcnt(vmcnt_imm(4 * PT));
  else if (MAXA >= 3 && n_after >= 3) __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * PT));
  else if (MAXA >= 2 && n_after >= 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * PT));
  else if (MAXA >= 1 && n_after >= 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm(PT));
  else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
}

// Stage loop shared by both passes over stages 0..ns-1 (stage k starts at
// token t_first + k*stride, tokens clamped to [lo, hi]) with an NS-slot LDS ring
// (slots are distinct LDS arrays so the compiler can tell the in-flight loads
// from the slot being read). After the first NS-1 stages are issued, pre()
// runs while they load. At step k: wait for stage k, barrier (stage k is
// complete and every wave has finished with stage k-1's slot), issue stage
// k+NS-1 into that freed slot, then body(slot, k) reduces stage k. The loads
// use cache policy AUX.
template <class S, int NS, int AUX, class Pre, class Body>
__device__ __forceinline__ void stage_loop(uint4* const* slot, const char* kbase, int64_t kv_st,
                                           int64_t t_first, int64_t stride, int ns, int64_t lo,
                                           int64_t hi, int wave, Pre pre, Body body) {
  const typename S::Plan p = S::plan(wave, kv_st);
  // Two workgroups share each CU; the one dispatched second is the younger,
  // and the SIMDs issue the older one's waves first, so it would finish
  // well after its partner and leave the CU half idle. It runs its first
  // 3/4 of the stages at a raised wave priority to even them out (a hint
  // only: results do not depend on it).
  const int prio_until = ((blockIdx.x / kCUs) & 1) ? ns * 3 / 4 : 0;
  if (prio_until > 0) __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int j = 0; j < NS - 1; ++j)
    if (j < ns) S::template fetch<AUX>(kbase, kv_st, t_first + j * stride, lo, hi, p, wave, slot[j]);
  pre();  // work that overlaps the first stages' loads
  for (int k0 = 0; k0 < ns; k0 += NS) {
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int k = k0 + j;
      if (k < ns) {
        const int left = ns - 1 - k;
        if (k == prio_until && prio_until > 0) __builtin_amdgcn_s_setprio(0);
        wait_stages<S::PT, NS - 2>(left < NS - 2 ? left : NS - 2);
        __builtin_amdgcn_s_barrier();
        if (k + NS - 1 < ns)
          S::template fetch<AUX>(kbase, kv_st, t_first + (k + NS - 1) * stride, lo, hi, p, wave,
                   slot[(j + NS - 1) % NS]);
        body(slot[j], k);
      }
    }
  }
  __syncthreads();
}

// Operand-reading and MFMA part shared by both passes: the wave's blocks of a
// stage are sub, sub + WPQ, ... (NB of them; the caller guarantees that they
// lie inside the stage) and its NQ query blocks' operands are q[0..NQ);
// acc[j][i] receives the 32x32 logit tile of query block j and key block i,
// queries x keys when KEYS_AS_ROWS is false, keys x queries otherwise. Every
// key operand is read from LDS once and used for all NQ query blocks, and the
// NQ*NB accumulation chains are interleaved, so the MFMA pipe never waits on
// a single dependent chain. Blocks past the prompt are computed too (their
// LDS rows are clamped copies) and the caller ignores them.
template <int DT, class S, int WPQ, int NQ, bool KEYS_AS_ROWS>
__device__ __forceinline__ void stage_tiles(const uint4* slot, const int* opoff,
                                            const uint4 (*q)[S::NC], f32x16 (*acc)[(S::BLOCKS + WPQ - 1) / WPQ]) {
  constexpr int NB = (S::BLOCKS + WPQ - 1) / WPQ;
  constexpr int NC = S::NC;
  uint4 kr[NB][NC];
#pragma unroll
  for (int i = 0; i < NB; ++i) S::operand(slot, i * WPQ, opoff, kr[i]);
#pragma unroll
  for (int j = 0; j < NQ; ++j)
#pragma unroll
    for (int i = 0; i < NB; ++i) acc[j][i] = f32x16{};
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int j = 0; j < NQ; ++j)
#pragma unroll
      for (int i = 0; i < NB; ++i)
        acc[j][i] = KEYS_AS_ROWS ? mfma_chunk<DT>(kr[i][c], q[j][c], acc[j][i])
                                 : mfma_chunk<DT>(q[j][c], kr[i][c], acc[j][i]);
}

// Stages of workgroup p of P over n_tok tokens: p, p+P, ... (none if p is
// past the last stage).
__device__ __forceinline__ int stages_of(int64_t n_tok, int st, int p, int P) {
  const int64_t n_st = (n_tok + st - 1) / st;
  return p < n_st ? (int)((n_st - p + P - 1) / P) : 0;
}

// Prompt and local workgroup index of workgroup b in a grid laid out by the
// per-prompt first-workgroup offsets off(t).
template <class Off>
__device__ __forceinline__ int find_seq(const LayerArgs& a, int b, Off off) {
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= off(a.seq[t])) s = t;
  return s;
}

// For K-pass workgroup `local` of a prompt: its KV group g, the row group
// (unit) j of that group, the unit's index u among the prompt's units, and
// the workgroup's index p among the unit's P workgroups (units are laid out
// in group order, group_split workgroups each).
__device__ __forceinline__ void kpass_locate(const LayerArgs& a, const SeqArgs& sq, int local,
                                             int& g, int& j, int& u, int& p, int& P) {
  int base = 0;
  u = 0;
  for (g = 0; g < a.n_kv; ++g) {
    const int cnt = a.grp_off[g + 1] - a.grp_off[g];
    const int nu = group_units(cnt, a.hpr);
    for (j = 0; j < nu; ++j, ++u) {
      P = group_split((unit_heads(cnt, a.hpr, j) * a.w8 + 31) >> 5, a.split_w, sq.n_split);
      if (local < base + P) {
        p = local - base;
        return;
      }
      base += P;
    }
  }
  // past the prompt's workgroups (the host launches exactly their number):
  // an empty unit
  g = a.n_kv - 1;
  j = group_units(a.grp_off[a.n_kv] - a.grp_off[g], a.hpr);
  p = P = 1;
}

// Causal mask of a 32-key block of window-sum logits (pass 2's layout: lane
// half h holds rows qb*32 + acc_row(v, h) of key tok): window row i of a
// head (padded row index modulo w8) sees keys up to Lw + i, where Lw = L - w
// is the window's first position. Only blocks that reach the window need it,
// and only when the window columns are scored (the keep-window flag off).
__device__ __forceinline__ void mask_window_block(f32x16& acc, int qb, int64_t tok, int64_t Lw,
                                                  int w8, int h) {
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int iw = (qb * 32 + acc_row(v, h)) % w8;
    if (tok > Lw + iw) acc[v] = -INFINITY;
  }
}

// ---------------------------------------------------------------------------
// Pass 1: row statistics.
// ---------------------------------------------------------------------------
template <int DT, int D, int WPQ, int NQ, class S, int NS>
__device__ __forceinline__ void rowstats_body(const LayerArgs& a, const SeqArgs& sq, int g, int u,
                                              int p, int P, int sel0, int n_sel, int nqb,
                                              uint4* const* slots, float2 (*red)[2][32]) {
  constexpr int NC = S::NC;
  constexpr int NB = (S::BLOCKS + WPQ - 1) / WPQ;
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int qg = wave / WPQ, sub = wave % WPQ;  // query group: blocks qg*NQ .. qg*NQ+NQ-1
  const int w8 = a.w8;
  const int64_t L = sq.L, Ls = L - a.w;
  const int64_t stride = (int64_t)P * S::ST;
  const float alpha = a.alpha;
  const char* kbase = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * S::EB;
  const int ns = stages_of(L, S::ST, p, P);
  const bool active = qg * NQ < nqb;

  // this lane's query row in each of its blocks (column of the MFMA result)
  // and that row's last visible key
  uint4 q[NQ][NC];
  int64_t last[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const int qb = qg * NQ + j;
    last[j] = Ls + (qb * 32 + l32) % w8;  // >= L for padding rows
    if (qb < nqb) load_queries<NC, S::EB>(a, sq, sel0, n_sel, qb, l32, h, q[j]);
    else
#pragma unroll
      for (int c = 0; c < NC; ++c) q[j][c] = make_uint4(0u, 0u, 0u, 0u);
  }
  int opoff[NC];
  S::operand_offsets(l32, h, opoff);
#pragma unroll
  for (int c = 0; c < NC; ++c) opoff[c] += sub * 32 * S::ROWB;
  float m_run[NQ], z_run[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    m_run[j] = -INFINITY;
    z_run[j] = 0.f;
  }

  // the keys stay cacheable: the window-sum pass that follows reads the
  // same keys, and finds part of them in the Infinity Cache
  stage_loop<S, NS, 0>(slots, kbase, sq.kv_st, (int64_t)p * S::ST, stride, ns, 0, L - 1, wave,
                    [] {}, [&](const uint4* slot, int k) {
    // waves past the stage's blocks (4 waves on a 2-block stage) sit out
    if (!active || sub >= S::BLOCKS) return;
    const int64_t ts = (int64_t)p * S::ST + k * stride + sub * 32;  // this wave's first block
    f32x16 acc[NQ][NB];
    stage_tiles<DT, S, WPQ, NQ, true>(slot, opoff, q, acc);
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      if (qg * NQ + j >= nqb) continue;  // a query block past the group's rows (uniform)
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        // acc[j][i][v]: key t0 + acc_row(v, h) of this lane's query row
        const int64_t t0 = ts + i * WPQ * 32;
        if (t0 + 32 > Ls) {  // keys inside the window or past the prompt: causal
                             // mask (a uniform branch; blocks past L mask all)
          const int64_t rel = last[j] - t0;
          const int lim = rel < -1 ? -1 : (rel > 32 ? 32 : (int)rel);
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (acc_row(v, h) > lim) acc[j][i][v] = -INFINITY;
        }
        float mx = acc[j][i][0];
#pragma unroll
        for (int v = 1; v < 16; ++v) mx = fmaxf(mx, acc[j][i][v]);
        const float m_new = fmaxf(m_run[j], mx);
        const float ms = m_new == -INFINITY ? 0.f : m_new * alpha;
        float z = z_run[j] * fast_exp2(m_run[j] * alpha - ms);
#pragma unroll
        for (int v = 0; v < 16; ++v) z += fast_exp2(fmaf(acc[j][i][v], alpha, -ms));
        z_run[j] = z;
        m_run[j] = m_new;
      }
    }
  });

  // merge the two lane halves (same query row, different keys), then the
  // waves that share the query group
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const float mo = __shfl_xor(m_run[j], 32);
    const float zo = __shfl_xor(z_run[j], 32);
    const float mn = fmaxf(m_run[j], mo);
    const float msn = mn == -INFINITY ? 0.f : mn * alpha;
    const float z = z_run[j] * fast_exp2(m_run[j] * alpha - msn) + zo * fast_exp2(mo * alpha - msn);
    if (h == 0) red[wave][j][l32] = make_float2(mn, z);
  }
  __syncthreads();
  if (tid < nqb * 32) {
    const int qq = tid >> 5, r = tid & 31;
    const int qgq = qq / NQ, jq = qq - qgq * NQ;
    float m = -INFINITY;
#pragma unroll
    for (int sw = 0; sw < WPQ; ++sw) m = fmaxf(m, red[qgq * WPQ + sw][jq][r].x);
    const float ms = m == -INFINITY ? 0.f : m * alpha;
    float z = 0.f;
#pragma unroll
    for (int sw = 0; sw < WPQ; ++sw)
      z += red[qgq * WPQ + sw][jq][r].y * fast_exp2(red[qgq * WPQ + sw][jq][r].x * alpha - ms);
    sq.partial[((int64_t)u * sq.n_split + p) * kMaxRows + tid] = make_float2(m, z);
  }
}

template <int DT, int D>
__device__ __forceinline__ void rowstats_block(const LayerArgs& a, const int b) {
  using S = Stager<DT, D, stage_bytes<DT, D>()>;
  constexpr int NS = 4;  // 4-slot ring
  __shared__ uint4 slot0[S::VEC];
  __shared__ uint4 slot1[S::VEC];
  __shared__ uint4 slot2[S::VEC];
  __shared__ uint4 slot3[S::VEC];
  __shared__ float2 red[kKpWaves][2][32];
  uint4* const slots[NS] = {slot0, slot1, slot2, slot3};

  const SeqArgs& sq = a.seq[find_seq(a, b, [](const SeqArgs& t) { return t.blk_kpass; })];
  int g, j, u, p, P;
  kpass_locate(a, sq, b - sq.blk_kpass, g, j, u, p, P);
  const int cnt = a.grp_off[g + 1] - a.grp_off[g];
  const int sel0 = a.grp_off[g] + j * a.hpr;
  const int n_sel = j < group_units(cnt, a.hpr) && cnt > 0 ? unit_heads(cnt, a.hpr, j) : 0;
  const int nqb = (n_sel * a.w8 + 31) >> 5;

  // the selection state starts from zero in every call (one per group, or
  // one per prompt when shared); the pooling kernel that accumulates into it
  // runs after this one
  if (p == 0 && j == 0 && a.do_hist && g < a.n_sg) {
    for (int i = threadIdx.x; i < kCtlWords; i += kKpThreads) sq.ctl[g * kCtlWords + i] = 0u;
    for (int i = threadIdx.x; i < kHistBins; i += kKpThreads)
      sq.hist[(int64_t)g * kHistBins + i] = 0u;
  }
  if (n_sel == 0) return;  // a group without chosen heads (shared scope) is not read
  const int wpq = waves_per_qblock(nqb);
  constexpr int W1 = kKpWaves, W2 = kKpWaves / 2, W4 = kKpWaves / 4;
  // 3-4 query blocks on a stage of 2+ key blocks: each wave takes two query
  // blocks and half the key blocks, so every key operand is read from LDS by
  // two waves instead of four
  if (S::BLOCKS >= 2 && nqb >= 3)
    rowstats_body<DT, D, 2, 2, S, NS>(a, sq, g, u, p, P, sel0, n_sel, nqb, slots, red);
  else if (wpq == W4) rowstats_body<DT, D, W4, 1, S, NS>(a, sq, g, u, p, P, sel0, n_sel, nqb, slots, red);
  else if (wpq == W2) rowstats_body<DT, D, W2, 1, S, NS>(a, sq, g, u, p, P, sel0, n_sel, nqb, slots, red);
  else rowstats_body<DT, D, W1, 1, S, NS>(a, sq, g, u, p, P, sel0, n_sel, nqb, slots, red);
}

template <int DT, int D>
__global__ __launch_bounds__(kKpThreads) __attribute__((amdgpu_waves_per_eu(2))) void rowstats_kernel(const LayerArgs a) {
  rowstats_block<DT, D>(a, blockIdx.x);
}

// The layer of workgroup b of a multi-layer K-pass launch.
__device__ __forceinline__ int layer_of(const LayersArgs& m, int b) {
  int l = 0;
#pragma unroll
  for (int i = 1; i < kLayersPerLaunch; ++i)
    if (i < m.n && b >= m.blk[i]) l = i;
  return l;
}

// The row-statistics passes of up to kLayersPerLaunch layers in one launch,
// layer l's workgroups at blk[l] .. blk[l+1]: one ramp-up and drain for them
// all.
template <int DT, int D>
__global__ __launch_bounds__(kKpThreads) __attribute__((amdgpu_waves_per_eu(2))) void rowstats_layers_kernel(const LayersArgs m) {
  const int l = layer_of(m, blockIdx.x);
  rowstats_block<DT, D>(m.lay[l], blockIdx.x - m.blk[l]);
}

// Online merge of (max logit, sum of exp2) pairs in exp2 units.
__device__ __forceinline__ void lse_merge(float& m, float& z, float m2, float z2, float alpha) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;  // both empty
  const float ms = mn * alpha;
  z = z * fast_exp2(m * alpha - ms) + z2 * fast_exp2(m2 * alpha - ms);
  m = mn;
}

// ---------------------------------------------------------------------------
// Pass 2: probabilities and per-head window sums.
// ---------------------------------------------------------------------------
constexpr int kGroupRows = kMaxRows / 8;  // 8-row groups of one group's rows
constexpr int kLseBatch = 16;             // partial loads in flight per thread
constexpr int kMergeLanes = kKpThreads / kMaxRows;  // threads per row in the lse merge

// QM (query-block mode, when w8 is a multiple of 32): every 32-row query
// block belongs to one head, so a lane sums its four 8-row groups in
// registers and the block's column sums are one row of gsum; otherwise
// gsum holds one row per 8-row group. DIRECT > 0 (QM, every head's DIRECT
// query blocks inside one wave's NQ): the wave adds its head's block sums in
// registers, in the order the fold would, and stores the window sums itself,
// so gsum and the fold are not used.
template <int DT, int D, int WPQ, int NQ, bool QM, int DIRECT, class S, int NS>
__device__ __forceinline__ void score_body(const LayerArgs& a, const SeqArgs& sq, int g, int u,
                                           int hs0, int p, int P, int sel0, int n_sel, int nqb,
                                           uint4* const* slots, float* gsum) {
  constexpr int NC = S::NC;
  constexpr int NB = (S::BLOCKS + WPQ - 1) / WPQ;
  constexpr int ST = S::ST;
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int qg = wave / WPQ, sub = wave % WPQ;  // query group: blocks qg*NQ .. qg*NQ+NQ-1
  const bool active = qg * NQ < nqb;
  // scored columns [0, Ls): the prefix when the window is kept by rule, the
  // whole prompt otherwise (window columns then take the causal mask)
  const int64_t Lw = sq.L - a.w, Ls = sq.L - a.tail;
  const bool window_cols = a.tail == 0;
  const int64_t stride = (int64_t)P * ST;
  const float alpha = a.alpha;
  const char* kbase = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * S::EB;
  const int ns = stages_of(Ls, ST, p, P);

  uint4 q[NQ][NC];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    if (qg * NQ + j < nqb) load_queries<NC, S::EB>(a, sq, sel0, n_sel, qg * NQ + j, l32, h, q[j]);
    else
#pragma unroll
      for (int c = 0; c < NC; ++c) q[j][c] = make_uint4(0u, 0u, 0u, 0u);
  }
  // lse of this lane's 16 result rows qb*32 + 8*a4 + 4*h + e of each of its
  // query blocks qb, in exp2 units: merged from pass 1's per-workgroup
  // partials while the first stages load
  float4 cv[NQ][4];
  auto merge_lse = [&] {
    // kMergeLanes threads per row, thread j merging partials j, j + kMergeLanes,
    // ...; their results meet in LDS in a fixed order (the gsum buffers are
    // not in use yet)
    float2* part = reinterpret_cast<float2*>(gsum);      // [kMergeLanes][kMaxRows]
    float* lse_l = gsum + 2 * kMergeLanes * kMaxRows;     // [kMaxRows]
    const int r = tid % kMaxRows, half = tid / kMaxRows;
    const int slot_h = r / a.w8, wrow = r - slot_h * a.w8;
    const bool valid = r < nqb * 32 && slot_h < n_sel && wrow < a.w;
    float m = -INFINITY, z = 0.f;
    if (valid && !a.lse_given) {
      const float2* pp = sq.partial + (int64_t)u * sq.n_split * kMaxRows + r;
      for (int c0 = half; c0 < P; c0 += kMergeLanes * kLseBatch) {
        float2 v[kLseBatch];
#pragma unroll
        for (int u = 0; u < kLseBatch; ++u) {
          const int c = c0 + kMergeLanes * u;
          v[u] = c < P ? pp[(int64_t)c * kMaxRows] : make_float2(-INFINITY, 0.f);
        }
#pragma unroll
        for (int u = 0; u < kLseBatch; ++u) lse_merge(m, z, v[u].x, v[u].y, alpha);
      }
    }
    part[half * kMaxRows + r] = make_float2(m, z);
    __syncthreads();
    if (tid < kMaxRows) {
      float mm = part[r].x, zz = part[r].y;
#pragma unroll
      for (int j = 1; j < kMergeLanes; ++j)
        lse_merge(mm, zz, part[j * kMaxRows + r].x, part[j * kMaxRows + r].y, alpha);
      // padding rows: +inf, so their probabilities are 0. Caller row
      // statistics are natural logs of the scaled logits' normaliser:
      // log2(e) times that is the same quantity in exp2 units.
      float v = INFINITY;
      if (valid)
        v = a.lse_given ? sq.lse[(int64_t)a.sel[sel0 + slot_h] * sq.lse_sh + wrow] * 1.4426950408889634f
                        : mm * alpha + log2f(zz);
      lse_l[r] = v;
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int j = 0; j < NQ; ++j)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          // rows of a block past nqb are padding (+inf) and never used
          const float* src = lse_l + (qg * NQ + j) * 32 + 8 * a4 + 4 * h;
          cv[j][a4] = make_float4(src[0], src[1], src[2], src[3]);
        }
    }
    __syncthreads();  // lse_l and part are gsum, which stage 0 overwrites
  };
  int opoff[NC];
  S::operand_offsets(l32, h, opoff);
#pragma unroll
  for (int c = 0; c < NC; ++c) opoff[c] += sub * 32 * S::ROWB;

  // Head window sums of stage kk: the head in slot hs owns gsum rows
  // [hs*rph, (hs+1)*rph) of buffer kk % 2 (rph = its query blocks in QM, its
  // 8-row groups otherwise); their fixed-order sum is written to
  // wsum[g][hs][token].
  const int rph = QM ? a.w8 / 32 : a.w8 / 8;
  float* wsum_g = sq.wsum + ((int64_t)g * sq.wsum_heads + hs0) * sq.ws_stride;  // this unit's heads
  auto fold = [&](int kk) {
    const float* gb = gsum + (kk & 1) * (kGroupRows * ST);
    const int64_t t0 = (int64_t)p * ST + kk * stride;
    for (int e = tid; e < n_sel * ST; e += kKpThreads) {
      const int hs = e / ST, c = e - hs * ST;
      if (t0 + c >= Ls) continue;
      float acc = gb[(hs * rph) * ST + c];
      for (int q8 = 1; q8 < rph; ++q8) acc += gb[(hs * rph + q8) * ST + c];
      __builtin_nontemporal_store(acc, wsum_g + (int64_t)hs * sq.ws_stride + t0 + c);
    }
  };

  // the last read of these keys: non-temporal loads leave the caches to the
  // data still to be read
  stage_loop<S, NS, kLoadNonTemporal>(slots, kbase, sq.kv_st, (int64_t)p * ST, stride, ns, 0,
                                      Ls - 1, wave,
                    merge_lse, [&](const uint4* slot, int k) {
    // the barrier before this step ordered every wave's gsum writes of stage
    // k-1 before these reads, and this fold's reads before stage k+1 reuses
    // the buffer
    if (DIRECT == 0 && k > 0) fold(k - 1);
    // waves past the stage's blocks (4 waves on a 2-block stage) sit out
    if (!active || sub >= S::BLOCKS) return;
    f32x16 acc[NQ][NB];
    stage_tiles<DT, S, WPQ, NQ, false>(slot, opoff, q, acc);
    const int64_t ts = (int64_t)p * ST + (int64_t)k * stride;  // the stage's first key
    if (window_cols && ts + ST > Lw) {  // a stage that reaches the window (uniform)
#pragma unroll
      for (int j = 0; j < NQ; ++j)
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int64_t t0 = ts + (sub + i * WPQ) * 32;
          if (t0 + 32 > Lw) mask_window_block(acc[j][i], qg * NQ + j, t0 + l32, Lw, a.w8, h);
        }
    }
    if constexpr (DIRECT > 0) {
      static_assert(QM && NQ % (DIRECT > 0 ? DIRECT : 1) == 0, "whole heads per wave");
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        // column sums of tile (j, i) over its 32 query rows, as in QM below
        float tq[NQ];
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
          float gs[4];
#pragma unroll
          for (int a4 = 0; a4 < 4; ++a4)
            gs[a4] = fast_exp2(fmaf(acc[j][i][4 * a4 + 0], alpha, -cv[j][a4].x)) +
                     fast_exp2(fmaf(acc[j][i][4 * a4 + 1], alpha, -cv[j][a4].y)) +
                     fast_exp2(fmaf(acc[j][i][4 * a4 + 2], alpha, -cv[j][a4].z)) +
                     fast_exp2(fmaf(acc[j][i][4 * a4 + 3], alpha, -cv[j][a4].w));
          tq[j] = (gs[0] + gs[1]) + (gs[2] + gs[3]);
          tq[j] += __shfl_xor(tq[j], 32);
        }
        const int64_t tok = ts + (sub + i * WPQ) * 32 + l32;
#pragma unroll
        for (int hw = 0; hw < NQ / DIRECT; ++hw) {
          const int hs = qg * (NQ / DIRECT) + hw;
          float t = tq[hw * DIRECT];
#pragma unroll
          for (int jj = 1; jj < DIRECT; ++jj) t += tq[hw * DIRECT + jj];
          if (h == 0 && hs < n_sel && tok < Ls) __builtin_nontemporal_store(t, wsum_g + (int64_t)hs * sq.ws_stride + tok);
        }
      }
      return;
    }
    float* gb = gsum + (k & 1) * (kGroupRows * ST);
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      const int qb = qg * NQ + j;
      if (qb >= nqb) continue;  // a query block past the group's rows (uniform)
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        // columns at or past Ls get values too; the fold never writes them out
        // acc[j][i][v]: query row qb*32 + acc_row(v, h), key (sub + i*WPQ)*32 +
        // l32 of the stage; prefix keys are visible to every window row, and
        // scored window keys were masked above.
        float gs[4];
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4)
          gs[a4] = fast_exp2(fmaf(acc[j][i][4 * a4 + 0], alpha, -cv[j][a4].x)) +
                   fast_exp2(fmaf(acc[j][i][4 * a4 + 1], alpha, -cv[j][a4].y)) +
                   fast_exp2(fmaf(acc[j][i][4 * a4 + 2], alpha, -cv[j][a4].z)) +
                   fast_exp2(fmaf(acc[j][i][4 * a4 + 3], alpha, -cv[j][a4].w));
        const int col = (sub + i * WPQ) * 32 + l32;
        if (QM) {
          float t = (gs[0] + gs[1]) + (gs[2] + gs[3]);
          t += __shfl_xor(t, 32);
          if (h == 0) gb[qb * ST + col] = t;
        } else {
#pragma unroll
          for (int a4 = 0; a4 < 4; ++a4) gs[a4] += __shfl_xor(gs[a4], 32);
          // lane half h stores 8-row groups a4 = h and h + 2
          gb[(qb * 4 + h) * ST + col] = h ? gs[1] : gs[0];
          gb[(qb * 4 + 2 + h) * ST + col] = h ? gs[3] : gs[2];
        }
      }
    }
  });
  // stage_loop ended with a barrier: the last stage's sums are complete
  if (DIRECT == 0 && ns > 0) fold(ns - 1);
}

template <int DT, int D>
__device__ __forceinline__ void score_block(const LayerArgs& a, const int b) {
  using S = Stager<DT, D, stage_bytes<DT, D>()>;
  constexpr int NS = 4;  // 4-slot ring
  __shared__ uint4 slot0[S::VEC];
  __shared__ uint4 slot1[S::VEC];
  __shared__ uint4 slot2[S::VEC];
  __shared__ uint4 slot3[S::VEC];
  // gsum[buf][r8][col]: sum over the 8 rows of 8-row group r8 of p at stage
  // column col, double-buffered by stage parity
  __shared__ __align__(16) float gsum[2 * kGroupRows * S::ST];
  static_assert(2 * kGroupRows * S::ST >= (2 * kMergeLanes + 1) * kMaxRows, "the lse merge fits in gsum");
  uint4* const slots[NS] = {slot0, slot1, slot2, slot3};

  const SeqArgs& sq = a.seq[find_seq(a, b, [](const SeqArgs& t) { return t.blk_kpass; })];
  // the selection stages of a multi-layer launch read this layer's argument
  // block from device memory: workgroup 0 puts it there
  if (a.table_out && b == 0) {
    static_assert(sizeof(LayerArgs) % 16 == 0, "argument block in 16-byte words");
    const uint4* src = reinterpret_cast<const uint4*>(&a);
    uint4* dst = static_cast<uint4*>(a.table_out);
    for (int i = threadIdx.x; i < (int)(sizeof(LayerArgs) / 16); i += kKpThreads) dst[i] = src[i];
  }
  int g, j, u, p, P;
  kpass_locate(a, sq, b - sq.blk_kpass, g, j, u, p, P);
  const int cnt = a.grp_off[g + 1] - a.grp_off[g];
  const int sel0 = a.grp_off[g] + j * a.hpr;
  const int n_sel = j < group_units(cnt, a.hpr) && cnt > 0 ? unit_heads(cnt, a.hpr, j) : 0;
  // without the row-statistics pass, this pass starts the selection state
  // from zero (the pooling kernel that accumulates into it runs after it)
  if (a.lse_given && p == 0 && j == 0 && a.do_hist && g < a.n_sg) {
    for (int i = threadIdx.x; i < kCtlWords; i += kKpThreads) sq.ctl[g * kCtlWords + i] = 0u;
    for (int i = threadIdx.x; i < kHistBins; i += kKpThreads)
      sq.hist[(int64_t)g * kHistBins + i] = 0u;
  }
  if (n_sel == 0) return;  // a group without chosen heads (shared scope) is not read
  const int nqb = (n_sel * a.w8 + 31) >> 5;
  const int wpq = waves_per_qblock(nqb);
  constexpr int W1 = kKpWaves, W2 = kKpWaves / 2, W4 = kKpWaves / 4;
  // the same wave mapping as the row-statistics pass
  const bool pair = S::BLOCKS >= 2 && nqb >= 3;
  if (pair && a.w8 == 64) {  // each wave's two query blocks are one head
    score_body<DT, D, 2, 2, true, 2, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
  } else if (pair && a.w8 == 32) {  // each query block is a head
    score_body<DT, D, 2, 2, true, 1, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
  } else if (a.w8 % 32 == 0) {
    if (pair) score_body<DT, D, 2, 2, true, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
    else if (wpq == W4) score_body<DT, D, W4, 1, true, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
    else if (wpq == W2) score_body<DT, D, W2, 1, true, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
    else score_body<DT, D, W1, 1, true, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
  } else {
    if (pair) score_body<DT, D, 2, 2, false, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
    else if (wpq == W4) score_body<DT, D, W4, 1, false, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
    else if (wpq == W2) score_body<DT, D, W2, 1, false, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
    else score_body<DT, D, W1, 1, false, 0, S, NS>(a, sq, g, u, j * a.hpr, p, P, sel0, n_sel, nqb, slots, gsum);
  }
}

template <int DT, int D>
__global__ __launch_bounds__(kKpThreads) __attribute__((amdgpu_waves_per_eu(2))) void score_kernel(const LayerArgs a) {
  score_block<DT, D>(a, blockIdx.x);
}

// The window-sum passes of up to kLayersPerLaunch layers in one launch.
template <int DT, int D>
__global__ __launch_bounds__(kKpThreads) __attribute__((amdgpu_waves_per_eu(2))) void score_layers_kernel(const LayersArgs m) {
  const int l = layer_of(m, blockIdx.x);
  score_block<DT, D>(m.lay[l], blockIdx.x - m.blk[l]);
}

// ---------------------------------------------------------------------------
// Pooling along the tokens, head mean, scores and the selection histogram.
// One workgroup per (prompt, selection group, kPoolTile scores), where the
// selection group is the KV group, or the whole layer when the selection is
// shared (then the mean runs over every chosen head); thread t owns the
// kPoolPer consecutive scores starting at t * kPoolPer. Window-sum rows are
// padded to a multiple of 4 floats, so a thread reads its scores and an
// R-wide halo on each side (rounded up to 4) with aligned 16-byte loads
// straight from global memory, the pool radius R being a template parameter
// so that only the needed taps are evaluated. The workgroup's histogram
// lives in LDS as packed 16-bit counters (a tile has at most 2048 scores),
// which keeps the kernel small enough in LDS to share a CU with two K-pass
// workgroups.
// ---------------------------------------------------------------------------
static_assert(kPoolPer * kThreads == kPoolTile && kUnitPoolTiles * kPoolTile <= 65535,
              "8 scores per thread, 16-bit bin counts");

// What one pooling workgroup needs, resolved from the argument block in the
// kernel itself (passing the block by reference down the radius dispatch
// would make the compiler copy it to scratch memory).
struct PoolJob {
  const float* const* rows;  // LDS table: window sums of the heads averaged
  int n_heads;
  int64_t Ls, j0;            // prefix length, first score of the first tile
  int n_out;                 // scores in this workgroup's tiles
  bool is_max, do_hist;
  float inv_kp;
  CKV_GLOBAL float* out;     // scores of the first tile
  uint32_t* ghist;           // the selection group's histogram
};

// Pools the workgroup's span of n_out <= KM * 4 * kThreads scores. Thread tid owns the
// 4-token chunks k = 0 .. KM-1 at offset (k * kThreads + tid) * 4, so that
// consecutive lanes load and store consecutive 16 bytes; the halo chunks come
// from the neighbouring lanes' loads (lanes at a wave's edge load theirs).
// All of a head's loads for a batch of KB chunks are issued before the first
// is used: a dependent load per chunk would leave the span latency-bound.
template <int R, int KM>
__device__ __forceinline__ void pool_tile(const PoolJob& jb, uint32_t* hist_lds) {
  constexpr int CH = (R + 3) / 4;  // 16-byte halo chunks on each side of an output chunk
  constexpr int NX = 4 * (2 * CH + 1);
  // chunks whose loads are in flight together (a main and a halo load each):
  // 2, or 1 with wider halos. Against one chunk at a time this measured 6%
  // faster on 32 layers of 131072 tokens, 15% on the ragged Qwen batch and
  // 30% on 32 layers of 32768 tokens; 8 at a time was 10% slower than one at
  // a time on the 131072-token layers
  constexpr int KB0 = CH <= 1 ? 2 : 1;
  constexpr int KB = KB0 < KM ? KB0 : KM;
  static_assert(KM % KB == 0, "chunk batches");
  const int tid = threadIdx.x, lane = tid & 63;
  const float pad = jb.is_max ? -INFINITY : 0.f;  // max ignores padding; avg counts it as 0
  const int64_t Ls = jb.Ls;
  // 16 bytes at token j (a multiple of 4), read unconditionally: positions
  // outside [0, Ls) read token 0 and are replaced by the padding afterwards;
  // rows are padded to a multiple of 4 floats, so j < Ls stays inside the row
  auto raw = [&](const CKV_GLOBAL float* row, int64_t j) {
    return *(const CKV_GLOBAL f32x4*)(row + (j >= 0 && j < Ls ? j : 0));
  };
  auto fix = [&](f32x4 c, int64_t j) {
    const bool in = j >= 0 && j < Ls;
    c.x = in ? c.x : pad;
    c.y = in && j + 1 < Ls ? c.y : pad;
    c.z = in && j + 2 < Ls ? c.z : pad;
    c.w = in && j + 3 < Ls ? c.w : pad;
    return c;
  };
#pragma unroll 1
  for (int k0 = 0; k0 < KM; k0 += KB) {
    float total[KB][4];
#pragma unroll
    for (int k = 0; k < KB; ++k)
      total[k][0] = total[k][1] = total[k][2] = total[k][3] = 0.f;
    for (int hh = 0; hh < jb.n_heads; ++hh) {
      const CKV_GLOBAL float* row = to_global(jb.rows[hh]);
      f32x4 c[KB], e[KB][CH];
#pragma unroll
      for (int k = 0; k < KB; ++k) c[k] = raw(row, jb.j0 + ((k0 + k) * kThreads + tid) * 4);
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const int64_t j = jb.j0 + ((k0 + k) * kThreads + tid) * 4;
#pragma unroll
        // every lane loads the chunk q away on its side of the wave, though
        // only the q edge lanes use it: a load under a branch would make the
        // compiler wait for every load before the first use
        for (int q = 1; q <= CH; ++q) e[k][q - 1] = raw(row, lane < 32 ? j - 4 * q : j + 4 * q);
      }
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const int64_t j = jb.j0 + ((k0 + k) * kThreads + tid) * 4;
        const f32x4 ck = fix(c[k], j);
        float x[NX];
        x[4 * CH] = ck.x;
        x[4 * CH + 1] = ck.y;
        x[4 * CH + 2] = ck.z;
        x[4 * CH + 3] = ck.w;
#pragma unroll
        for (int q = 1; q <= CH; ++q) {
          f32x4 lo, hi;
          lo.x = __shfl_up(ck.x, q); lo.y = __shfl_up(ck.y, q);
          lo.z = __shfl_up(ck.z, q); lo.w = __shfl_up(ck.w, q);
          hi.x = __shfl_down(ck.x, q); hi.y = __shfl_down(ck.y, q);
          hi.z = __shfl_down(ck.z, q); hi.w = __shfl_down(ck.w, q);
          if (lane < q) lo = fix(e[k][q - 1], j - 4 * q);
          if (lane + q >= 64) hi = fix(e[k][q - 1], j + 4 * q);
          const int l0 = 4 * (CH - q), h0 = 4 * (CH + q);
          x[l0] = lo.x; x[l0 + 1] = lo.y; x[l0 + 2] = lo.z; x[l0 + 3] = lo.w;
          x[h0] = hi.x; x[h0 + 1] = hi.y; x[h0 + 2] = hi.z; x[h0 + 3] = hi.w;
        }
        // both pools, one select: a branch on the pool kind per tap would split
        // the chunk into many small blocks
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float vm = x[4 * CH + u], va = vm;
#pragma unroll
          for (int dt = 1; dt <= R; ++dt) {
            const float a = x[4 * CH + u - dt], b = x[4 * CH + u + dt];
            vm = fmaxf(vm, fmaxf(a, b));
            va += a + b;
          }
          total[k][u] += jb.is_max ? vm : va * jb.inv_kp;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int t_off = ((k0 + k) * kThreads + tid) * 4;  // first token of the chunk in the span
      const int n_mine = jb.n_out - t_off;                // its scores inside the workgroup's range
      if (n_mine <= 0) continue;
      float sc[4];
      uint32_t bin[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        sc[u] = total[k][u] / (float)jb.n_heads;
        bin[u] = score_key(sc[u]) >> kHistShift;
      }
      CKV_GLOBAL float* o = jb.out + t_off;
      if (n_mine >= 4 && ((uintptr_t)o & 15u) == 0) {
        f32x4 w4 = {sc[0], sc[1], sc[2], sc[3]};
        *(CKV_GLOBAL f32x4*)o = w4;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (u < n_mine) o[u] = sc[u];
      }
      if (jb.do_hist) {
        // one LDS atomic per run of equal bins among the chunk's scores (max
        // pooling makes plateaus), not one per score
        uint32_t run = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (u >= n_mine) break;
          ++run;
          if (u + 1 < 4 && u + 1 < n_mine && bin[u + 1] == bin[u]) continue;
          atomicAdd(&hist_lds[bin[u] >> 1], run << ((bin[u] & 1u) * 16u));
          run = 0;
        }
      }
    }
  }
  if (!jb.do_hist) return;
  // this tile's part of the selection group's first-level histogram
  __syncthreads();
  for (int i = tid; i < kHistBins / 2; i += kThreads) {
    const uint32_t c = hist_lds[i];
    if (c & 0xFFFFu) atomicAdd(&jb.ghist[2 * i], c & 0xFFFFu);
    if (c >> 16) atomicAdd(&jb.ghist[2 * i + 1], c >> 16);
  }
}

template <int R>
__device__ __forceinline__ void pool_body(const LayerArgs& a, int b) {
  __shared__ uint32_t hist_lds[kHistBins / 2];  // two 16-bit counts per word
  __shared__ const float* rows[kMaxQHeads];
  const SeqArgs& sq = a.seq[find_seq(a, b, [](const SeqArgs& t) { return t.blk_pool; })];
  const int local = b - sq.blk_pool;
  const int g = local / sq.n_ptiles;  // selection group (0 when shared)
  const int tile = local - g * sq.n_ptiles;
  const int64_t Ls = sq.L - a.tail;  // scored length
  // the heads averaged here: the group's chosen heads, or every chosen head
  // of the layer when the selection is shared
  const int t0 = a.shared ? 0 : a.grp_off[g];
  const int t1 = a.shared ? a.grp_off[a.n_kv] : a.grp_off[g + 1];
  for (int t = t0 + (int)threadIdx.x; t < t1; t += kThreads) {
    const int gt = a.sel_grp[t];  // head t - grp_off[gt] of group gt
    rows[t - t0] = sq.wsum + ((int64_t)gt * sq.wsum_heads + (t - a.grp_off[gt])) * sq.ws_stride;
  }
  const bool do_hist = a.do_hist && sq.n_keep > 0;
  if (do_hist)
    for (int i = threadIdx.x; i < kHistBins / 2; i += kThreads) hist_lds[i] = 0u;
  __syncthreads();
  PoolJob jb;
  jb.rows = rows;
  jb.n_heads = t1 - t0;
  jb.Ls = Ls;
  jb.j0 = (int64_t)tile * kPoolTile;
  jb.n_out = Ls - jb.j0 < kPoolTile ? (int)(Ls - jb.j0) : kPoolTile;
  jb.is_max = a.pool != 0;
  jb.do_hist = do_hist;
  jb.inv_kp = 1.f / (float)a.kp;
  jb.out = to_global(sq.scores) + (int64_t)g * Ls + jb.j0;
  jb.ghist = sq.hist + (int64_t)g * kHistBins;
  pool_tile<R, kPoolTile / (4 * kThreads)>(jb, hist_lds);
}

// One kernel per pool radius R = kp / 2 (the host picks it): each then keeps
// only its own halo in registers, and the common small radii run at full
// occupancy.
template <int R>
__global__ __launch_bounds__(kThreads) void pool_kernel(const LayerArgs a) { pool_body<R>(a, blockIdx.x); }

// Pooling, head mean, scores and the first-level histogram of several layers
// at once (ckv_compress_stack): layer l's argument block is read from device
// memory, and each workgroup covers kUnitPoolTiles consecutive tiles of one
// (prompt, selection group), merging its histogram once.
template <int R>
__global__ __launch_bounds__(kThreads) void pool_units_kernel(const MultiArgs m) {
  __shared__ uint32_t hist_lds[kHistBins / 2];  // two 16-bit counts per word
  __shared__ const float* rows[kMaxQHeads];
  const int l = blockIdx.x / m.per_layer;
  const LayerArgs& a = layer_args(m, l);
  int local = blockIdx.x - l * m.per_layer;
  int s = 0;
  for (; s < a.num_seqs - 1; ++s) {
    const int n = a.n_sg * ((a.seq[s].n_ptiles + kUnitPoolTiles - 1) / kUnitPoolTiles);
    if (local < n) break;
    local -= n;
  }
  const SeqArgs& sq = a.seq[s];
  const int per_g = (sq.n_ptiles + kUnitPoolTiles - 1) / kUnitPoolTiles;
  const int g = local / per_g;
  const int chunk = local - g * per_g;
  const int64_t Ls = sq.L - a.tail;  // scored length
  const int t0 = a.shared ? 0 : a.grp_off[g];
  const int t1 = a.shared ? a.grp_off[a.n_kv] : a.grp_off[g + 1];
  for (int t = t0 + (int)threadIdx.x; t < t1; t += kThreads) {
    const int gt = a.sel_grp[t];
    rows[t - t0] = sq.wsum + ((int64_t)gt * sq.wsum_heads + (t - a.grp_off[gt])) * sq.ws_stride;
  }
  const bool do_hist = a.do_hist && sq.n_keep > 0;
  if (do_hist)
    for (int i = threadIdx.x; i < kHistBins / 2; i += kThreads) hist_lds[i] = 0u;
  __syncthreads();
  PoolJob jb;
  jb.rows = rows;
  jb.n_heads = t1 - t0;
  jb.Ls = Ls;
  jb.j0 = (int64_t)chunk * kUnitPoolTiles * kPoolTile;
  const int64_t left = Ls - jb.j0;
  jb.n_out = left < (int64_t)kUnitPoolTiles * kPoolTile ? (int)left : kUnitPoolTiles * kPoolTile;
  jb.is_max = a.pool != 0;
  jb.do_hist = do_hist;
  jb.inv_kp = 1.f / (float)a.kp;
  jb.out = to_global(sq.scores) + (int64_t)g * Ls + jb.j0;
  jb.ghist = sq.hist + (int64_t)g * kHistBins;
  pool_tile<R, kUnitPoolTiles * kPoolTile / (4 * kThreads)>(jb, hist_lds);
}


template <template <int, int> class KernelOf>
hipError_t launch_typed(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  if (dtype == 0) return a.d == 64 ? launch(KernelOf<0, 64>::fn, grid, kKpThreads, st, tm, a)
                                   : launch(KernelOf<0, 128>::fn, grid, kKpThreads, st, tm, a);
  if (dtype == 1) return a.d == 64 ? launch(KernelOf<1, 64>::fn, grid, kKpThreads, st, tm, a)
                                   : launch(KernelOf<1, 128>::fn, grid, kKpThreads, st, tm, a);
  return a.d == 64 ? launch(KernelOf<2, 64>::fn, grid, kKpThreads, st, tm, a)
                   : launch(KernelOf<2, 128>::fn, grid, kKpThreads, st, tm, a);
}

template <int DT, int D>
struct RowStatsOf {
  static constexpr auto fn = rowstats_kernel<DT, D>;
};
template <int DT, int D>
struct ScoreOf {
  static constexpr auto fn = score_kernel<DT, D>;
};
template <int DT, int D>
struct RowStatsLayersOf {
  static constexpr auto fn = rowstats_layers_kernel<DT, D>;
};
template <int DT, int D>
struct ScoreLayersOf {
  static constexpr auto fn = score_layers_kernel<DT, D>;
};

template <template <int, int> class KernelOf>
hipError_t launch_typed_layers(int dtype, const LayersArgs& m, int grid, hipStream_t st, const Timing& tm) {
  const int d = m.lay[0].d;
  if (dtype == 0) return d == 64 ? launch(KernelOf<0, 64>::fn, grid, kKpThreads, st, tm, m)
                                 : launch(KernelOf<0, 128>::fn, grid, kKpThreads, st, tm, m);
  if (dtype == 1) return d == 64 ? launch(KernelOf<1, 64>::fn, grid, kKpThreads, st, tm, m)
                                 : launch(KernelOf<1, 128>::fn, grid, kKpThreads, st, tm, m);
  return d == 64 ? launch(KernelOf<2, 64>::fn, grid, kKpThreads, st, tm, m)
                 : launch(KernelOf<2, 128>::fn, grid, kKpThreads, st, tm, m);
}

}  // namespace

hipError_t launch_rowstats(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch_typed<RowStatsOf>(dtype, a, grid, st, tm);
}

hipError_t launch_score(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch_typed<ScoreOf>(dtype, a, grid, st, tm);
}

hipError_t launch_rowstats_layers(int dtype, const LayersArgs& m, int grid, hipStream_t st,
                                  const Timing& tm) {
  return launch_typed_layers<RowStatsLayersOf>(dtype, m, grid, st, tm);
}

hipError_t launch_score_layers(int dtype, const LayersArgs& m, int grid, hipStream_t st,
                               const Timing& tm) {
  return launch_typed_layers<ScoreLayersOf>(dtype, m, grid, st, tm);
}

// The pooling kernels of radius r, looked up at run time.
template <int R>
const void* pool_fn(int r, bool units) {
  if constexpr (R >= kMaxPoolRadius) {
    return units ? reinterpret_cast<const void*>(pool_units_kernel<R>)
                 : reinterpret_cast<const void*>(pool_kernel<R>);
  } else {
    if (r != R) return pool_fn<R + 1>(r, units);
    return units ? reinterpret_cast<const void*>(pool_units_kernel<R>)
                 : reinterpret_cast<const void*>(pool_kernel<R>);
  }
}

hipError_t launch_pool(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  void* args[] = {const_cast<LayerArgs*>(&a)};
  return hipExtLaunchKernel(pool_fn<0>(a.kp >> 1, false), dim3(grid), dim3(kThreads), args, 0, st,
                            tm.start, tm.stop, 0);
}

hipError_t launch_pool_units(const MultiArgs& m, int radius, hipStream_t st, const Timing& tm) {
  void* args[] = {const_cast<MultiArgs*>(&m)};
  return hipExtLaunchKernel(pool_fn<0>(radius, true), dim3(m.n_layers * m.per_layer), dim3(kThreads),
                            args, 0, st, tm.start, tm.stop, 0);
}


}  // namespace ckv
