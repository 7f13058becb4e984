// gfx950 (MI355X) top-N selection and retain/evict of CompressKV's
// prefill-end token selection (arXiv 2508.02401, Sec. 3.3: the tokens with
// the N highest averaged scores keep their KV pairs, the others are evicted).
//
// Per (prompt, KV head) with n_keep = B - w prefix tokens to keep, keys are the
// fp32 bit patterns of the scores (scores >= 0, so integer order is score
// order) and ties go to the lower token index:
//   1. a 4096-bin histogram of key bits 30..19, built by the scoring kernel
//      (or by hist_kernel when the caller supplies the scores);
//   2. filter_kernel: every range of scores finds the bin b holding the
//      n_keep-th largest key, counts its keys above bin b and appends the keys
//      inside bin b (the candidates) to a list;
//   3. resolve_kernel: per group, the exact threshold by a radix select over
//      the candidates' low 19 bits, then per range how many keys it keeps and
//      at which output offset;
//   4. compact_kernel: every range writes its kept indices in ascending order
//      at its offset (keys above the threshold, then the first keys equal to
//      it), appends the window positions, and copies the kept K/V rows.
// Each step is its own launch, so stream order makes every hand-off visible
// without device-wide fences inside the kernels.
#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

constexpr int kStep = 4 * kThreads;  // scores per compaction step (4 per thread)

__device__ __forceinline__ int find_seq_sel(const LayerArgs& a, int b) {
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_sel) s = t;
  return s;
}

// Copy n rows of K and V: row src0 + i -> output row dst0 + i (contiguous runs).
__device__ __forceinline__ void copy_run(const LayerArgs& a, const SeqArgs& sq, int g, int64_t dst0,
                                         int64_t src0, int64_t n) {
  const int nv = a.d * a.elt / 16;
  const char* kb = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * a.elt;
  const char* vb = static_cast<const char*>(sq.v) + (int64_t)g * sq.kv_sh * a.elt;
  uint4* ko = static_cast<uint4*>(sq.k_out) + (int64_t)g * sq.n_ret * nv;
  uint4* vo = static_cast<uint4*>(sq.v_out) + (int64_t)g * sq.n_ret * nv;
  for (int64_t e = threadIdx.x; e < n * nv; e += kThreads) {
    const int64_t i = e / nv;
    const int c = (int)(e - i * nv);
    const int64_t j = src0 + i, p = dst0 + i;
    if (j < 0 || j >= sq.L || p < 0 || p >= sq.n_ret) continue;
    ko[p * nv + c] = reinterpret_cast<const uint4*>(kb + j * sq.kv_st * a.elt)[c];
    vo[p * nv + c] = reinterpret_cast<const uint4*>(vb + j * sq.kv_st * a.elt)[c];
  }
}

// Copy the listed rows: source token jl[i] -> output row pl[i].
__device__ __forceinline__ void copy_list(const LayerArgs& a, const SeqArgs& sq, int g,
                                          const int32_t* pl, const int32_t* jl, int n) {
  const int nv = a.d * a.elt / 16;
  const char* kb = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * a.elt;
  const char* vb = static_cast<const char*>(sq.v) + (int64_t)g * sq.kv_sh * a.elt;
  uint4* ko = static_cast<uint4*>(sq.k_out) + (int64_t)g * sq.n_ret * nv;
  uint4* vo = static_cast<uint4*>(sq.v_out) + (int64_t)g * sq.n_ret * nv;
  for (int e = threadIdx.x; e < n * nv; e += kThreads) {
    const int i = e / nv, c = e - i * nv;
    const int64_t j = jl[i], p = pl[i];
    if (j < 0 || j >= sq.L || p < 0 || p >= sq.n_ret) continue;
    ko[p * nv + c] = reinterpret_cast<const uint4*>(kb + j * sq.kv_st * a.elt)[c];
    vo[p * nv + c] = reinterpret_cast<const uint4*>(vb + j * sq.kv_st * a.elt)[c];
  }
}

// Zero the selection control words and histograms (ckv_select on caller
// scores; ckv_compress_layer clears them in the row-statistics kernel).
__global__ __launch_bounds__(kThreads) void clear_kernel(const LayerArgs a) {
  const int s = blockIdx.x / a.n_kv, g = blockIdx.x - s * a.n_kv;
  const SeqArgs& sq = a.seq[s];
  for (int i = threadIdx.x; i < kCtlWords; i += kThreads) sq.ctl[g * kCtlWords + i] = 0u;
  for (int i = threadIdx.x; i < kHistBins; i += kThreads)
    sq.hist[(int64_t)g * kHistBins + i] = 0u;
}

// First-level histogram of caller-supplied scores, one range per workgroup.
__global__ __launch_bounds__(kThreads) void hist_kernel(const LayerArgs a) {
  __shared__ uint32_t hist_lds[kHistBins];
  const int b = blockIdx.x;
  const int s = find_seq_sel(a, b);
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_sel;
  const int g = local / sq.n_ranges, r = local - g * sq.n_ranges;
  if (sq.n_keep <= 0) return;
  const int tid = threadIdx.x;
  const int64_t Ls = sq.L - a.w;
  const float* sc = sq.scores + (int64_t)g * Ls;
  const int64_t j0 = (int64_t)r * sq.range;
  const int64_t j1 = j0 + sq.range < Ls ? j0 + sq.range : Ls;
  for (int i = tid; i < kHistBins; i += kThreads) hist_lds[i] = 0u;
  __syncthreads();
  for (int64_t j = j0 + tid; j < j1; j += kThreads)
    atomicAdd(&hist_lds[score_key(sc[j]) >> kHistShift], 1u);
  __syncthreads();
  uint32_t* ghist = sq.hist + (int64_t)g * kHistBins;
  for (int i = tid; i < kHistBins; i += kThreads) {
    const uint32_t c = hist_lds[i];
    if (c) atomicAdd(&ghist[i], c);
  }
}

// Exact threshold among the candidates, then per-range kept counts and output
// offsets.
__device__ void resolve(const SeqArgs& sq, int g, int64_t Ls, uint32_t* ctl, uint32_t* lds_a,
                        uint32_t* lds_b, uint32_t* wsum, uint32_t* res) {
  const int tid = threadIdx.x;
  const uint32_t n_cand = ctl[kCtlNumCand];
  const uint2* cands = sq.cand + (int64_t)g * Ls;
  uint32_t prefix = ctl[kCtlBin];
  uint32_t need = (uint32_t)sq.n_keep - ctl[kCtlAbove];
  int shift = kHistShift;
  // radix select on bits 18..9, then 8..0, among keys still matching prefix
  for (int level = 0; level < 2; ++level) {
    const int nb = level == 0 ? 10 : 9;
    const int nshift = shift - nb;
    const int nbins = 1 << nb;
    for (int i = tid; i < nbins; i += kThreads) lds_a[i] = 0u;
    __syncthreads();
    for (uint32_t c = tid; c < n_cand; c += kThreads) {
      const uint32_t key = cands[c].x;
      if ((key >> shift) == prefix) atomicAdd(&lds_a[(key >> nshift) & (nbins - 1)], 1u);
    }
    __syncthreads();
    find_bin(nbins, need, [&](int bin) { return lds_a[bin]; }, wsum, res);
    prefix = (prefix << nb) | res[0];
    need -= res[1];
    shift = nshift;
    const uint32_t cnt = res[2];
    __syncthreads();
    if (cnt == need) break;  // every key of this bin is kept
  }
  // keys compare on key >> shift: above prefix kept, equal kept while need lasts
  const int n_ranges = sq.n_ranges;
  for (int i = tid; i < n_ranges; i += kThreads) {
    lds_a[i] = 0u;
    lds_b[i] = 0u;
  }
  __syncthreads();
  for (uint32_t c = tid; c < n_cand; c += kThreads) {
    const uint2 e = cands[c];
    const uint32_t p = e.x >> shift;
    const int r = (int)(e.y / (uint32_t)sq.range);
    if (p > prefix) atomicAdd(&lds_a[r], 1u);
    else if (p == prefix) atomicAdd(&lds_b[r], 1u);
  }
  __syncthreads();
  const uint32_t* rsure = sq.rsure + (int64_t)g * n_ranges;
  uint32_t* roff = sq.roff + (int64_t)g * n_ranges;
  uint32_t* reqb = sq.reqb + (int64_t)g * n_ranges;
  uint32_t eq_carry = 0, off_carry = 0;
  for (int base = 0; base < n_ranges; base += kThreads) {
    const int r = base + tid;
    const bool valid = r < n_ranges;
    const uint32_t eq = valid ? lds_b[r] : 0u;
    uint32_t tot_eq, tot_sel;
    const uint32_t eqb = eq_carry + block_excl_scan<kThreads>(eq, wsum, tot_eq);
    const uint32_t left = need > eqb ? need - eqb : 0u;
    const uint32_t chosen = eq < left ? eq : left;
    const uint32_t sel = valid ? rsure[r] + lds_a[r] + chosen : 0u;
    const uint32_t off = off_carry + block_excl_scan<kThreads>(sel, wsum, tot_sel);
    if (valid) {
      reqb[r] = eqb;
      roff[r] = off;
    }
    eq_carry += tot_eq;
    off_carry += tot_sel;
  }
  if (tid == 0) {
    ctl[kCtlPrefix] = prefix;
    ctl[kCtlShift] = (uint32_t)shift;
    ctl[kCtlNeedEq] = need;
  }
}

// Every range finds the threshold bin from the group's histogram (the range 0
// workgroup records it), counts its keys above the bin and appends the keys
// inside it to the candidate list.
__global__ __launch_bounds__(kThreads) void filter_kernel(const LayerArgs a) {
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t res[3];
  const int b = blockIdx.x;
  const int s = find_seq_sel(a, b);
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_sel;
  const int g = local / sq.n_ranges, r = local - g * sq.n_ranges;
  if (sq.n_keep <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t Ls = sq.L - a.w;
  uint32_t* ctl = sq.ctl + g * kCtlWords;
  const uint32_t* ghist = sq.hist + (int64_t)g * kHistBins;
  find_bin(kHistBins, (uint32_t)sq.n_keep, [&](int bin) { return ghist[bin]; }, wsum, res);
  const uint32_t bin = res[0];
  if (r == 0 && tid == 0) {
    ctl[kCtlBin] = res[0];
    ctl[kCtlAbove] = res[1];
    ctl[kCtlBinCount] = res[2];
  }
  const float* sc = sq.scores + (int64_t)g * Ls;
  uint2* cands = sq.cand + (int64_t)g * Ls;
  const int64_t j0 = (int64_t)r * sq.range;
  const int64_t j1 = j0 + sq.range < Ls ? j0 + sq.range : Ls;
  uint32_t sure = 0;
  for (int64_t j = j0 + tid; j < j1; j += kThreads) {
    const uint32_t key = score_key(sc[j]);
    const uint32_t kb = key >> kHistShift;
    sure += kb > bin;
    const bool isc = kb == bin;
    const uint64_t mask = __ballot(isc);
    if (mask) {
      const int leader = __ffsll((unsigned long long)mask) - 1;
      uint32_t base = 0;
      if (lane == leader) base = atomicAdd(&ctl[kCtlNumCand], (uint32_t)__popcll(mask));
      base = __shfl(base, leader);
      if (isc) {
        const uint32_t rank = (uint32_t)__popcll(mask & ((1ull << lane) - 1ull));
        cands[base + rank] = make_uint2(key, (uint32_t)j);
      }
    }
  }
  uint32_t total;
  block_excl_scan<kThreads>(sure, wsum, total);
  if (tid == 0) sq.rsure[(int64_t)g * sq.n_ranges + r] = total;
}

// One workgroup per (prompt, group): exact threshold and range offsets.
__global__ __launch_bounds__(kThreads) void resolve_kernel(const LayerArgs a) {
  __shared__ uint32_t lds_a[kMaxRanges];
  __shared__ uint32_t lds_b[kMaxRanges];
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t res[3];
  const int s = blockIdx.x / a.n_kv, g = blockIdx.x - s * a.n_kv;
  const SeqArgs& sq = a.seq[s];
  if (sq.n_keep <= 0) return;
  resolve(sq, g, sq.L - a.w, sq.ctl + g * kCtlWords, lds_a, lds_b, wsum, res);
}

__global__ __launch_bounds__(kThreads) void compact_kernel(const LayerArgs a) {
  __shared__ uint32_t wsum[kWaves];
  __shared__ int32_t pos_l[kStep];
  __shared__ int32_t tok_l[kStep];
  const int b = blockIdx.x;
  const int s = find_seq_sel(a, b);
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_sel;
  const int g = local / sq.n_ranges, r = local - g * sq.n_ranges;
  const int tid = threadIdx.x;
  const int w = a.w;
  const int64_t Ls = sq.L - w;
  int32_t* out = sq.idx + (int64_t)g * sq.n_ret;
  const int64_t j0 = (int64_t)r * sq.range;
  const int64_t j1 = j0 + sq.range < Ls ? j0 + sq.range : Ls;

  if (sq.n_keep < 0) {  // budget >= L: every token stays, in order
    for (int64_t j = j0 + tid; j < j1; j += kThreads) out[j] = (int32_t)j;
    if (r == 0)
      for (int i = tid; i < w; i += kThreads) out[Ls + i] = (int32_t)(Ls + i);
    if (a.do_gather) {
      copy_run(a, sq, g, j0, j0, j1 - j0);
      if (r == 0) copy_run(a, sq, g, Ls, Ls, w);
    }
    return;
  }
  const uint32_t nk = (uint32_t)sq.n_keep;
  if (r == 0) {  // the window is always kept, after the prefix tokens
    for (int i = tid; i < w; i += kThreads) out[nk + i] = (int32_t)(Ls + i);
    if (a.do_gather) copy_run(a, sq, g, nk, Ls, w);
  }
  if (nk == 0) return;
  const uint32_t* ctl = sq.ctl + g * kCtlWords;
  const uint32_t prefix = ctl[kCtlPrefix];
  const int shift = (int)ctl[kCtlShift];
  const uint32_t need = ctl[kCtlNeedEq];
  const uint32_t* roff = sq.roff + (int64_t)g * sq.n_ranges;
  uint32_t eq_carry = sq.reqb[(int64_t)g * sq.n_ranges + r];
  uint32_t pos_carry = roff[r];
  uint32_t end = r + 1 < sq.n_ranges ? roff[r + 1] : nk;
  end = end < nk ? end : nk;
  if (end == pos_carry) return;  // nothing kept in this range
  const float* sc = sq.scores + (int64_t)g * Ls;
  for (int64_t base = j0; base < j1 && pos_carry < end; base += kStep) {
    const int64_t jb = base + 4 * tid;
    int f[4];
    uint32_t neq = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[e] = 0;
      if (jb + e < j1) {
        const uint32_t p = score_key(sc[jb + e]) >> shift;
        f[e] = p > prefix ? 1 : (p == prefix ? 2 : 0);
      }
      neq += f[e] == 2;
    }
    uint32_t tot_eq, tot_sel;
    uint32_t eq_rank = eq_carry + block_excl_scan<kThreads>(neq, wsum, tot_eq);
    bool keep[4];
    uint32_t nsel = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      keep[e] = f[e] == 1;
      if (f[e] == 2) {
        keep[e] = eq_rank < need;
        ++eq_rank;
      }
      nsel += keep[e];
    }
    const uint32_t first = block_excl_scan<kThreads>(nsel, wsum, tot_sel);
    uint32_t pos = pos_carry + first;
    uint32_t li = first;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (keep[e] && pos < end) {
        out[pos] = (int32_t)(jb + e);
        pos_l[li] = (int32_t)pos;
        tok_l[li] = (int32_t)(jb + e);
        ++pos;
        ++li;
      }
    }
    if (a.do_gather) {
      __syncthreads();
      const uint32_t n = tot_sel < end - pos_carry ? tot_sel : end - pos_carry;
      copy_list(a, sq, g, pos_l, tok_l, (int)n);
      __syncthreads();
    }
    eq_carry += tot_eq;
    pos_carry += tot_sel;
  }
}

// Standalone retain/evict (ckv_gather): rows idx[g, r] of K and V.
__global__ __launch_bounds__(kThreads) void gather_kernel(const LayerArgs a) {
  const int b = blockIdx.x;
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_gather) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_gather;
  const int g = local / sq.n_gblk;
  const int r0 = (local - g * sq.n_gblk) * kGatherRows;
  const int nv = a.d * a.elt / 16;
  const int32_t* idx = sq.idx + (int64_t)g * sq.n_ret;
  const char* kb = static_cast<const char*>(sq.k) + (int64_t)g * sq.kv_sh * a.elt;
  const char* vb = static_cast<const char*>(sq.v) + (int64_t)g * sq.kv_sh * a.elt;
  uint4* ko = static_cast<uint4*>(sq.k_out) + (int64_t)g * sq.n_ret * nv;
  uint4* vo = static_cast<uint4*>(sq.v_out) + (int64_t)g * sq.n_ret * nv;
  for (int e = threadIdx.x; e < kGatherRows * nv; e += kThreads) {
    const int rr = e / nv, c = e - rr * nv;
    const int r = r0 + rr;
    if (r >= sq.n_ret) break;
    const int64_t t = idx[r];
    if (t < 0 || t >= sq.L) continue;  // out-of-range index: leave the row untouched
    ko[(int64_t)r * nv + c] = reinterpret_cast<const uint4*>(kb + t * sq.kv_st * a.elt)[c];
    vo[(int64_t)r * nv + c] = reinterpret_cast<const uint4*>(vb + t * sq.kv_st * a.elt)[c];
  }
}

}  // namespace

hipError_t launch_clear(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(clear_kernel, grid, kThreads, st, tm, a);
}

hipError_t launch_hist(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(hist_kernel, grid, kThreads, st, tm, a);
}

hipError_t launch_filter(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(filter_kernel, grid, kThreads, st, tm, a);
}

hipError_t launch_resolve(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(resolve_kernel, grid, kThreads, st, tm, a);
}

hipError_t launch_compact(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(compact_kernel, grid, kThreads, st, tm, a);
}

hipError_t launch_gather(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm) {
  return launch(gather_kernel, grid, kThreads, st, tm, a);
}

}  // namespace ckv
