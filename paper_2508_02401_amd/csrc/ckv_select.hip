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
// With the layer-shared scope there is one selection per prompt (selection
// group 0) and its rows are copied for every KV head.
// Each step is its own launch, so stream order makes every hand-off visible
// without device-wide fences inside the kernels.
#include <type_traits>

#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

constexpr int kCompactPer = 16;                      // scores per thread and compaction step
constexpr int kCompactStep = kCompactPer * kThreads;  // scores per compaction step
constexpr int kFilterPer = kRangeMin / kThreads;  // scores per thread loaded up front
constexpr int kCopyList = 1024;                   // kept rows listed in LDS per copy round

__device__ __forceinline__ int find_seq_sel(const LayerArgs& a, int b) {
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_sel) s = t;
  return s;
}

// Zero the selection control words and histograms (ckv_select on caller
// scores; ckv_compress_layer clears them in the row-statistics kernel).
__global__ __launch_bounds__(kThreads) void clear_kernel(const LayerArgs a) {
  const int s = blockIdx.x / a.n_sg, g = blockIdx.x - s * a.n_sg;
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
  const int64_t Ls = sq.L - a.tail;  // scored length
  const float* sc = sq.scores + (int64_t)g * Ls;
  const int64_t j0 = (int64_t)r * sq.range;
  const int64_t j1 = j0 + sq.range < Ls ? j0 + sq.range : Ls;
  // the first kFilterPer keys of this thread are loaded before the LDS
  // histogram is cleared, all in flight at once
  uint32_t key0[kFilterPer];
#pragma unroll
  for (int e = 0; e < kFilterPer; ++e) {
    const int64_t j = j0 + tid + (int64_t)e * kThreads;
    key0[e] = j < j1 ? score_key(sc[j]) : 0u;
  }
  for (int i = tid; i < kHistBins; i += kThreads) hist_lds[i] = 0u;
  __syncthreads();
#pragma unroll
  for (int e = 0; e < kFilterPer; ++e)
    if (j0 + tid + (int64_t)e * kThreads < j1) atomicAdd(&hist_lds[key0[e] >> kHistShift], 1u);
  for (int64_t j = j0 + tid + (int64_t)kFilterPer * kThreads; j < j1; j += kThreads)
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
__device__ void resolve(const SeqArgs& sq, int n_sg, int g, int64_t Ls, uint32_t* ctl,
                        uint32_t* lds_a, uint32_t* lds_b, uint32_t* wsum, uint32_t* res) {
  const int tid = threadIdx.x;
  const uint32_t n_cand = ctl[kCtlNumCand];
  const uint2* cands = sq.cand + (int64_t)g * Ls;
  uint32_t prefix = ctl[kCtlBin];
  uint32_t need = (uint32_t)sq.n_keep - ctl[kCtlAbove];
  int shift = kHistShift;
  // radix select on bits 18..9, then 8..0, among keys still matching prefix
  auto level = [&](auto nb_c) -> bool {
    constexpr int nb = decltype(nb_c)::value;
    constexpr int nbins = 1 << nb;
    const int nshift = shift - nb;
    for (int i = tid; i < nbins; i += kThreads) lds_a[i] = 0u;
    __syncthreads();
    for (uint32_t c = tid; c < n_cand; c += kThreads) {
      const uint32_t key = cands[c].x;
      if ((key >> shift) == prefix) atomicAdd(&lds_a[(key >> nshift) & (nbins - 1)], 1u);
    }
    __syncthreads();
    find_bin<nbins>(need, [&](int bin) { return lds_a[bin]; }, wsum, res);
    prefix = (prefix << nb) | res[0];
    need -= res[1];
    shift = nshift;
    const uint32_t cnt = res[2];
    __syncthreads();
    return cnt == need;  // every key of this bin is kept
  };
  static_assert(kHistShift == 19, "radix levels cover bits 18..0");
  if (!level(std::integral_constant<int, 10>{})) level(std::integral_constant<int, 9>{});
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
  uint32_t* roff = sq.rsure + ((int64_t)n_sg + g) * n_ranges;
  uint32_t* reqb = sq.rsure + (2 * (int64_t)n_sg + g) * n_ranges;
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
__device__ __forceinline__ void filter_body(const LayerArgs& a, int b) {
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t res[3];
  const int s = find_seq_sel(a, b);
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_sel;
  const int g = local / sq.n_ranges, r = local - g * sq.n_ranges;
  if (sq.n_keep <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t Ls = sq.L - a.tail;  // scored length
  uint32_t* ctl = sq.ctl + g * kCtlWords;
  const uint32_t* ghist = sq.hist + (int64_t)g * kHistBins;
  const float* sc = sq.scores + (int64_t)g * Ls;
  uint2* cands = sq.cand + (int64_t)g * Ls;
  const int64_t j0 = (int64_t)r * sq.range;
  const int64_t j1 = j0 + sq.range < Ls ? j0 + sq.range : Ls;
  // this thread's first kFilterPer keys are loaded before the threshold
  // search, so their latency overlaps it
  uint32_t key0[kFilterPer];
#pragma unroll
  for (int e = 0; e < kFilterPer; ++e) {
    const int64_t j = j0 + tid + (int64_t)e * kThreads;
    key0[e] = j < j1 ? score_key(sc[j]) : 0u;
  }
  find_bin<kHistBins>((uint32_t)sq.n_keep, [&](int bin) { return ghist[bin]; }, wsum, res);
  const uint32_t bin = res[0];
  if (r == 0 && tid == 0) {
    ctl[kCtlBin] = res[0];
    ctl[kCtlAbove] = res[1];
    ctl[kCtlBinCount] = res[2];
  }
  uint32_t sure = 0;
  // keys loaded up front: count, then one atomic per wave reserves the
  // wave's candidate slots, written in lane order
  {
    uint32_t mine = 0;
#pragma unroll
    for (int e = 0; e < kFilterPer; ++e) {
      const bool in = j0 + tid + (int64_t)e * kThreads < j1;
      const uint32_t kb = key0[e] >> kHistShift;
      sure += in && kb > bin;
      mine += in && kb == bin;
    }
    uint32_t incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    const uint32_t wave_total = __shfl(incl, 63);
    if (wave_total) {
      uint32_t base = 0;
      if (lane == 63) base = atomicAdd(&ctl[kCtlNumCand], wave_total);
      base = __shfl(base, 63);
      uint32_t at = base + incl - mine;
#pragma unroll
      for (int e = 0; e < kFilterPer; ++e) {
        const int64_t j = j0 + tid + (int64_t)e * kThreads;
        if (j < j1 && (key0[e] >> kHistShift) == bin) cands[at++] = make_uint2(key0[e], (uint32_t)j);
      }
    }
  }
  // ranges longer than kFilterPer * kThreads scores
  for (int64_t j = j0 + tid + (int64_t)kFilterPer * kThreads; j < j1; j += kThreads) {
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

__global__ __launch_bounds__(kThreads) void filter_kernel(const LayerArgs a) {
  filter_body(a, blockIdx.x);
}


// One workgroup per (prompt, group): exact threshold and range offsets.
__device__ __forceinline__ void resolve_body(const LayerArgs& a, int b) {
  __shared__ uint32_t lds_a[kMaxRanges];
  __shared__ uint32_t lds_b[kMaxRanges];
  __shared__ uint32_t wsum[kWaves];
  __shared__ uint32_t res[3];
  const int s = b / a.n_sg, g = b - s * a.n_sg;
  const SeqArgs& sq = a.seq[s];
  if (sq.n_keep <= 0) return;
  resolve(sq, a.n_sg, g, sq.L - a.tail, sq.ctl + g * kCtlWords, lds_a, lds_b, wsum, res);
}

__global__ __launch_bounds__(kThreads) void resolve_kernel(const LayerArgs a) {
  resolve_body(a, blockIdx.x);
}


// Kept indices of one range, in ascending order at the range's output offset,
// then the copies of their K/V rows. Thread t takes kCompactPer consecutive
// scores per step, so a thread's kept tokens are consecutive in the output.
__device__ __forceinline__ void compact_body(const LayerArgs& a, int b) {
  __shared__ uint32_t wsum[kWaves];
  __shared__ int32_t pos_l[kCopyList];
  __shared__ int32_t tok_l[kCopyList];
  const int s = find_seq_sel(a, b);
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_sel;
  const int g = local / sq.n_ranges, r = local - g * sq.n_ranges;
  const int tid = threadIdx.x;
  const int w = a.tail;  // tokens kept by rule after the ranked ones
  const int64_t Ls = sq.L - w;
  int32_t* out = sq.idx + (int64_t)g * sq.n_ret;
  const int64_t j0 = (int64_t)r * sq.range;
  const int64_t j1 = j0 + sq.range < Ls ? j0 + sq.range : Ls;

  // the KV heads whose rows this selection keeps: its own, or all of them
  // when the selection is shared (g is then 0)
  const int gk0 = a.shared ? 0 : g, gk1 = a.shared ? a.n_kv : g + 1;

  if (sq.n_keep < 0) {  // budget >= L: every token stays, in order
    for (int64_t j = j0 + tid; j < j1; j += kThreads) out[j] = (int32_t)j;
    if (r == 0)
      for (int i = tid; i < w; i += kThreads) out[Ls + i] = (int32_t)(Ls + i);
    if (a.do_gather) {
      for (int gk = gk0; gk < gk1; ++gk) {
        copy_run<kThreads>(a, sq, gk, j0, j0, j1 - j0);
        if (r == 0) copy_run<kThreads>(a, sq, gk, Ls, Ls, w);
      }
    }
    return;
  }
  const uint32_t nk = (uint32_t)sq.n_keep;
  if (r == 0) {  // the window is always kept, after the prefix tokens
    for (int i = tid; i < w; i += kThreads) out[nk + i] = (int32_t)(Ls + i);
    if (a.do_gather)
      for (int gk = gk0; gk < gk1; ++gk) copy_run<kThreads>(a, sq, gk, nk, Ls, w);
  }
  if (nk == 0) return;
  const uint32_t* ctl = sq.ctl + g * kCtlWords;
  const uint32_t* roff = sq.rsure + ((int64_t)a.n_sg + g) * sq.n_ranges;
  uint32_t pos_carry = roff[r];
  uint32_t end = r + 1 < sq.n_ranges ? roff[r + 1] : nk;
  uint32_t eq_carry = sq.rsure[(2 * (int64_t)a.n_sg + g) * sq.n_ranges + r];
  const uint32_t prefix = ctl[kCtlPrefix];
  const int shift = (int)ctl[kCtlShift];
  const uint32_t need = ctl[kCtlNeedEq];
  end = end < nk ? end : nk;
  if (end == pos_carry) return;  // nothing kept in this range
  const float* sc = sq.scores + (int64_t)g * Ls;
  for (int64_t base = j0; base < j1 && pos_carry < end; base += kCompactStep) {
    const int64_t jt = base + (int64_t)tid * kCompactPer;  // this thread's first score
    // flag 1: above the threshold, 2: equal to it, 0: below
    uint32_t key[kCompactPer];
#pragma unroll
    for (int e = 0; e < kCompactPer; ++e) key[e] = jt + e < j1 ? score_key(sc[jt + e]) : 0u;
    int f[kCompactPer];
    uint32_t neq = 0;
#pragma unroll
    for (int e = 0; e < kCompactPer; ++e) {
      const uint32_t p = key[e] >> shift;
      f[e] = jt + e >= j1 ? 0 : (p > prefix ? 1 : (p == prefix ? 2 : 0));
      neq += f[e] == 2;
    }
    uint32_t tot_eq, tot_sel;
    uint32_t eq_rank = eq_carry + block_excl_scan<kThreads>(neq, wsum, tot_eq);
    uint32_t kept = 0;  // bit e: score jt + e is kept
    uint32_t nsel = 0;
#pragma unroll
    for (int e = 0; e < kCompactPer; ++e) {
      bool keep = f[e] == 1;
      if (f[e] == 2) {  // equal keys: the lowest indices, while any are needed
        keep = eq_rank < need;
        ++eq_rank;
      }
      kept |= (uint32_t)keep << e;
      nsel += keep;
    }
    const uint32_t first = block_excl_scan<kThreads>(nsel, wsum, tot_sel);
    {
      uint32_t pos = pos_carry + first;
#pragma unroll
      for (int e = 0; e < kCompactPer; ++e) {
        if (((kept >> e) & 1u) && pos < end) out[pos++] = (int32_t)(jt + e);
      }
    }
    if (a.do_gather) {
      // the step's kept rows in rounds of kCopyList: this thread's kept
      // tokens have list numbers first, first + 1, ...
      const uint32_t n = tot_sel < end - pos_carry ? tot_sel : end - pos_carry;
      for (uint32_t r0 = 0; r0 < n; r0 += kCopyList) {
        uint32_t li = first;
#pragma unroll
        for (int e = 0; e < kCompactPer; ++e) {
          if ((kept >> e) & 1u) {
            if (li >= r0 && li < r0 + kCopyList && li < n) {
              pos_l[li - r0] = (int32_t)(pos_carry + li);
              tok_l[li - r0] = (int32_t)(jt + e);
            }
            ++li;
          }
        }
        __syncthreads();
        const uint32_t m = n - r0 < (uint32_t)kCopyList ? n - r0 : (uint32_t)kCopyList;
        for (int gk = gk0; gk < gk1; ++gk)
          copy_rows<kThreads>(a, sq, gk, m, [&](int64_t i) { return (int64_t)tok_l[i]; },
                    [&](int64_t i) { return (int64_t)pos_l[i]; });
        __syncthreads();
      }
    }
    eq_carry += tot_eq;
    pos_carry += tot_sel;
  }
}

__global__ __launch_bounds__(kThreads) void compact_kernel(const LayerArgs a) {
  compact_body(a, blockIdx.x);
}


// Retain/evict: rows idx[g, r] of K and V for the kGatherRows output rows of
// gather workgroup b of the layer. An out-of-range index leaves its output
// row untouched.
__device__ __forceinline__ void gather_body(const LayerArgs& a, int b, int32_t* tok_l) {
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_gather) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_gather;
  const int g = local / sq.n_gblk;
  const int r0 = (local - g * sq.n_gblk) * kGatherRows;
  const int n = sq.n_ret - r0 < kGatherRows ? sq.n_ret - r0 : kGatherRows;
  // the head's own index row, or the layer's one row when shared
  const int32_t* idx = sq.idx + (a.shared ? 0 : (int64_t)g * sq.n_ret);
  for (int i = threadIdx.x; i < n; i += kThreads) tok_l[i] = idx[r0 + i];
  __syncthreads();
  copy_rows<kThreads>(a, sq, g, n, [&](int64_t i) { return (int64_t)tok_l[i]; },
            [&](int64_t i) { return r0 + i; });
}

// Standalone retain/evict (ckv_gather).
__global__ __launch_bounds__(kThreads) void gather_kernel(const LayerArgs a) {
  __shared__ int32_t tok_l[kGatherRows];
  gather_body(a, blockIdx.x, tok_l);
}

// The gather of a batch of layers after the selection units wrote their
// indices: m.per_layer workgroups per layer, those past a layer's own grid
// idle.
__global__ __launch_bounds__(kThreads) void gather_layers_kernel(const MultiArgs m) {
  __shared__ int32_t tok_l[kGatherRows];
  const int l = blockIdx.x / m.per_layer;
  const int b = blockIdx.x - l * m.per_layer;
  const LayerArgs& a = layer_args(m, l);
  const SeqArgs& last = a.seq[a.num_seqs - 1];
  if (b >= last.blk_gather + last.n_gblk * a.n_kv) return;
  gather_body(a, b, tok_l);
}

// StreamingLLM-style selection, the comparison baseline that keeps the
// attention-sink tokens and the most recent ones: row r of the n_ret kept
// rows is token r for the first min(sinks, n_ret) rows and token
// L - n_ret + r after them (ascending, no scores). Writes the index row and
// copies the rows like gather_kernel, with the same grid.
__global__ __launch_bounds__(kThreads) void stream_gather_kernel(const LayerArgs a, int32_t sinks) {
  __shared__ int32_t tok_l[kGatherRows];
  const int b = blockIdx.x;
  int s = 0;
  for (int t = 1; t < a.num_seqs; ++t)
    if (b >= a.seq[t].blk_gather) s = t;
  const SeqArgs& sq = a.seq[s];
  const int local = b - sq.blk_gather;
  const int g = local / sq.n_gblk;
  const int r0 = (local - g * sq.n_gblk) * kGatherRows;
  const int n = sq.n_ret - r0 < kGatherRows ? sq.n_ret - r0 : kGatherRows;
  const int ns = sinks < sq.n_ret ? sinks : sq.n_ret;
  const int64_t recent0 = sq.L - sq.n_ret;  // token of row r >= ns is recent0 + r
  int32_t* idx = sq.idx + (a.shared ? 0 : (int64_t)g * sq.n_ret);
  const bool writer = !a.shared || g == 0;  // the layer's one index row when shared
  for (int i = threadIdx.x; i < n; i += kThreads) {
    const int r = r0 + i;
    const int32_t tok = r < ns ? r : (int32_t)(recent0 + r);
    tok_l[i] = tok;
    if (writer) idx[r] = tok;
  }
  __syncthreads();
  copy_rows<kThreads>(a, sq, g, n, [&](int64_t i) { return (int64_t)tok_l[i]; },
            [&](int64_t i) { return r0 + i; });
}

}  // namespace

hipError_t launch_stream_gather(const LayerArgs& a, int32_t sinks, int grid, hipStream_t st) {
  void* args[] = {const_cast<LayerArgs*>(&a), &sinks};
  return hipLaunchKernel(reinterpret_cast<const void*>(stream_gather_kernel), dim3(grid),
                         dim3(kThreads), args, 0, st);
}

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

hipError_t launch_gather_layers(const MultiArgs& m, hipStream_t st, const Timing& tm) {
  return launch(gather_layers_kernel, m.n_layers * m.per_layer, kThreads, st, tm, m);
}




}  // namespace ckv
