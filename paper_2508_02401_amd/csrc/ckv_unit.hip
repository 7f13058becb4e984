// gfx950 (MI355X) top-N selection and retain/evict of CompressKV's
// prefill-end token selection for a batch of layers (arXiv 2508.02401,
// Sec. 3.3: the tokens with the N highest averaged scores keep their KV
// pairs, the others are evicted).
//
// After the pooling kernel has written a batch's scores and first-level
// histograms, one workgroup of 512 threads owns one selection unit (layer,
// prompt, selection group) through to the compact cache, with no further
// kernel boundary or device-wide atomic:
//   1. the bin of the 4096-bin histogram (key bits 30..19) holding the N-th
//      largest key;
//   2. the exact threshold: the keys of that bin gathered into LDS (when at
//      most kCandCap) and ranked there, or ranked by further histogram passes
//      over the scores, 12 bits at a time, until the threshold key is exact
//      or every key of the bin is kept;
//   3. two LDS bitmaps per segment of 131072 tokens, one of the kept keys
//      (above the threshold) and one of the keys equal to it; walking them in
//      token order keeps the lowest-index equal keys, writes the indices in
//      ascending order and copies their K/V rows (or leaves the copies to a
//      gather launch when the batch keeps many rows per unit).
// For a prompt of at most 131072 tokens whose threshold bin fits in LDS,
// steps 2 and 3 read the scores once: the same pass marks the keys above the
// bin and gathers the bin's keys.
// Keys are the fp32 bit patterns of the scores (scores >= 0, so integer
// order is score order); ties go to the lower token index.
#include "ckv_device.h"

namespace ckv {
namespace {

using namespace dev;

constexpr int kUT = 512;                   // threads per unit workgroup
constexpr int kUW = kUT / 64;              // its waves
constexpr int kCandCap = 8192;             // threshold-bin keys ranked in LDS
constexpr int kSegWords = 4096;            // bitmap words of one output segment
constexpr int kSegTokens = kSegWords * 32; // tokens of one output segment
constexpr int kUnitList = 1024;            // kept rows listed per copy round
constexpr int kScanBatch = 32;             // score loads in flight per thread
constexpr int kBatchTokens = kUT * kScanBatch;  // tokens of one scan batch
static_assert(kSegWords % kUT == 0, "bitmap words per thread");
static_assert(kHistBins % kUT == 0 && kSegTokens % kBatchTokens == 0, "whole batches");

struct UnitLds {
  uint32_t hist[kHistBins];
  uint2 cand[kCandCap];      // (key, token) of the threshold bin's keys
  uint32_t kmap[kSegWords];  // keys above the threshold
  uint32_t emap[kSegWords];  // keys equal to it
  int32_t lpos[kUnitList];
  int32_t ltok[kUnitList];
  uint32_t wsum[kUW];
  uint32_t res[3];
  uint32_t n_cand;
};

// Bin of an LDS histogram of nbins (<= kHistBins) bins holding the need-th
// largest key (1 <= need <= total count): res = (bin, keys in higher bins,
// keys in the bin), for every thread.
constexpr int kBinsPer = kHistBins / kUT;
__device__ void find_bin_unit(UnitLds& sm, int nbins, uint32_t need) {
  const int per = (nbins + kUT - 1) / kUT;
  const int top = nbins - 1 - per * (int)threadIdx.x;
  uint32_t c[kBinsPer];
  uint32_t local = 0;
#pragma unroll
  for (int i = 0; i < kBinsPer; ++i) {
    c[i] = i < per && top - i >= 0 ? sm.hist[top - i] : 0u;
    local += c[i];
  }
  uint32_t tot;
  const uint32_t above = block_excl_scan<kUT>(local, sm.wsum, tot);
  if (above < need && need <= above + local) {
    uint32_t run = above;
    bool found = false;
#pragma unroll
    for (int i = 0; i < kBinsPer; ++i) {
      if (!found && need <= run + c[i]) {
        sm.res[0] = (uint32_t)(top - i);
        sm.res[1] = run;
        sm.res[2] = c[i];
        found = true;
      }
      run += c[i];
    }
  }
  __syncthreads();
}

// f(j, key, valid) for every token j in [j0, j1) of a score row, thread t
// taking j0 + t, j0 + t + kUT, ...; only tokens below jlim (>= 1) are valid,
// the others pass key 0. kScanBatch loads are in flight at once.
// Every thread calls f the same number of times, so f may use wave ballots:
// a wave's lanes hold 64 consecutive tokens.
template <class F>
__device__ __forceinline__ void scan_scores(const float* sc_p, int64_t j0, int64_t j1, int64_t jlim,
                                            F f) {
  const CKV_GLOBAL float* sc = to_global(sc_p);
  for (int64_t base = j0; base < j1; base += (int64_t)kUT * kScanBatch) {
    // every lane loads (tokens at or past jlim read the last valid one), so
    // the batch's loads are issued back to back, not one guarded load at a
    // time
    float v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const int64_t j = base + threadIdx.x + (int64_t)k * kUT;
      v[k] = sc[j < jlim ? j : jlim - 1];
    }
    uint32_t key[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const int64_t j = base + threadIdx.x + (int64_t)k * kUT;
      key[k] = j < jlim ? score_key(v[k]) : 0u;
    }
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const int64_t j = base + threadIdx.x + (int64_t)k * kUT;
      f(j, key[k], j < jlim);
    }
  }
}

__device__ __forceinline__ void unit_body(const LayerArgs& a, int u, bool copy, UnitLds& sm) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int s = u / a.n_sg, g = u - s * a.n_sg;
  const SeqArgs& sq = a.seq[s];
  const int w = a.tail;  // tokens kept by rule after the ranked ones
  const int64_t Ls = sq.L - w;
  // the KV heads whose rows this selection keeps
  const int gk0 = a.shared ? 0 : g, gk1 = a.shared ? a.n_kv : g + 1;
  const int64_t n_keep = sq.n_keep;
  const float* sc = sq.scores + (int64_t)g * Ls;
  CKV_GLOBAL int32_t* out = to_global(sq.idx) + (int64_t)g * sq.n_ret;
  if (n_keep < 0) {  // budget >= L: every token stays, in order
    for (int64_t j = tid; j < sq.L; j += kUT) out[j] = (int32_t)j;
    if (copy)
      for (int gk = gk0; gk < gk1; ++gk) copy_run<kUT>(a, sq, gk, 0, 0, sq.L);
    return;
  }
  // 1. the first-level bin from the pooling kernel's histogram, whose loads
  // are in flight while the window rows are copied
  const CKV_GLOBAL uint32_t* ghist = to_global(sq.hist) + (int64_t)g * kHistBins;
  uint32_t hv[kHistBins / kUT];
#pragma unroll
  for (int k = 0; k < kHistBins / kUT; ++k) hv[k] = ghist[tid + k * kUT];
  // the window is always kept, after the prefix tokens
  for (int i = tid; i < w; i += kUT) out[n_keep + i] = (int32_t)(Ls + i);
  if (copy)
    for (int gk = gk0; gk < gk1; ++gk) copy_run<kUT>(a, sq, gk, n_keep, Ls, w);
  if (n_keep == 0) return;
#pragma unroll
  for (int k = 0; k < kHistBins / kUT; ++k) sm.hist[tid + k * kUT] = hv[k];
  __syncthreads();
  find_bin_unit(sm, kHistBins, (uint32_t)n_keep);
  // keys compare on (key >> shift) against prefix: those above are kept, and
  // of those equal to it the `need` lowest-index ones
  uint32_t prefix = sm.res[0], need = (uint32_t)n_keep - sm.res[1], cnt = sm.res[2];
  int shift = kHistShift;
  __syncthreads();

  // gather the keys with `mine` set into the LDS candidate list (one atomic
  // per wave)
  auto gather = [&](uint32_t key, int64_t j, bool mine) {
    const uint64_t m = __ballot(mine);
    if (m) {
      const int leader = __ffsll((unsigned long long)m) - 1;
      uint32_t base = 0;
      if (lane == leader) base = atomicAdd(&sm.n_cand, (uint32_t)__popcll(m));
      base = __shfl(base, leader);
      if (mine) sm.cand[base + __popcll(m & ((1ull << lane) - 1ull))] = make_uint2(key, (uint32_t)j);
    }
  };

  // 2. the exact threshold
  bool in_lds = false, marked = false;
  if (Ls <= kSegTokens && need < cnt && cnt <= (uint32_t)kCandCap) {
    // one pass: the keys above the bin into the bitmap (a wave's 64
    // consecutive tokens give two whole words, written by its lane 0), the
    // bin's keys into LDS
    // the scan writes the bitmap words of whole batches up to Ls; the words
    // past them are cleared here (scanning all 131072 tokens for a short
    // prompt only wrote zeros there)
    const int scanned = (int)((Ls + kBatchTokens - 1) / kBatchTokens) * (kBatchTokens / 32);
    for (int i = tid; i < kSegWords; i += kUT) {
      sm.emap[i] = 0u;
      if (i >= scanned) sm.kmap[i] = 0u;
    }
    if (tid == 0) sm.n_cand = 0u;
    __syncthreads();
    const uint32_t bin = prefix;
    scan_scores(sc, 0, Ls, Ls, [&](int64_t j, uint32_t key, bool in) {
      const uint32_t kb = key >> kHistShift;
      const uint64_t above = __ballot(in && kb > bin);
      if (lane == 0) {
        const int wd = (int)(j >> 5);
        sm.kmap[wd] = (uint32_t)above;
        sm.kmap[wd + 1] = (uint32_t)(above >> 32);
      }
      gather(key, j, in && kb == bin);
    });
    in_lds = marked = true;
  }
  while (shift > 0 && need < cnt) {
    const int nb = shift < 12 ? shift : 12;
    const int nshift = shift - nb;
    const uint32_t nmask = (1u << nb) - 1u;
    if (!in_lds && cnt <= (uint32_t)kCandCap) {
      // gather the bin's keys once; the next levels rank them in LDS
      if (tid == 0) sm.n_cand = 0u;
      __syncthreads();
      scan_scores(sc, 0, Ls, Ls, [&](int64_t j, uint32_t key, bool in) {
        gather(key, j, in && (key >> shift) == prefix);
      });
      in_lds = true;
    }
    for (int i = tid; i <= (int)nmask; i += kUT) sm.hist[i] = 0u;
    __syncthreads();
    if (in_lds) {
      const uint32_t n = sm.n_cand;
      for (uint32_t c = tid; c < n; c += kUT) {
        const uint32_t key = sm.cand[c].x;
        if ((key >> shift) == prefix) atomicAdd(&sm.hist[(key >> nshift) & nmask], 1u);
      }
    } else {
      scan_scores(sc, 0, Ls, Ls, [&](int64_t, uint32_t key, bool in) {
        if (in && (key >> shift) == prefix) atomicAdd(&sm.hist[(key >> nshift) & nmask], 1u);
      });
    }
    __syncthreads();
    find_bin_unit(sm, 1 << nb, need);
    prefix = (prefix << nb) | sm.res[0];
    need -= sm.res[1];
    cnt = sm.res[2];
    shift = nshift;
    __syncthreads();
  }

  // 3. ascending output, one segment of tokens at a time
  uint32_t eq_carry = 0, pos_carry = 0;
  const int gk_n = gk1 - gk0;
  // the kept indices of the segment starting at seg0 from the bitmaps
  auto emit = [&](int64_t seg0) {
    // thread t owns words [t * kPer, (t + 1) * kPer) of the segment
    constexpr int kPer = kSegWords / kUT;
    uint32_t km[kPer], em[kPer];
    uint32_t ne = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      km[i] = sm.kmap[tid * kPer + i];
      em[i] = sm.emap[tid * kPer + i];
      ne += __popc(em[i]);
    }
    uint32_t tot_eq, tot_kept;
    uint32_t eq_rank = eq_carry + block_excl_scan<kUT>(ne, sm.wsum, tot_eq);
    uint32_t nk = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      uint32_t e = em[i];
      while (e) {  // equal keys in token order: the first `need` are kept
        const uint32_t bit = e & (0u - e);
        if (eq_rank < need) km[i] |= bit;
        ++eq_rank;
        e ^= bit;
      }
      nk += __popc(km[i]);
    }
    const uint32_t first = pos_carry + block_excl_scan<kUT>(nk, sm.wsum, tot_kept);
    {
      uint32_t pos = first;
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        uint32_t k = km[i];
        while (k) {
          const int b = __ffs(k) - 1;
          if (pos < (uint32_t)n_keep)
            out[pos] = (int32_t)(seg0 + (int64_t)(tid * kPer + i) * 32 + b);
          ++pos;
          k &= k - 1u;
        }
      }
    }
    // copies of the segment's kept rows, kUnitList rows per round
    const uint32_t n_seg = tot_kept < (uint32_t)n_keep - pos_carry ? tot_kept
                                                                    : (uint32_t)n_keep - pos_carry;
    for (uint32_t r0 = 0; copy && r0 < n_seg; r0 += kUnitList) {
      uint32_t li = first - pos_carry;
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        uint32_t k = km[i];
        while (k) {
          const int b = __ffs(k) - 1;
          if (li >= r0 && li < r0 + kUnitList && li < n_seg) {
            sm.lpos[li - r0] = (int32_t)(pos_carry + li);
            sm.ltok[li - r0] = (int32_t)(seg0 + (int64_t)(tid * kPer + i) * 32 + b);
          }
          ++li;
          k &= k - 1u;
        }
      }
      __syncthreads();
      const uint32_t m = n_seg - r0 < (uint32_t)kUnitList ? n_seg - r0 : (uint32_t)kUnitList;
      for (int gi = 0; gi < gk_n; ++gi)
        copy_rows<kUT>(a, sq, gk0 + gi, m, [&](int64_t i) { return (int64_t)sm.ltok[i]; },
                       [&](int64_t i) { return (int64_t)sm.lpos[i]; });
      __syncthreads();
    }
    eq_carry += tot_eq;
    pos_carry += tot_kept;
    __syncthreads();  // the bitmaps are rewritten by the next segment
  };

  if (marked) {
    // the bin's keys settle against the exact threshold: above it kept,
    // equal to it ranked by token
    const uint32_t n = sm.n_cand;
    for (uint32_t c = tid; c < n; c += kUT) {
      const uint2 e = sm.cand[c];
      const uint32_t p = e.x >> shift, bit = 1u << (e.y & 31u);
      if (p > prefix) atomicOr(&sm.kmap[e.y >> 5], bit);
      else if (p == prefix) atomicOr(&sm.emap[e.y >> 5], bit);
    }
    __syncthreads();
    emit(0);
    return;
  }
  for (int64_t seg0 = 0; seg0 < Ls && pos_carry < (uint32_t)n_keep; seg0 += kSegTokens) {
    const int64_t seg1 = Ls - seg0 < kSegTokens ? Ls : seg0 + kSegTokens;
    // the scan writes the words of whole batches up to seg1, the rest are
    // cleared (the previous segment's emit ended with a barrier)
    const int scanned = (int)((seg1 - seg0 + kBatchTokens - 1) / kBatchTokens) * (kBatchTokens / 32);
    for (int i = scanned + tid; i < kSegWords; i += kUT) sm.kmap[i] = sm.emap[i] = 0u;
    scan_scores(sc, seg0, seg1, seg1, [&](int64_t j, uint32_t key, bool in) {
      const uint32_t p = key >> shift;
      const uint64_t above = __ballot(in && p > prefix);
      const uint64_t equal = __ballot(in && p == prefix);
      if (lane == 0) {
        const int wd = (int)((j - seg0) >> 5);
        sm.kmap[wd] = (uint32_t)above;
        sm.kmap[wd + 1] = (uint32_t)(above >> 32);
        sm.emap[wd] = (uint32_t)equal;
        sm.emap[wd + 1] = (uint32_t)(equal >> 32);
      }
    });
    __syncthreads();
    emit(seg0);
  }
}

__global__ __launch_bounds__(kUT) void select_unit_kernel(const MultiArgs m) {
  __shared__ UnitLds sm;
  const int l = blockIdx.x / m.per_layer;
  unit_body(layer_args(m, l), blockIdx.x - l * m.per_layer, m.unit_copy != 0, sm);
}

}  // namespace

hipError_t launch_select_units(const MultiArgs& m, hipStream_t st, const Timing& tm) {
  return launch(select_unit_kernel, m.n_layers * m.per_layer, kUT, st, tm, m);
}

}  // namespace ckv
