// Internal launch interface between the C ABI layer (ckv_api.cpp) and the
// gfx950 kernels (ckv_score.hip, ckv_select.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ckv.h"

namespace ckv {

// Stores a HIP status for ckv_last_hip_error (per host thread) and returns
// CKV_ERR_HIP.
int record_hip_error(int hip_status);


constexpr int kMaxSeqs = 16;
constexpr int kMaxQHeads = 128;
constexpr int kMaxKvHeads = 64;
constexpr int kMaxRows = 128;      // chosen-head rows per group after padding each head to 8
constexpr int kKpThreads = 256;    // threads per K-pass workgroup
constexpr int kStageBytes = 16384; // K bytes per LDS stage of the two K passes
constexpr int kMaxSplit = 512;     // workgroups per (prompt, KV head) in a K pass
constexpr int kMinStagesPerWg = 65536 / kStageBytes; // K stages per workgroup (at least 64 KB)
constexpr int kTargetWgs = 512;    // K-pass workgroups per prompt: 2 on each of 256 CUs
constexpr int kCUs = 256;          // compute units of the MI355X
constexpr int kPoolTile = 2048;    // scores per pooling workgroup
constexpr int kUnitPoolTiles = 4;  // tiles per pooling workgroup of ckv_compress_stack
constexpr int kMaxPoolRadius = 15; // pool kernel <= 2*15+1
constexpr int kGatherRows = 64;    // retained rows per gather workgroup
// A selection batch whose largest unit keeps more rows than this copies them
// in a gather launch of its own: one workgroup per unit copies too slowly.
constexpr int kUnitCopyRows = 512;
constexpr int kHistBits = 12;      // first-level histogram: key bits 30..19
constexpr int kHistBins = 1 << kHistBits;
constexpr int kHistShift = 31 - kHistBits;
constexpr int kRangeMin = 4096;    // scores per selection workgroup (at least)
constexpr int kMaxRanges = 1024;   // selection ranges per KV head (at most)

// Per-(prompt, KV head) control words of the selection, in the workspace.
enum Ctl {
  kCtlBin = 0,         // first-level bin of the threshold key
  kCtlAbove = 1,       // keys in higher bins (all kept)
  kCtlBinCount = 2,    // keys in the threshold bin (the candidates)
  kCtlNumCand = 3,     // candidates appended so far
  kCtlPrefix = 4,      // threshold: keys compare on (key >> shift) against prefix
  kCtlShift = 5,
  kCtlNeedEq = 6,      // keys equal to the threshold to keep, lowest index first
  kCtlWords = 16
};

enum Stage {
  kStageRowStats = 0,
  kStageScore = 1,
  kStagePool = 2,
  kStageSelect = 3,
  kStageGather = 4,
  kNumStages = 5
};

// K-pass workgroups of one KV group (a prompt's groups together get at most
// kTargetWgs, rounded down: one workgroup past what the CUs hold at once
// would run after the others and double the launch). A stage costs a fixed
// part plus a part per 32-row query block of the group's chosen rows, so
// groups get workgroups in proportion to nqb + kSplitBias; w_total is that
// weight summed over the groups read, and cap bounds the count by the
// prompt's stages. A group without chosen heads (nqb == 0, shared scope only)
// gets one workgroup, which reads nothing.
constexpr int kSplitBias = 3;
// A KV group's chosen heads are read by the K passes in row groups ("units")
// of at most hpr heads (kMaxRows rows); a group without chosen heads is one
// unit that reads nothing. Unit j holds heads j*hpr .. of the group.
__host__ __device__ inline int group_units(int cnt, int hpr) {
  return cnt == 0 ? 1 : (cnt + hpr - 1) / hpr;
}
__host__ __device__ inline int unit_heads(int cnt, int hpr, int j) {
  const int r = cnt - j * hpr;
  return r < hpr ? r : hpr;
}

__host__ __device__ inline int group_split(int nqb, int w_total, int cap) {
  if (nqb == 0) return 1;
  const int p = (int)((int64_t)kTargetWgs * (nqb + kSplitBias) / w_total);
  return p < 1 ? 1 : (p > cap ? cap : p);
}

// Tokens per K stage for rows of row_bytes: kStageBytes, or one 32-token
// block of larger rows.
constexpr int stage_tokens(int row_bytes) {
  return 32 * row_bytes > kStageBytes ? 32 : kStageBytes / row_bytes;
}

// One prompt of the batch, in the form the kernels read.
struct SeqArgs {
  const void* q;
  const void* k;
  const void* v;
  int64_t q_sh, q_sr;      // elements
  int64_t kv_sh, kv_st;    // elements
  int64_t L;
  int32_t n_ret;           // min(B, L)
  int32_t n_keep;          // B - w prefix tokens kept, or -1 when B >= L (keep all)
  float* scores;           // [n_kv][L - w]
  int32_t* idx;            // [n_kv][n_ret]
  void* k_out;             // [n_kv][n_ret][d]
  void* v_out;
  const float* lse;        // caller's window-row log-sum-exp [H][w] (natural log), or null
  int64_t lse_sh;          // its head stride
  // workspace
  float2* partial;         // [unit][n_split][kMaxRows]: (max logit, sum exp2) per workgroup
  float* wsum;             // [n_kv][wsum_heads][ws_stride]: window sum of each chosen head
  uint32_t* ctl;           // [n_kv][kCtlWords]
  uint32_t* hist;          // [n_kv][kHistBins]
  uint2* cand;             // [n_kv][L - w]: (key, index) of threshold-bin candidates
  uint32_t* rsure;         // [3][n_sg][n_ranges], per range: keys above the threshold bin;
                           // then the output offset; then threshold-equal keys before it
  int32_t n_split;         // most K-pass workgroups of one KV head (group_split's cap)
  int32_t n_kpass;         // K-pass workgroups of this prompt (all KV heads)
  int64_t ws_stride;       // floats per window-sum row: L - w rounded up to 4
  int32_t wsum_heads;      // head slots per KV head in wsum
  int32_t n_ptiles;        // ceil((L - w) / kPoolTile)
  int32_t n_ranges;        // ceil((L - w) / range)
  int32_t range;           // scores per selection range (multiple of kRangeMin)
  int32_t blk_kpass;       // first workgroup of this prompt in the two K-pass grids
  int32_t blk_pool;        // ... in the pooling grid
  int32_t blk_sel;         // ... in the selection grids (n_kv * n_ranges per prompt)
  int32_t blk_gather;      // ... in the gather grid
  int32_t n_gblk;          // gather workgroups per KV head
};

// One layer call.
struct LayerArgs {
  int32_t num_seqs;
  int32_t n_kv;
  int32_t d;
  int32_t w;
  int32_t w8;              // w rounded up to a multiple of 8: rows reserved per chosen head
  float alpha;             // logit scale * log2(e): exp(scale*s) == exp2(alpha*s)
  int32_t pool;            // 0 average, 1 max
  int32_t kp;              // odd pool kernel
  int32_t hpr;             // chosen heads per K-pass row group: kMaxRows / w8
  int32_t elt;             // bytes per element of Q/K/V
  int32_t do_hist;         // scoring also builds the selection histogram
  int32_t do_gather;       // compaction also copies the kept K/V rows
  int32_t shared;          // one selection per prompt from the layer's chosen heads
  int32_t n_sg;            // selection groups per prompt: n_kv, or 1 when shared
  int32_t split_w;         // sum over the groups read of nqb + kSplitBias (group_split)
  int32_t lse_given;       // every prompt carries lse: the row-statistics pass is skipped
  void* table_out;         // the scoring kernel copies this block here (device), or null
  int16_t grp_off[kMaxKvHeads + 1];  // chosen heads of group g: sel[grp_off[g] .. grp_off[g+1])
  uint8_t sel[kMaxQHeads];
  uint8_t sel_grp[kMaxQHeads];       // KV group of chosen head t (sel[t] / G)
  int16_t tail;            // w when the window tokens are kept by rule (then only
                           // [0, L - w) is scored and ranked), 0 when every token competes
  SeqArgs seq[kMaxSeqs];
};

// The K passes of several layers in one launch (ckv_compress_stack): the
// argument blocks themselves travel as kernel arguments, layer l's
// workgroups at blk[l] .. blk[l+1].
constexpr int kLayersPerLaunch = CKV_STACK_LAYERS_PER_LAUNCH;
struct LayersArgs {
  LayerArgs lay[kLayersPerLaunch];
  int32_t n;                        // layers in this launch
  int32_t blk[kLayersPerLaunch + 1];
};

// Several layers' selection stages in one launch: layer l's argument block is
// in device memory at table + l * stride (the scoring kernel of that layer put
// it there), and every layer has per_layer workgroups.
struct MultiArgs {
  const char* table;
  int64_t stride;
  int32_t per_layer;
  int32_t n_layers;
  int32_t unit_copy;  // selection units copy their kept rows (else a gather launch follows)
  int32_t pad_;
};

// Decode attention of T query tokens over one KV cache: one prompt of a
// decode batch.
struct DecodeArgs {
  const void* q;           // [T][H][d]: token t, head h at t * q_st + h * q_sh
  int64_t q_st, q_sh;
  const void* k;           // [n_kv][n][d]
  const void* v;
  int64_t kv_sh, kv_st;
  int64_t n;               // cached tokens
  float* out;              // [T][H][d] fp32
  float* part;             // [n_kv][n_slots][prow][d + 2]: O rows, then (max, sum)
  int32_t T;
  int32_t prow;            // partial rows per slot: the group's query rows rounded up to 32
  int32_t chunk;           // cached tokens per workgroup
  int32_t n_chunks;
  int32_t n_slots;         // partial slots per KV head: n_chunks * 4
  int32_t pad_;
};

// Up to kMaxDecodeSeqs prompts (ragged caches) in one pair of launches: the
// decode workgroups of prompt i are [blk_off[i], blk_off[i+1]), its merge
// workgroups [mrg_off[i], mrg_off[i+1]).
constexpr int kProjSplit = 16;     // fewest K ranges of the W_O projection (partial tiles added in order)
constexpr int kProjRangeK = 256;   // most k per K range of the 16-bit projection
// K ranges of the W_O projection for K = H * d columns of W_O.
inline int proj_splits(int64_t K) {
  const int64_t n = (K + kProjRangeK - 1) / kProjRangeK;
  return n > kProjSplit ? (int)n : kProjSplit;
}
constexpr int kMaxDecodeSeqs = 24;
constexpr int kDecodeThreads = 256;  // threads of the decode and merge workgroups
struct DecodeBatch {
  DecodeArgs s[kMaxDecodeSeqs];
  int32_t blk_off[kMaxDecodeSeqs + 1];
  int32_t mrg_off[kMaxDecodeSeqs + 1];
  int32_t n;               // prompts
  int32_t H, n_kv, d;
  float alpha;             // logit scale * log2(e)
};
static_assert(sizeof(DecodeBatch) <= 4096, "decode batch is passed as kernel arguments");

// W_O projection and error ratios of one layer.
struct ErrorArgs {
  const float* a_full;     // [T][K] decode outputs with the full cache (K = H * d)
  const float* a_comp;     // [T][K] with the compressed cache
  const void* w;           // [D][K] W_O, row r at r * w_stride
  int64_t w_stride;
  int32_t T, D;
  int64_t K;
  float eps;
  float* part;             // [ceil(D / 32) + 1][2T]: column sums of Y^2 per 32 rows, then in all
  float* part_y;           // [n_split][ceil(D / 32)][ceil(2T / 32)][32][32]: Y tiles per K range
  int32_t n_split;         // K ranges: proj_splits(K)
  uint16_t* x_hl;          // 16-bit W_O: X = [A_full | A_comp - A_full] as [2][n_cols][K], the
                           // high parts, then the low parts (X - high), in W_O's 16-bit type
  int32_t n_cols;          // ceil(2T / 32) * 32
  float* ratio;            // [T]
  float* e;                // [1]
};

// Optional timing of one launch: start receives the kernel's start time and
// stop its end time (hipExtLaunchKernel events, which add no marker packets to
// the stream). Either may be null.
struct Timing {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// dtype codes match ckv_dtype. grid is the number of workgroups.
hipError_t launch_rowstats(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_score(int dtype, const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_rowstats_layers(int dtype, const LayersArgs& m, int grid, hipStream_t st,
                                  const Timing& tm);
hipError_t launch_score_layers(int dtype, const LayersArgs& m, int grid, hipStream_t st,
                               const Timing& tm);
hipError_t launch_pool(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_clear(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_hist(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_filter(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_resolve(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_compact(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
hipError_t launch_gather(const LayerArgs& a, int grid, hipStream_t st, const Timing& tm);
// pooling, head mean, scores and histograms of a batch of layers
// (per_layer = sum over prompts of selection groups * ceil(n_ptiles /
// kUnitPoolTiles)), then the top-N through compaction and gather of every
// selection unit (layer, prompt, selection group), one workgroup each
// (per_layer = prompts * selection groups)
hipError_t launch_pool_units(const MultiArgs& m, int radius, hipStream_t st, const Timing& tm);
// decode attention (partials, then their merge into a.out) and the error
// ratios (projection partials, then the ratios and their sum)
hipError_t launch_decode(int dtype, const DecodeBatch& b, hipStream_t st);
hipError_t launch_stream_gather(const LayerArgs& a, int32_t sinks, int grid, hipStream_t st);
hipError_t launch_error(int w_dtype, const ErrorArgs& a, hipStream_t st);
hipError_t launch_select_units(const MultiArgs& m, hipStream_t st, const Timing& tm);
// Gather of every layer of a batch: per_layer = the largest per-layer gather grid.
hipError_t launch_gather_layers(const MultiArgs& m, hipStream_t st, const Timing& tm);

}  // namespace ckv
