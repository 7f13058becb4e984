// C ABI of the CompressKV prefill-end KV eviction path: argument validation,
// workspace layout, launch sequencing, and the host-side Algorithm 1.
// Declarations and the contract of every entry point are in include/ckv.h.
#include "ckv.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include "ckv_internal.h"

namespace {

thread_local int g_last_hip_error = 0;
// ckv_compress_stack's kernel-argument staging for its multi-layer K-pass
// launches (about 12 KB, so not on the stack)
thread_local ckv::LayersArgs g_layers_args;
thread_local hipEvent_t g_ev_begin[ckv::kNumStages] = {};
thread_local hipEvent_t g_ev_end[ckv::kNumStages] = {};
thread_local bool g_events_on = false;
// ckv_compress_stack: per-layer stage events, and the fork/join events of its
// side stream per device (created on first use, kept for the process)
thread_local void* const* g_stack_begin = nullptr;
thread_local void* const* g_stack_end = nullptr;
thread_local int32_t g_stack_layers = 0;
constexpr int kMaxDevices = 16;
enum SyncEvent { kEvFork = 0, kEvScored = 1, kEvSelected = 2, kNumSyncEvents = 3 };
thread_local hipEvent_t g_sync_ev[kMaxDevices][kNumSyncEvents] = {};

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int elt_bytes(int dtype) { return dtype == CKV_F32 ? 4 : 2; }

// Scores per selection range: at least kRangeMin, and few enough ranges for
// the resolve step to count them in LDS.
int64_t range_size(int64_t Ls) {
  const int64_t per = ceil_div(Ls, ckv::kMaxRanges);
  return per <= ckv::kRangeMin ? ckv::kRangeMin : ceil_div(per, ckv::kRangeMin) * ckv::kRangeMin;
}

// Tokens at the end of a prompt that are kept by rule and not ranked: the
// window with CKV_KEEP_WINDOW, none without (then all L tokens are scored).
int64_t kept_tail(const ckv_layer_desc* d) { return (d->flags & CKV_KEEP_WINDOW) ? d->window : 0; }

// Selections per prompt: one per KV group, or one for the layer.
int64_t sel_groups(const ckv_layer_desc* d) {
  return (d->flags & CKV_SHARE_LAYER) ? 1 : d->num_kv_heads;
}

// K stages of one KV head of a prompt of seq_len tokens.
int64_t k_stages(const ckv_layer_desc* d, int64_t seq_len) {
  return ceil_div(seq_len, ckv::stage_tokens(d->head_dim * elt_bytes(d->dtype)));
}

// Most workgroups per KV head a K pass can use for this prompt.
int64_t max_split(const ckv_layer_desc* d, int64_t seq_len) {
  const int64_t p = ceil_div(k_stages(d, seq_len), ckv::kMinStagesPerWg);
  return p < ckv::kMaxSplit ? p : ckv::kMaxSplit;
}

// Head slots per KV head in the window-sum buffer: one per query head of the
// group (any of them may be chosen).
int64_t wsum_heads(const ckv_layer_desc* d) { return d->num_q_heads / d->num_kv_heads; }

// Chosen heads per K-pass row group (kMaxRows rows), and the most row groups
// ("units") a prompt can have: every KV group with all its heads chosen.
int heads_per_unit(const ckv_layer_desc* d) { return ckv::kMaxRows / ((d->window + 7) / 8 * 8); }
int64_t max_units(const ckv_layer_desc* d) {
  return (int64_t)d->num_kv_heads * ckv::group_units((int)wsum_heads(d), heads_per_unit(d));
}

// Floats per window-sum row: the scored length rounded up to 4, so that every
// row starts 16-byte aligned.
int64_t ws_stride(int64_t Ls) { return (Ls + 3) / 4 * 4; }

// Per-prompt workspace, in order: K-pass partials, head window sums, scores,
// selection control words, histograms, candidates, per-range counts/offsets.
struct WsLayout {
  size_t partial, wsum, scores, ctl, hist, cand, rsure, total;
};

WsLayout seq_ws_layout(const ckv_layer_desc* d, const ckv_seq* s) {
  const int64_t n_kv = d->num_kv_heads, n_sg = sel_groups(d);
  const int64_t Ls = s->seq_len - kept_tail(d);  // scored length
  const int64_t n_ranges = ceil_div(Ls, range_size(Ls));
  WsLayout w;
  size_t o = 0;
  w.partial = o; o += align_up((size_t)max_units(d) * max_split(d, s->seq_len) * ckv::kMaxRows * sizeof(float2));
  w.wsum = o;    o += align_up((size_t)n_kv * wsum_heads(d) * ws_stride(Ls) * sizeof(float));
  w.scores = o;  o += align_up((size_t)n_sg * Ls * sizeof(float));
  w.ctl = o;     o += align_up((size_t)n_sg * ckv::kCtlWords * sizeof(uint32_t));
  w.hist = o;    o += align_up((size_t)n_sg * ckv::kHistBins * sizeof(uint32_t));
  w.cand = o;    o += align_up((size_t)n_sg * Ls * sizeof(uint2));
  w.rsure = o;   o += align_up((size_t)3 * n_sg * n_ranges * sizeof(uint32_t));
  w.total = o;
  return w;
}

size_t seq_ws_bytes(const ckv_layer_desc* d, const ckv_seq* s) { return seq_ws_layout(d, s).total; }

// A call's workspace starts with room for its kernel argument block (the
// multi-layer selection launches of ckv_compress_stack read it from there),
// then holds every prompt's sections in order.
const size_t kWsHeader = align_up(sizeof(ckv::LayerArgs));

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_desc(const ckv_layer_desc* d) {
  if (!d) return CKV_ERR_INVALID_ARG;
  if (d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads)
    return CKV_ERR_INVALID_ARG;
  if (d->num_q_heads > CKV_MAX_Q_HEADS || d->num_kv_heads > CKV_MAX_KV_HEADS)
    return CKV_ERR_UNSUPPORTED;
  if (d->head_dim != 64 && d->head_dim != 128) return CKV_ERR_UNSUPPORTED;
  if (d->dtype != CKV_BF16 && d->dtype != CKV_F16 && d->dtype != CKV_F32) return CKV_ERR_UNSUPPORTED;
  if (d->window < 1) return CKV_ERR_INVALID_ARG;
  if (d->window > CKV_MAX_WINDOW) return CKV_ERR_UNSUPPORTED;
  if (d->pool != CKV_POOL_AVG && d->pool != CKV_POOL_MAX) return CKV_ERR_INVALID_ARG;
  if (d->pool_kernel < 1 || d->pool_kernel % 2 == 0) return CKV_ERR_INVALID_ARG;
  if (d->pool_kernel > CKV_MAX_POOL_KERNEL) return CKV_ERR_UNSUPPORTED;
  if (d->flags & ~(CKV_KEEP_WINDOW | CKV_SHARE_LAYER)) return CKV_ERR_UNSUPPORTED;
  if (!(d->scale > 0.f) && !(d->scale <= 0.f)) return CKV_ERR_INVALID_ARG;  // NaN
  if (isinf(d->scale)) return CKV_ERR_INVALID_ARG;
  return CKV_OK;
}

// What each stage reads/writes of a prompt.
enum Need : unsigned { kNeedQ = 1, kNeedK = 2, kNeedV = 4, kNeedScores = 8, kNeedIdx = 16, kNeedOut = 32 };

int check_seqs(const ckv_layer_desc* d, const ckv_seq* seqs, int32_t n, unsigned need) {
  if (!seqs || n < 1) return CKV_ERR_INVALID_ARG;
  if (n > CKV_MAX_SEQS) return CKV_ERR_UNSUPPORTED;
  const int64_t eb = elt_bytes(d->dtype);
  for (int32_t i = 0; i < n; ++i) {
    const ckv_seq& s = seqs[i];
    if (s.seq_len <= d->window || s.seq_len >= ((int64_t)1 << 31)) return CKV_ERR_INVALID_ARG;
    if (s.budget < (kept_tail(d) > 0 ? kept_tail(d) : 1)) return CKV_ERR_BUDGET;
    if ((need & kNeedQ) && (!s.q_win || !aligned16(s.q_win))) return CKV_ERR_INVALID_ARG;
    if (need & kNeedQ) {
      if (s.q_stride_head < 0 || s.q_stride_row < 0) return CKV_ERR_INVALID_ARG;
      if ((s.q_stride_head * eb) % 16 || (s.q_stride_row * eb) % 16) return CKV_ERR_INVALID_ARG;
      if (d->window > 1 && s.q_stride_row < d->head_dim) return CKV_ERR_INVALID_ARG;
    }
    if ((need & kNeedK) && (!s.k || !aligned16(s.k))) return CKV_ERR_INVALID_ARG;
    if ((need & kNeedV) && (!s.v || !aligned16(s.v))) return CKV_ERR_INVALID_ARG;
    if (need & (kNeedK | kNeedV)) {
      if (s.kv_stride_tok < d->head_dim || s.kv_stride_head < 0) return CKV_ERR_INVALID_ARG;
      if ((s.kv_stride_head * eb) % 16 || (s.kv_stride_tok * eb) % 16) return CKV_ERR_INVALID_ARG;
    }
    if ((need & kNeedScores) && (!s.scores || !aligned16(s.scores))) return CKV_ERR_INVALID_ARG;
    if ((need & kNeedIdx) && !s.idx) return CKV_ERR_INVALID_ARG;
    if ((need & kNeedOut) && (!s.k_out || !s.v_out || !aligned16(s.k_out) || !aligned16(s.v_out)))
      return CKV_ERR_INVALID_ARG;
    if (need & kNeedQ) {
      // caller row statistics: for every prompt or for none
      if ((s.lse != nullptr) != (seqs[0].lse != nullptr)) return CKV_ERR_INVALID_ARG;
      if (s.lse && (((uintptr_t)s.lse & 3u) || s.lse_stride_head < 0 ||
                    (d->window > 1 && s.lse_stride_head < d->window)))
        return CKV_ERR_INVALID_ARG;
    }
  }
  return CKV_OK;
}

// Fill the kernel argument block; workspace pointers are carved per prompt.
int build_args(const ckv_layer_desc* d, const uint8_t* mask, const ckv_seq* seqs, int32_t n,
               char* ws, bool scores_from_ws, ckv::LayerArgs& a) {
  memset(&a, 0, sizeof(a));
  a.num_seqs = n;
  a.n_kv = d->num_kv_heads;
  a.d = d->head_dim;
  a.w = d->window;
  a.w8 = (d->window + 7) / 8 * 8;
  const float scale = d->scale > 0.f ? d->scale : 1.0f / sqrtf((float)d->head_dim);
  a.alpha = (float)((double)scale * 1.4426950408889634);  // log2(e)
  a.pool = d->pool;
  a.kp = d->pool_kernel;
  a.shared = (d->flags & CKV_SHARE_LAYER) ? 1 : 0;
  a.n_sg = (int32_t)sel_groups(d);
  a.lse_given = seqs[0].lse != nullptr;
  a.tail = (int16_t)kept_tail(d);
  if (mask) {
    const int G = d->num_q_heads / d->num_kv_heads;
    int off = 0;
    for (int g = 0; g < d->num_kv_heads; ++g) {
      a.grp_off[g] = (int16_t)off;
      int cnt = 0;
      for (int t = 0; t < G; ++t) {
        const int h = g * G + t;
        if (mask[h]) {
          a.sel_grp[off] = (uint8_t)g;
          a.sel[off++] = (uint8_t)h;
          ++cnt;
        }
      }
      // per-group scope: every group selects with its own heads; shared
      // scope: a group may have none (it is not read)
      if (cnt == 0 && !a.shared) return CKV_ERR_MASK;
    }
    a.grp_off[d->num_kv_heads] = (int16_t)off;
    if (off == 0) return CKV_ERR_MASK;
  }
  // weight of the K-pass work: nqb + kSplitBias for every row group read
  // (groups without a chosen head are not read)
  a.hpr = heads_per_unit(d);
  if (mask)
    for (int g = 0; g < d->num_kv_heads; ++g) {
      const int cnt = a.grp_off[g + 1] - a.grp_off[g];
      if (cnt == 0) continue;
      for (int j = 0; j < ckv::group_units(cnt, a.hpr); ++j)
        a.split_w += (ckv::unit_heads(cnt, a.hpr, j) * a.w8 + 31) / 32 + ckv::kSplitBias;
    }
  a.elt = elt_bytes(d->dtype);
  int32_t blk_kpass = 0, blk_pool = 0, blk_sel = 0, blk_gather = 0;
  if (ws) ws += kWsHeader;
  for (int32_t i = 0; i < n; ++i) {
    const ckv_seq& s = seqs[i];
    ckv::SeqArgs& q = a.seq[i];
    const int64_t Ls = s.seq_len - a.tail;  // scored length
    q.q = s.q_win;
    q.k = s.k;
    q.v = s.v;
    q.q_sh = s.q_stride_head;
    q.q_sr = s.q_stride_row;
    q.kv_sh = s.kv_stride_head;
    q.kv_st = s.kv_stride_tok;
    q.L = s.seq_len;
    q.n_ret = (int32_t)(s.budget < s.seq_len ? s.budget : s.seq_len);
    q.n_keep = s.budget >= s.seq_len ? -1 : s.budget - a.tail;
    q.scores = s.scores;
    q.idx = s.idx;
    q.k_out = s.k_out;
    q.v_out = s.v_out;
    q.lse = s.lse;
    q.lse_sh = s.lse_stride_head;
    // K-pass workgroups of this prompt: about kTargetWgs over the KV heads it
    // reads, shared out by group_split, at least kMinStagesPerWg stages each.
    // They depend on the prompt and the mask alone, so a prompt's results do
    // not depend on the rest of the batch.
    q.n_split = (int32_t)max_split(d, s.seq_len);
    q.n_kpass = 0;
    if (mask)
      for (int g = 0; g < d->num_kv_heads; ++g) {
        const int cnt = a.grp_off[g + 1] - a.grp_off[g];
        for (int j = 0; j < ckv::group_units(cnt, a.hpr); ++j)
          q.n_kpass += ckv::group_split((ckv::unit_heads(cnt, a.hpr, j) * a.w8 + 31) / 32,
                                        a.split_w, q.n_split);
      }
    q.wsum_heads = (int32_t)wsum_heads(d);
    q.ws_stride = ws_stride(Ls);
    q.n_ptiles = (int32_t)ceil_div(Ls, ckv::kPoolTile);
    q.range = (int32_t)range_size(Ls);
    q.n_ranges = (int32_t)ceil_div(Ls, q.range);
    q.n_gblk = (int32_t)ceil_div(q.n_ret, ckv::kGatherRows);
    q.blk_kpass = blk_kpass;
    q.blk_pool = blk_pool;
    q.blk_sel = blk_sel;
    q.blk_gather = blk_gather;
    blk_kpass += q.n_kpass;
    blk_pool += q.n_ptiles * a.n_sg;
    blk_sel += q.n_ranges * a.n_sg;
    blk_gather += q.n_gblk * d->num_kv_heads;
    if (ws) {
      const WsLayout l = seq_ws_layout(d, &s);
      q.partial = reinterpret_cast<float2*>(ws + l.partial);
      q.wsum = reinterpret_cast<float*>(ws + l.wsum);
      if (scores_from_ws && !q.scores) q.scores = reinterpret_cast<float*>(ws + l.scores);
      q.ctl = reinterpret_cast<uint32_t*>(ws + l.ctl);
      q.hist = reinterpret_cast<uint32_t*>(ws + l.hist);
      q.cand = reinterpret_cast<uint2*>(ws + l.cand);
      q.rsure = reinterpret_cast<uint32_t*>(ws + l.rsure);
      ws += l.total;
    }
  }
  return CKV_OK;
}

int grid_kpass(const ckv::LayerArgs& a) {
  const ckv::SeqArgs& q = a.seq[a.num_seqs - 1];
  return q.blk_kpass + q.n_kpass;
}
int grid_pool(const ckv::LayerArgs& a) {
  const ckv::SeqArgs& q = a.seq[a.num_seqs - 1];
  return q.blk_pool + q.n_ptiles * a.n_sg;
}
int grid_sel(const ckv::LayerArgs& a) {
  const ckv::SeqArgs& q = a.seq[a.num_seqs - 1];
  return q.blk_sel + q.n_ranges * a.n_sg;
}
int grid_gather(const ckv::LayerArgs& a) {
  const ckv::SeqArgs& q = a.seq[a.num_seqs - 1];
  return q.blk_gather + q.n_gblk * a.n_kv;
}

int hip_fail(hipError_t e) { return ckv::record_hip_error((int)e); }

// Events of one launch: the stage's begin event on its first kernel and its
// end event on its last (kernel start and end times, no extra packets).
ckv::Timing timing(int stage, bool first, bool last) {
  ckv::Timing t;
  if (g_events_on) {
    if (first) t.start = g_ev_begin[stage];
    if (last) t.stop = g_ev_end[stage];
  }
  return t;
}

// The two K passes (row statistics, then window sums); with caller row
// statistics only the second.
int run_kpasses(const ckv_layer_desc* d, const ckv::LayerArgs& a, hipStream_t st) {
  hipError_t e;
  if (!a.lse_given && (e = ckv::launch_rowstats(d->dtype, a, grid_kpass(a), st,
                                                timing(ckv::kStageRowStats, true, true))) !=
                          hipSuccess)
    return hip_fail(e);
  if ((e = ckv::launch_score(d->dtype, a, grid_kpass(a), st,
                             timing(ckv::kStageScore, true, true))) != hipSuccess)
    return hip_fail(e);
  return CKV_OK;
}

int run_pool(const ckv::LayerArgs& a, hipStream_t st) {
  const hipError_t e = ckv::launch_pool(a, grid_pool(a), st, timing(ckv::kStagePool, true, true));
  return e == hipSuccess ? CKV_OK : hip_fail(e);
}

int run_score(const ckv_layer_desc* d, const ckv::LayerArgs& a, hipStream_t st) {
  const int rc = run_kpasses(d, a, st);
  return rc != CKV_OK ? rc : run_pool(a, st);
}

// Selection on scores already in place. With caller scores (ckv_select) the
// control words and histograms are built here; in ckv_compress_layer the
// scoring kernel built them.
int run_select(const ckv::LayerArgs& a, bool caller_scores, hipStream_t st) {
  hipError_t e;
  const int gs = grid_sel(a);
  const ckv::Timing none;
  if (caller_scores) {
    if ((e = ckv::launch_clear(a, a.num_seqs * a.n_sg, st, timing(ckv::kStageSelect, true, false))) !=
        hipSuccess)
      return hip_fail(e);
    if ((e = ckv::launch_hist(a, gs, st, none)) != hipSuccess) return hip_fail(e);
  }
  if ((e = ckv::launch_filter(a, gs, st, timing(ckv::kStageSelect, !caller_scores, false))) !=
      hipSuccess)
    return hip_fail(e);
  if ((e = ckv::launch_resolve(a, a.num_seqs * a.n_sg, st, timing(ckv::kStageSelect, false, true))) !=
      hipSuccess)
    return hip_fail(e);
  if ((e = ckv::launch_compact(a, gs, st, timing(ckv::kStageGather, true, true))) != hipSuccess)
    return hip_fail(e);
  return CKV_OK;
}

int run_gather(const ckv::LayerArgs& a, hipStream_t st) {
  const hipError_t e = ckv::launch_gather(a, grid_gather(a), st, timing(ckv::kStageGather, true, true));
  if (e != hipSuccess) return hip_fail(e);
  return CKV_OK;
}

}  // namespace

int ckv::record_hip_error(int hip_status) {
  g_last_hip_error = hip_status;
  return CKV_ERR_HIP;
}

extern "C" {

size_t ckv_workspace_bytes(const ckv_layer_desc* desc, const ckv_seq* seqs, int32_t num_seqs) {
  if (check_desc(desc) != CKV_OK || !seqs || num_seqs < 1 || num_seqs > CKV_MAX_SEQS) return 0;
  size_t total = kWsHeader;
  for (int32_t i = 0; i < num_seqs; ++i) {
    if (seqs[i].seq_len <= desc->window || seqs[i].seq_len >= ((int64_t)1 << 31)) return 0;
    total += seq_ws_bytes(desc, &seqs[i]);
  }
  return total;
}

int ckv_score(const ckv_layer_desc* desc, const uint8_t* head_mask, const ckv_seq* seqs,
              int32_t num_seqs, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_desc(desc);
  if (rc != CKV_OK) return rc;
  if (!head_mask) return CKV_ERR_INVALID_ARG;
  if ((rc = check_seqs(desc, seqs, num_seqs, kNeedQ | kNeedK | kNeedScores)) != CKV_OK) return rc;
  if (!workspace || workspace_bytes < ckv_workspace_bytes(desc, seqs, num_seqs) ||
      !aligned16(workspace))
    return CKV_ERR_WORKSPACE;
  ckv::LayerArgs a;
  if ((rc = build_args(desc, head_mask, seqs, num_seqs, (char*)workspace, false, a)) != CKV_OK)
    return rc;
  return run_score(desc, a, (hipStream_t)stream);
}

int ckv_select(const ckv_layer_desc* desc, const ckv_seq* seqs, int32_t num_seqs, void* workspace,
               size_t workspace_bytes, void* stream) {
  int rc = check_desc(desc);
  if (rc != CKV_OK) return rc;
  if ((rc = check_seqs(desc, seqs, num_seqs, kNeedScores | kNeedIdx)) != CKV_OK) return rc;
  if (!workspace || workspace_bytes < ckv_workspace_bytes(desc, seqs, num_seqs) ||
      !aligned16(workspace))
    return CKV_ERR_WORKSPACE;
  ckv::LayerArgs a;
  if ((rc = build_args(desc, nullptr, seqs, num_seqs, (char*)workspace, false, a)) != CKV_OK)
    return rc;
  a.do_gather = 0;
  return run_select(a, true, (hipStream_t)stream);
}

int ckv_gather(const ckv_layer_desc* desc, const ckv_seq* seqs, int32_t num_seqs, void* stream) {
  int rc = check_desc(desc);
  if (rc != CKV_OK) return rc;
  if ((rc = check_seqs(desc, seqs, num_seqs, kNeedK | kNeedV | kNeedIdx | kNeedOut)) != CKV_OK)
    return rc;
  ckv::LayerArgs a;
  if ((rc = build_args(desc, nullptr, seqs, num_seqs, nullptr, false, a)) != CKV_OK) return rc;
  return run_gather(a, (hipStream_t)stream);
}

int ckv_streaming_select(const ckv_layer_desc* desc, const ckv_seq* seqs, int32_t num_seqs,
                         int32_t n_sink, void* stream) {
  int rc = check_desc(desc);
  if (rc != CKV_OK) return rc;
  if (n_sink < 0) return CKV_ERR_INVALID_ARG;
  if ((rc = check_seqs(desc, seqs, num_seqs, kNeedK | kNeedV | kNeedIdx | kNeedOut)) != CKV_OK)
    return rc;
  ckv::LayerArgs a;
  if ((rc = build_args(desc, nullptr, seqs, num_seqs, nullptr, false, a)) != CKV_OK) return rc;
  const hipError_t e = ckv::launch_stream_gather(a, n_sink, grid_gather(a), (hipStream_t)stream);
  return e == hipSuccess ? CKV_OK : hip_fail(e);
}

int ckv_compress_layer(const ckv_layer_desc* desc, const uint8_t* head_mask, const ckv_seq* seqs,
                       int32_t num_seqs, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_desc(desc);
  if (rc != CKV_OK) return rc;
  if (!head_mask) return CKV_ERR_INVALID_ARG;
  if ((rc = check_seqs(desc, seqs, num_seqs, kNeedQ | kNeedK | kNeedV | kNeedIdx | kNeedOut)) !=
      CKV_OK)
    return rc;
  for (int32_t i = 0; i < num_seqs; ++i)
    if (seqs[i].scores && !aligned16(seqs[i].scores)) return CKV_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < ckv_workspace_bytes(desc, seqs, num_seqs) ||
      !aligned16(workspace))
    return CKV_ERR_WORKSPACE;
  ckv::LayerArgs a;
  if ((rc = build_args(desc, head_mask, seqs, num_seqs, (char*)workspace, true, a)) != CKV_OK)
    return rc;
  a.do_hist = 1;
  a.do_gather = 1;
  const hipStream_t st = (hipStream_t)stream;
  if ((rc = run_score(desc, a, st)) != CKV_OK) return rc;
  return run_select(a, false, st);
}

int ckv_compress_stack(const ckv_layer_desc* desc, int32_t n_layers, const uint8_t* head_masks,
                       const ckv_seq* seqs, int32_t num_seqs, void* workspace,
                       size_t workspace_bytes, void* stream, void* side_stream) {
  int rc = check_desc(desc);
  if (rc != CKV_OK) return rc;
  if (n_layers < 1 || !head_masks || !seqs) return CKV_ERR_INVALID_ARG;
  if (num_seqs < 1) return CKV_ERR_INVALID_ARG;
  if (num_seqs > CKV_MAX_SEQS) return CKV_ERR_UNSUPPORTED;
  const hipStream_t st = (hipStream_t)stream;
  const hipStream_t side = (hipStream_t)side_stream;
  const bool two = side != nullptr && side != st;
  // every layer is validated before anything is enqueued
  const size_t slot_bytes = ckv_workspace_bytes(desc, seqs, num_seqs);
  if (slot_bytes == 0) return CKV_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n_layers; ++l) {
    const ckv_seq* ls = seqs + (int64_t)l * num_seqs;
    if ((rc = check_seqs(desc, ls, num_seqs, kNeedQ | kNeedK | kNeedV | kNeedIdx | kNeedOut)) !=
        CKV_OK)
      return rc;
    for (int32_t i = 0; i < num_seqs; ++i) {
      if (ls[i].seq_len != seqs[i].seq_len) return CKV_ERR_INVALID_ARG;
      if (ls[i].scores && !aligned16(ls[i].scores)) return CKV_ERR_INVALID_ARG;
    }
    ckv::LayerArgs probe;
    if ((rc = build_args(desc, head_masks + (int64_t)l * desc->num_q_heads, ls, num_seqs, nullptr,
                         true, probe)) != CKV_OK)
      return rc;
  }
  // Layers go in batches of `batch`, one workspace slot per layer of a batch:
  // the K passes of the batch's layers, then its selection stages as two
  // launches that each cover the whole batch. With a side stream the K passes
  // of consecutive layers alternate between the two streams, so that one
  // layer's launches ramp up while the other's drain; the batch's selection
  // runs on the stream once both streams' K passes of the batch are done, and
  // the side stream starts the next batch only after that selection (it
  // reuses the slots).
  const size_t n_slots = workspace ? workspace_bytes / slot_bytes : 0;
  if (!workspace || !aligned16(workspace) || n_slots < 1) return CKV_ERR_WORKSPACE;
  const int32_t batch = n_slots < (size_t)n_layers ? (int32_t)n_slots : n_layers;
  // fork/join events of this thread on the current device
  hipEvent_t* ev = nullptr;
  if (two) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    if (dev < 0 || dev >= kMaxDevices) return CKV_ERR_UNSUPPORTED;
    ev = g_sync_ev[dev];
    for (int i = 0; i < kNumSyncEvents; ++i)
      if (!ev[i] && (e = hipEventCreateWithFlags(&ev[i], hipEventDisableTiming)) != hipSuccess)
        return hip_fail(e);
    if ((e = hipEventRecord(ev[kEvFork], st)) != hipSuccess) return hip_fail(e);
    if ((e = hipStreamWaitEvent(side, ev[kEvFork], 0)) != hipSuccess) return hip_fail(e);
  }
  // per-layer stage events replace the per-call ones for the duration
  const bool saved_on = g_events_on;
  hipEvent_t saved_b[ckv::kNumStages], saved_e[ckv::kNumStages];
  for (int i = 0; i < ckv::kNumStages; ++i) {
    saved_b[i] = g_ev_begin[i];
    saved_e[i] = g_ev_end[i];
  }
  const bool stack_timed = g_stack_begin != nullptr;
  auto use_layer_events = [&](int32_t l) {
    if (!stack_timed) return;
    g_events_on = l < g_stack_layers;
    for (int i = 0; i < ckv::kNumStages; ++i) {
      g_ev_begin[i] = g_events_on ? (hipEvent_t)g_stack_begin[l * ckv::kNumStages + i] : nullptr;
      g_ev_end[i] = g_events_on ? (hipEvent_t)g_stack_end[l * ckv::kNumStages + i] : nullptr;
    }
  };
  for (int32_t b0 = 0; b0 < n_layers && rc == CKV_OK; b0 += batch) {
    const int32_t nb = n_layers - b0 < batch ? n_layers - b0 : batch;
    char* base = static_cast<char*>(workspace);
    hipError_t e;
    // the previous batch's selection (on the stream) used these slots
    if (two && b0 > 0 &&
        ((e = hipEventRecord(ev[kEvSelected], st)) != hipSuccess ||
         (e = hipStreamWaitEvent(side, ev[kEvSelected], 0)) != hipSuccess)) {
      rc = hip_fail(e);
      break;
    }
    // The K passes in chunks of up to kLayersPerLaunch consecutive layers,
    // one launch per pass and chunk (the argument blocks travel as kernel
    // arguments): one ramp-up and drain per chunk rather than per layer.
    // Chunks alternate between the streams; a chunk's layers all have caller
    // row statistics or all have none. Stage events: the chunk's first layer.
    ckv::LayersArgs& la = g_layers_args;
    ckv::LayerArgs a;  // a layer of the batch (all have the same shape), for the selection below
    int64_t tokens = 0;  // per layer
    for (int32_t s = 0; s < num_seqs; ++s) tokens += seqs[s].seq_len;
    const int per_launch = tokens >= CKV_STACK_CHUNK_TOKENS ? 1
                           : (int)(CKV_STACK_CHUNK_TOKENS / tokens < ckv::kLayersPerLaunch
                                       ? CKV_STACK_CHUNK_TOKENS / tokens
                                       : ckv::kLayersPerLaunch);
    int gather_max = 0;   // the batch's largest per-layer gather grid
    int64_t ret_max = 0;  // and its most rows kept by one selection unit
    for (int32_t i = 0, chunk = 0; i < nb && rc == CKV_OK; ++chunk) {
      int n = 0, blk = 0;
      for (; n < per_launch && i + n < nb; ++n) {
        const int32_t l = b0 + i + n;
        char* ws = base + (size_t)(i + n) * slot_bytes;
        ckv::LayerArgs& al = la.lay[n];
        if ((rc = build_args(desc, head_masks + (int64_t)l * desc->num_q_heads,
                             seqs + (int64_t)l * num_seqs, num_seqs, ws, true, al)) != CKV_OK)
          break;
        if (n > 0 && al.lse_given != la.lay[0].lse_given) break;  // starts the next chunk
        al.do_hist = 1;
        al.do_gather = 1;
        al.table_out = ws;  // the argument block the selection launches read
        la.blk[n] = blk;
        blk += grid_kpass(al);
        if (grid_gather(al) > gather_max) gather_max = grid_gather(al);
        for (int s = 0; s < al.num_seqs; ++s)
          if (al.seq[s].n_ret > ret_max) ret_max = al.seq[s].n_ret;
      }
      if (rc != CKV_OK) break;
      la.n = n;
      la.blk[n] = blk;
      use_layer_events(b0 + i);
      const hipStream_t cs = two && (chunk & 1) ? side : st;
      if (n == 1) {  // one layer: the per-layer kernels
        if ((rc = run_kpasses(desc, la.lay[0], cs)) != CKV_OK) break;
      } else if (!la.lay[0].lse_given &&
          (e = ckv::launch_rowstats_layers(desc->dtype, la, blk, cs,
                                           timing(ckv::kStageRowStats, true, true))) != hipSuccess) {
        rc = hip_fail(e);
        break;
      }
      if (n > 1 && (e = ckv::launch_score_layers(desc->dtype, la, blk, cs,
                                                 timing(ckv::kStageScore, true, true))) != hipSuccess) {
        rc = hip_fail(e);
        break;
      }
      if (i + n == nb) a = la.lay[n - 1];
      i += n;
    }
    if (rc != CKV_OK) break;
    if (two && nb > 1 &&
        ((e = hipEventRecord(ev[kEvScored], side)) != hipSuccess ||
         (e = hipStreamWaitEvent(st, ev[kEvScored], 0)) != hipSuccess)) {
      rc = hip_fail(e);
      break;
    }
    // the batch's selection stages in two launches: the pooling (with the
    // scores and histograms), then one workgroup per selection unit (layer,
    // prompt, selection group) from the threshold to the gathered rows; a
    // third launch copies the rows when a unit keeps more than
    // kUnitCopyRows of them, spread over all CUs rather than one per unit.
    // Timed on the events of the batch's first layer.
    use_layer_events(b0);
    ckv::MultiArgs m;
    m.table = base;
    m.stride = (int64_t)slot_bytes;
    m.n_layers = nb;
    m.unit_copy = ret_max <= ckv::kUnitCopyRows;
    m.pad_ = 0;
    m.per_layer = 0;
    for (int i = 0; i < a.num_seqs; ++i)
      m.per_layer += a.n_sg * (int32_t)ceil_div(a.seq[i].n_ptiles, ckv::kUnitPoolTiles);
    if ((e = ckv::launch_pool_units(m, desc->pool_kernel >> 1, st, timing(ckv::kStagePool, true, true))) != hipSuccess) {
      rc = hip_fail(e);
      break;
    }
    m.per_layer = a.num_seqs * a.n_sg;
    ckv::Timing tm, tm_gather;
    if (g_events_on) {
      tm.start = g_ev_begin[ckv::kStageSelect];
      tm.stop = g_ev_end[ckv::kStageGather];
    }
    if (!m.unit_copy) {  // the gather launch ends the stage
      tm_gather.stop = tm.stop;
      tm.stop = nullptr;
    }
    if ((e = ckv::launch_select_units(m, st, tm)) != hipSuccess) {
      rc = hip_fail(e);
      break;
    }
    m.per_layer = gather_max;
    if (!m.unit_copy && (e = ckv::launch_gather_layers(m, st, tm_gather)) != hipSuccess) {
      rc = hip_fail(e);
      break;
    }
  }
  g_events_on = saved_on;
  for (int i = 0; i < ckv::kNumStages; ++i) {
    g_ev_begin[i] = saved_b[i];
    g_ev_end[i] = saved_e[i];
  }
  return rc;
}

int ckv_allocate_budgets(const double* err_norm, int32_t n_layers, int64_t total, int32_t m,
                         int32_t M, int32_t* out) {
  if (!err_norm || !out || n_layers < 1 || m < 0 || M < m) return CKV_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n_layers; ++i)
    if (!isfinite(err_norm[i])) return CKV_ERR_INVALID_ARG;
  // Every layer starts at the floor m; the remainder R is shared in
  // proportion to the errors, rounded half to even, and clipped to [m, M].
  int64_t sum = (int64_t)m * n_layers;
  const int64_t R = total - sum;
  sum = 0;
  for (int32_t i = 0; i < n_layers; ++i) {
    const int64_t v = (int64_t)m + (int64_t)nearbyint(err_norm[i] * (double)R);
    out[i] = (int32_t)(v < m ? m : (v > M ? M : v));
    sum += out[i];
  }
  // Then single tokens move to the highest-error layer with room (surplus) or
  // leave the lowest-error layer above the floor (deficit); lowest index on ties.
  int64_t delta = total - sum;
  while (delta != 0) {
    int32_t j = -1;
    if (delta > 0) {
      for (int32_t i = 0; i < n_layers; ++i)
        if (out[i] < M && (j < 0 || err_norm[i] > err_norm[j])) j = i;
      if (j < 0) break;
      // the errors do not change, so the same layer keeps winning until it
      // reaches M: move that many tokens at once
      const int64_t step = delta < (int64_t)(M - out[j]) ? delta : (int64_t)(M - out[j]);
      out[j] += (int32_t)step;
      delta -= step;
    } else {
      for (int32_t i = 0; i < n_layers; ++i)
        if (out[i] > m && (j < 0 || err_norm[i] < err_norm[j])) j = i;
      if (j < 0) break;
      // likewise the same layer keeps losing until it reaches m
      const int64_t step = -delta < (int64_t)(out[j] - m) ? -delta : (int64_t)(out[j] - m);
      out[j] -= (int32_t)step;
      delta += step;
    }
  }
  return delta == 0 ? CKV_OK : CKV_ERR_BUDGET;
}

// ---- compression-error profile ---------------------------------------------
namespace {

constexpr int kDecodeTargetWgs = 512;  // decode workgroups over all KV heads
constexpr int kDecodeSlotsPerChunk = 4;

int check_attn(const ckv_attn_desc* d, int32_t T) {
  if (!d || d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads)
    return CKV_ERR_INVALID_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return CKV_ERR_UNSUPPORTED;
  if (d->dtype != CKV_BF16 && d->dtype != CKV_F16 && d->dtype != CKV_F32) return CKV_ERR_UNSUPPORTED;
  if (!(d->scale > 0.f) && !(d->scale <= 0.f)) return CKV_ERR_INVALID_ARG;
  if (isinf(d->scale)) return CKV_ERR_INVALID_ARG;
  if (T < 1) return CKV_ERR_INVALID_ARG;
  if ((int64_t)(d->num_q_heads / d->num_kv_heads) * T > 128) return CKV_ERR_UNSUPPORTED;
  return CKV_OK;
}

int check_cache(const ckv_attn_desc* d, const ckv_kv_cache* c) {
  const int64_t eb = elt_bytes(d->dtype);
  if (!c || !c->k || !c->v || !aligned16(c->k) || !aligned16(c->v) || c->n < 1 ||
      c->n >= ((int64_t)1 << 31))
    return CKV_ERR_INVALID_ARG;
  if (c->stride_tok < d->head_dim || c->stride_head < 0 || (c->stride_tok * eb) % 16 ||
      (c->stride_head * eb) % 16)
    return CKV_ERR_INVALID_ARG;
  return CKV_OK;
}

int check_q(const ckv_attn_desc* d, const void* q, int64_t st, int64_t sh, int32_t T) {
  const int64_t eb = elt_bytes(d->dtype);
  if (!q || !aligned16(q) || st < 0 || sh < 0 || (st * eb) % 16 || (sh * eb) % 16)
    return CKV_ERR_INVALID_ARG;
  if (d->num_q_heads > 1 && sh < d->head_dim) return CKV_ERR_INVALID_ARG;
  if (T > 1 && st < d->head_dim) return CKV_ERR_INVALID_ARG;
  return CKV_OK;
}

// Tokens per decode workgroup for one launch over caches of sum_n tokens in
// all: about kDecodeTargetWgs workgroups over every KV head and prompt, each
// at least one 32-token block, the same length for every prompt.
int64_t decode_chunk_len(const ckv_attn_desc* d, int64_t sum_n) {
  const int64_t c = ceil_div(sum_n * d->num_kv_heads, kDecodeTargetWgs);
  return c <= 32 ? 32 : ceil_div(c, 32) * 32;
}

// Partial rows per slot: a group's T * (H / n_kv) query rows, whole 32-row blocks.
int32_t decode_rows(const ckv_attn_desc* d, int32_t T) {
  return (int32_t)(ceil_div((int64_t)(d->num_q_heads / d->num_kv_heads) * T, 32) * 32);
}

size_t decode_part_bytes(const ckv_attn_desc* d, int32_t T, int64_t n, int64_t chunk) {
  return align_up((size_t)d->num_kv_heads * ceil_div(n, chunk) * kDecodeSlotsPerChunk *
                  decode_rows(d, T) * (d->head_dim + 2) * sizeof(float));
}

void decode_batch_init(const ckv_attn_desc* d, ckv::DecodeBatch& b) {
  b.n = 0;
  b.H = d->num_q_heads;
  b.n_kv = d->num_kv_heads;
  b.d = d->head_dim;
  const float scale = d->scale > 0.f ? d->scale : 1.0f / sqrtf((float)d->head_dim);
  b.alpha = (float)((double)scale * 1.4426950408889634);
  b.blk_off[0] = 0;
  b.mrg_off[0] = 0;
}

// Appends one prompt (its partials at part, chunk tokens per workgroup).
void decode_batch_add(const ckv_attn_desc* d, const void* q, int64_t st, int64_t sh, int32_t T,
                      const ckv_kv_cache* c, float* out, float* part, int64_t chunk,
                      ckv::DecodeBatch& b) {
  ckv::DecodeArgs& a = b.s[b.n];
  a.q = q;
  a.q_st = st;
  a.q_sh = sh;
  a.k = c->k;
  a.v = c->v;
  a.kv_sh = c->stride_head;
  a.kv_st = c->stride_tok;
  a.n = c->n;
  a.out = out;
  a.part = part;
  a.T = T;
  a.prow = decode_rows(d, T);
  a.chunk = (int32_t)chunk;
  a.n_chunks = (int32_t)ceil_div(c->n, chunk);
  a.n_slots = a.n_chunks * kDecodeSlotsPerChunk;
  a.pad_ = 0;
  const int64_t merge_elems = (int64_t)d->num_q_heads * T * d->head_dim;
  b.blk_off[b.n + 1] = b.blk_off[b.n] + d->num_kv_heads * a.n_chunks;
  b.mrg_off[b.n + 1] = b.mrg_off[b.n] + (int32_t)ceil_div(merge_elems, ckv::kDecodeThreads);
  ++b.n;
}

// Partial Y tiles of the W_O projection: n_split K ranges x 32 x 32 tiles.
size_t proj_tiles_bytes(int32_t D, int32_t T, int64_t K) {
  return align_up((size_t)ckv::proj_splits(K) * ceil_div(D, 32) * ceil_div(2 * (int64_t)T, 32) *
                  1024 * sizeof(float));
}

// Columns of the projection's right-hand side X = [A_full | A_comp - A_full],
// padded to whole 32-column blocks, and the bytes of its two 16-bit parts.
int32_t proj_cols(int32_t T) { return (int32_t)(ceil_div(2 * (int64_t)T, 32) * 32); }
size_t proj_split_bytes(int32_t T, int64_t K) { return align_up((size_t)2 * proj_cols(T) * K * 2); }

int check_decode_seq(const ckv_attn_desc* d, const ckv_decode_seq* s) {
  int rc = check_attn(d, s->T);
  if (rc != CKV_OK) return rc;
  if ((rc = check_q(d, s->q, s->q_stride_t, s->q_stride_h, s->T)) != CKV_OK) return rc;
  if ((rc = check_cache(d, &s->cache)) != CKV_OK) return rc;
  if (!s->out || ((uintptr_t)s->out & 3u)) return CKV_ERR_INVALID_ARG;
  return CKV_OK;
}

// A batch goes to the GPU in runs of at most kMaxDecodeSeqs consecutive
// prompts, one launch each: the size of the run that starts at i0, and its
// chunk length.
int32_t decode_run(int32_t i0, int32_t num_seqs) {
  return num_seqs - i0 < ckv::kMaxDecodeSeqs ? num_seqs - i0 : ckv::kMaxDecodeSeqs;
}
int64_t decode_run_chunk(const ckv_attn_desc* d, const ckv_decode_seq* seqs, int32_t i0,
                         int32_t cnt) {
  int64_t sum_n = 0;
  for (int32_t i = i0; i < i0 + cnt; ++i) sum_n += seqs[i].cache.n;
  return decode_chunk_len(d, sum_n);
}

}  // namespace

size_t ckv_decode_workspace_bytes(const ckv_attn_desc* desc, int32_t T, int64_t n) {
  if (check_attn(desc, T) != CKV_OK || n < 1 || n >= ((int64_t)1 << 31)) return 0;
  return decode_part_bytes(desc, T, n, decode_chunk_len(desc, n));
}

int ckv_decode_attention(const ckv_attn_desc* desc, const void* q, int64_t q_stride_t,
                         int64_t q_stride_h, int32_t T, const ckv_kv_cache* cache, float* out,
                         void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_attn(desc, T);
  if (rc != CKV_OK) return rc;
  if ((rc = check_q(desc, q, q_stride_t, q_stride_h, T)) != CKV_OK) return rc;
  if ((rc = check_cache(desc, cache)) != CKV_OK) return rc;
  if (!out || ((uintptr_t)out & 3u)) return CKV_ERR_INVALID_ARG;
  if (!workspace || !aligned16(workspace) ||
      workspace_bytes < ckv_decode_workspace_bytes(desc, T, cache->n))
    return CKV_ERR_WORKSPACE;
  ckv::DecodeBatch b;
  decode_batch_init(desc, b);
  decode_batch_add(desc, q, q_stride_t, q_stride_h, T, cache, out, static_cast<float*>(workspace),
                   decode_chunk_len(desc, cache->n), b);
  const hipError_t e = ckv::launch_decode(desc->dtype, b, (hipStream_t)stream);
  return e == hipSuccess ? CKV_OK : hip_fail(e);
}

size_t ckv_decode_batch_workspace_bytes(const ckv_attn_desc* desc, const ckv_decode_seq* seqs,
                                        int32_t num_seqs) {
  if (!desc || !seqs || num_seqs < 1) return 0;
  for (int32_t i = 0; i < num_seqs; ++i)
    if (check_decode_seq(desc, &seqs[i]) != CKV_OK) return 0;
  size_t total = 0;
  for (int32_t i0 = 0; i0 < num_seqs; i0 += ckv::kMaxDecodeSeqs) {
    const int32_t cnt = decode_run(i0, num_seqs);
    const int64_t chunk = decode_run_chunk(desc, seqs, i0, cnt);
    for (int32_t i = i0; i < i0 + cnt; ++i)
      total += decode_part_bytes(desc, seqs[i].T, seqs[i].cache.n, chunk);
  }
  return total;
}

int ckv_decode_attention_batch(const ckv_attn_desc* desc, const ckv_decode_seq* seqs,
                               int32_t num_seqs, void* workspace, size_t workspace_bytes,
                               void* stream) {
  if (!desc || !seqs || num_seqs < 1) return CKV_ERR_INVALID_ARG;
  for (int32_t i = 0; i < num_seqs; ++i) {
    const int rc = check_decode_seq(desc, &seqs[i]);
    if (rc != CKV_OK) return rc;
  }
  if (!workspace || !aligned16(workspace) ||
      workspace_bytes < ckv_decode_batch_workspace_bytes(desc, seqs, num_seqs))
    return CKV_ERR_WORKSPACE;
  char* part = static_cast<char*>(workspace);
  for (int32_t i0 = 0; i0 < num_seqs; i0 += ckv::kMaxDecodeSeqs) {
    const int32_t cnt = decode_run(i0, num_seqs);
    const int64_t chunk = decode_run_chunk(desc, seqs, i0, cnt);
    ckv::DecodeBatch b;
    decode_batch_init(desc, b);
    for (int32_t i = i0; i < i0 + cnt; ++i) {
      const ckv_decode_seq& s = seqs[i];
      decode_batch_add(desc, s.q, s.q_stride_t, s.q_stride_h, s.T, &s.cache, s.out,
                       reinterpret_cast<float*>(part), chunk, b);
      part += decode_part_bytes(desc, s.T, s.cache.n, chunk);
    }
    const hipError_t err = ckv::launch_decode(desc->dtype, b, (hipStream_t)stream);
    if (err != hipSuccess) return hip_fail(err);
  }
  return CKV_OK;
}

size_t ckv_layer_error_workspace_bytes(const ckv_attn_desc* desc, int32_t T, int64_t n_full,
                                       int64_t n_comp, int32_t D) {
  if (check_attn(desc, T) != CKV_OK || D < 1 || n_full < 1 || n_comp < 1 ||
      n_full >= ((int64_t)1 << 31) || n_comp >= ((int64_t)1 << 31))
    return 0;
  const size_t outs = align_up((size_t)T * desc->num_q_heads * desc->head_dim * sizeof(float));
  const int64_t chunk = decode_chunk_len(desc, n_full + n_comp);
  const size_t parts = decode_part_bytes(desc, T, n_full, chunk) + decode_part_bytes(desc, T, n_comp, chunk);
  const size_t proj = align_up((size_t)(ceil_div(D, 32) + 1) * 2 * T * sizeof(float));
  const int64_t K = (int64_t)desc->num_q_heads * desc->head_dim;
  const size_t proj_y = proj_tiles_bytes(D, T, K);
  const size_t x_hl = proj_split_bytes(T, K);
  return 2 * outs + parts + proj + proj_y + x_hl;
}

int ckv_layer_error(const ckv_attn_desc* desc, const void* q, int64_t q_stride_t,
                    int64_t q_stride_h, int32_t T, const ckv_kv_cache* full,
                    const ckv_kv_cache* comp, const void* w_o, int64_t w_o_stride, int32_t D,
                    float eps, float* ratio, float* e, void* workspace, size_t workspace_bytes,
                    void* stream) {
  int rc = check_attn(desc, T);
  if (rc != CKV_OK) return rc;
  if ((rc = check_q(desc, q, q_stride_t, q_stride_h, T)) != CKV_OK) return rc;
  if ((rc = check_cache(desc, full)) != CKV_OK || (rc = check_cache(desc, comp)) != CKV_OK)
    return rc;
  const int64_t K = (int64_t)desc->num_q_heads * desc->head_dim;
  const int64_t eb = elt_bytes(desc->dtype);
  if (!w_o || !aligned16(w_o) || D < 1 || w_o_stride < K || (w_o_stride * eb) % 16)
    return CKV_ERR_INVALID_ARG;
  if (!(eps >= 0.f) || isinf(eps)) return CKV_ERR_INVALID_ARG;
  if (!ratio || !e || ((uintptr_t)ratio & 3u) || ((uintptr_t)e & 3u)) return CKV_ERR_INVALID_ARG;
  if (!workspace || !aligned16(workspace) ||
      workspace_bytes < ckv_layer_error_workspace_bytes(desc, T, full->n, comp->n, D))
    return CKV_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  const size_t outs = align_up((size_t)T * K * sizeof(float));
  float* a_full = reinterpret_cast<float*>(ws);
  float* a_comp = reinterpret_cast<float*>(ws + outs);
  char* part = ws + 2 * outs;
  // both decodes in one batch: the full cache and the compressed one
  const int64_t chunk = decode_chunk_len(desc, full->n + comp->n);
  const size_t pa = decode_part_bytes(desc, T, full->n, chunk);
  const size_t pb = decode_part_bytes(desc, T, comp->n, chunk);
  float* proj = reinterpret_cast<float*>(part + pa + pb);
  float* proj_y = reinterpret_cast<float*>(
      reinterpret_cast<char*>(proj) + align_up((size_t)(ceil_div(D, 32) + 1) * 2 * T * sizeof(float)));
  const hipStream_t st = (hipStream_t)stream;
  ckv::DecodeBatch db;
  decode_batch_init(desc, db);
  decode_batch_add(desc, q, q_stride_t, q_stride_h, T, full, a_full, reinterpret_cast<float*>(part),
                   chunk, db);
  decode_batch_add(desc, q, q_stride_t, q_stride_h, T, comp, a_comp,
                   reinterpret_cast<float*>(part + pa), chunk, db);
  hipError_t err;
  if ((err = ckv::launch_decode(desc->dtype, db, st)) != hipSuccess) return hip_fail(err);
  ckv::ErrorArgs ea;
  ea.a_full = a_full;
  ea.a_comp = a_comp;
  ea.w = w_o;
  ea.w_stride = w_o_stride;
  ea.T = T;
  ea.D = D;
  ea.K = K;
  ea.eps = eps;
  ea.part = proj;
  ea.part_y = proj_y;
  ea.x_hl = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(proj_y) + proj_tiles_bytes(D, T, K));
  ea.n_split = ckv::proj_splits(K);
  ea.n_cols = proj_cols(T);
  ea.ratio = ratio;
  ea.e = e;
  if ((err = ckv::launch_error(desc->dtype, ea, st)) != hipSuccess) return hip_fail(err);
  return CKV_OK;
}

int ckv_normalize_errors(const double* e, int32_t n_sets, int32_t n_layers, double* e_tilde) {
  if (!e || !e_tilde || n_sets < 1 || n_layers < 1) return CKV_ERR_INVALID_ARG;
  // every profiling set's errors as fractions of that set's total, the
  // fractions averaged over the sets, and the averages as fractions of
  // their own total
  double* acc = e_tilde;
  for (int32_t l = 0; l < n_layers; ++l) acc[l] = 0.0;
  for (int32_t s = 0; s < n_sets; ++s) {
    const double* row = e + (int64_t)s * n_layers;
    double total = 0.0;
    for (int32_t l = 0; l < n_layers; ++l) {
      if (!isfinite(row[l]) || row[l] < 0.0) return CKV_ERR_INVALID_ARG;
      total += row[l];
    }
    if (!(total > 0.0)) return CKV_ERR_INVALID_ARG;
    for (int32_t l = 0; l < n_layers; ++l) acc[l] += (row[l] / total) / (double)n_sets;
  }
  double total = 0.0;
  for (int32_t l = 0; l < n_layers; ++l) total += acc[l];
  for (int32_t l = 0; l < n_layers; ++l) e_tilde[l] = acc[l] / total;
  return CKV_OK;
}

const char* ckv_status_string(int status) {
  switch (status) {
    case CKV_OK: return "ok";
    case CKV_ERR_INVALID_ARG: return "invalid argument";
    case CKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case CKV_ERR_BUDGET: return "budget below the window or allocation infeasible";
    case CKV_ERR_MASK: return "a KV group has no chosen query head";
    case CKV_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case CKV_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int ckv_last_hip_error(void) { return g_last_hip_error; }

static_assert(ckv::kNumStages == CKV_NUM_STAGES, "stage count of the C ABI");
static_assert(sizeof(ckv::LayerArgs) <= 4096, "kernel argument block");

int ckv_set_stack_stage_events(void* const* begin, void* const* end, int32_t n_layers) {
  if (!begin || !end || n_layers <= 0) {
    g_stack_begin = g_stack_end = nullptr;
    g_stack_layers = 0;
    return CKV_OK;
  }
  g_stack_begin = begin;
  g_stack_end = end;
  g_stack_layers = n_layers;
  return CKV_OK;
}

int ckv_set_stage_events(void* const* begin, void* const* end) {
  if (!begin || !end) {
    g_events_on = false;
    for (int i = 0; i < ckv::kNumStages; ++i) g_ev_begin[i] = g_ev_end[i] = nullptr;
    return CKV_OK;
  }
  for (int i = 0; i < ckv::kNumStages; ++i) {
    g_ev_begin[i] = (hipEvent_t)begin[i];
    g_ev_end[i] = (hipEvent_t)end[i];
  }
  g_events_on = true;
  return CKV_OK;
}

}  // extern "C"
