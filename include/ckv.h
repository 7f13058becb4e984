/*
 * ckv.h -- C ABI of the MI355X (gfx950) CompressKV prefill-end KV eviction path.
 *
 * CompressKV (Lin et al., arXiv 2508.02401) evicts prompt KV pairs once, at the
 * end of prefill. Per layer and per KV head (GQA group), only the group's chosen
 * "semantic retrieval" query heads vote: their attention-score rows for the last
 * w prompt positions (the observation window) are summed over the window,
 * pooled along the token axis and averaged over the chosen heads; the tokens
 * with the N highest scores keep their K/V pairs, the rest are evicted
 * (paper Sec. 3.3, "Token Selection Driven by Semantic Retrieval Heads").
 * Per-layer budgets N come from Algorithm 1 (appendix "More Implementation
 * Details").
 *
 * Conventions shared by every entry point:
 *   - Every function returns an int status (CKV_OK or a negative CKV_ERR_*),
 *     never throws, never aborts, never prints.
 *   - All arguments are validated on the host before anything is enqueued; on
 *     error nothing is launched and no output is touched.
 *   - The caller owns every buffer. Device pointers are plain HIP device
 *     addresses (e.g. from torch or hipMalloc); host arrays (head mask,
 *     budgets, errors) are read during the call and not retained. The library
 *     allocates no device memory: scratch space is the caller's workspace,
 *     sized by ckv_workspace_bytes() (ckv_compress_layer_noalloc uses an array
 *     held by the library instead).
 *   - Device work is enqueued asynchronously on the caller's stream
 *     (`stream` is a hipStream_t; NULL means the default stream). Faults
 *     surface at the caller's next synchronisation. Calls that share one
 *     workspace must be ordered (same stream or synchronised).
 *   - The library keeps no state between calls apart from cached device
 *     properties and, for ckv_compress_stack, a few synchronisation events
 *     per host thread and device; it is safe to call from several host
 *     threads with distinct workspaces.
 */
#ifndef CKV_H_
#define CKV_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define CKV_OK 0
#define CKV_ERR_INVALID_ARG (-1) /* null pointer, bad size/stride/alignment, even pool kernel */
#define CKV_ERR_UNSUPPORTED (-2) /* dtype, head_dim, window or head count outside the built set */
#define CKV_ERR_BUDGET (-3)      /* budget below the window (or below 1); Algorithm 1 could not meet the total */
#define CKV_ERR_MASK (-4)        /* a KV group has no chosen query head (per-group scope), or no head at all */
#define CKV_ERR_WORKSPACE (-5)   /* workspace missing or smaller than ckv_workspace_bytes() */
#define CKV_ERR_HIP (-6)         /* a HIP runtime call failed; see ckv_last_hip_error() */

/* ---- enums ------------------------------------------------------------- */
typedef enum { CKV_BF16 = 0, CKV_F16 = 1, CKV_F32 = 2 } ckv_dtype;
typedef enum { CKV_POOL_AVG = 0, CKV_POOL_MAX = 1 } ckv_pool;

/* flags */
/* Window retention (the paper leaves it open; Sec. 3.3 follows SnapKV). With
 * this flag the w window tokens are always kept and count in B: only the
 * prefix [0, L-w) is scored and ranked, and the best B - w prefix tokens are
 * kept beside the window (requires B >= w). Without it every token competes:
 * all L columns are scored (window column L-w+c only by the window rows
 * i >= c that see it), pooled over [0, L), and the best B of all L tokens are
 * kept (requires B >= 1). Shapes that change with this flag are noted below. */
#define CKV_KEEP_WINDOW (1u << 0)
/* Head scope of the selection (paper Sec. 3.3). Without this flag every KV
 * group g ranks its tokens with its own chosen heads and keeps its own index
 * set. With it, the chosen heads of the whole layer (any groups; a group may
 * have none) rank the tokens together: each chosen head is scored against
 * its own group's keys, the pooled vectors of all chosen heads are averaged
 * (each head weighs the same), and one index set is kept for every KV head,
 * as the paper describes. Shapes that change under this flag are noted below. */
#define CKV_SHARE_LAYER (1u << 1)

/* Limits of this build (larger values return CKV_ERR_UNSUPPORTED). */
#define CKV_MAX_Q_HEADS 128
#define CKV_MAX_KV_HEADS 64
#define CKV_MAX_WINDOW 128
#define CKV_MAX_POOL_KERNEL 31
#define CKV_MAX_SEQS 16
/* ckv_compress_stack launches each K pass for n consecutive layers of a
 * batch at once, n = CKV_STACK_CHUNK_TOKENS / (sum of the prompt lengths of a
 * layer), clamped to [1, CKV_STACK_LAYERS_PER_LAUNCH]: short prompts share a
 * launch's ramp-up and drain, long ones keep one launch per layer (the second
 * pass then finds part of the layer's keys still in the Infinity Cache).
 * Per-layer stage events (ckv_set_stack_stage_events) are taken from the first
 * layer of each launch. */
#define CKV_STACK_LAYERS_PER_LAUNCH 3
#define CKV_STACK_CHUNK_TOKENS 98304
/* A KV group's chosen rows, n_chosen(g) * round_up(w, 8), are read from K in
 * row groups of at most this many: a group with more (e.g. 3 or 4 chosen
 * heads at w = 64) is read once per row group, which costs one more pass
 * over that group's keys in each K pass. */
#define CKV_ROWS_PER_READ 128

/* ---- layer descriptor ---------------------------------------------------
 * One attention layer's shape and the selection hyper-parameters.
 *   num_q_heads  H, num_kv_heads n_kv; H % n_kv == 0, group size G = H / n_kv.
 *                Query head h belongs to KV group h / G (contiguous GQA groups).
 *   head_dim     d in {64, 128}.
 *   window       w, the observation window (last w prompt positions), 1..128.
 *   dtype        element type of Q, K, V and of the compact K/V outputs.
 *   scale        logit scale; <= 0 selects 1/sqrt(head_dim). The softmax is
 *                taken over scale * <q, k> (paper Eq. 2 with the usual scale).
 *   pool         CKV_POOL_AVG (zero padding, divide by the kernel size) or
 *                CKV_POOL_MAX (padding ignored); pool_kernel odd, 1..31
 *                (1 = no pooling). Stride 1; the neighbourhood of token j is
 *                [j - k/2, j + k/2] clipped to the ranked prefix [0, L - w).
 *   flags        any of CKV_KEEP_WINDOW and CKV_SHARE_LAYER (other bits:
 *                CKV_ERR_UNSUPPORTED).
 */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t window;
  int32_t dtype;
  float scale;
  int32_t pool;
  int32_t pool_kernel;
  uint32_t flags;
  int32_t reserved;
} ckv_layer_desc;

/* ---- one prompt ---------------------------------------------------------
 * Strides are in elements; the last (head_dim) axis must be contiguous, every
 * pointer 16-byte aligned and every stride a multiple of 16 bytes.
 *   q_win   [H, w, d]: the queries of the last w prompt positions of every
 *           query head; row i of head h at q_win + h*q_stride_head + i*q_stride_row.
 *           Only the chosen heads' rows are read.
 *   k, v    [n_kv, L, d]: the prompt's key/value cache; token t of KV head g
 *           at k + g*kv_stride_head + t*kv_stride_tok (same strides for v).
 *   seq_len L > w, L < 2^31.
 *   budget  B, tokens kept per KV head. With CKV_KEEP_WINDOW it includes the
 *           w window tokens (B >= w) and the top B - w of the prefix
 *           [0, L - w) are kept; without it the top B of all L tokens are kept
 *           (B >= 1). B >= L keeps every token. Ties go to the lower index.
 *   scores  [n_kv, Lsc] fp32 ([Lsc] under CKV_SHARE_LAYER), Lsc = L - w with
 *           CKV_KEEP_WINDOW and L without: the averaged score of every ranked
 *           token. Written by ckv_score, read by ckv_select; may be NULL for
 *           ckv_compress_layer (the workspace holds it then).
 *   idx     [n_kv, min(B, L)] int32 ([min(B, L)] under CKV_SHARE_LAYER):
 *           retained token positions per KV head (or for every head) in
 *           ascending order (with CKV_KEEP_WINDOW the last w are L-w..L-1).
 *           Written by ckv_select, read by ckv_gather.
 *   k_out, v_out [n_kv, min(B, L), d] contiguous, dtype of the layer: the
 *           compact cache, row r of head g is K[g, idx[g, r], :] (idx[r] under
 *           CKV_SHARE_LAYER).
 *   lse     optional fp32 [H, w]: the natural-log log-sum-exp of every window
 *           row's scaled logits over its visible keys (row i of head h at
 *           lse + h*lse_stride_head + i), i.e. log of the softmax normaliser of
 *           paper Eq. 2 for that row, as a causal prefill attention kernel
 *           leaves it behind. Only the chosen heads' rows are read. When given
 *           (for every prompt of the call, or for none), the scoring skips its
 *           first pass over K (the row statistics) and takes these values
 *           instead, so K is read once. lse_stride_head >= w when w > 1;
 *           4-byte aligned. Values must be finite; they are not checked.
 */
typedef struct {
  const void *q_win;
  int64_t q_stride_head;
  int64_t q_stride_row;
  const void *k;
  const void *v;
  int64_t kv_stride_head;
  int64_t kv_stride_tok;
  int64_t seq_len;
  int32_t budget;
  int32_t reserved;
  float *scores;
  int32_t *idx;
  void *k_out;
  void *v_out;
  const float *lse;
  int64_t lse_stride_head;
} ckv_seq;

/* Bytes of device workspace the calls below need for this layer and batch
 * (an upper bound independent of the head mask). Returns 0 on invalid input. */
size_t ckv_workspace_bytes(const ckv_layer_desc *desc, const ckv_seq *seqs, int32_t num_seqs);

/* Token scoring, paper Sec. 3.3 (the chosen heads' attention-score matrices
 * over the observation window, summed over the window, pooled along the token
 * axis, averaged over the chosen heads). head_mask is a host array [H]; nonzero
 * marks a chosen head. Every KV group needs at least one, except under
 * CKV_SHARE_LAYER, where at least one head of the layer must be chosen and
 * groups without one are not read. Writes
 * seqs[s].scores for every prompt s. Window row i (position L-w+i) attends to
 * keys 0..L-w+i; its softmax runs over all of them. With CKV_KEEP_WINDOW only
 * the prefix columns [0, L-w) are scored; without it all L columns are, a
 * window column by the rows that see it. */
int ckv_score(const ckv_layer_desc *desc, const uint8_t *head_mask, const ckv_seq *seqs,
              int32_t num_seqs, void *workspace, size_t workspace_bytes, void *stream);

/* Top-N selection, paper Sec. 3.3 (the N best-scoring tokens are kept):
 * for every prompt and KV head, reads
 * scores (>= 0, finite) and writes idx: with CKV_KEEP_WINDOW the B - w best
 * prefix tokens (higher score first, lower index on ties) in ascending order,
 * then the window positions; without it the B best of all L tokens in
 * ascending order; 0..L-1 when B >= L. */
int ckv_select(const ckv_layer_desc *desc, const ckv_seq *seqs, int32_t num_seqs,
               void *workspace, size_t workspace_bytes, void *stream);

/* Retain/evict, paper Sec. 3.3 (the selected tokens' K/V pairs stay in the
 * cache, the rest are dropped): copies K and V rows idx[g, r] into k_out / v_out bit for bit.
 * idx entries must lie in [0, L). */
int ckv_gather(const ckv_layer_desc *desc, const ckv_seq *seqs, int32_t num_seqs, void *stream);

/* StreamingLLM-style preset, a comparison baseline the paper discusses
 * (Sec. 2): no scoring; per KV head (per prompt when CKV_SHARE_LAYER) keep
 * the first min(n_sink, n_ret) tokens (attention sinks) and the most recent
 * n_ret - that many, n_ret = min(B, L), ascending: idx_out[r] = r, then
 * L - n_ret + r. Writes idx_out and gathers k_out / v_out as ckv_gather
 * does; q_win, scores_out and lse are not used. n_sink >= 0, other checks
 * and errors as ckv_gather. Asynchronous on stream. (The SnapKV-style preset
 * is ckv_compress_layer with every head of every group in head_mask.) */
int ckv_streaming_select(const ckv_layer_desc *desc, const ckv_seq *seqs, int32_t num_seqs,
                         int32_t n_sink, void *stream);

/* The whole per-layer path: ckv_score, ckv_select and ckv_gather in order on
 * one stream (scores may be NULL). */
int ckv_compress_layer(const ckv_layer_desc *desc, const uint8_t *head_mask, const ckv_seq *seqs,
                       int32_t num_seqs, void *workspace, size_t workspace_bytes, void *stream);

/* The whole path over a stack of layers that share one descriptor (every
 * layer of a model at the end of prefill), paper Sec. 3.3 applied per layer.
 *   head_masks [n_layers][H]: layer l's mask at head_masks + l * H.
 *   seqs [n_layers][num_seqs]: layer l's prompts at seqs + l * num_seqs, with
 *       that layer's inputs, budgets and outputs (scores may be NULL); every
 *       layer has the same prompt lengths.
 * Every layer's results are those of ckv_compress_layer on it. The workspace
 * is cut into slots of S = ckv_workspace_bytes(desc, seqs, num_seqs) bytes
 * (n = workspace_bytes / S of them, at least 1). Layers go in batches of n:
 * the two K passes of each layer of a batch, then the batch's selection
 * stages (pooling, top-N, compaction with the gather) as two launches that
 * each cover the whole batch (three when a selection unit keeps more than
 * 512 rows: the gather then has a launch of its own); a slot per layer of the batch keeps its window
 * sums and selection state meanwhile. With side_stream non-NULL and different
 * from stream, the K passes of consecutive layers of a batch alternate
 * between stream and side_stream (one layer's launches start while the
 * other's finish), and the batch's selection runs on stream after both. The
 * call forks side_stream from stream and joins it back, so all its work is
 * ordered after earlier work on stream and before later work on stream, and
 * side_stream is only ordered after its own earlier work besides. On first
 * use with a side stream the library creates 3 events for the calling host
 * thread and device and keeps them until the process ends. If a launch fails
 * mid-way (CKV_ERR_HIP) the layers before it are enqueued and the fork may be
 * left open: synchronise both streams before reuse. */
int ckv_compress_stack(const ckv_layer_desc *desc, int32_t n_layers, const uint8_t *head_masks,
                       const ckv_seq *seqs, int32_t num_seqs, void *workspace,
                       size_t workspace_bytes, void *stream, void *side_stream);

/* ckv_compress_layer for callers that cannot allocate or pass device memory
 * of their own for scratch (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): same arguments apart from the
 * workspace, same checks, kernels and results. The workspace is a device
 * array inside the library of CKV_NOALLOC_MAX_WORKSPACE_BYTES, one per GPU,
 * allocated when the library's code is first loaded on that GPU and held
 * until the process ends; the call itself allocates nothing. It returns
 * CKV_ERR_WORKSPACE when ckv_workspace_bytes(desc, seqs, num_seqs) exceeds
 * that size (one 131072-token prompt of 32 query / 8 KV heads of dim 128
 * needs about 36 MiB), and CKV_ERR_INVALID_ARG when stream belongs to a
 * device other than the current one. Every call on a GPU uses that GPU's one
 * array: calls that may overlap on a GPU (different streams, host threads)
 * race and must be ordered by the caller. The array keeps the last call's
 * contents; nothing in it needs to start cleared. */
#define CKV_NOALLOC_MAX_WORKSPACE_BYTES ((size_t)64 << 20)
int ckv_compress_layer_noalloc(const ckv_layer_desc *desc, const uint8_t *head_mask,
                               const ckv_seq *seqs, int32_t num_seqs, void *stream);

/* Algorithm 1 (error-aware layer-adaptive cache allocation), host only,
 * synchronous. err_norm [n_layers] are the normalised per-layer errors,
 * total is B_total, [m, M] the per-layer bounds. out [n_layers] receives the
 * budgets. round() is round-half-to-even; argmax/argmin ties go to the lowest
 * layer. Returns CKV_OK when sum(out) == total, CKV_ERR_BUDGET when the bounds
 * made that impossible (out still holds the clipped allocation), or
 * CKV_ERR_INVALID_ARG. */
int ckv_allocate_budgets(const double *err_norm, int32_t n_layers, int64_t total, int32_t m,
                         int32_t M, int32_t *out);

/* ---- compression-error profile (paper Sec. 3.4) -------------------------
 * The per-layer errors that Algorithm 1 allocates by: decode attention of T
 * query tokens over the full cache and over the compressed one (Eq. 3-4 for
 * one query row per head, Eq. 2's softmax over every cached key), the
 * attention outputs of all heads concatenated head-major and projected by
 * W_O, and per decoding step t the ratio
 *   || W_O (A_comp,t - A_full,t) || / (|| W_O A_full,t || + eps)      (Eq. 6-8)
 * summed over the steps. Everything accumulates in fp32. */
typedef struct {
  int32_t num_q_heads;  /* H; head h reads KV head h / (H / n_kv) */
  int32_t num_kv_heads;
  int32_t head_dim;     /* 64 or 128 */
  int32_t dtype;        /* ckv_dtype of queries, caches and W_O */
  float scale;          /* <= 0 selects 1/sqrt(head_dim) */
  int32_t reserved;
} ckv_attn_desc;

/* One KV cache [n_kv][n][d] (d contiguous; pointers 16-byte aligned, strides in
 * elements and multiples of 16 bytes), e.g. a prompt's cache or the compact
 * cache ckv_compress_layer wrote (then n = min(B, L), stride_tok = d,
 * stride_head = n * d). */
typedef struct {
  const void *k;
  const void *v;
  int64_t stride_head;
  int64_t stride_tok;
  int64_t n;  /* cached tokens, >= 1 */
} ckv_kv_cache;

/* Workspace of ckv_decode_attention for T query tokens over n cached tokens
 * (0 on invalid input). */
size_t ckv_decode_workspace_bytes(const ckv_attn_desc *desc, int32_t T, int64_t n);

/* out[t][h][:] (fp32, [T][H][d] contiguous) = softmax over the n cached keys
 * of scale * <q[t][h], k[g][j]> applied to v[g][j], g = h / (H / n_kv).
 * q: token t, head h at q + t * q_stride_t + h * q_stride_h (elements; d
 * contiguous). Needs (H / n_kv) * T <= 128. Asynchronous on stream. */
int ckv_decode_attention(const ckv_attn_desc *desc, const void *q, int64_t q_stride_t,
                         int64_t q_stride_h, int32_t T, const ckv_kv_cache *cache, float *out,
                         void *workspace, size_t workspace_bytes, void *stream);

/* ---- decode over ragged caches (Eq. 2-4 at decoding time) ---------------
 * The consumer of the compressed caches: one decoding step of a batch of
 * prompts, each with its own queries and its own cache, e.g. the compact
 * caches ckv_compress_layer wrote for prompts of different lengths and
 * budgets (the cache lengths need not match). Prompt i computes exactly what
 * ckv_decode_attention computes for (q, T, cache, out) of seqs[i]. */
typedef struct {
  const void *q;          /* [T][H][d] at q + t * q_stride_t + h * q_stride_h (elements) */
  int64_t q_stride_t;
  int64_t q_stride_h;
  int32_t T;              /* query tokens; (H / n_kv) * T <= 128 */
  int32_t reserved;
  ckv_kv_cache cache;     /* this prompt's cache, n >= 1 tokens */
  float *out;             /* [T][H][d] fp32, contiguous */
} ckv_decode_seq;

/* Workspace of ckv_decode_attention_batch (0 on invalid input). */
size_t ckv_decode_batch_workspace_bytes(const ckv_attn_desc *desc, const ckv_decode_seq *seqs,
                                        int32_t num_seqs);

/* Decode attention of every prompt of seqs[0..num_seqs). The host array is
 * read during the call only; queries, caches and outputs are device memory
 * owned by the caller. The prompts go to the GPU in launches of up to 24
 * (one decode and one merge kernel each), their workgroups sized from the
 * launch's total cache length. Validates every prompt before any launch;
 * CKV_ERR_INVALID_ARG / CKV_ERR_UNSUPPORTED as ckv_decode_attention,
 * CKV_ERR_WORKSPACE when the workspace is short. Asynchronous on stream. */
int ckv_decode_attention_batch(const ckv_attn_desc *desc, const ckv_decode_seq *seqs,
                               int32_t num_seqs, void *workspace, size_t workspace_bytes,
                               void *stream);

/* Workspace of ckv_layer_error (0 on invalid input). */
size_t ckv_layer_error_workspace_bytes(const ckv_attn_desc *desc, int32_t T, int64_t n_full,
                                       int64_t n_comp, int32_t D);

/* One layer's error (Eq. 6-8) for T decoding steps with queries q (as in
 * ckv_decode_attention): W_O is [D][H*d] (row r at w_o + r * w_o_stride,
 * dtype of desc), eps the paper's 1e-6 or any >= 0. Writes ratio[T] (the
 * per-step terms) and e[0] (their sum), both fp32 device memory. */
int ckv_layer_error(const ckv_attn_desc *desc, const void *q, int64_t q_stride_t,
                    int64_t q_stride_h, int32_t T, const ckv_kv_cache *full,
                    const ckv_kv_cache *comp, const void *w_o, int64_t w_o_stride, int32_t D,
                    float eps, float *ratio, float *e, void *workspace, size_t workspace_bytes,
                    void *stream);

/* Eq. 10-12 on the host: e [n_sets][n_layers] (each set's layer errors, > 0
 * in sum) -> e_tilde [n_layers]: every set normalised to sum 1, the sets
 * averaged, the average normalised to sum 1. CKV_OK or CKV_ERR_INVALID_ARG. */
int ckv_normalize_errors(const double *e, int32_t n_sets, int32_t n_layers, double *e_tilde);

/* Static description of a status code. */
const char *ckv_status_string(int status);

/* hipError_t of the most recent CKV_ERR_HIP returned on this host thread. */
int ckv_last_hip_error(void);

/* Optional per-stage timing for profiling. While begin/end are non-NULL,
 * each stage's first kernel launch records its start time into begin[s] and
 * its last kernel records its end time into end[s] (hipExtLaunchKernel events:
 * no marker packets are added to the stream, so the timing does not perturb
 * the launches). Stages: 0 row statistics (K pass 1), 1 window sums (K pass
 * 2; the small merge kernel between the passes is not covered), 2 pooling,
 * head mean and histogram, 3 selection (threshold search), 4 compaction and
 * gather. Arrays are hipEvent_t[CKV_NUM_STAGES] owned by the caller, created
 * with timing enabled; a NULL entry leaves that stage untimed (each timed
 * launch costs a few microseconds of dispatch overlap); pass NULL arrays to
 * stop. Per host thread. */
#define CKV_NUM_STAGES 5
int ckv_set_stage_events(void *const *begin, void *const *end);

/* Per-layer stage timing of ckv_compress_stack: begin/end hold
 * n_layers * CKV_NUM_STAGES events (layer l, stage s at index
 * l * CKV_NUM_STAGES + s; NULL entries untimed) and apply to layers
 * 0..n_layers-1 of the following ckv_compress_stack calls on this host thread,
 * in place of the ckv_set_stage_events ones; NULL arrays stop it. The arrays
 * are read at each call, not copied: keep them alive while set. Stages 0-1
 * are per layer, on the stream; stages 2-4 cover a whole batch of layers and
 * use the entries of the batch's first layer (on the side stream when there
 * is one). */
int ckv_set_stack_stage_events(void *const *begin, void *const *end, int32_t n_layers);

#ifdef __cplusplus
}
#endif

#endif /* CKV_H_ */
