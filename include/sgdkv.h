/*
 * sgdkv.h -- C ABI of the SGD-KV hot path for AMD Instinct MI355X (gfx950).
 *
 * SGD-KV (Liu et al., "SGD-KV: Summarization Guided KV Cache Compression")
 * compresses a long prompt's KV cache per KV head: each head gets a budget
 * from its summarization score (Sec. 3.3, Eq. 2, redistributed by Appendix
 * A.1, Algorithm 1), and inside that budget it keeps the tokens with the
 * largest cumulative attention of a final observation window (Sec. 3.3, last
 * paragraph; Sec. 5), always keeping an initial sink and a recent window.
 * Budgets apply per KV head, before the heads are repeated for GQA
 * (Appendix A.2). Decode attention then reads the ragged compressed cache.
 *
 * Conventions shared by every entry point:
 *   - Every function returns an sgdkv_status; no exception crosses the ABI.
 *     Arguments are checked before anything is enqueued: on an
 *     INVALID_ARG, UNSUPPORTED or WORKSPACE error nothing has been written
 *     and nothing enqueued. SGDKV_ERR_HIP from a kernel launch partway
 *     through a call can leave the call's earlier kernels enqueued (their
 *     outputs are then undefined). sgdkv_last_error() describes the failure.
 *   - The caller owns all memory. The library never allocates device memory;
 *     scratch space comes from a caller buffer sized by *_workspace_size.
 *   - Device work is enqueued on `stream` (a hipStream_t passed as void*;
 *     NULL = the null stream) and is asynchronous. Device faults surface at
 *     the caller's next synchronisation.
 *   - Device pointers must be 16-byte aligned. Tensors are dense, row-major,
 *     in the layouts given below.
 *   - Outputs are bitwise reproducible run to run. The only atomics are
 *     integer histogram counts.
 *   - Calls on different streams are independent given distinct workspaces.
 */
#ifndef SGDKV_H
#define SGDKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sgdkv_status;
#define SGDKV_OK 0
#define SGDKV_ERR_INVALID_ARG 1 /* a size, pointer, alignment or value is out of range */
#define SGDKV_ERR_UNSUPPORTED 2 /* valid, but not built: head_dim, group size, ... */
#define SGDKV_ERR_WORKSPACE 3   /* workspace too small or misaligned */
#define SGDKV_ERR_HIP 4         /* the HIP runtime refused a call (no device, launch failure) */

#define SGDKV_DTYPE_F32 0
#define SGDKV_DTYPE_BF16 1

/* Thread-local description of the last failure on this thread; valid until
 * the next sgdkv_* call on the same thread. Never NULL. */
const char* sgdkv_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int32_t sgdkv_version(void);

/* ------------------------------------------------------------------ */
/* Head budgets (host only; never touches the device).                */

/* GQA reduction of per-attention-head summarization scores to one score per
 * KV head: the maximum over the G = Hq/Hkv query heads of each group
 * (Appendix A.7, where max beats mean). Query head q belongs to KV head q/G.
 * per_qhead: host [L][Hq] fp64. per_kvhead_out: host [L][Hkv] fp64.
 * Errors: L, Hq, Hkv < 1; Hq not a multiple of Hkv; NULL pointers. */
sgdkv_status sgdkv_reduce_query_head_scores(const double* per_qhead, int32_t L, int32_t Hq,
                                            int32_t Hkv, double* per_kvhead_out);

/* Total number of kept rows over all L*H KV heads for a budget ratio R.
 * of_middle = 0: R of all rows, floor(R*L*H*C) -- the "KV memory reduced by
 *                up to 75 %" reading at R = 25 % (abstract, Sec. 1).
 * of_middle = 1: Eq. 2 summed over heads, R applied to the compressible
 *                middle only: L*H*(s+W) + floor(R*L*H*(C-s-W)) (Sec. 3.3).
 * Errors: R outside [0,1]; L, H, C < 1; s, W < 0; s+W > C; a total that
 * cannot cover every head's sink and window (of_middle = 0). */
sgdkv_status sgdkv_total_from_ratio(double R, int32_t L, int32_t H, int64_t C, int64_t b_sink,
                                    int64_t b_window, int32_t of_middle, int64_t* total_out);

/* Per-KV-head budgets b_h for all L*H heads (Sec. 3.3, Eq. 2; Appendix A.1,
 * Algorithm 1). head_scores: host [L][H] fp64 raw summarization scores
 * (>= 0, finite), normalised internally over all L*H heads. Every head keeps
 * b_sink initial and b_window recent rows; the rest of total_budget,
 * T = total_budget - L*H*(b_sink+b_window), is shared over the middles of
 * length M = C - b_sink - b_window in proportion to the score:
 *   x_h = (sigma_h / sum(sigma)) * T   (all-zero scores: uniform shares),
 * evaluated in fp64 in exactly that order (the quotient first, then the
 * product; sum(sigma) added in flat layer-major order), since the rounding
 * decides the integer budgets.
 * mode 0 (default, Algorithm 1): x_h rounded by largest remainder (ties:
 *   larger score, then lower flat index); every middle capped at M; the
 *   excess handed to the remaining heads in descending score order (ties:
 *   lower index), each filled up to M before the next.
 * mode 1 (proportional water level): x_h = min(lambda*sigma_h, M) with the
 *   exact level lambda making the sum T, then rounded as above.
 * budgets_out: host [L][H] int64, b_h = b_sink + b_window + m_h, summing to
 * total_budget, each in [b_sink + b_window, C].
 * Errors: sizes as for sgdkv_total_from_ratio; a score < 0, NaN or Inf;
 * total_budget outside [L*H*(s+W), L*H*C]; mode not 0/1; NULL pointers. */
sgdkv_status sgdkv_allocate_budgets(const double* head_scores, int32_t L, int32_t H, int64_t C,
                                    int64_t b_sink, int64_t b_window, int64_t total_budget,
                                    int32_t mode, int64_t* budgets_out);

/* Allocation variants of the head-configuration ablation (Appendix A.7,
 * Table 5). With M = C - s - W and m_h the middle of the plain allocation:
 *   SGDKV_ALLOC_PLAIN           sgdkv_allocate_budgets.
 *   SGDKV_ALLOC_THR             scores strictly below the mean of all L*H
 *                               scores become 0, then the plain allocation
 *                               ("SGD-KV (thr)").
 *   SGDKV_ALLOC_REVERSE         each head keeps M - m_h middle rows instead of
 *                               m_h ("SGD-KV (Reverse)": 10 % becomes 90 %); the
 *                               budgets then sum to L*H*(C + s + W) - total.
 *   SGDKV_ALLOC_MIX             the plain allocation of the average of the
 *                               normalised head_scores and the normalised
 *                               second_scores (an all-zero vector normalises to
 *                               uniform) ("SGD-KV + HeadKV" with R2 scores).
 *   SGDKV_ALLOC_BINARY          the floor(full_fraction*L*H) heads first in
 *                               (score descending, index ascending) order get
 *                               C rows, the others s + W ("DuoAttention (Sum.)");
 *                               total_budget and mode are not used.
 *   SGDKV_ALLOC_BINARY_REVERSE  the same number of heads last in that order get
 *                               C rows ("DuoAttention (Sum., Reverse)").
 * second_scores: host [L][H], required by MIX only (else may be NULL).
 * budgets_out: host [L][H] int64. Errors (nothing written): those of
 * sgdkv_allocate_budgets for the variants that use it; an unknown variant;
 * MIX without valid second_scores; full_fraction outside [0,1] (BINARY*). */
#define SGDKV_ALLOC_PLAIN 0
#define SGDKV_ALLOC_THR 1
#define SGDKV_ALLOC_REVERSE 2
#define SGDKV_ALLOC_MIX 3
#define SGDKV_ALLOC_BINARY 4
#define SGDKV_ALLOC_BINARY_REVERSE 5
sgdkv_status sgdkv_allocate_budgets_variant(const double* head_scores, const double* second_scores, int32_t L,
                                            int32_t H, int64_t C, int64_t b_sink, int64_t b_window,
                                            int64_t total_budget, int32_t mode, int32_t variant,
                                            double full_fraction, int64_t* budgets_out);

/* Row offsets of the ragged per-KV-head cache of one layer (host only). The
 * cache is kept per KV head, before GQA repetition (Appendix A.2): segment
 * (b, h) holds the b_h kept rows of KV head h of sequence b, segments in
 * (b, h) order. With T_layer = sum_h layer_budgets[h]:
 *   offsets_out[b*Hkv + h] = b*T_layer + sum_{h' < h} layer_budgets[h'],
 *   offsets_out[B*Hkv]     = B*T_layer.
 * These are the values sgdkv_compress_layer writes to its device offsets_out
 * for the same budgets; sgdkv_decode_attention takes them as offsets_host.
 * layer_budgets: host [Hkv] int64 >= 0. offsets_out: host [B*Hkv+1] int64.
 * Errors (nothing written): batch or num_kv_heads < 1; a negative budget;
 * B*T_layer beyond 2^62; NULL pointers. */
sgdkv_status sgdkv_segment_offsets(const int64_t* layer_budgets, int32_t batch, int32_t num_kv_heads,
                                   int64_t* offsets_out);

/* ------------------------------------------------------------------ */
/* One layer's compression (device).                                   */

typedef struct sgdkv_compress_desc {
  int32_t batch;        /* B >= 1 sequences */
  int32_t num_q_heads;  /* Hq */
  int32_t num_kv_heads; /* Hkv, Hq % Hkv == 0, Hkv <= 64 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t obs_window;   /* w >= 1: the last w prompt positions are the window rows */
  int32_t pool_kernel;  /* odd k_p >= 1: average pooling, stride 1, zero padding */
  int64_t seq_len;      /* C: prompt length */
  int64_t b_sink;       /* s >= 0 initial rows always kept */
  int64_t b_window;     /* W >= w recent rows always kept (so every candidate has a score) */
  int32_t dtype;        /* SGDKV_DTYPE_F32 or SGDKV_DTYPE_BF16 for q_win, k, v, k_out, v_out */
  float scale;          /* logit scale; 0 selects 1/sqrt(head_dim) */
} sgdkv_compress_desc;

/* Bytes of device workspace sgdkv_compress_layer needs for `desc`
 * (the same for every budget vector). */
sgdkv_status sgdkv_compress_workspace_size(const sgdkv_compress_desc* desc, size_t* bytes);

/* Compress one layer: score, pool, select per KV head and gather.
 *
 * Window scores (Sec. 3.3 last paragraph, SnapKV-style; Sec. 5 Query-Aware
 * window): window row i of query head q sits at prompt position C-w+i and
 * attends causally to keys 0..C-w+i, logits l = scale*<q_i, k_j>. For every
 * scored key j in [0, C-w) the group mean over the G query heads of the
 * KV head of the window-summed softmax probabilities is
 *   a_j = (1/G) sum_q sum_i exp(l_{q,i,j} - lse_{q,i}),
 * then pooled_j = (1/k_p) sum_{|t-j| <= (k_p-1)/2} a_t (a_t = 0 outside).
 * Selection: for KV head h with budget b_h (m_h = b_h - s - W), the kept
 * positions are [0,s), the m_h candidates in [s, C-W) with the largest
 * pooled score (ties to the lower position) and [C-W, C), in ascending order.
 *
 * layer_budgets: HOST [Hkv] int64, each in [s+W, C] (one layer's slice of
 *   sgdkv_allocate_budgets); T_layer = sum_h layer_budgets[h].
 * q_win:   device [B][Hq][w][d]  window queries (post-RoPE), dtype.
 * k, v:    device [B][Hkv][C][d] the layer's full cache, dtype.
 * window_lse: optional device [B][Hq][w] fp32 natural-log LSE of each window
 *   row over its causal keys (prefill attention produces it); NULL = the
 *   library computes it (one extra pass over K).
 * k_out, v_out: device [B*T_layer][d] dtype; segment (b,h) occupies rows
 *   offsets_out[b*Hkv+h] .. offsets_out[b*Hkv+h+1]-1 in kept order.
 * kept_pos_out: device [B*T_layer] int32 prompt positions of the kept rows.
 * offsets_out: device [B*Hkv+1] int64, offsets[b*Hkv+h] = b*T_layer +
 *   sum_{h'<h} layer_budgets[h'] (sgdkv_segment_offsets gives the same
 *   values on the host).
 * k_out, v_out, kept_pos_out and offsets_out are either all non-NULL, or
 *   all NULL (scores-only mode: only scores_out is produced).
 * scores_out: optional device [B][Hkv][C-w] fp32 pooled scores (the values
 *   the selection used); required in scores-only mode.
 * workspace: device, 256-byte aligned, >= sgdkv_compress_workspace_size.
 * Errors (nothing enqueued): sizes < 1; Hq % Hkv; Hkv > 64; d not 64/128
 *   (UNSUPPORTED); G*w > 4096 (UNSUPPORTED); k_p even; s+W > C; W < w;
 *   a budget outside [s+W, C]; C > 2^31-1; misaligned or missing pointers;
 *   small workspace (WORKSPACE); no usable device (HIP). */
sgdkv_status sgdkv_compress_layer(const sgdkv_compress_desc* desc, const int64_t* layer_budgets,
                                  const void* q_win, const void* k, const void* v,
                                  const float* window_lse, void* k_out, void* v_out,
                                  int32_t* kept_pos_out, int64_t* offsets_out, float* scores_out,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* sgdkv_compress_layer with options (opts == NULL: the defaults, which make it
 * sgdkv_compress_layer):
 *
 * group_agg: how the G query heads of a KV head are aggregated into one
 * score per key (Appendix A.7, the "Ipt." rows of Table 5). With
 * A_g[j] = sum_i exp(l_{q,i,j} - lse_{q,i}) the window attention of query
 * head q = h*G + g and sigma_q = qhead_scores[q]:
 *   SGDKV_GROUP_MEAN      a_j = (1/G) sum_g A_g[j]  (default);
 *   SGDKV_GROUP_IPT_MAX   a_j = max_g sigma_q * A_g[j]  (the paper's best);
 *   SGDKV_GROUP_IPT_MEAN  a_j = (1/G) sum_g sigma_q * A_g[j];
 *   SGDKV_GROUP_IPT_ONLY  a_j = A_{g*}[j], g* the group's head with the
 *                         largest sigma (ties: lower g).
 * qhead_scores: HOST [Hq] fp64 >= 0 finite, this layer's per-attention-head
 *   summarization scores (used by the Ipt. modes; may be NULL for MEAN).
 * window_pos: position P0 of the first window row (Sec. 5). Row i sits at
 *   P0 + i and attends to the cached keys 0..min(P0 + i, C - 1); the keys
 *   [0, P0) are scored, so scores_out is [B][Hkv][P0] and every candidate
 *   needs a score: b_window >= C - P0. -1 selects C - w (the last w prompt
 *   tokens, Query-Aware); P0 < C - w places the window before a final
 *   question of C - w - P0 tokens (Query-Unaware); P0 = C places it after
 *   the prompt (Proxy-Query rows, which see every cached key; the softmax
 *   then runs over cached keys only unless window_lse is supplied).
 * gather_stream: NULL (or equal to `stream`): all work goes on `stream`.
 *   Otherwise the last step, copying the kept K and V rows into k_out and
 *   v_out, is enqueued on gather_stream, ordered after this call's selection
 *   on `stream` by an event the library records, as a grid of half as many
 *   workgroups as the device has compute units, so that it fits beside the
 *   work the caller enqueues next on `stream` (for example the next layer's
 *   window scoring, which leaves memory bandwidth unused). k_out and v_out are then complete only when
 *   gather_stream reaches this point, and k and v must stay unchanged until
 *   then; kept_pos_out, offsets_out and scores_out are complete on `stream`
 *   as usual. The copy does not touch the workspace, which is free for the
 *   next call on `stream` at once. Not used in scores-only mode.
 * Errors: those of sgdkv_compress_layer (with b_window >= C - P0 in place of
 *   b_window >= w); group_agg not 0..3; NULL or invalid qhead_scores for an
 *   Ipt. mode; Hq > 256 with an Ipt. mode (UNSUPPORTED); IPT_MAX with
 *   obs_window not a multiple of 16 or above 512 (UNSUPPORTED); window_pos outside
 *   [-1, C]; reserved not 0. */
#define SGDKV_GROUP_MEAN 0
#define SGDKV_GROUP_IPT_MAX 1
#define SGDKV_GROUP_IPT_MEAN 2
#define SGDKV_GROUP_IPT_ONLY 3
typedef struct sgdkv_compress_opts {
  int32_t group_agg;           /* SGDKV_GROUP_* */
  int32_t reserved;            /* must be 0 */
  const double* qhead_scores;  /* host [Hq], Ipt. modes */
  int64_t window_pos;          /* P0, or -1 for C - w */
  void* gather_stream;         /* hipStream_t for the row gather, or NULL */
} sgdkv_compress_opts;
sgdkv_status sgdkv_compress_layer_ex(const sgdkv_compress_desc* desc, const sgdkv_compress_opts* opts,
                                     const int64_t* layer_budgets, const void* q_win, const void* k,
                                     const void* v, const float* window_lse, void* k_out, void* v_out,
                                     int32_t* kept_pos_out, int64_t* offsets_out, float* scores_out,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ */
/* Decode attention over the ragged compressed cache (device).         */

typedef struct sgdkv_decode_desc {
  int32_t batch;        /* B */
  int32_t num_q_heads;  /* Hq */
  int32_t num_kv_heads; /* Hkv, Hq % Hkv == 0 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t kv_dtype;     /* dtype of q, k_c, v_c */
  int32_t out_dtype;    /* dtype of out */
  float scale;          /* 0 selects 1/sqrt(head_dim) */
} sgdkv_decode_desc;

/* Bytes of device workspace sgdkv_decode_attention needs for these segment
 * lengths (offsets_host: host [B*Hkv+1] int64, non-decreasing from 0): the
 * split partials, G*(d+2) floats per decode workgroup. With up to 512
 * segments (B*Hkv) these are the segments' own workgroups, about one per
 * 4 splits of about 12288 over the batch (past 512 workgroups, rounded to a
 * multiple of 512), however unequal the segments; with more segments every
 * segment holds as many as the longest one needs. */
sgdkv_status sgdkv_decode_workspace_size(const sgdkv_decode_desc* desc, const int64_t* offsets_host,
                                         size_t* bytes);

/* One decode step: query head q of sequence b attends to the rows of its
 * KV head's segment (b, q/G) of the compressed cache -- the cache is kept
 * per KV head, before GQA repetition (Appendix A.2):
 *   out = sum_r softmax_r(scale*<q, k_r>) v_r,  lse = log sum_r exp(scale*<q,k_r>).
 * An empty segment gives out = 0 and lse = -inf.
 * q: device [B][Hq][d] kv_dtype. k_c, v_c: device [rows][d] kv_dtype with
 * rows = offsets[B*Hkv]. offsets: device [B*Hkv+1] int64; offsets_host: the
 * same values on the host, used to plan the split without a device sync.
 * out: device [B][Hq][d] out_dtype. lse_out: optional device [B][Hq] fp32.
 * Errors: sizes < 1; Hq % Hkv; d not 64/128 (UNSUPPORTED); decreasing or
 * negative offsets; misaligned or missing pointers; small workspace. */
sgdkv_status sgdkv_decode_attention(const sgdkv_decode_desc* desc, const void* q, const void* k_c,
                                    const void* v_c, const int64_t* offsets,
                                    const int64_t* offsets_host, void* out, float* lse_out,
                                    void* workspace, size_t workspace_bytes, void* stream);

/* Generation after compression: every KV head (b, h) keeps, beside its
 * compressed segment, the rows appended since (one per generated token; the
 * cache stays one per KV head, Appendix A.2). They live in a caller-owned
 * region of `capacity` rows per (b, h); rows 0..n_new-1 are valid. */
typedef struct sgdkv_decode_tail {
  const void* k_new;  /* device [B][Hkv][capacity][d] kv_dtype */
  const void* v_new;  /* device [B][Hkv][capacity][d] kv_dtype */
  int64_t capacity;   /* rows per (b, h), >= 0 */
  int64_t n_new;      /* valid rows per (b, h), 0 <= n_new <= capacity */
} sgdkv_decode_tail;

/* Writes one generated token's K and V rows into row `slot` of every (b, h)
 * of the appended region. k_step, v_step: device [B][Hkv][d] kv_dtype;
 * k_new, v_new: device [B][Hkv][capacity][d] kv_dtype (caller-owned).
 * Errors (nothing enqueued): sizes as for sgdkv_decode_attention; slot
 * outside [0, capacity); a region of 4 GiB or more (UNSUPPORTED); missing
 * or misaligned pointers. */
sgdkv_status sgdkv_append_kv(const sgdkv_decode_desc* desc, const void* k_step, const void* v_step, void* k_new,
                             void* v_new, int64_t capacity, int64_t slot, void* stream);

/* Workspace for sgdkv_decode_attention_ex with appended regions of up to
 * `capacity` rows (capacity 0: the same as sgdkv_decode_workspace_size). */
sgdkv_status sgdkv_decode_workspace_size_ex(const sgdkv_decode_desc* desc, const int64_t* offsets_host,
                                            int64_t capacity, size_t* bytes);

/* sgdkv_decode_attention over each segment's compressed rows followed by
 * rows 0..tail->n_new-1 of its appended region (tail == NULL or n_new == 0:
 * the compressed rows alone):
 *   out = sum over both sets of softmax(scale*<q,k>) v, lse likewise.
 * Errors: those of sgdkv_decode_attention; capacity < 0; n_new outside
 *   [0, capacity]; NULL or misaligned k_new/v_new with n_new > 0; a region
 *   of 4 GiB or more (UNSUPPORTED); a workspace planned for a smaller
 *   capacity (WORKSPACE). */
sgdkv_status sgdkv_decode_attention_ex(const sgdkv_decode_desc* desc, const void* q, const void* k_c,
                                       const void* v_c, const int64_t* offsets, const int64_t* offsets_host,
                                       const sgdkv_decode_tail* tail, void* out, float* lse_out, void* workspace,
                                       size_t workspace_bytes, void* stream);

/* sgdkv_decode_attention_ex without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation). The split partials go to a static
 * device array of the library, 64 MiB per GPU, which every GPU the library
 * runs on holds from its first use until the process ends; the call allocates
 * nothing itself. The caller still passes q, the cache, the offsets, out and
 * lse_out as for sgdkv_decode_attention_ex, with the same results.
 * Calls on one GPU share that GPU's array: calls that overlap in time on one
 * GPU (on different streams, or from several threads) race and give
 * undefined results; calls ordered on one stream are safe. Nothing in the
 * array needs to persist or be cleared between calls.
 * Errors: those of sgdkv_decode_attention_ex except WORKSPACE; a decode whose
 * partials (sgdkv_decode_workspace_size_ex for the same arguments) exceed
 * 64 MiB (UNSUPPORTED, nothing enqueued). */
sgdkv_status sgdkv_decode_attention_noalloc(const sgdkv_decode_desc* desc, const void* q, const void* k_c,
                                            const void* v_c, const int64_t* offsets, const int64_t* offsets_host,
                                            const sgdkv_decode_tail* tail, void* out, float* lse_out,
                                            void* stream);

/* ------------------------------------------------------------------ */
/* Kernel timing for benchmarks (not part of the method).             */

/* While enabled (on != 0), every kernel the library launches is bracketed by
 * a pair of HIP events recorded on the launch stream. Costs two event
 * records per kernel; off by default. Thread-safe. */
sgdkv_status sgdkv_profile_enable(int32_t on);

/* Drops every recorded duration (waiting for pending events first). */
sgdkv_status sgdkv_profile_reset(void);

/* Waits for the recorded events and reports, per kernel name, the number of
 * launches and their total duration in milliseconds since the last reset.
 * names: host buffer of max_entries * 64 chars (NUL-terminated names);
 * counts, total_ms: host [max_entries]. *n_out receives the number of
 * kernels seen (entries beyond max_entries are not written).
 * Errors: negative max_entries; NULL buffers with max_entries > 0. */
sgdkv_status sgdkv_profile_read(int32_t max_entries, char* names, int64_t* counts, double* total_ms,
                                int32_t* n_out);

#ifdef __cplusplus
}
#endif

#endif /* SGDKV_H */
