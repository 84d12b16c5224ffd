/*
 * libcas: multi-cartridge prefix attention for AMD Instinct MI355X (gfx950).
 *
 * One attention layer of a frozen LLM in which each query token attends over
 * a concatenation of trainable KV prefixes ("cartridges") followed by the
 * row's own tokens under causal masking, with the backward pass that returns
 * dQ and the dK/dV of every cartridge and of the self tokens.
 *
 * The operation (paper: Section "Cartridges at Scale (CAS) Training",
 * Background paragraph, for the cartridge as a trainable KV prefix whose keys
 * and values alone receive gradients; Section "Inference" for the
 * concatenation of several cartridges in order ahead of the prompt; the
 * Limitations paragraph "Cartridge KV position" for ordinary causal masking of
 * the tokens that follow; the Budget Manager and Pool rotation paragraphs for
 * cartridges that move between host memory and the GPU):
 *
 *   For batch row b, query head h, query position t and kv = h / group_size,
 *   the visible keys are, in order, every token of every segment of row b,
 *   then self tokens 0..t. With s_j = softmax_scale * q . k_j:
 *     LSE = ln sum_j exp(s_j),  P_j = exp(s_j - LSE),  O = sum_j P_j v_j.
 *   Backward, given dO:  D = dO . O,  dS_j = P_j (dO . v_j - D),
 *     dQ = scale * sum_j dS_j k_j,  dK_j += scale * dS_j q,  dV_j += P_j dO,
 *   summed over every query (all heads of the group) that sees key j.
 *
 * Keys and queries are taken as given (post-RoPE); no positional operation is
 * applied. All calls are asynchronous on the caller's HIP stream; results are
 * valid once the stream reaches them.
 *
 * Thread safety: calls may be made from several host threads; the error
 * message is thread-local.
 */
#ifndef CAS_H_
#define CAS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CAS_ABI_VERSION 4

/* Bytes of the device scratch each GPU holds for cas_prefix_attn_fwd_noalloc. */
#define CAS_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

typedef enum {
  CAS_OK = 0,
  CAS_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, shape, segment table or aliasing */
  CAS_ERR_UNSUPPORTED = 2,      /* valid but not implemented (head_dim, dtype, table size) */
  CAS_ERR_ALIGNMENT = 3,        /* pointer or stride not a multiple of 16 bytes */
  CAS_ERR_NOT_PINNED = 4,       /* staging source is pageable host memory */
  CAS_ERR_WORKSPACE = 5,        /* workspace NULL or smaller than the size query returned */
  CAS_ERR_HIP = 6,              /* a HIP runtime call failed; see cas_last_error_message */
  CAS_ERR_IO = 7                /* a file operation of the pool's moment tier failed */
} cas_status_t;

typedef enum {
  CAS_DTYPE_BF16 = 0, /* bfloat16 tensors; MFMA in bf16 with fp32 accumulation */
  CAS_DTYPE_FP32 = 1  /* float32 tensors; MFMA in fp32 (no down-conversion anywhere) */
} cas_dtype_t;

/*
 * One cartridge block as seen by one batch row (one entry of the segment table).
 *
 * k, v:   device pointers. Element (token j, kv head h, channel c) lives at
 *         base + j*stride_tok + h*stride_head + c (in elements of the dtype).
 *         The channel stride is 1. Token-major [len, Hkv, d] and head-major
 *         [Hkv, len, d] storage, and padded token strides, are all expressible.
 * dk, dv: device pointers with the same strides, receiving the gradient
 *         (backward only; ignored by the forward). NULL means "do not return
 *         this gradient".
 * len:    tokens, >= 0. A zero-length entry is skipped and its pointers are
 *         not read.
 *
 * Entries with equal (k, v, len, stride_tok, stride_head) are the same
 * cartridge, referenced several times (by several rows, or twice in one row);
 * they must carry equal dk and dv, which then receive the SUM over all
 * references. Any other overlap between a gradient buffer and any tensor the
 * call reads or writes is rejected with CAS_ERR_INVALID_ARGUMENT.
 */
typedef struct {
  const void *k;
  const void *v;
  void *dk;
  void *dv;
  int64_t len;
  int64_t stride_tok;
  int64_t stride_head;
} cas_segment_t;

/*
 * Problem description, read only during the call (the host arrays may be
 * reused as soon as the call returns).
 *
 * Two query layouts. With q_offsets == NULL every batch row has q_len >= 1
 * query tokens (fixed-length batch). Otherwise the batch rows are packed
 * samples of different lengths (the training layout in which several
 * conversations, each with its own cartridges, share one token axis;
 * paper: Section "Training with Multiple Cartridges" and Eq. mixing):
 * q_offsets is a host array of batch+1 non-decreasing int32 with
 * q_offsets[0] == 0, row b owns tokens q_offsets[b] .. q_offsets[b+1]-1 of a
 * token axis of T = q_offsets[batch] >= 1 tokens, q_len must be 0, and each
 * row's self keys are its own tokens only (block-diagonal causal masking).
 * Rows may be empty. In both layouts let T be the token count (batch*q_len
 * when fixed) and Hq = num_kv_heads*group_size.
 *
 * Shapes (contiguous, in elements of dtype):
 *   q, o, d_o, dq:                    [T, Hq, head_dim]
 *   k_self, v_self, dk_self, dv_self: [T, num_kv_heads, head_dim]
 *   lse (always float32, natural log): [batch, Hq, q_len] (fixed) or [Hq, T] (packed)
 * (a fixed-length batch is [batch, q_len, ...] in these terms).
 * Query head h reads kv head h / group_size (contiguous GQA groups).
 * head_dim is 64 or 128. softmax_scale must be finite and > 0. T * Hq must
 * stay below 2^31.
 * seg_offsets is a host array of batch+1 non-decreasing int32 with
 * seg_offsets[0] == 0; row b uses segments[seg_offsets[b] .. seg_offsets[b+1]).
 * segments may be NULL when seg_offsets[batch] == 0.
 */
typedef struct {
  cas_dtype_t dtype;
  int32_t batch;
  int32_t q_len;
  int32_t num_kv_heads;
  int32_t group_size;
  int32_t head_dim;
  float softmax_scale;
  const cas_segment_t *segments;
  const int32_t *seg_offsets;
  const int32_t *q_offsets; /* NULL (fixed q_len per row) or batch+1 token offsets (packed) */
} cas_problem_t;

/*
 * Bytes of device workspace a forward (backward == 0) or backward
 * (backward != 0) call on this problem needs, written to *bytes. The size
 * depends on the problem, the current tuning (cas_set_tuning) and, through
 * the automatic key-axis splits, the compute-unit count of the current
 * device (the same on every whole MI355X): query it with the device current
 * that will run the call. Workspace is caller-owned, 256-byte aligned, and
 * may be reused by the next call once the stream has passed the previous
 * one. Besides the
 * segment tables and per-row statistics, a bf16 backward keeps a transposed
 * copy of q and d_o in it (about twice the bytes of q).
 */
cas_status_t cas_prefix_attn_workspace_size(const cas_problem_t *p, int backward, size_t *bytes);

/*
 * Forward (paper: Section "Inference", several cartridges concatenated in
 * order ahead of the prompt; Limitations, "Cartridge KV position", ordinary
 * causal masking of the tokens that follow): softmax attention of every
 * query over its row's segments in table order, then its own tokens 0..t.
 * Writes o (dtype) and, when lse != NULL, the row log-sum-exp lse
 * (float32, natural log). All tensors are device memory, 16-byte aligned
 * (lse 4-byte aligned). hip_stream is a hipStream_t (NULL = default stream).
 * Validation happens before anything is enqueued; on error nothing is
 * launched and the outputs are untouched.
 */
cas_status_t cas_prefix_attn_fwd(const cas_problem_t *p, const void *q, const void *k_self,
                                 const void *v_self, void *o, float *lse, void *workspace,
                                 size_t ws_bytes, void *hip_stream);

/*
 * Backward (paper: Section "Cartridges at Scale (CAS) Training", Background
 * paragraph: the model is frozen and only the cartridges' keys and values
 * are trained, so the gradient flows through the attention into every
 * referenced cartridge; a cartridge used several times gets the sum).
 * Backward of sum(d_o * o): consumes q, the self and segment K/V, and the o
 * and lse written by cas_prefix_attn_fwd on the same inputs, and OVERWRITES
 * dq, dk_self, dv_self and every non-NULL segments[i].dk / .dv (NULL outputs
 * are skipped). Gradients are returned in the input dtype; accumulation is in
 * fp32. Same pointer, alignment, stream and error rules as the forward.
 */
cas_status_t cas_prefix_attn_bwd(const cas_problem_t *p, const void *q, const void *k_self,
                                 const void *v_self, const void *o, const float *lse,
                                 const void *d_o, void *dq, void *dk_self, void *dv_self,
                                 void *workspace, size_t ws_bytes, void *hip_stream);

/*
 * The forward without any allocation, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc). Same problem, tensors, results and error rules as
 * cas_prefix_attn_fwd, without the workspace arguments: the workspace is a
 * static device array of CAS_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends, and the launch tables reach it
 * as kernel arguments (no pinned staging buffer). The call allocates nothing:
 * no hipMalloc, hipHostMalloc, hipFree or event creation (the first call on a
 * device only looks up that device's scratch address).
 *
 * When the forward would split the key axis into more partials than the
 * scratch holds, fewer splits are used (the result changes only in rounding
 * order). A problem whose launch tables alone exceed the scratch returns
 * CAS_ERR_UNSUPPORTED before anything is enqueued.
 *
 * All calls on one GPU share its scratch: calls that may overlap on that GPU
 * (different streams without ordering, or several host threads) race and
 * give wrong results; calls ordered on one stream are safe. Nothing in the
 * scratch needs clearing between calls.
 */
cas_status_t cas_prefix_attn_fwd_noalloc(const cas_problem_t *p, const void *q, const void *k_self,
                                         const void *v_self, void *o, float *lse, void *hip_stream);

/*
 * Cartridge staging (paper: Budget Manager and Pool rotation paragraphs,
 * cartridges offloaded to host memory and moved back onto the GPU).
 * Enqueues n host->device copies on side_stream (a hipStream_t) and, when
 * done_event (a hipEvent_t) is non-NULL, records it after the last copy so a
 * compute stream can hipStreamWaitEvent on it. Every host_src must lie in
 * pinned (page-locked) host memory, else CAS_ERR_NOT_PINNED and nothing is
 * enqueued: a pageable copy would silently serialise with the host. The
 * caller keeps host_src alive and unmodified until the event completes.
 * Consecutive entries whose source and destination both continue the
 * previous entry's are moved as one transfer (list a pool's cartridges in
 * address order to get large transfers); copies run in the given order.
 */
typedef struct {
  const void *host_src;
  void *dev_dst;
  size_t bytes;
} cas_stage_copy_t;

cas_status_t cas_cartridge_stage(const cas_stage_copy_t *copies, int32_t n, void *side_stream,
                                 void *done_event);

/*
 * Optimizer step of the trainable cartridges (paper: Section "Optimization
 * Dynamics", paragraphs "Optimizer" and "Per-cartridge LR warmup"; the
 * hyperparameter table's Adam (FP32), per-cartridge warmup W_c = 20 and one
 * frozen token). Adam (Kingma and Ba, Algorithm 1) with fp32 moments on bf16
 * parameters, one fused launch over every listed cartridge's K and V.
 *
 * For each element x of k and v (and its gradient g from dk / dv), with
 * t = step + 1 and lr_c = lr * cas_adam_lr_scale(step, warmup_steps,
 * warmup_buckets):
 *   m1 = beta1 m1 + (1 - beta1) g;   m2 = beta2 m2 + (1 - beta2) g g
 *   x  = bf16_rne(x - lr_c (m1 / (1 - beta1^t)) / (sqrt(m2 / (1 - beta2^t)) + eps))
 * all in fp32 with one rounding per operation, in this order (1 - beta^t is
 * evaluated in double and rounded to fp32). The first frozen_tokens tokens
 * of each cartridge (the BOS token) are neither read nor written.
 *
 * k, v, dk, dv: bf16 device tensors with the strides of cas_segment_t
 *   (element (j, h, c) at base + j*stride_tok + h*stride_head + c).
 * m1_k, m2_k, m1_v, m2_v: fp32 device moments, contiguous
 *   [len, num_kv_heads, head_dim], zero before a cartridge's first step.
 * step: optimizer steps the cartridge has already received (the caller
 *   increments it after the call; moving a cartridge out of the GPU pool and
 *   back keeps its step count and moments).
 * Every pointer 16-byte aligned, strides multiples of 8 elements; parameters
 * may not overlap their gradients or moments, or another cartridge's
 * tensors. Validation happens before anything is enqueued; on error nothing
 * runs. The workspace holds the launch tables (size from
 * cas_cartridge_adam_workspace_size; reusable once the stream has passed).
 */
typedef struct {
  void *k;
  void *v;
  const void *dk;
  const void *dv;
  float *m1_k;
  float *m2_k;
  float *m1_v;
  float *m2_v;
  int64_t len;
  int64_t stride_tok;
  int64_t stride_head;
  int32_t step;
  int32_t frozen_tokens;
} cas_adam_cartridge_t;

typedef struct {
  float lr;               /* eta_t of the global schedule at this step, >= 0 */
  float beta1, beta2;     /* in [0, 1) */
  float eps;              /* > 0 */
  int32_t warmup_steps;   /* W_c; 0 disables the per-cartridge warmup */
  int32_t warmup_buckets; /* N_b >= 1 */
} cas_adam_config_t;

/*
 * Per-cartridge warmup factor (host only): min(1, step / warmup_steps)
 * rounded up to one of warmup_buckets levels 1/N_b, 2/N_b, ..., 1 (the first
 * level also for step 0), so at most N_b distinct learning rates occur in a
 * step. 1 when warmup_steps <= 0; NaN for warmup_buckets < 1 or step < 0.
 */
float cas_adam_lr_scale(int32_t step, int32_t warmup_steps, int32_t warmup_buckets);

cas_status_t cas_cartridge_adam_workspace_size(const cas_adam_cartridge_t *carts, int32_t n,
                                               int32_t num_kv_heads, int32_t head_dim,
                                               size_t *bytes);

cas_status_t cas_cartridge_adam(const cas_adam_cartridge_t *carts, int32_t n, int32_t num_kv_heads,
                                int32_t head_dim, const cas_adam_config_t *cfg, void *workspace,
                                size_t ws_bytes, void *hip_stream);

/*
 * Short-query / decode attention over paged cartridges (paper: Section
 * "Inference" and paragraph "Cartridge RAG": the top-k retrieved cartridges'
 * KV caches are concatenated ahead of the prompt; appendix on cartridge
 * sizes: cartridges are whole 16-token pages of the serving engine's paged
 * KV cache). Forward only.
 *
 * K and V live in a page pool: k_pages, v_pages are bf16 device tensors
 * [num_pages, page_size, num_kv_heads, head_dim], contiguous. Request b owns
 * kv_lens[b] keys, stored in the pages page_ids[page_offsets[b] ..
 * page_offsets[b+1]) in key order (ceil(kv_lens[b] / page_size) pages; the
 * last may be partly filled): typically the pages of its selected cartridges
 * (shared with other requests, never copied) followed by the pages of its
 * own prompt and generated tokens. Its n_b = q_offsets[b+1] - q_offsets[b]
 * queries (1 <= n_b <= kv_lens[b]; n_b = 1 for a decode step) are the last
 * n_b positions of that key sequence: query i sees keys 0 .. kv_lens[b] -
 * n_b + i (causal among the new tokens). q and o are [Tq, Hq, head_dim]
 * (Tq = q_offsets[batch]), lse is [Hq, Tq] fp32 (may be NULL); query head h
 * reads kv head h / group_size. page_size is 16, 32, 64 or 128; head_dim 64
 * or 128; page ids lie in [0, num_pages). The key axis of each request is
 * split over several workgroups when the requests alone would not fill the
 * GPU (partials merged by their LSE). Validation before anything is
 * enqueued; on error nothing runs and the outputs are untouched.
 */
typedef struct {
  int32_t batch;
  int32_t num_kv_heads;
  int32_t group_size;
  int32_t head_dim;
  float softmax_scale;
  int32_t page_size;
  int64_t num_pages;
  const int32_t *q_offsets;    /* host, batch+1 */
  const int32_t *kv_lens;      /* host, batch */
  const int32_t *page_offsets; /* host, batch+1 */
  const int32_t *page_ids;     /* host, page_offsets[batch] entries */
} cas_decode_problem_t;

/* Workspace bytes of a cas_paged_decode_fwd call (launch tables and the
 * split partials), written to *bytes; like the prefix-attention query it
 * depends on the compute-unit count of the current device. */
cas_status_t cas_paged_decode_workspace_size(const cas_decode_problem_t *p, size_t *bytes);

cas_status_t cas_paged_decode_fwd(const cas_decode_problem_t *p, const void *q, const void *k_pages,
                                  const void *v_pages, void *o, float *lse, void *workspace,
                                  size_t ws_bytes, void *hip_stream);

/*
 * Budget manager (paper: paragraphs "Budget Manager" and "Pool rotation";
 * hyperparameter table: budget B = 20, rotation interval R = 10, swap
 * fraction phi = 0.5, least-trained cartridges first, Adam moments of
 * CPU-resident cartridges offloaded to NVMe). The pool owns a pinned host
 * copy of every cartridge's bf16 K/V and step count, and B active device
 * slots, plus floor(phi * B) staging slots into which the next rotation's
 * cartridges are copied ahead of time on the pool's own stream while the
 * current ones train.
 *
 * The fp32 Adam moments of the cartridges that are not on the GPU live in
 * one of two tiers: pinned host memory next to their K/V (moment_dir NULL),
 * or a file on a local (NVMe) file system (moment_dir names its directory:
 * the pool creates an unnamed file there, removed when the pool is
 * destroyed or the process ends, and keeps in pinned memory only two sets
 * of floor(phi * B) (at least one) moment buffers for the cartridges in
 * transit). The file tier's reads and writes run on a pool thread: an
 * eviction's moments are written after their copy back has landed, and the
 * next admissions' moments are read and copied to the GPU ahead of the
 * rotation that admits them, overlapped with the training steps between
 * rotations.
 *
 * Rotation, after every R-th cas_pool_end_step: the n = min(floor(phi * B),
 * N - B) active cartridges with the most optimizer steps (ties: lower id)
 * are copied back to host (parameters and moments, after the compute
 * stream's work so far) and leave the active set; the prefetched cartridges,
 * the n offloaded ones with the fewest steps (ties: lower id), take their
 * place; then the next admissions are prefetched into the freed slots.
 * Offloaded cartridges receive no gradient. cas_pool_plan_rotation is that
 * policy on its own (host only).
 *
 * Use: create; fill the host copies (cas_pool_host_cartridge: pinned views,
 * moments zero, step 0); cas_pool_load; then per training step read the
 * active set (cas_pool_active: device views of K/V, their gradient buffers
 * dk/dv, moments and step counts, ready for cas_cartridge_adam) and call
 * cas_pool_end_step after the optimizer step. cas_pool_flush copies every
 * active cartridge back and waits, after which all host copies (and the
 * moment file) are current. Calls on one pool must not overlap; streams are
 * the caller's except the pool's own copy stream (default priority). A
 * failed file read or write of the moment tier is reported as CAS_ERR_IO by
 * the next call on the pool; the pool is then unusable except for destroy.
 */
typedef struct cas_pool cas_pool_t;

typedef struct {
  int32_t num_cartridges;   /* N >= 1 */
  const int64_t *lens;      /* host, N token counts (>= 1) */
  int32_t num_kv_heads;
  int32_t head_dim;         /* 64 or 128 */
  int32_t budget;           /* B, 1 <= B <= N */
  int32_t rotate_every;     /* R >= 1 */
  float swap_fraction;      /* phi in [0, 1] */
  int32_t frozen_tokens;    /* reported in the views (BOS: 1) */
  const char *moment_dir;   /* NULL: moments in pinned host memory; else the file tier's directory */
} cas_pool_config_t;

cas_status_t cas_pool_plan_rotation(const int32_t *steps, const uint8_t *active, int32_t n, int32_t budget,
                                    float swap_fraction, int32_t *evict, int32_t *admit, int32_t *n_swap);
cas_status_t cas_pool_create(const cas_pool_config_t *cfg, cas_pool_t **pool);
cas_status_t cas_pool_destroy(cas_pool_t *pool);
/* Pinned host views of cartridge cart: k, v, step and frozen tokens, and
 * with the host moment tier its moments (NULL with the file tier: use
 * cas_pool_read_moments). */
cas_status_t cas_pool_host_cartridge(cas_pool_t *pool, int32_t cart, cas_adam_cartridge_t *host_view);
cas_status_t cas_pool_load(cas_pool_t *pool, void *compute_stream);
cas_status_t cas_pool_active(cas_pool_t *pool, int32_t *cart_ids, cas_adam_cartridge_t *views, int32_t cap,
                             int32_t *n);
cas_status_t cas_pool_end_step(cas_pool_t *pool, void *compute_stream);
cas_status_t cas_pool_flush(cas_pool_t *pool, void *compute_stream);
/*
 * Copies cartridge cart's fp32 moments, m1_k, m2_k, m1_v, m2_v (each
 * [len, num_kv_heads, head_dim], contiguous), into the host buffer dst
 * (4 * len * num_kv_heads * head_dim floats), from whichever tier holds
 * them. Current for every cartridge before cas_pool_load and after
 * cas_pool_flush; during training an active cartridge's copy is the one of
 * its last admission. Waits for the pool's pending file I/O.
 */
cas_status_t cas_pool_read_moments(cas_pool_t *pool, int32_t cart, float *dst);

/* Static description of a status code. */
const char *cas_status_string(cas_status_t s);
/* Message of the last failed call on this thread ("" if none). */
const char *cas_last_error_message(void);
/* CAS_ABI_VERSION of the built library. */
int32_t cas_abi_version(void);

/*
 * Tuning knobs (process-wide; 0 = automatic). They change the launch plan,
 * never the result beyond rounding order.
 *   fwd_splits:  key-axis splits of the forward (partial O/LSE merged after)
 *   dq_splits:   key-axis splits of the dQ pass (fp32 partials summed after)
 */
typedef struct {
  int32_t fwd_splits;
  int32_t dq_splits;
} cas_tuning_t;

cas_status_t cas_set_tuning(const cas_tuning_t *t);
cas_status_t cas_get_tuning(cas_tuning_t *t);

/*
 * Launch plan of a problem (host-side; no device access). For tests and
 * profiling tools.
 */
typedef struct {
  int32_t fwd_splits;       /* key-axis splits used by the forward */
  int32_t dq_splits;        /* key-axis splits used by the dQ pass */
  int32_t fwd_workgroups;   /* forward grid size */
  int32_t dkdv_workgroups;  /* dK/dV grid size */
  int32_t unique_segments;  /* distinct cartridges after alias folding */
  int32_t total_key_tiles;  /* dK/dV key tiles over unique cartridges and self */
  int64_t max_prefix_len;   /* longest row prefix, tokens */
  size_t ws_fwd_bytes;
  size_t ws_bwd_bytes;
} cas_plan_info_t;

cas_status_t cas_plan_info(const cas_problem_t *p, cas_plan_info_t *out);

/*
 * Per-kernel timing with HIP events, recorded on the stream each kernel is
 * launched on (a profiling aid; off by default). While enabled, every kernel
 * a call launches is bracketed by two events. cas_timing_read waits for the
 * recorded events and returns, per kernel name, the number of launches and
 * their summed duration since the last reset.
 */
typedef struct {
  char name[48];
  int32_t launches;
  double total_ms;
} cas_kernel_time_t;

cas_status_t cas_timing_enable(int enable);
cas_status_t cas_timing_reset(void);
cas_status_t cas_timing_read(cas_kernel_time_t *out, int32_t cap, int32_t *n_out);

#ifdef __cplusplus
}
#endif

#endif /* CAS_H_ */
