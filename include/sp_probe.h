/*
 * sp_probe.h — C ABI of the MI355X (gfx950) Speculative Probing classification forward.
 *
 * The operation (Sec. 3.2 "Speculative Probing", Sec. 3.3 Eq. 1-3 of the paper):
 * for every sequence b of a batch, whose speculative head (MTP / Eagle3, one
 * decoder layer) already holds the keys and values of the N_b committed tokens
 * in device memory, append k learned soft-prompt vectors at positions
 * N_b .. N_b+k-1 and run the frozen layer over those k rows only:
 *     RMSNorm -> Q/K/V projection -> RoPE -> attention of the k soft queries
 *     over [cached K/V ; the k new K/V] (causal among the new rows) ->
 *     o-projection + residual -> RMSNorm -> SwiGLU MLP + residual ->
 *     final RMSNorm -> read-out row(s) -> linear classifier -> logits[b, 0..C-1].
 * The new rows' keys and values live in a library-owned scratch area and are
 * never written into the caller's cache (Sec. 3.3, last paragraph).
 * sp_probe_forward_recursive runs the recursive form (SP-k with the MTP input
 * fusion, Sec. 3.1-3.2): k single-row steps, each fed the previous step's output.
 *
 * Conventions
 *  - Every pointer named "device" is a device address on the current HIP
 *    device; every other pointer is host memory read during the call only.
 *  - Matrices are row-major [out, in] (a row per output feature).
 *  - All calls return sp_status and never abort or throw.  Checks that can be
 *    made on the host run before anything is enqueued: on error no work is
 *    queued and the outputs are untouched.
 *  - sp_probe_forward (and _multi, _recursive) enqueues work on `stream` (a
 *    hipStream_t; NULL = the null stream) and returns without waiting; it
 *    allocates nothing, records no memset and never synchronises the host
 *    unless a debug/profiling call below says so, so a call can be captured
 *    into a HIP graph and replayed (without SP_FLAG_PROFILE / SP_FLAG_DEBUG).
 *  - One handle carries one workspace: forwards on the same handle must be
 *    ordered (same stream, or caller-synchronised).  Distinct handles are
 *    independent.
 */
#ifndef SP_PROBE_H
#define SP_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sp_status {
  SP_OK = 0,
  SP_ERR_INVALID_ARG = -1,   /* null pointer, bad size, stride or alignment */
  SP_ERR_UNSUPPORTED = -2,   /* valid but not implemented (e.g. head_dim 96) */
  SP_ERR_NO_DEVICE = -3,     /* no HIP device, or the current device is not gfx950 */
  SP_ERR_OUT_OF_MEMORY = -4, /* workspace allocation failed at init */
  SP_ERR_HIP = -5,           /* a HIP runtime call or kernel launch failed */
  SP_ERR_CAPACITY = -6,      /* batch larger than max_batch of the handle */
  SP_ERR_DEVICE_DATA = -7,   /* reported by sp_probe_check_device_error: a seq_len outside
                                [0, max_seq_len] (any mode), or (debug mode) an invalid block
                                id, class row or weight-image header */
  SP_ERR_RANGE = -8,         /* reported by sp_probe_check_device_error: an fp16 activation
                                (normed row, attention output, SwiGLU product) exceeded 65504 */
  SP_ERR_INTERNAL = -9       /* a library fault: reported by sp_probe_check_device_error when a
                                guard word between workspace areas was overwritten, or returned
                                by a forward whose plan does not fit the handle's workspace */
} sp_status;

typedef enum sp_dtype {
  SP_F32 = 0,   /* fp32 weights, soft prompt and KV cache; fp32 arithmetic throughout */
  SP_BF16 = 1   /* bf16 storage of weights, soft prompt and KV cache.  Projections: fp16
                   MFMA operands (bf16 weights converted exactly, activations rounded to
                   fp16), fp32 accumulation.  Attention: bf16 MFMA on the stored K and V
                   with the queries and probabilities split in bf16 hi + lo parts; each
                   split's output is kept as fp16 O/l until the merge.  fp32 norms,
                   softmax statistics, residual stream and logits.  Range: weight
                   and KV magnitudes must stay below 65504, and so must the fp16
                   activations (normed rows, attention outputs, SwiGLU products: |x| <= 65504);
                   an activation past that is stored as inf and reported by
                   sp_probe_check_device_error as SP_ERR_RANGE */
} sp_dtype;

typedef enum sp_pool {
  SP_POOL_LAST = 0,  /* classify the final-normed hidden state of the last soft row
                        (the read-out of the k-th step, Sec. 3.2) */
  SP_POOL_MEAN = 1   /* mean of the final-normed hidden states of the k soft rows
                        (the pooled read-out the Fig. 2 caption names) */
} sp_pool;

enum {
  SP_FLAG_DEBUG = 1,    /* validate device-resident seq_lens and block ids on every forward;
                           kernels then skip work after a failed check */
  SP_FLAG_PROFILE = 2,  /* record HIP events around every stage of each forward */
  SP_FLAG_LAST_ROW_ONLY = 4  /* one-pass forwards under SP_POOL_LAST compute only what the
                                read-out uses: every soft row's key and value, but the queries,
                                attention output, o-projection, MLP and final norm of the last
                                soft row of each task alone (the other rows reach the logits only
                                through their keys and values).  Same logits up to rounding order;
                                requires SP_POOL_LAST */
};

/* Shape of the frozen head and limits of a handle. */
typedef struct sp_probe_config {
  int32_t hidden;        /* d <= 16384: multiple of 32 (bf16) or of 4 (f32) */
  int32_t n_q_heads;     /* query heads */
  int32_t n_kv_heads;    /* KV heads; n_q_heads % n_kv_heads == 0 (grouped-query attention,
                            query head h reads KV head h / (n_q_heads / n_kv_heads)) */
  int32_t head_dim;      /* 64 or 128 */
  int32_t intermediate;  /* SwiGLU width: multiple of 32 (bf16) or of 4 (f32) */
  int32_t k;             /* soft-prompt rows per sequence, 1..64 */
  int32_t n_classes;     /* C, 1..64 */
  int32_t dtype;         /* sp_dtype */
  int32_t pool;          /* sp_pool */
  float rms_eps;         /* epsilon inside every RMSNorm square root */
  double rope_base;      /* RoPE base; pair (i, i + head_dim/2) turns by pos * base^(-2i/head_dim) */
  int32_t max_batch;     /* largest batch a forward may pass */
  int32_t max_seq_len;   /* largest context length N_b a forward may pass.  A seq_len outside
                            [0, max_seq_len] is clamped to that range (the sequence is then
                            classified on its first max_seq_len tokens) and reported by
                            sp_probe_check_device_error as SP_ERR_DEVICE_DATA, in any mode;
                            debug mode also skips the forward's later kernels */
  int32_t split_len;     /* tokens per attention split, a power of two >= 256; 0 = automatic */
  int32_t flags;         /* SP_FLAG_* */
  int32_t max_tasks;     /* largest task count of sp_probe_forward_multi, 1..64 (0 = 1);
                            max_tasks * k <= 1024 */
} sp_probe_config;

/* The head's resident KV cache (Sec. 3.3 Eq. 2-3: K_{1:n}, V_{1:n}), read-only.
 *
 * Storage is paged: sequence b's token t lives in logical block t / block_size
 * of that sequence, at slot t % block_size.  The physical block is
 * block_table[b * max_blocks_per_seq + t / block_size], or, when block_table is
 * NULL ("contiguous"), b * max_blocks_per_seq + t / block_size.
 * Inside physical block p, KV head g, with x = 16 / sizeof(element) (8 for bf16,
 * 4 for f32) and the cached keys post-RoPE:
 *   K(t, i) = k_base[p*k_stride_block + g*k_stride_head + ((i / x) * block_size + t) * x + i % x]
 *   V(t, i) = v_base[p*v_stride_block + g*v_stride_head + i * block_size + t]
 * (t = slot in block, i = 0..head_dim-1).  Strides are in elements.  Only
 * slots t < N_b of a sequence are read as data; other slots may hold anything,
 * including NaN.  Pointers and strides must be 16-byte aligned. */
typedef struct sp_kv_cache {
  const void* k_base;          /* device */
  const void* v_base;          /* device */
  int64_t num_blocks;          /* physical blocks in the pool (debug-mode bound for block ids) */
  int64_t k_stride_block, k_stride_head;
  int64_t v_stride_block, v_stride_head;
  int32_t block_size;          /* tokens per block: a power of two >= 16 */
  int32_t max_blocks_per_seq;  /* row length of block_table; >= ceil(N_b / block_size) */
  int32_t batch;               /* B, number of sequences; 0 is a no-op */
} sp_kv_cache;

/* Frozen head weights and the task's classifier, all device pointers in the
 * config's dtype except b_cls (fp32), 16-byte aligned, [out, in] row-major:
 *   in_norm[d], w_q[n_q*hd][d], w_k[n_kv*hd][d], w_v[n_kv*hd][d], w_o[d][n_q*hd],
 *   post_norm[d], w_gate[I][d], w_up[I][d], w_down[d][I], final_norm[d],
 *   w_cls[C][d], b_cls[C] (nullable: no bias).
 * Read-out through a vocabulary matrix (the frozen LM-head ablation, Sec. 6.7,
 * Table 7): with cls_rows set (device int32, one row index per class, [T][C]
 * for a multi-task call), class c reads row cls_rows[c] of w_cls, which is then
 * a [cls_vocab][d] matrix such as the head's LM head; with C = 2 and the rows of
 * the "yes" and "no" tokens, logits[b][0] - logits[b][1] is the paper's yes/no
 * score.  cls_rows NULL: w_cls is the trained [C][d] head (cls_vocab ignored).
 * Debug mode checks 0 <= cls_rows[i] < cls_vocab. */
typedef struct sp_probe_weights {
  const void* in_norm;
  const void* w_q;
  const void* w_k;
  const void* w_v;
  const void* w_o;
  const void* post_norm;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
  const void* final_norm;
  const void* w_cls;
  const float* b_cls;
  const int32_t* cls_rows;     /* nullable, device */
  int64_t cls_vocab;           /* rows of w_cls when cls_rows is set */
  /* nullable, device: an fp16 image of the seven projection matrices made by
   * sp_probe_pack_weights for this config (bf16 storage only).  When set, the
   * forwards read w_q, w_k, w_v, w_o, w_gate, w_up and w_down from the image
   * (those seven pointers may then be NULL) and skip the per-fragment
   * conversion; the results are identical bit for bit. */
  const void* packed;
} sp_probe_weights;

typedef struct sp_probe sp_probe_t;  /* opaque handle, library-owned */

/* Bytes of device workspace a handle with this config allocates on the
 * current device (0 if invalid).  The split plan depends on the device's
 * compute-unit count; with no device, 256 compute units are assumed. */
size_t sp_probe_workspace_bytes(const sp_probe_config* cfg);

/* The frozen head's fp16 weight image (Sec. 3.2: the head is frozen, so its
 * matrices can be converted once and reused by every forward).
 * sp_probe_packed_bytes: bytes of the image for cfg (0 if cfg is invalid or not
 * SP_BF16).  sp_probe_pack_weights: enqueues on `stream` the conversion of the
 * bf16 matrices w_q, w_k, w_v, w_o, w_gate, w_up, w_down of `weights` (device,
 * the layouts of sp_probe_weights) into `packed` (device, caller-owned,
 * 16-byte aligned, packed_bytes >= sp_probe_packed_bytes(cfg)): a 256-byte
 * header naming the shape, then the matrices as fp16.  The values are
 * converted exactly (the same conversion the projections otherwise apply per
 * fragment), so forwards with and without the image return identical logits.
 * The image is a snapshot: pack again after changing the matrices.  Errors:
 * SP_ERR_INVALID_ARG (null or misaligned pointers, packed_bytes too small),
 * SP_ERR_UNSUPPORTED (an SP_F32 config), SP_ERR_NO_DEVICE. */
size_t sp_probe_packed_bytes(const sp_probe_config* cfg);
int sp_probe_pack_weights(const sp_probe_config* cfg, const sp_probe_weights* weights, void* packed,
                          size_t packed_bytes, void* stream);

/* Validate cfg, check that the current HIP device is gfx950, allocate the
 * workspace (soft-row scratch K/V, queries, split partials, activations) for
 * max_batch x max_seq_len and return a handle in *out.  The only allocating call. */
int sp_probe_init(const sp_probe_config* cfg, sp_probe_t** out);

/* The classification forward (Sec. 3.2-3.3) for kv_cache->batch sequences.
 *   seq_lens    device int32[B]: committed-prefix length N_b of each sequence (may be 0)
 *   block_table device int32[B * max_blocks_per_seq] or NULL (contiguous storage)
 *   soft_prompt device [k][d]: the task's soft-prompt vectors, row j at position N_b + j
 *   weights     frozen head + classifier (host struct of device pointers)
 *   logits      device fp32 [B][C], written; raw scores before any sigmoid/softmax
 *   stream      hipStream_t
 * Device-resident seq_lens and block ids are trusted unless SP_FLAG_DEBUG is set. */
int sp_probe_forward(sp_probe_t* h, const sp_kv_cache* kv_cache, const int32_t* seq_lens,
                     const int32_t* block_table, const void* soft_prompt,
                     const sp_probe_weights* weights, float* logits, void* stream);

/* The MTP input fusion of the head (Sec. 3.1): the layer's input at a position
 * is W_fc [RMSNorm(h; gamma_h); RMSNorm(e; gamma_e)] for a hidden state h and an
 * embedding e.  Device pointers in the config's dtype, 16-byte aligned:
 *   fc_norm_hidden[d] = gamma_h, fc_norm_embed[d] = gamma_e,
 *   w_fc[d][2d] row-major: columns 0..d-1 multiply the normed hidden state,
 *   columns d..2d-1 the normed embedding (a checkpoint that stores the other
 *   order is passed with its two column halves swapped). */
typedef struct sp_probe_fusion {
  const void* fc_norm_hidden;
  const void* fc_norm_embed;
  const void* w_fc;
  /* Eagle3 input (Sec. 3.1, Eagle3 paragraph): NULL for the MTP head, whose first
   * hidden state is the base model's last layer (hidden_last [B][d]); else a
   * [d][3d] matrix, hidden_last is [B][3d] (three of the base model's hidden
   * states, low / mid / high layer, concatenated) and the first step's hidden
   * state is w_hidden_fuse . hidden_last[b]. */
  const void* w_hidden_fuse;
} sp_probe_fusion;

/* Recursive SP-k, the form the paper evaluates (Sec. 3.2, with the fusion of
 * Sec. 3.1): k steps of the head, one row per sequence each.  Step t = 0..k-1
 * takes the fused row x_t = W_fc [RMSNorm(h_t; gamma_h); RMSNorm(e_t; gamma_e)]
 * with e_t = soft_prompt row t, h_0 = hidden_last[b] (the base model's last
 * hidden state) and h_t = f_{t-1} (the final-normed output of the step before);
 * it sits at position N_b + t and attends to the N_b cached keys plus the soft
 * keys of steps 0..t.  The read-out is the config's pool over the steps' f_t
 * (SP_POOL_LAST: f_{k-1}, the output of the k-th step).  The cache is read once
 * per step.
 *   hidden_last  device [B][d] in the config's dtype ([B][3d] with w_hidden_fuse)
 *   fusion       host struct of device pointers
 * Every other argument, the checks and the error behaviour are those of
 * sp_probe_forward; the same handle serves both forwards. */
int sp_probe_forward_recursive(sp_probe_t* h, const sp_kv_cache* kv_cache, const int32_t* seq_lens,
                               const int32_t* block_table, const void* soft_prompt,
                               const void* hidden_last, const sp_probe_fusion* fusion,
                               const sp_probe_weights* weights, float* logits, void* stream);

/* Several monitoring tasks over one cache in one call (Sec. 3.3: one pass over
 * the cached K/V serves every task).  Task t has its own k soft-prompt rows and
 * its own classifier; the frozen head is shared.  Each task's soft rows sit at
 * positions N_b .. N_b+k-1 and attend to the cache and causally to the soft rows
 * of their own task only, so every task's logits equal those of sp_probe_forward
 * with that task's soft prompt and classifier.
 *   n_tasks      1 .. max_tasks of the handle
 *   soft_prompts device [n_tasks][k][d]
 *   weights      the frozen head as for sp_probe_forward; w_cls is [n_tasks][C][d]
 *                and b_cls (nullable) [n_tasks][C]
 *   logits       device fp32 [B][n_tasks][C]
 * Everything else as sp_probe_forward; sp_probe_forward is the n_tasks = 1 case. */
int sp_probe_forward_multi(sp_probe_t* h, const sp_kv_cache* kv_cache, const int32_t* seq_lens,
                           const int32_t* block_table, int32_t n_tasks, const void* soft_prompts,
                           const sp_probe_weights* weights, float* logits, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): sp_probe_forward
 * without a handle.  The workspace is a static device array of 64 MiB per
 * device (allocated when the library's code object loads, held until the
 * process ends); the call allocates nothing, host or device.  cfg is checked
 * as by sp_probe_init; every other argument, the checks and the results are
 * those of sp_probe_forward (the same kernels and plan: logits identical bit
 * for bit to a handle's).  Errors: SP_ERR_CAPACITY if the config's workspace
 * (sp_probe_plan_config) exceeds 64 MiB; SP_ERR_UNSUPPORTED for SP_FLAG_DEBUG
 * or SP_FLAG_PROFILE (no handle holds their flags or events; the status word
 * is not reported either).  All calls on one device share its array and the
 * last call's contents stay in it: calls that overlap on one device (other
 * streams, other threads) race and must be ordered by the caller.  The first
 * call on a device resolves the array's address there. */
int sp_probe_forward_noalloc(const sp_probe_config* cfg, const sp_kv_cache* kv_cache, const int32_t* seq_lens,
                             const int32_t* block_table, const void* soft_prompt,
                             const sp_probe_weights* weights, float* logits, void* stream);

/* Free the workspace and the handle (waits for the device). NULL is accepted. */
int sp_probe_destroy(sp_probe_t* h);

/* Human-readable name of a status code (static string). */
const char* sp_probe_status_string(int status);

/* Intermediate values of the last forward, for tests.  Row b*k + j is soft row
 * j (one-pass) or step j (recursive) of sequence b; with T tasks, row
 * (b*T + t)*k + j is soft row j of task t; with SP_FLAG_LAST_ROW_ONLY the
 * one-pass forwards fill row b*T + t with task t's last soft row.  Sizes are
 * for max_tasks tasks.  tap selects:
 *   SP_TAP_QKV   fp32 [T k][(n_q + 2 n_kv) hd]  projections of the normed soft rows
 *                                              (one-pass forwards only)
 *   SP_TAP_ATTN  [B T k][n_q hd]               attention output (fp16 for SP_BF16,
 *                                              fp32 for SP_F32)
 *   SP_TAP_A     fp32 [B T k][d]               residual after the o-projection
 *   SP_TAP_Y     fp32 [B T k][d]               residual after the MLP
 *   SP_TAP_X     fp32 [B k][d]                 fused input rows x_t (recursive forward only)
 * sp_probe_tap_bytes returns the size for a batch; sp_probe_copy_tap enqueues a
 * device-to-device copy of it into dst (device, dst_bytes >= that size). */
enum { SP_TAP_QKV = 0, SP_TAP_ATTN = 1, SP_TAP_A = 2, SP_TAP_Y = 3, SP_TAP_X = 4 };
size_t sp_probe_tap_bytes(const sp_probe_t* h, int tap, int32_t batch);
int sp_probe_copy_tap(sp_probe_t* h, int tap, int32_t batch, void* dst, size_t dst_bytes, void* stream);

/* Wait for `stream` and report what the forwards since the last call met on
 * the device, then clear it: SP_ERR_INTERNAL if a guard word of the workspace
 * was overwritten; SP_ERR_DEVICE_DATA for a seq_len outside [0, max_seq_len]
 * (any mode) or, in debug mode, an invalid block id, class row or weight-image
 * header; SP_ERR_RANGE if an fp16 activation exceeded 65504; else SP_OK.
 * Synchronises the host. */
int sp_probe_check_device_error(sp_probe_t* h, void* stream);

/* Profiling mode: per-stage device time summed over the forwards since the last
 * read (waits for them).  Stages, in order: 0 soft-row prep (norm, QKV, RoPE;
 * recursive: with the fusion), 1 split attention, 2 split merge, 3 o-projection,
 * 4 post-attention norm, 5 gate/up + SwiGLU, 6 down projection, 7 final norm +
 * classifier (recursive: the final norm of every step); a recursive forward adds
 * its k steps into the same stages.  stage_ms[n_stages] receives milliseconds,
 * *n_forwards the number of forwards counted: the last ones whose events fit a
 * pool of 256 * (SP_N_STAGES + 1) (256 one-pass forwards; 2304 / (8k + 1)
 * recursive ones). */
#define SP_N_STAGES 8
int sp_probe_profile_read(sp_probe_t* h, float* stage_ms, int32_t n_stages, int32_t* n_forwards);

/* Split plan of a handle: tokens per attention split and the launch grid of
 * the split-attention kernel of a one-task one-pass forward (honouring
 * SP_FLAG_LAST_ROW_ONLY) for a batch (for measurement and tests). */
int sp_probe_plan(const sp_probe_t* h, int32_t batch, int32_t* split_len, int32_t* max_splits,
                  int32_t* rows_per_kv_head, int32_t* query_groups);
/* The same for the attention of a recursive step (G query rows per KV head). */
int sp_probe_plan_recursive(const sp_probe_t* h, int32_t batch, int32_t* split_len,
                            int32_t* max_splits, int32_t* rows_per_kv_head, int32_t* query_groups);
/* The one-task one-pass split plan and the workspace size a handle with cfg
 * would use on a device of num_cus compute units; host only (no device
 * needed).  Any output pointer may be NULL.  SP_ERR_INVALID_ARG for num_cus
 * outside 1..65536, else the status of the config check. */
int sp_probe_plan_config(const sp_probe_config* cfg, int32_t num_cus, int32_t* split_len,
                         int32_t* max_splits, int32_t* rows_per_kv_head, int32_t* query_groups,
                         size_t* workspace_bytes);

/* Measurement: the rate of plain streaming reads of `bytes` (>= 16) at `buf`
 * (device, 16-byte aligned, read only) on the current device, the ceiling of a
 * read-bound kernel: one warm-up pass, then `reps` timed passes on `stream`
 * (each workgroup reads one contiguous slice with 16-byte non-temporal loads,
 * eight in flight per lane); *gbps receives the bytes read per second / 1e9.
 * `sink` (device, 4 bytes) may be written.  Synchronises the host.
 * SP_ERR_INVALID_ARG, SP_ERR_NO_DEVICE, SP_ERR_HIP. */
int sp_probe_measure_read(const void* buf, size_t bytes, int32_t reps, void* sink, float* gbps, void* stream);

/* Measurement: the dense fp16 matrix-core rate the current device sustains,
 * the practical ceiling of the projections: every SIMD runs eight waves, each
 * issuing `iters` x 4 independent 16x16x32 fp16 MFMAs (fp32 accumulation) with
 * no memory traffic; one warm-up launch, then one timed launch on `stream`.
 * *tflops receives the multiply-add FLOP per second / 1e12.  `sink` (device,
 * 4 bytes) may be written.  Synchronises the host.  SP_ERR_INVALID_ARG
 * (iters < 1, NULL pointers), SP_ERR_NO_DEVICE, SP_ERR_HIP. */
int sp_probe_measure_mfma(int32_t iters, void* sink, float* tflops, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SP_PROBE_H */
