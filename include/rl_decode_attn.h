/*
 * rl_decode_attn.h -- paged grouped-query decode attention for MI355X (gfx950).
 *
 * One call computes one decode step of one attention layer for a batch of
 * sequences: the operation that dominates rollout generation in RL
 * post-training (arXiv 2512.22492, Sec. 1 and Sec. 2.1: rollout runs in an
 * inference engine over a paged KV cache and takes most of post-training
 * time).  For every sequence b and query head h,
 *
 *     out[b,h,:] = sum_t softmax_t( scale * <q[b,h,:], K_b[t,kvh,:]> ) V_b[t,kvh,:]
 *
 * over the t = 0 .. seq_lens[b]-1 cached tokens, with kv head
 * kvh = h / (Hq / Hkv) (grouped-query attention: consecutive query heads share
 * a kv head).  Token t of sequence b is stored in physical page
 * block_table[b][t / page_size], slot t % page_size.
 *
 * Memory layouts (row-major, innermost last).  Every device pointer below is
 * owned by the caller; the library never frees or retains it past the call.
 *   q            [batch][Hq][head_dim]                         bf16
 *   k_pool       [num_pages][Hkv][page_size][head_dim]         bf16 or e4m3
 *                (layout RL_DA_LAYOUT_HND), or
 *                [num_pages][page_size][Hkv][head_dim]         (RL_DA_LAYOUT_NHD)
 *   v_pool       same as k_pool
 *                or, with RL_DA_LAYOUT_HND_KV, one allocation
 *                [num_pages][Hkv][2][page_size][head_dim] holding a (page, kv
 *                head)'s key slab and then its value slab: k_pool points at
 *                its start and v_pool exactly one slab (page_size * head_dim
 *                elements) further
 *   k_scale      [num_pages][Hkv] fp32, fp8 pools only: a stored code c of
 *   v_scale      slab (page, kvh) stands for e4m3(c) * scale[page][kvh]
 *   block_table  [batch][max_pages] int32 (row stride max_pages)
 *   seq_lens     [batch] int32
 *   out          [batch][Hq][head_dim]                         bf16
 * e4m3 is the OCP 8-bit float E4M3FN (bias 7, largest finite 448, no infinity).
 *
 * Execution.  run() enqueues its kernels on the caller's HIP stream and
 * returns without synchronising; the result is ready when the stream has
 * reached that point.  run() never allocates: the handle owns a workspace
 * sized at create() for max_batch and max_pages_per_seq.  Results are
 * deterministic: no atomics take part in any reduction, the split size is
 * fixed per handle and partial results merge in a fixed order, so a
 * sequence's output does not depend on the rest of the batch or on where its
 * pages sit in the pool.  With several splits per sequence and more work
 * units than the device holds at once, the split kernel runs persistent
 * work-groups that take units, longest first, from a counter in the handle's
 * workspace (the last work-group of each launch resets it); which work-group
 * computes a unit never changes a result.
 *
 * Concurrency.  The runs of one handle share its workspace: the per-split
 * partial results, the persistent schedule's unit counter and the error
 * word.  They must therefore be ordered on one stream (or otherwise never
 * overlap); two runs of one handle that overlap on two streams race on all
 * three and give wrong outputs without any error.  Use one handle per
 * stream; different handles never share state.  A run that returned
 * RL_DA_ERR_HIP, or whose stream later reports an error, may have stopped
 * with the unit counter not reset: destroy the handle and create a new one
 * before running again (after a device fault the HIP context itself is
 * unusable and must be re-created first).
 *
 * Errors.  Every entry point returns an rl_da_status; nothing is thrown
 * across the interface.  run() checks its host-visible arguments and returns
 * RL_DA_ERR_INVALID_ARG or RL_DA_ERR_UNSUPPORTED before launching anything.
 * It does not read device memory to check, so these are preconditions:
 *   0 <= block_table[b][j] < num_pages  for j < ceil(seq_lens[b] / page_size)
 *   seq_lens[b] <= max_pages * page_size
 * Block-table entries past a sequence's last page (inside the table row) may
 * hold anything and are never used as page indices; token slots past a
 * sequence's length are masked and may hold anything, including NaN.  A
 * sequence with seq_lens[b] <= 0 produces zeros.  With RL_DA_CHECKED set at
 * create(), the kernels test the preconditions, skip the offending work, and
 * record the violation in a device error word read by
 * rl_decode_attn_check_error().
 */
#ifndef RL_DECODE_ATTN_H
#define RL_DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rl_decode_attn rl_decode_attn; /* opaque handle */

typedef enum {
    RL_DA_OK = 0,
    RL_DA_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, bad size         */
    RL_DA_ERR_UNSUPPORTED = 2,   /* valid request this build does not serve   */
    RL_DA_ERR_OUT_OF_MEMORY = 3, /* workspace allocation failed in create()   */
    RL_DA_ERR_HIP = 4,           /* a HIP runtime call or launch failed       */
    RL_DA_ERR_SCRATCH_TOO_SMALL = 5 /* rl_decode_attn_run_noalloc: the step's  */
                                 /* workspace exceeds its fixed scratch       */
} rl_da_status;

typedef enum { RL_DA_KV_BF16 = 0, RL_DA_KV_FP8_E4M3 = 1 } rl_da_kv_dtype;

/* Order of a page's (kv head, token slot) rows in the pools.  HND keeps each
 * (page, kv head) slab contiguous; NHD keeps each token slot's kv heads
 * together (the page-major layout many serving engines allocate); HND_KV
 * puts a (page, kv head)'s value slab right after its key slab in one
 * allocation, so a decode step reads one contiguous block per (page, kv head)
 * (twice the slab: 4 KiB for e4m3, 8 KiB for bf16) instead of two.  The fp8
 * scales are [num_pages][Hkv] in every layout.  With HND_KV every entry point
 * that takes k_pool and v_pool returns INVALID_ARG unless v_pool is k_pool
 * plus one slab. */
typedef enum {
    RL_DA_LAYOUT_HND = 0,
    RL_DA_LAYOUT_NHD = 1,
    RL_DA_LAYOUT_HND_KV = 2
} rl_da_layout;

/* create() flag: kernels check block-table entries and lengths on device. */
#define RL_DA_CHECKED 0x1u
/* create() flag: form q.k with bf16 dot2 ops and DPP row sums on the vector
 * ALUs instead of packing the query group into an MFMA tile (same results up
 * to fp32 rounding; kept to measure one path against the other). */
#define RL_DA_SCORES_ON_VALU 0x2u
/* create() flag for token-major (RL_DA_LAYOUT_NHD) pools.  Such a handle
 * runs head-parallel units -- one work-group per (sequence, split, group of
 * up to 8 kv heads), one wavefront per kv head, so the group reads each
 * page's token rows together -- when its full-capacity batch cut into
 * four-wavefront units would fit on the device at once (768 work-groups);
 * a larger handle runs the head-major pools' units (four wavefronts per
 * (sequence, kv head, split)), which the persistent longest-first schedule
 * balances.  This flag always selects the four-wavefront units.  No effect
 * on head-major pools, with RL_DA_SCORES_ON_VALU, or with one kv head per
 * group (rl_decode_attn_unit_heads reports the choice). */
#define RL_DA_PER_HEAD_UNITS 0x4u
/* create() flag: accumulate the P.V product with vector-ALU FMAs on fp32
 * probabilities instead of on the matrix cores.  By default the four-wavefront
 * units form P.V with v_mfma_f32_16x16x16_bf16 over the page's values
 * transposed through LDS, each probability entering as two bf16 terms (hi +
 * lo, 2^-16 relative); kept to measure one path against the other.  Not
 * available for Hq / Hkv = 16 (UNSUPPORTED), whose accumulators only the
 * matrix-core pass holds; no effect on the head-parallel units, which keep
 * the vector-ALU pass. */
#define RL_DA_PV_ON_VALU 0x8u

/* Device error word bits reported by rl_decode_attn_check_error(). */
#define RL_DA_DEVERR_PAGE_OUT_OF_RANGE 0x1
#define RL_DA_DEVERR_LENGTH_TOO_LONG 0x2

typedef struct {
    int32_t num_q_heads;       /* Hq; a multiple of num_kv_heads               */
    int32_t num_kv_heads;      /* Hkv; Hq / Hkv in {1, 2, 4, 8, 16}            */
    int32_t head_dim;          /* 128                                         */
    int32_t page_size;         /* tokens per page: 16                         */
    int32_t max_batch;         /* largest batch a run() may pass (>= 1)       */
    int32_t max_pages_per_seq; /* largest block-table width a run() may pass  */
    int32_t kv_dtype;          /* rl_da_kv_dtype                              */
    int32_t layout;            /* rl_da_layout                                */
    int32_t split_tokens;      /* tokens per split-K work unit: a multiple of */
                               /* page_size, at most 4096; 0 = the longest of */
                               /* 4096, 2048, 1024, 512 that cuts max_batch   */
                               /* sequences of max_pages_per_seq pages into   */
                               /* >= 256 work-groups (a per-handle constant)  */
    uint32_t flags;            /* RL_DA_CHECKED, RL_DA_SCORES_ON_VALU,        */
                               /* RL_DA_PER_HEAD_UNITS, RL_DA_PV_ON_VALU, 0   */
} rl_da_config;

/*
 * Validates cfg and allocates a handle plus its device workspace on the
 * current HIP device.  On success *out owns both; on failure *out is NULL.
 * INVALID_ARG for null pointers or non-positive sizes, UNSUPPORTED for shapes
 * this build has no kernel for, OUT_OF_MEMORY / HIP when allocation fails.
 */
rl_da_status rl_decode_attn_create(const rl_da_config* cfg, rl_decode_attn** out);

/*
 * Enqueues one decode step on `stream` (a hipStream_t; NULL = null stream).
 * Pointers as in the layout table above; q, the pools and out must be 16-byte
 * aligned.  k_scale and v_scale must be non-NULL exactly for fp8 handles.
 * 0 <= batch <= max_batch, 1 <= max_pages <= max_pages_per_seq, num_pages >= 1,
 * scale finite.  batch == 0 enqueues nothing.
 */
rl_da_status rl_decode_attn_run(rl_decode_attn* h, const void* q,
                                const void* k_pool, const void* v_pool,
                                const float* k_scale, const float* v_scale,
                                int64_t num_pages, const int32_t* block_table,
                                int32_t max_pages, const int32_t* seq_lens,
                                int32_t batch, float scale, void* out,
                                void* stream);

/* Frees the handle and its workspace.  NULL is accepted.  The caller must
 * ensure no enqueued run() still uses the handle. */
rl_da_status rl_decode_attn_destroy(rl_decode_attn* h);

/* Static description of a status code. */
const char* rl_da_status_string(rl_da_status s);

/* Device workspace bytes create() would allocate for cfg (host only). */
rl_da_status rl_decode_attn_workspace_size(const rl_da_config* cfg,
                                           size_t* bytes);

/*
 * Checked handles only: waits for the stream of the handle's latest run()
 * (only that stream; other work on the device is not waited for), stores the
 * RL_DA_DEVERR_* bits accumulated since the previous call in *device_error
 * and clears them with a kernel enqueued on that stream.  UNSUPPORTED for a
 * handle created without RL_DA_CHECKED.
 */
rl_da_status rl_decode_attn_check_error(rl_decode_attn* h, int32_t* device_error);

/* Split-K geometry of a handle: tokens per split and the number of splits a
 * block table of max_pages columns is divided into. */
rl_da_status rl_decode_attn_split_info(const rl_decode_attn* h, int32_t max_pages,
                                       int32_t* split_tokens, int32_t* num_splits);

/* Work-unit family of a handle (host only): *kv_heads_per_unit = 1 for the
 * four-wavefront units of one kv head, or the number of kv heads of a
 * head-parallel unit (token-major pools). */
rl_da_status rl_decode_attn_unit_heads(const rl_decode_attn* h, int32_t* kv_heads_per_unit);

/*
 * Extend (prefill) attention: causal attention of several new tokens per
 * sequence over the paged cache, for multi-turn continuations and re-prefill
 * of trajectories (the rollout's multi-turn tool interactions, Sec. 2.1, and
 * the reassignment of a failed rollout's trajectories, Sec. 5.2.2).  The new
 * tokens' keys and values must already be in the cache (rl_kv_append or the
 * caller's own writes): sequence b's n_b = q_start[b+1] - q_start[b] new
 * tokens are the last n_b of its L_b = seq_lens[b] cached tokens.  Row
 * q_start[b] + i of q / out (new token i of b) attends to cached tokens
 * 0 .. L_b - n_b + i:
 *     out[r,h,:] = sum_t softmax_t(scale * <q[r,h,:], K_b[t,kvh,:]>) V_b[t,kvh,:]
 * q, out: [T][num_q_heads][head_dim] bf16 with T = q_start[batch]; q_start:
 * [batch+1] int32 device array, non-decreasing from 0; pools, block_table and
 * seq_lens as for rl_decode_attn_run.  max_q_per_seq >= every n_b (sizes the
 * grid).  Preconditions: n_b <= L_b <= max_pages * page_size and the table
 * entries of pages 0 .. (L_b-1)/page_size in [0, num_pages).  Needs no
 * handle and no workspace; enqueues one kernel on `stream`.  bf16 or e4m3
 * pools (k_scale and v_scale non-NULL exactly for e4m3, as for decode),
 * any rl_da_layout, head_dim 128, page_size 16, Hq/Hkv in {1, 2, 4, 8, 16}
 * and pages (all kv heads) under 2 GiB only (else UNSUPPORTED); q, the pools
 * and out 16-byte aligned.
 */
rl_da_status rl_extend_attn(const void* q, const int32_t* q_start, int32_t max_q_per_seq,
                            const void* k_pool, const void* v_pool, const float* k_scale,
                            const float* v_scale, int64_t num_pages, const int32_t* block_table,
                            int32_t max_pages, const int32_t* seq_lens, int32_t batch,
                            int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                            int32_t page_size, int32_t kv_dtype, int32_t layout, float scale,
                            void* out, void* stream);

/*
 * KV-cache append: the step before attention in every decode step (the
 * rollout engine generates one token per sequence per step, Sec. 2.1; the
 * new token's key and value join the paged cache the attention then reads).
 * For every sequence b with L = seq_lens[b] >= 0 (its length BEFORE the
 * append) and every kv head, the new token k_new[b][kvh][:], v_new[b][kvh][:]
 * (bf16, [batch][num_kv_heads][head_dim]) is written to page
 * block_table[b][L / page_size], slot L % page_size of k_pool / v_pool.  The
 * caller has already placed that page in the table and increments seq_lens
 * afterwards.
 *
 * bf16 pools: the token's bits are copied.  e4m3 pools keep one fp32 scale
 * per (page, kv head) that only grows (the paper is silent on re-scaling; this
 * is the build's reading), computed in fp32 and rounded to nearest even:
 *   slot 0 (fresh page):  scale = absmax(token) / 448, or 1 if zero
 *   other slots:  scale' = max(scale, absmax(token) / 448); when it grows,
 *     each earlier code c of the slab becomes e4m3(value(c) * (scale/scale'))
 *   the token:  e4m3(clamp(x / scale', -448, 448))
 * Different sequences must append into different (page, kv head) slabs.
 *
 * Bounds are checked on the device: a sequence whose L is at least
 * max_pages * page_size, or whose target page is outside [0, num_pages), is
 * skipped (nothing written) and, when device_error is non-NULL, reported in
 * that int32 device word with RL_DA_DEVERR_LENGTH_TOO_LONG /
 * RL_DA_DEVERR_PAGE_OUT_OF_RANGE (bits are only ever set).  Needs no handle;
 * enqueues one kernel on `stream`.  Pools in any rl_da_layout;
 * head_dim 128 and page_size 16 only (else UNSUPPORTED); k_new, v_new and the
 * pools 16-byte aligned; k_scale and v_scale non-NULL exactly for e4m3.
 */
rl_da_status rl_kv_append(const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                          float* k_scale, float* v_scale, int64_t num_pages,
                          const int32_t* block_table, int32_t max_pages,
                          const int32_t* seq_lens, int32_t batch, int32_t num_kv_heads,
                          int32_t head_dim, int32_t page_size, int32_t kv_dtype,
                          int32_t layout, int32_t* device_error, void* stream);

/*
 * Measurement hook (no counterpart in the paper): with both events non-NULL,
 * every later run() launches its split-K kernel with split_begin and
 * split_end attached to the launch itself (hipExtLaunchKernel), so they take
 * that kernel's start and end timestamps and hipEventElapsedTime gives its
 * duration, with nothing inserted between the launches of a step.  Events
 * are hipEvent_t owned by the caller; NULL, NULL turns recording off.
 * INVALID_ARG if exactly one event is NULL.
 */
rl_da_status rl_decode_attn_set_timing_events(rl_decode_attn* h, void* split_begin,
                                              void* split_end);

/* Bytes of device scratch that rl_decode_attn_run_noalloc uses on each device. */
#define RL_DA_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: one decode
 * step exactly as rl_decode_attn_run computes it for a handle created with
 * cfg (same kernels, same split size, bit-identical results), with the
 * handle's workspace replaced by a fixed array of
 * RL_DA_NOALLOC_SCRATCH_BYTES in device memory that the library holds on each
 * device it runs on until the process ends.  Calls no hipMalloc or hipFree
 * and allocates no host memory; the first call on a device looks up that
 * device's copy of the array.  Arguments and preconditions as for create()
 * plus run(); the caller still owns every input and output.
 *   RL_DA_ERR_SCRATCH_TOO_SMALL  when rl_decode_attn_workspace_size(cfg)
 *                                exceeds RL_DA_NOALLOC_SCRATCH_BYTES
 *                                (nothing is enqueued)
 *   RL_DA_ERR_UNSUPPORTED        with RL_DA_CHECKED (there is no handle whose
 *                                error word could be read)
 * Every call on one device shares that device's scratch, which keeps the
 * last call's contents: calls that can overlap on one device (two streams,
 * two host threads enqueueing concurrently) race on it and give wrong
 * results.  Order them on one stream.  Before each launch that uses the unit
 * queue, the queue is cleared by a kernel on the caller's stream.
 */
rl_da_status rl_decode_attn_run_noalloc(const rl_da_config* cfg, const void* q,
                                        const void* k_pool, const void* v_pool,
                                        const float* k_scale, const float* v_scale,
                                        int64_t num_pages, const int32_t* block_table,
                                        int32_t max_pages, const int32_t* seq_lens,
                                        int32_t batch, float scale, void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif
