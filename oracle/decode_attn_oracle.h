/*
 * decode_attn_oracle.h -- C interface of the fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY: used by tests, the smoke check and the benchmark's
 * CPU-baseline leg.  Independent of the GPU library (no shared code).
 *
 * Every pointer is a host pointer owned by the caller.  The oracle never
 * writes its inputs.  Layouts (row-major, innermost last):
 *   q            [batch][num_q_heads][head_dim]            bf16 bit patterns
 *   k_pool/v_pool [num_pages][num_kv_heads][page_size][head_dim] (layout HND)
 *                 or [num_pages][page_size][num_kv_heads][head_dim] (NHD);
 *                 bf16 bit patterns, or OCP e4m3 codes for the fp8 variant
 *   k_scale/v_scale [num_pages][num_kv_heads] fp32 (fp8 only, else unused)
 *   block_table  [batch][max_pages] int32 physical page indices
 *   seq_lens     [batch] int32 cached tokens per sequence (<= 0: empty)
 *   out          [num_rows][head_dim] fp64, one row per requested (b, h)
 */
#ifndef RL_DECODE_ATTN_ORACLE_H
#define RL_DECODE_ATTN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    RL_ORACLE_OK = 0,
    RL_ORACLE_ERR_ARG = 1,          /* malformed problem description          */
    RL_ORACLE_ERR_PRECONDITION = 2, /* page index or length out of range      */
    RL_ORACLE_ERR_NOMEM = 3
};

enum { RL_ORACLE_KV_BF16 = 0, RL_ORACLE_KV_FP8_E4M3 = 1 };

/* Pool layouts: [page][kv head][slot][dim] (HND) or [page][slot][kv head][dim]. */
enum { RL_ORACLE_LAYOUT_HND = 0, RL_ORACLE_LAYOUT_NHD = 1 };

typedef struct {
    int32_t batch, num_q_heads, num_kv_heads, head_dim, page_size;
    int32_t kv_dtype;   /* RL_ORACLE_KV_*                                  */
    int32_t layout;     /* RL_ORACLE_LAYOUT_*                              */
    int32_t max_pages;  /* columns of block_table                          */
    int64_t num_pages;  /* pages in each pool                              */
    double scale;       /* softmax scale applied to q.k                    */
    const void* q;
    const void* k_pool;
    const void* v_pool;
    const float* k_scale;
    const float* v_scale;
    const int32_t* block_table;
    const int32_t* seq_lens;
} rl_oracle_problem;

/*
 * out[r][:] = attention row (b, h) = (rows[2r], rows[2r+1]) for r < num_rows;
 * rows == NULL computes every (b, h), b-major.  Rows whose sequence is empty
 * are zero.  Fails with RL_ORACLE_ERR_PRECONDITION, writing nothing, when a
 * requested row reads a block-table entry outside [0, num_pages) or has a
 * length beyond max_pages * page_size.
 */
int rl_oracle_decode_attn(const rl_oracle_problem* p, const int32_t* rows,
                          int64_t num_rows, double* out);

/*
 * Extend (prefill) attention over the paged cache.  q is [T][num_q_heads]
 * [head_dim] bf16 bits with T = q_start[batch]; rows q_start[b] ..
 * q_start[b+1]-1 are sequence b's n_b new tokens, whose keys/values are the
 * last n_b of its seq_lens[b] cached tokens.  Row q_start[b] + i attends
 * causally to cache tokens 0 .. seq_lens[b] - n_b + i.  out is [T][Hq][D]
 * fp64.  p->batch, seq_lens, block_table, pools as for decode (p->q is the
 * [T][Hq][D] array).
 */
int rl_oracle_extend_attn(const rl_oracle_problem* p, const int32_t* q_start, double* out);

/*
 * One decode step's K/V cache append (the step before attention): the new
 * token of every sequence b (k_new/v_new [batch][num_kv_heads][head_dim] bf16
 * bits) is written to page block_table[b][L/page_size], slot L%page_size,
 * L = seq_lens[b] (length before the append; L < 0 skips b).  e4m3 pools keep
 * one fp32 scale per (page, kv head) that only grows; see the .c file for the
 * exact fp32 rules.  Pools and scales are updated in place.
 */
typedef struct {
    int32_t batch, num_kv_heads, head_dim, page_size;
    int32_t kv_dtype;
    int32_t layout;
    int32_t max_pages;
    int64_t num_pages;
    const void* k_new;
    const void* v_new;
    void* k_pool;
    void* v_pool;
    float* k_scale;
    float* v_scale;
    const int32_t* block_table;
    const int32_t* seq_lens;
} rl_oracle_append;

int rl_oracle_kv_append(const rl_oracle_append* p);

/* Round-to-nearest-even e4m3 code of x, |x| <= 448 (NaN -> 0x7F). */
uint8_t rl_oracle_e4m3_encode(float x);

/* Exact value of one OCP E4M3FN code (NaN for S.1111.111). */
double rl_oracle_e4m3_to_double(uint8_t code);

/* Exact value of one bf16 bit pattern. */
double rl_oracle_bf16_to_double(uint16_t bits);

/* OpenMP threads the oracle will use (1 without OpenMP). */
int rl_oracle_max_threads(void);

/* Sets the number of OpenMP threads for later calls (no effect without OpenMP). */
void rl_oracle_set_threads(int n);

#ifdef __cplusplus
}
#endif

#endif
