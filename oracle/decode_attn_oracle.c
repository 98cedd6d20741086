/*
 * decode_attn_oracle.c -- fp64 CPU oracle for one decode step of paged
 * grouped-query attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This file exists so that tests, the smoke check
 * and the CPU-baseline leg of the benchmark can check the GPU library.  No
 * product code may include, link or call it, and it includes and links
 * nothing from the GPU library: the two share no source, header, table or
 * helper.
 *
 * What is computed.  The paper (arXiv 2512.22492, Sec. 1 and Sec. 2.1) places
 * rollout generation in an inference engine with a paged KV cache
 * (PagedAttention, cited in Sec. 1 and Sec. 9); it prints no attention
 * formula.  The operation is the textbook scaled dot-product attention of one
 * new query token per sequence against that sequence's cached keys/values,
 * with grouped KV heads:
 *
 *     out[b,h,:] = sum_t softmax_t( scale * <q[b,h,:], K[b,kvh,t,:]> ) V[b,kvh,t,:]
 *     kvh = floor(h / G),  G = Hq / Hkv,  t = 0 .. seq_lens[b]-1
 *
 * where the cached token t of sequence b lives in physical page
 * block_table[b][t / page_size], slot t % page_size, and a pool is laid out
 * [num_pages][Hkv][page_size][D].  For fp8 pools every (page, kv head) slab
 * carries one fp32 scale, and a stored code c stands for e4m3(c) * scale.
 *
 * The oracle favours being checkable by eye over speed: every score is formed
 * in fp64 from the exactly decoded inputs, summed over d in increasing order,
 * then the maximum is subtracted, exponentiated, normalised and the weighted
 * sum of values formed, again in fp64.  Nothing is blocked or fused.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "decode_attn_oracle.h"

/* bf16 is the upper half of an IEEE binary32; widening is exact. */
static double oracle_bf16_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * OCP 8-bit floating point, E4M3 ("FN": finite, no infinities): sign bit,
 * 4 exponent bits with bias 7, 3 mantissa bits.  Exponent field 0 holds the
 * subnormals m/8 * 2^-6; the single code S.1111.111 is NaN; every other code
 * with exponent field 15 is a normal number (so the largest is 448).
 */
double rl_oracle_e4m3_to_double(uint8_t code)
{
    const int sign = (code >> 7) & 1;
    const int e = (code >> 3) & 0xF;
    const int m = code & 0x7;
    double mag;
    if (e == 0xF && m == 0x7)
        return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, -6);
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -mag : mag;
}

double rl_oracle_bf16_to_double(uint16_t bits)
{
    return oracle_bf16_to_double(bits);
}

/* Index of element d of token slot `slot`, kv head kvh, page `page`. */
static int64_t pool_index(int layout, int64_t page, int kvh, int slot, int d, int num_kv_heads,
                          int page_size, int head_dim)
{
    if (layout == RL_ORACLE_LAYOUT_NHD)
        return ((page * page_size + slot) * num_kv_heads + kvh) * (int64_t)head_dim + d;
    return ((page * num_kv_heads + kvh) * page_size + slot) * (int64_t)head_dim + d;
}

/* Decoded element d of token slot `slot` in slab (page, kvh) of a pool. */
static double pool_element(const rl_oracle_problem* p, const void* pool,
                           const float* slab_scale, int64_t page, int kvh,
                           int slot, int d)
{
    const int64_t idx = pool_index(p->layout, page, kvh, slot, d, p->num_kv_heads,
                                   p->page_size, p->head_dim);
    if (p->kv_dtype == RL_ORACLE_KV_BF16)
        return oracle_bf16_to_double(((const uint16_t*)pool)[idx]);
    return rl_oracle_e4m3_to_double(((const uint8_t*)pool)[idx]) *
           (double)slab_scale[(int64_t)page * p->num_kv_heads + kvh];
}

/* Checks the preconditions of one (b, h) row; nonzero when they hold. */
static int row_is_valid(const rl_oracle_problem* p, int b, int h)
{
    if (b < 0 || b >= p->batch || h < 0 || h >= p->num_q_heads)
        return 0;
    const int L = p->seq_lens[b];
    if (L <= 0)
        return 1;
    if ((int64_t)L > (int64_t)p->max_pages * p->page_size)
        return 0;
    const int used_pages = (L + p->page_size - 1) / p->page_size;
    for (int j = 0; j < used_pages; ++j) {
        const int32_t page = p->block_table[(int64_t)b * p->max_pages + j];
        if (page < 0 || (int64_t)page >= p->num_pages)
            return 0;
    }
    return 1;
}

/*
 * Attention of one query row qrow (head_dim bf16 values) over the first
 * `visible` cached tokens of sequence b, kv head kvh, written to dst[0..D-1].
 * `scores` is caller scratch of at least `visible` doubles; visible >= 1.
 */
static void attend_prefix(const rl_oracle_problem* p, const uint16_t* qrow, int b, int kvh,
                          int visible, double* scores, double* dst)
{
    const int D = p->head_dim;
    const int32_t* pages = p->block_table + (int64_t)b * p->max_pages;

    /* Scores s_t = scale * sum_d q[d] * k_t[d]. */
    for (int t = 0; t < visible; ++t) {
        const int64_t page = pages[t / p->page_size];
        const int slot = t % p->page_size;
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
            dot += oracle_bf16_to_double(qrow[d]) *
                   pool_element(p, p->k_pool, p->k_scale, page, kvh, slot, d);
        scores[t] = p->scale * dot;
    }

    /* Softmax weights w_t = exp(s_t - max_s) / sum_u exp(s_u - max_s). */
    double smax = scores[0];
    for (int t = 1; t < visible; ++t)
        if (scores[t] > smax)
            smax = scores[t];
    double z = 0.0;
    for (int t = 0; t < visible; ++t) {
        scores[t] = exp(scores[t] - smax);
        z += scores[t];
    }

    /* out[d] = sum_t w_t * v_t[d]. */
    for (int d = 0; d < D; ++d)
        dst[d] = 0.0;
    for (int t = 0; t < visible; ++t) {
        const int64_t page = pages[t / p->page_size];
        const int slot = t % p->page_size;
        const double w = scores[t] / z;
        for (int d = 0; d < D; ++d)
            dst[d] += w * pool_element(p, p->v_pool, p->v_scale, page, kvh,
                                       slot, d);
    }
}

/* Decode row out[b,h,:]: query q[b,h,:] over all seq_lens[b] tokens. */
static void attend_one_row(const rl_oracle_problem* p, int b, int h,
                           double* scores, double* dst)
{
    const int G = p->num_q_heads / p->num_kv_heads;
    const int L = p->seq_lens[b];
    if (L <= 0) {
        for (int d = 0; d < p->head_dim; ++d)
            dst[d] = 0.0;
        return;
    }
    const uint16_t* qrow =
        (const uint16_t*)p->q + ((int64_t)b * p->num_q_heads + h) * p->head_dim;
    attend_prefix(p, qrow, b, h / G, L, scores, dst);
}

int rl_oracle_decode_attn(const rl_oracle_problem* p, const int32_t* rows,
                          int64_t num_rows, double* out)
{
    if (p == NULL || out == NULL || p->q == NULL || p->k_pool == NULL ||
        p->v_pool == NULL || p->block_table == NULL || p->seq_lens == NULL)
        return RL_ORACLE_ERR_ARG;
    if (p->batch < 0 || p->num_q_heads <= 0 || p->num_kv_heads <= 0 ||
        p->num_q_heads % p->num_kv_heads != 0 || p->head_dim <= 0 ||
        p->page_size <= 0 || p->max_pages < 0 || p->num_pages < 0)
        return RL_ORACLE_ERR_ARG;
    if (p->kv_dtype != RL_ORACLE_KV_BF16 && p->kv_dtype != RL_ORACLE_KV_FP8_E4M3)
        return RL_ORACLE_ERR_ARG;
    if (p->layout != RL_ORACLE_LAYOUT_HND && p->layout != RL_ORACLE_LAYOUT_NHD)
        return RL_ORACLE_ERR_ARG;
    if (p->kv_dtype == RL_ORACLE_KV_FP8_E4M3 &&
        (p->k_scale == NULL || p->v_scale == NULL))
        return RL_ORACLE_ERR_ARG;

    /* rows == NULL means every (b, h) in order b-major. */
    const int64_t n =
        rows ? num_rows : (int64_t)p->batch * (int64_t)p->num_q_heads;
    int max_len = 1;
    for (int b = 0; b < p->batch; ++b)
        if (p->seq_lens[b] > max_len)
            max_len = p->seq_lens[b];

    for (int64_t r = 0; r < n; ++r) {
        const int b = rows ? rows[2 * r] : (int)(r / p->num_q_heads);
        const int h = rows ? rows[2 * r + 1] : (int)(r % p->num_q_heads);
        if (!row_is_valid(p, b, h))
            return RL_ORACLE_ERR_PRECONDITION;
    }

    int failed = 0;
#pragma omp parallel
    {
        double* scores = (double*)malloc(sizeof(double) * (size_t)max_len);
        if (scores == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < n; ++r) {
            if (scores == NULL)
                continue;
            const int b = rows ? rows[2 * r] : (int)(r / p->num_q_heads);
            const int h = rows ? rows[2 * r + 1] : (int)(r % p->num_q_heads);
            attend_one_row(p, b, h, scores, out + r * p->head_dim);
        }
        free(scores);
    }
    return failed ? RL_ORACLE_ERR_NOMEM : RL_ORACLE_OK;
}

/*
 * Extend (prefill) attention: n_b new query tokens per sequence whose keys and
 * values are already in the cache, i.e. the last n_b of its L_b = seq_lens[b]
 * cached tokens.  Query token i of sequence b (row q_start[b] + i of q/out)
 * sits at position L_b - n_b + i and attends causally to cache tokens
 * t <= L_b - n_b + i.  A decode step is the case n_b = 1.
 */
static void extend_one_row(const rl_oracle_problem* p, const int32_t* q_start, int64_t row,
                           int b, int h, double* scores, double* dst)
{
    const int G = p->num_q_heads / p->num_kv_heads;
    const int n_new = q_start[b + 1] - q_start[b];
    const int L = p->seq_lens[b];
    const int i = (int)(row - q_start[b]);
    const int visible = L - n_new + i + 1;  /* tokens 0 .. L-n_new+i */
    const uint16_t* qrow = (const uint16_t*)p->q + (row * p->num_q_heads + h) * p->head_dim;
    attend_prefix(p, qrow, b, h / G, visible, scores, dst);
}

int rl_oracle_extend_attn(const rl_oracle_problem* p, const int32_t* q_start, double* out)
{
    if (p == NULL || q_start == NULL || out == NULL || p->q == NULL || p->k_pool == NULL ||
        p->v_pool == NULL || p->block_table == NULL || p->seq_lens == NULL)
        return RL_ORACLE_ERR_ARG;
    if (p->batch < 0 || p->num_q_heads <= 0 || p->num_kv_heads <= 0 ||
        p->num_q_heads % p->num_kv_heads != 0 || p->head_dim <= 0 || p->page_size <= 0)
        return RL_ORACLE_ERR_ARG;
    if (p->kv_dtype == RL_ORACLE_KV_FP8_E4M3 && (p->k_scale == NULL || p->v_scale == NULL))
        return RL_ORACLE_ERR_ARG;
    if (p->layout != RL_ORACLE_LAYOUT_HND && p->layout != RL_ORACLE_LAYOUT_NHD)
        return RL_ORACLE_ERR_ARG;
    if (q_start[0] != 0)
        return RL_ORACLE_ERR_ARG;
    int max_len = 1;
    for (int b = 0; b < p->batch; ++b) {
        const int n = q_start[b + 1] - q_start[b];
        if (n < 0 || n > p->seq_lens[b])
            return RL_ORACLE_ERR_PRECONDITION;
        if (n > 0 && !row_is_valid(p, b, 0))
            return RL_ORACLE_ERR_PRECONDITION;
        if (p->seq_lens[b] > max_len)
            max_len = p->seq_lens[b];
    }
    const int64_t T = q_start[p->batch];
    int failed = 0;
#pragma omp parallel
    {
        double* scores = (double*)malloc(sizeof(double) * (size_t)max_len);
        if (scores == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < T * p->num_q_heads; ++r) {
            if (scores == NULL)
                continue;
            const int64_t row = r / p->num_q_heads;
            const int h = (int)(r % p->num_q_heads);
            int b = 0;
            while (q_start[b + 1] <= row)
                ++b;
            extend_one_row(p, q_start, row, b, h, scores, out + r * p->head_dim);
        }
        free(scores);
    }
    return failed ? RL_ORACLE_ERR_NOMEM : RL_ORACLE_OK;
}

/*
 * Round-to-nearest-even onto the OCP E4M3FN grid, from the format's
 * definition: 4 exponent bits with bias 7, 3 mantissa bits, subnormals
 * m/8 * 2^-6, largest finite 448.  Inputs are finite with |x| <= 448 (callers
 * clamp first); NaN encodes as 0x7F.  The sign of zero is kept.
 */
uint8_t rl_oracle_e4m3_encode(float x)
{
    if (x != x)
        return 0x7F;
    const uint8_t sign = signbit(x) ? 0x80 : 0x00;
    const double a = fabs((double)x);
    if (a < ldexp(1.0, -6)) {
        /* subnormal step 2^-9; rounding up to 8 steps yields code 0x08 = 2^-6 */
        const double steps = rint(a * 512.0);
        return sign | (uint8_t)steps;
    }
    int e = (int)floor(log2(a));
    if (ldexp(1.0, e) > a)  /* guard log2 rounding at exact powers of two */
        e -= 1;
    if (ldexp(1.0, e + 1) <= a)
        e += 1;
    double q = rint((a / ldexp(1.0, e) - 1.0) * 8.0);
    if (q == 8.0) {
        q = 0.0;
        e += 1;
    }
    return sign | (uint8_t)(((e + 7) << 3) | (int)q);
}

/* fp32 slab scale for a maximum magnitude: absmax / 448, or 1 for zero. */
static float slab_scale_for(float absmax)
{
    return absmax > 0.0f ? absmax / 448.0f : 1.0f;
}

static float clamp448(float v)
{
    return v > 448.0f ? 448.0f : (v < -448.0f ? -448.0f : v);
}

/*
 * Appends one token per (sequence, kv head) to a pool.  For bf16 pools the
 * token's bits are copied into page block_table[b][L/16], slot L%16
 * (L = seq_lens[b], the length before the append).  For e4m3 pools, in fp32:
 *   slot 0 (the page starts empty):  scale = absmax(token)/448 (1 if zero)
 *   later slots:  scale' = max(scale, absmax(token)/448); when it grows, every
 *     stored code c of the slab's earlier slots becomes
 *     e4m3(e4m3value(c) * (scale / scale'))
 *   the token:  e4m3(clamp(x / scale', +-448))
 * with e4m3() rounding to nearest even.  Sequences with L < 0 are skipped.
 */
int rl_oracle_kv_append(const rl_oracle_append* p)
{
    if (p == NULL || p->k_new == NULL || p->v_new == NULL || p->k_pool == NULL ||
        p->v_pool == NULL || p->block_table == NULL || p->seq_lens == NULL ||
        p->batch < 0 || p->num_kv_heads <= 0 || p->head_dim <= 0 || p->page_size <= 0 ||
        p->max_pages <= 0 || p->num_pages <= 0)
        return RL_ORACLE_ERR_ARG;
    const int fp8 = p->kv_dtype == RL_ORACLE_KV_FP8_E4M3;
    if (!fp8 && p->kv_dtype != RL_ORACLE_KV_BF16)
        return RL_ORACLE_ERR_ARG;
    if (p->layout != RL_ORACLE_LAYOUT_HND && p->layout != RL_ORACLE_LAYOUT_NHD)
        return RL_ORACLE_ERR_ARG;
    if (fp8 && (p->k_scale == NULL || p->v_scale == NULL))
        return RL_ORACLE_ERR_ARG;
    for (int b = 0; b < p->batch; ++b) {
        const int L = p->seq_lens[b];
        if (L < 0)
            continue;
        if ((int64_t)L >= (int64_t)p->max_pages * p->page_size)
            return RL_ORACLE_ERR_PRECONDITION;
        const int32_t page = p->block_table[(int64_t)b * p->max_pages + L / p->page_size];
        if (page < 0 || (int64_t)page >= p->num_pages)
            return RL_ORACLE_ERR_PRECONDITION;
    }
    const int D = p->head_dim, P = p->page_size, H = p->num_kv_heads;
    for (int b = 0; b < p->batch; ++b) {
        const int L = p->seq_lens[b];
        if (L < 0)
            continue;
        const int64_t page = p->block_table[(int64_t)b * p->max_pages + L / P];
        const int slot = L % P;
        for (int kvh = 0; kvh < H; ++kvh) {
            for (int which = 0; which < 2; ++which) {
                const uint16_t* src = (const uint16_t*)(which ? p->v_new : p->k_new) +
                                      ((int64_t)b * H + kvh) * D;
                const int64_t slab = page * H + kvh;
#define ELEM(sl, d) pool_index(p->layout, page, kvh, (sl), (d), H, P, D)
                if (!fp8) {
                    uint16_t* dst = (uint16_t*)(which ? p->v_pool : p->k_pool);
                    for (int d = 0; d < D; ++d)
                        dst[ELEM(slot, d)] = src[d];
                    continue;
                }
                uint8_t* codes = (uint8_t*)(which ? p->v_pool : p->k_pool);
                float* scale = (which ? p->v_scale : p->k_scale) + slab;
                float absmax = 0.0f;
                for (int d = 0; d < D; ++d) {
                    const float v = fabsf((float)rl_oracle_bf16_to_double(src[d]));
                    if (v > absmax)
                        absmax = v;
                }
                const float wanted = slab_scale_for(absmax);
                float s_new;
                if (slot == 0) {
                    s_new = wanted;
                } else {
                    const float s_old = *scale;
                    s_new = wanted > s_old ? wanted : s_old;
                    if (s_new != s_old) {
                        const float ratio = s_old / s_new;
                        for (int sl = 0; sl < slot; ++sl)
                            for (int d = 0; d < D; ++d) {
                                uint8_t* c = &codes[ELEM(sl, d)];
                                const float old = (float)rl_oracle_e4m3_to_double(*c);
                                *c = rl_oracle_e4m3_encode(old * ratio);
                            }
                    }
                }
                *scale = s_new;
                for (int d = 0; d < D; ++d) {
                    const float x = (float)rl_oracle_bf16_to_double(src[d]);
                    codes[ELEM(slot, d)] = rl_oracle_e4m3_encode(clamp448(x / s_new));
                }
#undef ELEM
            }
        }
    }
    return RL_ORACLE_OK;
}

int rl_oracle_max_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void rl_oracle_set_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}
