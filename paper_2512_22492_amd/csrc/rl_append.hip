// rl_append.hip -- KV-cache append (bf16 copy, e4m3 with growing slab scales).

#include "rl_common.h"

using namespace rl_da;

namespace {

// --------------------------------------------------------- KV append ---
//
// One work-group of two wavefronts per (sequence, kv head): wavefront 0 appends
// the key, wavefront 1 the value.  Lane l owns dims 2l and 2l+1.

struct AppendArgs {
    const uint16_t* k_new;      // bf16 bits [B][Hkv][D]
    const uint16_t* v_new;
    uint8_t* k_pool;
    uint8_t* v_pool;
    float* k_scale;
    float* v_scale;
    const int32_t* block_table;
    const int32_t* seq_lens;
    int32_t* dev_error;         // may be null
    int64_t num_pages;
    int64_t page_bytes;         // pool strides in bytes: per page,
    int32_t head_bytes;         //   per kv head within a page,
    int32_t row_bytes;          //   per token slot within a slab
    int32_t num_kv_heads;
    int32_t max_pages;
};

__device__ __forceinline__ float wave_max(float v)
{
    v = row16_max(v);
    v = fmaxf(v, __shfl_xor(v, 16));
    v = fmaxf(v, __shfl_xor(v, 32));
    return v;
}

// Two fp32 values to two e4m3 codes (round to nearest even) in the low 16 bits.
__device__ __forceinline__ uint32_t e4m3_pair(float a, float b)
{
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false) & 0xffffu;
}

__device__ __forceinline__ float clamp448(float v)
{
    // comparisons, not fminf/fmaxf, so that a NaN passes through unchanged
    return v > 448.0f ? 448.0f : (v < -448.0f ? -448.0f : v);
}

template <bool FP8>
__global__ __launch_bounds__(2 * kWave) void kv_append_kernel(AppendArgs a)
{
    const int b = blockIdx.x / a.num_kv_heads;
    const int kvh = blockIdx.x % a.num_kv_heads;
    const int which = threadIdx.x / kWave;  // 0: key, 1: value
    const int lane = threadIdx.x % kWave;
    const int L = a.seq_lens[b];
    if (L < 0)
        return;
    if (L >= a.max_pages * kPageSize) {
        if (a.dev_error != nullptr && threadIdx.x == 0 && kvh == 0)
            atomicOr(a.dev_error, RL_DA_DEVERR_LENGTH_TOO_LONG);
        return;
    }
    const int32_t page = a.block_table[(int64_t)b * a.max_pages + L / kPageSize];
    if (page < 0 || (int64_t)page >= a.num_pages) {
        if (a.dev_error != nullptr && threadIdx.x == 0)
            atomicOr(a.dev_error, RL_DA_DEVERR_PAGE_OUT_OF_RANGE);
        return;
    }
    const int slot = L % kPageSize;
    const int64_t slab = (int64_t)page * a.num_kv_heads + kvh;
    const uint16_t* src = (which ? a.v_new : a.k_new) + ((int64_t)b * a.num_kv_heads + kvh) * kHeadDim;
    const uint32_t bits = *reinterpret_cast<const uint32_t*>(src + 2 * lane);
    // token slot 0 of slab (page, kvh); slot j is j * row_bytes further
    uint8_t* codes = (which ? a.v_pool : a.k_pool) + page * a.page_bytes +
                     (int64_t)kvh * a.head_bytes;
    if (!FP8) {
        *reinterpret_cast<uint32_t*>(codes + slot * a.row_bytes + 4 * lane) = bits;
        return;
    }
    const float x0 = bf16_lo(bits), x1 = bf16_hi(bits);
    const float absmax = wave_max(fmaxf(fabsf(x0), fabsf(x1)));
    const float wanted = absmax > 0.0f ? absmax / 448.0f : 1.0f;
    float* scale = (which ? a.v_scale : a.k_scale) + slab;
    float s_new = wanted;
    if (slot != 0) {
        const float s_old = *scale;
        s_new = wanted > s_old ? wanted : s_old;
        if (s_new != s_old) {
            // re-encode the slab's earlier slots at the grown scale
            const float ratio = s_old / s_new;
            constexpr int kWordsPerRow = kHeadDim / 4;
            for (int w = lane; w < slot * kWordsPerRow; w += kWave) {
                uint32_t* word = reinterpret_cast<uint32_t*>(
                    codes + (w / kWordsPerRow) * a.row_bytes + 4 * (w % kWordsPerRow));
                const uint32_t c = *word;
                const floatx2_t lo = __builtin_amdgcn_cvt_pk_f32_fp8(c, false);
                const floatx2_t hi = __builtin_amdgcn_cvt_pk_f32_fp8(c, true);
                *word = e4m3_pair(lo.x * ratio, lo.y * ratio) |
                        (e4m3_pair(hi.x * ratio, hi.y * ratio) << 16);
            }
        }
    }
    const uint32_t pair = e4m3_pair(clamp448(x0 / s_new), clamp448(x1 / s_new));
    *reinterpret_cast<uint16_t*>(codes + slot * a.row_bytes + 2 * lane) = (uint16_t)pair;
    if (lane == 0)
        *scale = s_new;
}

}  // namespace

extern "C" {

rl_da_status rl_kv_append(const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                          float* k_scale, float* v_scale, int64_t num_pages,
                          const int32_t* block_table, int32_t max_pages,
                          const int32_t* seq_lens, int32_t batch, int32_t num_kv_heads,
                          int32_t head_dim, int32_t page_size, int32_t kv_dtype,
                          int32_t layout, int32_t* device_error, void* stream)
{
    if (k_new == nullptr || v_new == nullptr || k_pool == nullptr || v_pool == nullptr ||
        block_table == nullptr || seq_lens == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    if (batch < 0 || num_kv_heads <= 0 || max_pages < 1 || num_pages < 1)
        return RL_DA_ERR_INVALID_ARG;
    if (kv_dtype != RL_DA_KV_BF16 && kv_dtype != RL_DA_KV_FP8_E4M3)
        return RL_DA_ERR_INVALID_ARG;
    if (head_dim != kHeadDim || page_size != kPageSize)
        return RL_DA_ERR_UNSUPPORTED;
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool))
        return RL_DA_ERR_INVALID_ARG;
    const bool fp8 = kv_dtype == RL_DA_KV_FP8_E4M3;
    if (fp8 != (k_scale != nullptr) || fp8 != (v_scale != nullptr))
        return RL_DA_ERR_INVALID_ARG;
    if (!pools_paired(layout, k_pool, v_pool, fp8 ? 1 : 2))
        return RL_DA_ERR_INVALID_ARG;
    PoolStrides ps;
    if (!pool_strides(layout, num_kv_heads, fp8 ? 1 : 2, &ps))
        return RL_DA_ERR_INVALID_ARG;
    if (batch == 0)
        return RL_DA_OK;
    const int64_t blocks = (int64_t)batch * num_kv_heads;
    if (blocks > INT32_MAX)
        return RL_DA_ERR_UNSUPPORTED;
    AppendArgs aa;
    aa.k_new = (const uint16_t*)k_new;
    aa.v_new = (const uint16_t*)v_new;
    aa.k_pool = (uint8_t*)k_pool;
    aa.v_pool = (uint8_t*)v_pool;
    aa.k_scale = k_scale;
    aa.v_scale = v_scale;
    aa.block_table = block_table;
    aa.seq_lens = seq_lens;
    aa.dev_error = device_error;
    aa.num_pages = num_pages;
    aa.page_bytes = ps.page;
    aa.head_bytes = ps.head;
    aa.row_bytes = ps.row;
    aa.num_kv_heads = num_kv_heads;
    aa.max_pages = max_pages;
    hipStream_t st = (hipStream_t)stream;
    if (fp8)
        hipLaunchKernelGGL(kv_append_kernel<true>, dim3((unsigned)blocks), dim3(2 * kWave), 0,
                           st, aa);
    else
        hipLaunchKernelGGL(kv_append_kernel<false>, dim3((unsigned)blocks), dim3(2 * kWave), 0,
                           st, aa);
    return hipGetLastError() == hipSuccess ? RL_DA_OK : RL_DA_ERR_HIP;
}

}  // extern "C"
