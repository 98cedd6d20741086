// rl_extend.hip -- extend (prefill) attention over the paged KV cache.

#include "rl_common.h"

using namespace rl_da;

namespace {

// ---------------------------------------------------- extend attention ---
//
// Causal attention of each sequence's n_b new tokens (already appended: the
// last n_b of its L_b cached tokens).  A work unit is one work-group of four
// wavefronts for (sequence b, kv head, tile of 64/G new tokens); wavefront w
// owns 16/G of the tile's tokens and all G query heads of the kv head: 16
// query rows, row m = (token m / G, head m % G).  Every K/V page the tile can
// see is loaded once into LDS for the four wavefronts (K as [token][dim], V
// transposed to [dim][token]); each wavefront then forms its 16x16 score tile
// with four v_mfma_f32_16x16x32_bf16 (as the decode kernel), applies the
// causal mask where a page crosses a query position, keeps an online softmax
// per row, and accumulates O += P V with v_mfma_f32_16x16x16_bf16 over eight
// 16-dim blocks.  P goes to the PV MFMA as two bf16 terms (hi + lo), so the
// value sum keeps fp32-level accuracy; l sums the same fp32 probabilities.

constexpr int kExtendRows = 16;                   // query rows per wavefront
constexpr int kKRowPad = 8;                       // bf16 elements of row padding
constexpr int kVtRow = kPageSize + 4;             // [dim][token] row, padded

struct ExtendArgs {
    const uint16_t* q;          // bf16 [T][Hq][D]
    const int32_t* q_start;     // [B+1]
    const uint8_t* k_pool;
    const uint8_t* v_pool;
    const int32_t* block_table;
    const int32_t* seq_lens;
    uint16_t* out;              // bf16 [T][Hq][D]
    int64_t page_bytes;         // pool strides in bytes: per page,
    int32_t head_bytes;         //   per kv head within a page,
    int32_t row_bytes;          //   per token slot within a slab
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t max_pages;
    int32_t num_tiles;          // ceil(max_q_per_seq / tile tokens)
    float scale_log2;
};

template <int G>
__global__ __launch_bounds__(kWave * kUnitWaves) void extend_bf16(ExtendArgs a)
{
    static_assert(G >= 1 && G <= 16 && 16 % G == 0, "16 rows per wavefront hold whole groups");
    constexpr int kTokPerWave = kExtendRows / G;
    constexpr int kTileTok = kUnitWaves * kTokPerWave;
    __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kPageSize][kHeadDim + kKRowPad];
    __shared__ __attribute__((aligned(16))) uint16_t vt_lds[2][kHeadDim][kVtRow];
    __shared__ __attribute__((aligned(16))) uint16_t p_lds[kUnitWaves][2][kExtendRows][kVtRow];

    const int tile = blockIdx.x % a.num_tiles;
    const int bk = blockIdx.x / a.num_tiles;
    const int kvh = bk % a.num_kv_heads;
    const int b = bk / a.num_kv_heads;
    const int q0 = a.q_start[b];
    // lengths clamped to what the table row can hold, new tokens to the length
    const int L = min(a.seq_lens[b], a.max_pages * kPageSize);
    const int n_new = min(a.q_start[b + 1] - q0, L);
    const int tok0 = tile * kTileTok;
    if (tok0 >= n_new)
        return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int n = lane & 15, kg = lane >> 4;
    const int h0 = kvh * G;
    const int base_pos = L - n_new;  // position of new token 0

    // Query operand rows: lane holds row m = lane % 16 for the MFMA A operand.
    uint4 qa[4];
    {
        const int m = lane & 15;
        const int qi = tok0 + wave * kTokPerWave + m / G;
        const bool real = qi < n_new;
        const uint16_t* qrow =
            a.q + ((int64_t)(q0 + (real ? qi : 0)) * a.num_q_heads + h0 + m % G) * kHeadDim;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            qa[i] = real ? *reinterpret_cast<const uint4*>(qrow + 32 * i + 8 * kg)
                         : make_uint4(0, 0, 0, 0);
    }
    // Rows this lane holds in the C layout: m = 4kg + j.
    int row_pos[4];
    bool row_real[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int m = 4 * kg + j;
        const int qi = tok0 + wave * kTokPerWave + m / G;
        row_real[j] = qi < n_new;
        row_pos[j] = base_pos + qi;
    }
    const int tile_last = min(tok0 + kTileTok, n_new) - 1;
    const int npages = (base_pos + tile_last) / kPageSize + 1;  // pages the tile sees
    const int first_masked_page = (base_pos + tok0) / kPageSize;

    float m_run[4], lsum[4];
    floatx4_t o[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        m_run[j] = -INFINITY;
        lsum[j] = 0.0f;
    }
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
        o[nb] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // Staging: thread t moves 16 bytes of K and of V: token t/16, dims 8(t%16)..+8.
    const int st_tok = threadIdx.x / 16, st_dim = (threadIdx.x % 16) * 8;
    const int32_t* bt = a.block_table + (int64_t)b * a.max_pages;
    const int64_t st_off = (int64_t)kvh * a.head_bytes + st_tok * a.row_bytes + 2 * st_dim;
    auto fetch = [&](int j, uint4& kr, uint4& vr) {
        const int64_t off = bt[j] * a.page_bytes + st_off;
        kr = load_stream16(a.k_pool + off);
        vr = load_stream16(a.v_pool + off);
    };
    uint4 kr, vr;
    fetch(0, kr, vr);

    for (int j = 0; j < npages; ++j) {
        const int buf = j & 1;
        // slots past the sequence end may hold NaN: they must not reach P.V
        if (j * kPageSize + st_tok >= L) {
            kr = make_uint4(0, 0, 0, 0);
            vr = make_uint4(0, 0, 0, 0);
        }
        *reinterpret_cast<uint4*>(&k_lds[buf][st_tok][st_dim]) = kr;
        {
            const uint32_t w[4] = {vr.x, vr.y, vr.z, vr.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                vt_lds[buf][st_dim + 2 * e][st_tok] = (uint16_t)(w[e] & 0xffffu);
                vt_lds[buf][st_dim + 2 * e + 1][st_tok] = (uint16_t)(w[e] >> 16);
            }
        }
        if (j + 1 < npages)
            fetch(j + 1, kr, vr);
        __syncthreads();

        // scores S[row 4kg+jj][token n]
        floatx4_t sacc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint4 kb = *reinterpret_cast<const uint4*>(&k_lds[buf][n][32 * i + 8 * kg]);
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, qa[i]), __builtin_bit_cast(bf16x8_t, kb), sacc,
                0, 0, 0);
        }
        const int key = j * kPageSize + n;
        float s[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            float x = sacc[jj] * a.scale_log2;
            if (j >= first_masked_page)
                x = key <= row_pos[jj] ? x : -INFINITY;
            s[jj] = row_real[jj] ? x : 0.0f;  // rows past the tile's tokens stay finite
        }
        float mx[4];
        bool grow_any = false;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            mx[jj] = row16_max(s[jj]);   // finite: key 0 is visible to every row
            grow_any |= mx[jj] > m_run[jj] + kMaxSlack;
        }
        if (__any(grow_any)) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const float m_new = mx[jj] > m_run[jj] + kMaxSlack ? mx[jj] : m_run[jj];
                const float alpha = exp2_fast(m_run[jj] - m_new);
                m_run[jj] = m_new;
                lsum[jj] *= alpha;
#pragma unroll
                for (int nb = 0; nb < 8; ++nb)
                    o[nb][jj] *= alpha;
            }
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const float p = exp2_fast(s[jj] - m_run[jj]);
            lsum[jj] += p;
            const uint32_t hi = f32_to_bf16(p);
            const float rest = p - __uint_as_float(hi << 16);
            p_lds[wave][0][4 * kg + jj][n] = (uint16_t)hi;
            p_lds[wave][1][4 * kg + jj][n] = (uint16_t)f32_to_bf16(rest);
        }
        wave_lds_sync();
        const uint2 ph = *reinterpret_cast<const uint2*>(&p_lds[wave][0][n][4 * kg]);
        const uint2 pl = *reinterpret_cast<const uint2*>(&p_lds[wave][1][n][4 * kg]);
        wave_lds_sync();
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
            const uint2 vb = *reinterpret_cast<const uint2*>(&vt_lds[buf][16 * nb + n][4 * kg]);
            o[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
                __builtin_bit_cast(bf16x4_t, ph), __builtin_bit_cast(bf16x4_t, vb), o[nb], 0, 0, 0);
            o[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
                __builtin_bit_cast(bf16x4_t, pl), __builtin_bit_cast(bf16x4_t, vb), o[nb], 0, 0, 0);
        }
    }

    // out[row] = O[row] / l[row]; lane holds rows 4kg+jj, dims 16nb + n.
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
        const float l = row16_sum(lsum[jj]);
        if (!row_real[jj])
            continue;
        const int m = 4 * kg + jj;
        const int qi = tok0 + wave * kTokPerWave + m / G;
        uint16_t* orow = a.out + ((int64_t)(q0 + qi) * a.num_q_heads + h0 + m % G) * kHeadDim;
        const float inv = 1.0f / l;
#pragma unroll
        for (int nb = 0; nb < 8; ++nb)
            orow[16 * nb + n] = (uint16_t)f32_to_bf16(o[nb][jj] * inv);
    }
}

}  // namespace

extern "C" {

rl_da_status rl_extend_attn(const void* q, const int32_t* q_start, int32_t max_q_per_seq,
                            const void* k_pool, const void* v_pool, const float* k_scale,
                            const float* v_scale, int64_t num_pages, const int32_t* block_table,
                            int32_t max_pages, const int32_t* seq_lens, int32_t batch,
                            int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                            int32_t page_size, int32_t kv_dtype, int32_t layout, float scale,
                            void* out, void* stream)
{
    if (q == nullptr || q_start == nullptr || k_pool == nullptr || v_pool == nullptr ||
        block_table == nullptr || seq_lens == nullptr || out == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    if (batch < 0 || max_q_per_seq < 0 || num_q_heads <= 0 || num_kv_heads <= 0 ||
        num_q_heads % num_kv_heads != 0 || max_pages < 1 || num_pages < 1 || !isfinite(scale))
        return RL_DA_ERR_INVALID_ARG;
    if (kv_dtype != RL_DA_KV_BF16 && kv_dtype != RL_DA_KV_FP8_E4M3)
        return RL_DA_ERR_INVALID_ARG;
    if ((k_scale != nullptr) != (kv_dtype == RL_DA_KV_FP8_E4M3) ||
        (v_scale != nullptr) != (kv_dtype == RL_DA_KV_FP8_E4M3))
        return RL_DA_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
        return RL_DA_ERR_INVALID_ARG;
    PoolStrides ps;
    if (!pool_strides(layout, num_kv_heads, 2, &ps))
        return RL_DA_ERR_INVALID_ARG;
    const int G = num_q_heads / num_kv_heads;
    if (head_dim != kHeadDim || page_size != kPageSize || kv_dtype != RL_DA_KV_BF16 ||
        (G != 1 && G != 2 && G != 4 && G != 8 && G != 16))
        return RL_DA_ERR_UNSUPPORTED;
    if (batch == 0 || max_q_per_seq == 0)
        return RL_DA_OK;
    const int tile_tok = kUnitWaves * kExtendRows / G;
    ExtendArgs ea;
    ea.q = (const uint16_t*)q;
    ea.q_start = q_start;
    ea.k_pool = (const uint8_t*)k_pool;
    ea.v_pool = (const uint8_t*)v_pool;
    ea.block_table = block_table;
    ea.seq_lens = seq_lens;
    ea.out = (uint16_t*)out;
    ea.page_bytes = ps.page;
    ea.head_bytes = ps.head;
    ea.row_bytes = ps.row;
    ea.num_q_heads = num_q_heads;
    ea.num_kv_heads = num_kv_heads;
    ea.max_pages = max_pages;
    ea.num_tiles = (max_q_per_seq + tile_tok - 1) / tile_tok;
    ea.scale_log2 = scale * kLog2e;
    const int64_t blocks = (int64_t)batch * num_kv_heads * ea.num_tiles;
    if (blocks > INT32_MAX)
        return RL_DA_ERR_UNSUPPORTED;
    hipStream_t st = (hipStream_t)stream;
    const dim3 grid((unsigned)blocks), block(kWave * kUnitWaves);
    switch (G) {
    case 1: hipLaunchKernelGGL(extend_bf16<1>, grid, block, 0, st, ea); break;
    case 2: hipLaunchKernelGGL(extend_bf16<2>, grid, block, 0, st, ea); break;
    case 4: hipLaunchKernelGGL(extend_bf16<4>, grid, block, 0, st, ea); break;
    case 8: hipLaunchKernelGGL(extend_bf16<8>, grid, block, 0, st, ea); break;
    default: hipLaunchKernelGGL(extend_bf16<16>, grid, block, 0, st, ea); break;
    }
    return hipGetLastError() == hipSuccess ? RL_DA_OK : RL_DA_ERR_HIP;
}

}  // extern "C"
