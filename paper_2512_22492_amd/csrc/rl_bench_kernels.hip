// rl_bench_kernels.hip -- measurement-only kernels for the decode-attention
// benchmark (not part of the attention path).
//
//   rl_bench_copy         plain 16-byte-per-lane copy of a known byte count; its
//                         FETCH_SIZE / WRITE_SIZE readings calibrate the HBM
//                         traffic counters.
//   rl_bench_stream_read  contiguous read of a buffer, one contiguous share per
//                         work-group: the achievable HBM read bandwidth.
//   rl_bench_page_read    reads exactly the K/V bytes one decode step reads, with
//                         the split-K attention kernel's per-lane non-temporal
//                         load pattern (head-major slabs) and no arithmetic,
//                         the step's pages divided evenly over the work-groups
//                         (four wavefronts per (64 consecutive pages of the
//                         batch, kv head), kv heads adjacent): the ceiling of
//                         that access pattern.
//
// All pointers are device pointers owned by the caller.  Each function
// enqueues one kernel on `stream` and returns 0, or -1 on bad arguments, or the
// HIP error code of the launch.

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;
constexpr int kUnitWaves = 4;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream16(const uint8_t* p)
{
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__global__ __launch_bounds__(kBlock) void copy_kernel(uint4* __restrict__ dst,
                                                      const uint4* __restrict__ src, size_t n)
{
    const size_t stride = (size_t)gridDim.x * kBlock;
    for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
}

// Each work-group reads its own contiguous share of the buffer with
// non-temporal 16-byte loads, four in flight per lane (the fastest read
// pattern measured on this GPU).
__global__ __launch_bounds__(kBlock) void stream_read_kernel(const uint4* __restrict__ src,
                                                             size_t n, uint32_t* sink)
{
    const size_t per = (n + gridDim.x - 1) / gridDim.x;
    const size_t b0 = (size_t)blockIdx.x * per;
    const size_t b1 = b0 + per < n ? b0 + per : n;
    const uint8_t* base = reinterpret_cast<const uint8_t*>(src);
    uint32_t acc = 0;
    size_t i = b0 + threadIdx.x;
    for (; i + 3 * kBlock < b1; i += 4 * kBlock) {
        const uint4 a = load_stream16(base + 16 * i);
        const uint4 b = load_stream16(base + 16 * (i + kBlock));
        const uint4 c = load_stream16(base + 16 * (i + 2 * kBlock));
        const uint4 d = load_stream16(base + 16 * (i + 3 * kBlock));
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^
               d.y ^ d.z ^ d.w;
    }
    for (; i < b1; i += kBlock) {
        const uint4 a = load_stream16(base + 16 * i);
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    // one value per thread keeps every load live; the sink holds grid*block words
    sink[(size_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

struct PageReadArgs {
    const uint8_t* k_pool;
    const uint8_t* v_pool;
    const int32_t* block_table;
    const int32_t* page_prefix;  // [batch + 1]: pages of the sequences before b
    uint32_t* sink;
    int64_t total_pages;         // page_prefix[batch]
    int32_t num_kv_heads;
    int32_t max_pages;
    int32_t batch;
    int32_t unit_pages;
    int32_t slab_bytes;          // 4096 (bf16) or 2048 (e4m3)
};

__global__ __launch_bounds__(64 * kUnitWaves) void page_read_kernel(PageReadArgs a)
{
    const int kvh = blockIdx.x % a.num_kv_heads;
    const int64_t i0 = (int64_t)(blockIdx.x / a.num_kv_heads) * a.unit_pages;
    const int64_t i1 = min(i0 + (int64_t)a.unit_pages, a.total_pages);
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    int64_t i = i0 + wave;
    // sequence of page i: page_prefix[b] <= i < page_prefix[b + 1]
    int b = 0;
    if (i < i1) {
        int hi = a.batch;  // page_prefix[hi] = total_pages > i
        while (hi - b > 1) {
            const int mid = (b + hi) >> 1;
            if (a.page_prefix[mid] <= i)
                b = mid;
            else
                hi = mid;
        }
    }
    uint32_t acc = 0;
    const int koff = (lane & 15) * 256 + 16 * (lane >> 4);
    const int voff = lane * 16;
    for (; i < i1; i += kUnitWaves) {
        while (a.page_prefix[b + 1] <= i)  // ends: page_prefix[batch] > i
            ++b;
        const int j = (int)(i - a.page_prefix[b]);
        const int64_t page = a.block_table[(int64_t)b * a.max_pages + j];
        const int64_t slab = (page * a.num_kv_heads + kvh) * a.slab_bytes;
        if (a.slab_bytes == 4096) {
            uint4 k[4], v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                k[r] = load_stream16(a.k_pool + slab + koff + 64 * r);
                v[r] = load_stream16(a.v_pool + slab + voff + 1024 * r);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r)
                acc ^= k[r].x ^ k[r].y ^ k[r].z ^ k[r].w ^ v[r].x ^ v[r].y ^ v[r].z ^ v[r].w;
        } else {
            // e4m3 slabs: K and V both as whole 128-byte rows, eight per
            // instruction, as the decode kernel reads them
            uint4 k[2], v[2];
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                k[r] = load_stream16(a.k_pool + slab + voff + 1024 * r);
                v[r] = load_stream16(a.v_pool + slab + voff + 1024 * r);
            }
#pragma unroll
            for (int r = 0; r < 2; ++r)
                acc ^= k[r].x ^ k[r].y ^ k[r].z ^ k[r].w ^ v[r].x ^ v[r].y ^ v[r].z ^ v[r].w;
        }
    }
    a.sink[(size_t)blockIdx.x * 64 * kUnitWaves + threadIdx.x] = acc;
}

}  // namespace

extern "C" {

int rl_bench_copy(void* dst, const void* src, size_t bytes, void* stream)
{
    if (dst == nullptr || src == nullptr || bytes % 16 != 0)
        return -1;
    const size_t n = bytes / 16;
    const unsigned grid = 256 * 32;
    hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kBlock), 0, (hipStream_t)stream,
                       (uint4*)dst, (const uint4*)src, n);
    return (int)hipGetLastError();
}

// sink must hold grid_blocks * 256 uint32 words.
int rl_bench_stream_read(const void* src, size_t bytes, uint32_t* sink, int grid_blocks,
                         void* stream)
{
    if (src == nullptr || sink == nullptr || bytes % 16 != 0 || grid_blocks <= 0)
        return -1;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)grid_blocks), dim3(kBlock), 0,
                       (hipStream_t)stream, (const uint4*)src, bytes / 16, sink);
    return (int)hipGetLastError();
}

// Pools [P][Hkv][16][128] of 2-byte (slab_bytes 4096) or 1-byte (2048)
// elements; block_table [batch][max_pages].
// page_prefix: device int32 [batch + 1], page_prefix[b] = pages of sequences
// 0 .. b-1 (each sequence's ceil(min(len, 16 * max_pages) / 16)); total_pages
// = page_prefix[batch].  sink: grid * 256 words, grid = num_kv_heads *
// ceil(total_pages / unit_pages).
int rl_bench_page_read(const void* k_pool, const void* v_pool, const int32_t* block_table,
                       int32_t max_pages, const int32_t* page_prefix, int64_t total_pages,
                       int32_t batch, int32_t num_kv_heads, int32_t unit_pages,
                       int32_t slab_bytes, uint32_t* sink, void* stream)
{
    if (k_pool == nullptr || v_pool == nullptr || block_table == nullptr ||
        page_prefix == nullptr || sink == nullptr || batch <= 0 || num_kv_heads <= 0 ||
        max_pages <= 0 || unit_pages <= 0 || total_pages < 0 ||
        (slab_bytes != 4096 && slab_bytes != 2048))
        return -1;
    if (total_pages == 0)
        return 0;
    PageReadArgs a;
    a.k_pool = (const uint8_t*)k_pool;
    a.v_pool = (const uint8_t*)v_pool;
    a.block_table = block_table;
    a.page_prefix = page_prefix;
    a.sink = sink;
    a.total_pages = total_pages;
    a.num_kv_heads = num_kv_heads;
    a.max_pages = max_pages;
    a.batch = batch;
    a.unit_pages = unit_pages;
    a.slab_bytes = slab_bytes;
    const int64_t units = (int64_t)num_kv_heads * ((total_pages + unit_pages - 1) / unit_pages);
    hipLaunchKernelGGL(page_read_kernel, dim3((unsigned)units), dim3(64 * kUnitWaves), 0,
                       (hipStream_t)stream, a);
    return (int)hipGetLastError();
}

}  // extern "C"
