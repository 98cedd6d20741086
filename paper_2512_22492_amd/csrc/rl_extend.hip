// rl_extend.hip -- extend (prefill) attention over the paged KV cache.

#include <type_traits>

#include "rl_common.h"

using namespace rl_da;

namespace {

// ---------------------------------------------------- extend attention ---
//
// Causal attention of each sequence's n_b new tokens (already appended: the
// last n_b of its L_b cached tokens).  A work unit is one work-group of four
// wavefronts for (sequence b, kv head, tile of 128/G new tokens): 128 query
// rows, row r = (token r / G, head r % G); wavefront w owns rows 32w..32w+31 as
// two blocks of 16.  The keys the tile can see pass through LDS 64 at a time
// (four pages, K and V both as [key][dim] rows), double-buffered with one
// barrier per stage; the next stage's loads are in flight during the current
// stage's products.  bf16 pages go from global memory straight into LDS
// (direct loads, four whole key rows per instruction); e4m3 pages are
// widened to bf16 through registers.
//
// Both products run transposed so that every lane keeps one query row from
// the scores to the output.  S^T = K Q^T (v_mfma_f32_16x16x32_bf16, A = 16
// keys x 32 dims from LDS, B = Q^T held in registers) leaves lane l with row
// l%16 and keys 4(l/16)+j of each 16-key block; O^T += V^T P^T (same MFMA,
// 32 keys) takes P^T straight from those registers, with the k index of the
// product running over keys in the order (4g..4g+3, 16+4g..16+4g+3) for lane
// group g; the V^T operand in that order comes from the [key][dim] rows by
// the LDS transpose read.  Row max, rescale and sum are therefore lane-local
// but for two lane swaps per 64 keys.  P enters the PV product rounded to bf16
// (relative error at most 2^-8 per weight: 8 significant bits, round to
// nearest, as in common flash-attention kernels; an earlier two-term hi + lo
// split kept fp32-level accuracy at a third more MFMAs and conversion work).
// For bf16 pools l is the sum of the same rounded weights, taken by the PV
// product against a block of ones, so the output is a convex combination of
// the values with weights within 2^-7 relative of the exact ones; for e4m3
// pools (whose packed weights carry the page's v_scale) l sums the unrounded
// fp32 probabilities.
//
// Work-group order: consecutive work-groups go to the eight XCDs in turn,
// and the tiles of one (sequence, kv head) read the same keys, so they are
// placed on one XCD (one L2) -- see the unit mapping in the kernel.  The
// sequences are taken longest first (by length class), and each pair's
// tiles last tile first, so that the longest tiles do not start last and
// set the end of the launch.

constexpr int kRowBlocks = 2;                      // 16-row blocks per wavefront
constexpr int kTileRows = kUnitWaves * kRowBlocks * 16;
constexpr int kStageKeys = 64;                     // keys per LDS stage (4 pages)
constexpr int kStagePages = kStageKeys / kPageSize;
// K and V stage tiles are [key][dim] rows of 256 bytes whose sixteen 16-byte
// chunks are stored at position chunk ^ chunk_swizzle(row); every four rows
// stay one contiguous kilobyte (what a wavefront's direct global-to-LDS load
// fills).  The swizzle keeps both operand reads free of bank conflicts, as
// measured with the LDS counters on gfx950 (64 banks of 4 bytes):
// ds_read_b128 serves its 64 lanes sixteen at a time, lanes l and l ^ 1,
// l ^ 2, l ^ 20, l ^ 24 (and their combinations) together, so the K operand
// reads (lane 16g + i: row i, chunk (4ks + g) ^ swizzle(i)) need swizzle(r ^
// d) != swizzle(r) ^ (the g difference) for those lane pairs -- rows r and
// r ^ 8 in particular, which the XOR with (row & 8) separates (without it
// the reads were 2-way conflicted); ds_read_b64_tr_b16 serves 32 lanes at a
// time, so the transposed V reads (eight consecutive rows, two adjacent
// chunks each) need swizzle(row) >> 1 distinct over eight consecutive rows.
__device__ __forceinline__ int chunk_swizzle(int row)
{
    return (((row & 7) << 1) | ((row >> 3) & 1)) ^ (row & 8);
}

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4_t;

// Four bf16 of one dim from four consecutive key rows of a [key][dim] LDS
// tile (ds_read_b64_tr_b16).  Within each 16-lane group, lane j receives
// element j % 4 of the 8-byte chunks addressed by lanes j / 4 + 4e, e = 0..3:
// when lane s addresses row (base + s / 4), dims (d0 + 4 (s % 4)) .. +3, lane
// j gets rows base .. base + 3 of dim d0 + j.
__device__ __forceinline__ uint2 lds_read_transposed(const uint16_t* p)
{
    const short4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_t*)p);
    return __builtin_bit_cast(uint2, v);
}

// A lane's value and that of lane l ^ 16 (permlane16_swap exchanges 16-lane
// rows 1 <-> 0 and 3 <-> 2 between its two operands: with both equal to v,
// lane l receives v of lanes l & ~16 and l | 16), or of lane l ^ 32
// (permlane32_swap, the two halves).  Vector-ALU operations, no LDS round
// trip.  The maxima are IEEE `maximum` (no canonicalising copies of the
// operands); the row maxima they combine are finite or -inf.
__device__ __forceinline__ float max_lanes_xor16(float v)
{
    const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
    return __builtin_elementwise_maximum(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float max_lanes_xor32(float v)
{
    const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
    return __builtin_elementwise_maximum(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float sum_lanes_xor16(float v)
{
    const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
    return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}
__device__ __forceinline__ float sum_lanes_xor32(float v)
{
    const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
    return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// Length classes for the work-group order, longest first: class 0 holds
// lengths of 2^15 and more, class c lengths in [2^(15-c), 2^(16-c)), class 7
// everything below 2^9.
constexpr int kLengthClasses = 8;
__device__ __forceinline__ int length_class(int L)
{
    const int lg = 31 - __builtin_clz((unsigned)max(L, 1));
    return min(max(15 - lg, 0), kLengthClasses - 1);
}

// The sequence at place `rank` of the batch in longest-first order (length
// classes descending, sequence order within a class).  Every work-group
// derives the same order from the lengths (the counts do not depend on the
// order of the LDS atomics); called by all threads of the work-group.
// `classes` is LDS scratch of `capacity` bytes that keeps each sequence's
// class between the two passes (larger batches read the lengths again).
__device__ int sequence_at_rank(const int32_t* seq_lens, int cap, int batch, int rank,
                                uint8_t* classes, int capacity)
{
    __shared__ int count[kLengthClasses];
    __shared__ int wave_hits[kUnitWaves];
    __shared__ int pick;
    const int t = threadIdx.x, lane = t % kWave, w = t / kWave;
    if (t < kLengthClasses)
        count[t] = 0;
    __syncthreads();
    for (int i = t; i < batch; i += kWave * kUnitWaves) {
        const int cl = length_class(min(seq_lens[i], cap));
        if (i < capacity)
            classes[i] = (uint8_t)cl;
        atomicAdd(&count[cl], 1);
    }
    __syncthreads();
    int c = 0, k = rank;  // rank < batch, so some class holds it
    while (c < kLengthClasses - 1 && k >= count[c])
        k -= count[c++];
    if (count[c] == batch)  // one class: sequence order
        return rank;
    // the k-th sequence of class c, one chunk of 256 sequences at a time
    for (int base = 0; base < batch; base += kWave * kUnitWaves) {
        const int i = base + t;
        const bool hit =
            i < batch &&
            (i < capacity ? (int)classes[i] : length_class(min(seq_lens[i], cap))) == c;
        const uint64_t m = __ballot(hit);
        if (lane == 0)
            wave_hits[w] = __popcll(m);
        __syncthreads();
        int before = 0, total = 0;
#pragma unroll
        for (int v = 0; v < kUnitWaves; ++v) {
            before += v < w ? wave_hits[v] : 0;
            total += wave_hits[v];
        }
        if (hit && before + __popcll(m & ((1ull << lane) - 1)) == k)
            pick = i;
        __syncthreads();
        if (k < total)
            break;
        k -= total;
    }
    return pick;
}

// A direct global-to-LDS load of 16 bytes per lane, from a per-lane global
// address to LDS address lds + 16 * lane (lds uniform, in M0), written as
// inline assembly so that the compiler neither tracks these loads nor waits
// for them: the kernel waits for its own loads before each stage barrier,
// and the compiler, not knowing which LDS buffer a load fills, would
// otherwise wait for it before every read of the other buffer.  (The nop is
// the wait state between the M0 write and the load that reads it.)
__device__ __forceinline__ void dma16(const uint8_t* gaddr, uint32_t lds)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gaddr), "{m0}"(lds)
                 : "memory");
}

struct ExtendArgs {
    const uint16_t* q;          // bf16 [T][Hq][D]
    const int32_t* q_start;     // [B+1]
    const uint8_t* k_pool;
    const uint8_t* v_pool;
    const float* k_scale;       // [P][Hkv], e4m3 pools only
    const float* v_scale;
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
    float scale_log2;           // |scale| * log2(e)
    uint32_t q_sign;            // 0x80008000 for a negative scale: Q enters negated
};

// FP8: e4m3 pools.  Codes are staged as exact bf16 (scale 1); a page's
// k_scale multiplies its keys' scores and its v_scale the probabilities that
// weight its values (l sums the unscaled probabilities), as in decode.
template <int G, bool FP8>
__global__ __launch_bounds__(kWave * kUnitWaves)
__attribute__((amdgpu_waves_per_eu(2))) void extend_attn(ExtendArgs a)
{
    static_assert(G >= 1 && G <= 16 && 16 % G == 0, "16-row blocks hold whole groups");
    constexpr int kTileTok = kTileRows / G;
    // Two stage buffers per operand: stage j in buffer j % 2.
    __shared__ __attribute__((aligned(16))) uint16_t k_lds0[kStageKeys][kHeadDim];
    __shared__ __attribute__((aligned(16))) uint16_t k_lds1[kStageKeys][kHeadDim];
    __shared__ __attribute__((aligned(16))) uint16_t v_lds0[kStageKeys][kHeadDim];
    __shared__ __attribute__((aligned(16))) uint16_t v_lds1[kStageKeys][kHeadDim];
    // e4m3 pools: (k_scale, v_scale) of the stage's four pages
    __shared__ __attribute__((aligned(16))) float2 scale_lds[2][kStagePages];
    typedef uint16_t Tile[kStageKeys][kHeadDim];
    auto k_tile = [&](int sel) -> Tile& { return sel ? k_lds1 : k_lds0; };
    auto v_tile = [&](int sel) -> Tile& { return sel ? v_lds1 : v_lds0; };

    // Work-group g runs on XCD g % 8.  Pairs (sequence, kv head) are dealt
    // to the XCDs in turn, pair p to XCD p % 8 with all its tiles, so the
    // tiles that read the same keys share an L2 and every XCD takes every
    // eighth pair of the batch; pairs past the last whole eight follow in
    // grid order.  A pair's last tile (the one that sees the most keys) is
    // dealt first, so the shortest tiles fill the end of the launch.
    const int T = a.num_tiles;
    const int g = blockIdx.x;
    const int main_units = (int)(gridDim.x / T / 8) * 8 * T;
    int bk, tile;
    if (g < main_units) {
        bk = (g / 8 / T) * 8 + g % 8;
        tile = T - 1 - (g / 8) % T;
    } else {
        bk = g / T;
        tile = T - 1 - g % T;
    }
    // Pairs are taken longest sequence first, so that the longest tiles do
    // not start last and set the end of the launch.
    const int kvh = bk % a.num_kv_heads;
    // (the K staging buffer is free until the first stage is staged)
    const int b = sequence_at_rank(a.seq_lens, a.max_pages * kPageSize,
                                   (int)(gridDim.x / T / a.num_kv_heads), bk / a.num_kv_heads,
                                   reinterpret_cast<uint8_t*>(&k_lds0[0][0]), (int)sizeof(k_lds0));
    const int q0 = a.q_start[b];
    // lengths clamped to what the table row can hold, new tokens to the length
    const int L = min(a.seq_lens[b], a.max_pages * kPageSize);
    const int n_new = min(a.q_start[b + 1] - q0, L);
    const int tok0 = tile * kTileTok;
    if (tok0 >= n_new)
        return;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int i16 = lane & 15, g4 = lane >> 4;
    const int h0 = kvh * G;
    const int base_pos = L - n_new;  // position of new token 0

    const int tile_last = min(tok0 + kTileTok, n_new) - 1;
    const int nkeys = base_pos + tile_last + 1;           // keys the tile sees
    const int nstages = (nkeys + kStageKeys - 1) / kStageKeys;
    const int first_masked_stage = (base_pos + tok0) / kStageKeys;

    float m_run[kRowBlocks], lsum[kRowBlocks];
    // bf16 pools: the row sums come from the PV product itself -- a block of
    // all-ones "values" against the same bf16 probabilities -- so they sum
    // exactly the weights the numerator uses (every lane of a row block holds
    // its row's sum in each element).  e4m3 pools sum in lsum: their packed
    // probabilities carry the page's v_scale.
    floatx4_t lacc[kRowBlocks];
    const uint4 ones_bf16 = make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u);
    floatx4_t o[kRowBlocks][8];
#pragma unroll
    for (int rb = 0; rb < kRowBlocks; ++rb) {
        m_run[rb] = -INFINITY;
        lsum[rb] = 0.0f;
        lacc[rb] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int db = 0; db < 8; ++db)
            o[rb][db] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};
    }

    // Staging.  bf16 pools: direct global-to-LDS loads, no registers: lane l
    // of wavefront w fills chunk position l%16 of key row 16r + 4w + l/16
    // (slot 4w + l/16 of page r of the stage), r = 0..3, so that each load
    // instruction fills four whole rows, one contiguous kilobyte; the lane
    // reads the chunk the swizzle puts there.  A key past the sequence end
    // reads the sequence's last key instead (finite; its weight is 0 and its
    // score is masked to -inf).  e4m3 pools (128-byte rows): thread t loads
    // the codes of dims 16(t%8) .. +15 of keys 2(t/8) and 2(t/8) + 1 into
    // registers and widens them to bf16 as it stages them (16-byte loads;
    // whole-row staging would take 8-byte ones); value rows past the end are
    // zeroed.
    //
    // Loads are unconditional: page indices past the sequence are clamped to
    // its last page (whose scales are finite).
    // e4m3 register staging: thread t holds key rows st_row, st_row + 1,
    // codes of dims st_col .. st_col + 15
    constexpr int kRowsPerThread = 2;
    const int st_row = 2 * (threadIdx.x / 8);
    const int st_col = 16 * (threadIdx.x % 8);
    const int npages = (L + kPageSize - 1) / kPageSize;  // >= 1 here
    // The table row's address is uniform; held in vector registers, its
    // loads are vector loads, counted with the K/V loads and waited for at
    // the staging, instead of scalar loads, which share a counter with LDS
    // accesses and would be waited for at the next barrier and LDS read.
    typedef __attribute__((address_space(1))) const int32_t global_i32;
    global_i32* bt = (global_i32*)(a.block_table + (int64_t)b * a.max_pages);
    asm volatile("" : "+v"(bt));
    const int64_t st_off = (int64_t)kvh * a.head_bytes + st_col;
    uint4 kr[kRowsPerThread], vr[kRowsPerThread];  // e4m3 codes
    float ksr = 1.0f, vsr = 1.0f;                  // e4m3: scales of page t % 4
    // Key row (within the stage) of the thread's staging slot r.
    auto slot_row = [&](int r) { return st_row + r; };
    // The table entries of a stage are read one stage ahead, so that its K/V
    // loads do not wait on a table load: bf16, page r of the stage for slot
    // r; e4m3, the page of the thread's key pair (and page t % 4 for the
    // scales).
    int pages_next[kStagePages];
    auto stage_pages = [&](int stage, int* pg) {
#pragma unroll
        for (int r = 0; r < kStagePages; ++r) {
            const int idx = FP8 ? (r == 0 ? st_row / kPageSize : (threadIdx.x & 3)) : r;
            pg[r] = FP8 && r > 1 ? 0 : bt[min(stage * kStagePages + idx, npages - 1)];
        }
    };
    bool live[kRowsPerThread];
    // The tiles of one (sequence, kv head) read the same keys from one L2, so
    // K/V loads keep the default cache policy (2.5x fewer HBM bytes than
    // non-temporal loads).
    auto fetch = [&](int stage, const int* pg) {  // e4m3: into registers
#pragma unroll
        for (int r = 0; r < kRowsPerThread; ++r) {
            const int row = slot_row(r);
            live[r] = stage * kStageKeys + row < L;
            const int64_t off = (int64_t)pg[0] * a.page_bytes + st_off +
                                (int64_t)(row % kPageSize) * a.row_bytes;
            kr[r] = *reinterpret_cast<const uint4*>(a.k_pool + off);
            vr[r] = *reinterpret_cast<const uint4*>(a.v_pool + off);
        }
        const int64_t slab = (int64_t)pg[1] * a.num_kv_heads + kvh;
        ksr = a.k_scale[slab];
        vsr = a.v_scale[slab];
    };
    typedef __attribute__((address_space(3))) void lds_void;
    const int dma_slot = 4 * wave + lane / 16;  // key row within its page
    const int dma_chunk = (lane % 16) ^ chunk_swizzle(dma_slot);
    const int dead_slot = (L - 1) % kPageSize;
    // the lane's byte offset within a page (its key row's slot; under 2^31
    // like every in-page offset)
    const int32_t lane_off = kvh * a.head_bytes + dma_slot * a.row_bytes + 16 * dma_chunk;
    const uint32_t page_bytes32 = (uint32_t)a.page_bytes;  // < 2^31, checked by the host
    auto lds_addr = [](const void* p) { return (uint32_t)(uintptr_t)(lds_void*)p; };
    auto dma = [&](int stage, const int* pg, int sel) {  // bf16: into the stage tiles
        auto issue = [&](int r, int64_t off) {
            off += (int64_t)((uint64_t)(uint32_t)pg[r] * page_bytes32);
            dma16(a.k_pool + off, lds_addr(&k_tile(sel)[r * kPageSize + 4 * wave][0]));
            dma16(a.v_pool + off, lds_addr(&v_tile(sel)[r * kPageSize + 4 * wave][0]));
        };
        if ((stage + 1) * kStageKeys <= L) {  // every key of the stage exists
#pragma unroll
            for (int r = 0; r < kStagePages; ++r)
                issue(r, lane_off);
        } else {  // a key past the end reads the sequence's last key
            const int32_t dead_off = lane_off + (dead_slot - dma_slot) * a.row_bytes;
#pragma unroll
            for (int r = 0; r < kStagePages; ++r)
                issue(r, stage * kStageKeys + r * kPageSize + dma_slot < L ? lane_off : dead_off);
        }
    };
    // 16 e4m3 codes to 16 bf16 (exact), in order.
    auto widen = [](const uint4& c, uint4& lo, uint4& hi) {
        auto cvt = [](uint32_t w, auto upper) {
            return __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, decltype(upper)::value));
        };
        using F = std::false_type;
        using T = std::true_type;
        lo = make_uint4(cvt(c.x, F{}), cvt(c.x, T{}), cvt(c.y, F{}), cvt(c.y, T{}));
        hi = make_uint4(cvt(c.z, F{}), cvt(c.z, T{}), cvt(c.w, F{}), cvt(c.w, T{}));
    };
    auto stash = [&](int sel) {  // e4m3: widened codes at their swizzled chunks
#pragma unroll
        for (int r = 0; r < kRowsPerThread; ++r) {
            const int row = slot_row(r);
            const int sw = chunk_swizzle(row), c0 = st_col / 8;
            uint4* k0 = reinterpret_cast<uint4*>(&k_tile(sel)[row][8 * (c0 ^ sw)]);
            uint4* k1 = reinterpret_cast<uint4*>(&k_tile(sel)[row][8 * ((c0 + 1) ^ sw)]);
            uint4* v0 = reinterpret_cast<uint4*>(&v_tile(sel)[row][8 * (c0 ^ sw)]);
            uint4* v1 = reinterpret_cast<uint4*>(&v_tile(sel)[row][8 * ((c0 + 1) ^ sw)]);
            uint4 lo, hi;
            widen(kr[r], lo, hi);
            *k0 = lo;
            *k1 = hi;
            widen(vr[r], lo, hi);
            if (!live[r]) {  // slots past the sequence end may hold NaN
                lo = make_uint4(0, 0, 0, 0);
                hi = lo;
            }
            *v0 = lo;
            *v1 = hi;
        }
        if (threadIdx.x < kStagePages)
            scale_lds[sel][threadIdx.x] = make_float2(ksr, vsr);
    };

    // LDS operand offsets as a fixed lane part plus an XOR of the block
    // index (li = lane % 16, lg = lane / 16): the K operand's swizzled chunk
    // (4ks + lg) ^ s, s = chunk_swizzle(li), is 4 (ks ^ (s >> 2)) + (lg ^
    // (s & 3)), so the offset of dims 32ks.. is k_lane + (k_xor ^ 64ks), the
    // two parts in disjoint bits; likewise the V^T operand's chunk (2db + c)
    // ^ s is 2 (db ^ (s >> 1)) + (c ^ (s & 1)).  The twelve offsets (four K
    // dim blocks, eight V dim blocks) are made once per tile and held in
    // registers, so a stage spends no vector-ALU instruction on addresses.
    int k_lane, k_xor, v_lane, v_xor;
    {
        const int li = lane & 15, lg = lane >> 4;
        const int ks_sw = chunk_swizzle(li);
        k_lane = li * 256 + 16 * (lg ^ (ks_sw & 3));
        k_xor = 64 * (ks_sw >> 2);
        const int vrow = 4 * lg + (li >> 2), vsw = chunk_swizzle(vrow);
        v_lane = vrow * 256 + 16 * (((li & 3) >> 1) ^ (vsw & 1)) + 8 * (li & 1);
        v_xor = 32 * (vsw >> 1);
    }
    int koff_t[4], voff_t[8];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        koff_t[ks] = (k_xor ^ (64 * ks)) + k_lane;
        asm volatile("" : "+v"(koff_t[ks]));
    }
#pragma unroll
    for (int db = 0; db < 8; ++db) {
        voff_t[db] = (v_xor ^ (32 * db)) + v_lane;
        asm volatile("" : "+v"(voff_t[db]));
    }
    stage_pages(0, pages_next);
    if constexpr (FP8)
        fetch(0, pages_next);
    else
        dma(0, pages_next, 0);
    stage_pages(1, pages_next);
    // Q^T operand and the causal limit of this lane's row in each block,
    // read after the first stage's loads are issued (loads complete in order,
    // so the table reads those loads need wait for nothing else).  The eight
    // loads go first and unconditionally (a row past the tile's tokens reads
    // the sequence's first query), then the sign flip and a mask: a select on
    // each loaded value became a branch around its load, and every branch
    // waited for its load before the next one was issued.
    uint4 qb[kRowBlocks][4];
    int row_pos[kRowBlocks];
    bool row_real[kRowBlocks];
#pragma unroll
    for (int rb = 0; rb < kRowBlocks; ++rb) {
        const int r = wave * (kRowBlocks * 16) + rb * 16 + i16;
        const int qi = tok0 + r / G;
        row_real[rb] = qi < n_new;
        row_pos[rb] = base_pos + qi;
        const uint16_t* qrow =
            a.q + ((int64_t)(q0 + (row_real[rb] ? qi : 0)) * a.num_q_heads + h0 + r % G) *
                      kHeadDim;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            qb[rb][ks] = *reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g4);
    }
#pragma unroll
    for (int rb = 0; rb < kRowBlocks; ++rb) {
        const uint32_t keep = row_real[rb] ? 0xFFFFFFFFu : 0u;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            uint4& v = qb[rb][ks];
            v.x = (v.x ^ a.q_sign) & keep;
            v.y = (v.y ^ a.q_sign) & keep;
            v.z = (v.z ^ a.q_sign) & keep;
            v.w = (v.w ^ a.q_sign) & keep;
        }
    }
    // One stage; stages that cannot cross a query position (all but the
    // last one or two of a tile) are compiled without the causal mask.  sel:
    // the stage buffer (j % 2).
    auto stage = [&](const int j, auto masked_t, const int sel) __attribute__((always_inline)) {
        constexpr bool masked = decltype(masked_t)::value;
        const int buf = sel;
        if constexpr (FP8) {
            stash(sel);
            if (j + 1 < nstages) {
                fetch(j + 1, pages_next);
                stage_pages(j + 2, pages_next);
            }
            __syncthreads();
        } else {
            // this stage's direct loads have landed and every wavefront is
            // done with the other buffer, which the next stage's loads fill
            // once the score products are issued.  The compiler does not
            // track the direct loads, so this wavefront waits for its own
            // here, before the barrier.
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
            __syncthreads();
        }

        // Score multiplier (scale * log2 e, times k_scale) and value scale
        // of the stage's four pages; a page past the sequence carries the
        // finite scales of the page its index was clamped to (its keys are
        // masked and its values staged as zeros).
        float sl[4], vsc[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            sl[kb] = a.scale_log2;
            vsc[kb] = 1.0f;
            if (FP8) {
                const float2 ps = scale_lds[buf][kb];
                sl[kb] *= ps.x;
                vsc[kb] = ps.y;
            }
        }

        // The lane's byte offsets into the stage tiles, the same for both
        // buffers (each buffer's base folds into the LDS instructions'
        // offset field).
        const int (&koff)[4] = koff_t;
        const char* ktile = reinterpret_cast<const char*>(&k_tile(sel)[0][0]);
        const char* vtile = reinterpret_cast<const char*>(&v_tile(sel)[0][0]);

        // S^T for the stage's four 16-key blocks: lane holds row i16, keys
        // 16kb + 4g4 + jj.
        floatx4_t sacc[kRowBlocks][4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int rb = 0; rb < kRowBlocks; ++rb)
                sacc[rb][kb] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};
        // dims outermost: eight independent accumulators between dependent MFMAs.
        // The two product phases run at raised wave priority: of the two
        // wavefronts on a SIMD, one starting its products issues ahead of
        // one in its softmax, which keeps the MFMA unit fed.
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const uint4 kv =
                    *reinterpret_cast<const uint4*>(ktile + 16 * kb * 256 + koff[ks]);
#pragma unroll
                for (int rb = 0; rb < kRowBlocks; ++rb)
                    sacc[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8_t, kv), __builtin_bit_cast(bf16x8_t, qb[rb][ks]),
                        sacc[rb][kb], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        // bf16: the next stage's direct loads, issued after the K operand
        // reads so that their LDS writes do not compete with them
        if constexpr (!FP8) {
            if (j + 1 < nstages) {
                dma(j + 1, pages_next, 1 - sel);
                stage_pages(j + 2, pages_next);
            }
        }
        // Probabilities (masked only in stages that can cross a query
        // position; rows past the tile's tokens score 0 and stay finite) and
        // O^T += V^T P^T: lane holds dims 16db + 4g4 + jj of row i16.
        // Row max of the scaled scores (log2 units) over the stage for both
        // row blocks (lane-local over 16 keys, then the two other lane groups
        // of the row).  The multiply folds into the exponent,
        // p = 2^(raw * mult - m).  Stages below the diagonal see every key:
        // their max is each page's multiplier times its raw max (bf16 pools
        // have one multiplier, |scale| log2 e >= 0, Q carrying the scale's
        // sign), or times its raw min for a negative e4m3 multiplier, taken
        // with the IEEE maximum instructions, which need no canonicalising
        // copies of their operands.  Stages on the diagonal mask first: with
        // every page's multiplier positive the max is again multiplier times
        // raw max; a zero or negative one takes the general path -- scale,
        // then mask, so that masked keys stay at -inf for any scale -- with
        // mult 1.
        float sc[kRowBlocks][4][4], mx[kRowBlocks], mult[4];
        auto stage_max = [&](auto pre_scaled) {
#pragma unroll
            for (int rb = 0; rb < kRowBlocks; ++rb) {
                mx[rb] = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    float pm = -INFINITY;
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        float x = sacc[rb][kb][jj];
                        if (decltype(pre_scaled)::value)
                            x *= sl[kb];
                        if (masked)
                            x = j * kStageKeys + 16 * kb + 4 * g4 + jj <= row_pos[rb] ? x
                                                                                  : -INFINITY;
                        sc[rb][kb][jj] = x;
                        pm = fmaxf(pm, x);
                    }
                    // mult > 0 in the folded form: -inf stays -inf
                    mx[rb] = fmaxf(mx[rb], decltype(pre_scaled)::value ? pm : pm * sl[kb]);
                }
            }
        };
        if constexpr (!masked) {
            // the stage's page multipliers are the same in every lane
            const bool all_pos =
                !FP8 || __builtin_amdgcn_readfirstlane((sl[0] >= 0.0f) & (sl[1] >= 0.0f) &
                                                       (sl[2] >= 0.0f) & (sl[3] >= 0.0f));
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
                mult[kb] = sl[kb];
#pragma unroll
            for (int rb = 0; rb < kRowBlocks; ++rb) {
                const floatx4_t(&x)[4] = sacc[rb];
                if constexpr (FP8) {
                    float pm[4];
                    if (all_pos) {  // every page's multiplier >= 0: raw max times it
#pragma unroll
                        for (int kb = 0; kb < 4; ++kb)
                            pm[kb] = __builtin_elementwise_maximum(
                                         __builtin_elementwise_maximum(x[kb][0], x[kb][1]),
                                         __builtin_elementwise_maximum(x[kb][2], x[kb][3])) *
                                     sl[kb];
                    } else {
#pragma unroll
                        for (int kb = 0; kb < 4; ++kb) {
                            const float hi = __builtin_elementwise_maximum(
                                __builtin_elementwise_maximum(x[kb][0], x[kb][1]),
                                __builtin_elementwise_maximum(x[kb][2], x[kb][3]));
                            const float lo = __builtin_elementwise_minimum(
                                __builtin_elementwise_minimum(x[kb][0], x[kb][1]),
                                __builtin_elementwise_minimum(x[kb][2], x[kb][3]));
                            pm[kb] = (sl[kb] >= 0.0f ? hi : lo) * sl[kb];
                        }
                    }
                    mx[rb] = __builtin_elementwise_maximum(
                        __builtin_elementwise_maximum(pm[0], pm[1]),
                        __builtin_elementwise_maximum(pm[2], pm[3]));
                } else {
                    // one multiplier >= 0 for the stage: the max of the
                    // sixteen raw scores as a tree of three-input maxima
                    auto max3 = [](float a, float b, float c) {
                        return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
                    };
                    const float m0 = max3(x[0][0], x[0][1], x[0][2]);
                    const float m1 = max3(x[0][3], x[1][0], x[1][1]);
                    const float m2 = max3(x[1][2], x[1][3], x[2][0]);
                    const float m3 = max3(x[2][1], x[2][2], x[2][3]);
                    const float m4 = max3(x[3][0], x[3][1], x[3][2]);
                    mx[rb] = __builtin_elementwise_maximum(max3(m0, m1, m2), max3(m3, m4, x[3][3])) *
                             sl[0];
                }
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
                        sc[rb][kb][jj] = x[kb][jj];
            }
        } else {
            bool positive = true;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
                positive &= sl[kb] > 0.0f;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
                mult[kb] = positive ? sl[kb] : 1.0f;
            if (positive)
                stage_max(std::false_type{});
            else
                stage_max(std::true_type{});
        }
#pragma unroll
        for (int rb = 0; rb < kRowBlocks; ++rb)
            mx[rb] = max_lanes_xor16(mx[rb]);
#pragma unroll
        for (int rb = 0; rb < kRowBlocks; ++rb)
            mx[rb] = max_lanes_xor32(mx[rb]);  // finite: key 0 is visible
        bool grow = false;
#pragma unroll
        for (int rb = 0; rb < kRowBlocks; ++rb)
            grow |= mx[rb] > m_run[rb] + kMaxSlack;
        if (__builtin_expect(__any(grow), 0)) {  // rare: kept out of line
#pragma unroll
            for (int rb = 0; rb < kRowBlocks; ++rb) {
                const float m_new = mx[rb] > m_run[rb] + kMaxSlack ? mx[rb] : m_run[rb];
                const float alpha = exp2_fast(m_run[rb] - m_new);  // 0 on the first stage
                m_run[rb] = m_new;
                lsum[rb] *= alpha;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    lacc[rb][jj] *= alpha;
#pragma unroll
                for (int db = 0; db < 8; ++db)
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
                        o[rb][db][jj] *= alpha;
            }
        }
        // Probabilities as P^T operands: [rb][key half] bf16 x 8 (round to
        // nearest even; the normaliser sums the unrounded values).  Piece
        // (rb, kb, jp): keys 16kb + 4g4 + 2jp, +1 of row block rb.
        uint32_t pk[kRowBlocks][4][2];
        auto make_p = [&](int rb, int kb, int jp) {
            float p0 = exp2_fast(fmaf(sc[rb][kb][2 * jp], mult[kb], -m_run[rb]));
            float p1 = exp2_fast(fmaf(sc[rb][kb][2 * jp + 1], mult[kb], -m_run[rb]));
            if (FP8)
                lsum[rb] += p0 + p1;
            if (FP8) {
                p0 *= vsc[kb];
                p1 *= vsc[kb];
            }
            pk[rb][kb][jp] = pack_bf16x2(p0, p1);
        };
        uint4 pt[kRowBlocks][2];
        auto pack_half = [&](int kh) {
#pragma unroll
            for (int rb = 0; rb < kRowBlocks; ++rb)
                pt[rb][kh] = make_uint4(pk[rb][2 * kh][0], pk[rb][2 * kh][1],
                                        pk[rb][2 * kh + 1][0], pk[rb][2 * kh + 1][1]);
        };
        // keys 0..31 first
#pragma unroll
        for (int rb = 0; rb < kRowBlocks; ++rb)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int jp = 0; jp < 2; ++jp)
                    make_p(rb, kb, jp);
        pack_half(0);
        // O^T += V^T P^T: lane holds dims 16db + 4g4 + jj of row i16.  Steps
        // run over the first key half's eight dim blocks, then the second's,
        // so the two products into one accumulator are eight steps apart;
        // the second half's probabilities are made one piece per step of the
        // first half.  The V^T operand of the next step is read before this
        // one's MFMAs.  Lane i16 + 16g4 reads row 32kh + 4g4 + i16/4 (and
        // the row 16 below, same swizzle), dims 16db + 4(i16 % 4) .. +3:
        // chunk 2db + (i16 % 4)/2, half i16 % 2.
        auto vt_operand = [&](int step) {
            const int kh = step >> 3, db = step & 7;
            const int voff = voff_t[db];
            const uint16_t* vp =
                reinterpret_cast<const uint16_t*>(vtile + 32 * kh * 256 + voff);
            const uint2 va = lds_read_transposed(vp);
            const uint2 vb = lds_read_transposed(vp + 16 * kHeadDim);
            return make_uint4(va.x, va.y, vb.x, vb.y);
        };
        __builtin_amdgcn_s_setprio(1);
        uint4 vt_next = vt_operand(0);
#pragma unroll
        for (int step = 0; step < 16; ++step) {
            const uint4 vt = vt_next;
            if (step + 1 < 16)
                vt_next = vt_operand(step + 1);
            // keep the read ahead of this step's MFMAs (the scheduler would
            // otherwise sink it next to its own use)
            __builtin_amdgcn_sched_barrier(0);
            const int kh = step >> 3, db = step & 7;
#pragma unroll
            for (int rb = 0; rb < kRowBlocks; ++rb) {
                o[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8_t, vt), __builtin_bit_cast(bf16x8_t, pt[rb][kh]),
                    o[rb][db], 0, 0, 0);
            }
            if (step < 8) {
                make_p(step >> 2, 2 + ((step >> 1) & 1), step & 1);
                if (step == 7)
                    pack_half(1);
            }
        }
        if (!FP8) {
#pragma unroll
            for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                for (int rb = 0; rb < kRowBlocks; ++rb)
                    lacc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8_t, ones_bf16),
                        __builtin_bit_cast(bf16x8_t, pt[rb][kh]), lacc[rb], 0, 0, 0);
        }
        __builtin_amdgcn_s_setprio(0);
    };
    int j = 0;
    auto run = [&](int end, auto masked_t) {
        for (; j < end; ++j)
            stage(j, masked_t, j & 1);
    };
    run(min(first_masked_stage, nstages), std::false_type{});
    run(nstages, std::true_type{});

    // out[row] = O[row] / l[row]; lane holds row i16, dims 16db + 4g4 + jj.
#pragma unroll
    for (int rb = 0; rb < kRowBlocks; ++rb) {
        const float l = FP8 ? sum_lanes_xor32(sum_lanes_xor16(lsum[rb])) : lacc[rb][0];
        if (!row_real[rb])
            continue;
        const int r = wave * (kRowBlocks * 16) + rb * 16 + i16;
        const int qi = tok0 + r / G;
        uint16_t* orow = a.out + ((int64_t)(q0 + qi) * a.num_q_heads + h0 + r % G) * kHeadDim;
        const float inv = 1.0f / l;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const floatx4_t& v = o[rb][db];
            *reinterpret_cast<uint2*>(orow + 16 * db + 4 * g4) =
                make_uint2(f32_to_bf16(v[0] * inv) | (f32_to_bf16(v[1] * inv) << 16),
                           f32_to_bf16(v[2] * inv) | (f32_to_bf16(v[3] * inv) << 16));
        }
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
    const bool fp8 = kv_dtype == RL_DA_KV_FP8_E4M3;
    if (!pools_paired(layout, k_pool, v_pool, fp8 ? 1 : 2))
        return RL_DA_ERR_INVALID_ARG;
    PoolStrides ps;
    if (!pool_strides(layout, num_kv_heads, fp8 ? 1 : 2, &ps))
        return RL_DA_ERR_INVALID_ARG;
    if (ps.page >= ((int64_t)1 << 31))  // in-page offsets are 32-bit in the kernel
        return RL_DA_ERR_UNSUPPORTED;
    const int G = num_q_heads / num_kv_heads;
    if (head_dim != kHeadDim || page_size != kPageSize ||
        (G != 1 && G != 2 && G != 4 && G != 8 && G != 16))
        return RL_DA_ERR_UNSUPPORTED;
    if (batch == 0 || max_q_per_seq == 0)
        return RL_DA_OK;
    const int tile_tok = kTileRows / G;
    ExtendArgs ea;
    ea.q = (const uint16_t*)q;
    ea.q_start = q_start;
    ea.k_pool = (const uint8_t*)k_pool;
    ea.v_pool = (const uint8_t*)v_pool;
    ea.k_scale = k_scale;
    ea.v_scale = v_scale;
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
    ea.scale_log2 = fabsf(scale) * kLog2e;
    ea.q_sign = scale < 0.0f ? 0x80008000u : 0u;
    const int64_t blocks = (int64_t)batch * num_kv_heads * ea.num_tiles;
    if (blocks > INT32_MAX)
        return RL_DA_ERR_UNSUPPORTED;
    hipStream_t st = (hipStream_t)stream;
    const dim3 grid((unsigned)blocks), block(kWave * kUnitWaves);
    typedef void (*Kernel)(ExtendArgs);
    Kernel k;
    switch (G) {
    case 1: k = fp8 ? extend_attn<1, true> : extend_attn<1, false>; break;
    case 2: k = fp8 ? extend_attn<2, true> : extend_attn<2, false>; break;
    case 4: k = fp8 ? extend_attn<4, true> : extend_attn<4, false>; break;
    case 8: k = fp8 ? extend_attn<8, true> : extend_attn<8, false>; break;
    default: k = fp8 ? extend_attn<16, true> : extend_attn<16, false>; break;
    }
    hipLaunchKernelGGL(k, grid, block, 0, st, ea);
    return hipGetLastError() == hipSuccess ? RL_DA_OK : RL_DA_ERR_HIP;
}

}  // extern "C"
