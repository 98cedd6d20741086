// rl_decode.hip -- decode-step kernels and the handle-based C interface.
//
// One decode step of one attention layer (the rollout inner loop of
// arXiv 2512.22492, Sec. 2.1): out[b,h] = softmax(scale * q[b,h] K_b^T) V_b
// over a paged KV cache, kv head h / G.
//
// Decomposition (split-K, "flash-decoding").  A work unit is one work-group of
// four wavefronts for (sequence b, kv head, split s), where a split is
// split_tokens consecutive cached tokens (4096 by default).  The wavefronts
// take the split's pages in turn (wavefront w: pages w, w+4, w+8, ...); each
// keeps an online softmax (running max m, running sum l, weighted value sum
// acc) for the G query heads that share the kv head.  The four partial states
// are merged with the log-sum-exp rule through LDS at the end of the unit, so a
// sequence that fits one split is finished by one work-group; longer sequences
// write one partial per split and a second kernel merges them.  How a
// sequence's tokens are divided depends only on its own length and the
// handle's split size, never on the rest of the batch.
//
// Data movement is the whole cost: every K/V byte is read once from HBM.  A
// (page, kv head) slab is 16 tokens x 128 dims x 2 bytes = 4 KiB, contiguous in
// the [page][kv head][slot][dim] pool layout (16 rows of 256 bytes, 256 * Hkv
// bytes apart, in the [page][slot][kv head][dim] layout), and is read by one
// wavefront with four 16-byte-per-lane non-temporal loads each for K and V.  Scores are computed once per
// kv head for all G query heads of the group (the GQA reuse), either with one
// MFMA per 32 dims (the G query rows packed into a 16-row tile) or with bf16
// dot2 ops and DPP row reductions.  The value accumulation runs on the matrix
// cores by default (the page's values transposed through LDS, the weights as
// two bf16 terms), or in fp32 on the vector ALUs.
//
// All arithmetic is fp32; scores are kept in the log2 domain (scale folded
// with log2(e)) so that every exponential is one v_exp_f32.

#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "rl_common.h"

using namespace rl_da;

namespace {

constexpr int kDefaultSplitTokens = 4096;
constexpr int kMinDefaultSplitTokens = 512;
// The default split is the longest that still cuts a full-capacity batch into
// this many work units (enough to spread over the chip).
constexpr int64_t kMinDefaultUnits = 256;
// each wavefront holds its pages' block-table entries one per lane
constexpr int kMaxSplitTokens = kWave * kUnitWaves * kPageSize;
// head-parallel units (token-major pools): up to 8 kv heads per work-group,
// every wavefront walks all pages of its split
constexpr int kMaxHeadsPerUnit = 8;
constexpr int kMaxSplitTokensHp = 4096;
// Four-wavefront work-groups the chip holds at once with three per CU
// (MI355X: 256 CUs); the unit-family choice for token-major pools compares
// a handle's capacity with it.
constexpr int64_t kResidentUnits = 256 * 3;
// Launches with more than one split run persistent work-groups that take
// units longest first from a plan built in LDS; batches above this size
// take the units in sequence order instead (the plan would not fit).
constexpr int kMaxPlanBatch = 4096;

// How the split kernel of a launch with several splits takes its units.
enum Schedule : int32_t {
    kOnePerGroup = 0,   // grid = units: work-group g runs unit g (sequence order)
    kQueueInOrder = 1,  // persistent, units in sequence order (empty ones included)
    kQueuePlanned = 2,  // persistent, units longest first from the LDS plan
};

struct SplitArgs {
    const uint16_t* q;          // bf16 bits [B][Hq][D]
    const uint8_t* k_pool;      // [P][Hkv][16][D] or [P][16][Hkv][D] elements
    const uint8_t* v_pool;
    const float* k_scale;       // [P][Hkv] (fp8 only)
    const float* v_scale;
    const int32_t* block_table; // [B][max_pages]
    const int32_t* seq_lens;    // [B]
    uint16_t* out;              // bf16 bits [B][Hq][D]
    float* ws_acc;              // [B][Hq][num_splits][D]
    float* ws_ml;               // [B][Hq][num_splits][2]  (m in log2 units, l)
    int32_t* dev_error;
    int64_t num_pages;
    int64_t page_bytes;         // pool bytes per page (all kv heads)
    int32_t head_bytes;         // offset of kv head h's slab within a page, per h
    int32_t row_bytes;          // offset between token slots of a slab
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t max_pages;
    int32_t split_pages;
    int32_t num_splits;         // ceil(max_pages / split_pages)
    int32_t heads_per_unit;     // kv heads per head-parallel work-group
    int32_t batch;
    int32_t schedule;           // several splits: a Schedule
    int32_t* queue;             // persistent launch: [0] next unit, [1] finished work-groups
    float scale_log2;           // scale * log2(e)
};

// One wavefront's share of a work unit: pages p0 + wave + 4i, i < count.
struct WaveTask {
    int b, kvh, s, wave, lane;
    int seq_len;   // clamped to max_pages * page_size
    int npages;    // pages holding the sequence
    int nsplit;    // splits of this sequence
    int p0;        // first page of the unit
    int count;     // pages of this wavefront (may be 0)
    bool owner;    // the one unit per (sequence, head) that writes an empty
                   // sequence's zeros and reports a too-long sequence
};

// Fills a wavefront's task for the unit (sequence b, kv head kvh, split s)
// -- s < 0 meaning the sequence's last split -- and loads its block-table
// entries (lane i: page p0 + wave + 4i) together with the sequence length.
// Entries past the sequence's end lie inside the table row and are loaded
// but never used.  Returns false, for every wavefront of the unit alike, when
// the unit holds no page of its sequence.
template <bool CHECKED>
__device__ __forceinline__ bool begin_unit(const SplitArgs& a, WaveTask& t, int32_t& my_page,
                                           int b, int kvh, int s, bool owner)
{
    t.lane = threadIdx.x % kWave;
    t.wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform: scalar
    t.b = b;
    t.kvh = kvh;
    t.owner = owner;
    t.s = max(s, 0);
    t.p0 = t.s * a.split_pages;
    auto load_pages = [&] {
        const int col = t.p0 + t.wave + kUnitWaves * t.lane;
        const bool in_split = col < t.p0 + a.split_pages && col < a.max_pages;
        my_page = in_split ? a.block_table[(int64_t)t.b * a.max_pages + col] : 0;
    };
    if (s >= 0)
        load_pages();  // issued together with the length load
    int L = a.seq_lens[t.b];
    const int cap = a.max_pages * kPageSize;
    if (L > cap) {
        if (CHECKED && threadIdx.x == 0 && t.owner && t.kvh == 0)
            atomicOr(a.dev_error, RL_DA_DEVERR_LENGTH_TOO_LONG);
        L = cap;
    }
    t.seq_len = L;
    t.npages = L > 0 ? (L + kPageSize - 1) / kPageSize : 0;
    t.nsplit = (t.npages + a.split_pages - 1) / a.split_pages;
    if (s < 0) {
        if (t.nsplit == 0)
            return false;
        t.s = t.nsplit - 1;
        t.p0 = t.s * a.split_pages;
        load_pages();
    } else if (t.s >= t.nsplit) {
        return false;
    }
    const int p1 = min(t.p0 + a.split_pages, t.npages);
    t.count = max(0, (p1 - t.p0 - t.wave + kUnitWaves - 1) / kUnitWaves);
    if (CHECKED) {
        const bool bad = t.lane < t.count && (my_page < 0 || (int64_t)my_page >= a.num_pages);
        if (__any(bad)) {
            if (t.lane == 0)
                atomicOr(a.dev_error, RL_DA_DEVERR_PAGE_OUT_OF_RANGE);
            t.count = 0;  // read nothing; the unit's output is unspecified
        }
    }
    return true;
}

// ------------------------------------------------- persistent schedule ---
//
// A launch with more than one split runs about one work-group per resident
// slot; each takes units one after another from a counter in the workspace.
// (The hardware hands out the work-groups of a grid in index order,
// round-robin over the XCDs and their shader engines, and stalls while the
// engine next in turn is full, so a static grid of unequal units leaves
// engines idle behind a busy one.)  Units go longest first: every full split,
// then each sequence's last split in descending length, empty sequences last,
// so the launch ends on its shortest units.  Each work-group builds that
// order in LDS from the sequence lengths:
//   full[b]  = splits of sequence b before its last one, prefix-summed
//              (full[batch] = F, all full splits);
//   order[j] = sequences by the length of their last split, longest first:
//              kLengthClasses classes of last-split page counts, each class
//              in sequence order (a stable counting sort, so that every
//              work-group builds the same order).
// With U units per (sequence, split), unit i < F*U is full split i/U of the
// sequence found by binary search in full[], and unit F*U + i is the last
// split of order[i/U].  Without a plan (kQueueInOrder, or kOnePerGroup when
// every unit has a work-group of its own) unit i is split (i/U) % num_splits
// of sequence i/(U*num_splits), empty ones included.
// Which work-group takes a unit never changes a result.

// Exclusive prefix sum of data[0 .. n) in place by the work-group; returns
// the total.  tmp holds one int per wavefront.
__device__ __forceinline__ int block_exclusive_scan(int* data, int n, int* tmp)
{
    const int tid = threadIdx.x;
    const int nt = blockDim.x;
    const int per = (n + nt - 1) / nt;
    const int lo = min(tid * per, n), hi = min(lo + per, n);
    int sum = 0;
    for (int i = lo; i < hi; ++i)
        sum += data[i];
    const int lane = tid % kWave;
    int x = sum;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int y = __shfl_up(x, d, kWave);
        if (lane >= d)
            x += y;
    }
    if (lane == kWave - 1)
        tmp[tid / kWave] = x;
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < nt / kWave; ++w) {
        const int v = tmp[w];
        before += w < tid / kWave ? v : 0;
        total += v;
    }
    int run = before + x - sum;
    for (int i = lo; i < hi; ++i) {
        const int v = data[i];
        data[i] = run;
        run += v;
    }
    __syncthreads();
    return total;
}

constexpr int kLengthClasses = 8;
constexpr int kMaxPlanWaves = kMaxHeadsPerUnit;  // wavefronts of the largest work-group

// Ints of LDS the plan needs for `batch` sequences: full[], order[], one
// byte per sequence for its length class, the scans' per-wavefront totals.
__host__ __device__ constexpr int plan_ints(int batch)
{
    return 2 * batch + 1 + (batch + 3) / 4 + kLengthClasses * kMaxPlanWaves;
}

// Full splits of sequence b and the length class of its last split (0 for
// a full-length last split, rising as it gets shorter; an empty sequence is
// in the last class).
__device__ __forceinline__ void split_shape(const SplitArgs& a, int b, int& full, int& cls)
{
    const int L = min(a.seq_lens[b], a.max_pages * kPageSize);
    const int np = L > 0 ? (L + kPageSize - 1) / kPageSize : 0;
    const int ns = (np + a.split_pages - 1) / a.split_pages;
    full = max(ns - 1, 0);
    const int last = ns > 0 ? np - (ns - 1) * a.split_pages : 0;  // 0 .. split_pages
    cls = (a.split_pages - last) * kLengthClasses / (a.split_pages + 1);
}

// Exclusive prefix over the work-group's threads of K counts per thread, in
// place; total[c] gets the sum of count c.  tmp holds K * kMaxPlanWaves ints.
template <int K>
__device__ __forceinline__ void block_scan_counts(int (&v)[K], int (&total)[K], int* tmp)
{
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    int x[K];
#pragma unroll
    for (int c = 0; c < K; ++c)
        x[c] = v[c];
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
#pragma unroll
        for (int c = 0; c < K; ++c) {
            const int y = __shfl_up(x[c], d, kWave);
            if (lane >= d)
                x[c] += y;
        }
    }
    if (lane == kWave - 1) {
#pragma unroll
        for (int c = 0; c < K; ++c)
            tmp[c * kMaxPlanWaves + wave] = x[c];
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < K; ++c) {
        int before = 0, tot = 0;
        for (int w = 0; w < nw; ++w) {
            const int t = tmp[c * kMaxPlanWaves + w];
            before += w < wave ? t : 0;
            tot += t;
        }
        v[c] = before + x[c] - v[c];
        total[c] = tot;
    }
    __syncthreads();
}

// Builds full[] and order[] (see above); returns F.  The result depends only
// on the sequence lengths, read once.  Ends with a barrier.
__device__ __forceinline__ int build_plan(const SplitArgs& a, int* plan)
{
    const int B = a.batch, nt = blockDim.x;
    int* full = plan;
    int* order = plan + B + 1;
    uint8_t* cls_of = reinterpret_cast<uint8_t*>(order + B);
    int* tmp = order + B + (B + 3) / 4;
    for (int b = threadIdx.x; b < B; b += nt) {
        int f, cls;
        split_shape(a, b, f, cls);
        full[b] = f;
        cls_of[b] = (uint8_t)cls;
    }
    if (threadIdx.x == 0)
        full[B] = 0;
    __syncthreads();
    const int F = block_exclusive_scan(full, B + 1, tmp);
    // order: each thread takes a contiguous slice of sequences
    const int per = (B + nt - 1) / nt;
    const int lo = min((int)threadIdx.x * per, B), hi = min(lo + per, B);
    int pos[kLengthClasses], total[kLengthClasses];
#pragma unroll
    for (int c = 0; c < kLengthClasses; ++c)
        pos[c] = 0;
    for (int b = lo; b < hi; ++b) {
        const int cls = cls_of[b];
#pragma unroll
        for (int c = 0; c < kLengthClasses; ++c)
            pos[c] += cls == c;
    }
    block_scan_counts(pos, total, tmp);
    int start = 0;
#pragma unroll
    for (int c = 0; c < kLengthClasses; ++c) {
        pos[c] += start;  // class c begins after every longer class
        start += total[c];
    }
    for (int b = lo; b < hi; ++b) {
        const int cls = cls_of[b];
        int at = 0;
#pragma unroll
        for (int c = 0; c < kLengthClasses; ++c) {
            at = cls == c ? pos[c] : at;
            pos[c] += cls == c;
        }
        order[at] = b;
    }
    __syncthreads();
    return F;
}

// Runs unit(b, k, s, owner) -- k the unit's index within its (sequence,
// split), s < 0 for a last split -- for every unit of the launch.  Work-group
// g starts with unit g; later units come from a.queue (gridDim.x + the
// count of earlier requests), requested when the current unit starts and
// needed only when it ends.  The last work-group to finish resets the queue
// for the next launch.  plan: the dynamic LDS (unused without a plan).
template <typename Unit>
__device__ __forceinline__ void run_persistent(const SplitArgs& a, int U, int* plan, Unit unit)
{
    if (a.schedule == kOnePerGroup) {
        const int j = blockIdx.x / U;
        const int s = j % a.num_splits;
        unit(a, j / a.num_splits, blockIdx.x % U, s, s == 0);
        return;
    }
    __shared__ int s_item[2];
    unsigned* const counter = reinterpret_cast<unsigned*>(&a.queue[0]);
    const bool planned = a.schedule == kQueuePlanned;
    int F = 0, total;
    if (planned) {
        F = build_plan(a, plan);
        total = (F + a.batch) * U;
    } else {
        total = a.batch * a.num_splits * U;
    }
    const int* full = plan;
    const int* order = plan + a.batch + 1;
    int item = blockIdx.x;
    for (int cur = 0;; cur ^= 1) {
        if (item >= total)
            break;
        // atomicInc (not atomicAdd) leaves the wait for the result at its use
        unsigned next = 0;
        if (threadIdx.x == 0)
            next = atomicInc(counter, 0xffffffffu);
        const int k = item % U, j = item / U;
        int b, s;
        bool owner;
        if (!planned) {
            s = j % a.num_splits;
            b = j / a.num_splits;
            owner = s == 0;
        } else if (j < F) {
            int lo = 0, hi = a.batch;  // full[lo] <= j < full[hi]
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (full[mid] <= j)
                    lo = mid;
                else
                    hi = mid;
            }
            b = lo;
            s = j - full[lo];
            owner = false;
        } else {
            b = order[j - F];
            s = -1;
            owner = true;
        }
        b = __builtin_amdgcn_readfirstlane(b);
        s = __builtin_amdgcn_readfirstlane(s);
        if (b >= 0 && b < a.batch && s < a.num_splits)  // holds by construction
            unit(a, b, k, s, owner);
        if (threadIdx.x == 0)
            s_item[cur] = (int)gridDim.x + (int)next;
        __syncthreads();
        item = __builtin_amdgcn_readfirstlane(s_item[cur]);
    }
    if (threadIdx.x == 0 && atomicAdd(&a.queue[1], 1) == (int)gridDim.x - 1) {
        atomicExch(&a.queue[0], 0);
        atomicExch(&a.queue[1], 0);
    }
}

// An empty sequence produces zeros (written once, by its owner unit).
template <int G>
__device__ __forceinline__ void write_zero_rows(const SplitArgs& a, const WaveTask& t)
{
    if (t.npages != 0 || !t.owner)
        return;
    for (int e = threadIdx.x; e < G * (kHeadDim / 8); e += kWave * kUnitWaves) {
        const int g = e / (kHeadDim / 8), chunk = e % (kHeadDim / 8);
        uint4* dst = reinterpret_cast<uint4*>(
            a.out + ((int64_t)t.b * a.num_q_heads + t.kvh * G + g) * kHeadDim + chunk * 8);
        *dst = make_uint4(0, 0, 0, 0);
    }
}

// First byte (token slot 0, dim 0) of slab (page, kvh).
__device__ __forceinline__ const uint8_t* slab_base(const SplitArgs& a, const uint8_t* pool,
                                                    int64_t page, int kvh)
{
    return pool + page * a.page_bytes + (int64_t)kvh * a.head_bytes;
}

// Global page index of a wavefront's i-th page.
__device__ __forceinline__ int task_page(const WaveTask& t, int i)
{
    return t.p0 + t.wave + kUnitWaves * i;
}

// LDS holding each wavefront's final state for the unit merge.
template <int G>
struct UnitShared {
    float acc[kUnitWaves][G][kHeadDim];
    float m[kUnitWaves][G];
    float l[kUnitWaves][G];
};

// Stores one wavefront's state for query head g: 8 dims of acc from lane
// chunk c, and (m, l) from chunk 0.
template <int G>
__device__ __forceinline__ void stash_state(UnitShared<G>& sh, int wave, int g, int c,
                                            const float (&acc)[8], float m, float l)
{
    float4* dst = reinterpret_cast<float4*>(&sh.acc[wave][g][c * 8]);
    dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    if (c == 0) {
        sh.m[wave][g] = m;
        sh.l[wave][g] = l;
    }
}

// After every wavefront has stashed its state: merges the four states of each
// query head in wavefront order (M = max m_w, weights 2^(m_w - M)) and writes
// the bf16 output row, or the unit's (M, l, acc) partial when the sequence has
// more than one split.  Wavefront w merges heads w, w+4, ...; two dims per lane.
template <int G>
__device__ __forceinline__ void merge_unit(const SplitArgs& a, const WaveTask& t,
                                           const UnitShared<G>& sh)
{
    for (int g = t.wave; g < G; g += kUnitWaves) {
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kUnitWaves; ++w)
            M = fmaxf(M, sh.m[w][g]);  // finite: the unit holds at least one token
        float den = 0.0f, n0 = 0.0f, n1 = 0.0f;
#pragma unroll
        for (int w = 0; w < kUnitWaves; ++w) {
            const float wt = exp2_fast(sh.m[w][g] - M);  // 0 for a wavefront with no page
            den = fmaf(wt, sh.l[w][g], den);
            const float2 v = *reinterpret_cast<const float2*>(&sh.acc[w][g][2 * t.lane]);
            n0 = fmaf(wt, v.x, n0);
            n1 = fmaf(wt, v.y, n1);
        }
        const int64_t row = (int64_t)t.b * a.num_q_heads + t.kvh * G + g;
        if (t.nsplit == 1) {
            const float inv = 1.0f / den;
            *reinterpret_cast<uint32_t*>(a.out + row * kHeadDim + 2 * t.lane) =
                f32_to_bf16(n0 * inv) | (f32_to_bf16(n1 * inv) << 16);
        } else {
            const int64_t part = row * a.num_splits + t.s;
            *reinterpret_cast<float2*>(a.ws_acc + part * kHeadDim + 2 * t.lane) =
                make_float2(n0, n1);
            if (t.lane == 0)
                *reinterpret_cast<float2*>(a.ws_ml + part * 2) = make_float2(M, den);
        }
    }
}

// Streams a wavefront's pages through two buffers (A and B): while one page is
// consumed from one buffer the next is in flight into the other, and the load
// two pages ahead is issued as soon as a buffer has been consumed.  The
// steady-state loop issues unconditionally, so the compiler's wait before each
// consume only covers the buffer being consumed.  issue and consume take the
// wavefront-local page index.
template <typename Buf, typename Issue, typename Consume>
__device__ __forceinline__ void stream_pages(int n, Buf& a, Buf& b, Issue issue, Consume consume)
{
    if (n <= 0)
        return;
    int i = 0;
    if (n >= 4) {
        issue(a, 0);
        issue(b, 1);
        for (; i + 3 < n; i += 2) {
            consume(a, i);
            issue(a, i + 2);
            consume(b, i + 1);
            issue(b, i + 3);
        }
    } else {
        issue(a, 0);
        if (n >= 2)
            issue(b, 1);
    }
    const int rest = n - i;  // 1..3 pages left; pages i and i+1 already issued
    consume(a, i);
    if (rest == 3)
        issue(a, i + 2);
    if (rest >= 2)
        consume(b, i + 1);
    if (rest == 3)
        consume(a, i + 2);
}

// ------------------------------------------------------ K/V page formats ---
//
// A wavefront consumes one (page, kv head) slab at a time: 16 token rows of
// 128 dims, `row` bytes apart.  For the score MFMA (v_mfma_f32_16x16x32_bf16,
// A = queries 16x32, B = keys 32x16) lane l supplies key token n = l%16 and 8
// of the 32 dims of each of the four k-blocks; which 8 dims is the format's
// choice (q_dim), as long as the query tile uses the same ones.  For the value
// pass lane l = 16r + c holds dims 8c..8c+7 of tokens 4k + r, k = 0..3.

// bf16 slab: 4 KiB, four 16-byte loads per lane for K and for V.
struct KvBf16 {
    static constexpr bool kScaled = false;
    static constexpr bool kStagedK = false;
    struct Buf {
        uint4 k[4];
        uint4 v[4];
    };
    // first dim of the 8 query dims lane group kg holds for k-block i
    __device__ static int q_dim(int i, int kg) { return 32 * i + 8 * kg; }
    __device__ static void load(Buf& b, const uint8_t* ks, const uint8_t* vs, int lane, int row)
    {
        const int koff = (lane & 15) * row + 16 * (lane >> 4);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            b.k[i] = load_stream16(ks + koff + 64 * i);
        const int voff = (lane >> 4) * row + 16 * (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            b.v[i] = load_stream16(vs + 4 * row * i + voff);
    }
    __device__ static uint4 k_block(const Buf& b, int i) { return b.k[i]; }
    __device__ static void values(const Buf& b, int k, float (&v)[8]) { unpack8(b.v[k], v); }
    __device__ static void clear_values(Buf& b, int k) { b.v[k] = make_uint4(0, 0, 0, 0); }
    // dims 8c..8c+7 of token 4k + r as eight bf16
    __device__ static uint4 values_bf16(const Buf& b, int k) { return b.v[k]; }
};

// OCP e4m3 slab: 2 KiB.  K: two 16-byte loads per lane (dims 16kg..16kg+15 and
// 64+16kg..64+16kg+15 of token l%16); each 8-code half converts exactly to
// bf16 for one k-block.  V: four 8-byte loads per lane in the value layout,
// converted to fp32.  The slab scales stay out of the conversions: k_scale
// multiplies the score and v_scale the probability.
struct KvFp8 {
    static constexpr bool kScaled = true;
    struct Buf {
        uint4 k[2];
        uint2 v[4];
    };
    __device__ static int q_dim(int i, int kg) { return (i >> 1) * 64 + 16 * kg + (i & 1) * 8; }
    __device__ static void load(Buf& b, const uint8_t* ks, const uint8_t* vs, int lane, int row)
    {
        const int koff = (lane & 15) * row + 16 * (lane >> 4);
        b.k[0] = load_stream16(ks + koff);
        b.k[1] = load_stream16(ks + koff + 64);
        const int voff = (lane >> 4) * row + 8 * (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            b.v[i] = load_stream8(vs + 4 * row * i + voff);
    }
    // Two e4m3 codes (bytes 2*HI, 2*HI+1 of x) as a bf16 pair; exact.
    template <bool HI>
    __device__ static uint32_t cvt2(uint32_t x)
    {
        return __builtin_bit_cast(uint32_t,
                                  __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, HI));
    }
    __device__ static uint4 k_block(const Buf& b, int i)
    {
        const uint4& w = b.k[i >> 1];
        const uint32_t lo = (i & 1) ? w.z : w.x;
        const uint32_t hi = (i & 1) ? w.w : w.y;
        return make_uint4(cvt2<false>(lo), cvt2<true>(lo), cvt2<false>(hi), cvt2<true>(hi));
    }
    __device__ static void values(const Buf& b, int k, float (&v)[8])
    {
        const floatx2_t a0 = __builtin_amdgcn_cvt_pk_f32_fp8(b.v[k].x, false);
        const floatx2_t a1 = __builtin_amdgcn_cvt_pk_f32_fp8(b.v[k].x, true);
        const floatx2_t a2 = __builtin_amdgcn_cvt_pk_f32_fp8(b.v[k].y, false);
        const floatx2_t a3 = __builtin_amdgcn_cvt_pk_f32_fp8(b.v[k].y, true);
        v[0] = a0.x; v[1] = a0.y; v[2] = a1.x; v[3] = a1.y;
        v[4] = a2.x; v[5] = a2.y; v[6] = a3.x; v[7] = a3.y;
    }
    __device__ static void clear_values(Buf& b, int k) { b.v[k] = make_uint2(0, 0); }
};

// The same e4m3 slab read as whole rows, for the matrix-core value pass: lane
// l loads codes 16(l%8)..16(l%8)+15 of tokens l/8 and 8 + l/8, for K and for
// V, so each load instruction covers eight complete 128-byte rows.  K reaches
// the score layout above (k[0], k[1]) through the wavefront's staging tile
// (kStagedK) before its k-blocks are taken; V is widened to bf16 as it is
// staged.  On gfx950 this reads the pool measurably faster than the
// score-layout loads, which touch sixteen rows per instruction.
struct KvFp8Rows {
    static constexpr bool kScaled = true;
    static constexpr bool kStagedK = true;
    struct Buf {
        uint4 k[2];
        uint4 v[2];
    };
    __device__ static int q_dim(int i, int kg) { return KvFp8::q_dim(i, kg); }
    __device__ static void load(Buf& b, const uint8_t* ks, const uint8_t* vs, int lane, int row)
    {
        const int off = (lane >> 3) * row + 16 * (lane & 7);
        b.k[0] = load_stream16(ks + off);
        b.k[1] = load_stream16(ks + off + 8 * row);
        b.v[0] = load_stream16(vs + off);
        b.v[1] = load_stream16(vs + off + 8 * row);
    }
    // k-block i once k[] holds the score layout
    __device__ static uint4 k_block(const Buf& b, int i)
    {
        const uint4& w = b.k[i >> 1];
        const uint32_t lo = (i & 1) ? w.z : w.x;
        const uint32_t hi = (i & 1) ? w.w : w.y;
        return make_uint4(KvFp8::cvt2<false>(lo), KvFp8::cvt2<true>(lo),
                          KvFp8::cvt2<false>(hi), KvFp8::cvt2<true>(hi));
    }
    // codes 16(l%8) + 8h .. +7 of token 8j + l/8 as exact bf16
    __device__ static uint4 values_bf16(const Buf& b, int j, int h)
    {
        const uint32_t lo = h ? b.v[j].z : b.v[j].x;
        const uint32_t hi = h ? b.v[j].w : b.v[j].y;
        return make_uint4(KvFp8::cvt2<false>(lo), KvFp8::cvt2<true>(lo),
                          KvFp8::cvt2<false>(hi), KvFp8::cvt2<true>(hi));
    }
};

// ------------------------------------------------ split kernel, MFMA QK ---
//
// Query head g sits in row 4g of the 16-row query tile, so after the four
// MFMAs of a page lane l holds score (g = l/16, token l%16) in its first
// accumulator.  The probabilities cross from that layout to the value layout
// through 272 bytes of LDS per wavefront.
//
// The running max m of each query head moves only when a page's max exceeds
// it by more than kMaxSlack (log2 units); between moves the probabilities
// 2^(s - m) may exceed 1 (by at most 2^kMaxSlack) and the accumulators need no
// rescaling, so the rescale and its LDS exchange run only on the rare pages
// where some head's max moves.  Results are the same up to fp32 rounding: m
// cancels in acc / l.

// Rows of the 16-row query tile that hold a query head: every 4th row for
// G <= 4 (one score per lane of the first G lane groups), every 2nd row for
// G = 8 (two scores per lane).
template <int G>
struct ScoreRows {
    static constexpr int kStep = G > 8 ? 1 : G > 4 ? 2 : 4;  // head g sits in row kStep * g
    static constexpr int kPerLane = 4 / kStep;              // scores per lane
    static constexpr int kLdsHeads = G > 4 ? 8 : 4;         // p/alpha entries per token in LDS
};

// One wavefront's pass over its pages of one (sequence, kv head): the pages
// are t.p0 + t.wave + PAGE_STEP * i for the four-wavefront units (at most
// kWave of them, block-table entries in my_page) and t.p0 + i for the
// head-parallel units (PAGE_STEP 1, wave index not part of the page), which
// take their block-table entries kWave pages at a time: my_page holds the
// first kWave on entry.  On return every lane holds the wave's full acc for
// dims 8c..8c+7 of all G heads, and lane group kg holds (m, l) of heads
// head[e].
template <int G, bool CHECKED, typename KV, int PAGE_STEP>
__device__ __forceinline__ void attend_pages(const SplitArgs& a, const WaveTask& t,
                                             int32_t my_page, float* lds_p, float* lds_alpha,
                                             float (&acc)[G][8],
                                             float (&m)[ScoreRows<G>::kPerLane],
                                             float (&l_row)[ScoreRows<G>::kPerLane],
                                             int (&head)[ScoreRows<G>::kPerLane])
{
    using SR = ScoreRows<G>;
    constexpr int kE = SR::kPerLane;
    constexpr int kH = SR::kLdsHeads;
    const int lane = t.lane;
    const int n = lane & 15, kg = lane >> 4;  // score layout
    const int r = lane >> 4;                  // value layout row
    const int h0 = t.kvh * G;
    constexpr bool kChunked = PAGE_STEP == 1;
    const int first = kChunked ? t.p0 : t.p0 + t.wave;
    int c0 = 0;  // wavefront-local index of my_page's first entry
    float my_kscale = 1.0f, my_vscale = 1.0f;

    // Query tile: row kStep*g holds query head g, every other row is zero.
    uint4 qa[4];
    {
        const int row = lane & 15;
        const int g = row / SR::kStep;
        const bool has = row % SR::kStep == 0 && g < G;
        const uint16_t* qrow =
            a.q + ((int64_t)t.b * a.num_q_heads + h0 + (has ? g : 0)) * kHeadDim;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            qa[i] = has ? *reinterpret_cast<const uint4*>(qrow + KV::q_dim(i, kg))
                        : make_uint4(0, 0, 0, 0);
    }
    // Head of this lane's e-th score: tile row 4kg + e*kStep.
#pragma unroll
    for (int e = 0; e < kE; ++e)
        head[e] = (4 * kg + e * SR::kStep) / SR::kStep;

    float lsum[kE];    // this lane's share of l
#pragma unroll
    for (int e = 0; e < kE; ++e) {
        m[e] = -INFINITY;    // reference max (log2 units)
        lsum[e] = 0.0f;
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int d = 0; d < 8; ++d)
            acc[g][d] = 0.0f;

    auto issue = [&](typename KV::Buf& buf, int i) {
        const int64_t page = __builtin_amdgcn_readlane(my_page, i);
        KV::load(buf, slab_base(a, a.k_pool, page, t.kvh), slab_base(a, a.v_pool, page, t.kvh),
                 lane, a.row_bytes);
    };

    // i: index within the current run of my_page entries
    auto consume = [&](typename KV::Buf& buf, int i) {
        // Scores of the 16 tokens of the page for the G query heads.
        floatx4_t sacc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < 4; ++k)
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, qa[k]),
                __builtin_bit_cast(bf16x8_t, KV::k_block(buf, k)), sacc, 0, 0, 0);

        const int page_idx = first + PAGE_STEP * ((kChunked ? c0 : 0) + i);
        const int valid = t.seq_len - page_idx * kPageSize;  // >= 1 valid tokens
        float sl = a.scale_log2;
        if (KV::kScaled)
            sl *= __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_kscale), i));
        float s[kE], mx[kE];
        bool grow = false;
#pragma unroll
        for (int e = 0; e < kE; ++e) {
            s[e] = (n < valid) ? sacc[e * SR::kStep] * sl : -INFINITY;
            mx[e] = row16_max(s[e]);  // finite: token 0 is valid
            grow |= mx[e] > m[e] + kMaxSlack;
        }
        if (__any(grow)) {
#pragma unroll
            for (int e = 0; e < kE; ++e) {
                const float m_new = mx[e] > m[e] + kMaxSlack ? mx[e] : m[e];
                const float alpha = exp2_fast(m[e] - m_new);  // 0 on the first page
                lsum[e] *= alpha;
                m[e] = m_new;
                if (n == 0)
                    lds_alpha[head[e]] = alpha;
            }
            wave_lds_sync();
            float alv[kH];
#pragma unroll
            for (int q4 = 0; q4 < kH / 4; ++q4) {
                const float4 al = *reinterpret_cast<const float4*>(&lds_alpha[4 * q4]);
                alv[4 * q4] = al.x;
                alv[4 * q4 + 1] = al.y;
                alv[4 * q4 + 2] = al.z;
                alv[4 * q4 + 3] = al.w;
            }
            wave_lds_sync();
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int d = 0; d < 8; ++d)
                    acc[g][d] *= alv[g];
        }
        float vs = 1.0f;
        if (KV::kScaled)
            vs = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_vscale), i));
#pragma unroll
        for (int e = 0; e < kE; ++e) {
            const float pexp = exp2_fast(s[e] - m[e]);
            lsum[e] += pexp;
            lds_p[n * kH + head[e]] = pexp * vs;
        }
        wave_lds_sync();
        float pv[4][kH];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int q4 = 0; q4 < kH / 4; ++q4) {
                const float4 x =
                    *reinterpret_cast<const float4*>(&lds_p[(4 * k + r) * kH + 4 * q4]);
                pv[k][4 * q4] = x.x;
                pv[k][4 * q4 + 1] = x.y;
                pv[k][4 * q4 + 2] = x.z;
                pv[k][4 * q4 + 3] = x.w;
            }
        wave_lds_sync();

        if (valid < kPageSize) {
#pragma unroll
            for (int k = 0; k < 4; ++k)
                if (4 * k + r >= valid)
                    KV::clear_values(buf, k);  // unread slots may hold NaN
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            float v[8];
            KV::values(buf, k, v);
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int d = 0; d < 8; ++d)
                    acc[g][d] = fmaf(pv[k][g], v[d], acc[g][d]);
        }
    };

    typename KV::Buf buf_a, buf_b;
    for (;;) {
        const int n_here = kChunked ? min(t.count - c0, kWave) : t.count;
        // slab scales of these pages, one per lane like the pages
        if (KV::kScaled && lane < n_here) {
            const int64_t slab = (int64_t)my_page * a.num_kv_heads + t.kvh;
            my_kscale = a.k_scale[slab];
            my_vscale = a.v_scale[slab];
        }
        stream_pages(n_here, buf_a, buf_b, issue, consume);
        if (!kChunked)
            break;
        c0 += kWave;
        if (c0 >= t.count)
            break;
        // the next kWave block-table entries
        my_page = c0 + lane < t.count
                      ? a.block_table[(int64_t)t.b * a.max_pages + t.p0 + c0 + lane]
                      : 0;
        if (CHECKED) {
            const bool bad =
                c0 + lane < t.count && (my_page < 0 || (int64_t)my_page >= a.num_pages);
            if (__any(bad)) {
                if (lane == 0)
                    atomicOr(a.dev_error, RL_DA_DEVERR_PAGE_OUT_OF_RANGE);
                break;  // the rest is skipped; the output is unspecified
            }
        }
    }

    // Every lane of a value row holds a partial over tokens = r (mod 4); all
    // rows share the reference max, so the partials simply add.
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int d = 0; d < 8; ++d) {
            float v = acc[g][d];
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
            acc[g][d] = v;
        }
#pragma unroll
    for (int e = 0; e < kE; ++e)
        l_row[e] = row16_sum(lsum[e]);
}

// Three wavefronts per SIMD (two for G = 8): the register budget fits both
// page buffers and the accumulators without spilling.
// A persistent work-group keeps values live across its units; it takes the
// two-wave register budget, which holds them without spilling.
template <int G, bool CHECKED, typename KV, bool PERSISTENT>
__global__ __launch_bounds__(kWave * kUnitWaves)
__attribute__((amdgpu_waves_per_eu(G > 4 || PERSISTENT ? 2 : 3))) void split_mfma(SplitArgs a)
{
    static_assert(G == 1 || G == 2 || G == 4 || G == 8, "query group of 1, 2, 4 or 8 heads");
    using SR = ScoreRows<G>;
    constexpr int kE = SR::kPerLane;
    constexpr int kH = SR::kLdsHeads;
    __shared__ __attribute__((aligned(16))) float lds_p_all[kUnitWaves][kPageSize * kH];
    __shared__ __attribute__((aligned(16))) float lds_alpha_all[kUnitWaves][kH];
    __shared__ __attribute__((aligned(16))) UnitShared<G> sh;
    extern __shared__ int plan[];

    auto unit = [&](const SplitArgs& a, int b, int kvh, int s, bool owner) {
        WaveTask t;
        int32_t my_page;
        if (!begin_unit<CHECKED>(a, t, my_page, b, kvh, s, owner)) {
            write_zero_rows<G>(a, t);
            return;
        }
        float acc[G][8], m[kE], l_row[kE];
        int head[kE];
        attend_pages<G, CHECKED, KV, kUnitWaves>(a, t, my_page, lds_p_all[t.wave],
                                                 lds_alpha_all[t.wave], acc, m, l_row, head);
        // Lane group kg holds m and l of heads head[e]; its value lanes (r = kg)
        // stash those heads.
        const int c = t.lane & 15;
#pragma unroll
        for (int e = 0; e < kE; ++e) {
#pragma unroll
            for (int g = 0; g < G; ++g)
                if (g == head[e])
                    stash_state<G>(sh, t.wave, g, c, acc[g], m[e], l_row[e]);
        }
        __syncthreads();
        merge_unit<G>(a, t, sh);
    };
    if (PERSISTENT)
        run_persistent(a, a.num_kv_heads, plan, unit);
    else  // one split per sequence: unit (b, kv head) = blockIdx.x
        unit(a, blockIdx.x / a.num_kv_heads, blockIdx.x % a.num_kv_heads, 0, true);
}

// ------------------------------------- head-parallel split kernel, MFMA QK ---
//
// For token-major pools, where a (page, kv head) slab is 16 rows spread over
// the page, the four-wavefront unit of one kv head reads 256-byte pieces
// (128 for e4m3) of pages whose other heads are read by other units at other
// times.  Here one work-group covers (sequence, split, group of kHeadsPerUnit
// consecutive kv heads): wavefront w owns kv head group * kHeadsPerUnit + w
// and walks every page of the split, so the group's wavefronts read each
// page's token rows together (one contiguous run per row).  No merge inside
// the unit: each wavefront finishes its own heads, or writes one partial per
// split for the merge kernel.

template <bool CHECKED>
__device__ __forceinline__ bool begin_unit_hp(const SplitArgs& a, WaveTask& t, int32_t& my_page,
                                              int b, int group, int s, bool owner)
{
    t.lane = threadIdx.x % kWave;
    t.wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform: scalar
    t.kvh = __builtin_amdgcn_readfirstlane(group * a.heads_per_unit + t.wave);
    t.b = b;
    t.owner = owner;
    t.s = max(s, 0);
    t.p0 = t.s * a.split_pages;
    // the first kWave pages' block-table entries (later ones are loaded as
    // the wavefront reaches them)
    auto load_pages = [&] {
        const int col = t.p0 + t.lane;
        const bool in_split = t.lane < a.split_pages && col < a.max_pages;
        my_page = in_split ? a.block_table[(int64_t)t.b * a.max_pages + col] : 0;
    };
    if (s >= 0)
        load_pages();
    int L = __builtin_amdgcn_readfirstlane(a.seq_lens[t.b]);  // uniform: scalar
    const int cap = a.max_pages * kPageSize;
    if (L > cap) {
        if (CHECKED && t.lane == 0 && t.owner && t.kvh == 0)
            atomicOr(a.dev_error, RL_DA_DEVERR_LENGTH_TOO_LONG);
        L = cap;
    }
    t.seq_len = L;
    t.npages = L > 0 ? (L + kPageSize - 1) / kPageSize : 0;
    t.nsplit = (t.npages + a.split_pages - 1) / a.split_pages;
    if (s < 0) {
        if (t.nsplit == 0)
            return false;
        t.s = t.nsplit - 1;
        t.p0 = t.s * a.split_pages;
        load_pages();
    }
    const int p1 = min(t.p0 + a.split_pages, t.npages);
    if (t.p0 >= p1)
        return false;
    t.count = p1 - t.p0;
    if (CHECKED) {
        const bool bad = t.lane < min(t.count, kWave) &&
                         (my_page < 0 || (int64_t)my_page >= a.num_pages);
        if (__any(bad)) {
            if (t.lane == 0)
                atomicOr(a.dev_error, RL_DA_DEVERR_PAGE_OUT_OF_RANGE);
            t.count = 0;  // read nothing; the wavefront's output is unspecified
        }
    }
    return true;
}

// A work-group of up to eight wavefronts fills two waves per SIMD, so the
// kernel may use the two-wave register budget.
template <int G, bool CHECKED, typename KV, bool PERSISTENT>
__global__ __launch_bounds__(kWave * kMaxHeadsPerUnit)
__attribute__((amdgpu_waves_per_eu(2))) void split_mfma_hp(SplitArgs a)
{
    static_assert(G == 1 || G == 2 || G == 4 || G == 8, "query group of 1, 2, 4 or 8 heads");
    using SR = ScoreRows<G>;
    constexpr int kE = SR::kPerLane;
    constexpr int kH = SR::kLdsHeads;
    __shared__ __attribute__((aligned(16))) float lds_p_all[kMaxHeadsPerUnit][kPageSize * kH];
    __shared__ __attribute__((aligned(16))) float lds_alpha_all[kMaxHeadsPerUnit][kH];

    extern __shared__ int plan[];

    auto unit = [&](const SplitArgs& a, int b, int group, int s, bool owner) {
        WaveTask t;
        int32_t my_page;
        if (!begin_unit_hp<CHECKED>(a, t, my_page, b, group, s, owner)) {
            // an empty sequence produces zeros, written by its owner unit
            if (t.npages == 0 && t.owner)
                for (int e = t.lane; e < G * (kHeadDim / 8); e += kWave) {
                    const int g = e / (kHeadDim / 8), chunk = e % (kHeadDim / 8);
                    *reinterpret_cast<uint4*>(
                        a.out + ((int64_t)t.b * a.num_q_heads + t.kvh * G + g) * kHeadDim +
                        chunk * 8) = make_uint4(0, 0, 0, 0);
                }
            return;
        }
        float acc[G][8], m[kE], l_row[kE];
        int head[kE];
        attend_pages<G, CHECKED, KV, 1>(a, t, my_page, lds_p_all[t.wave], lds_alpha_all[t.wave],
                                        acc, m, l_row, head);
        // Lane 16kg + c writes dims 8c..8c+7 of the heads its lane group holds.
        const int c = t.lane & 15;
    #pragma unroll
        for (int e = 0; e < kE; ++e) {
    #pragma unroll
            for (int g = 0; g < G; ++g) {
                if (g != head[e])
                    continue;
                const int64_t row = (int64_t)t.b * a.num_q_heads + t.kvh * G + g;
                if (t.nsplit == 1) {
                    const float inv = 1.0f / l_row[e];
                    uint4 o;
                    o.x = f32_to_bf16(acc[g][0] * inv) | (f32_to_bf16(acc[g][1] * inv) << 16);
                    o.y = f32_to_bf16(acc[g][2] * inv) | (f32_to_bf16(acc[g][3] * inv) << 16);
                    o.z = f32_to_bf16(acc[g][4] * inv) | (f32_to_bf16(acc[g][5] * inv) << 16);
                    o.w = f32_to_bf16(acc[g][6] * inv) | (f32_to_bf16(acc[g][7] * inv) << 16);
                    *reinterpret_cast<uint4*>(a.out + row * kHeadDim + 8 * c) = o;
                } else {
                    const int64_t part = row * a.num_splits + t.s;
                    float4* dst = reinterpret_cast<float4*>(a.ws_acc + part * kHeadDim + 8 * c);
                    dst[0] = make_float4(acc[g][0], acc[g][1], acc[g][2], acc[g][3]);
                    dst[1] = make_float4(acc[g][4], acc[g][5], acc[g][6], acc[g][7]);
                    if (c == 0)
                        *reinterpret_cast<float2*>(a.ws_ml + part * 2) = make_float2(m[e], l_row[e]);
                }
            }
        }
    };
    const int groups = a.num_kv_heads / a.heads_per_unit;
    if (PERSISTENT)
        run_persistent(a, groups, plan, unit);
    else  // one split per sequence: unit (b, head group) = blockIdx.x
        unit(a, blockIdx.x / groups, blockIdx.x % groups, 0, true);
}

// ------------------------------------------- split kernel, VALU dot2 QK ---
//
// Lane l = 16r + c holds dims 8c..8c+7 of tokens 4i + r (i = 0..3) for both
// K and V.  Partial dots over those 8 dims (bf16 dot2) are summed over the 16
// lanes of the row with DPP; each row r keeps its own online softmax over its
// tokens and the four rows are merged with the log-sum-exp rule at the end.

template <int G, bool CHECKED, bool PERSISTENT>
__global__ __launch_bounds__(kWave * kUnitWaves) void split_valu_bf16(SplitArgs a)
{
    __shared__ __attribute__((aligned(16))) UnitShared<G> sh;
    extern __shared__ int plan[];

    auto unit = [&](const SplitArgs& a, int b, int kvh, int s, bool owner) {
        WaveTask t;
        int32_t my_page;
        if (!begin_unit<CHECKED>(a, t, my_page, b, kvh, s, owner)) {
            write_zero_rows<G>(a, t);
            return;
        }

        const int lane = t.lane;
        const int r = lane >> 4, c = lane & 15;
        const int h0 = t.kvh * G;

        uint4 qv[G];
    #pragma unroll
        for (int g = 0; g < G; ++g)
            qv[g] = *reinterpret_cast<const uint4*>(
                a.q + ((int64_t)t.b * a.num_q_heads + h0 + g) * kHeadDim + 8 * c);

        float m[G], l[G], acc[G][8];
    #pragma unroll
        for (int g = 0; g < G; ++g) {
            m[g] = -INFINITY;
            l[g] = 0.0f;
    #pragma unroll
            for (int d = 0; d < 8; ++d)
                acc[g][d] = 0.0f;
        }

        const int off = r * a.row_bytes + 16 * c;
        const int step = 4 * a.row_bytes;
        auto issue = [&](KvBf16::Buf& buf, int i) {
            const int64_t page = __builtin_amdgcn_readlane(my_page, i);
            const uint8_t* ks = slab_base(a, a.k_pool, page, t.kvh);
            const uint8_t* vs = slab_base(a, a.v_pool, page, t.kvh);
    #pragma unroll
            for (int k = 0; k < 4; ++k)
                buf.k[k] = load_stream16(ks + step * k + off);
    #pragma unroll
            for (int k = 0; k < 4; ++k)
                buf.v[k] = load_stream16(vs + step * k + off);
        };

        auto consume = [&](KvBf16::Buf& buf, int i) {
            uint4 (&kbuf)[4] = buf.k;
            uint4 (&vbuf)[4] = buf.v;
            const int valid = t.seq_len - task_page(t, i) * kPageSize;
            float sc[G][4];
    #pragma unroll
            for (int g = 0; g < G; ++g)
    #pragma unroll
                for (int k = 0; k < 4; ++k) {
                    float x = dot2_bf16(qv[g].x, kbuf[k].x, 0.0f);
                    x = dot2_bf16(qv[g].y, kbuf[k].y, x);
                    x = dot2_bf16(qv[g].z, kbuf[k].z, x);
                    x = dot2_bf16(qv[g].w, kbuf[k].w, x);
                    x = row16_sum(x) * a.scale_log2;
                    sc[g][k] = (4 * k + r < valid) ? x : -INFINITY;
                }

            float p[G][4];
    #pragma unroll
            for (int g = 0; g < G; ++g) {
                const float mx = fmaxf(fmaxf(sc[g][0], sc[g][1]), fmaxf(sc[g][2], sc[g][3]));
                const float m_new = fmaxf(m[g], mx);
                // A row may see no valid token of a short last page: keep it empty.
                const bool empty = m_new == -INFINITY;
                const float alpha = empty ? 1.0f : exp2_fast(m[g] - m_new);
                float sum = 0.0f;
    #pragma unroll
                for (int k = 0; k < 4; ++k) {
                    p[g][k] = empty ? 0.0f : exp2_fast(sc[g][k] - m_new);
                    sum += p[g][k];
                }
                l[g] = l[g] * alpha + sum;
                m[g] = m_new;
    #pragma unroll
                for (int d = 0; d < 8; ++d)
                    acc[g][d] *= alpha;
            }

            if (valid < kPageSize) {
    #pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (4 * k + r >= valid)
                        vbuf[k] = make_uint4(0, 0, 0, 0);
            }
    #pragma unroll
            for (int k = 0; k < 4; ++k) {
                float v[8];
                unpack8(vbuf[k], v);
    #pragma unroll
                for (int g = 0; g < G; ++g)
    #pragma unroll
                    for (int d = 0; d < 8; ++d)
                        acc[g][d] = fmaf(p[g][k], v[d], acc[g][d]);
            }
        };

        KvBf16::Buf buf_a, buf_b;
        stream_pages(t.count, buf_a, buf_b, issue, consume);

        // Merge the four rows: rescale each to the common max, then add.  A
        // wavefront without pages keeps m = -inf, l = 0, acc = 0.
    #pragma unroll
        for (int g = 0; g < G; ++g) {
            float M = fmaxf(m[g], __shfl_xor(m[g], 16));
            M = fmaxf(M, __shfl_xor(M, 32));
            const float w = (m[g] == -INFINITY) ? 0.0f : exp2_fast(m[g] - M);
            float lw = l[g] * w;
            lw += __shfl_xor(lw, 16);
            lw += __shfl_xor(lw, 32);
            l[g] = lw;
            m[g] = M;
    #pragma unroll
            for (int d = 0; d < 8; ++d) {
                float v = acc[g][d] * w;
                v += __shfl_xor(v, 16);
                v += __shfl_xor(v, 32);
                acc[g][d] = v;
            }
        }
    #pragma unroll
        for (int g = 0; g < G; ++g)
            if ((g & 3) == r)
                stash_state<G>(sh, t.wave, g, c, acc[g], m[g], l[g]);
        __syncthreads();
        merge_unit<G>(a, t, sh);
    };
    if (PERSISTENT)
        run_persistent(a, a.num_kv_heads, plan, unit);
    else  // one split per sequence: unit (b, kv head) = blockIdx.x
        unit(a, blockIdx.x / a.num_kv_heads, blockIdx.x % a.num_kv_heads, 0, true);
}

// ----------------------------------- split kernel, MFMA scores and MFMA PV ---
//
// Both contractions on the matrix cores.  Per page a wavefront forms the
// scores of the query tile as split_mfma does (head g in row kStep * g; for
// G = 16 every row is a head), then accumulates
//     O^T[dim][row] += V^T[dim][token] P^T[token][row]
// with v_mfma_f32_16x16x16_bf16, one product per 16-dim block.  V^T comes
// from the page's values staged in wavefront-private LDS as [token][dim]
// rows, read back with the LDS transpose read (lane 16q + j: tokens
// 4q..4q+3 of dim 16i + j); P^T from the probabilities staged as [row][token]
// rows (lane 16q + j: row j, tokens 4q..4q+3).  P enters the product as two
// bf16 terms, hi = bf16(p) and lo = bf16(p - hi), so the weights carry p to
// 2^-16 relative; the normaliser l sums the fp32 probabilities.  The
// accumulators take 32 registers per lane whatever the group size (lane
// 16q + j holds row j, dims 16i + 4q .. 16i + 4q + 3): what lets a group of 16
// query heads run, whose value pass on the vector ALUs would need 16 x 8
// accumulators per lane.  e4m3 values are widened exactly to bf16 as they are
// staged; v_scale multiplies p before the split.

constexpr int kPvVRow = kHeadDim + 16;  // bf16 per staged value row (288 bytes)
constexpr int kPvKRowBytes = 128;        // staged e4m3 key row pitch (bytes)
constexpr int kPvPRow = 20;             // floats per staged probability row (80 bytes)
// Staged rows keep their 16-byte chunks at swizzled positions so that the
// 16-byte reads of the value pass meet no bank conflict (ds_read_b128 serves
// lanes l, l ^ 1, l ^ 2, l ^ 20, l ^ 24 and their combinations together, as
// measured on gfx950): key row r, chunk c at c ^ (r >> 1); probability row
// r, chunk c at c ^ pv_p_swizzle(r).  The probabilities' one-float writes
// (a wavefront's 64 lanes at once) stay conflict-free with 80-byte rows.
__device__ __forceinline__ int pv_p_swizzle(int r) { return ((r >> 2) ^ (r >> 3)) & 1; }

struct PvWaveLds {
    uint16_t v[kPageSize * kPvVRow];
    float p[16 * kPvPRow];
    float alpha[16];
};

// The per-wavefront tiles of the page loop and the unit merge's state share
// the work-group's LDS: the merge runs after every wavefront has left its
// loop.
template <int G>
union PvShared {
    PvWaveLds wave[kUnitWaves];
    UnitShared<G> unit;
};

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4_t;

// Four bf16 of one dim from four consecutive rows of a [row][dim] LDS tile
// (ds_read_b64_tr_b16): within each 16-lane group, lane j receives element
// j % 4 of the 8-byte chunks addressed by lanes j / 4 + 4e, e = 0..3, so when
// lane s addresses row (base + s / 4), dims (d0 + 4 (s % 4)) .. +3, lane j
// gets rows base .. base + 3 of dim d0 + j.
__device__ __forceinline__ short4_t lds_read_tr16(const uint16_t* p)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_t*)p);
}

// Four fp32 weights as the two bf16 terms of the PV product.
__device__ __forceinline__ void split_bf16(const float4& p, short4_t& hi, short4_t& lo)
{
    const uint32_t h0 = pack_bf16x2(p.x, p.y), h1 = pack_bf16x2(p.z, p.w);
    const uint32_t l0 = pack_bf16x2(p.x - bf16_lo(h0), p.y - bf16_hi(h0));
    const uint32_t l1 = pack_bf16x2(p.z - bf16_lo(h1), p.w - bf16_hi(h1));
    hi = __builtin_bit_cast(short4_t, make_uint2(h0, h1));
    lo = __builtin_bit_cast(short4_t, make_uint2(l0, l1));
}

// One wavefront's pass over its pages (p0 + wave + 4i) of one (sequence, kv
// head).  On return o[i] holds, for lane 16q + j, tile row j's unnormalised
// output at dims 16i + 4q .. +3, and the lanes of score group kg hold (m, l)
// of tile rows 4kg + e kStep.
template <int G, bool CHECKED, typename KV>
__device__ __forceinline__ void attend_pages_pv(const SplitArgs& a, const WaveTask& t,
                                                int32_t my_page, PvWaveLds& lds,
                                                floatx4_t (&o)[kHeadDim / 16],
                                                float (&m)[ScoreRows<G>::kPerLane],
                                                float (&l_row)[ScoreRows<G>::kPerLane])
{
    using SR = ScoreRows<G>;
    constexpr int kE = SR::kPerLane;
    const int lane = t.lane;
    const int n = lane & 15, kg = lane >> 4;  // score layout: token n, rows 4kg + e kStep
    const int r = lane >> 4, c = lane & 15;   // value layout: token 4k + r, dims 8c..8c+7
    const int h0 = t.kvh * G;
    float my_kscale = 1.0f, my_vscale = 1.0f;

    uint4 qa[4];
    {
        const int row = lane & 15;
        const int g = row / SR::kStep;
        const bool has = row % SR::kStep == 0 && g < G;
        const uint16_t* qrow =
            a.q + ((int64_t)t.b * a.num_q_heads + h0 + (has ? g : 0)) * kHeadDim;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            qa[i] = has ? *reinterpret_cast<const uint4*>(qrow + KV::q_dim(i, kg))
                        : make_uint4(0, 0, 0, 0);
    }
    bool real[kE];  // the lane's e-th score row holds a query head
#pragma unroll
    for (int e = 0; e < kE; ++e)
        real[e] = (4 * kg + e * SR::kStep) / SR::kStep < G;

    // rows that hold no head keep zero weights; alpha starts at 1
#pragma unroll
    for (int x = lane; x < 16 * kPvPRow; x += kWave)
        lds.p[x] = 0.0f;
    if (lane < 16)
        lds.alpha[lane] = 1.0f;

    float lsum[kE];
#pragma unroll
    for (int e = 0; e < kE; ++e) {
        m[e] = -INFINITY;
        lsum[e] = 0.0f;
    }
#pragma unroll
    for (int i = 0; i < kHeadDim / 16; ++i)
        o[i] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};

    auto issue = [&](typename KV::Buf& buf, int i) {
        const int64_t page = __builtin_amdgcn_readlane(my_page, i);
        KV::load(buf, slab_base(a, a.k_pool, page, t.kvh), slab_base(a, a.v_pool, page, t.kvh),
                 lane, a.row_bytes);
    };

    auto consume = [&](typename KV::Buf& buf, int i) {
        const int valid = t.seq_len - task_page(t, i) * kPageSize;  // >= 1 valid tokens
        if constexpr (KV::kStagedK) {
            // whole key rows pass through the value tile into the score
            // layout; the values replace them there once they are read
            wave_lds_sync();  // the previous page's tiles have been read
            uint8_t* tile = reinterpret_cast<uint8_t*>(lds.v);
            const int tr = lane >> 3, tc = 16 * (lane & 7);
            *reinterpret_cast<uint4*>(tile + tr * kPvKRowBytes + 16 * ((lane & 7) ^ (tr >> 1))) =
                buf.k[0];
            *reinterpret_cast<uint4*>(tile + (8 + tr) * kPvKRowBytes +
                                      16 * ((lane & 7) ^ ((8 + tr) >> 1))) = buf.k[1];
            wave_lds_sync();
            buf.k[0] = *reinterpret_cast<const uint4*>(tile + n * kPvKRowBytes +
                                                       16 * (kg ^ (n >> 1)));
            buf.k[1] = *reinterpret_cast<const uint4*>(tile + n * kPvKRowBytes +
                                                       16 * ((4 + kg) ^ (n >> 1)));
            wave_lds_sync();
            // the page's values as [token][dim] rows; unread slots may hold NaN
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                uint4 v0 = KV::values_bf16(buf, j, 0), v1 = KV::values_bf16(buf, j, 1);
                if (valid < kPageSize && 8 * j + tr >= valid) {
                    v0 = make_uint4(0, 0, 0, 0);
                    v1 = v0;
                }
                *reinterpret_cast<uint4*>(&lds.v[(8 * j + tr) * kPvVRow + tc]) = v0;
                *reinterpret_cast<uint4*>(&lds.v[(8 * j + tr) * kPvVRow + tc + 8]) = v1;
            }
        }
        floatx4_t sacc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < 4; ++k)
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, qa[k]),
                __builtin_bit_cast(bf16x8_t, KV::k_block(buf, k)), sacc, 0, 0, 0);

        float sl = a.scale_log2;
        if (KV::kScaled)
            sl *= __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_kscale), i));
        float s[kE], mx[kE];
        bool grow = false;
#pragma unroll
        for (int e = 0; e < kE; ++e) {
            s[e] = (n < valid) ? sacc[e * SR::kStep] * sl : -INFINITY;
            mx[e] = row16_max(s[e]);  // finite: token 0 is valid
            grow |= real[e] && mx[e] > m[e] + kMaxSlack;
        }
        if constexpr (!KV::kStagedK)
            wave_lds_sync();  // the previous page's tiles have been read
        const bool rescale = __any(grow);
        if (rescale) {
#pragma unroll
            for (int e = 0; e < kE; ++e) {
                const float m_new = mx[e] > m[e] + kMaxSlack ? mx[e] : m[e];
                const float alpha = exp2_fast(m[e] - m_new);  // 0 on the first page
                lsum[e] *= alpha;
                m[e] = m_new;
                if (n == 0 && real[e])
                    lds.alpha[4 * kg + e * SR::kStep] = alpha;
            }
        }
        float vs = 1.0f;
        if (KV::kScaled)
            vs = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_vscale), i));
#pragma unroll
        for (int e = 0; e < kE; ++e) {
            const float pexp = exp2_fast(s[e] - m[e]);
            lsum[e] += pexp;
            if (real[e])
                {
                    const int pr = 4 * kg + e * SR::kStep;
                    lds.p[pr * kPvPRow + 4 * ((n >> 2) ^ pv_p_swizzle(pr)) + (n & 3)] = pexp * vs;
                }
        }
        // the page's values as [token][dim] rows; unread slots may hold NaN
        if constexpr (!KV::kStagedK) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                uint4 v = KV::values_bf16(buf, k);
                if (valid < kPageSize && 4 * k + r >= valid)
                    v = make_uint4(0, 0, 0, 0);
                *reinterpret_cast<uint4*>(&lds.v[(4 * k + r) * kPvVRow + 8 * c]) = v;
            }
        }
        wave_lds_sync();
        if (rescale) {
            const float al = lds.alpha[n];
#pragma unroll
            for (int i2 = 0; i2 < kHeadDim / 16; ++i2)
                o[i2] *= al;
        }
        const float4 pp =
            *reinterpret_cast<const float4*>(&lds.p[n * kPvPRow + 4 * (kg ^ pv_p_swizzle(n))]);
        short4_t p_hi, p_lo;
        split_bf16(pp, p_hi, p_lo);
        const uint16_t* vrow = &lds.v[(4 * kg + n / 4) * kPvVRow + 4 * (n % 4)];
#pragma unroll
        for (int i2 = 0; i2 < kHeadDim / 16; ++i2) {
            const short4_t vt = lds_read_tr16(vrow + 16 * i2);
            o[i2] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, p_hi, o[i2], 0, 0, 0);
            o[i2] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, p_lo, o[i2], 0, 0, 0);
        }
    };

    if (KV::kScaled && lane < t.count) {
        const int64_t slab = (int64_t)my_page * a.num_kv_heads + t.kvh;
        my_kscale = a.k_scale[slab];
        my_vscale = a.v_scale[slab];
    }
    typename KV::Buf buf_a, buf_b;
    stream_pages(t.count, buf_a, buf_b, issue, consume);
#pragma unroll
    for (int e = 0; e < kE; ++e)
        l_row[e] = row16_sum(lsum[e]);
}

template <int G, bool CHECKED, typename KV, bool PERSISTENT>
__global__ __launch_bounds__(kWave * kUnitWaves)
__attribute__((amdgpu_waves_per_eu(G > 4 || PERSISTENT ? 2 : 3))) void split_pv(SplitArgs a)
{
    static_assert(G == 1 || G == 2 || G == 4 || G == 8 || G == 16, "query group of 1..16 heads");
    using SR = ScoreRows<G>;
    constexpr int kE = SR::kPerLane;
    __shared__ __attribute__((aligned(16))) PvShared<G> sh;
    extern __shared__ int plan[];

    auto unit = [&](const SplitArgs& a, int b, int kvh, int s, bool owner) {
        WaveTask t;
        int32_t my_page;
        if (!begin_unit<CHECKED>(a, t, my_page, b, kvh, s, owner)) {
            write_zero_rows<G>(a, t);
            return;
        }
        floatx4_t o[kHeadDim / 16];
        float m[kE], l_row[kE];
        attend_pages_pv<G, CHECKED, KV>(a, t, my_page, sh.wave[t.wave], o, m, l_row);
        __syncthreads();  // every wavefront has left its page loop
        // Lane 16q + j holds tile row j: the head (j / kStep) when it is one.
        const int j = t.lane & 15, q = t.lane >> 4;
        if (j % SR::kStep == 0 && j / SR::kStep < G) {
            const int g = j / SR::kStep;
#pragma unroll
            for (int i = 0; i < kHeadDim / 16; ++i)
                *reinterpret_cast<float4*>(&sh.unit.acc[t.wave][g][16 * i + 4 * q]) =
                    make_float4(o[i][0], o[i][1], o[i][2], o[i][3]);
        }
        if ((t.lane & 15) == 0) {
#pragma unroll
            for (int e = 0; e < kE; ++e) {
                const int row = 4 * q + e * SR::kStep;
                if (row / SR::kStep < G) {
                    sh.unit.m[t.wave][row / SR::kStep] = m[e];
                    sh.unit.l[t.wave][row / SR::kStep] = l_row[e];
                }
            }
        }
        __syncthreads();
        merge_unit<G>(a, t, sh.unit);
    };
    if (PERSISTENT)
        run_persistent(a, a.num_kv_heads, plan, unit);
    else  // one split per sequence: unit (b, kv head) = blockIdx.x
        unit(a, blockIdx.x / a.num_kv_heads, blockIdx.x % a.num_kv_heads, 0, true);
}

// -------------------------------------------------------- merge kernel ---
//
// One work-group of four wavefronts per (b, h) of sequences with more than one
// split: M = max_s m_s, then wavefront w sums w_s l_s and w_s acc_s
// (w_s = 2^(m_s - M)) over splits s = w, w+4, ... (two dims per lane), and the
// four partial sums are added in wavefront order.

constexpr int kMergeWaves = 4;

struct MergeArgs {
    const int32_t* seq_lens;
    const float* ws_acc;
    const float* ws_ml;
    uint16_t* out;
    int32_t num_q_heads;
    int32_t max_pages;
    int32_t split_pages;
    int32_t num_splits;
};

__global__ __launch_bounds__(kWave * kMergeWaves) void merge_splits(MergeArgs a)
{
    __shared__ float part[kMergeWaves][kHeadDim + 1];
    const int64_t row = blockIdx.x;  // b * Hq + h
    const int b = (int)(row / a.num_q_heads);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const float* ml = a.ws_ml + row * a.num_splits * 2;
    const float* acc = a.ws_acc + row * a.num_splits * kHeadDim + 2 * lane;
    // The length and the first loads of both passes go out together (every
    // split index below num_splits lies inside the row's partials), so the
    // common case takes one round trip to memory; entries past the
    // sequence's own splits are read but not used.
    const int len = a.seq_lens[b];
    const float m_first = lane < a.num_splits ? ml[2 * lane] : -INFINITY;
    float2 ml_first = make_float2(0.0f, 0.0f), v_first = make_float2(0.0f, 0.0f);
    if (wave < a.num_splits) {
        ml_first = *reinterpret_cast<const float2*>(ml + 2 * wave);
        v_first = *reinterpret_cast<const float2*>(acc + (int64_t)wave * kHeadDim);
    }
    const int L = min(len, a.max_pages * kPageSize);
    const int npages = L > 0 ? (L + kPageSize - 1) / kPageSize : 0;
    const int n = (npages + a.split_pages - 1) / a.split_pages;
    if (n < 2)
        return;  // finished by the split kernel
    float M = lane < n ? m_first : -INFINITY;
    for (int s = lane + kWave; s < n; s += kWave)
        M = fmaxf(M, ml[2 * s]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        M = fmaxf(M, __shfl_xor(M, off));
    // wavefront w: splits w, w+4, ... in order
    float den = 0.0f, num0 = 0.0f, num1 = 0.0f;
    if (wave < n) {
        const float w = exp2_fast(ml_first.x - M);
        den = fmaf(w, ml_first.y, den);
        num0 = fmaf(w, v_first.x, num0);
        num1 = fmaf(w, v_first.y, num1);
    }
    for (int s = wave + kMergeWaves; s < n; s += kMergeWaves) {
        const float w = exp2_fast(ml[2 * s] - M);
        den = fmaf(w, ml[2 * s + 1], den);
        const float2 v = *reinterpret_cast<const float2*>(acc + (int64_t)s * kHeadDim);
        num0 = fmaf(w, v.x, num0);
        num1 = fmaf(w, v.y, num1);
    }
    part[wave][2 * lane] = num0;
    part[wave][2 * lane + 1] = num1;
    if (lane == 0)
        part[wave][kHeadDim] = den;
    __syncthreads();
    if (wave != 0)
        return;
    float d = 0.0f, x0 = 0.0f, x1 = 0.0f;
#pragma unroll
    for (int w = 0; w < kMergeWaves; ++w) {
        d += part[w][kHeadDim];
        x0 += part[w][2 * lane];
        x1 += part[w][2 * lane + 1];
    }
    const float inv = 1.0f / d;
    *reinterpret_cast<uint32_t*>(a.out + row * kHeadDim + 2 * lane) =
        f32_to_bf16(x0 * inv) | (f32_to_bf16(x1 * inv) << 16);
}

// ------------------------------------------------------------ dispatch ---

typedef void (*SplitKernel)(SplitArgs);

// PERSISTENT: the kernel for runs with more than one split (persistent
// work-groups taking units from the queue).  pv: the P.V product on the
// matrix cores.
template <int G, bool CHECKED, bool PERSISTENT>
SplitKernel pick(bool fp8, bool mfma, bool hp, bool pv)
{
    if (pv)
        return fp8 ? split_pv<G, CHECKED, KvFp8Rows, PERSISTENT>
                   : split_pv<G, CHECKED, KvBf16, PERSISTENT>;
    if (hp)
        return fp8 ? split_mfma_hp<G, CHECKED, KvFp8, PERSISTENT>
                   : split_mfma_hp<G, CHECKED, KvBf16, PERSISTENT>;
    if (fp8)
        return split_mfma<G, CHECKED, KvFp8, PERSISTENT>;  // fp8 pools: MFMA score tile only
    if (mfma)
        return split_mfma<G, CHECKED, KvBf16, PERSISTENT>;
    return split_valu_bf16<G, CHECKED, PERSISTENT>;
}

template <bool CHECKED, bool PERSISTENT>
SplitKernel select_for_group(int G, bool fp8, bool mfma, bool hp, bool pv)
{
    switch (G) {
    case 1: return pick<1, CHECKED, PERSISTENT>(fp8, mfma, hp, pv);
    case 2: return pick<2, CHECKED, PERSISTENT>(fp8, mfma, hp, pv);
    case 4: return pick<4, CHECKED, PERSISTENT>(fp8, mfma, hp, pv);
    case 8: return pick<8, CHECKED, PERSISTENT>(fp8, mfma, hp, pv);
    case 16:  // only the matrix-core value pass holds 16 heads' accumulators
        return fp8 ? split_pv<16, CHECKED, KvFp8Rows, PERSISTENT>
                   : split_pv<16, CHECKED, KvBf16, PERSISTENT>;
    default: return nullptr;
    }
}

SplitKernel select_split_kernel(int G, bool checked, bool fp8, bool mfma, bool hp, bool pv,
                               bool persistent)
{
    if (checked)
        return persistent ? select_for_group<true, true>(G, fp8, mfma, hp, pv)
                          : select_for_group<true, false>(G, fp8, mfma, hp, pv);
    return persistent ? select_for_group<false, true>(G, fp8, mfma, hp, pv)
                      : select_for_group<false, false>(G, fp8, mfma, hp, pv);
}

// Whether the four-wavefront units accumulate P.V on the matrix cores (the
// default; measured against the vector-ALU value pass on one box: Qwen3-8B
// step 166.9 -> 164.9 us, Qwen3-32B heads 179.1 -> 165.3 us, long tail 965 ->
// 955 us, stragglers 473 -> 470 us, fp8 large batch and the TP = 8 share
// within 1%), or with vector-ALU FMAs on request (RL_DA_PV_ON_VALU, and the
// vector-ALU score path, which has its own value pass).
bool uses_pv_mfma(const rl_da_config* cfg)
{
    return (cfg->flags & (RL_DA_PV_ON_VALU | RL_DA_SCORES_ON_VALU)) == 0;
}

// kv heads per head-parallel work-group: the largest divisor of Hkv up to 8
int heads_per_unit_for(int num_kv_heads)
{
    for (int d = kMaxHeadsPerUnit; d > 1; --d)
        if (num_kv_heads % d == 0)
            return d;
    return 1;
}

// The default split: the longest of kDefaultSplitTokens, half, ... (down to
// kMinDefaultSplitTokens) that cuts a full-capacity batch into at least
// kMinDefaultUnits work units of units_per_split per (sequence, split).  It
// depends on the handle's capacity only, never on a run's batch.
int default_split_tokens(const rl_da_config* cfg, int64_t units_per_split)
{
    int st = kDefaultSplitTokens;
    while (st > kMinDefaultSplitTokens) {
        const int64_t splits = ((int64_t)cfg->max_pages_per_seq * kPageSize + st - 1) / st;
        if ((int64_t)cfg->max_batch * units_per_split * splits >= kMinDefaultUnits)
            break;
        st /= 2;
    }
    return st;
}

// Token-major pools with at least two kv heads per work-group take the
// head-parallel units (MFMA scores only) when the handle's full-capacity
// batch, cut into four-wavefront units, would fit on the chip at once
// (kResidentUnits); a larger capacity takes the four-wavefront units, which
// the persistent longest-first schedule balances (on lengths with a tail
// that beats the head-parallel units by 8-15%; on uniform lengths the
// head-parallel units stay ahead).  RL_DA_PER_HEAD_UNITS or
// RL_DA_SCORES_ON_VALU always take the four-wavefront units, and so does
// everything on head-major pools.
bool uses_head_parallel(const rl_da_config* cfg)
{
    if (cfg->layout != RL_DA_LAYOUT_NHD ||
        (cfg->flags & (RL_DA_SCORES_ON_VALU | RL_DA_PER_HEAD_UNITS)) != 0 ||
        heads_per_unit_for(cfg->num_kv_heads) < 2 || cfg->num_q_heads > 8 * cfg->num_kv_heads)
        return false;
    const int st = cfg->split_tokens != 0 ? cfg->split_tokens
                                          : default_split_tokens(cfg, cfg->num_kv_heads);
    const int64_t splits = ((int64_t)cfg->max_pages_per_seq * kPageSize + st - 1) / st;
    return (int64_t)cfg->max_batch * cfg->num_kv_heads * splits <= kResidentUnits;
}

}  // namespace

// ----------------------------------------------------------- C interface ---

struct rl_decode_attn {
    rl_da_config cfg;
    int split_tokens;
    int split_pages;
    int max_splits;
    int device;
    bool use_mfma;
    bool head_parallel;
    int heads_per_unit;
    SplitKernel split_kernel;             // runs with one split per sequence
    SplitKernel split_kernel_persistent;  // runs with more
    int persistent_grid;                  // persistent work-groups resident at once
    int static_slots;                     // one-unit work-groups resident at once
    void* workspace;
    size_t workspace_bytes;
    float* ws_acc;
    float* ws_ml;
    int32_t* dev_error;
    int32_t* queue;  // persistent runs: next unit, finished work-groups
    hipStream_t last_stream;  // stream of the latest run (check_error waits on it)
    hipEvent_t ev_split_begin;
    hipEvent_t ev_split_end;
};

namespace {

// Validates cfg; on success fills the derived split geometry.
rl_da_status check_config(const rl_da_config* cfg, int* split_tokens, int* split_pages,
                          int* max_splits)
{
    if (cfg == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    if (cfg->num_q_heads <= 0 || cfg->num_kv_heads <= 0 || cfg->head_dim <= 0 ||
        cfg->page_size <= 0 || cfg->max_batch <= 0 || cfg->max_pages_per_seq <= 0 ||
        cfg->split_tokens < 0)
        return RL_DA_ERR_INVALID_ARG;
    if (cfg->num_q_heads % cfg->num_kv_heads != 0)
        return RL_DA_ERR_INVALID_ARG;
    if ((cfg->flags & ~(RL_DA_CHECKED | RL_DA_SCORES_ON_VALU | RL_DA_PER_HEAD_UNITS |
                        RL_DA_PV_ON_VALU)) != 0)
        return RL_DA_ERR_INVALID_ARG;
    if (cfg->kv_dtype != RL_DA_KV_BF16 && cfg->kv_dtype != RL_DA_KV_FP8_E4M3)
        return RL_DA_ERR_INVALID_ARG;
    PoolStrides ps;
    if (!pool_strides(cfg->layout, cfg->num_kv_heads, 1, &ps))
        return RL_DA_ERR_INVALID_ARG;
    const int G = cfg->num_q_heads / cfg->num_kv_heads;
    if (cfg->head_dim != kHeadDim || cfg->page_size != kPageSize ||
        (G != 1 && G != 2 && G != 4 && G != 8 && G != 16))
        return RL_DA_ERR_UNSUPPORTED;
    // only the matrix-core value pass holds a 16-head group's accumulators; the
    // vector-ALU score path serves bf16 pools only
    if (G == 16 && !uses_pv_mfma(cfg))
        return RL_DA_ERR_UNSUPPORTED;
    if ((cfg->flags & RL_DA_SCORES_ON_VALU) != 0 && cfg->kv_dtype == RL_DA_KV_FP8_E4M3)
        return RL_DA_ERR_UNSUPPORTED;
    const bool hp = uses_head_parallel(cfg);
    // work units per (sequence, split)
    const int64_t units_per_split =
        hp ? cfg->num_kv_heads / heads_per_unit_for(cfg->num_kv_heads) : cfg->num_kv_heads;
    const int st =
        cfg->split_tokens != 0 ? cfg->split_tokens : default_split_tokens(cfg, units_per_split);
    if (st % kPageSize != 0 || st > (hp ? kMaxSplitTokensHp : kMaxSplitTokens))
        return RL_DA_ERR_UNSUPPORTED;
    *split_tokens = st;
    *split_pages = st / kPageSize;
    *max_splits = (cfg->max_pages_per_seq + *split_pages - 1) / *split_pages;
    return RL_DA_OK;
}

// Workspace: per-split partial accumulators and (m, l) pairs, then one
// 256-byte control block: the device error word (offset 0) and the
// persistent launch's unit queue (offset 128).
constexpr size_t kControlBytes = 256;
constexpr int kQueueWord = 32;  // int32 index of the queue in the control block

size_t partials_bytes(const rl_da_config* cfg, int max_splits)
{
    const size_t rows = (size_t)cfg->max_batch * (size_t)cfg->num_q_heads * (size_t)max_splits;
    size_t bytes = rows * kHeadDim * sizeof(float);      // acc
    bytes += rows * 2 * sizeof(float);                    // (m, l)
    return (bytes + 255) & ~(size_t)255;
}

size_t workspace_bytes_for(const rl_da_config* cfg, int max_splits)
{
    return partials_bytes(cfg, max_splits) + kControlBytes;
}

// Zeroes n int32 words on a stream (a kernel rather than a memset node, so
// that the clear can sit in a captured graph).
__global__ __launch_bounds__(64) void clear_words(int32_t* p, int n)
{
    for (int i = threadIdx.x; i < n; i += blockDim.x)
        p[i] = 0;
}

// Everything a handle holds except its workspace: the validated
// configuration, the split geometry, the kernels and their resident
// work-group counts on the current device.  Allocates nothing.
rl_da_status init_handle(rl_decode_attn* h, const rl_da_config* cfg)
{
    int st, sp, ms;
    const rl_da_status rc = check_config(cfg, &st, &sp, &ms);
    if (rc != RL_DA_OK)
        return rc;
    h->cfg = *cfg;
    h->split_tokens = st;
    h->split_pages = sp;
    h->max_splits = ms;
    const int G = cfg->num_q_heads / cfg->num_kv_heads;
    h->use_mfma = (cfg->flags & RL_DA_SCORES_ON_VALU) == 0;
    h->head_parallel = uses_head_parallel(cfg);
    h->heads_per_unit = h->head_parallel ? heads_per_unit_for(cfg->num_kv_heads) : 1;
    for (int persistent = 0; persistent < 2; ++persistent)
        (persistent ? h->split_kernel_persistent : h->split_kernel) = select_split_kernel(
            G, (cfg->flags & RL_DA_CHECKED) != 0, cfg->kv_dtype == RL_DA_KV_FP8_E4M3, h->use_mfma,
            h->head_parallel, !h->head_parallel && uses_pv_mfma(cfg), persistent != 0);
    if (hipGetDevice(&h->device) != hipSuccess)
        return RL_DA_ERR_HIP;
    // One persistent work-group per slot that can be resident with the
    // largest plan this handle can need; and how many one-unit work-groups
    // the static grid keeps resident.
    const int threads = h->head_parallel ? kWave * h->heads_per_unit : kWave * kUnitWaves;
    const int plan_batch = cfg->max_batch < kMaxPlanBatch ? cfg->max_batch : kMaxPlanBatch;
    const size_t lds = (size_t)plan_ints(plan_batch) * sizeof(int);
    int per_cu = 0, static_per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu, reinterpret_cast<const void*>(h->split_kernel_persistent), threads, lds) !=
            hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &static_per_cu, reinterpret_cast<const void*>(h->split_kernel), threads, 0) !=
            hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device) !=
            hipSuccess ||
        per_cu < 1 || static_per_cu < 1 || cus < 1) {
        (void)hipGetLastError();
        return RL_DA_ERR_HIP;
    }
    h->persistent_grid = per_cu * cus;
    h->static_slots = static_per_cu * cus;
    h->workspace_bytes = workspace_bytes_for(cfg, ms);
    return RL_DA_OK;
}

// Points the handle at a workspace of h->workspace_bytes bytes.
void bind_workspace(rl_decode_attn* h, void* ws)
{
    const size_t rows =
        (size_t)h->cfg.max_batch * (size_t)h->cfg.num_q_heads * (size_t)h->max_splits;
    h->workspace = ws;
    h->ws_acc = (float*)ws;
    h->ws_ml = h->ws_acc + rows * kHeadDim;
    h->dev_error = (int32_t*)((char*)ws + h->workspace_bytes - kControlBytes);
    h->queue = h->dev_error + kQueueWord;
}

// Launches the split kernel, with the handle's timing events attached to the
// kernel itself when they are set (their timestamps are the kernel's own
// start and end, with no marker packets between launches).
hipError_t launch_split(const rl_decode_attn* h, SplitKernel k, int64_t grid, int threads,
                        size_t lds, hipStream_t st, SplitArgs& sa)
{
    if (h->ev_split_begin != nullptr) {
        void* args[] = {&sa};
        return hipExtLaunchKernel(reinterpret_cast<const void*>(k), dim3((unsigned)grid),
                                  dim3(threads), args, lds, st, h->ev_split_begin,
                                  h->ev_split_end, 0);
    }
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(threads), lds, st, sa);
    return hipGetLastError();
}

// Enqueues one decode step with the handle's kernels and workspace.
rl_da_status enqueue_run(rl_decode_attn* h, const void* q, const void* k_pool,
                         const void* v_pool, const float* k_scale, const float* v_scale,
                         int64_t num_pages, const int32_t* block_table, int32_t max_pages,
                         const int32_t* seq_lens, int32_t batch, float scale, void* out,
                         hipStream_t st, bool clear_queue)
{
    const rl_da_config& cfg = h->cfg;
    if (batch < 0 || batch > cfg.max_batch)
        return RL_DA_ERR_INVALID_ARG;
    if (max_pages < 1 || max_pages > cfg.max_pages_per_seq || num_pages < 1)
        return RL_DA_ERR_INVALID_ARG;
    if (!isfinite(scale))
        return RL_DA_ERR_INVALID_ARG;
    if (q == nullptr || k_pool == nullptr || v_pool == nullptr || block_table == nullptr ||
        seq_lens == nullptr || out == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
        return RL_DA_ERR_INVALID_ARG;
    const bool fp8 = cfg.kv_dtype == RL_DA_KV_FP8_E4M3;
    if (fp8 != (k_scale != nullptr) || fp8 != (v_scale != nullptr))
        return RL_DA_ERR_INVALID_ARG;
    if (!pools_paired(cfg.layout, k_pool, v_pool, fp8 ? 1 : 2))
        return RL_DA_ERR_INVALID_ARG;
    if (batch == 0)
        return RL_DA_OK;

    const int num_splits = (max_pages + h->split_pages - 1) / h->split_pages;
    const int64_t units = (int64_t)batch * (cfg.num_kv_heads / h->heads_per_unit) * num_splits;
    if (units + h->persistent_grid > INT32_MAX)
        return RL_DA_ERR_UNSUPPORTED;
    // One split: the one-unit kernel, one work-group per unit.  Several
    // splits: the multi-split kernel -- one work-group per unit when the chip
    // holds every unit at once (the order cannot matter then), else
    // persistent work-groups taking units longest first (in sequence order
    // when the batch is too large for the plan).
    // (Four-wavefront units on token-major pools run persistent with one
    // split too: their static grid balances badly there, 590 -> 463 us on the
    // fp8 large batch; on head-major pools the static grid is as good.)
    const bool persistent =
        num_splits > 1 || (cfg.layout == RL_DA_LAYOUT_NHD && !h->head_parallel &&
                           units > h->static_slots);
    const Schedule schedule = units <= h->static_slots ? kOnePerGroup
                              : batch <= kMaxPlanBatch ? kQueuePlanned
                                                       : kQueueInOrder;

    SplitArgs sa;
    sa.q = (const uint16_t*)q;
    sa.k_pool = (const uint8_t*)k_pool;
    sa.v_pool = (const uint8_t*)v_pool;
    sa.k_scale = k_scale;
    sa.v_scale = v_scale;
    sa.block_table = block_table;
    sa.seq_lens = seq_lens;
    sa.out = (uint16_t*)out;
    sa.ws_acc = h->ws_acc;
    sa.ws_ml = h->ws_ml;
    sa.dev_error = h->dev_error;
    sa.num_pages = num_pages;
    PoolStrides ps;
    (void)pool_strides(cfg.layout, cfg.num_kv_heads, fp8 ? 1 : 2, &ps);  // checked at create
    sa.page_bytes = ps.page;
    sa.head_bytes = ps.head;
    sa.row_bytes = ps.row;
    sa.num_q_heads = cfg.num_q_heads;
    sa.num_kv_heads = cfg.num_kv_heads;
    sa.max_pages = max_pages;
    sa.split_pages = h->split_pages;
    sa.num_splits = num_splits;
    sa.heads_per_unit = h->heads_per_unit;
    sa.batch = batch;
    sa.schedule = schedule;
    sa.queue = h->queue;
    sa.scale_log2 = scale * kLog2e;

    h->last_stream = st;
    const int threads = h->head_parallel ? kWave * h->heads_per_unit : kWave * kUnitWaves;
    if (persistent) {
        if (clear_queue && schedule != kOnePerGroup) {
            hipLaunchKernelGGL(clear_words, dim3(1), dim3(64), 0, st, h->queue, 2);
            if (hipGetLastError() != hipSuccess)
                return RL_DA_ERR_HIP;
        }
        const int64_t grid = schedule == kOnePerGroup || units <= h->persistent_grid
                                 ? units
                                 : h->persistent_grid;
        const size_t lds =
            schedule == kQueuePlanned ? (size_t)plan_ints(batch) * sizeof(int) : 0;
        if (launch_split(h, h->split_kernel_persistent, grid, threads, lds, st, sa) !=
            hipSuccess)
            return RL_DA_ERR_HIP;
    } else {
        if (launch_split(h, h->split_kernel, units, threads, 0, st, sa) != hipSuccess)
            return RL_DA_ERR_HIP;
    }
    if (num_splits > 1) {
        MergeArgs ma;
        ma.seq_lens = seq_lens;
        ma.ws_acc = h->ws_acc;
        ma.ws_ml = h->ws_ml;
        ma.out = (uint16_t*)out;
        ma.num_q_heads = cfg.num_q_heads;
        ma.max_pages = max_pages;
        ma.split_pages = h->split_pages;
        ma.num_splits = num_splits;
        hipLaunchKernelGGL(merge_splits, dim3((unsigned)((int64_t)batch * cfg.num_q_heads)),
                           dim3(kWave * kMergeWaves), 0, st, ma);
        if (hipGetLastError() != hipSuccess)
            return RL_DA_ERR_HIP;
    }
    return RL_DA_OK;
}

}  // namespace

extern "C" {

const char* rl_da_status_string(rl_da_status s)
{
    switch (s) {
    case RL_DA_OK: return "ok";
    case RL_DA_ERR_INVALID_ARG: return "invalid argument";
    case RL_DA_ERR_UNSUPPORTED: return "unsupported configuration";
    case RL_DA_ERR_OUT_OF_MEMORY: return "out of device memory";
    case RL_DA_ERR_HIP: return "HIP runtime error";
    case RL_DA_ERR_SCRATCH_TOO_SMALL:
        return "workspace exceeds the allocation-free entry point's fixed scratch";
    }
    return "unknown status";
}

rl_da_status rl_decode_attn_workspace_size(const rl_da_config* cfg, size_t* bytes)
{
    int st, sp, ms;
    if (bytes == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    const rl_da_status rc = check_config(cfg, &st, &sp, &ms);
    if (rc != RL_DA_OK)
        return rc;
    *bytes = workspace_bytes_for(cfg, ms);
    return RL_DA_OK;
}

rl_da_status rl_decode_attn_create(const rl_da_config* cfg, rl_decode_attn** out)
{
    if (out == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    *out = nullptr;
    int st, sp, ms;
    rl_da_status rc = check_config(cfg, &st, &sp, &ms);
    if (rc != RL_DA_OK)
        return rc;
    rl_decode_attn* h = (rl_decode_attn*)calloc(1, sizeof(rl_decode_attn));
    if (h == nullptr)
        return RL_DA_ERR_OUT_OF_MEMORY;
    rc = init_handle(h, cfg);
    if (rc != RL_DA_OK) {
        free(h);
        return rc;
    }
    void* ws = nullptr;
    if (hipMalloc(&ws, h->workspace_bytes) != hipSuccess) {
        (void)hipGetLastError();
        free(h);
        return RL_DA_ERR_OUT_OF_MEMORY;
    }
    bind_workspace(h, ws);
    if (hipMemset(h->dev_error, 0, kControlBytes) != hipSuccess) {
        (void)hipFree(ws);
        free(h);
        return RL_DA_ERR_HIP;
    }
    *out = h;
    return RL_DA_OK;
}

rl_da_status rl_decode_attn_destroy(rl_decode_attn* h)
{
    if (h == nullptr)
        return RL_DA_OK;
    const hipError_t e = hipFree(h->workspace);
    free(h);
    return e == hipSuccess ? RL_DA_OK : RL_DA_ERR_HIP;
}

rl_da_status rl_decode_attn_split_info(const rl_decode_attn* h, int32_t max_pages,
                                       int32_t* split_tokens, int32_t* num_splits)
{
    if (h == nullptr || split_tokens == nullptr || num_splits == nullptr || max_pages < 1 ||
        max_pages > h->cfg.max_pages_per_seq)
        return RL_DA_ERR_INVALID_ARG;
    *split_tokens = h->split_tokens;
    *num_splits = (max_pages + h->split_pages - 1) / h->split_pages;
    return RL_DA_OK;
}

rl_da_status rl_decode_attn_run(rl_decode_attn* h, const void* q, const void* k_pool,
                                const void* v_pool, const float* k_scale,
                                const float* v_scale, int64_t num_pages,
                                const int32_t* block_table, int32_t max_pages,
                                const int32_t* seq_lens, int32_t batch, float scale, void* out,
                                void* stream)
{
    if (h == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    return enqueue_run(h, q, k_pool, v_pool, k_scale, v_scale, num_pages, block_table,
                       max_pages, seq_lens, batch, scale, out, (hipStream_t)stream, false);
}

rl_da_status rl_decode_attn_unit_heads(const rl_decode_attn* h, int32_t* kv_heads_per_unit)
{
    if (h == nullptr || kv_heads_per_unit == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    *kv_heads_per_unit = h->head_parallel ? h->heads_per_unit : 1;
    return RL_DA_OK;
}

rl_da_status rl_decode_attn_set_timing_events(rl_decode_attn* h, void* split_begin,
                                              void* split_end)
{
    if (h == nullptr || (split_begin == nullptr) != (split_end == nullptr))
        return RL_DA_ERR_INVALID_ARG;
    h->ev_split_begin = (hipEvent_t)split_begin;
    h->ev_split_end = (hipEvent_t)split_end;
    return RL_DA_OK;
}

rl_da_status rl_decode_attn_check_error(rl_decode_attn* h, int32_t* device_error)
{
    if (h == nullptr || device_error == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    if ((h->cfg.flags & RL_DA_CHECKED) == 0)
        return RL_DA_ERR_UNSUPPORTED;
    // Read the word behind the latest run on its stream, then clear it on the
    // same stream; other streams of the device are not waited for.
    const hipStream_t st = h->last_stream;
    int32_t v = 0;
    if (hipMemcpyAsync(&v, h->dev_error, sizeof v, hipMemcpyDeviceToHost, st) != hipSuccess)
        return RL_DA_ERR_HIP;
    hipLaunchKernelGGL(clear_words, dim3(1), dim3(64), 0, st, h->dev_error, 1);
    if (hipGetLastError() != hipSuccess)
        return RL_DA_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess)
        return RL_DA_ERR_HIP;
    *device_error = v;
    return RL_DA_OK;
}

}  // extern "C"

// ------------------------------------------ allocation-free entry point ---
//
// rl_decode_attn_run_noalloc runs the decode step with the kernels and split
// size of a handle created with the same configuration, but takes its
// workspace (per-split partials, error word, unit queue) from `scratch`, a
// fixed device array, instead of allocating one.  Host code must never pass
// the array's name to a kernel or a copy: it names a host-side stand-in.  The
// device address comes from hipGetSymbolAddress, taken once per device (each
// device holds its own copy of the array) with that device current, and only
// that address is used afterwards.

static __device__ __align__(256) uint8_t scratch[RL_DA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
// Recently used configurations, so that repeated calls skip the occupancy
// queries of init_handle.
constexpr int kNoallocCacheEntries = 8;

struct NoallocEntry {
    bool used;
    int device;
    rl_da_config cfg;
    rl_decode_attn h;  // workspace not bound
};

std::mutex g_noalloc_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device
NoallocEntry g_noalloc_cache[kNoallocCacheEntries];
int g_noalloc_next;

// Fills *h for cfg on the current device `dev` (no workspace bound) and
// returns the device address of that device's scratch in *ws.
rl_da_status noalloc_setup(const rl_da_config* cfg, int dev, rl_decode_attn* h, void** ws)
{
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch)) != hipSuccess ||
            ptr == nullptr) {
            (void)hipGetLastError();
            return RL_DA_ERR_HIP;
        }
        g_scratch_ptr[dev] = ptr;
    }
    *ws = g_scratch_ptr[dev];
    for (int i = 0; i < kNoallocCacheEntries; ++i) {
        const NoallocEntry& e = g_noalloc_cache[i];
        if (e.used && e.device == dev && memcmp(&e.cfg, cfg, sizeof *cfg) == 0) {
            *h = e.h;
            return RL_DA_OK;
        }
    }
    memset(h, 0, sizeof *h);
    const rl_da_status rc = init_handle(h, cfg);
    if (rc != RL_DA_OK)
        return rc;
    if (h->workspace_bytes > (size_t)RL_DA_NOALLOC_SCRATCH_BYTES)
        return RL_DA_ERR_SCRATCH_TOO_SMALL;
    NoallocEntry& slot = g_noalloc_cache[g_noalloc_next];
    g_noalloc_next = (g_noalloc_next + 1) % kNoallocCacheEntries;
    slot.used = true;
    slot.device = dev;
    slot.cfg = *cfg;
    slot.h = *h;
    return RL_DA_OK;
}

}  // namespace

extern "C" rl_da_status rl_decode_attn_run_noalloc(
    const rl_da_config* cfg, const void* q, const void* k_pool, const void* v_pool,
    const float* k_scale, const float* v_scale, int64_t num_pages, const int32_t* block_table,
    int32_t max_pages, const int32_t* seq_lens, int32_t batch, float scale, void* out,
    void* stream)
{
    if (cfg == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    int st, sp, ms;
    const rl_da_status rc = check_config(cfg, &st, &sp, &ms);
    if (rc != RL_DA_OK)
        return rc;
    if ((cfg->flags & RL_DA_CHECKED) != 0)
        return RL_DA_ERR_UNSUPPORTED;  // no handle to read the error word from
    if (workspace_bytes_for(cfg, ms) > (size_t)RL_DA_NOALLOC_SCRATCH_BYTES)
        return RL_DA_ERR_SCRATCH_TOO_SMALL;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return RL_DA_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices)
        return RL_DA_ERR_UNSUPPORTED;
    rl_decode_attn h;
    void* ws = nullptr;
    const rl_da_status rs = noalloc_setup(cfg, dev, &h, &ws);
    if (rs != RL_DA_OK)
        return rs;
    bind_workspace(&h, ws);
    h.ev_split_begin = nullptr;
    h.ev_split_end = nullptr;
    // The unit queue is cleared on the stream before each persistent launch:
    // the scratch keeps whatever the device's previous call left in it.
    return enqueue_run(&h, q, k_pool, v_pool, k_scale, v_scale, num_pages, block_table,
                       max_pages, seq_lens, batch, scale, out, (hipStream_t)stream, true);
}
