// rl_weight_sync.hip -- layer-by-layer packing of model tensors into a
// transfer buffer (weight synchronisation, arXiv 2512.22492 Sec. 5.2.1) and
// the same copy into pinned host memory (per-step checkpoint, Sec. 3/Sec. 7).
//
// Plan on the host, copy on the GPU.  A chunk's pieces are cut into 32 KiB
// tiles; one work-group of 256 threads copies one tile, each thread eight
// 16-byte vectors with all loads issued before the stores (non-temporal
// loads, and non-temporal stores into device memory).  A work-group finds
// its piece by binary search over the pieces' first-tile numbers, so pieces of
// any size share one launch.  The copy is bound by HBM (read + write of every
// byte) when the buffer is device memory and by the host link when it is
// pinned host memory.

#include <stdlib.h>

#include <new>
#include <vector>

#include "rl_common.h"
#include "rl_weight_sync.h"

using namespace rl_da;

namespace {

constexpr int kCopyThreads = 256;
constexpr int kVecPerThread = 8;
constexpr uint64_t kTileBytes = (uint64_t)kCopyThreads * kVecPerThread * 16;  // 32 KiB

struct CopyPiece {
    uint8_t* tensor;        // first byte of the piece within its tensor
    uint8_t* buffer;        // first byte of the piece within the buffer (device-usable)
    uint64_t nbytes;
    uint64_t first_tile;    // tiles of the chunk before this piece
};

struct CopyArgs {
    const CopyPiece* pieces;  // the chunk's pieces, in plan order
    int32_t num_pieces;
    int32_t unpack;           // 0: tensor -> buffer, 1: buffer -> tensor
};

// STREAM_STORES: the destination is device memory and gets non-temporal
// stores (data written once, not read back soon; into pinned host memory
// they measured slower).  A template parameter, not a run-time flag: the
// branch made the compiler reorder the loads so that stores waited for
// seven of the eight.
template <bool STREAM_STORES>
__global__ __launch_bounds__(kCopyThreads) void copy_pieces(CopyArgs a)
{
    const uint64_t tile = blockIdx.x;
    // the last piece whose first tile is at or before this tile (every piece
    // has at least one tile, so it holds this one)
    int lo = 0, hi = a.num_pieces - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.pieces[mid].first_tile <= tile)
            lo = mid;
        else
            hi = mid - 1;
    }
    const CopyPiece pc = a.pieces[lo];
    const uint8_t* src = a.unpack ? pc.buffer : pc.tensor;
    uint8_t* dst = a.unpack ? pc.tensor : pc.buffer;
    const uint64_t begin = (tile - pc.first_tile) * kTileBytes;
    const uint64_t end = pc.nbytes < begin + kTileBytes ? pc.nbytes : begin + kTileBytes;
    const int t = threadIdx.x;
    if ((((uintptr_t)src | (uintptr_t)dst) & 15) != 0) {
        for (uint64_t i = begin + t; i < end; i += kCopyThreads)
            dst[i] = src[i];
        return;
    }
    const uint64_t nvec = (end - begin) / 16;
    const uint8_t* s = src + begin;
    uint4* d = reinterpret_cast<uint4*>(dst + begin);
    if (nvec == (uint64_t)kCopyThreads * kVecPerThread) {
        uint4 v[kVecPerThread];
#pragma unroll
        for (int i = 0; i < kVecPerThread; ++i)
            v[i] = load_stream16(s + 16 * (t + i * kCopyThreads));
#pragma unroll
        for (int i = 0; i < kVecPerThread; ++i) {
            if (STREAM_STORES) {
                const u32x4_t w = {v[i].x, v[i].y, v[i].z, v[i].w};
                __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(d + t + i * kCopyThreads));
            } else {
                d[t + i * kCopyThreads] = v[i];
            }
        }
        return;
    }
    for (uint64_t i = t; i < nvec; i += kCopyThreads)
        d[i] = load_stream16(s + 16 * i);
    for (uint64_t i = begin + 16 * nvec + t; i < end; i += kCopyThreads)
        dst[i] = src[i];
}

bool is_pow2(uint64_t x) { return x != 0 && (x & (x - 1)) == 0; }

// The plan of the header, written to `out` when non-null.
rl_da_status make_plan(const uint64_t* tensor_bytes, int32_t num_tensors, uint64_t capacity,
                       uint64_t align, std::vector<rl_ws_piece>* out, int64_t* num_pieces,
                       int32_t* num_chunks)
{
    if (num_tensors < 0 || (num_tensors > 0 && tensor_bytes == nullptr))
        return RL_DA_ERR_INVALID_ARG;
    if (capacity == 0 || !is_pow2(align) || capacity % align != 0)
        return RL_DA_ERR_INVALID_ARG;
    int64_t chunk = 0, pieces = 0;
    uint64_t cursor = 0;
    for (int32_t i = 0; i < num_tensors; ++i) {
        const uint64_t n = tensor_bytes[i];
        uint64_t done = 0;
        while (done < n) {
            uint64_t off = (cursor + align - 1) & ~(align - 1);  // <= capacity: align | capacity
            if (off >= capacity) {
                ++chunk;
                off = 0;
            }
            const uint64_t take = n - done < capacity - off ? n - done : capacity - off;
            if (out != nullptr)
                out->push_back(rl_ws_piece{i, (int32_t)chunk, done, off, take});
            ++pieces;
            done += take;
            cursor = off + take;
            if (chunk >= INT32_MAX)
                return RL_DA_ERR_UNSUPPORTED;
        }
    }
    *num_pieces = pieces;
    *num_chunks = pieces == 0 ? 0 : (int32_t)(chunk + 1);
    return RL_DA_OK;
}

// Device address at which a kernel may access `p`: device memory as is,
// pinned host memory through its device mapping; null for anything else.
// *on_device tells which.
void* device_view(const void* p, bool* on_device)
{
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    *on_device = attr.type == hipMemoryTypeDevice;
    if (attr.type == hipMemoryTypeDevice)
        return const_cast<void*>(p);
    if (attr.type == hipMemoryTypeHost) {
        void* d = nullptr;
        if (hipHostGetDevicePointer(&d, const_cast<void*>(p), 0) != hipSuccess) {
            (void)hipGetLastError();
            return nullptr;
        }
        return d;
    }
    return nullptr;
}

}  // namespace

struct rl_weight_sync {
    int32_t num_chunks;
    bool buffer_on_device;              // else pinned host memory
    std::vector<int64_t> chunk_first;   // index of each chunk's first piece; [num_chunks + 1]
    std::vector<uint64_t> chunk_tiles;  // tiles of each chunk
    std::vector<uint64_t> chunk_bytes;  // tensor bytes of each chunk
    CopyPiece* dev_pieces;              // every piece, in plan order
};

extern "C" {

rl_da_status rl_ws_plan(const uint64_t* tensor_bytes, int32_t num_tensors, uint64_t capacity,
                        uint64_t align, rl_ws_piece* pieces, int64_t max_pieces,
                        int64_t* num_pieces, int32_t* num_chunks)
{
    if (num_pieces == nullptr || num_chunks == nullptr || max_pieces < 0 ||
        (pieces == nullptr && max_pieces > 0))
        return RL_DA_ERR_INVALID_ARG;
    std::vector<rl_ws_piece> plan;
    const rl_da_status rc = make_plan(tensor_bytes, num_tensors, capacity, align,
                                      max_pieces > 0 ? &plan : nullptr, num_pieces, num_chunks);
    if (rc != RL_DA_OK)
        return rc;
    for (int64_t i = 0; i < max_pieces && i < (int64_t)plan.size(); ++i)
        pieces[i] = plan[i];
    return RL_DA_OK;
}

rl_da_status rl_ws_create(const rl_ws_tensor* tensors, int32_t num_tensors, void* buffer,
                          uint64_t capacity, uint64_t align, rl_weight_sync** out)
{
    if (out == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    *out = nullptr;
    if (num_tensors < 0 || (num_tensors > 0 && tensors == nullptr) || buffer == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    std::vector<uint64_t> sizes(num_tensors);
    for (int32_t i = 0; i < num_tensors; ++i) {
        sizes[i] = tensors[i].nbytes;
        if (sizes[i] == 0)
            continue;
        if (tensors[i].ptr == nullptr)
            return RL_DA_ERR_INVALID_ARG;
        hipPointerAttribute_t attr;
        if (hipPointerGetAttributes(&attr, tensors[i].ptr) != hipSuccess) {
            (void)hipGetLastError();
            return RL_DA_ERR_INVALID_ARG;
        }
        if (attr.type != hipMemoryTypeDevice)
            return RL_DA_ERR_INVALID_ARG;
    }
    bool buffer_on_device = false;
    uint8_t* buf = static_cast<uint8_t*>(device_view(buffer, &buffer_on_device));
    if (buf == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    std::vector<rl_ws_piece> plan;
    int64_t np = 0;
    int32_t nc = 0;
    rl_da_status rc = make_plan(sizes.data(), num_tensors, capacity, align, &plan, &np, &nc);
    if (rc != RL_DA_OK)
        return rc;

    rl_weight_sync* h = new (std::nothrow) rl_weight_sync();
    if (h == nullptr)
        return RL_DA_ERR_OUT_OF_MEMORY;
    h->num_chunks = nc;
    h->buffer_on_device = buffer_on_device;
    h->chunk_first.assign(nc + 1, np);
    h->chunk_tiles.assign(nc, 0);
    h->chunk_bytes.assign(nc, 0);
    std::vector<CopyPiece> host(np);
    for (int64_t k = 0; k < np; ++k) {
        const rl_ws_piece& p = plan[k];
        if (k == 0 || plan[k - 1].chunk != p.chunk)
            h->chunk_first[p.chunk] = k;
        host[k].tensor = static_cast<uint8_t*>(tensors[p.tensor].ptr) + p.tensor_offset;
        host[k].buffer = buf + p.buffer_offset;
        host[k].nbytes = p.nbytes;
        host[k].first_tile = h->chunk_tiles[p.chunk];
        h->chunk_tiles[p.chunk] += (p.nbytes + kTileBytes - 1) / kTileBytes;
        h->chunk_bytes[p.chunk] += p.nbytes;
    }
    for (int32_t c = 0; c < nc; ++c)
        if (h->chunk_tiles[c] > INT32_MAX) {
            delete h;
            return RL_DA_ERR_UNSUPPORTED;  // one launch per chunk: grid limit
        }
    h->dev_pieces = nullptr;
    if (np > 0) {
        if (hipMalloc(&h->dev_pieces, sizeof(CopyPiece) * (size_t)np) != hipSuccess) {
            (void)hipGetLastError();
            delete h;
            return RL_DA_ERR_OUT_OF_MEMORY;
        }
        if (hipMemcpy(h->dev_pieces, host.data(), sizeof(CopyPiece) * (size_t)np,
                      hipMemcpyHostToDevice) != hipSuccess) {
            (void)hipFree(h->dev_pieces);
            delete h;
            return RL_DA_ERR_HIP;
        }
    }
    *out = h;
    return RL_DA_OK;
}

rl_da_status rl_ws_num_chunks(const rl_weight_sync* h, int32_t* num_chunks)
{
    if (h == nullptr || num_chunks == nullptr)
        return RL_DA_ERR_INVALID_ARG;
    *num_chunks = h->num_chunks;
    return RL_DA_OK;
}

rl_da_status rl_ws_chunk_bytes(const rl_weight_sync* h, int32_t chunk, uint64_t* nbytes)
{
    if (h == nullptr || nbytes == nullptr || chunk < 0 || chunk >= h->num_chunks)
        return RL_DA_ERR_INVALID_ARG;
    *nbytes = h->chunk_bytes[chunk];
    return RL_DA_OK;
}

static rl_da_status launch_copy(rl_weight_sync* h, int32_t chunk, int unpack, void* stream)
{
    if (h == nullptr || chunk < 0 || chunk >= h->num_chunks)
        return RL_DA_ERR_INVALID_ARG;
    CopyArgs a;
    a.pieces = h->dev_pieces + h->chunk_first[chunk];
    a.num_pieces = (int32_t)(h->chunk_first[chunk + 1] - h->chunk_first[chunk]);
    a.unpack = unpack;
    const dim3 grid((unsigned)h->chunk_tiles[chunk]), block(kCopyThreads);
    if (unpack || h->buffer_on_device)  // destination in device memory
        hipLaunchKernelGGL(copy_pieces<true>, grid, block, 0, (hipStream_t)stream, a);
    else
        hipLaunchKernelGGL(copy_pieces<false>, grid, block, 0, (hipStream_t)stream, a);
    return hipGetLastError() == hipSuccess ? RL_DA_OK : RL_DA_ERR_HIP;
}

rl_da_status rl_ws_pack(rl_weight_sync* h, int32_t chunk, void* stream)
{
    return launch_copy(h, chunk, 0, stream);
}

rl_da_status rl_ws_unpack(rl_weight_sync* h, int32_t chunk, void* stream)
{
    return launch_copy(h, chunk, 1, stream);
}

rl_da_status rl_ws_destroy(rl_weight_sync* h)
{
    if (h == nullptr)
        return RL_DA_OK;
    const hipError_t e = h->dev_pieces != nullptr ? hipFree(h->dev_pieces) : hipSuccess;
    delete h;
    return e == hipSuccess ? RL_DA_OK : RL_DA_ERR_HIP;
}

}  // extern "C"
