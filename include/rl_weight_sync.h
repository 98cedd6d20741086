/*
 * rl_weight_sync.h -- one GPU's share of weight synchronisation and
 * checkpointing: layer-by-layer packing of model tensors into a reserved
 * transfer buffer, and the same copy into pinned host memory.
 *
 * Weight synchronisation (arXiv 2512.22492, Sec. 5.2.1, UCX weight update):
 * before a transfer the trainer places the model, layer by layer, into a
 * transfer buffer that is kept reserved (so the transfer cannot run out of
 * device memory) and is large enough to keep the network busy; the receiver
 * places the arriving bytes back into its own tensors.  Per-step checkpoint
 * (Sec. 3 and Sec. 7, checkpoint efficiency): the step blocks only for the
 * copy of the rank's shard from GPU memory to host memory.  The network
 * transfer and the disk write are not part of this library.
 *
 * Plan.  Tensors are taken in the caller's order (layer by layer).  A cursor
 * walks the buffer; each tensor's bytes go to the next `align`-aligned offset
 * and fill the buffer up to `capacity`; when the buffer is full (or the
 * aligned cursor reaches capacity) the next bytes start chunk c+1 at offset 0.
 * A tensor that does not fit the room left is split, so every piece boundary
 * inside a tensor falls on a multiple of `align`.  Chunk c is one fill of the
 * buffer: pack(c), transfer, then pack(c+1).  Zero-byte tensors get no piece.
 *
 * Memory.  Tensor addresses are device addresses owned by the caller, valid
 * for the handle's lifetime.  The buffer is device memory or pinned host
 * memory (hipHostMalloc, or torch's pin_memory); create() asks the HIP
 * runtime which one and rejects anything else.  Pack and unpack copy bytes
 * only; tensors whose address and the buffer are 16-byte aligned take the
 * vector path, others a byte path.  Bytes of the buffer between pieces are
 * never written.  Pack and unpack are asynchronous on the caller's stream:
 * host code that touches a pinned host buffer waits for the stream first.
 * Status codes are rl_da_status (rl_decode_attn.h).
 */
#ifndef RL_WEIGHT_SYNC_H
#define RL_WEIGHT_SYNC_H

#include <stdint.h>

#include "rl_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    void* ptr;         /* device address of the tensor's first byte (unpack writes it) */
    uint64_t nbytes;
} rl_ws_tensor;

/* One contiguous run of a tensor's bytes placed in one chunk of the buffer. */
typedef struct {
    int32_t tensor;          /* index in the tensor list                      */
    int32_t chunk;           /* fill of the buffer it belongs to (0, 1, ...)   */
    uint64_t tensor_offset;  /* first byte within the tensor                  */
    uint64_t buffer_offset;  /* first byte within the buffer                  */
    uint64_t nbytes;         /* >= 1                                          */
} rl_ws_piece;

/*
 * Host only (no HIP call): the plan above for num_tensors tensors of
 * tensor_bytes[i] bytes.  capacity >= 1 and align a power of two dividing
 * capacity, else INVALID_ARG.  Writes at most max_pieces pieces, in order;
 * *num_pieces and *num_chunks get the full counts even when max_pieces is too
 * small (pieces may be NULL with max_pieces 0 to ask for the counts).
 */
rl_da_status rl_ws_plan(const uint64_t* tensor_bytes, int32_t num_tensors, uint64_t capacity,
                        uint64_t align, rl_ws_piece* pieces, int64_t max_pieces,
                        int64_t* num_pieces, int32_t* num_chunks);

typedef struct rl_weight_sync rl_weight_sync; /* opaque handle */

/*
 * Plans the placement of tensors[0 .. num_tensors-1] into `buffer` (capacity
 * bytes, device memory or pinned host memory) and uploads the per-chunk copy
 * descriptors to the current device.  INVALID_ARG for null or non-device
 * tensor pointers, an unknown or pageable buffer, or bad capacity / align;
 * OUT_OF_MEMORY / HIP when the descriptor upload fails.
 */
rl_da_status rl_ws_create(const rl_ws_tensor* tensors, int32_t num_tensors, void* buffer,
                          uint64_t capacity, uint64_t align, rl_weight_sync** out);

/* Number of chunks (buffer fills) of the handle's plan; 0 if every tensor is empty. */
rl_da_status rl_ws_num_chunks(const rl_weight_sync* h, int32_t* num_chunks);

/* Bytes of tensor data in chunk `chunk` (the sum of its pieces). */
rl_da_status rl_ws_chunk_bytes(const rl_weight_sync* h, int32_t chunk, uint64_t* nbytes);

/* Enqueues one kernel on `stream` that copies every piece of `chunk` from its
 * tensor into the buffer.  INVALID_ARG for a chunk outside [0, num_chunks). */
rl_da_status rl_ws_pack(rl_weight_sync* h, int32_t chunk, void* stream);

/* The reverse copy: every piece of `chunk` from the buffer into its tensor. */
rl_da_status rl_ws_unpack(rl_weight_sync* h, int32_t chunk, void* stream);

/* Frees the handle and its device descriptors (not the tensors or buffer). */
rl_da_status rl_ws_destroy(rl_weight_sync* h);

#ifdef __cplusplus
}
#endif

#endif
