"""Oracle for the single-GPU share of weight synchronisation and checkpoint
copies.  TEST INFRASTRUCTURE ONLY: used by tests and the benchmark's CPU
baseline, never by the GPU library, with which it shares no code.

What is computed (arXiv 2512.22492, Sec. 5.2.1: the trainer places the model
layer by layer into a reserved transfer buffer before each transfer; Sec. 3
and Sec. 7: the per-step checkpoint blocks only for the GPU-to-host copy of
the rank's shard).  The paper gives no placement rule; the reading used here:
tensors in order, each starting at the next `align`-aligned offset, filling
the buffer up to `capacity` and splitting a tensor at the buffer's end, so
that one buffer fill (a chunk) follows another.

Everything is plain Python over integers and numpy byte arrays.
"""
import numpy as np


def align_up(x, a):
    return (x + a - 1) // a * a


def plan(tensor_bytes, capacity, align):
    """Pieces (tensor, chunk, tensor_offset, buffer_offset, nbytes) in order."""
    if capacity < 1 or align < 1 or align & (align - 1) or capacity % align:
        raise ValueError("capacity >= 1 and a power-of-two align dividing it")
    pieces = []
    chunk, cursor = 0, 0
    for i, n in enumerate(tensor_bytes):
        done = 0
        while done < n:
            off = align_up(cursor, align)
            if off >= capacity:          # this fill is full: start the next one
                chunk, off = chunk + 1, 0
            take = min(n - done, capacity - off)
            pieces.append((i, chunk, done, off, take))
            done += take
            cursor = off + take
    return pieces


def num_chunks(pieces):
    return pieces[-1][1] + 1 if pieces else 0


def pack(tensors, pieces, chunk, capacity, fill=0):
    """The buffer after packing `chunk`: tensors is a list of uint8 arrays;
    bytes outside every piece keep `fill`.  Returns (buffer, written mask)."""
    buf = np.full(capacity, fill, dtype=np.uint8)
    written = np.zeros(capacity, dtype=bool)
    for t, c, t_off, b_off, n in pieces:
        if c != chunk:
            continue
        buf[b_off:b_off + n] = tensors[t][t_off:t_off + n]
        written[b_off:b_off + n] = True
    return buf, written


def unpack(buffer, pieces, chunk, tensors):
    """Copies of `tensors` with `chunk`'s pieces taken from `buffer`."""
    out = [np.array(t, dtype=np.uint8, copy=True) for t in tensors]
    for t, c, t_off, b_off, n in pieces:
        if c == chunk:
            out[t][t_off:t_off + n] = buffer[b_off:b_off + n]
    return out
