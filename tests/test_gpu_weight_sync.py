"""GPU weight packing and checkpoint copies against the oracle, byte for
byte: every chunk of the transfer buffer after pack, the bytes between pieces
left untouched, and the tensors after unpack; with a device buffer and with a
pinned host buffer, aligned and misaligned tensors, tensors larger than the
buffer and empty tensors."""
import numpy as np
import pytest
import torch

from oracle import weight_sync as WS
from paper_2512_22492_amd import binding as B

from gpu_util import device

pytestmark = pytest.mark.gpu

SENTINEL = 0xA5


def make_tensors(sizes, seed, misalign=()):
    """uint8 device tensors of the given byte sizes; indices in `misalign`
    are views starting 3 bytes into their allocation."""
    gen = torch.Generator().manual_seed(seed)
    out = []
    for i, n in enumerate(sizes):
        host = torch.randint(0, 256, (n,), generator=gen, dtype=torch.uint8)
        if i in misalign:
            base = torch.empty(n + 16, dtype=torch.uint8, device=device())
            t = base[3:3 + n]
            t.copy_(host.to(device()))
        else:
            t = host.to(device())
        out.append(t)
    return out


def host_bytes(t):
    return t.cpu().numpy().copy()


def run_plan(sizes, capacity, align, seed, pinned=False, misalign=()):
    tensors = make_tensors(sizes, seed, misalign)
    want_tensors = [host_bytes(t) for t in tensors]
    if pinned:
        buf = torch.empty(capacity, dtype=torch.uint8, pin_memory=True)
    else:
        buf = torch.empty(capacity, dtype=torch.uint8, device=device())
    pieces = WS.plan(sizes, capacity, align)
    with B.WeightSync(tensors, buf, align=align) as ws:
        assert ws.num_chunks == WS.num_chunks(pieces)
        targets = [torch.zeros_like(t) for t in tensors]
        with B.WeightSync(targets, buf, align=align) as back:
            for c in range(ws.num_chunks):
                buf.fill_(SENTINEL)
                ws.pack(c)
                torch.cuda.synchronize()
                want, written = WS.pack(want_tensors, pieces, c, capacity, fill=SENTINEL)
                got = host_bytes(buf)
                assert np.array_equal(got, want), "chunk %d differs" % c
                assert ws.chunk_bytes(c) == int(written.sum())
                back.unpack(c)
                # a host buffer is refilled by the CPU: wait for the unpack first
                torch.cuda.synchronize()
        for i, (t, w) in enumerate(zip(targets, want_tensors)):
            assert np.array_equal(host_bytes(t), w), "tensor %d after unpack" % i


CASES = [
    # sizes, capacity, align
    ([10, 300, 5000, 0, 1, 7000], 4096, 256),
    ([40000, 17, 65536, 32768, 100001, 3], 1 << 16, 16),
    ([1 << 20, 5, 3 << 19, 12345], 1 << 20, 4096),
    ([999, 1, 2, 3, 31, 32, 33], 64, 1),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_pack_unpack_device_buffer(case):
    sizes, cap, align = CASES[case]
    print("case", case, flush=True)
    run_plan(sizes, cap, align, seed=case)


@pytest.mark.parametrize("case", [0, 1])
def test_pack_unpack_misaligned_tensors(case):
    sizes, cap, align = CASES[case]
    run_plan(sizes, cap, align, seed=10 + case, misalign={1, 2})


@pytest.mark.parametrize("case", [0, 2])
def test_pack_unpack_pinned_host_buffer(case):
    """The checkpoint form: the buffer lives in pinned host memory."""
    sizes, cap, align = CASES[case]
    run_plan(sizes, cap, align, seed=20 + case, pinned=True)


def test_model_layer_shapes_one_chunk_to_host():
    """One transformer layer of Qwen3-8B shapes (bf16) copied whole into pinned
    host memory, as a checkpoint shard copy."""
    shapes = [(4096, 4096), (1024, 4096), (1024, 4096), (4096, 4096), (12288, 4096),
              (12288, 4096), (4096, 12288), (4096,), (4096,), (128,), (128,)]
    gen = torch.Generator(device=device()).manual_seed(5)
    tensors = [torch.randn(s, generator=gen, device=device()).to(torch.bfloat16) for s in shapes]
    total = sum(t.numel() * 2 for t in tensors)
    buf = torch.empty(total + 256 * len(shapes), dtype=torch.uint8, pin_memory=True)
    with B.WeightSync(tensors, buf, align=256) as ws:
        assert ws.num_chunks == 1 and ws.chunk_bytes(0) == total
        ws.pack(0)
        torch.cuda.synchronize()
    pieces = WS.plan([t.numel() * 2 for t in tensors], buf.numel(), 256)
    want, written = WS.pack([t.view(torch.uint8).reshape(-1).cpu().numpy() for t in tensors],
                            pieces, 0, buf.numel())
    assert np.array_equal(buf.numpy()[written], want[written])


def test_create_validation():
    t = torch.zeros(100, dtype=torch.uint8, device=device())
    buf = torch.empty(4096, dtype=torch.uint8, device=device())
    host_t = torch.zeros(100, dtype=torch.uint8)                 # pageable host memory
    rc, h = B.rl_ws_create([(t, 100)], buf, 4096, 256)
    assert rc == B.RL_DA_OK
    assert B.rl_ws_pack(h, 1) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_pack(h, -1) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_chunk_bytes(h, 0) == (B.RL_DA_OK, 100)
    assert B.rl_ws_destroy(h) == B.RL_DA_OK
    assert B.rl_ws_create([(host_t, 100)], buf, 4096, 256)[0] == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_create([(t, 100)], host_t, 100, 4)[0] == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_create([(0, 100)], buf, 4096, 256)[0] == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_create([(t, 100)], buf, 4096, 3)[0] == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_create([(t, 100)], buf, 0, 1)[0] == B.RL_DA_ERR_INVALID_ARG
    rc, h = B.rl_ws_create([(t, 0), (0, 0)], buf, 4096, 256)     # nothing to copy
    assert rc == B.RL_DA_OK and B.rl_ws_num_chunks(h) == (B.RL_DA_OK, 0)
    assert B.rl_ws_pack(h, 0) == B.RL_DA_ERR_INVALID_ARG
    B.rl_ws_destroy(h)
