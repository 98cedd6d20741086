"""The library's weight-sync plan (host code behind the C interface, no GPU)
against the oracle's plan: identical pieces and chunk counts."""
import numpy as np
import pytest

from oracle import weight_sync as WS
from paper_2512_22492_amd import binding as B

from test_oracle_weight_sync import HAND_PIECES, HAND_SIZES, random_sizes


def test_hand_example():
    rc, pieces, nc = B.rl_ws_plan(HAND_SIZES, 4096, 256)
    assert rc == B.RL_DA_OK
    assert pieces == HAND_PIECES and nc == 4


@pytest.mark.parametrize("cap,align", [(4096, 256), (1 << 16, 16), (512, 512), (1000, 8),
                                       (64, 1), (3001, 1), (1 << 30, 4096)])
def test_matches_oracle_on_random_tensor_lists(cap, align):
    rng = np.random.default_rng(cap + align)
    for _ in range(5):
        sizes = random_sizes(rng, 80, 3 * cap if cap < (1 << 20) else 1 << 22)
        want = WS.plan(sizes, cap, align)
        rc, got, nc = B.rl_ws_plan(sizes, cap, align)
        assert rc == B.RL_DA_OK
        assert got == want
        assert nc == WS.num_chunks(want)


def test_model_sized_tensors():
    """Sizes beyond 32 bits (a 151936 x 4096 bf16 embedding, 1.24 GB, and a
    5 GB tensor) plan the same on both sides."""
    sizes = [151936 * 4096 * 2, 8192, 0, 5 << 30, 4096 * 2, 12288 * 4096 * 2]
    for cap in (1 << 30, 1 << 28, 3 << 29):
        rc, got, nc = B.rl_ws_plan(sizes, cap, 256)
        assert rc == B.RL_DA_OK and got == WS.plan(sizes, cap, 256)


def test_empty_and_zero_byte_lists():
    assert B.rl_ws_plan([], 64, 1) == (B.RL_DA_OK, [], 0)
    assert B.rl_ws_plan([0, 0], 64, 1) == (B.RL_DA_OK, [], 0)


@pytest.mark.parametrize("cap,align", [(0, 1), (100, 3), (100, 64), (64, 0)])
def test_bad_capacity_or_alignment(cap, align):
    rc, _, _ = B.rl_ws_plan([1, 2], cap, align)
    assert rc == B.RL_DA_ERR_INVALID_ARG


def test_count_query_and_short_output():
    import ctypes
    lib = B.load_library()
    sizes = (ctypes.c_uint64 * 3)(5000, 10, 9000)
    n, c = ctypes.c_int64(), ctypes.c_int32()
    assert lib.rl_ws_plan(sizes, 3, 4096, 256, None, 0, ctypes.byref(n), ctypes.byref(c)) == 0
    assert (n.value, c.value) == (len(WS.plan([5000, 10, 9000], 4096, 256)), 4)
    two = (B.rl_ws_piece * 2)()
    assert lib.rl_ws_plan(sizes, 3, 4096, 256, two, 2, ctypes.byref(n), ctypes.byref(c)) == 0
    assert n.value == 6 and [(p.tensor, p.nbytes) for p in two] == [(0, 4096), (0, 904)]
    assert lib.rl_ws_plan(sizes, 3, 4096, 256, None, 2, ctypes.byref(n),
                          ctypes.byref(c)) == B.RL_DA_ERR_INVALID_ARG
    assert lib.rl_ws_plan(None, 3, 4096, 256, None, 0, ctypes.byref(n),
                          ctypes.byref(c)) == B.RL_DA_ERR_INVALID_ARG
    assert lib.rl_ws_plan(sizes, -1, 4096, 256, None, 0, ctypes.byref(n),
                          ctypes.byref(c)) == B.RL_DA_ERR_INVALID_ARG


def test_create_and_copy_reject_null_arguments_without_gpu():
    import ctypes
    lib = B.load_library()
    h = ctypes.c_void_p()
    assert lib.rl_ws_create(None, 1, None, 64, 1, ctypes.byref(h)) == B.RL_DA_ERR_INVALID_ARG
    assert lib.rl_ws_create(None, 0, None, 64, 1, None) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_pack(None, 0) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_unpack(None, 0) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_num_chunks(None)[0] == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_chunk_bytes(None, 0)[0] == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_ws_destroy(None) == B.RL_DA_OK
