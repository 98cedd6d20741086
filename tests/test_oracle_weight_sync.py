"""Pins for the weight-sync / checkpoint oracle (CPU only).

The placement rule has no printed example in the paper, so the oracle is
pinned to a plan worked out by hand, to a closed form (with align 1 the chunks
are the consecutive capacity-sized slices of the concatenated byte stream), to
invariants any valid plan of this rule has (coverage, alignment, capacity,
order, a chunk ends only when the aligned cursor reaches capacity) and to the
pack/unpack round trip.  Each check is a function of the oracle module so that
the mutant test at the end can run the same checks against planted slips.
"""
import os

import numpy as np
import pytest

from oracle import weight_sync as WS

# Worked by hand: capacity 4096, align 256.
#   t0 10 B    -> chunk 0 @ 0                               cursor 10
#   t1 300 B   -> chunk 0 @ 256                             cursor 556
#   t2 5000 B  -> chunk 0 @ 768 takes 3328 (to 4096), rest 1672 -> chunk 1 @ 0
#   t3 0 B     -> no piece
#   t4 1 B     -> chunk 1 @ 1792 (align_up(1672))           cursor 1793
#   t5 7000 B  -> chunk 1 @ 2048 takes 2048; chunk 2 @ 0 takes 4096;
#                 chunk 3 @ 0 takes the last 856
HAND_SIZES = [10, 300, 5000, 0, 1, 7000]
HAND_PIECES = [
    (0, 0, 0, 0, 10),
    (1, 0, 0, 256, 300),
    (2, 0, 0, 768, 3328),
    (2, 1, 3328, 0, 1672),
    (4, 1, 0, 1792, 1),
    (5, 1, 0, 2048, 2048),
    (5, 2, 2048, 0, 4096),
    (5, 3, 6144, 0, 856),
]


def random_sizes(rng, n, big):
    kinds = rng.integers(0, 4, n)
    sizes = np.where(kinds == 0, 0, np.where(kinds == 1, rng.integers(1, 64, n),
                     np.where(kinds == 2, rng.integers(1, 5000, n), rng.integers(1, big, n))))
    return [int(x) for x in sizes]


def check_hand_example(ws):
    got = ws.plan(HAND_SIZES, 4096, 256)
    assert [tuple(p) for p in got] == HAND_PIECES
    assert ws.num_chunks(got) == 4


def check_align1_is_stream_slicing(ws):
    rng = np.random.default_rng(1)
    sizes = random_sizes(rng, 40, 20000)
    data = [rng.integers(0, 256, n, dtype=np.uint8) for n in sizes]
    stream = np.concatenate(data)
    cap = 3001
    pieces = ws.plan(sizes, cap, 1)
    assert ws.num_chunks(pieces) == -(-len(stream) // cap)
    for c in range(ws.num_chunks(pieces)):
        buf, written = ws.pack(data, pieces, c, cap)
        want = stream[c * cap:(c + 1) * cap]
        assert np.array_equal(buf[:len(want)], want)
        assert written[:len(want)].all() and not written[len(want):].any()


def check_invariants(ws):
    rng = np.random.default_rng(2)
    for cap, align in ((4096, 256), (1 << 16, 16), (512, 512), (1000, 8), (64, 1)):
        sizes = random_sizes(rng, 60, 3 * cap)
        pieces = ws.plan(sizes, cap, align)
        # each tensor is covered once, in order, by contiguous pieces
        for i, n in enumerate(sizes):
            mine = [p for p in pieces if p[0] == i]
            assert sum(p[4] for p in mine) == n
            off = 0
            for p in mine:
                assert p[2] == off and p[4] >= 1
                assert off % align == 0          # splits fall on multiples of align
                off += p[4]
        assert [p[0] for p in pieces] == sorted(p[0] for p in pieces)
        chunks = [p[1] for p in pieces]
        assert chunks == sorted(chunks)
        if pieces:
            assert sorted(set(chunks)) == list(range(chunks[-1] + 1))
        prev = None
        for p in pieces:
            assert p[3] % align == 0 and p[3] + p[4] <= cap
            if prev is not None:
                end = prev[3] + prev[4]
                if p[1] == prev[1]:
                    assert p[3] == -(-end // align) * align   # next aligned slot, no gap beyond
                else:
                    assert p[3] == 0 and -(-end // align) * align >= cap  # chunk was full
            prev = p


def check_round_trip(ws):
    rng = np.random.default_rng(3)
    sizes = random_sizes(rng, 30, 9000)
    data = [rng.integers(0, 256, n, dtype=np.uint8) for n in sizes]
    cap = 4096
    pieces = ws.plan(sizes, cap, 128)
    restored = [np.zeros(n, dtype=np.uint8) for n in sizes]
    for c in range(ws.num_chunks(pieces)):
        buf, _ = ws.pack(data, pieces, c, cap, fill=0xA5)
        restored = ws.unpack(buf, pieces, c, restored)
    for a, b in zip(data, restored):
        assert np.array_equal(a, b)


def check_one_chunk_closed_form(ws):
    """When everything fits, offsets are the aligned prefix sums."""
    sizes = [3, 0, 17, 256, 1, 100]
    pieces = ws.plan(sizes, 1 << 20, 64)
    offs, cursor = [], 0
    for n in sizes:
        if n:
            cursor = (cursor + 63) // 64 * 64
            offs.append(cursor)
            cursor += n
    assert [p[3] for p in pieces] == offs
    assert all(p[1] == 0 and p[2] == 0 for p in pieces)


CHECKS = [check_hand_example, check_align1_is_stream_slicing, check_invariants,
          check_round_trip, check_one_chunk_closed_form]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_pins(check):
    check(WS)


def test_bad_plan_arguments():
    for cap, align in ((0, 1), (100, 3), (100, 64), (64, 0)):
        with pytest.raises(ValueError):
            WS.plan([1], cap, align)
    assert WS.plan([], 64, 1) == [] and WS.num_chunks([]) == 0


MUTANTS = [
    ("chunk closes one byte late", "if off >= capacity:", "if off > capacity:"),
    ("no alignment", "return (x + a - 1) // a * a", "return x"),
    ("align rounds down", "return (x + a - 1) // a * a", "return x // a * a"),
    ("room ignores the cursor", "take = min(n - done, capacity - off)",
     "take = min(n - done, capacity)"),
    ("split restarts the tensor", "pieces.append((i, chunk, done, off, take))",
     "pieces.append((i, chunk, 0, off, take))"),
    ("pack reads the buffer offset", "buf[b_off:b_off + n] = tensors[t][t_off:t_off + n]",
     "buf[b_off:b_off + n] = tensors[t][b_off:b_off + n]"),
    ("unpack to the buffer offset", "out[t][t_off:t_off + n] = buffer[b_off:b_off + n]",
     "out[t][b_off:b_off + n] = buffer[b_off:b_off + n]"),
]


_RUN_CHECKS = """
import importlib.util, sys
sys.path.insert(0, {tests!r})
import test_oracle_weight_sync as T
spec = importlib.util.spec_from_file_location("ws_mutant", {path!r})
mod = importlib.util.module_from_spec(spec)
spec.loader.exec_module(mod)
for check in T.CHECKS:
    check(mod)
"""


def _checks_pass(path):
    """True if every check passes on the module at `path`; a check that runs
    past the time limit (a mutant that never ends) counts as failing."""
    import subprocess
    import sys
    code = _RUN_CHECKS.format(tests=os.path.dirname(os.path.abspath(__file__)), path=str(path))
    try:
        r = subprocess.run([sys.executable, "-c", code], stdout=subprocess.DEVNULL,
                           stderr=subprocess.DEVNULL, timeout=15,
                           cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    except subprocess.TimeoutExpired:
        return False
    return r.returncode == 0


def test_pins_catch_every_mutant(tmp_path):
    src = open(os.path.join(os.path.dirname(WS.__file__), "weight_sync.py")).read()
    control = tmp_path / "ws_control.py"
    control.write_text(src)
    assert _checks_pass(control), "unmodified oracle fails its pins"
    survivors = []
    for k, (name, old, new) in enumerate(MUTANTS):
        assert src.count(old) == 1, "mutation site not unique: " + name
        path = tmp_path / ("ws_mutant_%d.py" % k)
        path.write_text(src.replace(old, new))
        if _checks_pass(path):
            survivors.append(name)
    assert not survivors, "mutants not caught: %s" % survivors
