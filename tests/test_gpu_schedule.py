"""GPU tests of the persistent unit schedule (launches with several splits).

Which work-group computes a unit, and in which order, must never change a
result: every case is compared with the fp64 oracle, and runs that take the
units in different orders (longest-first plan, plain sequence order above the
plan's batch limit, other batch compositions) must agree bit for bit.
"""
import numpy as np
import pytest
import torch

from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import bf16_to_f64, check_close, decode_extra, device, oracle_ref, run_gpu

pytestmark = pytest.mark.gpu

# batches up to this size take the longest-first plan (it lives in LDS)
PLAN_BATCH_LIMIT = 4096


def problem(hq, hkv, lengths, seed, kv="bf16", layout="hnd", max_pages=None):
    return workloads.make_problem(
        "schedule", batch=len(lengths), num_q_heads=hq, num_kv_heads=hkv,
        lengths=list(lengths), kv_dtype=kv, seed=seed, layout=layout,
        max_pages=max_pages).to(device())


def sub_problem(p, rows):
    """The same sequences (same pages, same pool) as a smaller batch."""
    idx = torch.as_tensor(rows, device=p.q.device)
    return workloads.DecodeProblem(**{**p.__dict__, "batch": len(rows),
                                      "q": p.q[idx].contiguous(),
                                      "block_table": p.block_table[idx].contiguous(),
                                      "seq_lens": p.seq_lens[idx].contiguous()})


def short_lengths(n, seed, hi=300):
    rng = np.random.default_rng(seed)
    L = rng.integers(0, hi + 1, n)
    L[rng.random(n) < 0.05] = 0
    return [int(x) for x in L]


@pytest.mark.parametrize("flags", [0, B.RL_DA_CHECKED])
@pytest.mark.parametrize("batch", [PLAN_BATCH_LIMIT, PLAN_BATCH_LIMIT + 4])
@pytest.mark.parametrize("hq,hkv", [(8, 2), (16, 2)])
def test_large_batches_with_and_without_the_plan(batch, hq, hkv, flags):
    """At the plan's batch limit the plan is largest; one past it the units
    run in sequence order.  Both match the oracle, and a sub-batch (always
    planned) gives the same bits for its sequences."""
    print("case batch", batch, "hq", hq, "hkv", hkv, "flags", flags, flush=True)
    p = problem(hq, hkv, short_lengths(batch, seed=batch + hq), seed=batch + hq)
    got = run_gpu(p, split_tokens=64, flags=flags)
    print(check_close(bf16_to_f64(got), oracle_ref(p), "batch %d G=%d" % (batch, hq // hkv),
                      extra_abs=decode_extra(p, flags)))
    rows = list(range(0, batch, 7))
    part = run_gpu(sub_problem(p, rows), split_tokens=64, flags=flags)
    assert torch.equal(part.view(torch.int16), got[rows].view(torch.int16))


@pytest.mark.parametrize("kv,layout", [("bf16", "hnd"), ("fp8_e4m3", "hnd"), ("bf16", "nhd")])
def test_checked_mode_on_the_persistent_schedule(kv, layout):
    """A checked handle on a launch with many units (longest-first plan): a
    block-table entry out of range and a sequence longer than its table row
    are reported without a fault, and every other sequence's output keeps its
    bits."""
    lengths = [1000 + 37 * (i % 11) for i in range(300)]
    p = problem(8, 2, lengths, seed=71, kv=kv, layout=layout)
    with B.DecodeAttention.for_problem(p, flags=B.RL_DA_CHECKED, split_tokens=64) as attn:
        assert attn.unit_heads() == 1 and attn.split_info(p.max_pages)[1] > 1
        good = run_gpu(p, attn=attn)
        assert attn.check_error() == 0
        print(check_close(bf16_to_f64(good), oracle_ref(p), "checked persistent " + kv + layout,
                          extra_abs=decode_extra(p, B.RL_DA_CHECKED)))
        others = [b for b in range(len(lengths)) if b not in (5, 123)]
        bad_table = p.block_table.clone()
        bad_table[123, 7] = p.num_pages + 5        # inside sequence 123
        q = workloads.DecodeProblem(**{**p.__dict__, "block_table": bad_table})
        got = run_gpu(q, attn=attn)
        assert attn.check_error() & B.RL_DA_DEVERR_PAGE_OUT_OF_RANGE
        assert torch.equal(got[others].view(torch.int16), good[others].view(torch.int16))
        long_lens = p.seq_lens.clone()
        long_lens[5] = p.max_pages * 16 + 1        # longer than its table row
        q = workloads.DecodeProblem(**{**p.__dict__, "seq_lens": long_lens})
        got = run_gpu(q, attn=attn)
        assert attn.check_error() & B.RL_DA_DEVERR_LENGTH_TOO_LONG
        assert torch.equal(got[others].view(torch.int16), good[others].view(torch.int16))


@pytest.mark.parametrize("kv,layout,flags", [
    ("bf16", "hnd", 0), ("bf16", "hnd", B.RL_DA_SCORES_ON_VALU), ("fp8_e4m3", "hnd", 0),
    ("bf16", "nhd", 0), ("fp8_e4m3", "nhd", 0), ("bf16", "nhd", B.RL_DA_PER_HEAD_UNITS)])
def test_degenerate_length_mixes(kv, layout, flags):
    """All sequences empty (only the zero writes run), one long sequence among
    empty ones, one sequence alone, one token each.  Each mix runs as it is
    (few units: one work-group per unit) and padded with empty sequences to
    500 (many units: the longest-first plan); the padded run's rows for the
    original sequences are the same bits."""
    cases = {
        "all_empty": [0] * 37,
        "one_long": [0] * 20 + [5000] + [0] * 20,
        "alone": [4097],
        "one_token_each": [1] * 300,
    }
    for name, lengths in cases.items():
        print("case", kv, layout, flags, name, flush=True)
        # a table at least 64 pages wide: several 16-page splits per row
        width = max(64, max((L + 15) // 16 for L in lengths))
        padded = lengths + [0] * (500 - len(lengths))
        p = problem(8, 2, padded, seed=len(lengths), kv=kv, layout=layout, max_pages=width)
        assert p.max_pages > 16
        # one handle for both runs: the unit family (token-major pools) follows
        # the handle's capacity, and results are batch-invariant for a handle
        with B.DecodeAttention.for_problem(p, flags=flags, split_tokens=256) as attn:
            got_padded = run_gpu(p, attn=attn)
            got = run_gpu(sub_problem(p, list(range(len(lengths)))), attn=attn)
        assert torch.equal(got.view(torch.int16), got_padded[:len(lengths)].view(torch.int16))
        got = bf16_to_f64(got)
        assert np.all(bf16_to_f64(got_padded)[len(lengths):] == 0)
        if max(lengths) == 0:
            assert np.all(got == 0)
            continue
        sub = sub_problem(p, list(range(len(lengths))))
        print(check_close(got, oracle_ref(sub), name, extra_abs=decode_extra(sub, flags)))
        assert np.all(got[np.array(lengths) == 0] == 0)


def test_queue_is_reset_between_launches_of_any_shape():
    """One handle alternates persistent launches of different sizes with
    one-split launches; each result equals a fresh handle's."""
    long_tail = problem(8, 2, [4000, 17, 0, 2500, 900, 33, 1, 3000] * 8, seed=21)
    few = problem(8, 2, [1500, 0, 700], seed=22)
    one_split = problem(8, 2, [200, 90, 250, 3, 0, 16], seed=23)
    max_pages = max(x.max_pages for x in (long_tail, few, one_split))
    runs = [(long_tail, 256), (few, 256), (one_split, 256), (long_tail, 512), (few, 64)]
    fresh = [run_gpu(p, split_tokens=s) for p, s in runs]
    for p, s in runs:
        print(check_close(bf16_to_f64(run_gpu(p, split_tokens=s)), oracle_ref(p), "queue",
                          extra_abs=decode_extra(p, 0)))
    handles = {s: B.DecodeAttention(8, 2, 64, max_pages, split_tokens=s) for s in (64, 256, 512)}
    try:
        for rep in range(3):
            for (p, s), want in zip(runs, fresh):
                got = run_gpu(p, attn=handles[s])
                assert torch.equal(got.view(torch.int16), want.view(torch.int16)), (rep, s)
    finally:
        for h in handles.values():
            h.close()
