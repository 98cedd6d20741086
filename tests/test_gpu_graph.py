"""Decode and extend launches captured in a HIP graph and replayed.

A serving loop captures its per-step launches once and replays them.  The
decode step needs no memset node for that: the persistent schedule's unit
counter is reset by the kernel's last work-group, and the allocation-free
entry point clears its scratch with a kernel.  Each replay here must equal
the eager launch bit for bit, with other eager work on the same handle (a
different batch through the same workspace) and on the outputs between the
replays.
"""
import numpy as np
import pytest
import torch

from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import bf16_to_f64, check_close, decode_extra, device, oracle_ref

pytestmark = pytest.mark.gpu

REPLAYS = 4


def problem(hq, hkv, lengths, seed, kv="bf16", layout="hnd", max_pages=None):
    return workloads.make_problem("graph", batch=len(lengths), num_q_heads=hq,
                                  num_kv_heads=hkv, lengths=list(lengths), kv_dtype=kv,
                                  seed=seed, layout=layout, max_pages=max_pages,
                                  device=device())


def same_bits(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def capture(fn):
    """fn(stream) enqueues the launches; returns the graph after one warm-up
    call on a side stream."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn(torch.cuda.current_stream())
    torch.cuda.synchronize()
    return g


# (name, Hq, Hkv, kv dtype, layout, split_tokens, lengths)
CASES = [
    ("one_split", 32, 8, "bf16", "hnd", 0, [4096, 17, 0, 1000, 3333, 16]),
    ("persistent", 32, 8, "bf16", "hnd", 512,
     [3000 + 211 * i for i in range(40)] + [0, 1, 17]),
    ("nhd_head_parallel", 32, 8, "bf16", "nhd", 0, [4096] * 12 + [100, 3000, 5000]),
    ("fp8_g8_persistent", 64, 8, "fp8_e4m3", "hnd", 1024, [2500 + 401 * i for i in range(12)]),
    ("g16", 64, 4, "bf16", "hnd", 1024, [1, 700, 2049, 5000, 0, 4096]),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_decode_replays_equal_the_eager_run(case):
    name, hq, hkv, kv, layout, split, lengths = case
    print("case", name, flush=True)
    max_pages = max((L + 15) // 16 for L in lengths)
    p = problem(hq, hkv, lengths, seed=300, kv=kv, layout=layout, max_pages=max_pages)
    # another batch of the same shapes through the same handle between replays
    other = problem(hq, hkv, lengths[::-1], seed=301, kv=kv, layout=layout,
                    max_pages=max_pages)
    with B.DecodeAttention.for_problem(p, split_tokens=split) as a:
        eager = torch.full_like(p.q, float("nan"))
        a.run_problem(p, eager)
        torch.cuda.synchronize()
        print(check_close(bf16_to_f64(eager), oracle_ref(p), "eager " + name,
                          extra_abs=decode_extra(p, 0)))
        out = torch.full_like(p.q, float("nan"))
        g = capture(lambda s: a.run_problem(p, out, s))
        scratch = torch.empty_like(other.q)
        for i in range(REPLAYS):
            out.fill_(float("nan"))
            a.run_problem(other, scratch)
            g.replay()
            torch.cuda.synchronize()
            assert same_bits(out, eager), "replay %d" % i
        del g


def test_noalloc_replays_equal_the_handle():
    """The allocation-free entry point captured with its scratch clear: every
    replay equals the handle's eager output, with eager allocation-free calls
    on another batch between the replays."""
    lengths = [2000 + 313 * i for i in range(24)] + [0, 5]
    max_pages = max((L + 15) // 16 for L in lengths)
    p = problem(32, 8, lengths, seed=310, max_pages=max_pages)
    other = problem(32, 8, lengths[::-1], seed=311, max_pages=max_pages)
    cfg = B.make_config(32, 8, len(lengths), max_pages, split_tokens=512)
    with B.DecodeAttention.for_problem(p, split_tokens=512) as a:
        eager = torch.full_like(p.q, float("nan"))
        a.run_problem(p, eager)
        torch.cuda.synchronize()

    def noalloc(q_p, out, stream):
        rc = B.rl_decode_attn_run_noalloc(cfg, q_p.q, q_p.k_pool, q_p.v_pool, q_p.k_scale,
                                          q_p.v_scale, q_p.num_pages, q_p.block_table,
                                          q_p.max_pages, q_p.seq_lens, q_p.batch, q_p.scale,
                                          out, stream)
        assert rc == B.RL_DA_OK, B.rl_da_status_string(rc)

    out = torch.full_like(p.q, float("nan"))
    g = capture(lambda s: noalloc(p, out, s))
    scratch = torch.empty_like(other.q)
    for i in range(REPLAYS):
        out.fill_(float("nan"))
        noalloc(other, scratch, torch.cuda.current_stream())
        g.replay()
        torch.cuda.synchronize()
        assert same_bits(out, eager), "replay %d" % i
    del g


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_extend_replays_equal_the_eager_launch(kv):
    new, prior = [5, 70, 33, 1], [300, 1000, 17, 4000]
    lengths = [a + b for a, b in zip(new, prior)]
    p = problem(32, 8, lengths, seed=320, kv=kv)
    gen = torch.Generator().manual_seed(321)
    q = torch.randn((sum(new), 32, 128), generator=gen).to(torch.bfloat16).to(device())
    q_start = torch.tensor(np.concatenate([[0], np.cumsum(new)]), dtype=torch.int32,
                           device=device())
    eager = torch.full_like(q, float("nan"))
    B.extend_attention(p, q, q_start, max(new), eager)
    torch.cuda.synchronize()
    assert not torch.isnan(eager.float()).any()
    out = torch.full_like(q, float("nan"))
    g = capture(lambda s: B.extend_attention(p, q, q_start, max(new), out, s))
    for i in range(REPLAYS):
        out.fill_(float("nan"))
        B.extend_attention(p, q, q_start, max(new), torch.empty_like(q))
        g.replay()
        torch.cuda.synchronize()
        assert same_bits(out, eager), "replay %d" % i
    del g
