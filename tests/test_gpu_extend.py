"""GPU extend (prefill) attention against the fp64 oracle: ragged new-token
counts over ragged cached prefixes for every supported group size, poisoned
unread memory, causality, and argument checks."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import abs_value_host, bf16_to_f64, check_close, device, extend_extra

pytestmark = pytest.mark.gpu


def extend_problem(new, prior, seed, hq=8, hkv=2, layout="hnd", kv="bf16"):
    lengths = [a + b for a, b in zip(new, prior)]
    p = workloads.make_problem("ext", batch=len(new), num_q_heads=hq, num_kv_heads=hkv,
                               lengths=lengths, seed=seed, pool_factor=1.25,
                               layout=layout, kv_dtype=kv).to(device())
    gen = torch.Generator().manual_seed(seed + 3)
    q = torch.randn((int(sum(new)), hq, 128), generator=gen).to(torch.bfloat16).to(device())
    q_start = torch.tensor(np.concatenate([[0], np.cumsum(new)]), dtype=torch.int32,
                           device=device())
    return p, q, q_start


def run_extend(p, q, q_start, max_new):
    out = torch.full_like(q, float("nan"))
    B.extend_attention(p, q, q_start, max_new, out)
    torch.cuda.synchronize()
    return out


def oracle_extend(p, q, q_start, abs_values=False):
    """The oracle's extend attention of problem p; with abs_values, over the
    value pool of magnitudes |V| (same weights), which gives M1."""
    h = p.host_arrays()
    kw = {}
    if p.kv_dtype != "bf16":
        kw = dict(kv_dtype=oracle.KV_FP8_E4M3, k_scale=h["k_scale"], v_scale=h["v_scale"])
    v_pool = abs_value_host(p, h) if abs_values else h["v_pool"]
    return oracle.extend_attention(q.cpu().view(torch.int16).numpy().view(np.uint16),
                                   q_start.cpu().numpy(), h["k_pool"], v_pool,
                                   h["block_table"], h["seq_lens"],
                                   num_kv_heads=p.num_kv_heads, scale=p.scale,
                                   layout=h["layout"], **kw)


def check_extend(p, q, q_start, got, what):
    """Official bound, and one bf16 ulp plus the rounded-probability
    allowance derived from each row's own weights (extend_extra)."""
    ref = oracle_extend(p, q, q_start)
    extra = extend_extra(p.kv_dtype, ref, oracle_extend(p, q, q_start, abs_values=True))
    stats = check_close(bf16_to_f64(got), ref, what, extra_abs=extra)
    print(what, stats, flush=True)
    return stats


def check_rows_as_decode(p, got_row, q_bits_row, b, visible, what, kw=None):
    """New token of sequence b that sees `visible` cached tokens: all its heads
    against the oracle's decode attention over that prefix."""
    h = p.host_arrays()
    kw = kw or {}
    lens = h["seq_lens"].copy()
    lens[b] = visible
    qrow = np.repeat(q_bits_row, p.batch, axis=0)
    rows = [[b, hh] for hh in range(p.num_q_heads)]
    args = (h["k_pool"], h["block_table"], lens)
    ref = oracle.decode_attention(qrow, args[0], h["v_pool"], args[1], args[2],
                                  num_kv_heads=p.num_kv_heads, scale=p.scale, rows=rows, **kw)
    m1 = oracle.decode_attention(qrow, args[0], abs_value_host(p, h), args[1], args[2],
                                 num_kv_heads=p.num_kv_heads, scale=p.scale, rows=rows, **kw)
    return check_close(bf16_to_f64(got_row), ref, what,
                       extra_abs=extend_extra(p.kv_dtype, ref, m1))


CASES = [
    ([1, 3, 5, 16, 17, 33], [0, 7, 100, 4000, 15, 1]),
    ([64, 1, 100, 0, 2], [0, 63, 1000, 5, 9]),
    ([200], [3000]),
]


@pytest.mark.parametrize("hq,hkv", [(8, 2), (4, 4), (8, 4), (16, 2), (32, 2)])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_extend_matches_oracle(hq, hkv, case):
    new, prior = CASES[case]
    p, q, q_start = extend_problem(new, prior, seed=31 + case, hq=hq, hkv=hkv)
    got = run_extend(p, q, q_start, max(new))
    check_extend(p, q, q_start, got, "extend G=%d case %d" % (hq // hkv, case))


@pytest.mark.parametrize("pattern", ["every_other_negative", "all_negative", "zero_and_negative"])
def test_extend_fp8_slab_scales_of_either_sign(pattern):
    """e4m3 slab scales of either sign, or zero: a page whose k_scale is
    negative turns its largest codes into its smallest scores (below the
    diagonal its row max comes from the raw minimum), and a zero scale makes
    all its scores 0."""
    new, prior = [5, 70, 33, 1, 130], [300, 1000, 17, 4000, 64]
    p, q, q_start = extend_problem(new, prior, seed=90, kv="fp8_e4m3")
    if pattern == "every_other_negative":
        p.k_scale[::2] *= -1.0
    elif pattern == "all_negative":
        p.k_scale *= -1.0
    else:
        p.k_scale[::3] = 0.0
        p.k_scale[1::3] *= -1.0
    got = run_extend(p, q, q_start, max(new))
    check_extend(p, q, q_start, got, "extend fp8 k_scale " + pattern)


def test_extend_qwen3_8b_shapes_sampled():
    new, prior = [512, 300, 77, 1], [4096, 8000, 20, 12000]
    p, q, q_start = extend_problem(new, prior, seed=40, hq=32, hkv=8)
    got = run_extend(p, q, q_start, max(new))
    # oracle on a sample of rows: the oracle takes whole sequences, so restrict
    # each sequence's rows by passing a sub-problem of 4 chosen tokens each
    qs = q_start.cpu().numpy()
    q_bits = q.cpu().view(torch.int16).numpy().view(np.uint16)
    for b in range(4):
        n = new[b]
        for i in sorted({0, n // 2, n - 1}):
            r = qs[b] + i
            print(check_rows_as_decode(p, got[r], q_bits[r:r + 1], b, prior[b] + i + 1,
                                       "row b=%d i=%d" % (b, i)))


@pytest.mark.parametrize("config,n", [("qwen3_8b_step", 512), ("fp8_large_batch", 128)])
def test_extend_bench_workloads_sampled(config, n):
    """The inputs `bench.py --op extend` times, built the same way (every
    sequence gets n new tokens after its drawn length), in the same launch:
    new tokens 0, n/2 and n-1 of the longest, the shortest and two other
    sequences match the oracle, each as a decode query over its visible
    prefix."""
    cfg = dict(workloads.CONFIGS[config])
    seed = cfg.pop("seed")
    prior = workloads.draw_lengths(np.random.default_rng(seed), cfg["batch"], cfg["lengths"])
    cfg["lengths"] = [int(x) + n for x in prior]
    p = workloads.make_problem(config + "+extend", seed=seed, device=device(), **cfg)
    T = n * p.batch
    gen = torch.Generator(device=device()).manual_seed(seed + 1)
    q = torch.randn((T, p.num_q_heads, p.head_dim), generator=gen,
                    device=device()).to(torch.bfloat16)
    q_start = torch.arange(0, T + 1, n, dtype=torch.int32, device=device())
    got = run_extend(p, q, q_start, n)
    assert torch.isfinite(got.float()).all()
    h = p.host_arrays()
    kw = {}
    if p.kv_dtype != "bf16":
        kw = dict(kv_dtype=oracle.KV_FP8_E4M3, k_scale=h["k_scale"], v_scale=h["v_scale"])
    order = np.argsort(np.asarray(prior), kind="stable")
    seqs = sorted({int(order[-1]), int(order[0]), int(order[len(order) // 3]),
                   int(order[2 * len(order) // 3])})
    q_bits = q.cpu().view(torch.int16).numpy().view(np.uint16)
    for b in seqs:
        for i in sorted({0, n // 2, n - 1}):
            r = b * n + i
            print(check_rows_as_decode(p, got[r], q_bits[r:r + 1], b, int(prior[b]) + i + 1,
                                       "%s b=%d i=%d" % (config, b, i), kw))


def test_extend_ignores_unread_memory_and_is_causal():
    new, prior = [20, 5], [13, 40]
    p, q, q_start = extend_problem(new, prior, seed=41)
    base = run_extend(p, q, q_start, 20)
    bt = p.block_table.cpu().numpy()
    nan = float("nan")
    for b, L in enumerate([33, 45]):
        last, tail = int(bt[b, (L - 1) // 16]), L % 16
        if tail:
            p.k_pool[last, :, tail:, :] = nan
            p.v_pool[last, :, tail:, :] = nan
    assert torch.equal(run_extend(p, q, q_start, 20).view(torch.int16), base.view(torch.int16))
    # the last cached token of sequence 0 is visible only to its last new token
    last, slot = int(bt[0, 32 // 16]), 32 % 16
    p.k_pool[last, :, slot, :] *= -3.0
    moved = run_extend(p, q, q_start, 20)
    assert torch.equal(moved[:19].view(torch.int16), base[:19].view(torch.int16))
    assert not torch.equal(moved[19].view(torch.int16), base[19].view(torch.int16))
    assert torch.equal(moved[20:].view(torch.int16), base[20:].view(torch.int16))


@pytest.mark.parametrize("kv,layout", [("bf16", "hnd"), ("fp8_e4m3", "hnd"), ("bf16", "nhd"),
                                       ("fp8_e4m3", "nhd")])
def test_extend_ignores_unstaged_memory_and_the_table_tail(kv, layout):
    """Keys past a sequence's end are read from a slot of its last page and
    discarded; table entries past a sequence's pages are never read; pages
    no sequence uses are never read.  With the slots past each sequence's end
    NaN, an unused page 0 NaN (codes and, for e4m3 pools, scales) and every
    table row's tail out of range, each output keeps its bits."""
    new, prior = [37, 1, 64, 20, 9], [70, 0, 130, 300, 7]   # partial pages and stages
    p, q, q_start = extend_problem(new, prior, seed=44, hq=16, hkv=4, layout=layout, kv=kv)
    bt = p.block_table.clone()
    lens = [int(L) for L in p.seq_lens.cpu()]
    pages = [(L + 15) // 16 for L in lens]
    used = {int(x) for b, n in enumerate(pages) for x in bt[b, :n].cpu()}
    if 0 in used:  # move page 0's tokens to a spare page
        spare = next(x for x in range(1, p.num_pages) if x not in used)
        for t in (p.k_pool, p.v_pool) + ((p.k_scale, p.v_scale) if kv != "bf16" else ()):
            t[spare] = t[0]
        for b, n in enumerate(pages):
            row = bt[b, :n]
            row[row == 0] = spare
    p = workloads.DecodeProblem(**{**p.__dict__, "block_table": bt})
    base = run_extend(p, q, q_start, max(new))
    check_extend(p, q, q_start, base, "unstaged " + kv + layout)
    nan_code = float("nan") if kv == "bf16" else 0x7F   # e4m3 NaN
    for pool in (p.k_pool, p.v_pool):
        pool[0] = nan_code
        for b, L in enumerate(lens):
            last, tail = int(bt[b, (L - 1) // 16]), L % 16
            if tail:
                if layout == "hnd":
                    pool[last, :, tail:, :] = nan_code
                else:
                    pool[last, tail:, :, :] = nan_code
    if kv != "bf16":
        p.k_scale[0] = float("nan")
        p.v_scale[0] = float("nan")
    tail = bt.clone()
    for b, n in enumerate(pages):
        tail[b, n:] = 1 << 30
    got = run_extend(workloads.DecodeProblem(**{**p.__dict__, "block_table": tail}),
                     q, q_start, max(new))
    assert torch.equal(got.view(torch.int16), base.view(torch.int16))


def test_extend_longest_first_order_on_a_large_batch():
    """Work-groups take the sequences longest first; every work-group derives
    the order from the lengths, keeping each sequence's length class in LDS
    for the first 36864 sequences and reading the lengths again past that.
    A batch of 37000 sequences, nearly all empty, with real ones of six
    length classes on both sides of that index: their rows match the oracle."""
    batch = 37000
    real = {5: (3000, 40), 300: (20, 5), 9000: (33000, 17), 36863: (700, 64),
            36864: (5000, 33), 36999: (100, 1), 20000: (1, 1), 15000: (12000, 2)}
    prior = [0] * batch
    new = [0] * batch
    for b, (pre, n) in real.items():
        prior[b], new[b] = pre, n
    p, q, q_start = extend_problem(new, prior, seed=45, hq=4, hkv=1)
    got = run_extend(p, q, q_start, max(new))
    rows = sorted(real)
    sub = workloads.DecodeProblem(**{**p.__dict__, "batch": len(rows),
                                     "block_table": p.block_table[rows].contiguous(),
                                     "seq_lens": p.seq_lens[rows].contiguous()})
    qs = q_start.cpu().numpy()
    sub_q = torch.cat([q[qs[b]:qs[b + 1]] for b in rows])
    sub_start = torch.tensor(np.concatenate([[0], np.cumsum([new[b] for b in rows])]),
                             dtype=torch.int32, device=q.device)
    check_extend(sub, sub_q, sub_start, got, "longest-first, 37000 sequences")


def test_extend_argument_validation():
    p, q, q_start = extend_problem([3, 2], [4, 4], seed=42)
    out = torch.empty_like(q)

    def call(**kw):
        args = dict(q=q, q_start=q_start, max_q_per_seq=3, k_pool=p.k_pool, v_pool=p.v_pool,
                    k_scale=None, v_scale=None, num_pages=p.num_pages,
                    block_table=p.block_table, max_pages=p.max_pages, seq_lens=p.seq_lens,
                    batch=2, num_q_heads=8, num_kv_heads=2, scale=p.scale, out=out)
        args.update(kw)
        return B.rl_extend_attn(**args)

    assert call() == B.RL_DA_OK
    assert call(q=None) == B.RL_DA_ERR_INVALID_ARG
    assert call(num_q_heads=7) == B.RL_DA_ERR_INVALID_ARG
    assert call(out=out.data_ptr() + 2) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_scale=p.seq_lens) == B.RL_DA_ERR_INVALID_ARG
    assert call(head_dim=64) == B.RL_DA_ERR_UNSUPPORTED
    assert call(num_q_heads=6) == B.RL_DA_ERR_UNSUPPORTED
    assert call(layout=3) == B.RL_DA_ERR_INVALID_ARG
    assert call(max_q_per_seq=0) == B.RL_DA_OK
    torch.cuda.synchronize()


@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (4, 1)])
def test_extend_nhd_pools_match_oracle_and_the_hnd_result(hq, hkv):
    new, prior = CASES[0]
    pn, q, q_start = extend_problem(new, prior, seed=40 + hq, hq=hq, hkv=hkv, layout="nhd")
    ph, _, _ = extend_problem(new, prior, seed=40 + hq, hq=hq, hkv=hkv)
    got = run_extend(pn, q, q_start, max(new))
    check_extend(pn, q, q_start, got, "extend nhd G=%d" % (hq // hkv))
    same = run_extend(ph, q, q_start, max(new))
    assert torch.equal(got.view(torch.int16), same.view(torch.int16))


@pytest.mark.parametrize("layout", ["hnd", "nhd"])
@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (16, 16)])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_extend_fp8_pools_match_oracle(hq, hkv, case, layout):
    """e4m3 pools with per-slab scales: codes staged as exact bf16, k_scale on
    the scores, v_scale on the probabilities."""
    new, prior = CASES[case]
    p, q, q_start = extend_problem(new, prior, seed=50 + case, hq=hq, hkv=hkv, layout=layout,
                                   kv="fp8_e4m3")
    got = run_extend(p, q, q_start, max(new))
    check_extend(p, q, q_start, got, "extend fp8 %s G=%d case %d" % (layout, hq // hkv, case))


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (64, 4)])
def test_extend_hnd_kv_pools_match_oracle_and_the_hnd_result(kv, hq, hkv):
    """Key and value slabs side by side in one allocation: the same bits as
    head-major pools holding the same values."""
    new, prior = CASES[0]
    pk, q, q_start = extend_problem(new, prior, seed=60 + hq, hq=hq, hkv=hkv, layout="hnd_kv",
                                    kv=kv)
    ph, _, _ = extend_problem(new, prior, seed=60 + hq, hq=hq, hkv=hkv, kv=kv)
    got = run_extend(pk, q, q_start, max(new))
    check_extend(pk, q, q_start, got, "extend hnd_kv %s G=%d" % (kv, hq // hkv))
    same = run_extend(ph, q, q_start, max(new))
    assert torch.equal(got.view(torch.int16), same.view(torch.int16))


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_extend_rows_do_not_depend_on_the_rest_of_the_batch(kv):
    """A sequence's tiles, their key stages and the order of every sum depend
    only on its own cached length and new-token count, so its output rows are
    the same bits extended alone, in a batch, or at another batch position
    (the work-group order does change with the batch: longest first)."""
    new, prior = [7, 70, 1, 33, 100], [4000, 17, 900, 2500, 64]
    p, q, q_start = extend_problem(new, prior, seed=51, hq=32, hkv=8, kv=kv)
    full = run_extend(p, q, q_start, max(new))
    starts = q_start.cpu().numpy()
    for rows in ([1], [3, 0], [4, 2, 1]):
        idx = torch.as_tensor(rows, device=p.q.device)
        sub = workloads.DecodeProblem(**{**p.__dict__, "batch": len(rows),
                                         "block_table": p.block_table[idx].contiguous(),
                                         "seq_lens": p.seq_lens[idx].contiguous()})
        sub_new = [new[b] for b in rows]
        sub_q = torch.cat([q[starts[b]:starts[b + 1]] for b in rows]).contiguous()
        sub_start = torch.tensor(np.concatenate([[0], np.cumsum(sub_new)]), dtype=torch.int32,
                                 device=device())
        got = run_extend(sub, sub_q, sub_start, max(sub_new))
        at = 0
        for b, n in zip(rows, sub_new):
            assert torch.equal(got[at:at + n].view(torch.int16),
                               full[starts[b]:starts[b] + n].view(torch.int16)), (rows, b)
            at += n
