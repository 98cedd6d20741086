"""The allocation-free decode entry point against the handle-based one.

rl_decode_attn_run_noalloc takes its workspace from a fixed device array
instead of a handle's allocation, with the same kernels and split size as a
handle created with the same configuration: its output must equal that
handle's output bit for bit (and so the oracle's, within the gate the
decode tests apply), on two calls in a row, the second with a smaller input,
so that the second call runs over whatever the first left in the scratch.
"""
import numpy as np
import pytest
import torch

from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import bf16_to_f64, check_close, decode_extra, device, oracle_ref

pytestmark = pytest.mark.gpu


def problem(hq, hkv, lengths, seed, kv="bf16", layout="hnd", max_pages=None):
    return workloads.make_problem("noalloc", batch=len(lengths), num_q_heads=hq,
                                  num_kv_heads=hkv, lengths=list(lengths), kv_dtype=kv,
                                  seed=seed, layout=layout, max_pages=max_pages,
                                  device=device())


def run_noalloc(cfg, p, stream=None):
    out = torch.full_like(p.q, float("nan"))
    rc = B.rl_decode_attn_run_noalloc(cfg, p.q, p.k_pool, p.v_pool, p.k_scale, p.v_scale,
                                      p.num_pages, p.block_table, p.max_pages, p.seq_lens,
                                      p.batch, p.scale, out, stream)
    assert rc == B.RL_DA_OK, B.rl_da_status_string(rc)
    return out


def run_handle(cfg, p):
    out = torch.full_like(p.q, float("nan"))
    rc, h = B.rl_decode_attn_create(cfg)
    assert rc == B.RL_DA_OK
    try:
        assert B.rl_decode_attn_run(h, p.q, p.k_pool, p.v_pool, p.k_scale, p.v_scale,
                                    p.num_pages, p.block_table, p.max_pages, p.seq_lens,
                                    p.batch, p.scale, out) == B.RL_DA_OK
        torch.cuda.synchronize()
    finally:
        B.rl_decode_attn_destroy(h)
    return out


# (name, Hq, Hkv, kv dtype, layout, split_tokens, first lengths, second lengths)
# The first call of each case is the larger; the handle is sized for it.
CASES = [
    # several splits, more units than the chip holds: persistent longest-first
    # schedule with the unit queue in the scratch, then the merge kernel
    ("persistent", 32, 8, "bf16", "hnd", 512,
     [3000 + 211 * i for i in range(48)] + [0, 1, 17], [700, 5000, 16, 2049, 0, 9000]),
    # e4m3 pools, one split per sequence at the default split
    ("fp8", 32, 8, "fp8_e4m3", "hnd", 0,
     [512 + 37 * i for i in range(64)], [600, 2048, 513]),
    # token-major pools, head-parallel units over several splits
    ("nhd", 32, 8, "bf16", "nhd", 0, [4096] * 16 + [100, 3000], [4096, 17, 1025]),
    # Qwen3-32B heads (G = 8), several splits
    ("g8", 64, 8, "bf16", "hnd", 1024, [2500 + 401 * i for i in range(12)], [40, 3333]),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_the_handle_on_two_calls(case):
    name, hq, hkv, kv, layout, split, first, second = case
    print("case", name, flush=True)
    max_pages = max((L + 15) // 16 for L in first + second)
    cfg = B.make_config(hq, hkv, len(first), max_pages, kv_dtype=B.KV_DTYPES[kv],
                        layout=B.LAYOUTS[layout], split_tokens=split)
    rc, need = B.rl_decode_attn_workspace_size(cfg)
    assert rc == B.RL_DA_OK and need <= B.RL_DA_NOALLOC_SCRATCH_BYTES
    pa = problem(hq, hkv, first, seed=500 + hq, kv=kv, layout=layout, max_pages=max_pages)
    pb = problem(hq, hkv, second, seed=600 + hq, kv=kv, layout=layout, max_pages=max_pages)
    got_a = run_noalloc(cfg, pa)
    got_b = run_noalloc(cfg, pb)          # right after, over the first call's scratch
    torch.cuda.synchronize()
    for p, got in ((pa, got_a), (pb, got_b)):
        want = run_handle(cfg, p)
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), name
        stats = check_close(bf16_to_f64(got), oracle_ref(p), "noalloc " + name,
                            extra_abs=decode_extra(p, cfg.flags))
        print(name, p.batch, stats, flush=True)
        assert np.all(bf16_to_f64(got)[p.lengths() == 0] == 0)


def test_noalloc_rejects_a_step_beyond_its_scratch():
    p = problem(32, 8, [40, 70], seed=700)
    big = B.make_config(32, 8, 1024, 4096, split_tokens=512)
    out = torch.full_like(p.q, 7.0)
    rc = B.rl_decode_attn_run_noalloc(big, p.q, p.k_pool, p.v_pool, None, None, p.num_pages,
                                      p.block_table, p.max_pages, p.seq_lens, p.batch,
                                      p.scale, out)
    assert rc == B.RL_DA_ERR_SCRATCH_TOO_SMALL
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)        # nothing was enqueued
