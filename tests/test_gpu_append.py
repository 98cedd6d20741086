"""GPU KV-cache append against the oracle: pools and slab scales must match
byte for byte (integer/byte work, and every fp8 decision is made in fp32 on
both sides), over many decode steps that cross page boundaries, grow and
keep e4m3 slab scales; then attention over the appended cache must match the
oracle's attention over the oracle-appended cache."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import PV_ROUND, KV, bf16_to_f64, check_close, device, oracle_ref, run_gpu

pytestmark = pytest.mark.gpu


def grown_problem(kv, lengths, steps, seed, hq=8, hkv=2, layout="hnd"):
    """Pages for lengths + steps tokens are in the table already; seq_lens
    start at lengths."""
    p = workloads.make_problem("append", batch=len(lengths), num_q_heads=hq,
                               num_kv_heads=hkv, lengths=[L + steps for L in lengths],
                               kv_dtype=kv, seed=seed, pool_factor=1.5,
                               layout=layout).to(device())
    p.seq_lens.copy_(torch.tensor(lengths, dtype=torch.int32, device=device()))
    return p


def new_tokens(p, step, gen):
    """Per-step tokens with magnitudes that both grow and shrink the slab scales."""
    mag = [1.0, 50.0, 1e-3, 3.0, 0.25][step % 5]
    shape = (p.batch, p.num_kv_heads, p.head_dim)
    k = (torch.randn(shape, generator=gen) * mag).to(torch.bfloat16)
    v = (torch.randn(shape, generator=gen) * mag).to(torch.bfloat16)
    return k, v


def host_bits(t):
    return t.view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("layout", ["hnd", "nhd", "hnd_kv"])
@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_append_steps_match_oracle_byte_for_byte(kv, layout):
    lengths = [0, 1, 14, 15, 16, 31, 100, 4095, 4096, 5000]
    steps = 20
    p = grown_problem(kv, lengths, steps, seed=21, hkv=2 if layout == "hnd" else 4,
                      hq=8, layout=layout)
    h = p.host_arrays()
    ok, ov = h["k_pool"], h["v_pool"]
    oks, ovs = h.get("k_scale"), h.get("v_scale")
    gen = torch.Generator().manual_seed(22)
    for step in range(steps):
        k, v = new_tokens(p, step, gen)
        lens = p.seq_lens.cpu().numpy()
        B.kv_append(p, k.to(device()), v.to(device()))
        ok, ov, oks, ovs = oracle.kv_append(host_bits(k), host_bits(v), ok, ov,
                                            h["block_table"], lens, kv_dtype=KV[kv],
                                            k_scale=oks, v_scale=ovs, layout=h["layout"])
        p.seq_lens += 1
        torch.cuda.synchronize()
        got = p.host_arrays()
        assert np.array_equal(got["k_pool"], ok), "K pool differs after step %d" % step
        assert np.array_equal(got["v_pool"], ov), "V pool differs after step %d" % step
        if kv != "bf16":
            assert np.array_equal(got["k_scale"], oks), "k_scale differs after step %d" % step
            assert np.array_equal(got["v_scale"], ovs), "v_scale differs after step %d" % step
    # attention over the appended cache
    ref, m1 = [oracle.decode_attention(
        got["q_bits"], ok, v, h["block_table"], p.seq_lens.cpu().numpy(),
        num_kv_heads=p.num_kv_heads, scale=p.scale, kv_dtype=KV[kv], k_scale=oks,
        v_scale=ovs, layout=h["layout"])
        for v in (ov, ov & (np.uint16(0x7FFF) if ov.dtype == np.uint16 else np.uint8(0x7F)))]
    print(check_close(bf16_to_f64(run_gpu(p)), ref, "attention after appends " + kv,
                      extra_abs=PV_ROUND * m1))


def test_negative_length_is_skipped_and_errors_are_reported():
    p = grown_problem("fp8_e4m3", [5, 7, 9], 1, seed=23)
    before = p.host_arrays()
    err = torch.zeros(1, dtype=torch.int32, device=device())
    gen = torch.Generator().manual_seed(24)
    k, v = new_tokens(p, 0, gen)
    p.seq_lens.copy_(torch.tensor([-1, p.max_pages * 16, 9], dtype=torch.int32,
                                  device=device()))
    bad_table = p.block_table.clone()
    bad_table[2, 0] = p.num_pages + 3         # page of token 9 is out of range
    good_table = p.block_table
    p.block_table = bad_table
    B.kv_append(p, k.to(device()), v.to(device()), device_error=err)
    torch.cuda.synchronize()
    p.block_table = good_table
    after = p.host_arrays()
    for name in ("k_pool", "v_pool", "k_scale", "v_scale"):
        assert np.array_equal(before[name], after[name]), name
    bits = int(err.item())
    assert bits & B.RL_DA_DEVERR_LENGTH_TOO_LONG
    assert bits & B.RL_DA_DEVERR_PAGE_OUT_OF_RANGE


def test_append_argument_validation():
    p = grown_problem("bf16", [3, 4], 1, seed=25)
    k = torch.zeros((2, 2, 128), dtype=torch.bfloat16, device=device())

    def call(**kw):
        args = dict(k_new=k, v_new=k, k_pool=p.k_pool, v_pool=p.v_pool, k_scale=None,
                    v_scale=None, num_pages=p.num_pages, block_table=p.block_table,
                    max_pages=p.max_pages, seq_lens=p.seq_lens, batch=2, num_kv_heads=2)
        args.update(kw)
        return B.rl_kv_append(**args)

    assert call() == B.RL_DA_OK
    assert call(batch=-1) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_new=None) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_pool=p.k_pool.data_ptr() + 2) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_scale=p.seq_lens) == B.RL_DA_ERR_INVALID_ARG
    assert call(head_dim=64) == B.RL_DA_ERR_UNSUPPORTED
    assert call(page_size=32) == B.RL_DA_ERR_UNSUPPORTED
    assert call(kv_dtype=5) == B.RL_DA_ERR_INVALID_ARG
    assert call(layout=3) == B.RL_DA_ERR_INVALID_ARG
    assert call(layout=2) == B.RL_DA_ERR_INVALID_ARG   # two pools, not one slab apart
    assert call(batch=0) == B.RL_DA_OK
    torch.cuda.synchronize()
