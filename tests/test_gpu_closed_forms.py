"""GPU results against closed forms of the definition, computed here in
numpy rather than by the oracle: one cached token gives V_0; equal keys, or
scale 0, give the mean of the visible values; every output lies in the
convex hull of its values.  Both pool layouts, both kv encodings."""
import numpy as np
import pytest
import torch

from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import (PV_ROUND, abs_value_host, bf16_to_f64, bf16_ulp, check_close, device,
                      extend_extra, run_gpu, uses_pv)

pytestmark = pytest.mark.gpu

LAYOUTS = ["hnd", "nhd"]
KVS = ["bf16", "fp8_e4m3"]
# (Hq, Hkv, create flags): four heads per kv head on either value pass, and
# sixteen (the matrix-core value pass only)
HEADS = {"g4": (32, 8, 0), "g4valu": (32, 8, B.RL_DA_PV_ON_VALU), "g16": (64, 4, 0)}


def problem(lengths, kv, layout, seed, hq=32, hkv=8, pool_factor=1.25):
    return workloads.make_problem("closed", batch=len(lengths), num_q_heads=hq,
                                  num_kv_heads=hkv, lengths=list(lengths), kv_dtype=kv,
                                  seed=seed, layout=layout,
                                  pool_factor=pool_factor).to(device())


_decoded = {}


def decoded_values(p):
    """V as float64 [P, Hkv, 16, D] whatever the layout (cached per pool)."""
    key = (p.v_pool.data_ptr(), p.v_pool._version,
           None if p.v_scale is None else p.v_scale._version)
    if key not in _decoded:
        _decoded.clear()
        _decoded[key] = _decode(p)
    return _decoded[key]


def _decode(p):
    if p.kv_dtype == "bf16":
        v = p.v_pool.float().double()
    else:
        v = p.v_pool.view(torch.float8_e4m3fn).double()
    if p.layout == "nhd":
        v = v.transpose(1, 2)
    if p.kv_dtype != "bf16":
        v = v * p.v_scale.double()[:, :, None, None]
    return v.cpu().numpy()


def visible_values(p, b, kvh, upto=None):
    """[L, D] values of sequence b, kv head kvh, tokens 0..upto-1."""
    v = decoded_values(p)
    L = int(p.seq_lens[b]) if upto is None else upto
    bt = p.block_table[b].cpu().numpy()
    t = np.arange(L)
    return v[bt[t // 16], kvh, t % 16, :]


@pytest.mark.parametrize("heads", list(HEADS))
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("kv", KVS)
def test_one_token_returns_its_value(kv, layout, heads):
    hq, hkv, flags = HEADS[heads]
    p = problem([1] * 16, kv, layout, seed=61, hq=hq, hkv=hkv)
    got = bf16_to_f64(run_gpu(p, flags=flags))
    G = p.num_q_heads // p.num_kv_heads
    for b in range(p.batch):
        for h in range(p.num_q_heads):
            want = visible_values(p, b, h // G)[0]
            if kv == "bf16":
                assert np.array_equal(got[b, h], want), (b, h)   # weight exactly 1
            else:
                assert np.all(np.abs(got[b, h] - want) <= bf16_ulp(want)), (b, h)


@pytest.mark.parametrize("heads", list(HEADS))
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("kv", KVS)
@pytest.mark.parametrize("how", ["equal_keys", "zero_scale"])
def test_uniform_weights_give_the_mean(kv, layout, how, heads):
    hq, hkv, flags = HEADS[heads]
    lengths = [1, 16, 17, 300, 4096, 5000, 9000]
    p = problem(lengths, kv, layout, seed=62, hq=hq, hkv=hkv)
    if how == "equal_keys":
        # every key of every page the same row: all scores equal
        row = p.k_pool.reshape(-1, p.head_dim)[0].clone()
        p.k_pool.reshape(-1, p.head_dim)[:] = row
        if kv != "bf16":
            p.k_scale.fill_(1.0)
    else:
        p.scale = 0.0
    for split in (0, 1024):
        got = bf16_to_f64(run_gpu(p, split_tokens=split, flags=flags))
        G = p.num_q_heads // p.num_kv_heads
        want = np.stack([[visible_values(p, b, h // G).mean(axis=0)
                          for h in range(p.num_q_heads)] for b in range(p.batch)])
        extra = 0.0
        if uses_pv(p, flags):   # equal weights: M1 is the mean magnitude
            extra = PV_ROUND * np.stack([[np.abs(visible_values(p, b, h // G)).mean(axis=0)
                                          for h in range(p.num_q_heads)]
                                         for b in range(p.batch)])
        print(check_close(got, want, "%s %s %s split %d" % (how, kv, layout, split),
                          extra_abs=extra))


@pytest.mark.parametrize("heads", list(HEADS))
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("kv", KVS)
def test_outputs_lie_in_the_convex_hull_of_the_values(kv, layout, heads):
    hq, hkv, flags = HEADS[heads]
    lengths = [3, 100, 700, 2049]
    p = problem(lengths, kv, layout, seed=63, hq=hq, hkv=hkv)
    p.q.mul_(8.0)                        # peaked softmax: outputs near single values
    got = bf16_to_f64(run_gpu(p, flags=flags))
    G = p.num_q_heads // p.num_kv_heads
    for b in range(p.batch):
        for h in range(p.num_q_heads):
            v = visible_values(p, b, h // G)
            lo, hi = v.min(axis=0), v.max(axis=0)
            slack = bf16_ulp(np.maximum(np.abs(lo), np.abs(hi)))
            assert np.all(got[b, h] >= lo - slack) and np.all(got[b, h] <= hi + slack), (b, h)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_extend_with_zero_scale_gives_causal_prefix_means(layout):
    new, prior = [5, 40, 1], [11, 70, 0]
    lengths = [a + b for a, b in zip(new, prior)]
    p = problem(lengths, "bf16", layout, seed=64, hq=8, hkv=2)
    T = sum(new)
    gen = torch.Generator().manual_seed(65)
    q = torch.randn((T, 8, 128), generator=gen).to(torch.bfloat16).to(device())
    q_start = torch.tensor(np.concatenate([[0], np.cumsum(new)]), dtype=torch.int32,
                           device=device())
    p.scale = 0.0
    out = torch.full_like(q, float("nan"))
    B.extend_attention(p, q, q_start, max(new), out)
    torch.cuda.synchronize()
    got = bf16_to_f64(out)
    want = np.zeros_like(got)
    m1 = np.zeros_like(got)
    for b in range(len(new)):
        for i in range(new[b]):
            row = int(q_start[b]) + i
            for h in range(8):
                vis = visible_values(p, b, h // 4, upto=prior[b] + i + 1)
                want[row, h] = vis.mean(axis=0)
                m1[row, h] = np.abs(vis).mean(axis=0)
    # equal weights: the rounded-probability allowance with M1 = mean |v|
    print(check_close(got, want, "extend zero scale " + layout,
                      extra_abs=extend_extra("bf16", want, m1)))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_negative_and_zero_scales_match_the_oracle(layout):
    """The softmax scale is any finite number: a negative one turns the
    largest dot products into the smallest weights."""
    import oracle
    from gpu_util import decode_extra, oracle_ref
    for scale in (-0.09, 0.0):
        p = problem([1, 17, 300, 4100], "bf16", layout, seed=66)
        p.scale = scale
        print(check_close(bf16_to_f64(run_gpu(p)), oracle_ref(p), "decode scale %g" % scale,
                          extra_abs=decode_extra(p, 0)))
        new, prior = [3, 70], [14, 200]
        pe = problem([a + b for a, b in zip(new, prior)], "bf16", layout, seed=67, hq=8, hkv=2)
        pe.scale = scale
        gen = torch.Generator().manual_seed(68)
        q = torch.randn((sum(new), 8, 128), generator=gen).to(torch.bfloat16).to(device())
        q_start = torch.tensor(np.concatenate([[0], np.cumsum(new)]), dtype=torch.int32,
                               device=device())
        out = torch.full_like(q, float("nan"))
        B.extend_attention(pe, q, q_start, max(new), out)
        torch.cuda.synchronize()
        h = pe.host_arrays()
        refs = [oracle.extend_attention(q.cpu().view(torch.int16).numpy().view(np.uint16),
                                        q_start.cpu().numpy(), h["k_pool"], v,
                                        h["block_table"], h["seq_lens"], num_kv_heads=2,
                                        scale=scale, layout=layout)
                for v in (h["v_pool"], abs_value_host(pe, h))]
        print(check_close(bf16_to_f64(out), refs[0], "extend scale %g" % scale,
                          extra_abs=extend_extra("bf16", refs[0], refs[1])))
