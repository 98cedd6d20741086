"""bench.py's oracle legs on the host (CPU): with the oracle's own result in
place of the device output they report exact agreement, and a planted
one-byte change is found.  Small problems, short timing loops."""
import importlib.util
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import weight_sync as ows
from paper_2512_22492_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_legs", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def tiny(kv, **kw):
    cfg = dict(workloads.CONFIGS["tiny"])
    seed = cfg.pop("seed")
    cfg.update(kv_dtype=kv, **kw)
    return workloads.make_problem("tiny", seed=seed, device="cpu", layout="hnd", **cfg)


def bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_extend_leg(bench, kv):
    n, prior = 24, np.array([100, 37, 250, 16])
    p = tiny(kv, lengths=[int(x) + n for x in prior])
    q = torch.randn((len(prior) * n, p.num_q_heads, p.head_dim),
                    generator=torch.Generator().manual_seed(5)).to(torch.bfloat16)
    h = p.host_arrays()
    ref = oracle.extend_attention(
        bits(q), np.arange(0, q.shape[0] + 1, n, dtype=np.int32), h["k_pool"], h["v_pool"],
        h["block_table"], h["seq_lens"], num_kv_heads=p.num_kv_heads, scale=p.scale,
        kv_dtype=oracle.KV_BF16 if kv == "bf16" else oracle.KV_FP8_E4M3,
        k_scale=h.get("k_scale"), v_scale=h.get("v_scale"))
    out = torch.from_numpy(ref).float().to(torch.bfloat16)
    base, par = bench.extend_cpu_baseline(p, q, n, prior, out, min_seconds=0.01)
    assert base["kind"] == "oracle" and base["unit"] == "TFLOP/s" and base["value"] > 0
    assert par["official_bound_holds"] and par["max_ulp"] <= 0.5
    assert par["max_err_over_weight_bound"] < 1
    out[0, 0, 0] = out[0, 0, 0] + 1.0
    _, bad = bench.extend_cpu_baseline(p, q, n, prior, out, min_seconds=0.01)
    assert not bad["official_bound_holds"] and bad["max_err_over_weight_bound"] > 1


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_append_leg(bench, kv):
    p = tiny(kv)
    shape = (p.batch, p.num_kv_heads, p.head_dim)
    g = torch.Generator().manual_seed(1)
    k = torch.randn(shape, generator=g).to(torch.bfloat16)
    v = torch.randn(shape, generator=g).to(torch.bfloat16)
    before = {a: np.array(b, copy=True) if isinstance(b, np.ndarray) else b
              for a, b in p.host_arrays().items()}
    res = oracle.kv_append(bits(k), bits(v), before["k_pool"], before["v_pool"],
                           before["block_table"], before["seq_lens"],
                           kv_dtype=oracle.KV_BF16 if kv == "bf16" else oracle.KV_FP8_E4M3,
                           k_scale=before.get("k_scale"), v_scale=before.get("v_scale"))
    dst = [p.k_pool, p.v_pool] + ([p.k_scale, p.v_scale] if kv != "bf16" else [])
    for t, r in zip(dst, res):    # the device's result, as the oracle gives it
        t.view(torch.uint8).reshape(-1).copy_(
            torch.from_numpy(np.ascontiguousarray(r).view(np.uint8).reshape(-1)))
    base, par = bench.append_cpu_baseline(p, before, k, v, min_seconds=0.01)
    assert base["unit"] == "us" and par["bit_exact"] and par["bytes_compared"] > 0
    p.v_pool.view(torch.uint8).reshape(-1)[7] ^= 1
    _, bad = bench.append_cpu_baseline(p, before, k, v, min_seconds=0.01)
    assert bad["mismatched_bytes"] == 1 and not bad["bit_exact"]


def test_weight_sync_leg(bench):
    g = torch.Generator().manual_seed(3)
    tensors = [torch.randint(-30000, 30000, (n,), generator=g, dtype=torch.int16)
               .view(torch.bfloat16) for n in (1000, 70000, 33, 400000, 5)]
    cap = 1 << 18
    pieces = ows.plan([t.numel() * 2 for t in tensors], cap, 256)
    host = [t.view(torch.uint8).numpy() for t in tensors]
    for chunk in range(ows.num_chunks(pieces)):
        buf, written = ows.pack(host, pieces, chunk, cap, fill=7)
        base, par = bench.weight_sync_cpu_baseline(tensors, buf, chunk, cap, 256,
                                                   min_seconds=0.01)
        assert par == {"bytes_compared": int(written.sum()), "mismatched_bytes": 0,
                       "bit_exact": True}
        buf[np.flatnonzero(written)[3]] ^= 0x80
        _, bad = bench.weight_sync_cpu_baseline(tensors, buf, chunk, cap, 256, min_seconds=0.01)
        assert bad["mismatched_bytes"] == 1
