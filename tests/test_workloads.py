"""Seeded workload generators (CPU only): reproducibility, length
distributions, page placement and the e4m3 storage encoding."""
import math

import numpy as np
import pytest
import torch

from paper_2512_22492_amd import workloads


def test_same_seed_same_problem():
    a = workloads.make_config("tiny")
    b = workloads.make_config("tiny")
    for name in ("q", "k_pool", "v_pool", "block_table", "seq_lens"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    c = workloads.make_config("tiny", seed=1)
    assert not torch.equal(a.q, c.q)


def test_tiny_config_shapes():
    p = workloads.make_config("tiny")
    assert p.q.shape == (4, 8, 128) and p.q.dtype == torch.bfloat16
    assert p.k_pool.shape == (200, 2, 16, 128)
    L = p.lengths()
    assert np.all((L >= 1) & (L <= 512))
    assert p.scale == 1.0 / math.sqrt(128)


@pytest.mark.parametrize("spec,lo,hi", [
    (("uniform", 1, 512), 1, 512),
    (("uniform", 32768, 65536), 32768, 65536),
    (("lognormal", 4096, 0.8, 256, 32768), 256, 32768),
])
def test_length_bounds(spec, lo, hi):
    rng = np.random.default_rng(0)
    L = workloads.draw_lengths(rng, 20000, spec)
    assert L.min() >= lo and L.max() <= hi
    if spec[0] == "lognormal":
        assert abs(np.median(L) - 4096) < 150
        assert np.mean(L == hi) < 0.01


def test_uniform_lengths_reach_both_ends():
    rng = np.random.default_rng(1)
    L = workloads.draw_lengths(rng, 5000, ("uniform", 1, 8))
    assert set(np.unique(L)) == set(range(1, 9))


def test_pages_form_a_permutation_slice():
    rng = np.random.default_rng(2)
    L = np.array([1, 16, 17, 100, 0, 33])
    table, P, pad = workloads.place_pages(rng, L, 16, None, 1.25)
    used = (L + 15) // 16
    assert P == math.ceil(1.25 * used.sum())
    pages = np.concatenate([table[b, :n] for b, n in enumerate(used)])
    assert len(set(pages.tolist())) == used.sum()
    assert pages.min() >= 0 and pages.max() < P
    assert pad not in set(pages.tolist())
    for b, n in enumerate(used):
        assert np.all(table[b, n:] == pad)


def _e4m3_values():
    vals = []
    for c in range(256):
        s, e, m = c >> 7, (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            continue
        mag = (m / 8.0) * 2.0 ** -6 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7)
        vals.append((-mag if s else mag, c))
    return vals


def _encode_nearest_even(x):
    """Brute-force round-to-nearest-even onto the finite e4m3 grid."""
    table = _e4m3_values()
    positive = {val: c for val, c in table if c < 0x80}     # magnitude -> code
    mags = sorted(positive)
    out = np.empty(x.shape, dtype=np.uint8)
    for i, v in enumerate(x.ravel()):
        a = abs(float(v))
        best = min(mags, key=lambda m: (abs(m - a), 0))
        ties = [m for m in mags if abs(m - a) == abs(best - a)]
        if len(ties) > 1:            # pick the even mantissa (code LSB 0)
            best = [m for m in ties if positive[m] % 2 == 0][0]
        code = positive[best]
        if v < 0 or (v == 0 and math.copysign(1, v) < 0):
            code |= 0x80
        out.ravel()[i] = code
    return out


def test_e4m3_quantisation_is_nearest_even_with_slab_scale():
    gen = torch.Generator().manual_seed(3)
    x = torch.randn((6, 64), generator=gen)
    x[0, :8] = torch.tensor([0.0, 448.0, -448.0, 1.0625, 1.1875, 3.0, -0.5, 1e-9])
    codes, scale = workloads.quantize_e4m3_slabs(x)
    absmax = x.abs().amax(dim=1)
    assert torch.equal(scale, absmax / 448.0)
    y = (x / scale[:, None]).clamp(-448, 448).numpy()
    assert np.array_equal(codes.numpy(), _encode_nearest_even(y))
    # each slab's largest magnitude lands exactly on +-448
    dec = codes.view(torch.float8_e4m3fn).to(torch.float32).abs().amax(dim=1)
    assert torch.all(dec == 448.0)


def test_e4m3_ties_round_to_even():
    # 1.0625 lies halfway between 1.0 (code 0x38) and 1.125 (0x39): even is 0x38;
    # 1.1875 lies halfway between 1.125 (0x39) and 1.25 (0x3A): even is 0x3A.
    x = torch.tensor([[1.0625, 1.1875, -1.0625, 448.0]])
    codes, scale = workloads.quantize_e4m3_slabs(x)
    assert scale.item() == 1.0
    assert codes.tolist() == [[0x38, 0x3A, 0xB8, 0x7E]]


def test_kv_bytes_of_qwen3_8b_step():
    cfg = workloads.CONFIGS["qwen3_8b_step"]
    # 64 sequences x 4096 tokens x 8 kv heads x 128 dims x (K and V) x 2 bytes
    expected = 64 * 4096 * 8 * 128 * 2 * 2
    p = workloads.make_problem("c2-shape", device="cpu", **{
        k: v for k, v in cfg.items() if k not in ("seed",)
    } | dict(batch=2, seed=0))
    assert p.kv_bytes() == 2 * 4096 * 8 * 128 * 2 * 2
    assert expected == 1073741824


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_hnd_kv_layout_views_one_allocation(kv):
    """'hnd_kv' problems hold the head-major values in one [P, Hkv, 2, 16, D]
    allocation, value slab right after key slab, through copies and moves."""
    kw = dict(batch=3, num_q_heads=8, num_kv_heads=2, lengths=[5, 40, 17], kv_dtype=kv, seed=3)
    h = workloads.make_problem("x", layout="hnd", **kw)
    p = workloads.make_problem("x", layout="hnd_kv", **kw)
    for q in (p, p.to("cpu"), p.clone_pools()):
        assert q.kv_pool.shape == (q.num_pages, 2, 2, 16, 128) and q.kv_pool.is_contiguous()
        slab = 16 * 128 * q.k_pool.element_size()
        assert q.k_pool.data_ptr() == q.kv_pool.data_ptr()
        assert q.v_pool.data_ptr() == q.k_pool.data_ptr() + slab
        assert torch.equal(q.k_pool, h.k_pool) and torch.equal(q.v_pool, h.v_pool)
        arrays = q.host_arrays()
        assert arrays["layout"] == "hnd" and arrays["k_pool"].shape == (q.num_pages, 2, 16, 128)
    c = p.clone_pools()
    assert c.kv_pool.data_ptr() != p.kv_pool.data_ptr()
