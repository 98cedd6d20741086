"""Pins for the oracle's KV-cache append and its e4m3 encoder (CPU only).

The encoder is checked against torch's float8_e4m3fn conversion (a library
routine) on every e4m3 value, every midpoint between neighbours (ties go to
the even code) and random values; the append against direct consequences of
its definition: bf16 tokens land bit-exactly in their slot and nowhere else,
an fp8 token on an empty page is quantised exactly like a one-token slab by
the workload generator (which uses torch's cast), a token inside the current
range leaves the scale and the earlier codes alone, and a growing token
raises the scale to its own absmax/448 with the earlier values preserved to
within one e4m3 rounding.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22492_amd import workloads


def torch_e4m3(x):
    return torch.tensor(np.asarray(x, dtype=np.float32)).to(
        torch.float8_e4m3fn).view(torch.uint8).numpy()


def e4m3_values():
    codes = np.arange(256, dtype=np.uint8)
    vals = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    return codes, vals


def test_encoder_round_trips_every_code():
    for c, v in zip(*e4m3_values()):
        if math.isnan(v):
            assert oracle.e4m3_encode(float("nan")) == 0x7F
            continue
        assert oracle.e4m3_encode(v) == c, (hex(c), v)


def test_encoder_ties_and_random_values_match_torch():
    _, vals = e4m3_values()
    pos = np.unique(vals[(vals >= 0) & np.isfinite(vals)])
    mids = (pos[:-1] + pos[1:]) / 2                      # exact midpoints (fp32-representable)
    rng = np.random.default_rng(0)
    rand = np.concatenate([rng.uniform(-448, 448, 3000), rng.normal(0, 1e-2, 2000),
                           rng.uniform(-2 ** -6, 2 ** -6, 2000)])
    xs = np.concatenate([mids, -mids, rand]).astype(np.float32)
    want = torch_e4m3(xs)
    got = np.array([oracle.e4m3_encode(float(x)) for x in xs], dtype=np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(float(xs[i]), hex(got[i]), hex(want[i])) for i in bad[:5]]


def _append_problem(seed, kv, lengths, hkv=2, d=16, page=4, layout="hnd"):
    """Pools laid out for lengths + 1 (the engine has already given every
    sequence the page its new token goes to); seq_lens = lengths."""
    p = workloads.make_problem("app", batch=len(lengths), num_q_heads=hkv, num_kv_heads=hkv,
                               head_dim=d, page_size=page,
                               lengths=[L + 1 for L in lengths], kv_dtype=kv, seed=seed,
                               pool_factor=2.0, layout=layout)
    h = p.host_arrays()
    h["seq_lens"] = (h["seq_lens"] - 1).astype(np.int32)
    gen = torch.Generator().manual_seed(seed + 1)
    kn = torch.randn((len(lengths), hkv, d), generator=gen).to(torch.bfloat16)
    vn = torch.randn((len(lengths), hkv, d), generator=gen).to(torch.bfloat16)
    bits = lambda t: t.view(torch.int16).numpy().view(np.uint16)
    return p, h, bits(kn), bits(vn)


def _run(h, kn, vn, kv):
    code = oracle.KV_BF16 if kv == "bf16" else oracle.KV_FP8_E4M3
    return oracle.kv_append(kn, vn, h["k_pool"], h["v_pool"], h["block_table"],
                            h["seq_lens"], kv_dtype=code, k_scale=h.get("k_scale"),
                            v_scale=h.get("v_scale"), layout=h["layout"])


def test_bf16_append_writes_exactly_one_slot_per_head():
    lengths = [0, 3, 4, 9, 15]
    p, h, kn, vn = _append_problem(1, "bf16", lengths)
    k2, v2, _, _ = _run(h, kn, vn, "bf16")
    kd, vd = h["k_pool"].copy(), h["v_pool"].copy()
    for b, L in enumerate(lengths):
        page, slot = h["block_table"][b, L // 4], L % 4
        assert np.array_equal(k2[page, :, slot, :], kn[b])
        assert np.array_equal(v2[page, :, slot, :], vn[b])
        kd[page, :, slot, :] = kn[b]
        vd[page, :, slot, :] = vn[b]
    assert np.array_equal(k2, kd) and np.array_equal(v2, vd)   # nothing else touched


def test_bf16_append_to_token_major_pools_writes_one_row_per_head():
    lengths = [0, 3, 4, 9, 15]
    p, h, kn, vn = _append_problem(1, "bf16", lengths, layout="nhd")
    k2, v2, _, _ = _run(h, kn, vn, "bf16")
    kd, vd = h["k_pool"].copy(), h["v_pool"].copy()
    for b, L in enumerate(lengths):
        page, slot = h["block_table"][b, L // 4], L % 4
        kd[page, slot, :, :] = kn[b]
        vd[page, slot, :, :] = vn[b]
    assert np.array_equal(k2, kd) and np.array_equal(v2, vd)


@pytest.mark.parametrize("grow", [1.0, 50.0])
def test_fp8_append_is_the_same_in_both_layouts(grow):
    """Same tokens into the same values stored in either order: the appended
    pools are each other's transposes and the scales are equal."""
    lengths = [0, 5, 6, 11]
    res = {}
    for layout in ("hnd", "nhd"):
        p, h, kn, vn = _append_problem(9, "fp8_e4m3", lengths, layout=layout)
        big = torch.from_numpy(kn.view(np.int16).copy()).view(torch.bfloat16).float() * grow
        kn = big.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        res[layout] = _run(h, kn, vn, "fp8_e4m3")
    for a, b in zip(res["hnd"][:2], res["nhd"][:2]):
        assert np.array_equal(a.transpose(0, 2, 1, 3), b)
    for a, b in zip(res["hnd"][2:], res["nhd"][2:]):
        assert np.array_equal(a, b)
    assert not np.array_equal(res["hnd"][2], _append_problem(9, "fp8_e4m3", lengths)[1]["k_scale"])


def test_fp8_append_on_an_empty_page_matches_one_token_slab_quantisation():
    lengths = [0, 4, 8]                      # every append starts a new page
    p, h, kn, vn = _append_problem(2, "fp8_e4m3", lengths)
    k2, v2, ks2, vs2 = _run(h, kn, vn, "fp8_e4m3")
    for b, L in enumerate(lengths):
        page = h["block_table"][b, L // 4]
        for kvh in range(2):
            for new, pool, sc in ((kn, k2, ks2), (vn, v2, vs2)):
                x = torch.from_numpy(new[b, kvh].view(np.int16).copy()).view(
                    torch.bfloat16).float()[None, :]
                codes, scale = workloads.quantize_e4m3_slabs(x)
                assert sc[page, kvh] == scale.item()
                assert np.array_equal(pool[page, kvh, 0, :], codes.numpy()[0])


def test_fp8_append_inside_the_range_keeps_scale_and_codes():
    lengths = [5, 6]
    p, h, kn, vn = _append_problem(3, "fp8_e4m3", lengths)
    # shrink the new tokens so they fit the page's current range
    small = (torch.from_numpy(kn.view(np.int16).copy()).view(torch.bfloat16).float() * 1e-3)
    kn = small.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    vn = kn.copy()
    k2, v2, ks2, vs2 = _run(h, kn, vn, "fp8_e4m3")
    for b, L in enumerate(lengths):
        page, slot = h["block_table"][b, L // 4], L % 4
        assert np.array_equal(ks2[page], h["k_scale"][page])
        assert np.array_equal(k2[page, :, :slot, :], h["k_pool"][page, :, :slot, :])
        for kvh in range(2):
            x = torch.from_numpy(kn[b, kvh].view(np.int16).copy()).view(torch.bfloat16).float()
            want = torch_e4m3(np.clip((x / float(ks2[page, kvh])).numpy(), -448, 448))
            assert np.array_equal(k2[page, kvh, slot, :], want)


def test_fp8_append_that_grows_the_scale_reencodes_earlier_slots():
    lengths = [5, 7]
    p, h, kn, vn = _append_problem(4, "fp8_e4m3", lengths)
    big = torch.from_numpy(kn.view(np.int16).copy()).view(torch.bfloat16).float() * 50.0
    kn = big.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    k2, _, ks2, _ = _run(h, kn, vn, "fp8_e4m3")
    dec = lambda c: torch.from_numpy(c.copy()).view(torch.float8_e4m3fn).double().numpy()
    for b, L in enumerate(lengths):
        page, slot = h["block_table"][b, L // 4], L % 4
        for kvh in range(2):
            x = torch.from_numpy(kn[b, kvh].view(np.int16).copy()).view(torch.bfloat16).float()
            s_new = float(ks2[page, kvh])
            assert s_new == np.float32(x.abs().max().item()) / np.float32(448.0)
            assert s_new > h["k_scale"][page, kvh]
            old = dec(h["k_pool"][page, kvh, :slot]) * float(h["k_scale"][page, kvh])
            new = dec(k2[page, kvh, :slot]) * s_new
            # one e4m3 rounding at the new scale: half a step of 2^-3 relative,
            # or half the subnormal step
            tol = np.maximum(np.abs(old) * 2.0 ** -4, 2.0 ** -10 * s_new) * 1.0001
            assert np.all(np.abs(new - old) <= tol)
            assert np.max(np.abs(dec(k2[page, kvh]))) <= 448.0


def test_filling_a_page_ends_with_the_one_shot_scale():
    """Appending 16 tokens one by one leaves the page's scale equal to the
    absmax/448 of all of them, as one-shot quantisation of the slab would."""
    rng = torch.Generator().manual_seed(5)
    tokens = torch.randn((16, 1, 32), generator=rng).to(torch.bfloat16)
    P = 2
    k_pool = np.zeros((P, 1, 16, 32), dtype=np.uint8)
    v_pool = np.zeros_like(k_pool)
    ks = np.ones((P, 1), dtype=np.float32)
    vs = np.ones((P, 1), dtype=np.float32)
    bt = np.array([[1]], dtype=np.int32)
    for t in range(16):
        bits = tokens[t:t + 1].view(torch.int16).numpy().view(np.uint16)
        k_pool, v_pool, ks, vs = oracle.kv_append(
            bits, bits, k_pool, v_pool, bt, np.array([t], dtype=np.int32),
            kv_dtype=oracle.KV_FP8_E4M3, k_scale=ks, v_scale=vs)
    _, scale = workloads.quantize_e4m3_slabs(tokens.float().reshape(1, -1))
    assert ks[1, 0] == scale.item() and vs[1, 0] == scale.item()
    assert ks[0, 0] == 1.0                     # the other page is untouched


def test_append_preconditions():
    p, h, kn, vn = _append_problem(6, "bf16", [3, 4])
    bad = h["block_table"].copy()
    bad[1, 1] = h["k_pool"].shape[0]
    with pytest.raises(oracle.OracleError):
        oracle.kv_append(kn, vn, h["k_pool"], h["v_pool"], bad, h["seq_lens"])
    full = h["seq_lens"].copy()
    full[0] = h["block_table"].shape[1] * 4
    with pytest.raises(oracle.OracleError):
        oracle.kv_append(kn, vn, h["k_pool"], h["v_pool"], h["block_table"], full)
