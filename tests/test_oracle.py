"""Pins for the fp64 oracle (CPU only).

The paper prints no attention values, so the oracle is pinned to mathematics:
a dense brute force written independently in numpy, torch's float64
scaled-dot-product attention (a library routine), closed forms (one token,
equal keys, scale 0, hand-worked weights), invariants (page permutation,
poisoned unread memory, convex hull) and block-table probes.  Each pin is
chosen so that a plausible slip in the oracle -- a dropped scale, a flipped
sign, a wrong head or slot index, a missing max subtraction, a transposed
operand, an off-by-one in the length mask -- fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22492_amd import workloads


# ---------------------------------------------------------------- helpers ---

def bf16_bits_to_f64(bits):
    """bf16 bit patterns -> float64 (bf16 is the top half of binary32)."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x):
    """Exact conversion for values representable in bf16 (test inputs only)."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not representable in bf16"
    return (u >> 16).astype(np.uint16)


def decode_pool(arr, kv_dtype, scales, layout="hnd"):
    if kv_dtype == oracle.KV_BF16:
        return bf16_bits_to_f64(arr)
    vals = torch.from_numpy(arr.copy()).view(torch.float8_e4m3fn).to(
        torch.float64).numpy()
    sc = scales.astype(np.float64)
    # scales are [page][kv head]; the kv-head axis is 1 (hnd) or 2 (nhd)
    return vals * (sc[:, :, None, None] if layout == "hnd" else sc[:, None, :, None])


def dense_bruteforce(h, kv_dtype=oracle.KV_BF16, layout="hnd"):
    """Independent dense reference: gather with fancy indexing, repeat heads,
    einsum, max-subtracted softmax."""
    q = bf16_bits_to_f64(h["q_bits"])
    K = decode_pool(h["k_pool"], kv_dtype, h.get("k_scale"), layout)
    V = decode_pool(h["v_pool"], kv_dtype, h.get("v_scale"), layout)
    bt, lens = h["block_table"], h["seq_lens"]
    B, Hq, D = q.shape
    if layout == "hnd":
        Hkv, page = K.shape[1], K.shape[2]
    else:
        page, Hkv = K.shape[1], K.shape[2]
    G = Hq // Hkv
    out = np.zeros((B, Hq, D))
    for b in range(B):
        L = int(lens[b])
        if L <= 0:
            continue
        t = np.arange(L)
        pages = bt[b, t // page]
        if layout == "hnd":
            Kb = K[pages, :, t % page, :]        # [L, Hkv, D]
            Vb = V[pages, :, t % page, :]
        else:
            Kb = K[pages, t % page, :, :]
            Vb = V[pages, t % page, :, :]
        Kh = np.repeat(Kb, G, axis=1)            # [L, Hq, D]
        Vh = np.repeat(Vb, G, axis=1)
        s = np.einsum("hd,thd->ht", q[b], Kh) * h["scale"]
        s = s - s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w = w / w.sum(axis=1, keepdims=True)
        out[b] = np.einsum("ht,thd->hd", w, Vh)
    return out


def run_oracle(h, kv_dtype=oracle.KV_BF16, rows=None):
    kw = dict(num_kv_heads=h["num_kv_heads"], scale=h["scale"],
              kv_dtype=kv_dtype, rows=rows, layout=h.get("layout", "hnd"))
    if kv_dtype == oracle.KV_FP8_E4M3:
        kw.update(k_scale=h["k_scale"], v_scale=h["v_scale"])
    return oracle.decode_attention(h["q_bits"], h["k_pool"], h["v_pool"],
                                   h["block_table"], h["seq_lens"], **kw)


def small_problem(seed, *, batch=3, hq=4, hkv=2, d=16, page=4,
                  lengths=("uniform", 1, 23), kv="bf16", pool_factor=1.5,
                  scale=None):
    return workloads.make_problem(
        "small", batch=batch, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
        page_size=page, lengths=lengths, kv_dtype=kv, seed=seed,
        pool_factor=pool_factor, scale=scale)


KV = {"bf16": oracle.KV_BF16, "fp8_e4m3": oracle.KV_FP8_E4M3}


# ------------------------------------------------------ brute-force pins ---

SHAPES = [
    # (batch, hq, hkv, d, page, lengths)
    (3, 4, 2, 16, 4, ("uniform", 1, 23)),
    (2, 8, 1, 8, 16, ("explicit", [1, 40])),
    (4, 8, 8, 5, 3, ("uniform", 0, 10)),
    (2, 32, 8, 128, 16, ("explicit", [17, 64])),
    (5, 6, 3, 12, 5, ("explicit", [4, 5, 6, 0, 11])),
]


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("seed", [1, 2])
def test_matches_dense_bruteforce(shape, seed, kv):
    batch, hq, hkv, d, page, lengths = shape
    lens = lengths if lengths[0] != "explicit" else list(lengths[1])
    p = workloads.make_problem("bf", batch=batch, num_q_heads=hq,
                               num_kv_heads=hkv, head_dim=d, page_size=page,
                               lengths=lens, kv_dtype=kv, seed=seed)
    h = p.host_arrays()
    got = run_oracle(h, KV[kv])
    want = dense_bruteforce(h, KV[kv])
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("shape", SHAPES)
def test_token_major_pools_match_dense_bruteforce(shape, kv):
    """[page][slot][kv head][dim] pools: the brute force indexes them directly."""
    batch, hq, hkv, d, page, lengths = shape
    lens = lengths if lengths[0] != "explicit" else list(lengths[1])
    p = workloads.make_problem("nhd", batch=batch, num_q_heads=hq, num_kv_heads=hkv,
                               head_dim=d, page_size=page, lengths=lens, kv_dtype=kv,
                               seed=7, layout="nhd")
    h = p.host_arrays()
    assert h["k_pool"].shape[1:] == (page, hkv, d)
    got = run_oracle(h, KV[kv])
    want = dense_bruteforce(h, KV[kv], layout="nhd")
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_layouts_store_the_same_values_and_give_the_same_result(kv):
    """The two layouts of one seeded problem hold the same values, and the
    oracle reads them in the same order, so the results are bit-identical."""
    kw = dict(batch=4, num_q_heads=8, num_kv_heads=4, head_dim=16, page_size=4,
              lengths=[0, 1, 9, 30], kv_dtype=kv, seed=8)
    a = workloads.make_problem("hnd", **kw).host_arrays()
    b = workloads.make_problem("nhd", layout="nhd", **kw).host_arrays()
    assert np.array_equal(a["k_pool"].transpose(0, 2, 1, 3), b["k_pool"])
    assert np.array_equal(a["v_pool"].transpose(0, 2, 1, 3), b["v_pool"])
    assert np.array_equal(run_oracle(a, KV[kv]), run_oracle(b, KV[kv]))


@pytest.mark.parametrize("seed", [3, 4])
def test_matches_torch_sdpa_float64(seed):
    p = small_problem(seed, batch=4, hq=8, hkv=2, d=32, page=16,
                      lengths=("uniform", 1, 70))
    h = p.host_arrays()
    got = run_oracle(h)
    q = torch.from_numpy(bf16_bits_to_f64(h["q_bits"]))
    K = torch.from_numpy(bf16_bits_to_f64(h["k_pool"]))
    V = torch.from_numpy(bf16_bits_to_f64(h["v_pool"]))
    G = 8 // 2
    for b in range(4):
        L = int(h["seq_lens"][b])
        t = np.arange(L)
        pages = torch.from_numpy(h["block_table"][b, t // 16].astype(np.int64))
        slots = torch.from_numpy(t % 16)
        Kb = K[pages, :, slots, :].permute(1, 0, 2).repeat_interleave(G, 0)
        Vb = V[pages, :, slots, :].permute(1, 0, 2).repeat_interleave(G, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(
            q[b][:, None, :], Kb, Vb, scale=h["scale"])[:, 0, :]
        np.testing.assert_allclose(got[b], ref.numpy(), rtol=1e-12, atol=1e-14)


# -------------------------------------------------------- closed forms ---

@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_length_one_returns_first_value_exactly(kv):
    p = small_problem(5, batch=3, lengths=("explicit", [1, 1, 1]), kv=kv)
    h = p.host_arrays()
    got = run_oracle(h, KV[kv])
    V = decode_pool(h["v_pool"], KV[kv], h.get("v_scale"))
    G = 2
    for b in range(3):
        page = h["block_table"][b, 0]
        for hh in range(4):
            assert np.array_equal(got[b, hh], V[page, hh // G, 0, :])


def _equal_keys_problem(seed, scale=None):
    p = small_problem(seed, batch=3, lengths=("explicit", [1, 9, 22]),
                      scale=scale)
    h = p.host_arrays()
    k = h["k_pool"]
    k[...] = k[0, 0, 0, :]          # every key in the pool identical
    return h


def _mean_of_values(h):
    V = bf16_bits_to_f64(h["v_pool"])
    B, Hq, D = h["q_bits"].shape
    G = Hq // h["num_kv_heads"]
    out = np.zeros((B, Hq, D))
    for b in range(B):
        L = int(h["seq_lens"][b])
        t = np.arange(L)
        vals = V[h["block_table"][b, t // 4], :, t % 4, :]   # [L, Hkv, D]
        out[b] = np.repeat(vals.mean(axis=0), G, axis=0)
    return out


def test_equal_keys_give_mean_of_values():
    h = _equal_keys_problem(6)
    np.testing.assert_allclose(run_oracle(h), _mean_of_values(h),
                               rtol=1e-13, atol=1e-15)


def test_zero_scale_gives_mean_of_values():
    p = small_problem(7, batch=3, lengths=("explicit", [1, 9, 22]), scale=0.0)
    h = p.host_arrays()
    np.testing.assert_allclose(run_oracle(h), _mean_of_values(h),
                               rtol=1e-13, atol=1e-15)


def _handmade(scores, values, scale):
    """One sequence, one head, D=2, page=2: keys chosen so that q.k_t equals
    `scores[t]` (q = e0, k_t = scores[t] e0) and v_t = values[t]."""
    L = len(scores)
    page = 2
    P = (L + page - 1) // page + 1
    q = f64_to_bf16_bits(np.array([[[1.0, 0.0]]]))
    k = np.zeros((P, 1, page, 2))
    v = np.zeros((P, 1, page, 2))
    # logical page j lives in physical page P-1-j (reversed placement)
    bt = np.array([[P - 1 - j for j in range((L + page - 1) // page)]],
                  dtype=np.int32)
    for t in range(L):
        k[bt[0, t // page], 0, t % page, 0] = scores[t]
        v[bt[0, t // page], 0, t % page, :] = values[t]
    return dict(q_bits=q, k_pool=f64_to_bf16_bits(k), v_pool=f64_to_bf16_bits(v),
                block_table=bt, seq_lens=np.array([L], dtype=np.int32),
                num_kv_heads=1, scale=scale)


def test_hand_worked_weights():
    # scores 0, 1, 2 times scale ln 2 -> exp weights 1 : 2 : 4, i.e. 1/7, 2/7, 4/7
    values = [[7.0, -1.0], [14.0, 3.0], [0.0, 5.0]]
    h = _handmade([0.0, 1.0, 2.0], values, math.log(2.0))
    got = run_oracle(h)[0, 0]
    want = np.array([(7 + 28 + 0) / 7.0, (-1 + 6 + 20) / 7.0])
    np.testing.assert_allclose(got, want, rtol=1e-15, atol=0)


def test_golden_worked_examples():
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden",
                        "worked_examples.json")
    with open(path) as f:
        cases = json.load(f)["cases"]
    assert cases
    for case in cases:
        h = _handmade(case["qk"], case["values"], math.log(case["scale_exp"]))
        got = run_oracle(h)[0, 0]
        np.testing.assert_allclose(got, case["out"], rtol=1e-14, atol=1e-15,
                                   err_msg=case["name"])


def test_grouped_heads_map_contiguously():
    # Hq=4, Hkv=2: heads 0,1 read kv head 0 and heads 2,3 read kv head 1.
    p = small_problem(8, batch=1, hq=4, hkv=2, d=4, page=4,
                      lengths=("explicit", [5]))
    h = p.host_arrays()
    v = bf16_bits_to_f64(h["v_pool"])
    v[:, 0] = 1.0
    v[:, 1] = -2.0
    h["v_pool"] = f64_to_bf16_bits(v)
    got = run_oracle(h)
    # weights sum to 1 up to fp64 rounding
    np.testing.assert_allclose(got[0, :2], 1.0, rtol=1e-14)
    np.testing.assert_allclose(got[0, 2:], -2.0, rtol=1e-14)


def test_large_scores_do_not_overflow():
    p = small_problem(9, batch=2, d=16, lengths=("explicit", [30, 7]),
                      scale=40.0)
    h = p.host_arrays()
    got = run_oracle(h)
    assert np.all(np.isfinite(got))
    np.testing.assert_allclose(got, dense_bruteforce(h), rtol=1e-11, atol=1e-13)


def test_empty_sequences_are_zero():
    p = small_problem(10, batch=3, lengths=("explicit", [0, 5, -3]))
    h = p.host_arrays()
    got = run_oracle(h)
    assert np.all(got[0] == 0) and np.all(got[2] == 0)
    assert np.any(got[1] != 0)


# ---------------------------------------------------------- invariants ---

@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_page_permutation_invariance_is_bit_exact(kv):
    p = small_problem(11, batch=4, lengths=("uniform", 1, 40), kv=kv)
    h = p.host_arrays()
    base = run_oracle(h, KV[kv])
    rng = np.random.default_rng(0)
    P = h["k_pool"].shape[0]
    pi = rng.permutation(P)
    h2 = dict(h)
    for name in ("k_pool", "v_pool"):
        arr = np.empty_like(h[name])
        arr[pi] = h[name]
        h2[name] = arr
    if kv != "bf16":
        for name in ("k_scale", "v_scale"):
            arr = np.empty_like(h[name])
            arr[pi] = h[name]
            h2[name] = arr
    h2["block_table"] = pi[h["block_table"]].astype(np.int32)
    assert np.array_equal(run_oracle(h2, KV[kv]), base)


def test_output_inside_convex_hull_of_values():
    p = small_problem(12, batch=4, lengths=("uniform", 1, 40))
    h = p.host_arrays()
    got = run_oracle(h)
    V = bf16_bits_to_f64(h["v_pool"])
    for b in range(4):
        L = int(h["seq_lens"][b])
        t = np.arange(L)
        vals = V[h["block_table"][b, t // 4], :, t % 4, :]     # [L, Hkv, D]
        lo = np.repeat(vals.min(axis=0), 2, axis=0)
        hi = np.repeat(vals.max(axis=0), 2, axis=0)
        assert np.all(got[b] >= lo - 1e-12) and np.all(got[b] <= hi + 1e-12)


def test_unread_memory_never_leaks():
    """NaN in tail slots, unused pages and padding must not reach outputs."""
    p = small_problem(13, batch=4, lengths=("explicit", [1, 6, 8, 13]),
                      pool_factor=2.0)
    h = p.host_arrays()
    base = run_oracle(h)
    nan_bits = np.uint16(0x7FC0)
    used = set()
    for b in range(4):
        L = int(h["seq_lens"][b])
        n = (L + 3) // 4
        for j in range(n):
            used.add(int(h["block_table"][b, j]))
        last = h["block_table"][b, n - 1]
        tail = L - (n - 1) * 4
        for name in ("k_pool", "v_pool"):
            h[name][last, :, tail:, :] = nan_bits
        h["block_table"][b, n:] = p.pad_page     # pad page is unused -> NaN
    for pg in range(h["k_pool"].shape[0]):
        if pg not in used:
            h["k_pool"][pg] = nan_bits
            h["v_pool"][pg] = nan_bits
    got = run_oracle(h)
    assert np.array_equal(got, base)


def test_one_hot_probe_reports_physical_location():
    """q = 8 e0 and scale 16; key t* has dim0 = 8 and every other key is 0, so
    the score gap is 1024 nats, exp(-1024) underflows to 0 in fp64, and the
    output equals the value stored at t*'s physical (page, slot, kv head),
    which the values encode as small integers."""
    p = small_problem(14, batch=3, hq=4, hkv=2, d=8, page=4,
                      lengths=("explicit", [9, 4, 13]), pool_factor=1.0)
    h = p.host_arrays()
    P = h["k_pool"].shape[0]
    q = np.zeros((3, 4, 8))
    q[:, :, 0] = 8.0
    h["q_bits"] = f64_to_bf16_bits(q)
    h["scale"] = 16.0          # score gap 8 * 8 * 16 = 1024 nats
    v = np.zeros((P, 2, 4, 8))
    for pg in range(P):
        for kvh in range(2):
            for s in range(4):
                v[pg, kvh, s, :3] = [pg, s, kvh]
    h["v_pool"] = f64_to_bf16_bits(v)
    for b in range(3):
        L = int(h["seq_lens"][b])
        for target in range(L):
            k = np.zeros((P, 2, 4, 8))
            k[h["block_table"][b, target // 4], :, target % 4, 0] = 8.0
            h["k_pool"] = f64_to_bf16_bits(k)
            got = run_oracle(h, rows=[[b, 0], [b, 3]])
            for r, kvh in ((0, 0), (1, 1)):
                assert got[r, 0] == h["block_table"][b, target // 4]
                assert got[r, 1] == target % 4
                assert got[r, 2] == kvh


def test_row_selection_matches_full_output():
    p = small_problem(15, batch=4, lengths=("uniform", 1, 30))
    h = p.host_arrays()
    full = run_oracle(h)
    rows = np.array([[3, 1], [0, 0], [2, 3], [3, 1]], dtype=np.int32)
    part = run_oracle(h, rows=rows)
    for r, (b, hh) in enumerate(rows):
        assert np.array_equal(part[r], full[b, hh])


# -------------------------------------------------------- preconditions ---

def test_out_of_range_page_is_rejected():
    p = small_problem(16, batch=2, lengths=("explicit", [5, 9]))
    h = p.host_arrays()
    h["block_table"][1, 2] = h["k_pool"].shape[0]
    with pytest.raises(oracle.OracleError):
        run_oracle(h)


def test_too_long_sequence_is_rejected():
    p = small_problem(17, batch=2, lengths=("explicit", [5, 9]))
    h = p.host_arrays()
    h["seq_lens"][0] = h["block_table"].shape[1] * 4 + 1
    with pytest.raises(oracle.OracleError):
        run_oracle(h)
