"""Pins for the oracle's extend (prefill) attention (CPU only): a decode step
is the one-token case; every query row equals a decode at its own position;
an independent numpy brute force with an explicit causal mask and torch's
float64 scaled-dot-product attention with a boolean mask agree; keys past a
query's position never affect it."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22492_amd import workloads

from test_oracle import bf16_bits_to_f64, decode_pool, run_oracle


def extend_problem(seed, new, prior, hq=8, hkv=2, d=16, page=4, kv="bf16", layout="hnd"):
    lengths = [a + b for a, b in zip(new, prior)]
    p = workloads.make_problem("ext", batch=len(new), num_q_heads=hq, num_kv_heads=hkv,
                               head_dim=d, page_size=page, lengths=lengths, kv_dtype=kv,
                               seed=seed, pool_factor=1.5, layout=layout)
    h = p.host_arrays()
    T = int(sum(new))
    gen = torch.Generator().manual_seed(seed + 7)
    q = torch.randn((T, hq, d), generator=gen).to(torch.bfloat16)
    h["q_bits"] = q.view(torch.int16).numpy().view(np.uint16)
    h["q_start"] = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    return p, h


def run_extend(h, kv=oracle.KV_BF16):
    kw = dict(num_kv_heads=h["num_kv_heads"], scale=h["scale"], kv_dtype=kv,
              layout=h.get("layout", "hnd"))
    if kv == oracle.KV_FP8_E4M3:
        kw.update(k_scale=h["k_scale"], v_scale=h["v_scale"])
    return oracle.extend_attention(h["q_bits"], h["q_start"], h["k_pool"], h["v_pool"],
                                   h["block_table"], h["seq_lens"], **kw)


def dense_causal(h, kv=oracle.KV_BF16):
    q = bf16_bits_to_f64(h["q_bits"])
    layout = h.get("layout", "hnd")
    K = decode_pool(h["k_pool"], kv, h.get("k_scale"), layout)
    V = decode_pool(h["v_pool"], kv, h.get("v_scale"), layout)
    if layout == "nhd":                 # view as [page][kv head][slot][dim]
        K, V = K.transpose(0, 2, 1, 3), V.transpose(0, 2, 1, 3)
    T, Hq, D = q.shape
    Hkv, page = K.shape[1], K.shape[2]
    G = Hq // Hkv
    out = np.zeros((T, Hq, D))
    qs = h["q_start"]
    for b in range(len(h["seq_lens"])):
        L = int(h["seq_lens"][b])
        n = qs[b + 1] - qs[b]
        if n == 0:
            continue
        t = np.arange(L)
        pages = h["block_table"][b, t // page]
        Kh = np.repeat(K[pages, :, t % page, :], G, axis=1)      # [L, Hq, D]
        Vh = np.repeat(V[pages, :, t % page, :], G, axis=1)
        s = np.einsum("nhd,thd->nht", q[qs[b]:qs[b + 1]], Kh) * h["scale"]
        pos = L - n + np.arange(n)
        s = np.where(t[None, None, :] <= pos[:, None, None], s, -np.inf)
        s = s - s.max(axis=2, keepdims=True)
        w = np.exp(s)
        w /= w.sum(axis=2, keepdims=True)
        out[qs[b]:qs[b + 1]] = np.einsum("nht,thd->nhd", w, Vh)
    return out


@pytest.mark.parametrize("layout", ["hnd", "nhd"])
@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("new,prior", [([1, 3, 5], [0, 7, 2]), ([8, 1, 0, 12], [4, 0, 9, 1]),
                                       ([17], [40])])
def test_matches_dense_causal_bruteforce(new, prior, kv, layout):
    code = oracle.KV_BF16 if kv == "bf16" else oracle.KV_FP8_E4M3
    p, h = extend_problem(1, new, prior, kv=kv, layout=layout)
    np.testing.assert_allclose(run_extend(h, code), dense_causal(h, code), rtol=1e-12,
                               atol=1e-14)


def test_matches_torch_sdpa_with_causal_mask():
    new, prior = [6, 2], [10, 3]
    p, h = extend_problem(2, new, prior, d=32, page=16)
    got = run_extend(h)
    q = torch.from_numpy(bf16_bits_to_f64(h["q_bits"]))
    K = torch.from_numpy(bf16_bits_to_f64(h["k_pool"]))
    V = torch.from_numpy(bf16_bits_to_f64(h["v_pool"]))
    for b in range(2):
        L, n = new[b] + prior[b], new[b]
        t = np.arange(L)
        pages = torch.from_numpy(h["block_table"][b, t // 16].astype(np.int64))
        slots = torch.from_numpy(t % 16)
        Kb = K[pages, :, slots, :].permute(1, 0, 2).repeat_interleave(4, 0)   # [Hq, L, D]
        Vb = V[pages, :, slots, :].permute(1, 0, 2).repeat_interleave(4, 0)
        qb = q[h["q_start"][b]:h["q_start"][b + 1]].permute(1, 0, 2)           # [Hq, n, D]
        mask = torch.from_numpy(t[None, :] <= (L - n + np.arange(n))[:, None])
        ref = torch.nn.functional.scaled_dot_product_attention(
            qb, Kb, Vb, attn_mask=mask, scale=h["scale"]).permute(1, 0, 2)
        np.testing.assert_allclose(got[h["q_start"][b]:h["q_start"][b + 1]], ref.numpy(),
                                   rtol=1e-12, atol=1e-14)


def test_one_new_token_is_a_decode_step():
    p, h = extend_problem(3, [1, 1, 1, 1], [0, 5, 16, 30])
    got = run_extend(h)
    dec = dict(h)
    dec["q_bits"] = h["q_bits"]                       # [B, Hq, D] since n_b = 1
    assert np.array_equal(got, run_oracle(dec))


def test_each_row_equals_a_decode_at_its_position():
    new, prior = [5, 3], [6, 0]
    p, h = extend_problem(4, new, prior)
    got = run_extend(h)
    for b in range(2):
        for i in range(new[b]):
            row = h["q_start"][b] + i
            dec = dict(h)
            dec["q_bits"] = np.repeat(h["q_bits"][row:row + 1], 2, axis=0)
            lens = h["seq_lens"].copy()
            lens[b] = prior[b] + i + 1
            dec["seq_lens"] = lens
            assert np.array_equal(got[row], run_oracle(dec)[b])


def test_keys_after_a_query_do_not_affect_it():
    new, prior = [6], [9]
    p, h = extend_problem(5, new, prior)
    base = run_extend(h)
    L = 15
    last_page, last_slot = h["block_table"][0, (L - 1) // 4], (L - 1) % 4
    h["k_pool"] = h["k_pool"].copy()
    h["v_pool"] = h["v_pool"].copy()
    h["k_pool"][last_page, :, last_slot, :] ^= 0x1234
    h["v_pool"][last_page, :, last_slot, :] ^= 0x0F0F
    moved = run_extend(h)
    assert np.array_equal(moved[:-1], base[:-1])          # only the last query sees it
    assert not np.array_equal(moved[-1], base[-1])


def test_extend_preconditions():
    p, h = extend_problem(6, [3, 2], [1, 1])
    bad = dict(h)
    bad["q_start"] = np.array([0, 3, 7], dtype=np.int32)   # 4 new tokens > length 3
    bad["q_bits"] = np.zeros((7, 8, 16), dtype=np.uint16)
    with pytest.raises(oracle.OracleError):
        run_extend(bad)
