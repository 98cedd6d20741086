"""Maximum sizes: pools whose pages lie beyond 4 GiB (64-bit page offsets in
decode, extend and append, both layouts) and a weight tensor larger than
4 GiB packed through a 1 GiB buffer."""
import numpy as np
import pytest
import torch

import oracle
from oracle import weight_sync as WS
from paper_2512_22492_amd import binding as B
from paper_2512_22492_amd import workloads

from gpu_util import (KV, abs_value_host, bf16_to_f64, check_close, decode_extra, device,
                      extend_extra, oracle_ref, run_gpu)

pytestmark = pytest.mark.gpu

POOL_PAGES = 140000      # 140000 x 8 heads x 4 KiB = 4.6 GB per bf16 pool


def top_of_pool_problem(kv, layout, lengths, seed):
    """Sequences whose pages are the highest page indices of a > 4 GiB pool."""
    p = workloads.make_problem("large", batch=len(lengths), num_q_heads=32, num_kv_heads=8,
                               lengths=list(lengths), kv_dtype=kv, seed=seed, layout=layout,
                               pool_pages=POOL_PAGES, device=device())
    need = [(L + 15) // 16 for L in lengths]
    bt = p.block_table.clone()
    nxt = POOL_PAGES - 1
    for b, n in enumerate(need):
        for j in range(n):
            bt[b, j] = nxt
            nxt -= 1
    p.block_table = bt
    return p


@pytest.mark.parametrize("layout", ["hnd", "nhd"])
@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_decode_reads_pages_beyond_4gib(kv, layout):
    lengths = [1, 700, 4100, 9000]
    p = top_of_pool_problem(kv, layout, lengths, seed=71)
    assert p.k_pool.numel() * p.k_pool.element_size() > (1 << 32) or kv != "bf16"
    rows = np.array([(b, h) for b in range(len(lengths)) for h in (0, 5, 31)], dtype=np.int32)
    out = run_gpu(p)
    got = bf16_to_f64(out[torch.from_numpy(rows[:, 0]).long(), torch.from_numpy(rows[:, 1]).long()])
    print(check_close(got, oracle_ref(p, rows=rows), "decode > 4 GiB %s %s" % (kv, layout),
                      extra_abs=decode_extra(p, 0, rows=rows)))


@pytest.mark.parametrize("layout", ["hnd", "nhd"])
def test_extend_and_append_beyond_4gib(layout):
    lengths = [300, 2000]
    p = top_of_pool_problem("bf16", layout, [L + 1 for L in lengths], seed=72)
    p.seq_lens.copy_(torch.tensor(lengths, dtype=torch.int32, device=device()))
    # append one token per sequence, then compare the written rows
    gen = torch.Generator().manual_seed(73)
    k = torch.randn((2, 8, 128), generator=gen).to(torch.bfloat16)
    v = torch.randn((2, 8, 128), generator=gen).to(torch.bfloat16)
    B.kv_append(p, k.to(device()), v.to(device()))
    torch.cuda.synchronize()
    bt = p.block_table.cpu().numpy()
    for b, L in enumerate(lengths):
        page, slot = int(bt[b, L // 16]), L % 16
        got_k = p.k_pool[page, :, slot] if layout == "hnd" else p.k_pool[page, slot]
        assert torch.equal(got_k.cpu().view(torch.int16), k[b].view(torch.int16))
    p.seq_lens += 1
    # extend: the last 1 and 17 cached tokens as new tokens
    new = [1, 17]
    q = torch.randn((sum(new), 32, 128), generator=gen).to(torch.bfloat16).to(device())
    q_start = torch.tensor([0, 1, 18], dtype=torch.int32, device=device())
    out = torch.full_like(q, float("nan"))
    B.extend_attention(p, q, q_start, max(new), out)
    torch.cuda.synchronize()
    # oracle over the gathered sequences only (the full pool is too large to copy)
    h = p.host_arrays()
    ref, m1 = [oracle.extend_attention(q.cpu().view(torch.int16).numpy().view(np.uint16),
                                       q_start.cpu().numpy(), h["k_pool"], v,
                                       h["block_table"], h["seq_lens"], num_kv_heads=8,
                                       scale=p.scale, layout=layout)
               for v in (h["v_pool"], abs_value_host(p, h))]
    print(check_close(bf16_to_f64(out), ref, "extend > 4 GiB " + layout,
                      extra_abs=extend_extra("bf16", ref, m1)))


def test_pack_a_tensor_larger_than_4gib():
    n = (4 << 30) + 12345
    big = torch.empty(n, dtype=torch.uint8, device=device())
    big.view(-1)[: n // 4 * 4].view(torch.int32).copy_(
        torch.arange(n // 4, dtype=torch.int32, device=device()) * 1103515245)
    small = torch.randint(0, 256, (1000,), dtype=torch.uint8, device=device())
    sizes = [1000, n, 1000]
    tensors = [small, big, small.clone()]
    cap = 1 << 30
    buf = torch.empty(cap, dtype=torch.uint8, device=device())
    pieces = WS.plan(sizes, cap, 256)
    back = [torch.zeros_like(t) for t in tensors]
    with B.WeightSync(tensors, buf, align=256) as ws, B.WeightSync(back, buf, align=256) as un:
        assert ws.num_chunks == WS.num_chunks(pieces) == 5
        for c in range(ws.num_chunks):
            ws.pack(c)
            torch.cuda.synchronize()
            for t, ch, t_off, b_off, nb in pieces:
                if ch == c:
                    assert torch.equal(buf[b_off:b_off + nb], tensors[t][t_off:t_off + nb]), \
                        (c, t, t_off)
            un.unpack(c)
            torch.cuda.synchronize()
    for a, b in zip(tensors, back):
        assert torch.equal(a, b)
