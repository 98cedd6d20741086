"""The binding's argument checks (CPU): what every entry point runs on each
tensor before its C call, so a wrong dtype, shape, layout or device raises
ValueError instead of reaching a kernel."""
import pytest
import torch

from paper_2512_22492_amd import binding as B


def test_check_tensor_accepts_matching_tensors():
    t = torch.empty((4, 8, 128), dtype=torch.bfloat16)
    B._check_tensor("t", t, dtype=torch.bfloat16, shape=(4, 8, 128), device=t.device)
    B._check_tensor("t", t, dtype=(torch.uint8, torch.bfloat16), shape=(None, 8, None))
    B._check_tensor("t", t, ndim=3)
    B._check_tensor("t", t[:, :4], contiguous=False, shape=(4, 4, 128))


@pytest.mark.parametrize("kw", [
    dict(dtype=torch.float32),
    dict(dtype=(torch.uint8, torch.int32)),
    dict(shape=(4, 8, 64)),
    dict(shape=(4, 8)),
    dict(shape=(4, 8, 128, 1)),
    dict(shape=(None, 4, None)),
    dict(ndim=2),
    dict(device=torch.device("meta")),
])
def test_check_tensor_rejects(kw):
    t = torch.empty((4, 8, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        B._check_tensor("t", t, **kw)


def test_check_tensor_rejects_non_tensors_and_strided_views():
    t = torch.empty((4, 8, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        B._check_tensor("t", [1, 2, 3])
    with pytest.raises(ValueError):
        B._check_tensor("t", t[:, ::2], shape=(4, 4, 128))


def test_check_table_and_pools():
    bt = torch.zeros((3, 5), dtype=torch.int32)
    sl = torch.ones(3, dtype=torch.int32)
    B._check_table(bt, sl, 3, bt.device)
    for args in [(bt.long(), sl, 3), (bt, sl.long(), 3), (bt, sl, 2), (bt[:, ::2], sl, 3),
                 (bt, sl[:2], 3)]:
        with pytest.raises(ValueError):
            B._check_table(*args, bt.device)
    k = torch.empty((6, 2, 16, 128), dtype=torch.bfloat16)
    v = torch.empty_like(k)
    kw = dict(kv_dtype=B.RL_DA_KV_BF16, layout=B.RL_DA_LAYOUT_HND, num_kv_heads=2,
              head_dim=128, page_size=16, device=k.device)
    assert B._check_pools(k, v, None, None, **kw) == 6
    with pytest.raises(ValueError):
        B._check_pools(k, v[:5], None, None, **kw)
    with pytest.raises(ValueError):
        B._check_pools(k, v, torch.ones((6, 2)), torch.ones((6, 2)), **kw)
    with pytest.raises(ValueError):          # token-major pools checked as head-major
        B._check_pools(k.transpose(1, 2).contiguous(), v.transpose(1, 2).contiguous(),
                       None, None, **kw)
    k8 = torch.empty((6, 2, 16, 128), dtype=torch.uint8)
    kw8 = dict(kw, kv_dtype=B.RL_DA_KV_FP8_E4M3)
    assert B._check_pools(k8, k8.clone(), torch.ones((6, 2)), torch.ones((6, 2)), **kw8) == 6
    with pytest.raises(ValueError):
        B._check_pools(k8, k8.clone(), None, None, **kw8)
    with pytest.raises(ValueError):
        B._check_pools(k8, k8.clone(), torch.ones((6, 3)), torch.ones((6, 2)), **kw8)
