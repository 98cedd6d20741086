"""Helpers shared by the GPU tests: run the HIP library through its C
interface and compare against the fp64 oracle."""
import math

import numpy as np
import torch

import oracle
from paper_2512_22492_amd import binding

OFFICIAL_ATOL = 1e-2
OFFICIAL_RTOL = 1e-2
# fp32 accumulation error allowance on top of one bf16 ulp (see check_close).
TIGHT_ABS = 1e-6

KV = {"bf16": oracle.KV_BF16, "fp8_e4m3": oracle.KV_FP8_E4M3}


def device():
    return torch.device("cuda:0")


def run_gpu(p, *, flags=0, split_tokens=0, attn=None, stream=None):
    """One decode step of problem p (tensors on the GPU); returns bf16 out."""
    out = torch.full_like(p.q, float("nan"))
    if attn is None:
        with binding.DecodeAttention.for_problem(p, flags=flags,
                                                 split_tokens=split_tokens) as a:
            a.run_problem(p, out, stream)
            torch.cuda.synchronize()
    else:
        attn.run_problem(p, out, stream)
        torch.cuda.synchronize()
    return out


def oracle_ref(p, rows=None):
    h = p.host_arrays()
    return oracle.decode_attention(kv_dtype=KV[p.kv_dtype], rows=rows, **h)


def bf16_to_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (8 significant bits)."""
    a = np.abs(x)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.maximum(e, -126)
    return np.where(a > 0, np.exp2(e - 7), 0.0)


def rne_bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float64)).float().to(
        torch.bfloat16).double().numpy()


def check_close(got, ref, what="", extra_abs=0.0):
    """Asserts the official tolerance |err| <= 1e-2 + 1e-2 |ref| and the tight
    one: the bf16 output is within one bf16 ulp of the fp64 reference (plus
    1e-6 absolute for fp32 accumulation), which rounding an fp32 result that
    carries ~1e-6 relative error guarantees; extra_abs widens the tight bound
    for paths whose arithmetic carries a known extra error.  Returns error
    statistics."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "%s: non-finite output" % what
    err = np.abs(got - ref)
    official = OFFICIAL_ATOL + OFFICIAL_RTOL * np.abs(ref)
    worst = np.unravel_index(np.argmax(err - official), err.shape)
    assert np.all(err <= official), (
        "%s: |err| %.3g > tolerance at %s (ref %.6g got %.6g)"
        % (what, err[worst], worst, ref[worst], got[worst]))
    ulp = bf16_ulp(ref)
    tight = ulp + TIGHT_ABS + extra_abs
    worst = np.unravel_index(np.argmax(err - tight), err.shape)
    assert np.all(err <= tight), (
        "%s: |err| %.3g exceeds one bf16 ulp (%.3g) at %s (ref %.8g got %.8g)"
        % (what, err[worst], ulp[worst], worst, ref[worst], got[worst]))
    with np.errstate(invalid="ignore", divide="ignore"):
        ulps = np.where(ulp > 0, err / ulp, 0.0)
    return dict(max_abs_err=float(err.max()), max_ulp=float(ulps.max()),
                frac_rne_equal=float(np.mean(got == rne_bf16(ref))))


def sample_rows(p, n, seed=0):
    """(b, h) pairs: the longest and shortest sequences in full, plus random."""
    rng = np.random.default_rng(seed)
    L = p.lengths()
    Hq = p.num_q_heads
    rows = set()
    for b in (int(np.argmax(L)), int(np.argmin(L))):
        for h in range(0, Hq, max(1, Hq // 8)):
            rows.add((b, h))
    while len(rows) < n:
        rows.add((int(rng.integers(p.batch)), int(rng.integers(Hq))))
    return np.array(sorted(rows), dtype=np.int32)


def max_pages_for(lengths, page=16):
    L = np.asarray(lengths)
    return max(1, int(math.ceil(max(1, L.max()) / page)))
