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


def oracle_ref(p, rows=None, abs_values=False):
    """The oracle's decode attention of problem p; with abs_values, over the
    value pool of magnitudes |V| (same weights): M1 = sum w |v| / sum w."""
    h = p.host_arrays()
    if abs_values:
        h["v_pool"] = abs_value_host(p, h)
    return oracle.decode_attention(kv_dtype=KV[p.kv_dtype], rows=rows, **h)


# The matrix-core value pass (the default of the four-wavefront units) feeds
# each weight to the product as hi = bf16(p) plus lo = bf16(p - hi), which
# carries p to 2^-16 relative, and normalises by the fp32 sum of the weights:
# the result moves by at most 2^-16 M1 beyond fp32 rounding (the e4m3 case of
# the analysis above with the residual term).
PV_ROUND = 2.0 ** -16 * (1.0 + 2.0 ** -8)


def uses_pv(p, flags):
    """Whether a handle created with `flags` may take the matrix-core value
    pass (token-major handles with head-parallel units do not; the allowance
    applies to them too, as a bound)."""
    return not flags & (binding.RL_DA_PV_ON_VALU | binding.RL_DA_SCORES_ON_VALU)


def decode_extra(p, flags, rows=None):
    """Allowance on top of one ulp for the decode path a handle with `flags`
    takes: 0 for the vector-ALU value pass, PV_ROUND * M1 for the
    matrix-core one."""
    if not uses_pv(p, flags):
        return 0.0
    return PV_ROUND * oracle_ref(p, rows=rows, abs_values=True)


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
    ref_rms = float(np.sqrt(np.mean(ref * ref)))
    return dict(max_abs_err=float(err.max()), max_ulp=float(ulps.max()),
                frac_rne_equal=float(np.mean(got == rne_bf16(ref))),
                rel_rms_err=float(np.sqrt(np.mean(err * err))) / ref_rms if ref_rms > 0 else 0.0,
                elements=int(err.size))


# Extend attention feeds the P.V product with each probability rounded to
# bf16 (8 significant bits, round to nearest even): w_t (1 + d_t) with
# |d_t| <= 2^-8.  Writing o = sum w v / sum w:
#   bf16 pools normalise by the sum of the same rounded weights, so the fp32
#   result is sum w (1+d) v / sum w (1+d) = o + sum w d (v - o) / sum w (1+d),
#   off by at most 2^-8 / (1 - 2^-8) * sum w |v - o| / sum w
#   <= 2^-8 (1 + 2^-7) (M1 + |o|),  M1 = sum w |v| / sum w;
#   e4m3 pools normalise by the unrounded weights: off by at most 2^-8 M1.
# M1 is the attention output over the same weights with every value replaced
# by its magnitude (one more oracle call on a pool with the sign bits cleared).
P_ROUND = 2.0 ** -8 * (1.0 + 2.0 ** -7)


def extend_extra(kv_dtype, ref, abs_ref):
    """Per-element allowance of the rounded probabilities (above), given the
    reference o and the weighted mean magnitude M1 of the values."""
    ref = np.abs(np.asarray(ref, dtype=np.float64))
    abs_ref = np.asarray(abs_ref, dtype=np.float64)
    assert np.all(abs_ref >= ref * (1 - 1e-12)), "M1 must bound |o|"
    if kv_dtype == "bf16":
        return P_ROUND * (abs_ref + ref)
    return P_ROUND * abs_ref


def abs_value_host(p, h=None):
    """Host copy of problem p's value pool with every sign bit cleared (bf16
    bit 15, e4m3 bit 7): the pool of |V| under the same slab scales."""
    h = h if h is not None else p.host_arrays()
    v = h["v_pool"]
    return v & (np.uint16(0x7FFF) if v.dtype == np.uint16 else np.uint8(0x7F))


def max_pages_for(lengths, page=16):
    L = np.asarray(lengths)
    return max(1, int(math.ceil(max(1, L.max()) / page)))
