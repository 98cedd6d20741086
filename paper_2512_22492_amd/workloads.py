"""Seeded synthetic decode-attention workloads.

This module generates inputs only: sequence lengths, the placement of each
sequence's pages in a shuffled page pool, random query/key/value values and
their storage encodings (bf16 rounding, per-slab e4m3 quantisation).  It
contains none of the attention arithmetic and is shared by the GPU library's
tests and benchmark and by the oracle's tests.

The shapes follow the paper's rollout workload (Sec. 7.1: Qwen3-8B rollouts,
64 prompts per batch, text up to 65536 tokens; Sec. 7.3: a rollout length tail
beyond 4k tokens).  The paper's datasets are not used; attention cost depends
only on shapes and lengths, and values are N(0, 1).

Pool layout is [num_pages][num_kv_heads][page_size][head_dim] ("hnd"),
[num_pages][page_size][num_kv_heads][head_dim] ("nhd"), or one allocation
[num_pages][num_kv_heads][2][page_size][head_dim] holding each (page, kv
head)'s key slab and then its value slab ("hnd_kv"; k_pool and v_pool are
views of it): the same values, only stored in that order.  Pages are drawn
from one random permutation of the
whole pool and sequence b takes the next ceil(L_b / page_size) entries for its
logical pages 0, 1, ...
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

E4M3_MAX = 448.0

# Named workloads.  "lengths" is (kind, *params); "uniform" bounds are
# inclusive at both ends.
CONFIGS = {
    "tiny": dict(
        batch=4, num_q_heads=8, num_kv_heads=2, head_dim=128, page_size=16,
        lengths=("uniform", 1, 512), pool_pages=200, kv_dtype="bf16",
        seed=20251222),
    "qwen3_8b_step": dict(
        batch=64, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16,
        lengths=("fixed", 4096), pool_factor=1.25, kv_dtype="bf16",
        seed=20251223),
    "long_tail": dict(
        batch=256, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16,
        lengths=("lognormal", 4096, 0.8, 256, 32768), pool_factor=1.25,
        kv_dtype="bf16", seed=20251224),
    "straggler": dict(
        batch=16, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16,
        lengths=("uniform", 32768, 65536), pool_factor=1.25, kv_dtype="bf16",
        seed=20251225),
    "fp8_large_batch": dict(
        batch=1024, num_q_heads=32, num_kv_heads=8, head_dim=128,
        page_size=16, lengths=("uniform", 512, 2048), pool_factor=1.25,
        kv_dtype="fp8_e4m3", seed=20251226),
}

# Variant shapes (not among the five headline workloads): the per-GPU share of
# the Qwen3-8B step at the paper's rollout tensor parallelism of 8 (Sec. 7.1:
# one kv head and its 4 query heads per GPU), and the Qwen3-32B head layout
# (64 query heads, 8 kv heads; the paper evaluates 32B rollouts, Sec. 7.1,
# without stating its head counts).
CONFIGS.update({
    "tp8_share_step": dict(
        batch=64, num_q_heads=4, num_kv_heads=1, head_dim=128, page_size=16,
        lengths=("fixed", 4096), pool_factor=1.25, kv_dtype="bf16", seed=20251227),
    "qwen3_32b_step": dict(
        batch=64, num_q_heads=64, num_kv_heads=8, head_dim=128, page_size=16,
        lengths=("fixed", 4096), pool_factor=1.25, kv_dtype="bf16", seed=20251228),
    # a group of 16 query heads per kv head: the Qwen3-235B-A22B attention
    # layout (64 query heads, 4 kv heads), whose rollouts the paper also
    # evaluates (Sec. 7.1) without stating head counts
    "qwen3_235b_step": dict(
        batch=64, num_q_heads=64, num_kv_heads=4, head_dim=128, page_size=16,
        lengths=("fixed", 4096), pool_factor=1.25, kv_dtype="bf16", seed=20251229),
})

CONFIG_ORDER = ["tiny", "qwen3_8b_step", "long_tail", "straggler",
                "fp8_large_batch"]


@dataclasses.dataclass
class DecodeProblem:
    """One decode step's inputs.  Tensors live on one device."""
    name: str
    seed: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    kv_dtype: str               # "bf16" or "fp8_e4m3"
    layout: str                 # "hnd" or "nhd"
    scale: float
    q: torch.Tensor             # bf16 [B, Hq, D]
    k_pool: torch.Tensor        # bf16 or uint8 (e4m3 codes) [P, Hkv, page, D] or [P, page, Hkv, D]
    v_pool: torch.Tensor
    k_scale: Optional[torch.Tensor]   # fp32 [P, Hkv] (fp8 only)
    v_scale: Optional[torch.Tensor]
    block_table: torch.Tensor   # int32 [B, max_pages]
    seq_lens: torch.Tensor      # int32 [B]
    pad_page: int               # page index written into unused table slots
    kv_pool: Optional[torch.Tensor] = None  # "hnd_kv": [P, Hkv, 2, page, D]; k/v_pool view it

    @property
    def num_pages(self) -> int:
        return int(self.k_pool.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def device(self) -> torch.device:
        return self.q.device

    def lengths(self) -> np.ndarray:
        return self.seq_lens.cpu().numpy().astype(np.int64)

    def kv_bytes(self) -> int:
        """Bytes of K and V the step must read (plus fp8 slab scales)."""
        L = np.clip(self.lengths(), 0, None)
        elt = 2 if self.kv_dtype == "bf16" else 1
        total = int(L.sum()) * self.num_kv_heads * self.head_dim * 2 * elt
        if self.kv_dtype != "bf16":
            pages = (L + self.page_size - 1) // self.page_size
            total += int(pages.sum()) * self.num_kv_heads * 2 * 4
        return total

    def to(self, device) -> "DecodeProblem":
        def mv(t):
            return None if t is None else t.to(device)
        if self.kv_pool is not None:   # keep each value slab next to its key slab
            kv = self.kv_pool.to(device)
            k_pool, v_pool = kv[:, :, 0], kv[:, :, 1]
        else:
            kv, k_pool, v_pool = None, mv(self.k_pool), mv(self.v_pool)
        return dataclasses.replace(
            self, q=mv(self.q), k_pool=k_pool, v_pool=v_pool, kv_pool=kv,
            k_scale=mv(self.k_scale), v_scale=mv(self.v_scale),
            block_table=mv(self.block_table), seq_lens=mv(self.seq_lens))

    def clone_pools(self) -> "DecodeProblem":
        """The same problem over copies of the K/V pools and slab scales."""
        if self.kv_pool is not None:
            kv = self.kv_pool.clone()
            k_pool, v_pool = kv[:, :, 0], kv[:, :, 1]
        else:
            kv, k_pool, v_pool = None, self.k_pool.clone(), self.v_pool.clone()
        return dataclasses.replace(
            self, k_pool=k_pool, v_pool=v_pool, kv_pool=kv,
            k_scale=None if self.k_scale is None else self.k_scale.clone(),
            v_scale=None if self.v_scale is None else self.v_scale.clone())

    def host_arrays(self) -> dict:
        """numpy views for the oracle: bf16 as uint16 bits, e4m3 as uint8."""
        def bits(t):
            t = t.detach().cpu().contiguous()
            if t.dtype == torch.bfloat16:
                return t.view(torch.int16).numpy().view(np.uint16)
            return t.numpy()
        # "hnd_kv" views copy out as head-major pools
        layout = "hnd" if self.layout == "hnd_kv" else self.layout
        out = dict(q_bits=bits(self.q), k_pool=bits(self.k_pool),
                   v_pool=bits(self.v_pool),
                   block_table=self.block_table.cpu().numpy(),
                   seq_lens=self.seq_lens.cpu().numpy(),
                   num_kv_heads=self.num_kv_heads, scale=self.scale, layout=layout)
        if self.kv_dtype != "bf16":
            out["k_scale"] = self.k_scale.cpu().numpy()
            out["v_scale"] = self.v_scale.cpu().numpy()
        return out


def draw_lengths(rng: np.random.Generator, batch: int, spec) -> np.ndarray:
    kind = spec[0]
    if kind == "fixed":
        return np.full(batch, int(spec[1]), dtype=np.int64)
    if kind == "uniform":
        lo, hi = int(spec[1]), int(spec[2])
        return rng.integers(lo, hi, size=batch, endpoint=True, dtype=np.int64)
    if kind == "lognormal":
        median, sigma, lo, hi = spec[1:]
        z = rng.standard_normal(batch)
        L = np.rint(np.exp(math.log(median) + sigma * z))
        return np.clip(L, lo, hi).astype(np.int64)
    if kind == "explicit":
        L = np.asarray(spec[1], dtype=np.int64)
        if L.shape != (batch,):
            raise ValueError("explicit lengths must have one entry per sequence")
        return L
    raise ValueError("unknown length distribution %r" % (kind,))


def place_pages(rng: np.random.Generator, lengths: np.ndarray, page_size: int,
                pool_pages: Optional[int], pool_factor: float,
                max_pages: Optional[int] = None):
    """Block table from one random permutation of the pool.

    Returns (block_table int32 [B, max_pages], num_pages, pad_page).  Table
    slots past a sequence's last page hold pad_page, a valid page index that
    no sequence uses when the pool has a spare page.
    """
    used = np.where(lengths > 0, (lengths + page_size - 1) // page_size, 0)
    total = int(used.sum())
    if pool_pages is None:
        pool_pages = max(1, int(math.ceil(pool_factor * total)))
    if pool_pages < total:
        raise ValueError("pool of %d pages cannot hold %d" % (pool_pages, total))
    width = int(max(1, used.max(initial=0)))
    if max_pages is not None:
        if max_pages < width:
            raise ValueError("max_pages too small for the longest sequence")
        width = int(max_pages)
    perm = rng.permutation(pool_pages).astype(np.int64)
    pad_page = int(perm[total]) if pool_pages > total else int(perm[0])
    table = np.full((lengths.shape[0], width), pad_page, dtype=np.int32)
    off = 0
    for b, n in enumerate(used):
        table[b, :n] = perm[off:off + n]
        off += n
    return table, pool_pages, pad_page


def _randn_bf16(shape, gen: torch.Generator, device, chunk: int = 1 << 26):
    """N(0, 1) drawn in fp32 and rounded to bf16 (round-to-nearest-even)."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    for s in range(0, flat.numel(), chunk):
        n = min(chunk, flat.numel() - s)
        flat[s:s + n] = torch.randn(n, generator=gen, device=device,
                                    dtype=torch.float32).to(torch.bfloat16)
    return out


def quantize_e4m3_slabs(x: torch.Tensor):
    """Per-slab e4m3 quantisation of fp32 rows x [S, slab_elems].

    scale = absmax / 448 in fp32 (1 when the slab is all zero); codes are
    round-to-nearest-even e4m3 of clamp(x / scale, -448, 448).  Returns
    (codes uint8 [S, slab_elems], scale fp32 [S]).
    """
    absmax = x.abs().amax(dim=1)
    scale = absmax / E4M3_MAX
    scale = torch.where(absmax == 0, torch.ones_like(scale), scale)
    y = (x / scale[:, None]).clamp_(-E4M3_MAX, E4M3_MAX)
    codes = y.to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, scale


def _randn_e4m3_pool(num_slabs: int, slab_elems: int, gen: torch.Generator,
                     device, chunk_slabs: int = 1 << 15):
    codes = torch.empty((num_slabs, slab_elems), dtype=torch.uint8, device=device)
    scales = torch.empty((num_slabs,), dtype=torch.float32, device=device)
    for s in range(0, num_slabs, chunk_slabs):
        n = min(chunk_slabs, num_slabs - s)
        x = torch.randn((n, slab_elems), generator=gen, device=device,
                        dtype=torch.float32)
        c, sc = quantize_e4m3_slabs(x)
        codes[s:s + n] = c
        scales[s:s + n] = sc
    return codes, scales


def make_problem(name: str = "custom", *, batch: int, num_q_heads: int,
                 num_kv_heads: int, head_dim: int = 128, page_size: int = 16,
                 lengths, kv_dtype: str = "bf16", seed: int = 0,
                 pool_pages: Optional[int] = None, pool_factor: float = 1.25,
                 max_pages: Optional[int] = None, scale: Optional[float] = None,
                 layout: str = "hnd", device="cpu") -> DecodeProblem:
    """Build one seeded problem.  `lengths` is a distribution spec or an array.
    The values do not depend on `layout`."""
    if layout not in ("hnd", "nhd", "hnd_kv"):
        raise ValueError("layout must be 'hnd', 'nhd' or 'hnd_kv'")
    rng = np.random.default_rng(seed)
    if isinstance(lengths, (list, tuple)) and lengths and isinstance(lengths[0], str):
        L = draw_lengths(rng, batch, lengths)
    else:
        L = draw_lengths(rng, batch, ("explicit", lengths))
    table, P, pad = place_pages(rng, L, page_size, pool_pages, pool_factor,
                                max_pages)
    device = torch.device(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) * 7919 + 17)
    q = _randn_bf16((batch, num_q_heads, head_dim), gen, device)
    pool_shape = (P, num_kv_heads, page_size, head_dim)
    if kv_dtype == "bf16":
        k_pool = _randn_bf16(pool_shape, gen, device)
        v_pool = _randn_bf16(pool_shape, gen, device)
        k_scale = v_scale = None
    elif kv_dtype == "fp8_e4m3":
        slab = page_size * head_dim
        kc, ks = _randn_e4m3_pool(P * num_kv_heads, slab, gen, device)
        vc, vs = _randn_e4m3_pool(P * num_kv_heads, slab, gen, device)
        k_pool, v_pool = kc.view(pool_shape), vc.view(pool_shape)
        k_scale = ks.view(P, num_kv_heads)
        v_scale = vs.view(P, num_kv_heads)
    else:
        raise ValueError("kv_dtype must be 'bf16' or 'fp8_e4m3'")
    kv_pool = None
    if layout == "nhd":
        k_pool = k_pool.transpose(1, 2).contiguous()
        v_pool = v_pool.transpose(1, 2).contiguous()
    elif layout == "hnd_kv":
        kv_pool = torch.stack([k_pool, v_pool], dim=2)
        k_pool, v_pool = kv_pool[:, :, 0], kv_pool[:, :, 1]
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    return DecodeProblem(
        name=name, seed=int(seed), batch=batch, num_q_heads=num_q_heads,
        num_kv_heads=num_kv_heads, head_dim=head_dim, page_size=page_size,
        kv_dtype=kv_dtype, layout=layout, scale=float(scale), q=q, k_pool=k_pool,
        v_pool=v_pool, k_scale=k_scale, v_scale=v_scale,
        block_table=torch.from_numpy(table).to(device),
        seq_lens=torch.from_numpy(L.astype(np.int32)).to(device),
        pad_page=pad, kv_pool=kv_pool)


def make_config(name: str, device="cpu", seed: Optional[int] = None,
                layout: str = "hnd") -> DecodeProblem:
    """One of the named workloads, generated on `device`, pools in `layout`."""
    cfg = dict(CONFIGS[name])
    cfg_seed = cfg.pop("seed")
    return make_problem(name, seed=cfg_seed if seed is None else seed,
                        device=device, layout=layout, **cfg)


def describe(name: str) -> str:
    cfg = CONFIGS[name]
    return ("B=%d Hq=%d Hkv=%d D=%d page=%d lengths=%s kv=%s"
            % (cfg["batch"], cfg["num_q_heads"], cfg["num_kv_heads"],
               cfg["head_dim"], cfg["page_size"], cfg["lengths"],
               cfg["kv_dtype"]))
