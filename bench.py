#!/usr/bin/env python3
"""Decode-attention benchmark: one layer, one decode step, one GPU.

A step is one rl_decode_attn_run() (split-K kernel + merge kernel) over one
batch.  Inputs are seeded synthetic tensors resident in HBM before timing
starts.  Prints one JSON line:
  value      = KV bytes read per step / step time  (GB/s, the metric's unit)
  roofline   = the split-K kernel's achieved bytes/s against 8 TB/s: the
               step's algorithmic bytes over the kernel's mean duration --
               the timed pass's GPU time per step (an event pair around the K
               back-to-back steps) when a step is that kernel alone, else HIP
               events attached to each of its launches in a second pass of K
               steps (the first pass, which gives value, has none)
  cpu_baseline = the fp64 oracle timed on the host on a sample of the step
  parity     = the GPU output of that sample against the oracle's
--op extend reports TFLOP/s against the bf16 MFMA peak, with the oracle's
extend attention timed on the launch's first sequences as its cpu_baseline
and the GPU output's error statistics on them as its parity.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# default warm-up of --op extend, in milliseconds of back-to-back launches
EXTEND_WARMUP_MS = 60.0
# PCIe 5.0 x16, one direction: 32 GT/s x 16 lanes x 128/130 / 8
PCIE5_X16_GBS = 63.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
COPY_CALIBRATION_BYTES = 1 << 30


def bench_kernels():
    """ctypes handle of the measurement-only kernel library."""
    import ctypes
    import torch  # noqa: F401  (binds the library to torch's HIP runtime)
    from paper_2512_22492_amd import build
    lib = ctypes.CDLL(build.BENCH_LIB_PATH)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    lib.rl_bench_copy.argtypes = [vp, vp, sz, vp]
    lib.rl_bench_stream_read.argtypes = [vp, sz, vp, ctypes.c_int, vp]
    lib.rl_bench_page_read.argtypes = [vp, vp, vp, i32, vp, ctypes.c_int64, i32, i32, i32,
                                       i32, vp, vp]
    for f in (lib.rl_bench_copy, lib.rl_bench_stream_read, lib.rl_bench_page_read):
        f.restype = ctypes.c_int
    return lib


def read_ceilings(p, stream):
    """Achievable read bandwidth: a contiguous 4 GiB stream, and the decode
    step's own K/V page reads with no arithmetic, divided evenly over the
    work-groups (64 pages of one kv head each).  Best of several runs."""
    import numpy as np
    import torch
    lib = bench_kernels()
    s = stream.cuda_stream
    nbytes = 4 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    best_stream = 0.0
    for grid in (1024, 2048, 8192):
        sink = torch.empty(grid * 256, dtype=torch.int32, device="cuda")
        for it in range(6):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            assert lib.rl_bench_stream_read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, s) == 0
            e1.record(stream)
            e1.synchronize()
            if it:
                best_stream = max(best_stream, nbytes / (e0.elapsed_time(e1) / 1e3) / 1e9)
    del buf
    unit_pages = 64
    pages = (np.clip(p.lengths(), 0, p.max_pages * p.page_size) + p.page_size - 1) // p.page_size
    prefix = np.concatenate([[0], np.cumsum(pages)]).astype(np.int32)
    total_pages = int(prefix[-1])
    prefix_dev = torch.from_numpy(prefix).to("cuda")
    units = p.num_kv_heads * ((total_pages + unit_pages - 1) // unit_pages)
    sink = torch.empty(max(units, 1) * 256, dtype=torch.int32, device="cuda")
    best_page = 0.0
    kv = p.kv_bytes()
    slab = p.page_size * p.head_dim * (2 if p.kv_dtype == "bf16" else 1)
    for it in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        assert lib.rl_bench_page_read(p.k_pool.data_ptr(), p.v_pool.data_ptr(),
                                      p.block_table.data_ptr(), p.max_pages,
                                      prefix_dev.data_ptr(), total_pages, p.batch,
                                      p.num_kv_heads, unit_pages, slab, sink.data_ptr(),
                                      s) == 0
        e1.record(stream)
        e1.synchronize()
        if it:
            best_page = max(best_page, kv / (e0.elapsed_time(e1) / 1e3) / 1e9)
    # the page-read kernel walks head-major slabs whatever the pool's layout
    return {"stream_read_GBs": round(best_stream, 1), "page_read_GBs": round(best_page, 1),
            "page_read_layout": "hnd"}


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before the timed ones (default 5; for --op extend, "
                         "as many launches as fill %d ms, since a stream of matrix work "
                         "raises the clock over its first tens of milliseconds)"
                         % EXTEND_WARMUP_MS)
    ap.add_argument("--config", default="qwen3_8b_step",
                    help="workload name (see paper_2512_22492_amd.workloads.CONFIGS)")
    ap.add_argument("--replicas", type=int, default=2,
                    help="copies of the KV pools visited round-robin, so that no step "
                         "reads data a previous step left in the caches")
    ap.add_argument("--scores", choices=["mfma", "valu"], default="mfma",
                    help="score path of the split-K kernel")
    ap.add_argument("--pv", choices=["mfma", "valu"], default="mfma",
                    help="P.V product of the split-K kernel: the matrix cores (default), or "
                         "vector-ALU FMAs (not for 16 query heads per kv head)")
    ap.add_argument("--split-tokens", type=int, default=0)
    ap.add_argument("--layout", choices=["hnd", "nhd", "hnd_kv"], default="hnd",
                    help="pool layout: [page][kv head][slot][dim], [page][slot][kv head][dim], "
                         "or [page][kv head][K|V][slot][dim] in one allocation")
    ap.add_argument("--per-head-units", action="store_true",
                    help="token-major pools: four-wavefront units per kv head")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-input-digests", action="store_true",
                    help="skip the SHA-256 of the input buffers")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="do not record events around the split kernel (profiling runs)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the read-ceiling measurements")
    ap.add_argument("--pmc-calibrate", action="store_true",
                    help="launch one plain copy of %d bytes first, so that a counter "
                         "run can scale FETCH_SIZE/WRITE_SIZE" % COPY_CALIBRATION_BYTES)
    ap.add_argument("--op", choices=["attention", "append", "extend", "pack", "d2h"],
                    default="attention",
                    help="attention (the decode step, default), the KV-cache append that "
                         "precedes it, or extend (prefill) attention of --new-tokens per "
                         "sequence after the workload's cached lengths (separate JSON lines "
                         "with their own metrics)")
    ap.add_argument("--new-tokens", type=int, default=512,
                    help="new tokens per sequence for --op extend")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, "
                         "WRITE_SIZE) of a --pmc-calibrate run into profiles/traffic.json")
    return ap.parse_args()


def _pmc_means(path, counter):
    """Mean counter value per kernel name in a rocprofv3 counter_collection.csv."""
    import csv
    sums = {}
    with open(path) as f:
        for row in csv.DictReader(f):
            if row.get("Counter_Name") != counter:
                continue
            name = row["Kernel_Name"]
            tot, n = sums.get(name, (0.0, 0))
            sums[name] = (tot + float(row["Counter_Value"]), n + 1)
    return {k: v[0] / v[1] for k, v in sums.items()}


# Per measured operation: the kernel whose counters are summarised (name
# prefix in the profiler's output) and the sources it is built from.
OP_KERNELS = {
    "attention": ("void (anonymous namespace)::split_", ("rl_common.h", "rl_decode.hip")),
    "pack": ("void (anonymous namespace)::copy_pieces<true>", ("rl_common.h", "rl_weight_sync.hip")),
}


def summarize_pmc(fetch_csv, write_csv, config, op="attention"):
    """HBM bytes per launch of the op's kernel, each counter scaled by its
    reading for the calibration copy (which moves COPY_CALIBRATION_BYTES each
    way)."""
    fetch = _pmc_means(fetch_csv, "FETCH_SIZE")
    write = _pmc_means(write_csv, "WRITE_SIZE")

    def pick(d, key):
        names = [k for k in d if k.startswith(key)]
        if len(names) != 1:
            raise SystemExit("expected one kernel matching %r, got %s" % (key, names))
        return d[names[0]]

    copy_kib = COPY_CALIBRATION_BYTES / 1024.0
    copy_name = "(anonymous namespace)::copy_kernel"
    split_name = OP_KERNELS[op][0]
    f_scale = copy_kib / pick(fetch, copy_name)
    w_scale = copy_kib / pick(write, copy_name)
    split_f = pick(fetch, split_name)
    split_w = pick(write, split_name)
    entry = {
        "kernel_source_sha256": kernel_source_sha(op),
        "fetch_kib_raw": split_f, "write_kib_raw": split_w,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "bytes_per_launch": int(round((split_f * f_scale + split_w * w_scale) * 1024)),
    }
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    data[config] = entry
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(entry))


def algorithmic_bytes(p):
    """Bytes one decode step must move: K and V of every cached token (plus
    fp8 slab scales), the queries, the outputs, the used block-table entries
    and seq_lens.  Returns (total, KV part)."""
    import numpy as np
    L = np.clip(p.lengths(), 0, None)
    pages = (L + p.page_size - 1) // p.page_size
    kv = p.kv_bytes()
    q = p.batch * p.num_q_heads * p.head_dim * 2
    out = q
    return kv + q + out + int(pages.sum()) * 4 + p.batch * 4, kv


def load_traffic(config, kernel_source_sha):
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    entry = data.get(config)
    if not entry or entry.get("kernel_source_sha256") != kernel_source_sha:
        return None
    return entry.get("bytes_per_launch")


def kernel_source_sha(op="attention"):
    """sha256 over the sources of the op's kernel (shared header first)."""
    import hashlib
    h = hashlib.sha256()
    for name in OP_KERNELS[op][1]:
        with open(os.path.join(ROOT, "paper_2512_22492_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (8 significant bits)."""
    import numpy as np
    a = np.abs(x)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(np.maximum(e, -126) - 7), 0.0)


def parity_stats(got, ref):
    """Error of the GPU's bf16 output against the fp64 oracle: the official
    bound (|err| <= 1e-2 + 1e-2 |ref|), max |err|, max error in bf16 ulps of
    the reference, the fraction of elements equal to the correctly rounded
    reference, and the relative RMS error."""
    import numpy as np
    import torch
    err = np.abs(got - ref)
    ulp = _bf16_ulp(ref)
    with np.errstate(invalid="ignore", divide="ignore"):
        ulps = np.where(ulp > 0, err / ulp, 0.0)
    rne = torch.from_numpy(ref).float().to(torch.bfloat16).double().numpy()
    rms = float(np.sqrt(np.mean(ref * ref)))
    return {
        "elements": int(err.size),
        "official_bound_holds": bool(np.all(err <= 1e-2 + 1e-2 * np.abs(ref))),
        "max_abs_err": float(err.max()),
        "max_ulp": round(float(ulps.max()), 4),
        # the tests' internal gate: one bf16 ulp of the reference plus 1e-6
        # (fp32 accumulation; it dominates where |ref| is below ~1e-4)
        "max_err_over_ulp_gate": round(float((err / (ulp + 1e-6)).max()), 4),
        "frac_rne_equal": round(float(np.mean(got == rne)), 6),
        "rel_rms_err": float(np.sqrt(np.mean(err * err))) / rms if rms > 0 else 0.0,
    }


class _host_oracle:
    """Builds the oracle for this host (-O3 -march=native, no FMA contraction:
    the same results as the test build) in a temporary directory and makes it
    the library the oracle module calls; yields a description of the build."""

    def __enter__(self):
        import tempfile

        import oracle
        self._tmp = tempfile.mkdtemp(prefix="oracle_native_")
        try:
            lib, build = oracle.build_native(self._tmp), \
                "gcc -O3 -march=native -ffp-contract=off -fopenmp"
        except Exception as e:  # no compiler on this host: the portable build
            print("bench: native oracle build failed (%s); timing the portable build" % e,
                  file=sys.stderr, flush=True)
            lib, build = oracle.LIB_PATH, "gcc -O2 -ffp-contract=off -fopenmp (portable)"
        self._using = oracle.using_library(lib)
        self._using.__enter__()
        return build

    def __exit__(self, *exc):
        import shutil
        try:
            return self._using.__exit__(*exc)
        finally:
            shutil.rmtree(self._tmp, ignore_errors=True)


def cpu_baseline(p, gpu_out, min_seconds=10.0):
    """Times the oracle on the host, built for this host (-O3 -march=native,
    no FMA contraction: the same results as the test build).  The sample is
    the whole step (every (sequence, head) row) when that is bounded, else
    the first sequences.  The oracle's output of the sample also gives the
    GPU output's error statistics."""
    import numpy as np
    import oracle
    kv_code = oracle.KV_BF16 if p.kv_dtype == "bf16" else oracle.KV_FP8_E4M3
    h = p.host_arrays()
    L = np.clip(p.lengths(), 0, None)
    # bound the sample to ~5e10 fp64 multiply-adds (a few seconds on 16 cores)
    per_seq = L * p.num_q_heads * p.head_dim * 2
    nseq = int(np.searchsorted(np.cumsum(per_seq), 5e10, side="right"))
    nseq = max(1, min(p.batch, nseq))
    rows = np.array([(b, hh) for b in range(nseq) for hh in range(p.num_q_heads)],
                    dtype=np.int32)
    with _host_oracle() as build:
        # repeat the sample until about min_seconds of CPU work have been timed
        reps, dt, ref = 0, 0.0, None
        while reps == 0 or dt < min_seconds:
            t0 = time.perf_counter()
            ref = oracle.decode_attention(kv_dtype=kv_code, rows=rows, **h)
            dt += time.perf_counter() - t0
            reps += 1
        cores = oracle.max_threads()
        # one thread, on the first sequence's rows (a few seconds)
        rows1 = rows[:p.num_q_heads]
        oracle.set_threads(1)
        try:
            t0 = time.perf_counter()
            oracle.decode_attention(kv_dtype=kv_code, rows=rows1, **h)
            dt1 = time.perf_counter() - t0
        finally:
            oracle.set_threads(cores)
    elt = 2 if p.kv_dtype == "bf16" else 1
    kv = int(L[:nseq].sum()) * p.num_kv_heads * p.head_dim * 2 * elt * reps
    kv1 = int(L[0]) * p.num_kv_heads * p.head_dim * 2 * elt
    got = gpu_out[:nseq].float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    return {
        "value": kv / dt / 1e9,
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": "%d of %d sequences (%d query-head rows, all tokens), fp64, %d passes "
                  "in %.2f s; %.1f query-tokens/s" % (nseq, p.batch, len(rows), reps, dt,
                                                     nseq * reps / dt),
        "build": build,
        "single_thread_GBs": round(kv1 / dt1 / 1e9, 4),
        "single_thread_sample": "sequence 0 (%d tokens, %d query heads), 1 pass"
                                % (int(L[0]), p.num_q_heads),
        "cpu_model": _cpu_model(),
        "seconds": dt,
    }, parity_stats(got, ref)


def _cpu_model():
    """The host CPU as /proc/cpuinfo names it: model name, family, model,
    stepping, and the logical CPUs this process may run on."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if ":" not in line:
                    if info:
                        break
                    continue
                k, v = (x.strip() for x in line.split(":", 1))
                if k in ("vendor_id", "model name", "cpu family", "model", "stepping",
                         "cpu MHz") and k not in info:
                    info[k] = v
    except OSError:
        return None
    try:
        info["usable_cpus"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        info["usable_cpus"] = os.cpu_count()
    return info


def input_digests(p):
    """SHA-256 of every input buffer of a decode problem (host copies)."""
    import hashlib
    import torch
    out = {}
    for name in ("q", "k_pool", "v_pool", "k_scale", "v_scale", "block_table", "seq_lens"):
        t = getattr(p, name)
        if t is None:
            continue
        h = hashlib.sha256()
        flat = t.reshape(-1).view(torch.uint8) if t.dtype != torch.uint8 else t.reshape(-1)
        step = 1 << 28
        for i in range(0, flat.numel(), step):
            h.update(flat[i:i + step].cpu().numpy().tobytes())
        out[name] = h.hexdigest()[:16]
    return out


def bench_append(args, base, stream):
    """Times K KV-cache appends (one new token per sequence and kv head) on the
    workload's shapes; every sequence appends at its current length."""
    import numpy as np
    import torch
    from paper_2512_22492_amd import binding
    L = base.lengths()
    room = L < base.max_pages * base.page_size
    if not room.all():
        # append at the last slot of the last page instead of past the table
        base.seq_lens.copy_(torch.from_numpy(np.minimum(L, base.max_pages * base.page_size - 1)
                                             .astype(np.int32)).to(base.seq_lens.device))
    # A token that opens a page goes to a page of its own, taken from the
    # pool's unused pages, as a serving engine would allocate it (the table's
    # padding slots all name one shared page, which several sequences would
    # otherwise write at once).
    L = base.lengths()
    table = base.block_table.cpu().numpy().copy()
    opens = (L % base.page_size == 0) & (L // base.page_size < base.max_pages)
    if opens.any():
        in_use = np.zeros(base.num_pages, dtype=bool)
        in_use[table.reshape(-1)] = True
        free = np.flatnonzero(~in_use)
        if free.size < int(opens.sum()):
            raise SystemExit("the pool has too few unused pages for the new tokens")
        rows = np.flatnonzero(opens)
        table[rows, L[rows] // base.page_size] = free[:rows.size]
        base.block_table.copy_(torch.from_numpy(table).to(base.block_table.device))
    gen = torch.Generator(device=base.q.device).manual_seed(1)
    shape = (base.batch, base.num_kv_heads, base.head_dim)
    k = torch.randn(shape, generator=gen, device=base.q.device).to(torch.bfloat16)
    v = torch.randn(shape, generator=gen, device=base.q.device).to(torch.bfloat16)
    # the cache before the first append, for the oracle leg (appending the
    # same tokens at the same lengths again changes nothing: an e4m3 page's
    # scale only grows, to the largest token's absmax / 448)
    before = None if args.no_cpu_baseline else base.host_arrays()
    # the cache is checked once; each call checks only the new tokens
    append = binding.KvAppender(base)
    for _ in range(args.warmup):
        append(k, v, stream=stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        append(k, v, stream=stream)
    torch.cuda.synchronize()
    us = (time.perf_counter() - t0) * 1e6 / args.steps
    elt = 2 if base.kv_dtype == "bf16" else 1
    tok = base.batch * base.num_kv_heads * base.head_dim
    moved = 2 * (tok * 2 + tok * elt) + base.batch * 8   # read new K/V, write slots, table
    record = {
        "metric": "KV-cache append (one token per sequence) us per call, 1 GPU",
        "value": round(us, 3), "unit": "us", "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "dtype": base.kv_dtype, "data": "synthetic",
        "config": {"workload": "%s: %s" % (args.config, _describe(args.config)),
                   "batch": base.batch, "num_kv_heads": base.num_kv_heads,
                   "layout": base.layout},
        "bytes_per_call": moved, "GBs": round(moved / us / 1e3, 2),
    }
    if before is not None:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        record["cpu_baseline"], record["parity"] = append_cpu_baseline(base, before, k, v)
    return record


def append_cpu_baseline(p, before, k, v, min_seconds=5.0):
    """The oracle's append of the same tokens to the cache as it was before
    the first call, timed on the host (whole step; the oracle returns updated
    copies of the pools, so copying them is part of its time), and the GPU's
    pools and scales after the timed calls compared with it byte for byte."""
    import numpy as np
    import oracle
    import torch
    kv_code = oracle.KV_BF16 if p.kv_dtype == "bf16" else oracle.KV_FP8_E4M3
    bits = lambda t: t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    kw = dict(kv_dtype=kv_code, layout=before["layout"], k_scale=before.get("k_scale"),
              v_scale=before.get("v_scale"))
    reps, dt = 0, 0.0
    while reps == 0 or dt < min_seconds:
        t0 = time.perf_counter()
        ref = oracle.kv_append(bits(k), bits(v), before["k_pool"], before["v_pool"],
                               before["block_table"], before["seq_lens"], **kw)
        dt += time.perf_counter() - t0
        reps += 1
    after = p.host_arrays()
    names = ["k_pool", "v_pool"] + (["k_scale", "v_scale"] if p.kv_dtype != "bf16" else [])
    compared = mismatched = 0
    for name, want in zip(names, ref):
        got = np.ascontiguousarray(after[name]).view(np.uint8).reshape(-1)
        want = np.ascontiguousarray(want).view(np.uint8).reshape(-1)
        compared += want.size
        mismatched += int(np.count_nonzero(got != want))
    return {
        "value": dt / reps * 1e6,
        "unit": "us",
        "cores": 1,
        "kind": "oracle",
        "sample": "the whole step (%d sequences x %d kv heads), %d calls in %.2f s"
                  % (p.batch, p.num_kv_heads, reps, dt),
        "cpu_model": _cpu_model(),
    }, {"bytes_compared": compared, "mismatched_bytes": mismatched,
        "bit_exact": mismatched == 0}


def bench_extend(args, dev):
    """Times K extend-attention launches: every sequence of the workload gets
    --new-tokens new tokens after its cached length; FLOPs are the causal
    count 4 * D * Hq * sum over new tokens of the keys they see."""
    import numpy as np
    import torch
    from paper_2512_22492_amd import binding, workloads
    cfg = dict(workloads.CONFIGS[args.config])
    seed = cfg.pop("seed")
    n = args.new_tokens
    prior = workloads.draw_lengths(np.random.default_rng(seed), cfg["batch"], cfg["lengths"])
    cfg["lengths"] = [int(x) + n for x in prior]
    p = workloads.make_problem(args.config + "+extend", seed=seed, device=dev,
                               layout=args.layout, **cfg)
    T = n * p.batch
    gen = torch.Generator(device=dev).manual_seed(seed + 1)
    q = torch.randn((T, p.num_q_heads, p.head_dim), generator=gen, device=dev).to(torch.bfloat16)
    q_start = torch.arange(0, T + 1, n, dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    if args.warmup is None:
        # launch until EXTEND_WARMUP_MS of back-to-back launches have passed:
        # under matrix load the clock settles only after tens of milliseconds
        # (per XCD from about 1.5 to 2.0 GHz over the first ~30 ms, with the
        # cycle count per launch unchanged)
        args.warmup = 0
        t_end = time.perf_counter() + EXTEND_WARMUP_MS / 1e3
        while args.warmup < 5 or time.perf_counter() < t_end:
            for _ in range(5):
                binding.extend_attention(p, q, q_start, n, out)
            args.warmup += 5
            torch.cuda.synchronize()
    else:
        for _ in range(args.warmup):
            binding.extend_attention(p, q, q_start, n, out)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        binding.extend_attention(p, q, q_start, n, out)
    torch.cuda.synchronize()
    s = (time.perf_counter() - t0) / args.steps
    visible = sum(int(L) * n + n * (n + 1) // 2 for L in prior)
    flops = 4.0 * p.head_dim * p.num_q_heads * visible
    tf = flops / s / 1e12
    record = {
        "metric": "extend (prefill) attention TFLOP/s, causal, 1 GPU",
        "value": round(tf, 2), "unit": "TFLOP/s", "higher_is_better": True,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(s * 1e3, 4),
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "%s cached prefixes + %d new tokens per sequence" % (args.config, n),
                   "batch": p.batch, "num_q_heads": p.num_q_heads,
                   "num_kv_heads": p.num_kv_heads, "new_tokens": T, "layout": args.layout,
                   "kv_dtype": p.kv_dtype},
        "roofline": {"bound": "mfma", "achieved": round(tf, 2), "peak": 2500.0,
                     "unit": "TFLOP/s", "frac": round(tf / 2500.0, 4)},
    }
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        record["cpu_baseline"], record["parity"] = extend_cpu_baseline(p, q, n, prior, out)
    return record


def extend_cpu_baseline(p, q, n, prior, gpu_out, min_seconds=10.0):
    """The oracle's extend attention timed on the host on the launch's first
    sequences (about 2e10 fp64 multiply-adds for bf16 pools, 2e9 for e4m3
    ones, whose elements the oracle decodes one by one; one sequence at least),
    repeated until about min_seconds of CPU work have been timed; its output
    also gives the GPU output's error statistics on those sequences."""
    import numpy as np
    import oracle
    import torch
    kv_code = oracle.KV_BF16 if p.kv_dtype == "bf16" else oracle.KV_FP8_E4M3
    h = p.host_arrays()
    visible = np.array([int(L) * n + n * (n + 1) // 2 for L in prior], dtype=np.float64)
    macs = visible * p.num_q_heads * p.head_dim * 2          # both products
    budget = 2e10 if p.kv_dtype == "bf16" else 2e9
    nseq = max(1, min(p.batch, int(np.searchsorted(np.cumsum(macs), budget, side="right"))))
    q_bits = q[:nseq * n].cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    q_start = np.arange(0, nseq * n + 1, n, dtype=np.int32)
    kw = dict(num_kv_heads=p.num_kv_heads, scale=p.scale, kv_dtype=kv_code,
              layout=h["layout"], k_scale=h.get("k_scale"), v_scale=h.get("v_scale"))
    with _host_oracle() as build:
        reps, dt, ref = 0, 0.0, None
        while reps == 0 or dt < min_seconds:
            t0 = time.perf_counter()
            ref = oracle.extend_attention(q_bits, q_start, h["k_pool"], h["v_pool"],
                                          h["block_table"][:nseq], h["seq_lens"][:nseq], **kw)
            dt += time.perf_counter() - t0
            reps += 1
        cores = oracle.max_threads()
        # M1, the weighted mean of |v| per output: the same attention over
        # the value pool with every sign bit cleared (bf16 bit 15, e4m3 bit 7)
        v_abs = h["v_pool"] & (np.uint16(0x7FFF) if h["v_pool"].dtype == np.uint16
                               else np.uint8(0x7F))
        m1 = oracle.extend_attention(q_bits, q_start, h["k_pool"], v_abs,
                                     h["block_table"][:nseq], h["seq_lens"][:nseq], **kw)
    got = gpu_out[:nseq * n].float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    flops = 4.0 * p.head_dim * p.num_q_heads * float(visible[:nseq].sum()) * reps
    parity = parity_stats(got, ref)
    # The kernel rounds each weight to bf16 before the value product (8
    # significant bits, relative error <= 2^-8); with the normaliser summing
    # the same rounded weights (bf16 pools) an output moves by at most
    # 2^-8 (1 + 2^-7) (M1 + |o|), with the unrounded ones (e4m3 pools) by
    # 2^-8 (1 + 2^-7) M1, on top of one bf16 ulp of the output plus 1e-6.
    # The decode kernels' one-ulp gate does not apply here.
    del parity["max_err_over_ulp_gate"]
    p_round = 2.0 ** -8 * (1.0 + 2.0 ** -7)
    extra = p_round * (np.abs(m1) + (np.abs(ref) if p.kv_dtype == "bf16" else 0.0))
    parity["max_err_over_weight_bound"] = round(float(
        (np.abs(got - ref) / (_bf16_ulp(ref) + 1e-6 + extra)).max()), 4)
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": "%d of %d sequences (%d new tokens each, every query head), fp64, %d passes "
                  "in %.2f s" % (nseq, p.batch, n, reps, dt),
        "build": build,
        "cpu_model": _cpu_model(),
    }, parity


# Qwen3-8B weight tensors of one decoder layer, [out, in] (bf16): q, k, v, o
# projections, gate, up, down, the two layer norms and the q/k norms.
QWEN3_8B_LAYER = [(4096, 4096), (1024, 4096), (1024, 4096), (4096, 4096), (12288, 4096),
                  (12288, 4096), (4096, 12288), (4096,), (4096,), (128,), (128,)]
QWEN3_8B_LAYERS = 36
QWEN3_8B_VOCAB = 151936


def qwen3_8b_shapes(shard=1):
    """Tensor shapes in layer order (embedding, 36 layers, final norm, lm head);
    shard > 1 gives one rank's row slice of every matrix (rollout TP)."""
    def cut(shape):
        return (shape[0] // shard,) + tuple(shape[1:]) if len(shape) == 2 else shape
    shapes = [cut((QWEN3_8B_VOCAB, 4096))]
    for _ in range(QWEN3_8B_LAYERS):
        shapes += [cut(s) for s in QWEN3_8B_LAYER]
    return shapes + [(4096,), cut((QWEN3_8B_VOCAB, 4096))]


def _weights(shapes, dev, seed):
    import torch
    gen = torch.Generator(device=dev).manual_seed(seed)
    return [torch.empty(s, dtype=torch.bfloat16, device=dev).normal_(generator=gen)
            for s in shapes]


def _time_launches(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def bench_pack(args, dev):
    """Layer-by-layer packing of the Qwen3-8B weights (bf16, 16.4 GB) through a
    1 GiB device transfer buffer: one step packs every chunk in turn.  HBM
    traffic is one read and one write of every weight byte."""
    import torch
    from paper_2512_22492_amd import binding
    tensors = _weights(qwen3_8b_shapes(), dev, 7)
    total = sum(t.numel() * 2 for t in tensors)
    cap = 1 << 30
    buf = torch.empty(cap, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    if args.pmc_calibrate:
        calibrate_counters(dev, stream)
    with binding.WeightSync(tensors, buf, align=256) as ws:
        def step():
            for c in range(ws.num_chunks):
                ws.pack(c, stream)
        s = _time_launches(step, args.steps, args.warmup)
        chunks = ws.num_chunks
        torch.cuda.synchronize()
        baseline = None
        if not args.no_cpu_baseline:
            # the buffer holds the last chunk of the last step
            print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
            baseline = weight_sync_cpu_baseline(tensors, buf.cpu().numpy(), chunks - 1, cap, 256)
    # plain device copy of one buffer's worth, for the achievable copy rate
    copy_s = None
    if not args.no_ceilings:
        src = torch.empty(cap, dtype=torch.uint8, device=dev)
        lib = bench_kernels()
        copy_s = _time_launches(lambda: lib.rl_bench_copy(buf.data_ptr(), src.data_ptr(), cap,
                                                          stream.cuda_stream), 10, 2)
    gbs = total / s / 1e9
    hbm = 2 * total / s / 1e9
    record = {
        "metric": "weight-sync pack GB/s of weights (layer by layer into a transfer buffer), 1 GPU",
        "value": round(gbs, 1), "unit": "GB/s", "higher_is_better": True,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(s * 1e3, 4),
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "Qwen3-8B weights, %d tensors, %.2f GB, 1 GiB buffer, %d chunks"
                               % (len(tensors), total / 1e9, chunks)},
        "roofline": {"bound": "hbm", "achieved": round(hbm, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(hbm / HBM_PEAK_GBS, 4),
                     "traffic": load_traffic(traffic_key(args), kernel_source_sha("pack")),
                     "bytes_per_launch": 2 * total // chunks},
        "plain_copy_GBs_rw": None if copy_s is None else round(2 * cap / copy_s / 1e9, 1),
    }
    if baseline is not None:
        record["cpu_baseline"], record["parity"] = baseline
    return record


def weight_sync_cpu_baseline(tensors, gpu_buffer, chunk, capacity, align, min_seconds=5.0):
    """The oracle's pack of one chunk (numpy, one thread) timed on the host,
    repeated until about min_seconds, and the GPU's buffer for that chunk
    compared with it byte for byte over every byte the chunk's pieces write."""
    import numpy as np
    import torch
    from oracle import weight_sync as ows
    sizes = [t.numel() * t.element_size() for t in tensors]
    pieces = ows.plan(sizes, capacity, align)
    used = sorted({t for t, c, _, _, _ in pieces if c == chunk})
    host = [np.empty(0, dtype=np.uint8)] * len(tensors)
    for i in used:
        host[i] = tensors[i].detach().contiguous().view(torch.uint8).reshape(-1).cpu().numpy()
    reps, dt = 0, 0.0
    while reps == 0 or dt < min_seconds:
        t0 = time.perf_counter()
        ref, written = ows.pack(host, pieces, chunk, capacity)
        dt += time.perf_counter() - t0
        reps += 1
    nbytes = int(written.sum())
    mismatches = int(np.count_nonzero(gpu_buffer[:capacity][written] != ref[written]))
    return {
        "value": nbytes * reps / dt / 1e9,
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": "chunk %d (%d bytes of %d tensors), numpy, %d passes in %.2f s"
                  % (chunk, nbytes, len(used), reps, dt),
        "cpu_model": _cpu_model(),
    }, {"bytes_compared": nbytes, "mismatched_bytes": mismatches, "bit_exact": mismatches == 0}


def bench_d2h(args, dev):
    """Checkpoint copy of one rank's shard (the Qwen3-8B weights cut 8 ways,
    2.05 GB) into pinned host memory with the pack kernel; the runtime's DMA
    copy of the same number of contiguous bytes is timed beside it."""
    import torch
    from paper_2512_22492_amd import binding
    tensors = _weights(qwen3_8b_shapes(shard=8), dev, 8)
    total = sum(t.numel() * 2 for t in tensors)
    cap = (total + 256 * len(tensors) + 4095) // 4096 * 4096
    host = torch.empty(cap, dtype=torch.uint8, pin_memory=True)
    stream = torch.cuda.current_stream()
    with binding.WeightSync(tensors, host, align=256) as ws:
        assert ws.num_chunks == 1
        s = _time_launches(lambda: ws.pack(0, stream), args.steps, args.warmup)
        torch.cuda.synchronize()
        baseline = None
        if not args.no_cpu_baseline:
            # before the runtime copy below overwrites the host buffer
            print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
            baseline = weight_sync_cpu_baseline(tensors, host.numpy(), 0, cap, 256)
    flat = torch.empty(total, dtype=torch.uint8, device=dev)
    dma_s = _time_launches(lambda: host[:total].copy_(flat, non_blocking=True), 5, 1)
    gbs = total / s / 1e9
    record = {
        "metric": "checkpoint GPU-to-host copy GB/s (pinned host memory), 1 GPU",
        "value": round(gbs, 2), "unit": "GB/s", "higher_is_better": True,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(s * 1e3, 3),
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "Qwen3-8B weights / 8 (one rank's shard), %d tensors, %.3f GB"
                               % (len(tensors), total / 1e9)},
        "roofline": {"bound": "host-link", "achieved": round(gbs, 2), "peak": PCIE5_X16_GBS,
                     "unit": "GB/s", "frac": round(gbs / PCIE5_X16_GBS, 4)},
        "dma_copy_GBs": round(total / dma_s / 1e9, 2),
    }
    if baseline is not None:
        record["cpu_baseline"], record["parity"] = baseline
    return record


def traffic_key(args):
    """Entry of the counter file for this workload and pool layout, or op."""
    if args.op == "pack":
        return "pack:qwen3_8b_weights"
    key = args.config if args.layout == "hnd" else args.config + ":" + args.layout
    return key + (":per-head" if args.per_head_units and args.layout != "hnd" else "")


def calibrate_counters(dev, stream):
    """One plain 16-byte-per-lane copy of COPY_CALIBRATION_BYTES, whose counter
    readings scale the op kernel's readings."""
    import torch
    src = torch.empty(COPY_CALIBRATION_BYTES, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    assert bench_kernels().rl_bench_copy(dst.data_ptr(), src.data_ptr(),
                                         COPY_CALIBRATION_BYTES, stream.cuda_stream) == 0
    torch.cuda.synchronize()


def _describe(name):
    from paper_2512_22492_amd import workloads
    return workloads.describe(name)


def main():
    args = parse_args()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], traffic_key(args), args.op)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(decode attention shards by sequence or kv head with no exchange; "
              "the per-GPU figure is the --gpus 1 line)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2512_22492_amd import binding, workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    print("bench: generating %s (%s)" % (args.config, workloads.describe(args.config)),
          file=sys.stderr, flush=True)
    if args.op == "extend":
        print(json.dumps(bench_extend(args, dev)), flush=True)
        return
    if args.warmup is None:
        args.warmup = 5
    if args.op == "pack":
        print(json.dumps(bench_pack(args, dev)), flush=True)
        return
    if args.op == "d2h":
        print(json.dumps(bench_d2h(args, dev)), flush=True)
        return
    base = workloads.make_config(args.config, device=dev, layout=args.layout)
    replicas = [base]
    for _ in range(1, max(1, args.replicas)):
        replicas.append(base.clone_pools())
    if args.op == "append":
        print(json.dumps(bench_append(args, base, torch.cuda.current_stream())), flush=True)
        return
    out = torch.empty_like(base.q)
    flags = binding.RL_DA_SCORES_ON_VALU if args.scores == "valu" else 0
    if args.per_head_units:
        flags |= binding.RL_DA_PER_HEAD_UNITS
    if args.pv == "valu":
        flags |= binding.RL_DA_PV_ON_VALU
    attn = binding.DecodeAttention.for_problem(base, flags=flags,
                                               split_tokens=args.split_tokens)
    split_tokens, num_splits = attn.split_info(base.max_pages)
    unit_heads = attn.unit_heads()
    stream = torch.cuda.current_stream()

    nev = args.steps
    ev_b = [torch.cuda.Event(enable_timing=True) for _ in range(nev)]
    ev_e = [torch.cuda.Event(enable_timing=True) for _ in range(nev)]
    for e in ev_b + ev_e:
        e.record(stream)          # materialises the underlying hipEvent_t
    torch.cuda.synchronize()

    if args.pmc_calibrate:
        calibrate_counters(dev, stream)

    for i in range(args.warmup):
        attn.run_problem(replicas[i % len(replicas)], out, stream)
    torch.cuda.synchronize()
    print("bench: warmup done, timing %d steps" % args.steps, file=sys.stderr, flush=True)

    # Timed region: exactly K steps, nothing else enqueued; one event pair on
    # the stream around the K steps gives their GPU time.
    pass_b = torch.cuda.Event(enable_timing=True)
    pass_e = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    pass_b.record(stream)
    for i in range(args.steps):
        attn.run_problem(replicas[i % len(replicas)], out, stream)
    pass_e.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    gpu_ms_per_step = pass_b.elapsed_time(pass_e) / args.steps

    # Second timed pass of K steps whose split-kernel launches carry HIP
    # events attached to the launch itself (hipExtLaunchKernel): each pair
    # holds that kernel's own start and end.  Its wall time bounds the sum of
    # the kernel times from above.
    split_ms = None
    pass2_ms = None
    if not args.no_kernel_events:
        t2 = time.perf_counter()
        for i in range(args.steps):
            binding.rl_decode_attn_set_timing_events(attn.handle, ev_b[i].cuda_event,
                                                     ev_e[i].cuda_event)
            attn.run_problem(replicas[i % len(replicas)], out, stream)
        torch.cuda.synchronize()
        pass2_ms = (time.perf_counter() - t2) * 1e3 / args.steps
        binding.rl_decode_attn_set_timing_events(attn.handle, None, None)
        split_ms = np.array([b.elapsed_time(e) for b, e in zip(ev_b, ev_e)])

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    alg_bytes, kv_bytes = algorithmic_bytes(base)
    value = kv_bytes / (ms_per_step / 1e3) / 1e9
    seed = workloads.CONFIGS[args.config]["seed"]
    record = {
        "metric": "decode-attention KV-read GB/s (fraction of HBM peak) + query-tokens/s, 1 GPU",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": base.kv_dtype if base.kv_dtype == "bf16" else "fp8_e4m3",
        "data": "synthetic",
        "config": {
            "workload": "%s: %s" % (args.config, workloads.describe(args.config)),
            "seed": seed,
            "batch": base.batch, "num_q_heads": base.num_q_heads,
            "num_kv_heads": base.num_kv_heads, "head_dim": base.head_dim,
            "page_size": base.page_size, "seq_len_mean": float(base.lengths().mean()),
            "split_tokens": split_tokens, "num_splits": num_splits,
            "scores": args.scores,
            "pv": "valu" if args.scores == "valu" or args.pv == "valu" or unit_heads > 1
                  else "mfma",
            "replicas": len(replicas), "layout": base.layout,
            "units": "per-head" if unit_heads == 1
                     else "head-parallel (%d kv heads)" % unit_heads,
        },
        "query_tokens_per_s": round(base.batch / (ms_per_step / 1e3), 1),
        "kv_bytes_per_step": kv_bytes,
        "hbm_frac": round(value / HBM_PEAK_GBS, 4),
    }
    if not args.no_input_digests:
        record["config"]["input_sha256_16"] = input_digests(base)
    if split_ms is not None:
        kernel_avg = float(split_ms.mean())
        # every kernel runs inside its step
        assert kernel_avg <= pass2_ms * (1 + 1e-6), (kernel_avg, pass2_ms)
        if num_splits == 1:
            # a step is the split kernel alone: its time is the timed pass's
            # GPU time per step (back-to-back launches), which cannot exceed
            # the step's wall time
            avg, source = gpu_ms_per_step, "event pair around the K timed steps (one kernel per step)"
        elif kernel_avg <= ms_per_step:
            avg, source = kernel_avg, "events attached to each split-kernel launch"
        else:
            # a launch-attached start event can fire while the launch still
            # waits in the queue (slow launches, e.g. under a profiler): take
            # the whole step's GPU time (split and merge kernels) instead
            avg, source = gpu_ms_per_step, ("event pair around the K timed steps (split + merge "
                                            "kernels; launch-attached events exceeded the step)")
        assert avg <= ms_per_step, (avg, ms_per_step)
        achieved = alg_bytes / (avg / 1e3) / 1e9
        record["roofline"] = {
            "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": load_traffic(traffic_key(args), kernel_source_sha()),
            "kernel": "split-K decode kernel", "avg_us": round(avg * 1e3, 2),
            "avg_us_source": source,
            "kernel_events_avg_us": round(kernel_avg * 1e3, 2),
            "kernel_events_min_us": round(float(split_ms.min()) * 1e3, 2),
            "kernel_events_p10_p50_p90_us": [round(float(x) * 1e3, 2)
                                             for x in np.percentile(split_ms, [10, 50, 90])],
            "bytes_per_launch": alg_bytes,
        }
    attn.close()
    if not args.no_ceilings:
        print("bench: measuring read ceilings", file=sys.stderr, flush=True)
        ceil = read_ceilings(base, stream)
        record["read_ceiling"] = ceil
        if "roofline" in record:
            record["roofline"]["frac_of_stream_read"] = round(
                record["roofline"]["achieved"] / ceil["stream_read_GBs"], 4)
            record["roofline"]["frac_of_page_read"] = round(
                record["roofline"]["achieved"] / ceil["page_read_GBs"], 4)
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        # the output of the last timed step, from the first replica's inputs
        attn = binding.DecodeAttention.for_problem(base, flags=flags,
                                                   split_tokens=args.split_tokens)
        attn.run_problem(base, out, stream)
        torch.cuda.synchronize()
        attn.close()
        record["cpu_baseline"], record["parity"] = cpu_baseline(base, out)
        del record["cpu_baseline"]["seconds"]
    print(json.dumps(record), flush=True)

if __name__ == "__main__":
    main()
