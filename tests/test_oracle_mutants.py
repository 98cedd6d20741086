"""The oracle's pins must catch plausible mistakes (CPU only).

Each case below plants one slip in a private copy of the oracle's C source,
builds it, and runs the pin suites (attention, append, codecs) against that
build in a fresh process.  The suite must fail for every mutant and pass for the
unmodified source built the same way.
"""
import concurrent.futures
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "decode_attn_oracle.c")

# (name, exact text in the source, replacement)
MUTANTS = [
    ("dropped scale", "scores[t] = p->scale * dot;", "scores[t] = dot;"),
    ("flipped score sign", "scores[t] = p->scale * dot;",
     "scores[t] = -p->scale * dot;"),
    ("interleaved head grouping", "attend_prefix(p, qrow, b, h / G, L, scores, dst);",
     "attend_prefix(p, qrow, b, h % p->num_kv_heads, L, scores, dst);"),
    ("query row of the kv head",
     "((int64_t)b * p->num_q_heads + h) * p->head_dim;",
     "((int64_t)b * p->num_q_heads + h / G) * p->head_dim;"),
    ("slot off by one", "const int slot = t % p->page_size;\n        double dot",
     "const int slot = (t + 1) % p->page_size;\n        double dot"),
    ("every token from logical page 0",
     "const int64_t page = pages[t / p->page_size];\n        const int slot = t % p->page_size;\n        const double w",
     "const int64_t page = pages[0];\n        const int slot = t % p->page_size;\n        const double w"),
    ("token-major pool layout",
     "return ((page * num_kv_heads + kvh) * page_size + slot)",
     "return ((page * page_size + slot) * num_kv_heads + kvh)"),
    ("NHD pools read head-major",
     "return ((page * page_size + slot) * num_kv_heads + kvh)",
     "return ((page * num_kv_heads + kvh) * page_size + slot)"),
    ("no max subtraction", "scores[t] = exp(scores[t] - smax);",
     "scores[t] = exp(scores[t]);"),
    ("no normalisation", "const double w = scores[t] / z;",
     "const double w = scores[t];"),
    ("last token dropped from values",
     "for (int t = 0; t < visible; ++t) {\n        const int64_t page = pages[t / p->page_size];\n        const int slot = t % p->page_size;\n        const double w",
     "for (int t = 0; t < visible - 1; ++t) {\n        const int64_t page = pages[t / p->page_size];\n        const int slot = t % p->page_size;\n        const double w"),
    ("e4m3 exponent bias 8", "mag = ldexp(1.0 + (double)m / 8.0, e - 7);",
     "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    ("e4m3 subnormal scale", "mag = ldexp((double)m / 8.0, -6);",
     "mag = ldexp((double)m / 8.0, -7);"),
    ("values scaled by the key scale",
     "dst[d] += w * pool_element(p, p->v_pool, p->v_scale,",
     "dst[d] += w * pool_element(p, p->v_pool, p->k_scale,"),
    ("bf16 read as low half", "uint32_t u = (uint32_t)bits << 16;",
     "uint32_t u = (uint32_t)bits << 15;"),
    ("append to the next slot", "codes[ELEM(slot, d)] = rl_oracle_e4m3_encode(",
     "codes[ELEM((slot + 1) % P, d)] = rl_oracle_e4m3_encode("),
    ("bf16 append to the next slot", "dst[ELEM(slot, d)] = src[d];",
     "dst[ELEM((slot + 1) % P, d)] = src[d];"),
    ("append scale never grows", "s_new = wanted > s_old ? wanted : s_old;",
     "s_new = s_old;"),
    ("append rescale ratio inverted", "const float ratio = s_old / s_new;",
     "const float ratio = s_new / s_old;"),
    ("append reads kv head 0", "((int64_t)b * H + kvh) * D;", "((int64_t)b * H) * D;"),
    ("encoder ties away from zero", "double q = rint((a / ldexp(1.0, e) - 1.0) * 8.0);",
     "double q = round((a / ldexp(1.0, e) - 1.0) * 8.0);"),
    ("encoder subnormal step", "const double steps = rint(a * 512.0);",
     "const double steps = rint(a * 256.0);"),
    ("extend sees its own next token", "const int visible = L - n_new + i + 1;",
     "const int visible = L - n_new + i + 2 <= L ? L - n_new + i + 2 : L;"),
    ("extend without causal mask", "const int visible = L - n_new + i + 1;",
     "const int visible = L;"),
    ("extend query row of the first new token",
     "(const uint16_t*)p->q + (row * p->num_q_heads + h) * p->head_dim;",
     "(const uint16_t*)p->q + ((int64_t)q_start[b] * p->num_q_heads + h) * p->head_dim;"),
    ("extend kv head of the query head",
     "attend_prefix(p, qrow, b, h / G, visible, scores, dst);",
     "attend_prefix(p, qrow, b, h % p->num_kv_heads, visible, scores, dst);"),
]


def _build(src_text, workdir, name):
    c_path = os.path.join(workdir, name + ".c")
    so_path = os.path.join(workdir, name + ".so")
    with open(c_path, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
                    "-fPIC", "-shared", "-I", os.path.join(ROOT, "oracle"),
                    c_path, "-o", so_path, "-lm"], check=True)
    return so_path


PIN_FILES = ["test_oracle.py", "test_oracle_append.py", "test_oracle_extend.py",
             "test_codecs.py"]


def _run_pins(so_path):
    env = dict(os.environ, RL_ORACLE_LIB=so_path, OMP_NUM_THREADS="2")
    r = subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider"] +
        [os.path.join(ROOT, "tests", f) for f in PIN_FILES],
        cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
        timeout=600)
    return r.returncode, r.stdout.decode(errors="replace")[-2000:]


def test_pins_catch_every_mutant():
    with open(SRC) as f:
        source = f.read()
    with tempfile.TemporaryDirectory() as work:
        jobs = {"unmodified": _build(source, work, "control")}
        for i, (name, old, new) in enumerate(MUTANTS):
            assert source.count(old) == 1, "mutation site not unique: " + name
            jobs[name] = _build(source.replace(old, new), work, "m%d" % i)
        with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
            results = dict(zip(jobs, ex.map(_run_pins, jobs.values())))
    rc, log = results.pop("unmodified")
    assert rc == 0, "unmodified oracle failed its pins:\n" + log
    survivors = [name for name, (rc, _) in results.items() if rc == 0]
    assert not survivors, "mutants not caught by any pin: %s" % survivors
