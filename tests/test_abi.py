"""The C interface: every declared symbol is exported, and host-side
validation answers with the documented status codes (CPU only: create()
validates its configuration before touching the HIP runtime)."""
import ctypes
import glob
import os
import re

import pytest

from paper_2512_22492_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for path in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(path).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"\b(rl_\w+)\s*\(", text)
    return names


def test_every_declared_function_is_exported():
    lib = B.load_library()
    names = declared_functions()
    assert set(names) == set(B.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_library_needs_no_torch():
    # The boundary is plain C over the HIP runtime: no torch/c10 dependency.
    import subprocess
    out = subprocess.run(["readelf", "-d", B.library_path()], stdout=subprocess.PIPE,
                         universal_newlines=True, check=True).stdout
    needed = re.findall(r"\(NEEDED\)\s+Shared library: \[(.+?)\]", out)
    assert "libamdhip64.so.7" in needed
    assert not [n for n in needed if "torch" in n or "c10" in n], needed


def test_config_struct_matches_the_header(tmp_path):
    """ctypes' rl_da_config has the C struct's size and field offsets."""
    import subprocess
    fields = [f for f, _ in B.rl_da_config._fields_]
    src = tmp_path / "offsets.c"
    src.write_text(
        "#include <stddef.h>\n#include <stdio.h>\n#include \"rl_decode_attn.h\"\n"
        "int main(void) {\n  printf(\"%zu\", sizeof(rl_da_config));\n" +
        "".join('  printf(" %%zu", offsetof(rl_da_config, %s));\n' % f for f in fields) +
        "  return 0;\n}\n")
    exe = tmp_path / "offsets"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = [int(x) for x in subprocess.run([str(exe)], stdout=subprocess.PIPE,
                                          check=True).stdout.split()]
    want = [ctypes.sizeof(B.rl_da_config)] + [getattr(B.rl_da_config, f).offset
                                              for f in fields]
    assert got == want


def test_status_strings():
    assert B.rl_da_status_string(B.RL_DA_OK) == "ok"
    for s in (1, 2, 3, 4, 5):
        assert B.rl_da_status_string(s) not in ("ok", "unknown status")
    assert B.rl_da_status_string(99) == "unknown status"


def cfg(**kw):
    base = dict(num_q_heads=32, num_kv_heads=8, max_batch=64, max_pages_per_seq=256)
    base.update(kw)
    hq, hkv, mb, mp = (base.pop(k) for k in ("num_q_heads", "num_kv_heads", "max_batch",
                                             "max_pages_per_seq"))
    return B.make_config(hq, hkv, mb, mp, **base)


def test_workspace_size_formula():
    rc, n = B.rl_decode_attn_workspace_size(cfg())
    assert rc == B.RL_DA_OK
    splits = 256 // 256                      # default 4096-token splits of 16-token pages
    rows = 64 * 32 * splits
    expect = (rows * 128 * 4 + rows * 2 * 4 + 255) // 256 * 256 + 256
    assert n == expect
    rc, n2 = B.rl_decode_attn_workspace_size(cfg(split_tokens=512))
    assert rc == B.RL_DA_OK and n2 > n
    # a small handle gets a shorter default split: 2 x 1 x 16 pages -> 512 tokens
    rc, n3 = B.rl_decode_attn_workspace_size(cfg(max_batch=2, num_q_heads=4, num_kv_heads=1,
                                                 max_pages_per_seq=16))
    rows3 = 2 * 4 * 1
    assert rc == B.RL_DA_OK
    assert n3 == (rows3 * 128 * 4 + rows3 * 2 * 4 + 255) // 256 * 256 + 256


def test_token_major_pools_default_split():
    """Token-major pools with several kv heads per work-group use one
    work-group per (sequence, split, eight kv heads), so the default split
    that still gives 256 work-groups is 1024 tokens here; the workspace
    follows."""
    rc, n = B.rl_decode_attn_workspace_size(cfg(layout=B.RL_DA_LAYOUT_NHD))
    rows = 64 * 32 * 4                       # 256 pages -> four 1024-token splits
    assert rc == B.RL_DA_OK
    assert n == (rows * 128 * 4 + rows * 2 * 4 + 255) // 256 * 256 + 256
    # the VALU score path keeps the four-wavefront units and their 4096 default
    rc, n1 = B.rl_decode_attn_workspace_size(cfg(layout=B.RL_DA_LAYOUT_NHD,
                                                 flags=B.RL_DA_SCORES_ON_VALU))
    assert rc == B.RL_DA_OK and n1 == B.rl_decode_attn_workspace_size(cfg())[1]


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=0), B.RL_DA_ERR_INVALID_ARG),
    (dict(num_kv_heads=-1), B.RL_DA_ERR_INVALID_ARG),
    (dict(num_q_heads=30, num_kv_heads=8), B.RL_DA_ERR_INVALID_ARG),
    (dict(max_batch=0), B.RL_DA_ERR_INVALID_ARG),
    (dict(max_pages_per_seq=0), B.RL_DA_ERR_INVALID_ARG),
    (dict(split_tokens=-16), B.RL_DA_ERR_INVALID_ARG),
    (dict(flags=0x80), B.RL_DA_ERR_INVALID_ARG),
    (dict(flags=0x10), B.RL_DA_ERR_INVALID_ARG),
    (dict(kv_dtype=7), B.RL_DA_ERR_INVALID_ARG),
    (dict(layout=3), B.RL_DA_ERR_INVALID_ARG),
    (dict(head_dim=64), B.RL_DA_ERR_UNSUPPORTED),
    (dict(page_size=32), B.RL_DA_ERR_UNSUPPORTED),
    (dict(num_q_heads=24, num_kv_heads=8), B.RL_DA_ERR_UNSUPPORTED),   # G = 3
    (dict(num_q_heads=256, num_kv_heads=8), B.RL_DA_ERR_UNSUPPORTED),  # G = 32
    (dict(num_q_heads=128, num_kv_heads=8, flags=B.RL_DA_SCORES_ON_VALU),
     B.RL_DA_ERR_UNSUPPORTED),                                          # G = 16, VALU scores
    (dict(num_q_heads=128, num_kv_heads=8, flags=B.RL_DA_PV_ON_VALU),
     B.RL_DA_ERR_UNSUPPORTED),                                          # G = 16, VALU values
    (dict(split_tokens=24), B.RL_DA_ERR_UNSUPPORTED),
    (dict(kv_dtype=B.RL_DA_KV_FP8_E4M3, flags=B.RL_DA_SCORES_ON_VALU), B.RL_DA_ERR_UNSUPPORTED),
    (dict(split_tokens=4112), B.RL_DA_ERR_UNSUPPORTED),
    (dict(layout=B.RL_DA_LAYOUT_NHD, split_tokens=4112), B.RL_DA_ERR_UNSUPPORTED),
])
def test_create_rejects_bad_config_without_gpu(kw, status):
    c = cfg(**kw)
    rc, h = B.rl_decode_attn_create(c)
    assert rc == status and h is None
    rc2, _ = B.rl_decode_attn_workspace_size(c)
    assert rc2 == status


def test_null_arguments():
    lib = B.load_library()
    h = ctypes.c_void_p()
    assert lib.rl_decode_attn_create(None, ctypes.byref(h)) == B.RL_DA_ERR_INVALID_ARG
    assert lib.rl_decode_attn_create(ctypes.byref(cfg()), None) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_decode_attn_destroy(None) == B.RL_DA_OK
    assert lib.rl_decode_attn_run(None, 1, 1, 1, None, None, 1, 1, 1, 1, 1, 1.0, 1,
                                  None) == B.RL_DA_ERR_INVALID_ARG
    v = ctypes.c_int32()
    assert lib.rl_decode_attn_check_error(None, ctypes.byref(v)) == B.RL_DA_ERR_INVALID_ARG
    assert lib.rl_decode_attn_workspace_size(None, None) == B.RL_DA_ERR_INVALID_ARG


def test_noalloc_entry_point_host_checks():
    """The allocation-free entry point rejects, before touching the device:
    no configuration, a configuration create() rejects, checked mode, and a
    step whose workspace exceeds its fixed scratch."""
    lib = B.load_library()
    args = (1, 1, 1, None, None, 1, 1, 1, 1, 1, 1.0, 1, None)
    assert lib.rl_decode_attn_run_noalloc(None, *args) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_decode_attn_run_noalloc(cfg(head_dim=64), *args) == B.RL_DA_ERR_UNSUPPORTED
    assert B.rl_decode_attn_run_noalloc(cfg(max_batch=0), *args) == B.RL_DA_ERR_INVALID_ARG
    assert B.rl_decode_attn_run_noalloc(cfg(flags=B.RL_DA_CHECKED), *args) == \
        B.RL_DA_ERR_UNSUPPORTED
    big = cfg(max_batch=1024, max_pages_per_seq=4096, split_tokens=512)
    rc, need = B.rl_decode_attn_workspace_size(big)
    assert rc == B.RL_DA_OK and need > B.RL_DA_NOALLOC_SCRATCH_BYTES
    assert B.rl_decode_attn_run_noalloc(big, *args) == B.RL_DA_ERR_SCRATCH_TOO_SMALL


def test_extend_host_checks_without_gpu():
    """rl_extend_attn refuses bad requests before touching the device: null
    or misaligned pointers, e4m3 scales given for bf16 pools, shapes it has
    no kernel for, and pages of 2 GiB or more (its kernels address within a
    page with 32-bit offsets).  The pointers are never dereferenced."""
    fake = 1 << 20

    def call(**kw):
        args = dict(q=fake, q_start=fake, max_q_per_seq=4, k_pool=fake, v_pool=fake,
                    k_scale=None, v_scale=None, num_pages=16, block_table=fake, max_pages=4,
                    seq_lens=fake, batch=2, num_q_heads=32, num_kv_heads=8, out=fake)
        args.update(kw)
        return B.rl_extend_attn(**args)

    assert call(q=None) == B.RL_DA_ERR_INVALID_ARG
    assert call(out=fake + 8) == B.RL_DA_ERR_INVALID_ARG             # misaligned
    # nothing to do: success without touching the device
    assert call(batch=0) == B.RL_DA_OK
    assert call(max_q_per_seq=0) == B.RL_DA_OK
    assert call(batch=-1) == B.RL_DA_ERR_INVALID_ARG
    assert call(max_q_per_seq=-1) == B.RL_DA_ERR_INVALID_ARG
    assert call(scale=float("nan")) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_scale=fake, v_scale=fake) == B.RL_DA_ERR_INVALID_ARG
    assert call(layout=3) == B.RL_DA_ERR_INVALID_ARG
    assert call(head_dim=64) == B.RL_DA_ERR_UNSUPPORTED
    assert call(num_q_heads=24, num_kv_heads=8) == B.RL_DA_ERR_UNSUPPORTED   # G = 3
    assert call(num_q_heads=256, num_kv_heads=8) == B.RL_DA_ERR_UNSUPPORTED  # G = 32
    # 2^19 kv heads: 2 GiB per bf16 page in every layout
    for layout in (B.RL_DA_LAYOUT_HND, B.RL_DA_LAYOUT_NHD):
        assert call(num_q_heads=1 << 19, num_kv_heads=1 << 19,
                    layout=layout) == B.RL_DA_ERR_UNSUPPORTED


def test_kv_append_host_checks_without_gpu():
    """rl_kv_append refuses bad requests before touching the device (null or
    misaligned pointers, scales given exactly for e4m3 pools, shapes it has no
    kernel for) and succeeds on an empty batch without launching anything.
    The pointers are never dereferenced."""
    fake = 1 << 20

    def call(**kw):
        args = dict(k_new=fake, v_new=fake, k_pool=fake, v_pool=fake, k_scale=None,
                    v_scale=None, num_pages=16, block_table=fake, max_pages=4, seq_lens=fake,
                    batch=2, num_kv_heads=8)
        args.update(kw)
        return B.rl_kv_append(**args)

    assert call(batch=0) == B.RL_DA_OK
    assert call(batch=-1) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_new=None) == B.RL_DA_ERR_INVALID_ARG
    assert call(seq_lens=None) == B.RL_DA_ERR_INVALID_ARG
    assert call(v_pool=fake + 8) == B.RL_DA_ERR_INVALID_ARG            # misaligned
    assert call(num_kv_heads=0) == B.RL_DA_ERR_INVALID_ARG
    assert call(max_pages=0) == B.RL_DA_ERR_INVALID_ARG
    assert call(k_scale=fake, v_scale=fake) == B.RL_DA_ERR_INVALID_ARG   # scales on bf16
    assert call(kv_dtype=B.RL_DA_KV_FP8_E4M3) == B.RL_DA_ERR_INVALID_ARG  # e4m3 without
    assert call(kv_dtype=7) == B.RL_DA_ERR_INVALID_ARG
    assert call(layout=3) == B.RL_DA_ERR_INVALID_ARG
    assert call(head_dim=64) == B.RL_DA_ERR_UNSUPPORTED
    assert call(page_size=32) == B.RL_DA_ERR_UNSUPPORTED
