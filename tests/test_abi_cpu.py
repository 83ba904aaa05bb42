"""The C ABI without a GPU: libkvio.so loads, exports every function that
include/kvio.h declares, and host-side validation rejects bad arguments
before any device work."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "kvio.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvio_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("kvio_load", "kvio_offload", "kvio_load_layer", "kvio_pool_create", "kvio_pool_destroy",
                 "kvio_check", "kvio_strerror", "kvio_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol():
    import paper_2508_18572_amd as kv
    lib = ctypes.CDLL(kv.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(kv.EXPORTS) == declared_functions()


def test_strerror_and_last_error():
    import paper_2508_18572_amd as kv
    for code in (kv.KVIO_OK, kv.KVIO_EINVAL, kv.KVIO_ERANGE, kv.KVIO_EALIGN, kv.KVIO_ENOTMAPPED,
                 kv.KVIO_EHIP, kv.KVIO_ENOMEM):
        assert kv.kvio_strerror(code).startswith("KVIO_")
    assert kv.kvio_strerror(-99) == "unknown kvio_status"


def test_host_side_validation_without_device():
    import paper_2508_18572_amd as kv
    with pytest.raises(kv.KvioError) as e:                      # null layer pointers
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4096, [0, 0], [0, 0])
    assert e.value.status == kv.KVIO_EINVAL and "layer 0 is null" in e.value.detail
    with pytest.raises(kv.KvioError) as e:                      # R = 3 * 5 * 2 = 30 B
        kv.kvio_pool_create(2, 3, 5, 2, 16, 4096, [16, 16], [16, 16])
    assert e.value.status == kv.KVIO_EALIGN
    with pytest.raises(kv.KvioError) as e:                      # S % P != 0
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4100, [16, 16], [16, 16])
    assert e.value.status == kv.KVIO_EINVAL
    with pytest.raises(kv.KvioError) as e:                      # bad launch shape
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16], load_launch=kv.launch(threads=96))
    assert e.value.status == kv.KVIO_EINVAL
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16], offload_launch=kv.launch(tile_kib=5))
    assert e.value.status == kv.KVIO_EINVAL
    staged = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    with pytest.raises(kv.KvioError) as e:                      # staged: not for page-first chunks
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16], load_launch=staged,
                            host_layout=kv.KVIO_HOST_PAGE_FIRST)
    assert e.value.status == kv.KVIO_EINVAL and "token-major" in e.value.detail
    with pytest.raises(kv.KvioError) as e:                      # staging below one page of K and V rows
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16], offload_launch=staged,
                            staging_bytes=2 * 16 * 512 - 16)
    assert e.value.status == kv.KVIO_EINVAL and "staging_bytes" in e.value.detail
    with pytest.raises(kv.KvioError) as e:                      # unknown flag bit
        kv.kvio_pool_create(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16], load_launch=kv.launch(flags=0x80))
    assert e.value.status == kv.KVIO_EINVAL
    with pytest.raises(kv.KvioError) as e:                      # null pool handle
        kv.kvio_load(0, [], 0, 1)
    assert e.value.status == kv.KVIO_EINVAL
    kv.kvio_pool_destroy(0)                                     # NULL is accepted
    kv.kvio_memcpy(0, 0, 0)                                     # zero bytes: no-op
    kv.kvio_kernel_memcpy(0, 0, 0)
    for dst, src, n, what in ((0, 4096, 16, "null"), (4096, 4096, 24, "multiple of 16"),
                              (4104, 4096, 16, "aligned"), (4096, 4100, 32, "aligned")):
        with pytest.raises(kv.KvioError) as e:                  # checked before anything is enqueued
            kv.kvio_kernel_memcpy(dst, src, n)
        assert e.value.status == kv.KVIO_EINVAL and what in e.value.detail
    lib = kv.kvio._lib                                          # stream arguments, checked before HIP
    out = ctypes.c_void_p()
    zero = (ctypes.c_uint32 * 2)()
    assert lib.kvio_stream_create(zero, 2, ctypes.byref(out)) == kv.KVIO_EINVAL
    assert "empty CU mask" in kv.kvio_last_error()
    assert lib.kvio_stream_create(None, 1, ctypes.byref(out)) == kv.KVIO_EINVAL
    assert lib.kvio_stream_create(None, 0, None) == kv.KVIO_EINVAL
    assert lib.kvio_stream_destroy(None) == kv.KVIO_EINVAL


def test_noalloc_argument_checks_without_device():
    """kvio_load_noalloc refuses what its static table cannot hold before it
    touches the device."""
    import paper_2508_18572_amd as kv
    desc, keep = kv.pool_desc(kv.KVIO_NOALLOC_MAX_LAYERS + 1, 4, 64, 2, 16, 4096, [16] * 129, [16] * 129)
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(desc, [], 0, 1)
    assert e.value.status == kv.KVIO_EINVAL and "layers exceed" in e.value.detail
    desc, keep = kv.pool_desc(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16],
                              load_launch=kv.launch(flags=kv.KVIO_LAUNCH_STAGED))
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(desc, [], 0, 2)
    assert e.value.status == kv.KVIO_EINVAL and "staged" in e.value.detail
    desc, keep = kv.pool_desc(2, 3, 5, 2, 16, 4096, [16, 16], [16, 16])     # R = 30 B
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(desc, [], 0, 2)
    assert e.value.status == kv.KVIO_EALIGN
    desc, keep = kv.pool_desc(2, 4, 64, 2, 16, 4096, [16, 16], [16, 16])
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(desc, [(0, 0, 0, 0)] * (kv.KVIO_MAX_SPANS_PER_LAUNCH + 1), 0, 2)
    assert e.value.status == kv.KVIO_EINVAL


def test_package_refuses_to_import_without_the_library(tmp_path):
    """No fallback: without libkvio.so the package raises at import."""
    import shutil
    import subprocess
    import sys
    pkg = os.path.join(ROOT, "paper_2508_18572_amd")
    shutil.copytree(pkg, tmp_path / "paper_2508_18572_amd",
                    ignore=lambda d, names: [n for n in names if n.endswith(".so") or n == "__pycache__"])
    r = subprocess.run([sys.executable, "-c", "import paper_2508_18572_amd"], cwd=tmp_path,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "is not built" in r.stderr


def test_python_constants_match_the_header():
    import paper_2508_18572_amd.kvio as K
    text = open(os.path.join(ROOT, "include", "kvio.h")).read()
    consts = {m.group(1): int(m.group(2), 0)
              for m in re.finditer(r"#define (KVIO_[A-Z0-9_]+) (0x[0-9a-fA-F]+|-?\d+)\b", text)}
    consts.update({m.group(1): int(m.group(2))
                   for m in re.finditer(r"\b(KVIO_E[A-Z]+|KVIO_OK) = (-?\d+)", text)})
    assert len(consts) >= 19          # 8 status codes and 11 #defines
    for name, value in consts.items():
        assert getattr(K, name) == value, name


STRUCTS = {
    "kvio_launch": ["workgroups", "threads", "tile_kib", "flags"],
    "kvio_pool_desc": ["num_layers", "num_kv_heads", "head_dim", "elem_bytes", "page_size", "host_layout",
                       "num_slots", "k_layers", "v_layers", "load_launch", "offload_launch", "staging_bytes"],
    "kvio_span": ["host", "host_tokens", "num_tokens", "page_idx"],
    "kvio_request": ["load_tokens", "compute_tokens", "context", "transient_matches"],
    "kvio_batch_policy": ["max_tokens", "max_requests", "reserved", "loading_bound_ratio", "delay_hit_threshold"],
    "kvio_disk_store": ["fd", "disk_layout", "num_disk_pages", "num_layers", "page_size", "row_bytes"],
}


def test_ctypes_structs_match_the_c_layout(tmp_path):
    """Every struct the binding passes across the ABI has the size and field
    offsets gcc gives the header's declaration."""
    import subprocess
    import paper_2508_18572_amd.kvio as K
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "kvio.h"', "int main(void) {"]
    for st, fields in STRUCTS.items():
        lines.append(f'    printf("{st} size %zu\\n", sizeof({st}));')
        for f in fields:
            lines.append(f'    printf("{st} {f} %zu\\n", offsetof({st}, {f}));')
    lines += ["    return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = str(tmp_path / "layout")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), str(src), "-o", exe],
                   check=True)
    out = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split("\n")
    c = {(a, b): int(v) for a, b, v in (ln.split() for ln in out if ln)}
    for st, fields in STRUCTS.items():
        cls = getattr(K, st)
        assert [f[0] for f in cls._fields_] == fields, st
        assert ctypes.sizeof(cls) == c[(st, "size")], st
        for f in fields:
            assert getattr(cls, f).offset == c[(st, f)], (st, f)
