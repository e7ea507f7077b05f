"""C ABI checks that need no GPU: the library loads, exports every function
the public headers declare, and answers layout queries."""
import ctypes
import glob
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"\b(pb_[a-z0-9_]+)\s*\(", text):
            names.add(m.group(1))
    return sorted(names)


def test_headers_declare_the_boundary():
    names = _declared()
    for required in ("pb_model_create", "pb_stream_layers", "pb_attach_lora",
                     "pb_prefill_first_token", "pb_destroy", "pb_last_error"):
        assert required in names


def test_headers_are_plain_c(tmp_path):
    """The boundary is a C ABI: both headers compile as strict C99 (and as
    C++), and every declared function can be named from C."""
    import shutil
    import subprocess

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "boundary.c"
    refs = "\n".join("    (void (*)(void))%s," % n for n in _declared())
    src.write_text('#include "pipeboost.h"\n#include "pipeboost_ops.h"\n'
                   "void (*boundary_functions[])(void) = {\n%s\n};\n" % refs)
    inc = os.path.join(ROOT, "include")
    for lang in (["-std=c99"], ["-x", "c++", "-std=c++11"]):
        r = subprocess.run([cc] + lang + ["-Wall", "-Wextra", "-pedantic", "-Werror",
                                          "-c", "-I" + inc, str(src), "-o", str(tmp_path / "b.o")],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


@pytest.mark.parametrize("name", _declared())
def test_library_exports_declared_symbol(name):
    from paper_2503_17707_amd import binding as pb

    assert hasattr(pb.lib(), name)


def test_layout_queries():
    from paper_2503_17707_amd import binding as pb

    w = synth.WORKLOADS["opt-1.3b"]
    cfg = pb.make_config(w)
    L = pb.lib()
    lb = L.pb_layer_bytes(ctypes.byref(cfg))
    d, f = w.d_model, w.d_ffn
    assert lb >= 2 * w.layer_params()
    assert lb - 2 * w.layer_params() < 4096  # only alignment padding
    off_q, n_q = pb.layer_tensor(cfg, "wq")
    off_k, _ = pb.layer_tensor(cfg, "wk")
    off_v, _ = pb.layer_tensor(cfg, "wv")
    assert n_q == d * d and off_k == off_q + d * d and off_v == off_k + d * d
    off_bq, _ = pb.layer_tensor(cfg, "bq")
    off_bk, _ = pb.layer_tensor(cfg, "bk")
    assert off_bk == off_bq + d
    # tensors do not overlap and fit the blob
    spans = sorted(pb.layer_tensor(cfg, n) for n in synth.LAYER_TENSORS)
    for (o1, n1), (o2, _) in zip(spans, spans[1:]):
        assert o1 + n1 <= o2
    assert spans[-1][0] + spans[-1][1] <= lb // 2
    gb = L.pb_globals_bytes(ctypes.byref(cfg))
    assert gb >= 2 * w.global_params()
    # LoRA blob: A [r, d] then B [d, r] per target, q before v
    mask = 1 | 4
    assert L.pb_lora_layer_bytes(ctypes.byref(cfg), 16, mask) == 2 * 2 * 2 * 16 * d
    assert pb.lora_tensor(cfg, 16, mask, "q", "A") == (0, 16 * d)
    assert pb.lora_tensor(cfg, 16, mask, "q", "B") == (16 * d, 16 * d)
    assert pb.lora_tensor(cfg, 16, mask, "v", "A") == (32 * d, 16 * d)
    assert L.pb_arena_bytes(ctypes.byref(cfg)) > w.storage_bytes()
    del f


def test_invalid_configs_are_refused():
    from paper_2503_17707_amd import binding as pb

    L = pb.lib()
    base = pb.make_config(synth.WORKLOADS["tiny"])
    for field, value in (("d_model", 200), ("n_heads", 3), ("d_ffn", 100), ("n_layers", 0),
                         ("dtype", 7), ("max_rank", 0), ("max_adapters", 17)):
        cfg = pb.Config.from_buffer_copy(base)
        setattr(cfg, field, value)
        assert L.pb_arena_bytes(ctypes.byref(cfg)) == 0, field
        off = ctypes.c_size_t()
        assert L.pb_layer_tensor(ctypes.byref(cfg), 0, ctypes.byref(off), None) == pb.PB_EINVAL
        assert L.pb_last_error().decode()


def test_pageable_blob_binds_to_a_numa_node_before_first_touch():
    import numpy as np

    from paper_2503_17707_amd import binding as pb

    b = pb.Pageable(3 << 20, 0)  # node 0 exists on every Linux host
    assert b.bound
    assert b.ptr % 4096 == 0
    v = b.view()
    v[:] = 5
    assert int(v.sum()) == 5 * (3 << 20)
    assert not pb.Pageable(1 << 20, -1).bound
