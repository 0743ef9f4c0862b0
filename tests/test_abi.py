"""The C ABI library loads and exports what include/taurus.h declares; host
functions and argument validation work without a GPU (no compute calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "taurus.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(taurus_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def native():
    from paper_2607_17374_amd import _native as N
    return N


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("taurus_layer_init", "taurus_push_chunk", "taurus_finalize", "taurus_sampled_edges",
                     "taurus_build_csr", "taurus_layer_destroy", "taurus_last_error", "taurus_hash",
                     "taurus_plan_create", "taurus_plan_destroy"):
        assert required in names


def test_library_exports_every_declared_symbol(native):
    L = native.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
        assert name in native.SIGNATURES, f"binding lacks {name}"


def header_constants():
    """TAURUS_* constants of the header's enums and #defines -> values."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    vals = {}
    for name, val in re.findall(r"\b(TAURUS_[A-Z0-9_]+)\s*=\s*(-?\d+)", text):
        vals[name] = int(val)
    for name, a, b in re.findall(r"#define\s+(TAURUS_[A-Z0-9_]+)\s+\((\d+)ll\s*<<\s*(\d+)\)", text):
        vals[name] = int(a) << int(b)
    return vals


def test_binding_constants_match_header(native):
    vals = header_constants()
    for name, val in vals.items():
        short = name[len("TAURUS_"):]
        if short in ("OK",) or hasattr(native, short):
            assert getattr(native, short) == val, name
        else:
            raise AssertionError(f"binding lacks {name}")


def test_binding_signatures_match_header(native):
    """Each declared function takes as many arguments in the binding as in
    the header."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for name, params in re.findall(r"\b(taurus_[a-z_0-9]+)\s*\(([^)]*)\)\s*;", text):
        params = params.strip()
        n = 0 if params in ("", "void") else params.count(",") + 1
        assert len(native.SIGNATURES[name][1]) == n, name


def test_binding_structs_match_header_layout(native):
    # field order and sizes as declared in taurus.h (x86-64 alignment)
    assert ctypes.sizeof(native.Graph) == 32
    assert native.LayerDesc.weight.offset == 24 and native.LayerDesc.seed.offset == 48
    assert native.LayerDesc.out.offset == 80 and native.LayerDesc.stream.offset == 96
    assert native.LayerDesc.plan.offset == 112 and native.LayerDesc.eviction.offset == 120
    assert native.LayerDesc.attn.offset == 128 and native.LayerDesc.d_hidden.offset == 136
    assert native.LayerDesc.weight2.offset == 144 and native.LayerDesc.bias2.offset == 152
    assert native.LayerDesc.setup_stream.offset == 160
    assert ctypes.sizeof(native.LayerDesc) == 168
    assert ctypes.sizeof(native.Stats) == 17 * 8 + 7 * 8 + 4 * 8 + 5 * 8


def test_binding_structs_match_compiled_header(native, tmp_path):
    """Every field offset and struct size of the binding's structures equals
    what a C compiler makes of include/taurus.h."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"taurus_graph": native.Graph, "taurus_layer_desc": native.LayerDesc,
               "taurus_stats": native.Stats, "taurus_stream_stats": native.StreamStats}
    lines = ["#include <stdio.h>", "#include <stddef.h>", f'#include "{HEADER}"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'    printf("{cname} sizeof %zu\\n", sizeof({cname}));')
        for field, _ in py._fields_:
            lines.append(f'    printf("{cname} {field} %zu\\n", offsetof({cname}, {field}));')
    lines += ["    return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c11", "-o", str(exe), str(src)], check=True, capture_output=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.splitlines():
        cname, field, value = line.split()
        got[(cname, field)] = int(value)
    for cname, py in structs.items():
        assert got[(cname, "sizeof")] == ctypes.sizeof(py), cname
        for field, _ in py._fields_:
            assert got[(cname, field)] == getattr(py, field).offset, (cname, field)


def test_hash_matches_published_splitmix64(golden_dir):
    from paper_2607_17374_amd.api import hash_u64
    G = 0x9e3779b97f4a7c15
    refs = [int(l, 16) for l in open(f"{golden_dir}/splitmix64_state0.txt") if l.strip() and not l.startswith("#")]
    for k, ref in enumerate(refs):
        assert hash_u64(0, (k * G) % 2**64) == ref


def test_invalid_arguments_rejected_before_device_work(native):
    L = native.lib()
    g = native.Graph(0, 0, None, None)
    d = native.LayerDesc()
    h = ctypes.c_void_p()
    assert L.taurus_layer_init(ctypes.byref(g), ctypes.byref(d), ctypes.byref(h)) == native.E_INVALID
    assert "graph size" in native.last_error()
    assert L.taurus_layer_init(None, None, ctypes.byref(h)) == native.E_INVALID
    assert L.taurus_push_chunk(None, 0, 1, None, 0) == native.E_INVALID
    assert L.taurus_finalize(None, None) == native.E_INVALID
    assert L.taurus_sampled_edges(None, None, None) == native.E_INVALID
    assert L.taurus_build_csr(0, 0, None, None, None, None, None) == native.E_INVALID
    # the allocation-free build refuses more edges than its scratch holds,
    # before touching any pointer or the device
    assert L.taurus_build_csr_noalloc(10, (1 << 20) + 1, 8, 8, 8, 8, None) == native.E_INVALID
    assert "exceed the limit" in native.last_error()
    L.taurus_layer_destroy(None)
    L.taurus_plan_destroy(None)
    hp = ctypes.c_void_p()
    assert L.taurus_plan_create(None, 16, None, ctypes.byref(hp)) == native.E_INVALID
    g1 = native.Graph(10, 0, 1, None)
    assert L.taurus_plan_create(ctypes.byref(g1), 0, None, ctypes.byref(hp)) == native.E_INVALID
    # width not a multiple of 4
    g = native.Graph(10, 0, 1, None)
    w = np.zeros(16, np.float32)
    d = native.LayerDesc(agg=0, d_in=6, d_out=4, weight=w.ctypes.data, chunk=4, out=1)
    assert L.taurus_layer_init(ctypes.byref(g), ctypes.byref(d), ctypes.byref(h)) == native.E_INVALID
    assert "multiples of 4" in native.last_error()
