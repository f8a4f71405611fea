"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function declared in include/olive_score.h,
describe every status code, and reject malformed arguments on the host before it
touches the device.
"""
import ctypes
import os
import re

import pytest

from paper_2609_36246_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "olive_score.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        from paper_2609_36246_amd import build
        build.build()
    return L.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(olive_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("olive_score_init", "olive_token_logprobs", "olive_kl_masked",
              "olive_score_free", "olive_status_string", "olive_score_last_error",
              "olive_score_last_stats", "olive_score_kernel_times", "olive_score_batch",
              "olive_score_batch_spans", "olive_score_backward"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_status_strings(lib):
    seen = set()
    for code in L.STATUS_CODES:
        s = L.olive_status_string(code)
        assert s.startswith("OLIVE_")
        seen.add(s)
    assert len(seen) == len(L.STATUS_CODES)
    assert "unknown" in L.olive_status_string(99)


STRUCTS = ("olive_score_desc", "olive_batch", "olive_score_outputs", "olive_spans",
           "olive_grad_outputs")


def header_layouts(tmp_path):
    """sizeof and offsetof of every field of the public structs, from the header
    itself compiled by the host C compiler."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "olive_score.h"',
             "int main(void) {"]
    for name in STRUCTS:
        lines.append('printf("%s __sizeof__ %%zu\\n", sizeof(%s));' % (name, name))
        for f, _ in getattr(L, name)._fields_:
            lines.append('printf("%s %s %%zu\\n", offsetof(%s, %s));' % (name, f, name, f))
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    return {tuple(l.split()[:2]): int(l.split()[2]) for l in out.splitlines()}


def test_struct_layouts_match_header(tmp_path):
    got = header_layouts(tmp_path)
    for name in STRUCTS:
        st = getattr(L, name)
        assert got[(name, "__sizeof__")] == ctypes.sizeof(st), name
        for f, _ in st._fields_:
            assert got[(name, f)] == getattr(st, f).offset, (name, f)
    assert ctypes.sizeof(L.olive_score_outputs) == 112
    assert L.olive_score_outputs.topk_teacher.offset == 96
    assert L.olive_score_outputs.jsd.offset == 104


def test_header_constants_match_the_binding():
    """Every numeric #define of the header has the same value in the Python binding."""
    text = open(HEADER).read()
    defs = re.findall(r"^#define\s+(OLIVE_[A-Z0-9_]+)\s+(\d+)\s*$", text, re.M)
    assert len(defs) >= 6
    for name, value in defs:
        assert getattr(L, name) == int(value), name


def _init(desc, ws=1, wt=1):
    return L.olive_score_init(desc, ws, wt, stream=None, check=False)


@pytest.mark.parametrize("field,value,expect", [
    ("dtype", 7, L.OLIVE_E_DTYPE),
    ("w_layout", 5, L.OLIVE_E_DTYPE),
    ("vocab", 0, L.OLIVE_E_SHAPE),
    ("vocab", 1 << 31, L.OLIVE_E_SHAPE),
    ("d_student", 0, L.OLIVE_E_SHAPE),
    ("d_teacher", -1, L.OLIVE_E_SHAPE),
    ("max_positions", 0, L.OLIVE_E_SHAPE),
    ("max_seqs", 0, L.OLIVE_E_SHAPE),
    ("d_student", 12289, L.OLIVE_E_UNSUPPORTED),
    ("logit_scale_student", 0.0, L.OLIVE_E_RANGE),
    ("logit_scale_student", float("inf"), L.OLIVE_E_RANGE),
    ("logit_scale_teacher", -1.0, L.OLIVE_E_RANGE),
    ("logit_scale_teacher", float("nan"), L.OLIVE_E_RANGE),
    ("flags", 64, L.OLIVE_E_RANGE),
])
def test_init_rejects_bad_descriptors_on_host(lib, field, value, expect):
    d = L.make_desc(1000, 64, 96, max_positions=64, max_seqs=2)
    setattr(d, field, value)
    status, handle = _init(d)
    assert status == expect and handle is None


def test_init_null_pointers(lib):
    d = L.make_desc(1000, 64, 96, max_positions=64, max_seqs=2)
    assert _init(d, ws=None)[0] == L.OLIVE_E_NULL
    assert _init(d, wt=None)[0] == L.OLIVE_E_NULL
    h = ctypes.c_void_p()
    assert lib.olive_score_init(ctypes.byref(h), None, 1, 1, None) == L.OLIVE_E_NULL
    assert lib.olive_score_init(None, ctypes.byref(d), 1, 1, None) == L.OLIVE_E_NULL


def test_calls_on_null_context(lib):
    b = L.olive_batch()
    assert lib.olive_token_logprobs(None, ctypes.byref(b), 1, None, None, None,
                                    None) == L.OLIVE_E_NULL
    assert lib.olive_kl_masked(None, ctypes.byref(b), 1, None, None, None, None, None, None,
                               None) == L.OLIVE_E_NULL
    assert lib.olive_score_free(None) == L.OLIVE_OK
    v = ctypes.c_int32()
    assert lib.olive_score_last_error(None, ctypes.byref(v)) == L.OLIVE_E_NULL
    out = (ctypes.c_int64 * 4)()
    assert lib.olive_score_last_stats(None, out) == L.OLIVE_E_NULL
    f = (ctypes.c_float * 4)()
    assert lib.olive_score_kernel_times(None, f, 1) == L.OLIVE_E_NULL
    o = L.make_outputs()
    assert lib.olive_score_batch(None, ctypes.byref(b), ctypes.byref(o), None) == L.OLIVE_E_NULL
    gr = L.make_grad_outputs()
    assert lib.olive_score_backward(None, ctypes.byref(b), None, ctypes.byref(gr),
                                    None) == L.OLIVE_E_NULL
    sp = L.olive_spans()
    assert lib.olive_score_batch_spans(None, ctypes.byref(b), ctypes.byref(sp), ctypes.byref(o),
                                       None) == L.OLIVE_E_NULL


def test_binding_refuses_to_run_without_the_library(monkeypatch, tmp_path):
    monkeypatch.setattr(L, "_lib", None)
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        L.load()


def test_library_and_torch_share_one_hip_runtime(lib):
    """Loading the binding before torch must still leave a single HIP runtime mapped."""
    import subprocess
    import sys
    code = ("from paper_2609_36246_amd import _lib as L\n"
            "L.load()\n"
            "import torch\n"
            "paths = set()\n"
            "for line in open('/proc/self/maps'):\n"
            "    f = line.split()[-1]\n"
            "    if 'libamdhip64' in f:\n"
            "        paths.add(__import__('os').path.realpath(f))\n"
            "print(len(paths), sorted(paths))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr
    n = int(r.stdout.split()[0])
    assert n == 1, r.stdout
