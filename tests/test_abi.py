"""The C-ABI library loads on a machine without a GPU, exports every entry
point include/grand.h declares, its structs match the Python binding, and
host-only argument checks work.  No compute call is made here."""
import ctypes
import os
import re
import subprocess

import pytest

from conftest import ROOT
from paper_2608_21163_amd import grand

HEADER = os.path.join(ROOT, "include", "grand.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(grand_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = grand.load_library()
    names = declared_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", grand.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (grand_\w+)", out))
    assert set(names) <= exported
    assert set(grand.EXPORTED) == set(names)


def test_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    fields_p = [f for f, _ in grand.Params._fields_]
    fields_s = [f for f, _ in grand.Stats._fields_]
    lines = ['#include <stddef.h>', '#include <stdio.h>', f'#include "{HEADER}"', 'int main(void) {',
             'printf("%zu %zu\\n", sizeof(grand_params), sizeof(grand_stats_t));']
    lines += [f'printf("%zu\\n", offsetof(grand_params, {f}));' for f in fields_p]
    lines += [f'printf("%zu\\n", offsetof(grand_stats_t, {f}));' for f in fields_s]
    lines += ["return 0; }"]
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", str(src), "-o", str(exe)])
    vals = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert vals[0] == ctypes.sizeof(grand.Params) and vals[1] == ctypes.sizeof(grand.Stats)
    offs = vals[2:]
    assert offs[: len(fields_p)] == [getattr(grand.Params, f).offset for f in fields_p]
    assert offs[len(fields_p):] == [getattr(grand.Stats, f).offset for f in fields_s]


def test_default_params_are_the_papers():
    p = grand.Params()
    grand.load_library().grand_default_params(ctypes.byref(p))
    assert p.struct_size == ctypes.sizeof(grand.Params)
    assert abs(p.alpha - 1.2) < 1e-6 and p.P == 64 and p.c == 2 and p.k_repair == 50   # Section 5.4
    assert p.algo == grand.VAMANA and p.metric == grand.L2 and p.cas_mode == grand.CAS_GROUPED


@pytest.mark.parametrize("field,value", [("R", 0), ("R", 65), ("L_build", 300), ("P", 0), ("k_repair", 65),
                                         ("dim", 0), ("capacity", 0), ("max_iters", 10), ("struct_size", 12)])
def test_create_rejects_bad_parameters_before_touching_the_gpu(field, value):
    lib = grand.load_library()
    p = grand.Params()
    lib.grand_default_params(ctypes.byref(p))
    setattr(p, field, value)
    h = ctypes.c_void_p()
    assert lib.grand_create(ctypes.byref(p), ctypes.byref(h)) == grand.E_ARG
    assert not h.value


def test_create_rejects_unsupported_metric_combinations():
    lib = grand.load_library()
    p = grand.Params()
    lib.grand_default_params(ctypes.byref(p))
    p.metric = grand.IP          # Vamana on IP: the paper augments IP data to L2 instead
    h = ctypes.c_void_p()
    assert lib.grand_create(ctypes.byref(p), ctypes.byref(h)) == grand.E_ARG
    p.algo, p.dtype = grand.CAGRA, grand.U8
    assert lib.grand_create(ctypes.byref(p), ctypes.byref(h)) == grand.E_ARG


def test_null_handle_is_rejected():
    lib = grand.load_library()
    assert lib.grand_insert_batch(None, None, None, 0) == grand.E_ARG
    assert lib.grand_destroy(None) == grand.OK
    assert lib.grand_last_error(None) == b"null handle"
