"""Host-only checks of the C ABI library: it is built, it loads, and it
exports every function include/ifvs.h declares (no GPU calls)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ifvs.h")
LIB = os.path.join(ROOT, "paper_2607_22922_amd", "libifvs.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(ifvs_[a-z_]+)\s*\(",
                                 text, flags=re.M)))


def test_header_declares_the_four_path_calls():
    names = declared_functions()
    for n in ("ifvs_load_index", "ifvs_select_codebook", "ifvs_build_lut", "ifvs_filtered_search"):
        assert n in names
    assert len(names) >= 9


def test_library_loads_and_exports_every_declared_symbol():
    assert os.path.exists(LIB), "build the library first: python -m paper_2607_22922_amd.build"
    lib = ctypes.CDLL(LIB)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in ifvs.h but not exported"


def _c_layout(tmp_path):
    """sizeof/offsetof of the header's structs as the C compiler lays them out."""
    from paper_2607_22922_amd import ifvs as B
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ifvs.h"', "int main(void) {"]
    for cname, cls in (("ifvs_index_desc", B.IndexDesc), ("ifvs_clause", B.Clause),
                       ("ifvs_predicate", B.Predicate)):
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f in cls._fields_:
            lines.append(f'printf("{cname} {f[0]} %zu\\n", offsetof({cname}, {f[0]}));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    return {tuple(l.split()[:2]): int(l.split()[2]) for l in out.splitlines()}


def test_binding_mirrors_header_structs(tmp_path):
    from paper_2607_22922_amd import ifvs as B
    layout = _c_layout(tmp_path)
    for cname, cls in (("ifvs_index_desc", B.IndexDesc), ("ifvs_clause", B.Clause),
                       ("ifvs_predicate", B.Predicate)):
        assert layout[(cname, "size")] == ctypes.sizeof(cls), cname
        for f in cls._fields_:
            assert layout[(cname, f[0])] == getattr(cls, f[0]).offset, (cname, f[0])
    # same field order as the header
    text = open(HEADER).read()
    body = text[text.index("typedef struct {\n  int64_t n;"):text.index("} ifvs_index_desc;")]
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    assert [f[0] for f in B.IndexDesc._fields_] == re.findall(r"\b\**\s*([a-zA-Z_]+)(?:\[\d+\])?;", body)
    assert set(B.EXPORTED) == set(declared_functions())


def test_null_handle_and_error_text_without_gpu():
    from paper_2607_22922_amd import ifvs as B
    lib = B.lib()
    assert lib.ifvs_set_option(None, B.OPT_QTILE, 1) == B.E_STATE
    assert b"NULL" in lib.ifvs_last_error()
    assert lib.ifvs_load_index(None, None) == B.E_INVALID
    lib.ifvs_free_index(None)


def test_encoder_parameter_count_matches_the_documented_layout():
    """ifvs_encoder_params (a host-only function) counts the floats of the
    layout include/ifvs.h documents; sizes out of range give -1."""
    lib = ctypes.CDLL(LIB)
    fn = lib.ifvs_encoder_params
    fn.argtypes = [ctypes.c_int32] * 6
    fn.restype = ctypes.c_int64
    for H, heads, L, F, A, D in [(64, 4, 2, 128, 1, 96), (16, 16, 1, 16, 3, 7), (128, 8, 8, 256, 2, 960)]:
        per_layer = 2 * H + 3 * H * H + 3 * H + H * H + H + 2 * H + H * F + F + F * H + H
        assert fn(H, heads, L, F, A, D) == A * H + 2 * H + 2 * H + L * per_layer + 2 * H + H * D + D
    for bad in [(8, 1, 1, 16, 1, 4), (48 + 1, 1, 1, 16, 1, 4), (64, 3, 1, 16, 1, 4), (64, 4, 0, 16, 1, 4),
                (64, 4, 9, 16, 1, 4), (64, 32, 1, 16, 1, 4), (64, 4, 1, 272, 1, 4), (144, 4, 1, 16, 1, 4), (64, 4, 1, 16, 0, 4)]:
        assert fn(*bad) == -1, bad
