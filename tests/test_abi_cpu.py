"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and its struct layouts agree with the binding's."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

import paper_2407_00051_amd as sg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sagips.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sagips_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    if not os.path.exists(sg.LIB_PATH):
        pytest.skip("library not built")
    lib = ctypes.CDLL(sg.LIB_PATH)
    names = declared_functions()
    assert set(names) == set(sg.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n


def test_struct_layout_matches_header(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc unavailable")
    src = tmp_path / "layout.c"
    src.write_text("""
#include <stddef.h>
#include <stdio.h>
#include "sagips.h"
#define P(T, f) printf(#T "." #f " %zu\\n", offsetof(T, f))
int main(void) {
  printf("sagips_source %zu\\n", sizeof(sagips_source));
  printf("sagips_mlp %zu\\n", sizeof(sagips_mlp));
  printf("sagips_disc_out %zu\\n", sizeof(sagips_disc_out));
  printf("sagips_gen %zu\\n", sizeof(sagips_gen));
  printf("sagips_param_set %zu\\n", sizeof(sagips_param_set));
  P(sagips_source, events_per_theta); P(sagips_source, seed); P(sagips_source, stream);
  P(sagips_mlp, W); P(sagips_mlp, b); P(sagips_mlp, leaky_slope); P(sagips_mlp, features);
  P(sagips_disc_out, dW); P(sagips_disc_out, dLg_dx); P(sagips_disc_out, dLg_dtheta);
  P(sagips_gen, W); P(sagips_gen, b); P(sagips_gen, n_members); P(sagips_gen, leaky_slope);
  P(sagips_param_set, param); P(sagips_param_set, grad); P(sagips_param_set, m); P(sagips_param_set, v);
  P(sagips_param_set, size);
  return 0;
}
""")
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)])
    got = dict(line.split() for line in subprocess.check_output([str(exe)], text=True).splitlines())
    py = {"sagips_source": ctypes.sizeof(sg.Source), "sagips_mlp": ctypes.sizeof(sg.Mlp),
          "sagips_disc_out": ctypes.sizeof(sg.DiscOut), "sagips_gen": ctypes.sizeof(sg.GenStack),
          "sagips_param_set": ctypes.sizeof(sg.ParamSet)}
    for k, v in py.items():
        assert int(got[k]) == v, k
    for k, v in got.items():
        if "." in k:
            st, f = k.split(".")
            cls = {"sagips_source": sg.Source, "sagips_mlp": sg.Mlp, "sagips_disc_out": sg.DiscOut,
                   "sagips_gen": sg.GenStack, "sagips_param_set": sg.ParamSet}[st]
            assert getattr(cls, f).offset == int(v), k


def test_last_error_never_null():
    if not os.path.exists(sg.LIB_PATH):
        pytest.skip("library not built")
    lib = sg.load_library()
    assert isinstance(lib.sagips_last_error(None), bytes)
