"""The ctypes mirrors of the public structs match the C header byte for byte.

A small C program built with the host compiler prints sizeof and offsetof of
every field of the structs declared in include/muonbp.h; the binding's
ctypes.Structure classes must agree.  No GPU and no library load needed.
"""

import os
import shutil
import subprocess

import pytest

from paper_2510_16981_amd import muonbp as mb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

STRUCTS = {
    "muonbp_matrix": mb.Matrix,
    "muonbp_options": mb.Options,
    "muonbp_plan_info": mb.PlanInfo,
    "muonbp_profile": mb.Profile,
    "muonbp_adamw_options": mb.AdamwOptions,
}


def _c_layout(tmp_path):
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "muonbp.h"', "int main(void) {"]
    for cname, cls in STRUCTS.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in cls._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", f"{ROOT}/include", str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    table = {}
    for line in out.splitlines():
        cname, field, value = line.split()
        table[(cname, field)] = int(value)
    return table


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs a host C compiler")
def test_ctypes_structs_match_header(tmp_path):
    import ctypes
    table = _c_layout(tmp_path)
    for cname, cls in STRUCTS.items():
        assert ctypes.sizeof(cls) == table[(cname, "size")], cname
        for fname, _ in cls._fields_:
            assert getattr(cls, fname).offset == table[(cname, fname)], (cname, fname)
