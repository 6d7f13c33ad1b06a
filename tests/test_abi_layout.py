"""The ctypes mirrors of the boundary's structs match the C layout: every struct's size and
every field's offset, as a C compiler (gcc) lays out include/miriam.h.  Runs on the host."""
import ctypes
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PAIRS = [  # (C type, ctypes mirror in _lib)
    ("miriam_op_desc", "OpDesc"),
    ("miriam_op_info", "OpInfo"),
    ("miriam_device_desc", "DeviceDesc"),
    ("miriam_config", "Config"),
    ("miriam_launch_record", "LaunchRecord"),
    ("miriam_completion", "Completion"),
    ("miriam_stats", "Stats"),
]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_ctypes_structs_match_the_c_layout(tmp_path):
    from paper_2307_04339_amd import _lib as L
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "miriam.h"', "int main(void) {"]
    for ctype, py in PAIRS:
        lines.append(f'    printf("{py} size %zu\\n", sizeof({ctype}));')
        for name, _ in getattr(L, py)._fields_:
            lines.append(f'    printf("{py} {name} %zu\\n", offsetof({ctype}, {name}));')
    lines += ["    return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {}
    for line in out:
        if line.strip():
            py, name, val = line.split()
            got[(py, name)] = int(val)
    for _, py in PAIRS:
        st = getattr(L, py)
        assert got[(py, "size")] == ctypes.sizeof(st), py
        for name, _ in st._fields_:
            assert got[(py, name)] == getattr(st, name).offset, (py, name)
