"""The Python binding's ctypes structs against the C header (CPU): gcc
compiles a program that prints sizeof and offsetof of every field of every
struct the binding declares, and each must match ctypes' layout.  A field
added to the header but not to the binding (or in another order, or of
another width) would make the library read or write the wrong bytes."""
import ctypes
import os
import shutil
import subprocess

import pytest

import paper_2511_07035_amd as g

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

STRUCTS = ["gockpt_config", "gockpt_window_opts", "gockpt_step_record", "gockpt_window_stats", "gockpt_ckpt_meta",
           "gockpt_arena_layout", "gockpt_plan_params", "gockpt_plan_result", "gockpt_ckpt_info", "gockpt_io_stats"]


def test_ctypes_layout_matches_header(tmp_path):
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no C compiler")
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "gockpt.h"', 'int main(void) {']
    expect = []
    for name in STRUCTS:
        cls = getattr(g, name)
        lines.append(f'  printf("{name} size %zu\\n", sizeof({name}));')
        expect.append(f"{name} size {ctypes.sizeof(cls)}")
        for fname, _ in cls._fields_:
            lines.append(f'  printf("{name}.{fname} %zu %zu\\n", offsetof({name}, {fname}), '
                         f'sizeof((({name}*)0)->{fname}));')
            f = getattr(cls, fname)
            expect.append(f"{name}.{fname} {f.offset} {f.size}")
    lines += ['  return 0;', '}']
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", f"-I{ROOT}/include", str(src), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    got = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = [ln for ln in got if ln]
    assert got == expect


def test_every_header_struct_is_bound():
    """Every struct typedef of the header has a ctypes twin in the test above."""
    import re
    text = open(os.path.join(ROOT, "include", "gockpt.h")).read()
    names = set(re.findall(r"\}\s*(gockpt_\w+)\s*;", text))
    assert names == set(STRUCTS), names ^ set(STRUCTS)
