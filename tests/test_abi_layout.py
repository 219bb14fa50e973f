"""The ctypes mirrors of the C ABI's structs (paper_2306_03622_amd/torpor.py) against the C
compiler's layout of include/torpor.h: every struct's size and every field's offset, so that a
field added on one side only fails here instead of corrupting memory at a call."""
import ctypes
import os
import shutil
import subprocess

import pytest

from paper_2306_03622_amd import torpor as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
STRUCTS = ["tp_tensor_desc", "tp_model_desc", "tp_config", "tp_arena_stats_t", "tp_model_info_t", "tp_request",
           "tp_request_result", "tp_sched_config", "tp_sched_stats"]


def test_ctypes_layout_matches_the_header(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if not cc:
        pytest.skip("no C compiler")
    src = ["#include <stdio.h>", "#include <stddef.h>", '#include "torpor.h"', "int main(void) {"]
    for s in STRUCTS:
        src.append(f'  printf("{s} %zu\\n", sizeof({s}));')
        for f, _ in getattr(T, s)._fields_:
            src.append(f'  printf("{s}.{f} %zu\\n", offsetof({s}, {f}));')
    src += ["  return 0;", "}"]
    c_file, exe = tmp_path / "layout.c", tmp_path / "layout"
    c_file.write_text("\n".join(src) + "\n")
    subprocess.run([cc, "-std=c11", "-I", os.path.join(ROOT, "include"), str(c_file), "-o", str(exe)], check=True)
    got = dict(line.split() for line in subprocess.run([str(exe)], check=True, capture_output=True,
                                                        text=True).stdout.splitlines())
    for s in STRUCTS:
        cls = getattr(T, s)
        assert int(got[s]) == ctypes.sizeof(cls), s
        for f, _ in cls._fields_:
            assert int(got[f"{s}.{f}"]) == getattr(cls, f).offset, f"{s}.{f}"
