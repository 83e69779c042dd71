"""The binding's ctypes structures and trace dtype have the sizes and field
offsets of the C structures in include/bart.h, as the host C compiler lays
them out: a field added, dropped or reordered on one side only would shift
every later argument the library reads."""
from __future__ import annotations

import ctypes
import os
import shutil
import subprocess
import tempfile

import pytest

from paper_2410_23244_amd import bart as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CC = shutil.which("gcc") or shutil.which("cc")

# binding name -> C name where Python needs another spelling
RENAMED = {"lam": "lambda"}


def _c_layout(struct: str, fields: list[str]) -> tuple[int, list[int]]:
    """sizeof(struct) and offsetof(struct, f) for each field, from a C program
    compiled against the header."""
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "bart.h"', "int main(void) {",
             f'  printf("%zu\\n", sizeof({struct}));']
    lines += [f'  printf("%zu\\n", offsetof({struct}, {f}));' for f in fields]
    lines += ["  return 0;", "}"]
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "layout.c"), os.path.join(d, "layout")
        with open(src, "w") as fh:
            fh.write("\n".join(lines) + "\n")
        subprocess.run([CC, "-std=c11", "-I", os.path.join(ROOT, "include"), src, "-o", exe],
                       check=True, capture_output=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.split()
    vals = [int(v) for v in out]
    return vals[0], vals[1:]


@pytest.mark.skipif(CC is None, reason="no host C compiler")
@pytest.mark.parametrize("cls,struct", [(B.Config, "bart_config"), (B.State, "bart_state"),
                                        (B.LaunchInfo, "bart_launch")])
def test_ctypes_structures_match_the_header(cls, struct):
    names = [f for f, _ in cls._fields_]
    size, offs = _c_layout(struct, [RENAMED.get(f, f) for f in names])
    assert ctypes.sizeof(cls) == size
    for f, off in zip(names, offs):
        assert getattr(cls, f).offset == off, f


@pytest.mark.skipif(CC is None, reason="no host C compiler")
def test_trace_dtype_matches_the_header():
    dt = B.TRACE_DTYPE
    size, offs = _c_layout("bart_trace", list(dt.names))
    assert dt.itemsize == size
    for f, off in zip(dt.names, offs):
        assert dt.fields[f][1] == off, f
