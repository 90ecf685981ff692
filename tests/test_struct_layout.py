"""The ctypes mirrors of the C-ABI structs have the C compiler's layout:
gcc compiles a program that prints sizeof and every field's offset of each
struct as declared in include/acache.h, and the binding must agree."""

import ctypes
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

STRUCTS = {  # C typedef -> ctypes class name in the binding
    "acache_dims": "Dims",
    "acache_layer_weights": "LayerWeights",
    "acache_ragged": "Ragged",
    "acache_score_args": "ScoreArgs",
    "acache_layout": "Layout",
    "acache_paging": "Paging",
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_ctypes_structs_match_c_layout(tmp_path):
    from paper_2608_26140_amd import acache as B
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "acache.h"', "int main(void) {"]
    for cname, pyname in STRUCTS.items():
        lines.append(f'  printf("{cname} sizeof %zu\\n", sizeof({cname}));')
        for f, _ in getattr(B, pyname)._fields_:
            lines.append(f'  printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for cname, pyname in STRUCTS.items():
        cls = getattr(B, pyname)
        assert got[(cname, "sizeof")] == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert got[(cname, f)] == getattr(cls, f).offset, f"{cname}.{f}"
