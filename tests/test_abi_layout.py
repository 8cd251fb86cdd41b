"""The binding's ctypes mirrors of the boundary's structs against the header:
a small C program compiled with the host compiler against include/gsraster.h
prints each struct's size and each field's offset, and every one must equal
what ctypes lays out (a field added, dropped or reordered on one side only
would otherwise pass arguments shifted, silently)."""
import ctypes
import os
import shutil
import subprocess

import pytest

from paper_2609_05255_amd import gsraster as gs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MIRRORS = {
    "gs_camera": gs.Camera,
    "gs_gaussians": gs.Gaussians,
    "gs_appearance": gs.Appearance,
    "gs_preprocessed": gs.Preprocessed,
    "gs_grads": gs.Grads,
    "gs_adam_tensor": gs.AdamTensor,
}


# where the binding reads each field of a 64-byte splat record, in 4-byte words
SPLAT_WORDS = sorted(gs.SPLAT_WORDS.items(), key=lambda kv: kv[1])


def c_layout(tmp_path):
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "gsraster.h"', "int main(void) {"]
    for cname, cls in MIRRORS.items():
        lines.append('    printf("%s size %%zu\\n", sizeof(%s));' % (cname, cname))
        for fname, _ in cls._fields_:
            lines.append('    printf("%s %s %%zu\\n", offsetof(%s, %s));' % (cname, fname, cname, fname))
    for fname, _ in SPLAT_WORDS:
        lines.append('    printf("gs_splat %s %%zu\\n", offsetof(gs_splat, %s));' % (fname, fname))
    lines.append('    printf("gs_splat size %zu\\n", sizeof(gs_splat));')
    lines += ["    return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    layout = {}
    for line in out.splitlines():
        struct, field, value = line.split()
        layout[(struct, field)] = int(value)
    return layout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no host C compiler")
def test_ctypes_mirrors_match_the_header(tmp_path):
    layout = c_layout(tmp_path)
    for cname, cls in MIRRORS.items():
        assert layout[(cname, "size")] == ctypes.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert layout[(cname, fname)] == getattr(cls, fname).offset, (cname, fname)
    assert layout[("gs_splat", "size")] == 64
    for fname, word in SPLAT_WORDS:
        assert layout[("gs_splat", fname)] == 4 * word, fname
