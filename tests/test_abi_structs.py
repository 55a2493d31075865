"""The binding's ctypes structures against the C declarations of
include/seg.h (CPU only): a C probe compiled with the host compiler prints
sizeof of every structure and offsetof of every field the binding names,
and both must equal what ctypes computes.  A field added to one side only
would otherwise shift every later pointer of the structure."""
import ctypes
import os
import shutil
import subprocess

import pytest

from paper_2607_11185_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
STRUCTS = {
    "seg_problem": _lib.SegProblem,
    "seg_sizes": _lib.SegSizes,
    "seg_layout": _lib.SegLayout,
    "seg_loss_cfg": _lib.SegLossCfg,
    "seg_layer_cfg": _lib.SegLayerCfg,
    "seg_layer_weights": _lib.SegLayerWeights,
    "seg_layer_saved": _lib.SegLayerSaved,
    "seg_layer_grads": _lib.SegLayerGrads,
}


def _probe(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("no host C compiler or HIP headers")
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "seg.h"', "int main(void) {"]
    for cname, py in STRUCTS.items():
        lines.append(f'  printf("{cname} sizeof %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'  printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "probe.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "probe"
    subprocess.run([cc, "-x", "c", "-std=c99", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__", str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    return {tuple(line.split()[:2]): int(line.split()[2]) for line in out.splitlines()}


def test_ctypes_structs_match_header(tmp_path):
    c = _probe(tmp_path)
    for cname, py in STRUCTS.items():
        assert ctypes.sizeof(py) == c[(cname, "sizeof")], cname
        for f, _ in py._fields_:
            assert getattr(py, f).offset == c[(cname, f)], (cname, f)


def test_header_fields_all_mirrored():
    """Every field declared in a mirrored structure has a ctypes field of the
    same name (the probe above cannot see a field the binding omits at the
    end of a structure)."""
    import re
    with open(os.path.join(ROOT, "include", "seg.h")) as f:
        hdr = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
    for cname, py in STRUCTS.items():
        m = re.search(r"typedef struct\s*\{([^{}]*)\}\s*" + cname + r"\s*;", hdr)
        assert m, cname
        declared = []
        for decl in m.group(1).split(";"):
            decl = decl.strip()
            if not decl:
                continue
            names = decl.split(None, 1)[1] if " " in decl else decl
            for part in names.split(","):
                nm = re.sub(r"\[.*?\]", "", part).replace("*", "").replace("const", "").strip()
                nm = nm.split()[-1]
                declared.append(nm)
        assert declared == [f for f, _ in py._fields_], (cname, declared)
