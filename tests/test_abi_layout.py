"""The binding's ctypes structures match the C declarations of
include/qlinear.h field by field (sizes and offsets), checked by compiling a
small C program against the header with the host compiler (CPU only)."""
import ctypes
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIP_INCLUDE = "/opt/rocm/include"

STRUCTS = {
    "ql_linear": ["fmt", "X", "xdt", "M", "K", "N", "codes", "scales", "Y"],
    "ql_epilogue": ["bias", "act", "residual", "ydt", "steer_dir", "steer_norm",
                    "steer_strength", "y_bf16_copy"],
    "ql_linear_ep": ["lin", "ep"],
}


def c_layout():
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None or not os.path.isdir(os.path.join(HIP_INCLUDE, "hip")):
        pytest.skip("no host C compiler or HIP headers")
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "qlinear.h"',
             'int main(void) {']
    for name, fields in STRUCTS.items():
        lines.append(f'printf("{name} size %zu\\n", sizeof({name}));')
        for f in fields:
            lines.append(f'printf("{name} {f} %zu\\n", offsetof({name}, {f}));')
    lines.append("return 0; }")
    d = tempfile.mkdtemp(prefix="abi_layout_")
    try:
        src, exe = os.path.join(d, "l.c"), os.path.join(d, "l")
        open(src, "w").write("\n".join(lines))
        subprocess.run([cc, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", HIP_INCLUDE, src, "-o", exe], check=True, capture_output=True)
        out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    finally:
        shutil.rmtree(d, ignore_errors=True)
    res = {}
    for line in out.splitlines():
        parts = line.split()
        res[tuple(parts[:-1])] = int(parts[-1])
    return res


def test_ctypes_structs_match_header():
    from paper_2607_08526_amd.qlinear import _Epilogue, _Linear, _LinearEp
    c = c_layout()
    for name, cls in (("ql_linear", _Linear), ("ql_epilogue", _Epilogue),
                      ("ql_linear_ep", _LinearEp)):
        assert ctypes.sizeof(cls) == c[(name, "size")], name
        for f in STRUCTS[name]:
            assert getattr(cls, f).offset == c[(name, f)], (name, f)
