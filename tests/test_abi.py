"""The C-ABI library loads and exports every function include/recis_mi355x.h declares (CPU only)."""
import ctypes
import os
import re

from paper_2509_20883_amd import recis as R


def _declared():
    src = open(R.HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^(?:rs_status|int|size_t|const char\s*\*)\s*([A-Za-z_][A-Za-z0-9_]*)\s*\(", src, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("ht_create", "ht_find_or_insert", "lookup_pool_fwd", "lookup_pool_bwd", "sparse_opt_step"):
        assert n in names


def test_library_exports_every_declared_symbol():
    assert os.path.exists(R.LIB_PATH), "build the library first (paper_2509_20883_amd/build.py)"
    lib = ctypes.CDLL(R.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert R.lib().rs_version() == 10


def test_binding_struct_layouts_match_header(tmp_path):
    """ctypes mirrors of the header's structs have the C compiler's sizes and offsets."""
    import subprocess
    prog = tmp_path / "layout.c"
    fields = {"rs_table_desc": [f[0] for f in R.TableDesc._fields_],
              "rs_opt_params": [f[0] for f in R.OptParams._fields_],
              "rs_ctx": [f[0] for f in R.RsCtx._fields_]}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "recis_mi355x.h"', "int main(void) {"]
    for st, fs in fields.items():
        lines.append(f'printf("%zu\\n", sizeof({st}));')
        for f in fs:
            lines.append(f'printf("%zu\\n", offsetof({st}, {f}));')
    lines.append("return 0; }")
    prog.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(R.HEADER), str(prog), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()]
    want = []
    for cls in (R.TableDesc, R.OptParams, R.RsCtx):
        want.append(ctypes.sizeof(cls))
        want += [getattr(cls, f[0]).offset for f in cls._fields_]
    assert got == want
