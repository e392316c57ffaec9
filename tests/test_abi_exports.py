"""The C-ABI library loads and exports every function include/lattice.h
declares, and the host-side queries that launch nothing answer on a machine
without a GPU.  No compute entry point is called here."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2512_09200_amd import _abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lattice.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    # the header declares no function pointers or macros with arguments, so
    # every "lattice_<name>(" left after stripping comments is a declaration
    return sorted(set(re.findall(r"\b(lattice_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("lattice_embbag_fwd", "lattice_embbag_bwd", "lattice_interact_fwd",
                     "lattice_interact_bwd", "lattice_mlp_heads_fwd", "lattice_mlp_heads_bwd",
                     "lattice_step", "lattice_forward", "lattice_step_plan", "lattice_validate_batch",
                     "lattice_status_string", "lattice_last_error", "lattice_abi_version"):
        assert required in names, required


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_abi.LIB_PATH):
        pytest.fail(f"{_abi.LIB_PATH} is not built (run __graft_entry__.build())")
    return ctypes.CDLL(_abi.LIB_PATH)


def test_library_exports_every_declared_function(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, f"declared in lattice.h but not exported: {missing}"


def test_exports_are_c_symbols():
    out = subprocess.run(["nm", "-D", "--defined-only", _abi.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    for n in declared_functions():
        assert n in exported, f"{n} is not an unmangled text symbol"


def test_host_queries_without_gpu(lib):
    lib.lattice_abi_version.restype = ctypes.c_int
    version = int(re.search(r"#define LATTICE_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert lib.lattice_abi_version() == version
    lib.lattice_status_string.restype = ctypes.c_char_p
    lib.lattice_status_string.argtypes = [ctypes.c_int]
    msgs = {code: lib.lattice_status_string(code).decode() for code in _abi.STATUS}
    assert all(msgs.values()) and len(set(msgs.values())) == len(msgs), msgs
    assert "unknown" in lib.lattice_status_string(99).decode()


def test_binding_structs_match_the_header(tmp_path):
    """Every ctypes structure of the binding has the size and field offsets
    of the C struct of the same name, as a C compiler lays it out."""
    structs = [getattr(_abi, n) for n in dir(_abi)
               if n.startswith("lattice_") and isinstance(getattr(_abi, n), type)
               and issubclass(getattr(_abi, n), ctypes.Structure)]
    assert structs
    lines = ['#include <stddef.h>', '#include <stdio.h>', f'#include "{HEADER}"', "int main(void) {"]
    expect = []
    for S in structs:
        lines.append(f'  printf("%zu\\n", sizeof({S.__name__}));')
        expect.append((S.__name__, "sizeof", ctypes.sizeof(S)))
        for f in S._fields_:
            lines.append(f'  printf("%zu\\n", offsetof({S.__name__}, {f[0]}));')
            expect.append((S.__name__, f[0], getattr(S, f[0]).offset))
    lines.append("  return 0;\n}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-o", str(exe), str(src)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    bad = [(s, f, want, g) for (s, f, want), g in zip(expect, got) if want != g]
    assert len(got) == len(expect) and not bad, bad
