"""The C-ABI library loads on the host and exports every symbol include/dro.h declares.

CPU only: no entry point that needs a device is called here.
"""
import ctypes as ct
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dro.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(",
                       src, flags=re.M)
    return sorted(set(n for n in names if n not in {"if", "while", "for", "return"}))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_16892_amd import _native
    if not os.path.exists(_native.LIB_PATH):
        from paper_2607_16892_amd import build
        build.build()
    return _native.load()


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("dro_cost_eval", "dro_argmin_reservation", "class_quantile", "bcd_block_step",
              "bcd_init_state", "dro_create", "dro_destroy", "dro_validate", "dro_strerror",
              "dro_last_error", "dro_cost_eval_noalloc"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in _declared():
        assert hasattr(lib, n), n


def test_binding_covers_every_declared_symbol():
    from paper_2607_16892_amd import _native
    assert set(_declared()) == set(_native.EXPORTS)


def test_strerror_codes(lib):
    assert lib.dro_strerror(0) == b"ok"
    assert lib.dro_strerror(-1) == b"invalid argument"
    assert lib.dro_strerror(-5) == b"beyond the exactness limits"
    assert lib.dro_strerror(-99) == b"unknown error"


def test_null_context_is_rejected_without_device_work(lib):
    from paper_2607_16892_amd import _native
    ps = _native.ProblemStruct()
    assert lib.dro_cost_eval(None, ct.byref(ps), 1, None, None, None, None, None) == -1
    assert lib.dro_argmin_reservation(None, ct.byref(ps), 1, None, None, None, None, None, None,
                                      None) == -1
    assert lib.class_quantile(None, ct.byref(ps), None, None, None) == -1
    assert lib.bcd_block_step(None, ct.byref(ps), None, None, None, None, None) == -1
    assert lib.dro_baseline_reservations(None, 1, None, None, None, None, 0, None, None, 16, None,
                                         None, None, None) == -1
    assert lib.dro_last_error(None) == b"no context"


def test_product_has_no_cpu_fallback():
    """The product package neither imports the oracle nor computes on the host."""
    pkg = os.path.join(ROOT, "paper_2607_16892_amd")
    for fn in os.listdir(pkg):
        if fn.endswith(".py"):
            txt = open(os.path.join(pkg, fn)).read()
            assert "import oracle" not in txt and "from oracle" not in txt, fn


def test_header_is_plain_c_and_links(lib, tmp_path):
    """include/dro.h compiles as C99 (no C++ types in the ABI) and a C program
    that calls through it links against libdro.so (no entry point that needs a
    device is called: it is only linked)."""
    import shutil
    import subprocess
    from paper_2607_16892_amd import _native
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use_dro.c"
    src.write_text(
        '#include "dro.h"\n'
        "#include <stdio.h>\n"
        "int main(void) {\n"
        "    dro_problem p = {0};\n"
        "    int32_t k = 0; double w = 0.0;\n"
        "    int rc = dro_argmin_reservation(NULL, &p, 1, NULL, NULL, NULL, &k, &w, NULL, NULL);\n"
        '    printf("%d %s\\n", rc, dro_strerror(rc));\n'
        "    return rc == DRO_EINVAL ? 0 : 1;\n"
        "}\n")
    exe = tmp_path / "use_dro"
    libdir = os.path.dirname(_native.LIB_PATH)
    r = subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-pedantic", "-I",
                        os.path.join(ROOT, "include"), str(src), "-o", str(exe), "-L", libdir,
                        "-ldro", f"-Wl,-rpath,{libdir}"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0 and run.stdout.startswith("-1 invalid argument"), run.stdout + run.stderr
