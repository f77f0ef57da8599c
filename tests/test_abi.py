"""Host-side checks of liboptima.so: it loads, exports every function that
include/optima.h declares, and its host-only paths (status strings, defaults,
workspace queries, argument validation that returns before any launch)
behave as the header states. No kernel is launched here."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "optima.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(optima_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2512_13886_amd as L
    return ctypes.CDLL(L.library_path())


def test_header_declares_the_four_calls():
    names = _declared_functions()
    for n in ("optima_hessian_accumulate", "optima_hessian_damp", "optima_spectral_norm",
              "optima_qp_solve_batched"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_product_library_has_no_phase_stamps(lib):
    # The clock stamps exist only in the instrumented build (build.py phases);
    # the library the package loads must not carry them.
    import paper_2512_13886_amd as L
    if os.path.basename(L.library_path()) == "liboptima.so":
        assert not hasattr(lib, "optima_phase_stamps")


def test_status_strings_and_version():
    import paper_2512_13886_amd as L
    assert L.optima_abi_version() >= 1
    assert "INVAL" in L.optima_status_string(-1)
    assert "NONFINITE" in L.optima_status_string(-3)
    assert "WORKSPACE" in L.optima_status_string(-4)
    assert "unknown" in L.optima_status_string(42)


def test_default_options_follow_table_8():
    import paper_2512_13886_amd as L
    o = L.SolverOpts.default()
    assert o.max_iters == 100000 and o.check_every == 64
    assert o.eps_rel == pytest.approx(0.01) and o.eps_abs == pytest.approx(0.01)
    assert o.restarts == 1 and o.fixed_iters == 0
    assert o.precision == L.PREC_BF16X3
    assert o.method == L.METHOD_RAPDHG
    assert o.sparse == 1
    assert o.cooperative == 1


def test_workspace_queries():
    import paper_2512_13886_amd as L
    a = L.optima_qp_workspace_bytes(4096, 4096)
    assert a >= 6 * 4096 * 4096 * 4
    assert L.optima_qp_workspace_bytes(4096, 2048) < a
    assert L.optima_qp_workspace_bytes(100, 3) >= 128 * 128 * 4  # padded copy of H
    assert L.optima_qp_workspace_bytes(0, 3) == 0
    h = L.optima_hessian_workspace_bytes(262144, 4096, L.DTYPE_BF16)
    assert h >= 4096 * 65536 * 2
    assert L.optima_hessian_workspace_bytes(10, 4096, 7) == 0
    assert L.optima_spectral_norm_workspace_bytes(4096) >= 2 * 4096 * 4
    assert L.optima_spectral_norm_workspace_bytes(4096, 16) >= 2 * 16 * 4096 * 4
    assert L.optima_spectral_norm_workspace_bytes(4096, 17) == 0
    assert L.optima_spectral_norm_workspace_bytes(4096, 0) == 0
    # The Lanczos basis: one fp32 row of d per step, at most d steps.
    assert L.optima_spectral_lanczos_workspace_bytes(4096, 64) >= 64 * 4096 * 4
    assert L.optima_spectral_lanczos_workspace_bytes(10, 256) < \
        L.optima_spectral_lanczos_workspace_bytes(10, 1) + 10 * 64 * 4 + 4096
    assert L.optima_spectral_lanczos_workspace_bytes(4096, L.LANCZOS_MAX_STEPS + 1) == 0
    assert L.optima_spectral_lanczos_workspace_bytes(4096, 0) == 0
    assert L.SPECTRAL_MAX_BLOCK == 16


def test_validation_returns_before_launch(lib):
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    f = lib.optima_hessian_accumulate
    f.restype = ctypes.c_int
    f.argtypes = [vp, ctypes.c_int, i64, i64, vp, ctypes.c_int, vp, ctypes.c_size_t, vp]
    assert f(None, 0, 10, 8, None, 0, None, 0, None) == -1          # H is NULL
    assert f(None, 9, 10, 8, vp(256), 0, None, 0, None) == -5       # dtype
    assert f(vp(512), 0, 10, 8, vp(1 << 20), 0, None, 0, None) == -4  # no workspace
    q = lib.optima_qp_solve_batched
    q.restype = ctypes.c_int
    q.argtypes = [vp, i64, vp, vp, vp, i64, vp, vp, ctypes.c_size_t, vp, vp, vp, vp]
    assert q(None, 8, None, None, None, 4, None, None, 0, None, None, None, None) == -1
    g = lib.optima_spectral_norm
    g.restype = ctypes.c_int
    g.argtypes = [vp, i64, vp, ctypes.c_int, ctypes.c_int, ctypes.c_float, vp, ctypes.c_size_t,
                  vp, vp, vp]
    assert g(vp(256), 8, vp(512), 1, 0, 1e-6, None, 0, vp(1024), None, None) == -1  # max_iters
    assert g(vp(256), 8, vp(512), 0, 10, 1e-6, None, 0, vp(1024), None, None) == -1  # block
    assert g(vp(256), 8, vp(512), 17, 10, 1e-6, None, 0, vp(1024), None, None) == -1
    assert g(vp(256), 8, vp(512), 4, 10, 1e-6, None, 0, vp(1024), None, None) == -4  # ws


def test_forward_queries_and_validation(lib):
    import paper_2512_13886_amd as L
    assert L.ACT_NONE == 0 and L.ACT_SILU == 1
    b = L.optima_linear_forward_workspace_bytes(1000, 128, 100)
    assert b >= 128 * 128 * 2  # bf16 weights, rows padded to the tile
    assert L.optima_linear_forward_workspace_bytes(1000, 100, 100) == 0   # d_in % 64
    assert L.optima_linear_forward_workspace_bytes(1000, 128, 102) == 0   # d_out % 4
    assert L.optima_linear_forward_workspace_bytes(-1, 128, 100) == 0
    i64, vp, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    f = lib.optima_linear_forward
    f.restype = ctypes.c_int
    f.argtypes = [vp, i64, i64, vp, i64, i32, vp, i32, vp, vp, vp, ctypes.c_size_t, vp]
    X, W, Y = vp(1 << 20), vp(2 << 20), vp(4 << 20)
    assert f(X, 10, 128, None, 8, 0, Y, 1, None, None, None, 0, None) == -1   # W is NULL
    assert f(X, 10, 128, W, 8, 0, None, 1, None, None, None, 0, None) == -1   # nothing to do
    assert f(X, 10, 128, W, 8, 5, Y, 1, None, None, None, 0, None) == -1      # act
    assert f(X, 10, 128, W, 8, 0, Y, 7, None, None, None, 0, None) == -1      # y_dtype
    assert f(X, 10, 128, W, 8, 0, None, 1, Y, None, None, 0, None) == -1      # Y_ref w/o err
    assert f(X, 10, 128, W, 8, 0, None, 1, None, Y, None, 0, None) == -1      # err w/o Y_ref
    assert f(vp((1 << 20) + 8), 10, 128, W, 8, 0, Y, 1, None, None, None, 0, None) == -1  # align
    assert f(X, 10, 128, W, 8, 0, Y, 1, None, None, None, 0, None) == -4      # no workspace


def _header_struct(name):
    """(type, field) pairs of `typedef struct { ... } name;` in the header."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    m = re.search(r"typedef struct\s*\{([^}]*)\}\s*" + name + r"\s*;", text)
    assert m, name
    fields = []
    for decl in m.group(1).split(";"):
        decl = " ".join(decl.split())
        if decl:
            t, f = decl.rsplit(" ", 1)
            if f.startswith("*"):
                t, f = t + "*", f[1:]
            fields.append((t, f))
    return fields


@pytest.mark.parametrize("c_name,py_name", [("optima_solver_opts", "_Opts"),
                                            ("optima_solve_stats", "_Stats"),
                                            ("optima_solve_info", "_Info")])
def test_binding_structs_mirror_the_header(c_name, py_name):
    # The ctypes structs of the binding list the header's fields in order,
    # with the same C types (the library's ABI version pins this layout).
    from paper_2512_13886_amd import _lib
    ctype = {"int64_t": ctypes.c_int64, "int32_t": ctypes.c_int32, "float": ctypes.c_float,
             "double": ctypes.c_double}
    header = _header_struct(c_name)
    mirror = getattr(_lib, py_name)._fields_
    assert [f for _, f in header] == [f for f, _ in mirror]
    for (t, f), (_, pt) in zip(header, mirror):
        if t.endswith("*"):
            assert pt is ctypes.c_void_p, f
        else:
            assert pt is ctype[t], (f, t)
